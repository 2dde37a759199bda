// INT8 projection GEMMs with a fused fixed-point requantization epilogue.
//
// Every linear layer of the block (Q, K, V, the relative-position projection and
// the output projection) is Eq. 7: an int8 x int8 product accumulated in int32,
// rescaled by a per-output-channel multiplier m and a right shift n with round to
// nearest (ties up), and clamped to the symmetric int8 grid.
//
// Kernel shape: one 256-thread workgroup computes a TN (channels) x TM (tokens) tile
// with v_mfma_i32_32x32x32_i8; the four waves form a 2 x 2 grid of (TN/2) x (TM/2)
// sub-tiles.  K advances in 128-byte steps, so every global row segment is a whole
// cache line; the next step is fetched into registers while the current one is
// multiplied out of LDS.  LDS rows are 128 bytes with the eight 16-byte chunks
// XOR-swizzled by the row index, which keeps both the 16-byte stores of the fetch
// and the 16-byte MFMA operand reads free of bank conflicts.
//
// Token tiles never straddle two utterances (each utterance is tiled on its own), so
// every destination layout receives whole aligned 16-byte pieces.  Tiles are dealt
// to the eight XCDs in contiguous, roughly square groups of the tile grid, so the
// operand rows one XCD touches fit its L2.
//
// Epilogue: the requantization y = clamp8(floor((acc m + 2^(n-1)) / 2^n)) is
// evaluated exactly in float64 as floor(acc * (m 2^-n) + 128.5) clamped to [1, 255],
// the biased code y + 128: |acc m| < 2^51, so acc * (m 2^-n) + 128.5 is a multiple of
// 2^-n below 2^52 units and the fused multiply-add is exact.  Each lane then owns 4
// consecutive outputs per accumulator group; one exchange with the lane 32 away gives
// it 16 consecutive bytes, stored with one 16-byte write.  Channel-major V^T is
// produced by swapping the MFMA operands in the waves whose channels are V, so that
// its 16-byte pieces run along tokens.
#include <type_traits>

#include "ipk_internal.h"

namespace ipk {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

enum OutMode { OUT_QKV = 0, OUT_POS = 1, OUT_ROWMAJOR = 2 };

struct GemmProblem {
  const int8_t* x;      // [nb][rows][K] activations
  const int8_t* w;      // [N][K] weights
  const double* scale;  // [N] m * 2^-n per output channel
  int nb, rows, N, K;
  int mode;
  int tile_begin;   // first logical tile of this problem
  int tiles_n;      // tiles along N
  int tiles_m_per;  // token tiles per utterance
  int band;         // token tiles per band of the logical order
};

struct GemmArgs {
  GemmProblem prob[2];
  int nprob;
  int tiles_total;
  int per_xcd;  // logical tiles dealt to each XCD
  int8_t *q, *k, *vt, *p, *y;
  int T_al, H, DK, d, p_rows, p_base;
};

constexpr int BK = 128;  // bytes of K per step
constexpr int BUF_WORD3 = 0x00020000;  // buffer resource word 3 for gfx9-family raw loads

// Byte offset of 16-byte chunk c of LDS row r.  Rows are 128 bytes; the chunk index
// is XORed with (r ^ r/8) mod 8, so any 16 consecutive rows (16-row aligned) that
// read one logical chunk touch 16 distinct (row parity, chunk) bank groups.
__device__ __forceinline__ int lds_off(int r, int c) { return r * BK + ((c ^ ((r ^ (r >> 3)) & 7)) << 4); }

// biased code y + 128 of one accumulator (exact, see the header comment)
__device__ __forceinline__ uint32_t requant_code(int acc, double scale) {
  const double t = __builtin_fma((double)acc, scale, 128.5);
  return (uint32_t)(int)__builtin_fmin(__builtin_fmax(t, 1.0), 255.0);
}

// four biased codes -> four int8 bytes (code - 128 == code ^ 0x80 for code in [1, 255])
__device__ __forceinline__ uint32_t pack4(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3) {
  return (c0 | (c1 << 8) | (c2 << 16) | (c3 << 24)) ^ 0x80808080u;
}

template <int TN, int TM>
__global__ __launch_bounds__(256) void gemm_i8_requant(GemmArgs args) {
  constexpr int FN = TN / 64;               // 32-row MFMA tiles per wave along N
  constexpr int FM = TM / 64;               // 32-col MFMA tiles per wave along M
  constexpr int LW = TN * (BK / 16) / 256;  // 16-byte global loads per thread, W tile
  constexpr int LX = TM * (BK / 16) / 256;  // same for the X tile
  __shared__ __align__(16) int8_t sw[TN * BK];
  __shared__ __align__(16) int8_t sx[TM * BK];
  __shared__ double ssc[TN];

  // XCD-aware deal: workgroup i runs on XCD i % 8; XCD x owns logical tiles
  // [x * per_xcd, (x + 1) * per_xcd)
  const int lin = blockIdx.x;
  const int tile = (lin & 7) * args.per_xcd + (lin >> 3);
  if (tile >= args.tiles_total) return;
  const int pi = (args.nprob > 1 && tile >= args.prob[1].tile_begin) ? 1 : 0;
  const GemmProblem& P = args.prob[pi];
  // logical order inside a problem: bands of `band` token tiles, channels outer,
  // tokens inner within a band
  const int local = tile - P.tile_begin;
  const int tiles_m = P.nb * P.tiles_m_per;
  const int band_idx = local / (P.band * P.tiles_n);
  const int in_band = local - band_idx * P.band * P.tiles_n;
  const int band_m = min(P.band, tiles_m - band_idx * P.band);
  const int nt = in_band / band_m;
  const int mt = band_idx * P.band + (in_band - nt * band_m);
  const int n0 = nt * TN;
  const int ub = mt / P.tiles_m_per;               // utterance
  const int t0 = (mt - ub * P.tiles_m_per) * TM;   // first token of the tile
  const int K = P.K, rows = P.rows;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave & 1, wm = wave >> 1;

  if (tid < TN) ssc[tid] = P.scale[min(n0 + tid, P.N - 1)];

  // thread -> (row, chunk) of the fetch: 8 threads cover one 128-byte row segment.
  // Raw buffer loads: rows past the end of the operand (their whole offset is in the
  // per-lane operand, which the bounds check covers) read as zeros.
  const int fchunk = tid & 7, frow = tid >> 3;  // rows frow + 32 r
  const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(P.w + (size_t)n0 * K), (short)0, (P.N - n0) * K, BUF_WORD3);
  const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(P.x + ((size_t)ub * rows + t0) * K), (short)0, (rows - t0) * K, BUF_WORD3);
  const int foff = frow * K + fchunk * 16;

  v4i rw[LW], rx[LX];
  // K is a multiple of 64: the last step of an odd multiple fills its upper half with zeros
  auto fetch = [&](int k0) {
    if (k0 + fchunk * 16 < K) {
#pragma unroll
      for (int r = 0; r < LW; ++r)
        rw[r] = (v4i)__builtin_amdgcn_raw_buffer_load_b128(wres, foff + 32 * r * K + k0, 0, 0);
#pragma unroll
      for (int r = 0; r < LX; ++r)
        rx[r] = (v4i)__builtin_amdgcn_raw_buffer_load_b128(xres, foff + 32 * r * K + k0, 0, 0);
    } else {
#pragma unroll
      for (int r = 0; r < LW; ++r) rw[r] = (v4i){};
#pragma unroll
      for (int r = 0; r < LX; ++r) rx[r] = (v4i){};
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int r = 0; r < LW; ++r) *(v4i*)(sw + lds_off(frow + 32 * r, fchunk)) = rw[r];
#pragma unroll
    for (int r = 0; r < LX; ++r) *(v4i*)(sx + lds_off(frow + 32 * r, fchunk)) = rx[r];
  };

  // waves whose channels are V produce the transposed product (tokens along MFMA rows)
  const int nw0 = n0 + wn * (TN / 2);
  const bool vwave = P.mode == OUT_QKV && nw0 >= 2 * args.d;

  v16i acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = (v16i){};

  // operand fragments: lane l reads row (l % 32), 16 bytes at k = 32 ks + 16 (l / 32)
  const int frag_row = lane & 31, half = lane >> 5;
  const int nk = (K + BK - 1) / BK;
  // the K loop, instantiated once per operand order so that the order is not a
  // branch inside it
  auto kloop = [&](auto swap_tag) {
    constexpr bool SWAP = decltype(swap_tag)::value;
    fetch(0);
    for (int kt = 0; kt < nk; ++kt) {
      stash();
      __syncthreads();
      if (kt + 1 < nk) fetch((kt + 1) * BK);
#pragma unroll
      for (int ks = 0; ks < BK / 32; ++ks) {
        v4i af[FN], bf[FM];
#pragma unroll
        for (int i = 0; i < FN; ++i)
          af[i] = *(const v4i*)(sw + lds_off(wn * (TN / 2) + i * 32 + frag_row, 2 * ks + half));
#pragma unroll
        for (int j = 0; j < FM; ++j)
          bf[j] = *(const v4i*)(sx + lds_off(wm * (TM / 2) + j * 32 + frag_row, 2 * ks + half));
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
          for (int j = 0; j < FM; ++j)
            acc[i][j] = SWAP ? __builtin_amdgcn_mfma_i32_32x32x32_i8(bf[j], af[i], acc[i][j], 0, 0, 0)
                             : __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
      }
      __syncthreads();
    }
  };
  if (vwave) kloop(std::true_type{});
  else kloop(std::false_type{});

  // Epilogue.  Accumulator g * 4 + e of a lane sits at MFMA row g * 8 + half * 4 + e
  // and column lane % 32.  After requantization each lane holds dwords D[g] (4 rows);
  // trading D[2], D[3] of the low half for D[0], D[1] of the high half gives the low
  // half rows 0..15 and the high half rows 16..31, 16 bytes each.
  const int col = lane & 31;
  const int tw0 = t0 + wm * (TM / 2);
#pragma unroll
  for (int i = 0; i < FN; ++i) {
    const int nl = wn * (TN / 2) + i * 32;  // first channel of this sub-tile, tile-local
#pragma unroll
    for (int j = 0; j < FM; ++j) {
      uint32_t D[4];
      if (vwave) {
        // rows are tokens, the column is the channel
        const double sc = ssc[nl + col];
#pragma unroll
        for (int g = 0; g < 4; ++g)
          D[g] = pack4(requant_code(acc[i][j][g * 4 + 0], sc), requant_code(acc[i][j][g * 4 + 1], sc),
                       requant_code(acc[i][j][g * 4 + 2], sc), requant_code(acc[i][j][g * 4 + 3], sc));
      } else {
        // rows are channels, the column is the token
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int c = nl + g * 8 + half * 4;
          D[g] = pack4(requant_code(acc[i][j][g * 4 + 0], ssc[c]), requant_code(acc[i][j][g * 4 + 1], ssc[c + 1]),
                       requant_code(acc[i][j][g * 4 + 2], ssc[c + 2]), requant_code(acc[i][j][g * 4 + 3], ssc[c + 3]));
        }
      }
      const uint32_t s0 = __shfl_xor(half ? D[0] : D[2], 32);
      const uint32_t s1 = __shfl_xor(half ? D[1] : D[3], 32);
      v4i out;
      if (half == 0) out = (v4i){(int)D[0], (int)s0, (int)D[1], (int)s1};
      else out = (v4i){(int)s0, (int)D[2], (int)s1, (int)D[3]};

      if (vwave) {
        // 16 consecutive tokens of channel n; tokens up to the next multiple of 16
        // stay inside the padded key range of V^T
        const int n = n0 + nl + col;
        const int t = tw0 + j * 32 + half * 16;
        if (n < P.N && t < rows) {
          const int c = n - 2 * args.d;
          const int h = c / args.DK, kk = c - h * args.DK;
          int8_t* base = args.vt + ((size_t)ub * args.H + h) * args.T_al * args.DK;
          *(v4i*)(base + vt_index(t, kk, args.DK)) = out;
        }
      } else {
        // 16 consecutive channels of token t
        const int n = n0 + nl + half * 16;
        const int t = tw0 + j * 32 + col;
        if (n < P.N && t < rows) {
          if (P.mode == OUT_QKV) {
            const int which = n / args.d;
            const int c = n - which * args.d;
            const int h = c / args.DK, kk = c - h * args.DK;
            int8_t* base = (which == 0 ? args.q : args.k) + ((size_t)ub * args.H + h) * args.T_al * args.DK;
            *(v4i*)(base + frag_index(t, kk, args.DK)) = out;
          } else if (P.mode == OUT_POS) {
            const int h = n / args.DK, kk = n - h * args.DK;
            *(v4i*)(args.p + (size_t)h * args.p_rows * args.DK + frag_index(args.p_base + t, kk, args.DK)) = out;
          } else {
            *(v4i*)(args.y + ((size_t)ub * rows + t) * P.N + n) = out;
          }
        }
      }
    }
  }
}

static int add_problem(GemmArgs& a, int idx, const int8_t* x, const int8_t* w, const double* scale, int nb,
                       int rows, int N, int K, int mode, int tile_begin, int TN, int TM) {
  GemmProblem& p = a.prob[idx];
  p.x = x;
  p.w = w;
  p.scale = scale;
  p.nb = nb;
  p.rows = rows;
  p.N = N;
  p.K = K;
  p.mode = mode;
  p.tile_begin = tile_begin;
  p.tiles_n = (N + TN - 1) / TN;
  p.tiles_m_per = (rows + TM - 1) / TM;
  const int tiles_m = nb * p.tiles_m_per;
  const int tiles = p.tiles_n * tiles_m;
  // band height: an XCD's share of about tiles/8 tiles covers ~band token tiles and
  // ~share/band channel tiles; weight rows per channel tile (TN) are worth TN/TM
  // token tiles, so the square in bytes has band ~ sqrt(share * TN / TM)
  const double share = (tiles + 7) / 8;
  const int band = (int)(sqrt(share * TN / TM) + 0.5);
  p.band = band < 1 ? 1 : (band > tiles_m ? tiles_m : band);
  return tiles;
}

static void fill_dest(GemmArgs& a, const RunShape& rs, const Workspace& ws, int8_t* y) {
  a.q = ws.q;
  a.k = ws.k;
  a.vt = ws.vt;
  a.p = ws.p;
  a.y = y;
  a.T_al = rs.T_al;
  a.H = rs.H;
  a.DK = rs.DK;
  a.d = rs.d;
  a.p_rows = p_rows(rs.T_al);
  a.p_base = rs.p_base;
}

template <int TN, int TM>
static hipError_t launch_gemm(GemmArgs& a, int tiles, hipStream_t st, const LaunchEv& ev) {
  a.tiles_total = tiles;
  a.per_xcd = (tiles + 7) / 8;
  return launch_kernel(gemm_i8_requant<TN, TM>, dim3(8 * a.per_xcd), dim3(256), 0, st, ev, a);
}

hipError_t launch_projections(const RunShape& rs, const Weights& w, const Workspace& ws, const int8_t* x,
                              const int8_t* pos_table, hipStream_t st, const LaunchEv& ev) {
  GemmArgs a{};
  fill_dest(a, rs, ws, nullptr);
  constexpr int TN = 256, TM = 128;
  int tiles = add_problem(a, 0, x, w.w_qkv, w.scale_qkv, rs.B, rs.T, 3 * rs.d, rs.d, OUT_QKV, 0, TN, TM);
  tiles += add_problem(a, 1, pos_table, w.w_pos, w.scale_pos, 1, 2 * rs.T - 1, rs.d, rs.d, OUT_POS, tiles, TN, TM);
  a.nprob = 2;
  return launch_gemm<TN, TM>(a, tiles, st, ev);
}

hipError_t launch_out_projection(const RunShape& rs, const Weights& w, const Workspace& ws, int8_t* y,
                                 hipStream_t st, const LaunchEv& ev) {
  GemmArgs a{};
  fill_dest(a, rs, ws, y);
  constexpr int TN = 128, TM = 64;
  int tiles = add_problem(a, 0, ws.ctx, w.w_out, w.scale_out, rs.B, rs.T, rs.d, rs.d, OUT_ROWMAJOR, 0, TN, TM);
  a.nprob = 1;
  return launch_gemm<TN, TM>(a, tiles, st, ev);
}

}  // namespace ipk
