// INT8 projection GEMMs with a fused fixed-point requantization epilogue.
//
// Every linear layer of the block (Q, K, V, the relative-position projection and
// the output projection) is Eq. 7: an int8 x int8 product accumulated in int32,
// rescaled by a per-output-channel multiplier m and a right shift n with round to
// nearest (ties up), and clamped to the symmetric int8 grid.
//
// Kernel shape: one workgroup of WN x WM waves computes a TN (channels) x TM (tokens)
// tile with v_mfma_i32_32x32x32_i8; the waves form a WN x WM grid of (TN/WN) x (TM/WM)
// sub-tiles.  K advances in 128-byte steps, so every global row segment is a whole
// cache line.  The weights are stored in MFMA operand-fragment order (each 32-channel x
// 32-byte fragment a contiguous 1 KB block in lane order), so every wave loads its own
// weight fragments straight into registers with fully coalesced 16-byte loads, one K
// step ahead.  The token tile is fetched into registers one step ahead (two for the
// small output-projection tiles) and staged in LDS, whose rows are 128 bytes with the eight 16-byte chunks XOR-swizzled by the row
// index, which keeps both the 16-byte stores of the fetch and the 16-byte MFMA operand
// reads free of bank conflicts.
//
// The large projections use 256 x 256 tiles of eight waves (two per SIMD, 64 channels x
// 128 tokens each, accumulators in VGPRs).  Per K step a workgroup then moves 32 KB of
// token tile and 128 KB of token fragments through LDS and streams 64 KB of weight
// fragments (each block read by the two waves that share its channels); with both
// operands staged in LDS the step moved 256 KB through LDS and ran about 17 % slower.
//
// Token tiles never straddle two utterances (each utterance is tiled on its own), so
// every destination layout receives whole aligned 16-byte pieces.  Tiles are dealt
// to the eight XCDs in contiguous, roughly square groups of the tile grid, so the
// operand rows one XCD touches fit its L2.
//
// Epilogue: the requantization y = clamp8(floor((acc m + 2^(n-1)) / 2^n)) in integers.
// When every channel of the matrix allows it (n <= 16, m' = m 2^(16-n) < 2^23 and
// one clamp bound A for all channels, at least ceil(2^23 / m') + 1 for each, with
// A m' + 2^15 < 2^31), the accumulator is first clamped to [-A, A] (beyond a channel's
// own bound the result saturates anyway), then one 24-bit multiply-add gives
// t = a m' + 2^15, whose clamp to [-127 2^16, 127 2^16 + 2^16 - 1] holds the int8
// result in byte 2: three full-rate instructions per value, one multiplier register per
// value, and a byte permute gathers four results into a dword.  Otherwise the value
// is evaluated in 64-bit integers, its constants read from LDS per value.  Each lane owns 4 consecutive outputs per accumulator group; one
// exchange with the lane 32 away gives it 16 consecutive bytes, stored with one 16-byte
// write.  Channel-major V^T is produced by swapping the MFMA operands in the waves whose
// channels are V, so that its 16-byte pieces run along tokens.
#include <type_traits>
#include <utility>

#include "ipk_internal.h"

namespace ipk {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

enum OutMode { OUT_QKV = 0, OUT_POS = 1, OUT_ROWMAJOR = 2 };
// Epilogues of row-major outputs: the requantized int8 values themselves, the residual
// add of Eq. 2 (with z1 laid out as the output), or the integer Swish of Eq. 12 and
// its requantization, applied through a 256-entry table indexed by the biased code.
enum Epilogue { EPI_PLAIN = 0, EPI_RESID = 1, EPI_SWISH = 2 };

struct GemmProblem {
  const int8_t* x;      // [nb][rows][K] activations
  const int8_t* w;      // [N][K] weights
  const int32_t* req;   // [2][N] per output channel: multiplier, and shift in the wide form (Requant)
  int wide;             // 64-bit evaluation
  int clamp;            // the fast form's clamp bound
  int nb, rows, N, K;
  int mode;
  int tile_begin;   // first logical tile of this problem
  int tiles_n;      // tiles along N
  int tiles_m_per;  // token tiles per utterance
  int band;         // token tiles per band of the logical order
  DivU dv_band_span, dv_band, dv_last_band, dv_tiles_m_per;  // divisors of the tile decomposition
};

struct GemmArgs {
  GemmProblem prob[2];
  int nprob;
  int tiles_total;
  int per_xcd;  // logical tiles dealt to each XCD
  int8_t *q, *k, *vt, *p, *y;
  int T_al, H, dk_shift, d, p_rows, p_base;  // d_k = 2^dk_shift
  // residual add of the MHSA module (row-major outputs only): y := clamp8(RS(m_z z1 +
  // m_y y, 1, shift_r)) with z1 laid out as y
  const int8_t* z1;
  int m_z, m_y, shift_r;
  const uint8_t* swtab;  // EPI_SWISH: output byte of each biased code h + 128
};

constexpr int BK = 128;  // bytes of K per step

// Byte offset of 16-byte chunk c of LDS row r.  Rows are 128 bytes; the chunk index
// is XORed with (r ^ r/8) mod 8, so any 16 consecutive rows (16-row aligned) that
// read one logical chunk touch 16 distinct (row parity, chunk) bank groups.
__device__ __forceinline__ int lds_off(int r, int c) { return r * BK + ((c ^ ((r ^ (r >> 3)) & 7)) << 4); }

// f(integral_constant<int, 0>), ..., f(integral_constant<int, N - 1>), in order
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// byte 2 of four words -> one dword (v_perm_b32 selector bytes: 0-3 pick the second
// operand's bytes, 4-7 the first's, 0x0c a zero byte)
__device__ __forceinline__ uint32_t pack_b2(uint32_t v0, uint32_t v1, uint32_t v2, uint32_t v3) {
  return __builtin_amdgcn_perm(v1, v0, 0x0c0c0602u) | __builtin_amdgcn_perm(v3, v2, 0x06020c0cu);
}

// v_med3_i32 with the low bound in a scalar register and the high one in a vector
// register (the compiler forms med3 from min/max only with constant bounds)
__device__ __forceinline__ int med3_sv(int x, int lo, int hi) {
  int r;
  asm("v_med3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "s"(lo), "v"(hi));
  return r;
}

// a b + c for a, b in the signed 24-bit range (v_mad_i32_i24; the compiler cannot
// see the range of a clamp to runtime bounds and would sign-extend both first)
__device__ __forceinline__ int mad24_s(int a, int b, int c) {
  int r;
  asm("v_mad_i32_i24 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "s"(c));
  return r;
}

// Eq. 7 on the 16 accumulators of one MFMA output block, fast form: m[e] is element
// e's multiplier m', -A and A (negA, Av) the matrix's clamp bounds; v[e] receives the
// int8 result in byte 2.
__device__ __forceinline__ void requant16_fast(const v16i& a, const int (&m)[16], int negA, int Av, int (&v)[16]) {
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int c = med3_sv(a[e], negA, Av);
    v[e] = min(max(mad24_s(c, m[e], 1 << 15), -127 * 65536), 127 * 65536 + 65535);
  }
}

// The wide form: element e's multiplier and shift are sm[ch(e)], sn[ch(e)] (LDS).
template <typename CH>
__device__ __forceinline__ void requant16_wide(const v16i& a, const int* sm, const int* sn, CH ch, int (&v)[16]) {
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int m = sm[ch(e)], n = sn[ch(e)];
    const long long q = ((long long)a[e] * m + (1ll << (n - 1))) >> n;
    v[e] = (int)(q < -127 ? -127 : (q > 127 ? 127 : q)) << 16;
  }
}

// The 16 results (byte 2 of v[e]) packed four per dword: D[g] holds elements 4g .. 4g + 3.
// With SW, each int8 result h goes through the Swish table `stab` (LDS, indexed by h + 128).
template <bool SW = false>
__device__ __forceinline__ void pack16(const int (&v)[16], uint32_t (&D)[4], const uint8_t* stab = nullptr) {
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    if constexpr (SW) {
      uint32_t o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = stab[(((uint32_t)v[4 * g + e] >> 16) & 0xffu) ^ 0x80u];
      D[g] = o[0] | (o[1] << 8) | (o[2] << 16) | (o[3] << 24);
    } else {
      D[g] = pack_b2((uint32_t)v[4 * g], (uint32_t)v[4 * g + 1], (uint32_t)v[4 * g + 2], (uint32_t)v[4 * g + 3]);
    }
  }
}

// The residual add of Eq. 2 on 16 int8 pairs: clamp8(floor((m_z z + m_y y + 2^(n-1)) / 2^n)).
// m_z z + m_y y is exact in int32 (multipliers below 2^23, |z|, |y| <= 128); the
// rounding term and the shift (n <= 40) need 64 bits.
__device__ __forceinline__ v4i residual16(const v4i& y, const v4i& z, int m_z, int m_y, int shift) {
  const long long half = 1ll << (shift - 1);
  v4i r;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t o = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int yb = (y[w] << (24 - 8 * b)) >> 24, zb = (z[w] << (24 - 8 * b)) >> 24;
      const long long q = ((long long)(m_z * zb + m_y * yb) + half) >> shift;
      o |= ((uint32_t)(int)min(max(q, -127ll), 127ll) & 0xFFu) << (8 * b);
    }
    r[w] = (int)o;
  }
  return r;
}

// WN x WM waves (NWAVE = WN WM) each own a (TN/WN) x (TM/WM) sub-tile.  The weights
// come pre-packed in MFMA fragment order (wfrag_index): each wave streams its own
// fragments from memory straight into registers, one K step ahead, and only the token
// tile goes through LDS.  EPI: the epilogue of row-major outputs.  TPF: register sets of
// the token tile in flight (2 fetches each step's tile two steps before it is stored, for
// long K loops whose operands come from beyond the L2).  WIDE: some problem of the
// launch takes the wide form of Eq. 7 (its code costs registers even where unused, so
// launches in the fast form alone leave it out).
template <int TN, int TM, int NWAVE, int WN, int EPI, int TPF, bool WIDE>
__global__ __launch_bounds__(64 * NWAVE) void gemm_i8_requant(GemmArgs args) {
  constexpr int NTH = 64 * NWAVE;
  constexpr int WM = NWAVE / WN;            // waves along M
  constexpr int WTN = TN / WN;              // channels per wave
  constexpr int WTM = TM / WM;              // tokens per wave
  constexpr int FN = WTN / 32;              // 32-row MFMA tiles per wave along N
  constexpr int FM = WTM / 32;              // 32-col MFMA tiles per wave along M
  constexpr int LX = TM * (BK / 16) / NTH;  // 16-byte global loads per thread of the token tile
  constexpr int FROWS = NTH / 8;            // rows one pass of the fetch covers
  constexpr int KSL = BK / 32;              // 32-byte K slices per step
  static_assert(FN >= 1 && FM >= 1 && LX >= 1 && WTM % 32 == 0 && NTH >= TN && NWAVE % WN == 0, "tile shape");
  // two LDS buffers: the next K step is stored while the current one is multiplied
  __shared__ __align__(16) int8_t sx[2][TM * BK];
  __shared__ __align__(16) int sreq[2][TN];  // Eq. 7 constants of the tile's channels
  __shared__ uint32_t stab32[EPI == EPI_SWISH ? 64 : 1];  // the Swish table (read after the K loop)

  // XCD-aware deal: workgroup i runs on XCD i % 8; XCD x owns logical tiles
  // [x * per_xcd, (x + 1) * per_xcd)
  const int lin = blockIdx.x;
  const int tile = (lin & 7) * args.per_xcd + (lin >> 3);
  if (tile >= args.tiles_total) return;
  const int pi = (args.nprob > 1 && tile >= args.prob[1].tile_begin) ? 1 : 0;
  const GemmProblem& P = args.prob[pi];
  // the problem's scalars, all loaded at once: left alone the compiler loads each one
  // where it is first used, and every division below would wait for its own load
  int tile_begin = P.tile_begin, nb = P.nb, tiles_m_per = P.tiles_m_per, band = P.band, tiles_n = P.tiles_n;
  uint32_t m_span = P.dv_band_span.m, m_band = P.dv_band.m, m_last = P.dv_last_band.m, m_tmp = P.dv_tiles_m_per.m;
  int K = P.K, rows = P.rows, N = P.N, mode = P.mode;
  asm volatile(""
               : "+s"(tile_begin), "+s"(nb), "+s"(tiles_m_per), "+s"(band), "+s"(tiles_n), "+s"(m_span), "+s"(m_band),
                 "+s"(m_last), "+s"(m_tmp), "+s"(K), "+s"(rows), "+s"(N), "+s"(mode));
  // logical order inside a problem: bands of `band` token tiles, channels outer,
  // tokens inner within a band
  const int local = tile - tile_begin;
  const int tiles_m = nb * tiles_m_per;
  const int band_idx = (int)div_u(local, DivU{0u, m_span});
  const int in_band = local - band_idx * band * tiles_n;
  const int band_m = min(band, tiles_m - band_idx * band);
  const int nt = (int)div_u(in_band, DivU{0u, band_m == band ? m_band : m_last});
  const int mt = band_idx * band + (in_band - nt * band_m);
  const int n0 = nt * TN;
  const int ub = (int)div_u(mt, DivU{0u, m_tmp});  // utterance
  const int t0 = (mt - ub * tiles_m_per) * TM;      // first token

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave % WN, wm = wave / WN;

  if (tid < TN) {
    const int c = min(n0 + tid, N - 1);
    sreq[0][tid] = P.req[c];
    sreq[1][tid] = P.req[N + c];
  }
  const int rq_wide = WIDE ? __builtin_amdgcn_readfirstlane(P.wide) : 0, rq_clamp = __builtin_amdgcn_readfirstlane(P.clamp);
  if (EPI == EPI_SWISH && tid < 64) stab32[tid] = ((const uint32_t*)args.swtab)[tid];

  // thread -> (row, chunk) of the fetch: 8 threads cover one 128-byte row segment.
  // Raw buffer loads: rows past the end of the operand (their whole offset is in the
  // per-lane operand, which the bounds check covers) read as zeros.
  const int fchunk = tid & 7, frow = tid >> 3;  // rows frow + FROWS r
  const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc((void*)P.w, (short)0, N * K, BUF_WORD3);
  const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(P.x + ((size_t)ub * rows + t0) * K), (short)0, (rows - t0) * K, BUF_WORD3);
  const int foff = frow * K + fchunk * 16;

  // the next step's token tile in registers
  static_assert(TPF == 1 || TPF == 2, "token prefetch depth");
  v4i rx[TPF][LX];
  // this wave's weight fragments of one K step (FN channel blocks x KSL slices, 1 KB
  // each, the slices of a block contiguous), two steps in registers.  A slice past K
  // (odd multiples of 64) meets zero tokens, so its contents do not matter; reads past
  // the matrix return zeros.
  v4i wf[2][FN][KSL];
  const int cb0 = (n0 + wn * WTN) >> 5;  // first 32-channel block of this wave
  auto wfetch = [&](int kt, auto set_tag) {
    constexpr int SET = decltype(set_tag)::value;
#pragma unroll
    for (int i = 0; i < FN; ++i) {
      const int base = __builtin_amdgcn_readfirstlane(((cb0 + i) * (K >> 5) + kt * KSL) * 1024);
#pragma unroll
      for (int ks = 0; ks < KSL; ++ks)
        wf[SET][i][ks] = (v4i)__builtin_amdgcn_raw_buffer_load_b128(wres, lane * 16 + ks * 1024, base, 0);
    }
  };
  // K is a multiple of 64: the last step of an odd multiple fills its upper half with zeros
  auto fetch = [&](int k0, int set) {
    if (k0 + fchunk * 16 < K) {
#pragma unroll
      for (int r = 0; r < LX; ++r)
        rx[set][r] = (v4i)__builtin_amdgcn_raw_buffer_load_b128(xres, foff + FROWS * r * K + k0, 0, 0);
    } else {
#pragma unroll
      for (int r = 0; r < LX; ++r) rx[set][r] = (v4i){};
    }
  };
  auto stash = [&](int buf, int set) {
#pragma unroll
    for (int r = 0; r < LX; ++r) *(v4i*)(sx[buf] + lds_off(frow + FROWS * r, fchunk)) = rx[set][r];
  };

  // waves whose channels are V produce the transposed product (tokens along MFMA rows)
  const int nw0 = n0 + wn * WTN;
  const bool vwave = mode == OUT_QKV && nw0 >= 2 * args.d;

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
    auto mma = [&](const int buf, auto wset_tag) {
      constexpr int WSET = decltype(wset_tag)::value;
#pragma unroll
      for (int ks = 0; ks < KSL; ++ks) {
        v4i bf[FM];
#pragma unroll
        for (int j = 0; j < FM; ++j)
          bf[j] = *(const v4i*)(sx[buf] + lds_off(wm * WTM + j * 32 + frag_row, 2 * ks + half));
#pragma unroll
        for (int i = 0; i < FN; ++i)
#pragma unroll
          for (int j = 0; j < FM; ++j)
            acc[i][j] = SWAP ? __builtin_amdgcn_mfma_i32_32x32x32_i8(bf[j], wf[WSET][i][ks], acc[i][j], 0, 0, 0)
                             : __builtin_amdgcn_mfma_i32_32x32x32_i8(wf[WSET][i][ks], bf[j], acc[i][j], 0, 0, 0);
      }
    };
    // step k is multiplied out of LDS buffer k % 2 (and weight set k % 2) while step
    // k + 1 (fetched into token set (k + 1) % TPF, TPF steps earlier) is stored into the
    // other buffer; one barrier per step orders both.  Unrolled twice so that the weight
    // and token sets are static.
    wfetch(0, std::integral_constant<int, 0>{});
    fetch(0, 0);
    stash(0, 0);
    if (nk > 1) {
      fetch(BK, 1 % TPF);
      wfetch(1, std::integral_constant<int, 1>{});
    }
    if (TPF == 2 && nk > 2) fetch(2 * BK, 0);
    __syncthreads();
    for (int kt = 0; kt < nk; kt += 2) {
      static_for<2>([&](auto ph) {
        constexpr int P2 = decltype(ph)::value;  // (kt + P2) % 2
        if (kt + P2 < nk) {
          mma(P2, ph);
          if (kt + P2 + 1 < nk) {
            stash(P2 ^ 1, (P2 + 1) % TPF);
            if (kt + P2 + 1 + TPF < nk) fetch((kt + P2 + 1 + TPF) * BK, (P2 + 1) % TPF);
            if (kt + P2 + 2 < nk) wfetch(kt + P2 + 2, ph);
          }
          __syncthreads();
        }
      });
    }
  };
  if (vwave) kloop(std::true_type{});
  else kloop(std::false_type{});

  // Epilogue.  Accumulator g * 4 + e of a lane sits at MFMA row g * 8 + half * 4 + e
  // and column lane % 32.  After requantization each lane holds dwords D[g] (4 rows);
  // v_permlane32_swap trades the low half's D[2], D[3] for the high half's D[0], D[1],
  // which leaves the low half with rows 0..15 and the high half with rows 16..31 of
  // its column, 16 bytes each.  A 32-channel sub-tile never straddles N, a head or the
  // Q/K/V boundary (N and d_k are multiples of 64), so its destination is uniform.
  //
  // V^T is written up to T_al, so the padded keys hold zeros (a wave's WTM tokens are
  // WTM / 64 whole 64-key blocks of V^T, two 32-token MFMA columns each).
  const int col = lane & 31;
  const int tw0 = t0 + wm * WTM;
  // the epilogue's arguments, loaded together (one wait, not one per first use)
  int8_t *o_q = args.q, *o_k = args.k, *o_vt = args.vt, *o_p = args.p, *o_y = args.y;
  const int8_t* o_z1 = args.z1;
  int o_T_al = args.T_al, o_H = args.H, o_d = args.d, o_prows = args.p_rows, o_pbase = args.p_base, dks = args.dk_shift;
  asm volatile(""
               : "+s"(o_q), "+s"(o_k), "+s"(o_vt), "+s"(o_p), "+s"(o_y), "+s"(o_z1), "+s"(o_T_al), "+s"(o_H), "+s"(o_d),
                 "+s"(o_prows), "+s"(o_pbase), "+s"(dks));
  const int DK = 1 << dks, DKm = DK - 1;
  const size_t head_bytes = (size_t)o_T_al << dks;  // one (utterance, head) block of Q, K or V^T
  // frag_index / vt_index with d_k = 2^dks
  auto frag_off = [&](int row, int kk) {
    return ((size_t)(row >> 4) << (dks + 4)) + (size_t)((kk >> 6) << 10) + (((((kk >> 4) & 3) << 4) + (row & 15)) << 4) +
           (kk & 15);
  };
  auto vt_off = [&](int t, int kk) {
    return ((size_t)(t >> 6) << (dks + 6)) + (size_t)((kk >> 4) << 10) + (((((t >> 4) & 3) << 4) + (kk & 15)) << 4) +
           (t & 15);
  };
#pragma unroll
  for (int i = 0; i < FN; ++i) {
    const int nl = wn * WTN + i * 32;  // first channel of this sub-tile, tile-local
    const int nb = n0 + nl;
    if (nb >= N) continue;
    int8_t* dst;
    const int8_t* zsrc = nullptr;  // residual input, laid out as dst (row-major mode)
    int kk = 0;  // channel of the sub-tile's first row inside its head
    int hd = 0;  // its head
    if (mode == OUT_QKV) {
      const int which = (nb >= o_d) + (nb >= 2 * o_d);
      const int c = nb - which * o_d;
      hd = c >> dks;
      dst = (which == 0 ? o_q : which == 1 ? o_k : o_vt) + ((size_t)ub * o_H + hd) * head_bytes;
      kk = c & DKm;
    } else if (mode == OUT_POS) {
      hd = nb >> dks;
      dst = o_p + ((size_t)hd * o_prows << dks);
      kk = nb & DKm;
    } else {
      dst = o_y + (size_t)ub * rows * N + nb;
      zsrc = o_z1 + (size_t)ub * rows * N + nb;
    }
    // the tile-local channel of element e: with rows as tokens (V^T) the column, else
    // row g * 8 + half * 4 + e' of element e = 4g + e'
    auto chan = [&](int e) { return vwave ? nl + col : nl + (e >> 2) * 8 + half * 4 + (e & 3); };
    // the fast form's multipliers, the same for all the sub-tile's token columns
    int mc[16];
    if (vwave) {
      const int m1 = sreq[0][nl + col];
#pragma unroll
      for (int e = 0; e < 16; ++e) mc[e] = m1;
    } else {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const v4i q = *(const v4i*)&sreq[0][nl + g * 8 + half * 4];
#pragma unroll
        for (int e = 0; e < 4; ++e) mc[4 * g + e] = q[e];
      }
    }
    // this lane's destination for token column j = 0 (relative to dst, under 2^31),
    // the first token it stores and the bound on tokens: one 32-token column further
    // is a uniform step (jstep; for V^T, 512 bytes within a 64-key block, and the
    // next block at even columns)
    int tl, tmax;
    uint32_t off0;
    if (vwave) {
      tl = tw0 + half * 16;
      tmax = o_T_al;
      off0 = (uint32_t)vt_off(tl, kk + col);
    } else {
      tl = tw0 + col;
      tmax = rows;
      off0 = mode == OUT_ROWMAJOR ? (uint32_t)(tl * N + half * 16)
                                  : (uint32_t)frag_off((mode == OUT_POS ? o_pbase : 0) + tl, kk + half * 16);
    }
    const uint32_t jstep = mode == OUT_ROWMAJOR ? 32u * (uint32_t)N : 2u << (dks + 4);
#pragma unroll
    for (int j = 0; j < FM; ++j) {
      int v[16];
      if (rq_wide) {
        // a compiler barrier keeps the wide form's LDS reads here instead of letting
        // them be hoisted into live registers next to the fast form's
        asm volatile("" ::: "memory");
        requant16_wide(acc[i][j], sreq[0], sreq[1], chan, v);
      } else {
        requant16_fast(acc[i][j], mc, -rq_clamp, rq_clamp, v);
      }
      uint32_t D[4];
      pack16<EPI == EPI_SWISH>(v, D, (const uint8_t*)stab32);
      const auto x02 = __builtin_amdgcn_permlane32_swap(D[0], D[2], false, false);
      const auto x13 = __builtin_amdgcn_permlane32_swap(D[1], D[3], false, false);
      v4i out = (v4i){(int)x02[0], (int)x02[1], (int)x13[0], (int)x13[1]};

      // V^T: 16 consecutive tokens of one channel, stored up to T_al (zeros past the
      // utterance: the operand rows there read as zeros); otherwise 16 consecutive
      // channels of one token
      const uint32_t joff = vwave ? ((uint32_t)(j >> 1) << (dks + 6)) + (uint32_t)(j & 1) * 512u : (uint32_t)j * jstep;
      if (tl + j * 32 < tmax) {
        if (EPI == EPI_RESID)
          out = residual16(out, *(const v4i*)(zsrc + (off0 + joff)), args.m_z, args.m_y, args.shift_r);
        *(v4i*)(dst + (off0 + joff)) = out;
      }
    }
  }
}

static int add_problem(GemmArgs& a, int idx, const int8_t* x, const int8_t* w, const Requant& rq, int nb,
                       int rows, int N, int K, int mode, int tile_begin, int TN, int TM) {
  GemmProblem& p = a.prob[idx];
  p.x = x;
  p.w = w;
  p.req = rq.req;
  p.wide = rq.wide;
  p.clamp = rq.clamp;
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
  const int last = tiles_m - (tiles_m - 1) / p.band * p.band;  // token tiles of the last band
  p.dv_band_span = make_div((uint32_t)(p.band * p.tiles_n));
  p.dv_band = make_div((uint32_t)p.band);
  p.dv_last_band = make_div((uint32_t)last);
  p.dv_tiles_m_per = make_div((uint32_t)p.tiles_m_per);
  return tiles;
}

static void fill_dest(GemmArgs& a, const RunShape& rs, const Workspace& ws, int8_t* y) {
  a.q = ws.q;
  a.k = ws.k;
  a.vt = ws.vt;
  a.p = ws.p;
  a.z1 = nullptr;
  a.y = y;
  a.T_al = rs.T_al;
  a.H = rs.H;
  a.dk_shift = rs.DK == 128 ? 7 : 6;  // d_k is 64 or 128
  a.d = rs.d;
  a.p_rows = rs.p_rows;
  a.p_base = rs.p_base;
}

template <int TN, int TM, int NWAVE, int WN, int EPI = EPI_PLAIN, int TPF = 1>
static hipError_t launch_gemm(GemmArgs& a, int tiles, hipStream_t st, const LaunchEv& ev) {
  a.tiles_total = tiles;
  a.per_xcd = (tiles + 7) / 8;
  const bool wide = a.prob[0].wide || (a.nprob > 1 && a.prob[1].wide);
  return wide ? launch_kernel(gemm_i8_requant<TN, TM, NWAVE, WN, EPI, TPF, true>, dim3(8 * a.per_xcd), dim3(64 * NWAVE),
                              0, st, ev, a)
              : launch_kernel(gemm_i8_requant<TN, TM, NWAVE, WN, EPI, TPF, false>, dim3(8 * a.per_xcd),
                              dim3(64 * NWAVE), 0, st, ev, a);
}

// Token-tile height for a launch of `tiles_of(TM)` tiles: every tile of a launch runs at
// once when the tiles fit the CUs, so a launch takes about (rounds over the CUs) x (one
// tile's K loop, proportional to TM).  The smaller height wins only when it needs
// fewer rounds x rows (ties keep the larger tile, which has less overhead per row).
constexpr int kGemmCUs = 256;
template <typename F>
static int pick_tile_rows(int big, int small, F tiles_of) {
  auto cost = [&](int tm) { return (long)((tiles_of(tm) + kGemmCUs - 1) / kGemmCUs) * tm; };
  return cost(small) < cost(big) ? small : big;
}

// A tile shape of the projection launch (channels, tokens, waves, waves along channels,
// token-tile prefetch depth).
template <int TN_, int TM_, int NWAVE_, int WN_, int TPF_>
struct ProjShape {
  static constexpr int tn = TN_, tm = TM_, nwave = NWAVE_, wn = WN_, tpf = TPF_;
};

hipError_t launch_projections(const RunShape& rs, const Weights& w, const Workspace& ws, const int8_t* x,
                              const int8_t* pos_table, hipStream_t st, const LaunchEv& ev) {
  // 256-channel tiles of eight waves in a 4 x 2 grid (64 channels x TM/2 tokens each):
  // with TM = 256, per K step a workgroup moves 32 KB of token tile and 128 KB of token
  // fragments through LDS and streams 64 KB of weight fragments (each wave's own, two
  // waves per block).  TM = 128 halves the tiles' height when that fills the CUs better
  // (Q|K|V alone at T = 2500: 240 tiles in one round instead of 120 of twice the work).
  constexpr int TN = 256, NWAVE = 8, WN = 4;
  auto tiles_of = [&](int tm) {
    long t = (long)rs.B * ((rs.T + tm - 1) / tm) * ((3 * rs.d + TN - 1) / TN);
    if (pos_table) t += (long)((2 * rs.T - 1 + tm - 1) / tm) * ((rs.d + TN - 1) / TN);
    return t;
  };
  const int TMr = pick_tile_rows(256, 128, tiles_of);
  auto go = [&](auto shape_tag) {
    using S = decltype(shape_tag);
    constexpr int TNs = S::tn, TMs = S::tm, NW = S::nwave, WNs = S::wn, TPFs = S::tpf;
    // V^T's 64-key blocks: a wave's tokens are whole blocks
    static_assert((TMs / (NW / WNs)) % KCHUNK == 0 && (TNs / WNs) % 32 == 0, "projection tile shape");
    GemmArgs a{};
    fill_dest(a, rs, ws, nullptr);
    int tiles = add_problem(a, 0, x, w.w_qkv, w.rq_qkv, rs.B, rs.T, 3 * rs.d, rs.d, OUT_QKV, 0, TNs, TMs);
    a.nprob = 1;
    if (pos_table) {
      tiles += add_problem(a, 1, pos_table, w.w_pos, w.rq_pos, 1, 2 * rs.T - 1, rs.d, rs.d, OUT_POS, tiles, TNs, TMs);
      a.nprob = 2;
    }
    return launch_gemm<TNs, TMs, NW, WNs, EPI_PLAIN, TPFs>(a, tiles, st, ev);
  };
  // a short call (few frames): where the 256-channel tiles would leave more than half of
  // the CUs idle, 128-channel x 64-token tiles of four waves (32 channels x 64 tokens
  // each, the token tile fetched two steps ahead) spread it over several times as many
  // workgroups
  if (tiles_of(TMr) < kGemmCUs / 2) return go(ProjShape<128, 64, 4, 4, 2>{});
  return TMr == 128 ? go(ProjShape<TN, 128, NWAVE, WN, 1>{}) : go(ProjShape<TN, 256, NWAVE, WN, 1>{});
}

hipError_t launch_pos_projection(const RunShape& rs, const Weights& w, int8_t* p, const int8_t* pos_table,
                                 hipStream_t st) {
  GemmArgs a{};
  Workspace ws{};
  ws.p = p;
  fill_dest(a, rs, ws, nullptr);
  constexpr int TN = 256, TM = 256, NWAVE = 8, WN = 4;
  const int tiles = add_problem(a, 0, pos_table, w.w_pos, w.rq_pos, 1, 2 * rs.T - 1, rs.d, rs.d, OUT_POS, 0, TN, TM);
  a.nprob = 1;
  return launch_gemm<TN, TM, NWAVE, WN>(a, tiles, st, LaunchEv{});
}

hipError_t launch_out_projection(const RunShape& rs, const Weights& w, const Workspace& ws, int8_t* y,
                                 hipStream_t st, const LaunchEv& ev, const Residual* res, const int8_t* z1) {
  GemmArgs a{};
  fill_dest(a, rs, ws, y);
  if (res) {
    a.z1 = z1;
    a.m_z = res->m_z;
    a.m_y = res->m_y;
    a.shift_r = res->shift_r;
  }
  // small tiles (640 at T = 2500): with K = d_model and few 64-token blocks the launch
  // is bound by load latency, and larger tiles measured no faster
  constexpr int TN = 64, TM = 64, NWAVE = 4, WN = 2;
  int tiles = add_problem(a, 0, ws.ctx, w.w_out, w.rq_out, rs.B, rs.T, rs.d, rs.d, OUT_ROWMAJOR, 0, TN, TM);
  a.nprob = 1;
  // the token tile two steps ahead: 0.6 - 0.7 us less per call at T = 2500 (interleaved A/B)
  if (res) return launch_gemm<TN, TM, NWAVE, WN, EPI_RESID, 2>(a, tiles, st, ev);
  return launch_gemm<TN, TM, NWAVE, WN, EPI_PLAIN, 2>(a, tiles, st, ev);
}

// ---------------------------------------------------------------------------
// The feed-forward module of Eq. 1: W1 with the integer Swish in its epilogue, W2
// with the residual add in its epilogue.

// The integer Swish of Eq. 12 and its requantization to FFN2's input grid, for every
// int8 input h (one thread per biased code h + 128; code 0 is never looked up):
//   L = (min(|h|, q_c) - q_c)^2 + q_1,  q = -(|h| L + h q_1),  o = clamp8(RS(q, m, n)).
// The host checks that |q m| + 2^(n-1) stays below 2^62 for every h.
__global__ __launch_bounds__(256) void swish_table(uint8_t* tab, long long q_c, long long q_1, long long m,
                                                   int shift) {
  const long long h = (long long)threadIdx.x - 128;
  const long long ah = h < 0 ? -h : h;
  const long long t = (ah < q_c ? ah : q_c) - q_c;
  const long long L = t * t + q_1;
  const long long q = -(ah * L + h * q_1);
  const long long o = (q * m + (1ll << (shift - 1))) >> shift;
  tab[threadIdx.x] = (uint8_t)(int)(o < -127 ? -127 : (o > 127 ? 127 : o));
}

hipError_t launch_swish_table(uint8_t* tab, long long q_c, long long q_1, long long m, int shift, hipStream_t st) {
  hipLaunchKernelGGL(swish_table, dim3(1), dim3(256), 0, st, tab, q_c, q_1, m, shift);
  return hipGetLastError();
}

hipError_t launch_ffn_up(const int8_t* x, int rows, int d, int d_ff, const int8_t* w1, const Requant& rq1,
                         const uint8_t* swtab, int8_t* o, hipStream_t st) {
  // 256-channel tiles of eight waves; 192-token tiles when they need no more rounds
  // over the CUs than 256-token ones (2500 rows: 224 tiles instead of 160 of 4/3 the work)
  constexpr int TN = 256, NWAVE = 8, WN = 4;
  auto tiles_of = [&](int tm) { return (long)((rows + tm - 1) / tm) * ((d_ff + TN - 1) / TN); };
  auto go = [&](auto tm_tag) {
    constexpr int TM = decltype(tm_tag)::value;
    GemmArgs a{};
    a.y = o;
    a.swtab = swtab;
    const int tiles = add_problem(a, 0, x, w1, rq1, 1, rows, d_ff, d, OUT_ROWMAJOR, 0, TN, TM);
    a.nprob = 1;
    return launch_gemm<TN, TM, NWAVE, WN, EPI_SWISH>(a, tiles, st, LaunchEv{});
  };
  return pick_tile_rows(256, 192, tiles_of) == 192 ? go(std::integral_constant<int, 192>{})
                                                   : go(std::integral_constant<int, 256>{});
}

hipError_t launch_linear_resid(const int8_t* x, int rows, int N, int K, const int8_t* w, const Requant& rq,
                               const int8_t* z, int m_z, int m_y, int shift_r, int8_t* z_out, hipStream_t st) {
  GemmArgs a{};
  a.y = z_out;
  a.z1 = z;
  a.m_z = m_z;
  a.m_y = m_y;
  a.shift_r = shift_r;
  // 128 x 128 tiles of eight waves (32 channels x 64 tokens each): for the feed-forward
  // module's W2 (K = d_ff) measured against 64 x 64, 128 x 64, 128 x 96, 64 x 192,
  // 256 x 128 and 128 x 256 tiles at 2500 and 4000 rows
  constexpr int TN = 128, TM = 128, NWAVE = 8, WN = 4;
  const int tiles = add_problem(a, 0, x, w, rq, 1, rows, N, K, OUT_ROWMAJOR, 0, TN, TM);
  a.nprob = 1;
  return launch_gemm<TN, TM, NWAVE, WN, EPI_RESID>(a, tiles, st, LaunchEv{});
}

hipError_t launch_linear(const int8_t* x, int rows, int K, int N, const int8_t* w, const Requant& rq, int8_t* y,
                         hipStream_t st) {
  constexpr int TN = 256, NWAVE = 8, WN = 4;
  auto tiles_of = [&](int tm) { return (long)((rows + tm - 1) / tm) * ((N + TN - 1) / TN); };
  int TMr = pick_tile_rows(256, 192, tiles_of);
  TMr = pick_tile_rows(TMr, 128, tiles_of);
  auto go = [&](auto tm_tag) {
    constexpr int TM = decltype(tm_tag)::value;
    GemmArgs a{};
    a.y = y;
    const int tiles = add_problem(a, 0, x, w, rq, 1, rows, N, K, OUT_ROWMAJOR, 0, TN, TM);
    a.nprob = 1;
    return launch_gemm<TN, TM, NWAVE, WN>(a, tiles, st, LaunchEv{});
  };
  // 128-channel x 192-token tiles (eight waves of 32 x 96) when they leave the busiest
  // CU less work than the 256-channel shape picked above (2500 rows, N = 2048: 224 tiles
  // of 24.6 K outputs against 160 of 32.8 K)
  const long t128 = (long)((rows + 191) / 192) * ((N + 127) / 128);
  const long rounds_wide = (tiles_of(TMr) + kGemmCUs - 1) / kGemmCUs, rounds128 = (t128 + kGemmCUs - 1) / kGemmCUs;
  if (rounds128 * 128 * 192 < rounds_wide * TN * TMr) {
    GemmArgs a{};
    a.y = y;
    const int tiles = add_problem(a, 0, x, w, rq, 1, rows, N, K, OUT_ROWMAJOR, 0, 128, 192);
    a.nprob = 1;
    return launch_gemm<128, 192, 8, 4>(a, tiles, st, LaunchEv{});
  }
  if (TMr == 128) return go(std::integral_constant<int, 128>{});
  if (TMr == 192) return go(std::integral_constant<int, 192>{});
  return go(std::integral_constant<int, 256>{});
}

// one thread per 16-byte piece of the destination
__global__ __launch_bounds__(256) void pack_wfrag(const int8_t* __restrict__ w, int8_t* __restrict__ dst, int N,
                                                  int K, DivU dv_ksl) {
  const long p = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= (long)N * K / 16) return;
  const int l = (int)(p & 63);
  const int frag = (int)(p >> 6);
  const int cb = (int)div_u((uint32_t)frag, dv_ksl), ks = frag - cb * (int)dv_ksl.d;
  const int8_t* src = w + (size_t)(cb * 32 + (l & 31)) * K + ks * 32 + (l >> 5) * 16;
  *(uint4*)(dst + p * 16) = *(const uint4*)src;
}

hipError_t pack_weight_fragments(const int8_t* w, int8_t* dst, int N, int K, hipStream_t st) {
  if (N % 32 || K % 32) return hipErrorInvalidValue;
  const long pieces = (long)N * K / 16;
  hipLaunchKernelGGL(pack_wfrag, dim3((unsigned)((pieces + 255) / 256)), dim3(256), 0, st, w, dst, N, K,
                     make_div((uint32_t)(K >> 5)));
  return hipGetLastError();
}

}  // namespace ipk
