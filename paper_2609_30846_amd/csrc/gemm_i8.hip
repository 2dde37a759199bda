// INT8 projection GEMMs with a fused fixed-point requantization epilogue.
//
// Every linear layer of the block (Q, K, V, the relative-position projection and
// the output projection) is Eq. 7: an int8 x int8 product accumulated in int32,
// rescaled by a per-output-channel multiplier m and a right shift n with round to
// nearest (ties up), and clamped to the symmetric int8 grid.
//
// Kernel shape: one 256-thread workgroup computes a TN x TM tile of
// D[n][m] = sum_k W[n][k] X[m][k] with v_mfma_i32_32x32x32_i8 (4 waves in a 2x2
// grid, each (TN/2) x (TM/2)).  K is walked in 64-byte steps through a double
// buffer in LDS whose rows are padded to 80 bytes, which keeps the 16-byte operand
// reads of 8 consecutive lanes on distinct banks.  Output channels run along the
// MFMA rows, so each lane ends with 4 consecutive channels of one token per group
// of accumulators: the epilogue requantizes them and writes 4 bytes at once into
// the head-major workspace layouts (V goes out transposed, byte by byte).
// Several problems share one launch (Q|K|V stacked plus the position projection).
#include "ipk_internal.h"

namespace ipk {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

enum OutMode { OUT_QKV = 0, OUT_POS = 1, OUT_ROWMAJOR = 2 };

struct GemmProblem {
  const int8_t* x;       // [M][K] activations
  const int8_t* w;       // [N][K] weights
  const int32_t* mult;   // [N]
  const int32_t* shift;  // [N]
  int M, N, K;
  int mode;
  int tile_begin;  // first linear tile index of this problem
  int tiles_n;     // tiles along N (N fastest)
};

struct GemmArgs {
  GemmProblem prob[2];
  int nprob;
  int8_t *q, *k, *vt, *p, *y;
  int T, T_al, H, DK, d, p_rows, p_base;
};

constexpr int BK = 64;
constexpr int SROW = BK + 16;  // padded LDS row (bytes)

__device__ __forceinline__ int requant8(int acc, int mult, int shift) {
  int64_t t = (int64_t)acc * (int64_t)mult + ((int64_t)1 << (shift - 1));
  int64_t r = t >> shift;  // arithmetic shift: floor division by 2^shift
  return r < -127 ? -127 : (r > 127 ? 127 : (int)r);
}

template <int TN, int TM>
__global__ __launch_bounds__(256) void gemm_i8_requant(GemmArgs args) {
  constexpr int FN = TN / 64;  // 32-row MFMA tiles per wave along N
  constexpr int FM = TM / 64;  // 32-col MFMA tiles per wave along M
  constexpr int LW = TN * 4 / 256;  // 16-byte global loads per thread, W tile
  constexpr int LX = TM * 4 / 256;  // same for the X tile
  __shared__ __align__(16) int8_t sw[2][TN * SROW];
  __shared__ __align__(16) int8_t sx[2][TM * SROW];

  // locate the problem and tile
  int tile = blockIdx.x;
  int pi = (args.nprob > 1 && tile >= args.prob[1].tile_begin) ? 1 : 0;
  const GemmProblem& P = args.prob[pi];
  const int local = tile - P.tile_begin;
  const int n0 = (local % P.tiles_n) * TN;
  const int m0 = (local / P.tiles_n) * TM;
  const int K = P.K;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave & 1, wm = wave >> 1;

  // global -> register staging
  v4i rw[LW], rx[LX];
  auto load_tile = [&](int k0) {
#pragma unroll
    for (int r = 0; r < LW; ++r) {
      int id = tid + 256 * r, row = id >> 2, kc = id & 3;
      int n = min(n0 + row, P.N - 1);
      rw[r] = *(const v4i*)(P.w + (size_t)n * K + k0 + kc * 16);
    }
#pragma unroll
    for (int r = 0; r < LX; ++r) {
      int id = tid + 256 * r, row = id >> 2, kc = id & 3;
      int m = min(m0 + row, P.M - 1);
      rx[r] = *(const v4i*)(P.x + (size_t)m * K + k0 + kc * 16);
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int r = 0; r < LW; ++r) {
      int id = tid + 256 * r, row = id >> 2, kc = id & 3;
      *(v4i*)(&sw[buf][row * SROW + kc * 16]) = rw[r];
    }
#pragma unroll
    for (int r = 0; r < LX; ++r) {
      int id = tid + 256 * r, row = id >> 2, kc = id & 3;
      *(v4i*)(&sx[buf][row * SROW + kc * 16]) = rx[r];
    }
  };

  v16i acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = (v16i){};

  const int nk = K / BK;
  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_tile((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      v4i af[FN], bf[FM];
#pragma unroll
      for (int i = 0; i < FN; ++i)
        af[i] = *(const v4i*)(&sw[buf][(wn * (TN / 2) + i * 32 + (lane & 31)) * SROW + ks * 32 + (lane >> 5) * 16]);
#pragma unroll
      for (int j = 0; j < FM; ++j)
        bf[j] = *(const v4i*)(&sx[buf][(wm * (TM / 2) + j * 32 + (lane & 31)) * SROW + ks * 32 + (lane >> 5) * 16]);
#pragma unroll
      for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) store_tile(buf ^ 1);
    __syncthreads();
  }

  // epilogue: lane holds token m = .. + (lane & 31); accumulator e holds channel
  // n = .. + (e / 4) * 8 + (lane / 32) * 4 + (e % 4)
#pragma unroll
  for (int j = 0; j < FM; ++j) {
    const int m = m0 + wm * (TM / 2) + j * 32 + (lane & 31);
    if (m >= P.M) continue;
#pragma unroll
    for (int i = 0; i < FN; ++i) {
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const int n = n0 + wn * (TN / 2) + i * 32 + grp * 8 + (lane >> 5) * 4;
        if (n >= P.N) continue;
        int qv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) qv[e] = requant8(acc[i][j][grp * 4 + e], P.mult[n + e], P.shift[n + e]);
        const uint32_t packed = (uint32_t)(qv[0] & 0xff) | ((uint32_t)(qv[1] & 0xff) << 8) |
                                ((uint32_t)(qv[2] & 0xff) << 16) | ((uint32_t)(qv[3] & 0xff) << 24);
        if (P.mode == OUT_QKV) {
          const int which = n / args.d, c = n - which * args.d;
          const int h = c / args.DK, kk = c - h * args.DK;
          const int b = m / args.T, t = m - b * args.T;
          const size_t bh = (size_t)b * args.H + h;
          if (which < 2) {
            int8_t* base = (which == 0 ? args.q : args.k) + bh * args.T_al * args.DK;
            *(uint32_t*)(base + frag_index(t, kk, args.DK)) = packed;
          } else {
            int8_t* base = args.vt + bh * args.T_al * args.DK;
#pragma unroll
            for (int e = 0; e < 4; ++e) base[vt_index(t, kk + e, args.DK)] = (int8_t)qv[e];
          }
        } else if (P.mode == OUT_POS) {
          const int h = n / args.DK, kk = n - h * args.DK;
          int8_t* base = args.p + (size_t)h * args.p_rows * args.DK;
          *(uint32_t*)(base + frag_index(args.p_base + m, kk, args.DK)) = packed;
        } else {
          *(uint32_t*)(args.y + (size_t)m * P.N + n) = packed;
        }
      }
    }
  }
}

static int add_problem(GemmArgs& a, int idx, const int8_t* x, const int8_t* w, const int32_t* mult,
                       const int32_t* shift, int M, int N, int K, int mode, int tile_begin, int TN, int TM) {
  GemmProblem& p = a.prob[idx];
  p.x = x;
  p.w = w;
  p.mult = mult;
  p.shift = shift;
  p.M = M;
  p.N = N;
  p.K = K;
  p.mode = mode;
  p.tile_begin = tile_begin;
  p.tiles_n = (N + TN - 1) / TN;
  return p.tiles_n * ((M + TM - 1) / TM);
}

static void fill_dest(GemmArgs& a, const RunShape& rs, const Workspace& ws, int8_t* y) {
  a.q = ws.q;
  a.k = ws.k;
  a.vt = ws.vt;
  a.p = ws.p;
  a.y = y;
  a.T = rs.T;
  a.T_al = rs.T_al;
  a.H = rs.H;
  a.DK = rs.DK;
  a.d = rs.d;
  a.p_rows = p_rows(rs.T_al);
  a.p_base = rs.p_base;
}

hipError_t launch_projections(const RunShape& rs, const Weights& w, const Workspace& ws, const int8_t* x,
                              const int8_t* pos_table, hipStream_t st) {
  GemmArgs a{};
  fill_dest(a, rs, ws, nullptr);
  constexpr int TN = 128, TM = 128;
  const int M = rs.B * rs.T;
  int tiles = add_problem(a, 0, x, w.w_qkv, w.mult_qkv, w.shift_qkv, M, 3 * rs.d, rs.d, OUT_QKV, 0, TN, TM);
  tiles += add_problem(a, 1, pos_table, w.w_pos, w.mult_pos, w.shift_pos, 2 * rs.T - 1, rs.d, rs.d, OUT_POS, tiles,
                       TN, TM);
  a.nprob = 2;
  hipLaunchKernelGGL((gemm_i8_requant<TN, TM>), dim3(tiles), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_out_projection(const RunShape& rs, const Weights& w, const Workspace& ws, int8_t* y,
                                 hipStream_t st) {
  GemmArgs a{};
  fill_dest(a, rs, ws, y);
  constexpr int TN = 128, TM = 64;
  const int M = rs.B * rs.T;
  int tiles = add_problem(a, 0, ws.ctx, w.w_out, w.mult_out, w.shift_out, M, rs.d, rs.d, OUT_ROWMAJOR, 0, TN, TM);
  a.nprob = 1;
  hipLaunchKernelGGL((gemm_i8_requant<TN, TM>), dim3(tiles), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace ipk
