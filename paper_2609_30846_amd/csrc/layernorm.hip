// Integer LayerNorm of the Conformer block (Eq. 1 - 4: every module normalizes its input
// first, and the block ends with one; the paper takes LayerNorm's integer form from
// I-BERT).
//
// For a row z of d int8 values:
//   mu    = floor((2 sum z + d) / (2 d))                 mean, ties up
//   sigma = max(1, floor(sqrt(sum (z - mu)^2)))          integer square root
//   F     = floor(2^31 / sigma)
//   u_k   = floor((z_k - mu) F / 2)
//   x_k   = clamp8(floor((u_k g_k + c_k + 2^(n-1)) / 2^n))
// g and c fold gamma, beta and the move to the block's input grid into one
// fixed-point step per channel (the rounding term comes pre-added to c).
//
// The work is a few bytes per element, so the kernel is bound by moving the rows
// (HBM or L2) and by the latency of doing so: one wave per row, each lane holding
// 16-byte pieces of it in registers, so the row is read once; the per-channel
// constants of the lane's pieces (4 + 8 bytes a channel, the same for every row) are
// requested together with the row, so their latency hides behind the row's and the
// sums'.  Both sums come from one pass: sum z and sum z^2 by
// v_dot4 against ones and against z itself, and
//   sum (z - mu)^2 = sum z^2 - 2 mu sum z + d mu^2
// exactly in integers, and the wave sums are DPP adds.  The mean (a binary search over
// its 9-bit range), floor(sqrt(v)) (bit by bit) and floor(2^31 / sigma) (restoring
// division) are wave-uniform integer sequences: no floating-point instruction runs.
#include "ipk_internal.h"

namespace ipk {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef long long v2l __attribute__((ext_vector_type(2)));

struct LnArgs {
  const int8_t* z;
  int8_t* x;
  const int32_t* g;
  const int64_t* c;  // bias plus 2^(shift-1)
  long rows;
  int d, shift;
};

constexpr int LN_WAVES = 4;  // rows per workgroup

// Sum over the wave: DPP adds leave every lane of a 16-lane row with the row's sum
// (quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror, row_mirror), and the four
// row sums are read as scalars.  Integer adds, so the order does not matter.
__device__ __forceinline__ int wave_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false);
  return __builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16) + __builtin_amdgcn_readlane(v, 32) +
         __builtin_amdgcn_readlane(v, 48);
}

// floor(x / D) for |x| <= 257 D / 2, D <= 2^15: the largest mu in [-256, 255] with
// mu D <= x, by binary search (every product stays below 2^23 in magnitude)
__device__ __forceinline__ int floor_div_small(int x, int D) {
  int mu = -256;
#pragma unroll
  for (int step = 256; step >= 1; step >>= 1)
    if ((mu + step) * D <= x) mu += step;
  return mu;
}

// floor(sqrt(v)) for 0 <= v < 2^32, bit by bit
__device__ __forceinline__ uint32_t isqrt_u32(uint32_t v) {
  uint32_t res = 0, one = 1u << 30;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    if (v >= res + one) {
      v -= res + one;
      res = (res >> 1) + one;
    } else {
      res >>= 1;
    }
    one >>= 2;
  }
  return res;
}

// floor(2^31 / s) for 1 <= s < 2^16 by restoring division (the remainder stays below s)
__device__ __forceinline__ uint32_t div_2p31(uint32_t s) {
  uint32_t r = 1, q = 0;  // the dividend's only one bit, bit 31, enters first
#pragma unroll
  for (int i = 31; i >= 0; --i) {
    const bool c = r >= s;
    if (c) r -= s;
    q |= (c ? 1u : 0u) << i;
    r <<= 1;
  }
  return q;
}

// NP: 16-byte pieces per lane (d <= 1024 NP).  With NP <= 2 the lane's constants
// are loaded up front (at most 104 registers); wider rows load them per piece.
template <int NP>
__global__ __launch_bounds__(64 * LN_WAVES) void layernorm_i8(LnArgs a) {
  constexpr bool PRE = NP <= 2;
  const int lane = threadIdx.x & 63;
  const long row = (long)blockIdx.x * LN_WAVES + (threadIdx.x >> 6);
  if (row >= a.rows) return;
  const int d = a.d, npieces = d >> 4;
  const int8_t* src = a.z + row * d;
  v4i zv[NP];
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int p = lane + 64 * k;
    zv[k] = p < npieces ? *(const v4i*)(src + 16 * p) : (v4i){0, 0, 0, 0};
  }
  // the constants of the lane's 16 channels per piece: multipliers (4 x 16 bytes) and
  // biases (8 x 16 bytes)
  v4i gv[PRE ? NP : 1][4];
  v2l cv[PRE ? NP : 1][8];
  auto load_consts = [&](int c0, v4i (&g)[4], v2l (&c)[8]) {
#pragma unroll
    for (int w = 0; w < 4; ++w) g[w] = *(const v4i*)(a.g + c0 + 4 * w);
#pragma unroll
    for (int j = 0; j < 8; ++j) c[j] = *(const v2l*)(a.c + c0 + 2 * j);
  };
  if constexpr (PRE) {
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      const int p = lane + 64 * k;
      if (p < npieces) load_consts(16 * p, gv[k], cv[k]);
    }
  }
  int s = 0, q = 0;
#pragma unroll
  for (int k = 0; k < NP; ++k) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      s = __builtin_amdgcn_sdot4(zv[k][w], 0x01010101, s, false);
      q = __builtin_amdgcn_sdot4(zv[k][w], zv[k][w], q, false);
    }
  }
  // |sum z| <= 128 d < 2^21 and sum z^2 <= 2^14 d < 2^29 for d <= 16384
  s = wave_sum(s);
  q = wave_sum(q);
  // mean, ties up: floor((2 sum z + d) / (2 d)), with |2 sum z + d| <= 257 d
  const int mu = floor_div_small(2 * s + d, 2 * d);
  const long long var = (long long)q - 2ll * mu * s + (long long)d * mu * mu;  // sum (z - mu)^2 < 2^31
  uint32_t sg = isqrt_u32((uint32_t)var);
  if (sg < 1) sg = 1;
  const long long F = div_2p31(sg);  // floor(2^31 / sigma), sigma < 2^16
  // u = floor(y F / 2) for y = z - mu, in 32 bits: with F = 2 Fh + Fo,
  // u = y Fh + Fo floor(y / 2), and |y Fh| <= |y| F / 2 <= 2^30 since |y| <= sigma
  const int Fh = (int)(F >> 1), Fo = (F & 1) ? -1 : 0;
  const int shift = a.shift;
  const int m = mu;
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int p = lane + 64 * k;
    if (p >= npieces) continue;
    const int c0 = 16 * p;
    v4i g[4];
    v2l c[8];
    if constexpr (PRE) {
#pragma unroll
      for (int w = 0; w < 4; ++w) g[w] = gv[k][w];
#pragma unroll
      for (int j = 0; j < 8; ++j) c[j] = cv[k][j];
    } else {
      load_consts(c0, g, c);
    }
    v4i out;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      uint32_t o = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int zb = (zv[k][w] << (24 - 8 * b)) >> 24;
        const int y = zb - m;
        const int u = y * Fh + ((y >> 1) & Fo);
        const int e = 4 * w + b;
        const long long t = ((long long)u * g[w][b] + c[e >> 1][e & 1]) >> shift;
        o |= ((uint32_t)(int)min(max(t, -127ll), 127ll) & 0xFFu) << (8 * b);
      }
      out[w] = (int)o;
    }
    *(v4i*)(a.x + row * d + c0) = out;
  }
}

static hipError_t launch_ln(long rows, int d, const Residual& r, const int8_t* z, int8_t* out, hipStream_t st,
                            const LaunchEv& ev) {
  LnArgs a{};
  a.z = z;
  a.x = out;
  a.g = r.ln_mult;
  a.c = r.ln_bias;
  a.rows = rows;
  a.d = d;
  a.shift = r.ln_shift;
  const dim3 grid((unsigned)((a.rows + LN_WAVES - 1) / LN_WAVES)), block(64 * LN_WAVES);
  const int np = (d + 1023) / 1024;
  if (d % 16) return hipErrorInvalidValue;
  if (np <= 1) return launch_kernel(layernorm_i8<1>, grid, block, 0, st, ev, a);
  if (np <= 2) return launch_kernel(layernorm_i8<2>, grid, block, 0, st, ev, a);
  if (np <= 4) return launch_kernel(layernorm_i8<4>, grid, block, 0, st, ev, a);
  if (np <= 8) return launch_kernel(layernorm_i8<8>, grid, block, 0, st, ev, a);
  if (np <= 16) return launch_kernel(layernorm_i8<16>, grid, block, 0, st, ev, a);
  return hipErrorInvalidValue;
}

hipError_t launch_layernorm(const RunShape& rs, const Residual& r, const int8_t* z, int8_t* out, hipStream_t st,
                            const LaunchEv& ev) {
  return launch_ln((long)rs.B * rs.T, rs.d, r, z, out, st, ev);
}

hipError_t launch_layernorm_rows(long rows, int d, const Residual& r, const int8_t* z, int8_t* out, hipStream_t st) {
  return launch_ln(rows, d, r, z, out, st, LaunchEv{});
}

}  // namespace ipk
