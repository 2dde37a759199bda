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
// (HBM or L2): one wave per row, each lane holding 16-byte pieces of it in registers,
// so the row is read once.  Both sums come from one pass: sum z and sum z^2 by
// v_dot4 against ones and against z itself, and
//   sum (z - mu)^2 = sum z^2 - 2 mu sum z + d mu^2
// exactly in integers, and the wave sums are DPP adds.  floor(sqrt(v)) is the correctly
// rounded double square root truncated and then checked against v (v < 2^31, so the
// double is within one of the root and one correction step suffices either way).
#include "ipk_internal.h"

namespace ipk {

typedef int v4i __attribute__((ext_vector_type(4)));

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

// floor(a / b) for b > 0
__device__ __forceinline__ long long floor_div(long long a, long long b) {
  const long long q = a / b;
  return (q * b > a) ? q - 1 : q;
}

// NP: 16-byte pieces per lane (d <= 1024 NP)
template <int NP>
__global__ __launch_bounds__(64 * LN_WAVES) void layernorm_i8(LnArgs a) {
  const int lane = threadIdx.x & 63;
  const long row = (long)blockIdx.x * LN_WAVES + (threadIdx.x >> 6);
  if (row >= a.rows) return;
  const int d = a.d, npieces = d >> 4;
  const int8_t* src = a.z + row * d;
  v4i zv[NP];
  int s = 0, q = 0;
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int p = lane + 64 * k;
    zv[k] = p < npieces ? *(const v4i*)(src + 16 * p) : (v4i){0, 0, 0, 0};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      s = __builtin_amdgcn_sdot4(zv[k][w], 0x01010101, s, false);
      q = __builtin_amdgcn_sdot4(zv[k][w], zv[k][w], q, false);
    }
  }
  // |sum z| <= 128 d < 2^21 and sum z^2 <= 2^14 d < 2^29 for d <= 16384
  s = wave_sum(s);
  q = wave_sum(q);
  const long long mu = floor_div(2ll * s + d, 2ll * d);
  const long long var = (long long)q - 2 * mu * s + (long long)d * mu * mu;  // sum (z - mu)^2
  long long sg = (long long)sqrt((double)var);
  if (sg * sg > var) --sg;
  if ((sg + 1) * (sg + 1) <= var) ++sg;
  if (sg < 1) sg = 1;
  // floor(2^31 / sigma) from the correctly rounded double quotient: unless sigma divides
  // 2^31 the quotient lies at least 1 / sigma >= 2^-16 below the next integer, far more
  // than its rounding error (2^31 2^-53), so truncating it gives the floor
  const long long F = (long long)(2147483648.0 / (double)sg);
  // u = floor(y F / 2) for y = z - mu, in 32 bits: with F = 2 Fh + Fo,
  // u = y Fh + Fo floor(y / 2), and |y Fh| <= |y| F / 2 <= 2^30 since |y| <= sigma
  const int Fh = (int)(F >> 1), Fo = (F & 1) ? -1 : 0;
  const int shift = a.shift;
  const int m = (int)mu;
#pragma unroll
  for (int k = 0; k < NP; ++k) {
    const int p = lane + 64 * k;
    if (p >= npieces) continue;
    const int c0 = 16 * p;
    v4i out;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const v4i gv = *(const v4i*)(a.g + c0 + 4 * w);
      uint32_t o = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int zb = (zv[k][w] << (24 - 8 * b)) >> 24;
        const int y = zb - m;
        const int u = y * Fh + ((y >> 1) & Fo);
        const long long t = ((long long)u * gv[b] + a.c[c0 + 4 * w + b]) >> shift;
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
