// Relative-position attention core of the integer MHSA block (Sec. 3.1).
//
// One 256-thread workgroup owns (utterance b, head h, a block of 16*NRT query
// rows).  Each wave owns one 16-row tile and a contiguous range of 64-key chunks
// (4/NRT waves split the keys of a tile).  Per 16x16 score tile:
//
//  * content score   c = Q K^T + (u.K_j)    -- v_mfma_i32_16x16x64_i8; the rank-1
//                                              term seeds the accumulator
//  * position score  G = Q P_win^T + (v.P_r) for the two 16-row windows of the
//                    table that the tile's relative positions j-i+T-1 touch;
//                    Phi is then a per-row rotation inside each 16-lane row
//                    group: every source lane picks the window its value belongs
//                    to and ds_bpermute moves it to the lane of its key
//  * fused requant   s = clamp8(RS(m_c c + m_p p, 1, shift_s))  (Eq. 11), exact
//                    in 64-bit
//  * masked keys (j >= L_b) are stored as -128, a code below every valid score
//
// The int8 scores of the workgroup's rows stay in LDS (never in HBM).  Then:
// row max (wave shuffles + LDS across the waves of a tile), I-BERT integer exp
// and row sum, F = floor(2^32 / sum), and a = min(floor(e F / 2^24), 255).
// The A.V contraction runs on v_mfma_i32_16x16x64_i8 with a - 128 as the signed
// operand; the exact correction 128 * sum_j V_j over the same keys comes from
// per-chunk prefix sums of V.  Partial contexts of the waves sharing a tile are
// added in LDS (int32, exact) and requantized with (m_o, shift_o).
#include "ipk_internal.h"

namespace ipk {

typedef int v4i __attribute__((ext_vector_type(4)));

struct AttnArgs {
  const int8_t *q, *k, *vt, *p;
  const int32_t *bu, *bv, *vsum;
  int8_t* ctx;
  Lengths lens;
  int T, T_al, H, d, p_rows;
  int32_t m_c, m_p, shift_s, m_o, shift_o, q_ln2, q_b, q_c;
};

constexpr int SCORE_PAD = 16;  // bytes added to each LDS score row

__device__ __forceinline__ uint32_t iexp_int(int d, int q_ln2, int q_b, int q_c) {
  // I-BERT integer exp of -d: d = z q_ln2 - r, r in (-q_ln2, 0]
  const int z = d / q_ln2;
  const int r = z * q_ln2 - d;
  const int poly = (r + q_b) * (r + q_b) + q_c;  // < 2^24 (checked at create)
  return z >= 32 ? 0u : ((uint32_t)poly >> z);
}

template <int DK, int NRT>
__global__ __launch_bounds__(256) void relpos_attn_core(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int WPT = 4 / NRT;   // waves per 16-row tile
  constexpr int NKS = DK / 64;   // MFMA K-steps over d_k
  constexpr int NT = DK / 16;    // 16-wide output tiles of the context

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int rt = w % NRT, ks = w / NRT;
  const int b = blockIdx.z, h = blockIdx.y;
  const int i_base = blockIdx.x * 16 * NRT;
  const int i0 = i_base + 16 * rt;
  const int L = a.lens.len[b];
  const int T = a.T, T_al = a.T_al;
  const int srow = T_al + SCORE_PAD;
  const int sbuf_bytes = 16 * NRT * srow;
  const int red_bytes = 4 * 16 * DK * 4;
  int8_t* sbuf = (int8_t*)smem;
  int32_t* red = (int32_t*)smem;  // reused after the scores are consumed
  int32_t* smax = (int32_t*)(smem + (sbuf_bytes > red_bytes ? sbuf_bytes : red_bytes));
  uint32_t* ssum = (uint32_t*)(smax + 64);

  const int col = lane & 15, g = lane >> 4;
  const int nkc = (L + KCHUNK - 1) / KCHUNK;
  const int c_begin = ks * nkc / WPT, c_end = (ks + 1) * nkc / WPT;
  const bool active = i0 < L;
  const size_t bh = (size_t)b * a.H + h;
  const int8_t* Qh = a.q + bh * T_al * DK;
  const int8_t* Kh = a.k + bh * T_al * DK;
  const int8_t* VTh = a.vt + bh * DK * T_al;
  const int8_t* Ph = a.p + (size_t)h * a.p_rows * DK;
  const int32_t* bu = a.bu + bh * T_al;
  const int32_t* bv = a.bv + (size_t)h * a.p_rows;
  const int32_t* vs = a.vsum + bh * (size_t)(T_al / KCHUNK + 1) * DK;
  int8_t* srows = sbuf + (size_t)(16 * rt) * srow;

  // ---------------- phase 1: fused scores into LDS, running row max
  int mx[4] = {-128, -128, -128, -128};
  if (active) {
    v4i qa[NKS];
#pragma unroll
    for (int s = 0; s < NKS; ++s) qa[s] = *(const v4i*)(Qh + (size_t)(i0 + col) * DK + s * 64 + g * 16);
    bool take_hi[4];
    int src_addr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int arow = 4 * g + i;
      take_hi[i] = (col + arow) < 16;                           // as a source lane
      src_addr[i] = (g * 16 + ((col - arow) & 15)) * 4;         // as a destination lane
    }
    const int64_t half = (int64_t)1 << (a.shift_s - 1);
    for (int c = c_begin; c < c_end; ++c) {
      for (int sub = 0; sub < 4; ++sub) {
        const int j0 = c * KCHUNK + sub * 16;
        const int bu_j = bu[j0 + col];
        v4i cs = {bu_j, bu_j, bu_j, bu_j};
#pragma unroll
        for (int s = 0; s < NKS; ++s) {
          const v4i kf = *(const v4i*)(Kh + (size_t)(j0 + col) * DK + s * 64 + g * 16);
          cs = __builtin_amdgcn_mfma_i32_16x16x64_i8(qa[s], kf, cs, 0, 0, 0);
        }
        // relative position of (row i0, key j0) is table row j0 - i0 + T - 1
        const int rlo = P_PADLO + j0 - i0 + T - 1 - 16, rhi = rlo + 16;
        const int bvl = bv[rlo + col], bvh = bv[rhi + col];
        v4i glo = {bvl, bvl, bvl, bvl}, ghi = {bvh, bvh, bvh, bvh};
#pragma unroll
        for (int s = 0; s < NKS; ++s) {
          const v4i pl = *(const v4i*)(Ph + (size_t)(rlo + col) * DK + s * 64 + g * 16);
          const v4i ph = *(const v4i*)(Ph + (size_t)(rhi + col) * DK + s * 64 + g * 16);
          glo = __builtin_amdgcn_mfma_i32_16x16x64_i8(qa[s], pl, glo, 0, 0, 0);
          ghi = __builtin_amdgcn_mfma_i32_16x16x64_i8(qa[s], ph, ghi, 0, 0, 0);
        }
        const int j = j0 + col;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int sel = take_hi[i] ? ghi[i] : glo[i];
          const int pt = __builtin_amdgcn_ds_bpermute(src_addr[i], sel);
          const int64_t t = (int64_t)a.m_c * cs[i] + (int64_t)a.m_p * pt + half;
          const int64_t r = t >> a.shift_s;
          int sv = r < -127 ? -127 : (r > 127 ? 127 : (int)r);
          if (j >= L) sv = -128;
          mx[i] = sv > mx[i] ? sv : mx[i];
          srows[(4 * g + i) * srow + j] = (int8_t)sv;
        }
      }
    }
  }
  // row max over the 16 key lanes of each row group
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int v = mx[i];
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      const int u = __shfl_xor(v, o);
      v = u > v ? u : v;
    }
    mx[i] = v;
  }
  if (col == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) smax[w * 16 + 4 * g + i] = mx[i];
  }
  __syncthreads();

  // from here on lane (g, col) works on row `col` of its tile and keys g*16.. of a chunk
  int M = -128;
#pragma unroll
  for (int k2 = 0; k2 < WPT; ++k2) {
    const int v = smax[(rt + NRT * k2) * 16 + col];
    M = v > M ? v : M;
  }

  // ---------------- phase 2: row sums of the integer exp
  uint32_t sum = 0;
  if (active) {
    for (int c = c_begin; c < c_end; ++c) {
      const v4i sv16 = *(const v4i*)(srows + col * srow + c * KCHUNK + g * 16);
#pragma unroll
      for (int wd = 0; wd < 4; ++wd)
#pragma unroll
        for (int by = 0; by < 4; ++by) {
          const int s = (int)(int8_t)((uint32_t)sv16[wd] >> (8 * by));
          if (s != -128) sum += iexp_int(M - s, a.q_ln2, a.q_b, a.q_c);
        }
    }
  }
  sum += __shfl_xor(sum, 16);
  sum += __shfl_xor(sum, 32);
  if (g == 0) ssum[w * 16 + col] = sum;
  __syncthreads();
  uint32_t tot = 0;
#pragma unroll
  for (int k2 = 0; k2 < WPT; ++k2) tot += ssum[(rt + NRT * k2) * 16 + col];
  const uint64_t F = tot ? ((uint64_t)1 << 32) / tot : 0;

  // ---------------- phase 3: a = softmax codes, A.V on MFMA
  v4i acc[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) acc[nt] = (v4i){0, 0, 0, 0};
  if (active) {
    for (int c = c_begin; c < c_end; ++c) {
      const v4i sv16 = *(const v4i*)(srows + col * srow + c * KCHUNK + g * 16);
      v4i af;
#pragma unroll
      for (int wd = 0; wd < 4; ++wd) {
        uint32_t packed = 0;
#pragma unroll
        for (int by = 0; by < 4; ++by) {
          const int s = (int)(int8_t)((uint32_t)sv16[wd] >> (8 * by));
          uint32_t av = 0;
          if (s != -128) {
            const uint64_t e = iexp_int(M - s, a.q_ln2, a.q_b, a.q_c);
            const uint64_t v = (e * F) >> 24;
            av = v > 255 ? 255u : (uint32_t)v;
          }
          packed |= ((av ^ 0x80u) & 0xffu) << (8 * by);  // a - 128 as a signed byte
        }
        af[wd] = (int)packed;
      }
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const v4i vf = *(const v4i*)(VTh + (size_t)(nt * 16 + col) * T_al + c * KCHUNK + g * 16);
        acc[nt] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, vf, acc[nt], 0, 0, 0);
      }
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int n = nt * 16 + col;
      const int corr = 128 * (vs[(size_t)c_end * DK + n] - vs[(size_t)c_begin * DK + n]);
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[nt][i] += corr;
    }
  }
  __syncthreads();  // all waves are done with the scores; reuse LDS for the partials
  // lane holds context channel n = nt*16 + col of rows 4g + i
#pragma unroll
  for (int nt = 0; nt < NT; ++nt)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[(w * 16 + 4 * g + i) * DK + nt * 16 + col] = acc[nt][i];
  __syncthreads();
  const int half_o = 1 << (a.shift_o - 1);
  for (int idx = threadIdx.x; idx < 16 * NRT * DK; idx += 256) {
    const int row = idx / DK, n = idx - row * DK;
    const int rt2 = row >> 4, ar = row & 15;
    const int i = i_base + row;
    if (i >= T) continue;
    int v = 0;
    if (i < L) {
      int tot2 = 0;
#pragma unroll
      for (int k2 = 0; k2 < WPT; ++k2) tot2 += red[((rt2 + NRT * k2) * 16 + ar) * DK + n];
      const int64_t r = ((int64_t)tot2 * a.m_o + half_o) >> a.shift_o;
      v = r < -127 ? -127 : (r > 127 ? 127 : (int)r);
    }
    a.ctx[((size_t)b * T + i) * a.d + (size_t)h * DK + n] = (int8_t)v;
  }
}

// ---------------------------------------------------------------------------
// Rank-1 bias terms and prefix sums of V over 64-key chunks.
struct BiasArgs {
  const int8_t *k, *vt, *p, *u, *v;
  int32_t *bu, *bv, *vsum;
  int BH, H, T_al, DK, p_rows;
};

__global__ __launch_bounds__(256) void bias_terms(BiasArgs a) {
  const long n_bu = (long)a.BH * a.T_al;
  const long n_bv = (long)a.H * a.p_rows;
  const long n_vs = (long)a.BH * a.DK;
  long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx < n_bu) {
    const long bh = idx / a.T_al;
    const int h = (int)(bh % a.H);
    const int8_t* kr = a.k + idx * a.DK;
    const int8_t* ur = a.u + (size_t)h * a.DK;
    int acc = 0;
    for (int kk = 0; kk < a.DK; ++kk) acc += (int)ur[kk] * (int)kr[kk];
    a.bu[idx] = acc;
    return;
  }
  idx -= n_bu;
  if (idx < n_bv) {
    const int h = (int)(idx / a.p_rows);
    const int8_t* pr = a.p + idx * a.DK;
    const int8_t* vr = a.v + (size_t)h * a.DK;
    int acc = 0;
    for (int kk = 0; kk < a.DK; ++kk) acc += (int)vr[kk] * (int)pr[kk];
    a.bv[idx] = acc;
    return;
  }
  idx -= n_bv;
  if (idx < n_vs) {
    const long bh = idx / a.DK;
    const int n = (int)(idx % a.DK);
    const int8_t* row = a.vt + idx * a.T_al;
    int32_t* out = a.vsum + bh * (long)(a.T_al / KCHUNK + 1) * a.DK + n;
    int run = 0;
    out[0] = 0;
    for (int c = 0; c < a.T_al / KCHUNK; ++c) {
      for (int t = 0; t < KCHUNK; ++t) run += (int)row[c * KCHUNK + t];
      out[(size_t)(c + 1) * a.DK] = run;
    }
  }
}

// ---------------------------------------------------------------------------
// Copies a workspace tensor back to the documented [B][T][d] / [2T-1][d] layouts.
struct GatherArgs {
  const int8_t* src;
  int8_t* dst;
  int which, B, T, T_al, H, DK, d, p_rows;
};

__global__ __launch_bounds__(256) void gather_intermediate(GatherArgs a) {
  const long rows = a.which == 3 ? (long)(2 * a.T - 1) : (long)a.B * a.T;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= rows * a.d) return;
  const long m = idx / a.d;
  const int c = (int)(idx % a.d);
  const int h = c / a.DK, kk = c % a.DK;
  int8_t v;
  if (a.which == 3) {
    v = a.src[((size_t)h * a.p_rows + P_PADLO + m) * a.DK + kk];
  } else if (a.which == 4) {
    v = a.src[idx];
  } else {
    const long b = m / a.T, t = m % a.T;
    const size_t bh = (size_t)b * a.H + h;
    if (a.which == 2)
      v = a.src[(bh * a.DK + kk) * a.T_al + t];
    else
      v = a.src[(bh * a.T_al + t) * a.DK + kk];
  }
  a.dst[idx] = v;
}

// ---------------------------------------------------------------------------
template <int DK, int NRT>
static hipError_t launch_attn_cfg(const AttnArgs& args, int B, int H, int T, int T_al, hipStream_t st) {
  const int sbuf = 16 * NRT * (T_al + SCORE_PAD);
  const int red = 4 * 16 * DK * 4;
  const size_t shmem = (size_t)(sbuf > red ? sbuf : red) + 2 * 64 * 4;
  hipError_t e = hipFuncSetAttribute((const void*)relpos_attn_core<DK, NRT>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)shmem);
  if (e != hipSuccess) return e;
  const int rows_per_wg = 16 * NRT;
  dim3 grid((T + rows_per_wg - 1) / rows_per_wg, H, B);
  hipLaunchKernelGGL((relpos_attn_core<DK, NRT>), grid, dim3(256), shmem, st, args);
  return hipGetLastError();
}

// Largest query block (16, 32 or 64 rows) whose scores fit the LDS budget.
int attn_rows_per_block(int T_al) {
  const int budget = 160 * 1024 - 1024;
  for (int nrt = 4; nrt >= 1; nrt >>= 1)
    if (16 * nrt * (T_al + SCORE_PAD) <= budget) return 16 * nrt;
  return 0;
}

hipError_t launch_attention(const RunShape& rs, const Scalars& sc, const Workspace& ws, const Lengths& lens,
                            hipStream_t st) {
  AttnArgs a{};
  a.q = ws.q;
  a.k = ws.k;
  a.vt = ws.vt;
  a.p = ws.p;
  a.bu = ws.bu;
  a.bv = ws.bv;
  a.vsum = ws.vsum;
  a.ctx = ws.ctx;
  a.lens = lens;
  a.T = rs.T;
  a.T_al = rs.T_al;
  a.H = rs.H;
  a.d = rs.d;
  a.p_rows = p_rows(rs.T_al);
  a.m_c = sc.m_c;
  a.m_p = sc.m_p;
  a.shift_s = sc.shift_s;
  a.m_o = sc.m_o;
  a.shift_o = sc.shift_o;
  a.q_ln2 = sc.q_ln2;
  a.q_b = sc.q_b;
  a.q_c = sc.q_c;
  const int rows = attn_rows_per_block(rs.T_al);
  if (rs.DK == 128) {
    if (rows == 64) return launch_attn_cfg<128, 4>(a, rs.B, rs.H, rs.T, rs.T_al, st);
    if (rows == 32) return launch_attn_cfg<128, 2>(a, rs.B, rs.H, rs.T, rs.T_al, st);
    if (rows == 16) return launch_attn_cfg<128, 1>(a, rs.B, rs.H, rs.T, rs.T_al, st);
  } else if (rs.DK == 64) {
    if (rows == 64) return launch_attn_cfg<64, 4>(a, rs.B, rs.H, rs.T, rs.T_al, st);
    if (rows == 32) return launch_attn_cfg<64, 2>(a, rs.B, rs.H, rs.T, rs.T_al, st);
    if (rows == 16) return launch_attn_cfg<64, 1>(a, rs.B, rs.H, rs.T, rs.T_al, st);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_bias_terms(const RunShape& rs, const Weights& w, const Workspace& ws, const Lengths& lens,
                             hipStream_t st) {
  (void)lens;
  BiasArgs a{};
  a.k = ws.k;
  a.vt = ws.vt;
  a.p = ws.p;
  a.u = w.u;
  a.v = w.v;
  a.bu = ws.bu;
  a.bv = ws.bv;
  a.vsum = ws.vsum;
  a.BH = rs.B * rs.H;
  a.H = rs.H;
  a.T_al = rs.T_al;
  a.DK = rs.DK;
  a.p_rows = p_rows(rs.T_al);
  const long total = (long)a.BH * a.T_al + (long)a.H * a.p_rows + (long)a.BH * a.DK;
  hipLaunchKernelGGL(bias_terms, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gather_intermediate(const RunShape& rs, const Workspace& ws, int which, int8_t* dst,
                                      hipStream_t st) {
  GatherArgs a{};
  a.src = which == 0 ? ws.q : which == 1 ? ws.k : which == 2 ? ws.vt : which == 3 ? ws.p : ws.ctx;
  a.dst = dst;
  a.which = which;
  a.B = rs.B;
  a.T = rs.T;
  a.T_al = rs.T_al;
  a.H = rs.H;
  a.DK = rs.DK;
  a.d = rs.d;
  a.p_rows = p_rows(rs.T_al);
  const long rows = which == 3 ? (long)(2 * rs.T - 1) : (long)rs.B * rs.T;
  const long total = rows * rs.d;
  hipLaunchKernelGGL(gather_intermediate, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace ipk
