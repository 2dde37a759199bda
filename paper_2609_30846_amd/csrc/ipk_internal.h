// Internal declarations of the ipk library (not part of the C ABI).
//
// Workspace layout in HBM for one run of (B, T), with T_al = T rounded up to the
// 64-key chunk and H heads of width DK.  Every layout is chosen so that an MFMA
// operand fragment of the attention core (16 rows x 64 bytes of K-dimension) is a
// contiguous 1 KB block in lane order: lane (g, col) of the fragment's load, which
// feeds row col with bytes 16 g .. 16 g + 15, finds them at byte 16 (16 g + col).
// A load whose lanes walk 16-byte pieces in address order streams about twice as
// fast through the vector memory path as one whose neighbouring lanes sit 64 bytes
// apart.
//   q, k   int8  [B][H] fragment-major rows: row t, channel kk sits at
//                frag_index(t, kk) = (t/16)*16*DK + (kk/64)*1024
//                                    + (16*((kk%64)/16) + t%16)*16 + kk%16
//   vt     int8  [B][H] V transposed, chunk-major (the fragment rows are channels,
//                its K-dimension keys): key t, channel kk sits at
//                vt_index(t, kk) = (t/64)*64*DK + (kk/16)*1024
//                                  + (16*((t%64)/16) + kk%16)*16 + t%16;
//                keys T .. T_al-1 hold zeros
//   p      int8  [H] fragment-major rows of the projected relative-position table;
//                table row r is stored at row p_base + r, where p_base >= P_PADLO is
//                chosen per run so that the table row j-i+T-1 of every 16-query by
//                16-key tile starts a 16-row block.  The rows around the table keep
//                every padded tile in bounds (their contents are never used).
//   ctx    int8  [B][T][d]          attention output, heads concatenated
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ipk {

constexpr int KCHUNK = 64;    // keys per chunk of the A.V contraction (MFMA K = 64)
constexpr int P_PADLO = 128;  // rows kept before relative-position row 0
constexpr int P_PADHI = 128;  // rows kept after the last table row
constexpr int BUF_WORD3 = 0x00020000;  // buffer resource word 3 for gfx9-family raw loads

inline int round_up(int v, int m) { return (v + m - 1) / m * m; }

// Division by a divisor known only at launch, in integers: the compiler's lowering of a
// 32-bit division uses a floating-point reciprocal.  With m = floor(2^32 / d) + 1,
// floor(x / d) = mulhi(x, m) exactly whenever x d < 2^32 (the error term x (m - 2^32/d)
// / 2^32 stays below 1/d, the smallest gap to the next multiple); d = 1 has m = 0 and
// passes x, through a select rather than a branch (no load waits on another).
struct DivU {
  uint32_t d, m;
};
inline DivU make_div(uint32_t d) { return DivU{d, d <= 1 ? 0u : (uint32_t)((1ull << 32) / d + 1)}; }
__device__ __forceinline__ uint32_t div_u(uint32_t x, const DivU& v) {
  return __umulhi(x, v.m) + (v.m == 0u ? x : 0u);
}
inline int t_aligned(int T) { return round_up(T, KCHUNK); }
inline int p_rows(int T_al) { return P_PADLO + 2 * T_al + P_PADHI; }
// Row of table row 0: the smallest value >= P_PADLO with (p_base + T - 1) % 16 == 0.
inline int p_base_row(int T) { return P_PADLO + (16 - (T - 1) % 16) % 16; }

__host__ __device__ inline size_t frag_index(int row, int kk, int DK) {
  return (size_t)(row >> 4) * (16 * DK) + (size_t)(kk >> 6) * 1024 + ((((kk >> 4) & 3) << 4) + (row & 15)) * 16 +
         (kk & 15);
}
__host__ __device__ inline size_t vt_index(int t, int kk, int DK) {
  return (size_t)(t >> 6) * (64 * DK) + (size_t)(kk >> 4) * 1024 + ((((t >> 4) & 3) << 4) + (kk & 15)) * 16 + (t & 15);
}

struct Workspace {
  int8_t *q, *k, *vt, *p, *ctx;
  int8_t* xln;  // LayerNorm output [B][T][d] of the MHSA module's runs
};

// LayerNorm and residual constants of the MHSA module (Eq. 2) on the device.
struct Residual {
  const int32_t* ln_mult;  // [d]
  const int64_t* ln_bias;  // [d]: ln_bias + 2^(ln_shift - 1), the rounding term folded in
  int32_t ln_shift;
  int32_t m_z, m_y, shift_r;
};

// Fragment order of a weight matrix W [N][K] (N, K multiples of 32) for the A operand of
// v_mfma_i32_32x32x32_i8: the fragment of channels 32 cb .. 32 cb + 31 and bytes
// 32 ks .. 32 ks + 31 is the 1 KB block (cb K/32 + ks), and the lane l that feeds channel
// 32 cb + l % 32 with bytes 32 ks + 16 (l / 32) .. + 15 finds them at byte 16 l of it.
__host__ __device__ inline size_t wfrag_index(int n, int k, int K) {
  return ((size_t)(n >> 5) * (K >> 5) + (k >> 5)) * 1024 + (size_t)(((((k >> 4) & 1) << 5) + (n & 31)) << 4) +
         (k & 15);
}

// Eq. 7 requantization constants of one weight matrix's N output channels (a stack of
// matrices, e.g. Q, K and V, shares one form), on the device as int32 [2][N]:
//  * fast (wide == 0): every part has n <= 16; row 0 holds m' = m 2^(16-n) < 2^23, and
//    `clamp` is one bound A for the whole matrix with A >= ceil(2^23 / m') + 1 for every
//    channel, A < 2^23 and A max(m') + 2^15 < 2^31.  Then clamp8(RS(a, m, n)) =
//    clamp8(floor((clamp(a, -A, A) m' + 2^15) / 2^16)): inside [-A, A] the value is the
//    exact one, past it the result saturates either way (each channel's own bound is at
//    most A), and the 24-bit product cannot overflow.  Such an A exists when the largest
//    m' is below about 2^8 times the smallest nonzero one;
//  * wide (wide == 1): row 0 holds m, row 1 the channel's shift n, and the epilogue
//    evaluates Eq. 7 in 64-bit integers.
struct Requant {
  const int32_t* req;
  int wide;
  int clamp;  // A of the fast form
};

struct Weights {
  int8_t* w_qkv;       // [3d][d]: w_q, w_k, w_v stacked, in fragment order (wfrag_index)
  int8_t* w_pos;       // [d][d], in fragment order
  int8_t* w_out;       // [d][d], in fragment order
  int8_t *u, *v;       // [H][DK]
  uint32_t* etab;      // [256] I-BERT integer exp of every score distance (0 at 255)
  // Eq. 7 constants per output channel (Requant)
  Requant rq_qkv;  // 3d channels: Q, K, V stacked (one form for the three)
  Requant rq_pos;  // d channels
  Requant rq_out;  // d channels
};

struct Scalars {
  int32_t m_c, m_p, shift_s;
  int32_t m_o, shift_o;
  int32_t q_ln2, q_b, q_c;
  // Eq. 11 as evaluated by the attention core: in 32-bit integers
  // (t = mc24 c + mp24 p + bias32 with the biased code in bits 16..23; exact when the
  // bound on |t| proven at create holds), otherwise in 64-bit integers.
  bool fs_wide;
  int32_t fs_mc24, fs_mp24, fs_bias32;
};

// Per-utterance valid lengths, passed by value to the kernels that mask.
struct Lengths {
  int32_t len[256];
};

struct RunShape {
  int B, T, T_al, H, DK, d;
  int p_base;  // workspace row of relative-position table row 0
  int p_rows;  // rows per head of the projected table's buffer
};

// Optional timing events of one kernel launch, carried by the dispatch itself
// (hipExtLaunchKernel): start is stamped when the kernel starts, stop when it ends.
struct LaunchEv {
  hipEvent_t start = nullptr, stop = nullptr;
};

template <typename K, typename... Args>
inline hipError_t launch_kernel(K kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t st, const LaunchEv& ev,
                                Args... args) {
  if (ev.start || ev.stop)
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, st, ev.start, ev.stop, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, shmem, st, args...);
  return hipGetLastError();
}

// Enqueue the kernels of one run; return the first HIP error.
// pos_table == nullptr: Q|K|V only (the projected table is already in ws.p)
hipError_t launch_projections(const RunShape& rs, const Weights& w, const Workspace& ws, const int8_t* x,
                              const int8_t* pos_table, hipStream_t st, const LaunchEv& ev = {});
// The I-BERT integer exp of every score distance into tab[256] (create time).
hipError_t launch_iexp_table(uint32_t* tab, int q_ln2, int q_b, int q_c, hipStream_t st);
hipError_t launch_attention(const RunShape& rs, const Weights& w, const Scalars& sc, const Workspace& ws,
                            const Lengths& lens, hipStream_t st, const LaunchEv& ev = {});
// res != nullptr: the epilogue adds the residual, y := clamp8(RS(m_z z1 + m_y y, 1, shift_r))
hipError_t launch_out_projection(const RunShape& rs, const Weights& w, const Workspace& ws, int8_t* y,
                                 hipStream_t st, const LaunchEv& ev = {}, const Residual* res = nullptr,
                                 const int8_t* z1 = nullptr);
// The position projection alone, of a table of T_table rows, into `p` (rs.p_base, rs.p_rows).
hipError_t launch_pos_projection(const RunShape& rs, const Weights& w, int8_t* p, const int8_t* pos_table,
                                 hipStream_t st);
// Integer LayerNorm of rows [B][T][d] of z into ws.xln.
hipError_t launch_layernorm(const RunShape& rs, const Residual& r, const int8_t* z, int8_t* out, hipStream_t st,
                            const LaunchEv& ev = {});
// The feed-forward module (Eq. 1): the Swish table of every int8 input, W1 with the
// Swish in its epilogue (x [rows][d] -> o [rows][d_ff]), W2 with the residual add in
// its epilogue (o -> z_out [rows][d]).
hipError_t launch_swish_table(uint8_t* tab, long long q_c, long long q_1, long long m, int shift, hipStream_t st);
hipError_t launch_ffn_up(const int8_t* x, int rows, int d, int d_ff, const int8_t* w1, const Requant& rq1,
                         const uint8_t* swtab, int8_t* o, hipStream_t st);
// A row-major linear layer y = clamp8(RS(x W^T)) of `rows` rows (K -> N), and one with the
// residual add z_out = clamp8(RS(m_z z + m_y y, 1, shift_r)) in its epilogue.
hipError_t launch_linear(const int8_t* x, int rows, int K, int N, const int8_t* w, const Requant& rq, int8_t* y,
                         hipStream_t st);
hipError_t launch_linear_resid(const int8_t* x, int rows, int N, int K, const int8_t* w, const Requant& rq,
                               const int8_t* z, int m_z, int m_y, int shift_r, int8_t* z_out, hipStream_t st);

// The middle of the convolution module (Eq. 5): GLU, depthwise convolution with folded
// BatchNorm to the INT16 grid, Swish, requantization to PW2's int8 input.
struct ConvMiddle {
  const int8_t* w_dw;     // [d][9]
  const int32_t* bias_dw;  // [d]
  const int32_t* mult_dw;  // [d]
  int shift_dw;
  long long glu_qc, glu_q1, m_glu;
  int shift_glu;
  const int8_t* swtab16;  // [65535] Swish output of each int16 value v, at v + 32767
  const int8_t* glutab;   // [256][256] GLU output of each int8 pair (a, b), at (a + 128) 256 + b + 128
};
hipError_t launch_swish16_table(int8_t* tab, long long q_c, long long q_1, long long m, int shift, hipStream_t st);
hipError_t launch_glu_table(int8_t* tab, long long q_c, long long q_1, long long m, int shift, hipStream_t st);
hipError_t launch_conv_middle(const ConvMiddle& m, const int8_t* u, const Lengths& lens, int B, int T, int d,
                              int8_t* o, int16_t* v, hipStream_t st);
hipError_t launch_layernorm_rows(long rows, int d, const Residual& r, const int8_t* z, int8_t* out, hipStream_t st);

// Workgroup shapes of the attention core for a run: the first shape's nqb1 query
// blocks per (utterance, head), then (c2.ksplit != 0) the second shape's nqb2 blocks
// for the remaining queries.  c1.ksplit == 0 when T_al does not fit LDS.
struct AttnCfg {
  int ksplit, ntl;  // key splits per query set, 16-query tiles per wave
};
struct AttnPlan {
  AttnCfg c1;
  int nqb1;
  AttnCfg c2;
  int nqb2;
};
AttnPlan attn_plan(int DK, int T_al, long bh_count, int T);

// Rearranges a row-major int8 matrix [N][K] into fragment order (wfrag_index).
hipError_t pack_weight_fragments(const int8_t* w, int8_t* dst, int N, int K, hipStream_t st);

// The no-allocation run's workspace on the current device: a static device array of
// `bytes` bytes (its address looked up once per device).
hipError_t noalloc_scratch(uint8_t** base, size_t* bytes);

hipError_t launch_gather_intermediate(const RunShape& rs, const Workspace& ws, int which, int8_t* dst,
                                      hipStream_t st);

}  // namespace ipk
