// Internal declarations of the ipk library (not part of the C ABI).
//
// Workspace layout in HBM for one run of (B, T), with T_al = T rounded up to the
// 64-key chunk and H heads of width DK:
//   q, k   int8  [B][H][T_al][DK]   head-major rows: one 128-byte (DK=128) line per token
//   vt     int8  [B][H][DK][T_al]   V transposed, so the A.V contraction reads keys
//                                   contiguously for each output channel
//   p      int8  [H][P_ROWS][DK]    projected relative-position table; table row r
//                                   is stored at row P_PADLO + r, and the rows around
//                                   it keep the index map j-i+T-1 in bounds for every
//                                   padded tile (their contents are never used)
//   bu     int32 [B][H][T_al]       u . K_j  (rank-1 part of the content score)
//   bv     int32 [H][P_ROWS]        v . P_r  (rank-1 part of the position score)
//   vsum   int32 [B][H][T_al/64+1][DK] prefix sums of V over 64-key chunks
//   ctx    int8  [B][T][d]          attention output, heads concatenated
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ipk {

constexpr int KCHUNK = 64;    // keys per chunk of the A.V contraction (MFMA K = 64)
constexpr int P_PADLO = 128;  // rows kept before relative-position row 0
constexpr int P_PADHI = 128;  // rows kept after the last table row

inline int round_up(int v, int m) { return (v + m - 1) / m * m; }
inline int t_aligned(int T) { return round_up(T, KCHUNK); }
inline int p_rows(int T_al) { return P_PADLO + 2 * T_al + P_PADHI; }

struct Workspace {
  int8_t *q, *k, *vt, *p, *ctx;
  int32_t *bu, *bv, *vsum;
};

struct Weights {
  int8_t* w_qkv;       // [3d][d]: w_q, w_k, w_v stacked
  int8_t* w_pos;       // [d][d]
  int8_t* w_out;       // [d][d]
  int8_t *u, *v;       // [H][DK]
  int32_t* mult_qkv;   // [3d]
  int32_t* shift_qkv;  // [3d]
  int32_t* mult_pos;   // [d]
  int32_t* shift_pos;  // [d]
  int32_t* mult_out;   // [d]
  int32_t* shift_out;  // [d]
};

struct Scalars {
  int32_t m_c, m_p, shift_s;
  int32_t m_o, shift_o;
  int32_t q_ln2, q_b, q_c;
};

// Per-utterance valid lengths, passed by value to the kernels that mask.
struct Lengths {
  int32_t len[256];
};

struct RunShape {
  int B, T, T_al, H, DK, d;
};

// Enqueue the kernels of one run; return the first HIP error.
hipError_t launch_projections(const RunShape& rs, const Weights& w, const Workspace& ws, const int8_t* x,
                              const int8_t* pos_table, hipStream_t st);
hipError_t launch_bias_terms(const RunShape& rs, const Weights& w, const Workspace& ws, const Lengths& lens,
                             hipStream_t st);
hipError_t launch_attention(const RunShape& rs, const Scalars& sc, const Workspace& ws, const Lengths& lens,
                            hipStream_t st);
hipError_t launch_out_projection(const RunShape& rs, const Weights& w, const Workspace& ws, int8_t* y,
                                 hipStream_t st);
hipError_t launch_gather_intermediate(const RunShape& rs, const Workspace& ws, int which, int8_t* dst,
                                      hipStream_t st);

}  // namespace ipk
