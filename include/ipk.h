/*
 * ipk: integer-only relative-positional multi-head self-attention on MI355X (gfx950).
 *
 * The block is the MHSA term of the Conformer block (Eq. 2) of "I-Parakeet:
 * Integer-Only Conformer ASR on Mobile NPU", computed entirely in integers as in
 * Sec. 3.1:
 *
 *   Q, K, V  = clamp8(RS(x W^T, mult[c], shift))            (Eq. 7, per channel)
 *   P        = clamp8(RS(pe W_pos^T, mult_pos[c], shift))    (Eq. 7)
 *   c_ij     = (Q_i + u) . K_j                                (Eq. 8, content)
 *   p_ij     = (Q_i + v) . P_{j-i+T-1}                        (Eq. 8 with Phi as
 *                                                              an index map)
 *   s_ij     = clamp8(RS(m_c c_ij + m_p p_ij, 1, shift_s))    (Eq. 11)
 *   a_ij     = I-BERT integer softmax of s_i. (8-bit, grid 2^-8)
 *   ctx_i    = clamp8(RS(sum_j a_ij V_j, m_o, shift_o))       (Eq. 7)
 *   y        = clamp8(RS(ctx W_out^T, mult_out[c], shift))    (Eq. 7)
 *
 * with RS(a, m, n) = floor((a m + 2^(n-1)) / 2^n) (round to nearest, ties up) and
 * clamp8(v) = min(max(v, -127), 127) (symmetric int8 grid, Eq. 6 with b = 8).
 * The I-BERT softmax over the valid keys j < L_b of row i is: M = max_j s_ij;
 * d = M - s_ij; z = floor(d / q_ln2); r = z q_ln2 - d; e_ij = ((r + q_b)^2 + q_c) >> z;
 * F = floor(2^32 / sum_j e_ij); a_ij = min(floor(e_ij F / 2^24), 255).
 * Rows i >= L_b of y are zero.
 *
 * All run-time arguments are integers; real scales never reach the library.
 * Every entry point returns an ipk_status and never throws.  The text of the
 * last error on the calling thread is available from ipk_last_error().
 */
#ifndef IPK_H
#define IPK_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define IPK_ABI_VERSION 5

/* Status codes. */
typedef enum ipk_status {
  IPK_OK = 0,
  IPK_ERR_INVALID_ARG = -1,   /* a pointer, size or constant outside its documented range */
  IPK_ERR_UNSUPPORTED = -2,   /* valid per the method but outside this implementation's limits */
  IPK_ERR_OUT_OF_MEMORY = -3, /* a device or host allocation failed */
  IPK_ERR_HIP = -4            /* the HIP runtime reported an error (launch, copy, device) */
} ipk_status;

/* Implementation limits (checked by ipk_relpos_attn_create / _run). */
#define IPK_MAX_BATCH 256 /* utterances per call */
#define IPK_MAX_T 8192    /* frames per utterance */

/*
 * Block descriptor, read only during ipk_relpos_attn_create.
 *
 * Shapes: d_model = n_heads * d_k, d_k in {64, 128}; max_batch in [1, IPK_MAX_BATCH]
 * and max_T in [1, IPK_MAX_T] size the handle's workspace.  The attention core keeps a
 * workgroup's score rows on chip, which limits max_T to 8000 (IPK_ERR_UNSUPPORTED above).
 *
 * Weights (DEVICE pointers, int8, [d_out = d_model][d_in = d_model], row-major,
 * nn.Linear convention y = x W^T): w_q, w_k, w_v (the three projections of
 * Eq. 8's Q, K, V), w_pos (projection of the sinusoidal relative-position
 * embeddings, Sec. 3.1), w_out (output projection).
 * pos_bias_u, pos_bias_v (DEVICE, int8, [n_heads][d_k]): the learned biases u, v of
 * Eq. 8, on the grid of Q.
 *
 * Requantization (HOST pointers, int32, [d_model]): mult_{q,k,v,pos,out}[c] is
 * the fixed-point multiplier m of Eq. 7 for output channel c (per-channel weight
 * scales, Sec. 2.2; per-tensor scales are the case of equal entries), with the
 * shared shift shift_{q,k,v,pos,out} (the paper's n = 16).
 * Fused score (Eq. 11): m_c, m_p, shift_s.  Context requant (A V, Eq. 7): m_o, shift_o.
 * Ranges: 0 <= mult < 2^23 for every multiplier; 1 <= shift <= 40.
 *
 * Softmax constants (I-BERT integer exp for the score grid S_s):
 * q_ln2 = floor(ln2 / S_s) >= 1, q_b = floor(b / S_s) >= 0,
 * q_c = floor(c / (a S_s^2)) >= 0 with (a, b, c) = (0.3585, 1.353, 0.344).
 * Implementation limits: the polynomial (r + q_b)^2 + q_c must stay below 2^24
 * for r in (-q_ln2, 0], must be at least 2^8 at r = 0, and max_T times its maximum
 * must stay below 2^32 (IPK_ERR_UNSUPPORTED otherwise).
 *
 * Zero points zp_x, zp_y must be 0: quantization is symmetric (Eq. 6).
 */
typedef struct ipk_relpos_attn_desc {
  int32_t d_model, n_heads, d_k;
  int32_t max_batch, max_T;
  const int8_t *w_q, *w_k, *w_v, *w_pos, *w_out;
  const int8_t *pos_bias_u, *pos_bias_v;
  const int32_t *mult_q, *mult_k, *mult_v, *mult_pos, *mult_out;
  int32_t shift_q, shift_k, shift_v, shift_pos, shift_out;
  int32_t m_c, m_p, shift_s;
  int32_t m_o, shift_o;
  int32_t q_ln2, q_b, q_c;
  int32_t zp_x, zp_y;
} ipk_relpos_attn_desc;

typedef struct ipk_relpos_attn ipk_relpos_attn_t;

/*
 * Validates the descriptor, allocates the handle and its device workspace for
 * (max_batch, max_T), and copies the weights, biases and multipliers into it on
 * the current HIP device.  Synchronizes its own copies, so the caller may free its
 * buffers when it returns.
 * Returns IPK_OK and sets *out, or a negative status with *out = NULL and nothing
 * leaked (IPK_ERR_INVALID_ARG, IPK_ERR_UNSUPPORTED, IPK_ERR_OUT_OF_MEMORY, IPK_ERR_HIP).
 */
int ipk_relpos_attn_create(const ipk_relpos_attn_desc* desc, ipk_relpos_attn_t** out);

/*
 * Runs the block on `stream` (a hipStream_t; NULL is the default stream).
 * x        DEVICE int8 [B][T][d_model]   block input
 * pos_table DEVICE int8 [2T-1][d_model]  sinusoidal relative-position table; row r
 *                                        holds relative position T-1-r; NULL uses the
 *                                        projection kept by ipk_relpos_attn_cache_positions
 * lengths  HOST int32 [B] valid frames L_b in [1, T], or NULL for all T; exactly B
 *          entries are read (the array must hold them), and the values are captured
 *          when the call returns (the array may be reused at once)
 * y        DEVICE int8 [B][T][d_model]   block output; rows t >= L_b are zero
 * x, pos_table and y must be 16-byte aligned.
 * The call is asynchronous: it enqueues kernels and returns.  Pointers are borrowed
 * until the stream work completes.  The handle's workspace is shared by all calls:
 * calls on one handle must be ordered on one stream (calls on different streams
 * race).  x and y may not overlap.
 * Errors: IPK_ERR_INVALID_ARG (null handle/x/y, B < 1, T < 1, B > max_batch,
 * T > max_T, a length outside [1, T], a NULL pos_table with no kept projection of at
 * least T rows); IPK_ERR_HIP (launch failure).
 * On an error nothing is enqueued.
 */
int ipk_relpos_attn_run(ipk_relpos_attn_t* h, const int8_t* x, const int8_t* pos_table, const int32_t* lengths,
                        int32_t B, int32_t T, int8_t* y, void* stream);

/*
 * ipk_relpos_attn_run without any device allocation, for callers that cannot allocate
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * Same arguments, results and errors as ipk_relpos_attn_run; the run's workspace (Q,
 * K, V^T, the projected position table unless pos_table is NULL, and the context)
 * lives in one static device array of IPK_NOALLOC_SCRATCH_BYTES per GPU instead of
 * the handle's: the library's code object holds it, each GPU the library
 * runs on keeps its copy until the process ends, and its address is looked up on the
 * device's first call.  The call allocates nothing and calls no allocating routine.
 * Workspace bytes, each part rounded up to 256:
 *   3 B H T_al d_k + H (2 T_al + 256) d_k (only with a pos_table) + B T d_model,
 *   T_al = T rounded up to 64
 * (one 2500-frame utterance at d_model 1024, 8 heads: 15.9 MB; 16 x 375 frames:
 * 26.1 MB).
 * All no-allocation calls on one GPU share that array, whatever their handle or
 * stream, and it keeps the last call's contents (nothing in it has to start at zero:
 * every byte a run reads was written by the same run, or is masked): calls that
 * overlap on one GPU race, so order them (one stream, or events).  After such a call,
 * ipk_relpos_attn_intermediate reads the array, valid until the next one on the GPU.
 * Errors: those of ipk_relpos_attn_run, and IPK_ERR_UNSUPPORTED when (B, T) needs more
 * than IPK_NOALLOC_SCRATCH_BYTES (nothing is enqueued); IPK_ERR_HIP when the array's
 * address cannot be looked up.
 */
#define IPK_NOALLOC_SCRATCH_BYTES (32u * 1024u * 1024u)
int ipk_relpos_attn_run_noalloc(ipk_relpos_attn_t* h, const int8_t* x, const int8_t* pos_table,
                                const int32_t* lengths, int32_t B, int32_t T, int8_t* y, void* stream);

/* Frees the handle and its workspace after synchronizing the device; NULL is a no-op.
 * Returns IPK_OK (or IPK_ERR_HIP if the device reported an error). */
int ipk_relpos_attn_destroy(ipk_relpos_attn_t* h);

/*
 * Copies one intermediate of the last run from its workspace (the handle's, or the
 * GPU's shared array after ipk_relpos_attn_run_noalloc) into a caller buffer (DEVICE
 * pointer `dst` of `bytes` bytes), on `stream`, for tests and debugging.  Layouts for
 * the last run's (B, T):
 *   IPK_INTER_Q, IPK_INTER_K:  int8 [B][T][d_model]
 *   IPK_INTER_V:               int8 [B][T][d_model]
 *   IPK_INTER_P:               int8 [2T-1][d_model]
 *   IPK_INTER_CTX:             int8 [B][T][d_model] (attention output before W_out)
 *   IPK_INTER_XLN:             int8 [B][T][d_model] (LayerNorm output; only after
 *                              ipk_mhsa_residual_run)
 * Errors: IPK_ERR_INVALID_ARG (no run yet, unknown `which`, bytes too small, null,
 * IPK_INTER_XLN when the last run was not ipk_mhsa_residual_run), IPK_ERR_HIP.
 */
enum { IPK_INTER_Q = 0, IPK_INTER_K = 1, IPK_INTER_V = 2, IPK_INTER_P = 3, IPK_INTER_CTX = 4, IPK_INTER_XLN = 5 };
int ipk_relpos_attn_intermediate(ipk_relpos_attn_t* h, int32_t which, void* dst, int64_t bytes, void* stream);

/*
 * Stage timing for profiling: the NEXT run on `h` records the IPK_NUM_STAGES + 1
 * caller-created HIP events events[0..3] (hipEvent_t, created with timing enabled)
 * on its stream: events[0..2] when the three stages start (the Q|K|V and position
 * projections; the attention core; the output projection), events[3] when the output projection
 * ends.  The events are carried by the kernel dispatches themselves, so recording
 * them adds no work to the stream.  The events are used once; later runs record
 * nothing until this is called again.  events = NULL clears a pending request.
 * Errors: IPK_ERR_INVALID_ARG (null handle, or a null entry in events).
 */
enum { IPK_NUM_STAGES = 3 };
int ipk_relpos_attn_record_stages(ipk_relpos_attn_t* h, void* const* events);

/*
 * Kernel timing for profiling: enqueues the attention core of the last run on `h`
 * (Eq. 8-11, the integer softmax and A.V: the middle stage above) `count` more times,
 * back to back on `stream`, with that run's shapes, lengths and score path.  It reads
 * the projections the last run left in the handle's workspace (or the kept position
 * projection, as it is now) and rewrites the context there with the same bytes; nothing
 * outside the handle is touched, so two events around the call time the kernel alone,
 * with no event between its launches.  The last run must have used the handle's own
 * workspace (ipk_relpos_attn_run or ipk_mhsa_residual_run, not the no-allocation run,
 * whose array other calls share), on the current device.
 * Errors: IPK_ERR_INVALID_ARG (null handle, no run yet, the last run was the
 * no-allocation one, count outside [1, IPK_MAX_REPEAT], another current device),
 * IPK_ERR_HIP (launch failure).
 */
#define IPK_MAX_REPEAT 100000
int ipk_relpos_attn_repeat_core(ipk_relpos_attn_t* h, int32_t count, void* stream);

/*
 * How the attention core evaluates the fused score of Eq. 11.  Both paths are exact
 * integer arithmetic and give the same bytes.  IPK_SCORE_AUTO (what create selects)
 * takes 32-bit multiply-adds when create proves m_c |c| + m_p |p| plus the rounding and
 * code bias below 2^31 for every possible score (|c|, |p| <= d_k 255 127), and 64-bit
 * ones otherwise; IPK_SCORE_WIDE forces the 64-bit path, so that tests can exercise it on
 * descriptors that would take the 32-bit one.  Takes effect from the next run.
 * ipk_relpos_attn_score_path returns the path the next run takes (IPK_SCORE_NARROW or
 * IPK_SCORE_WIDE), or a negative status.
 * Errors: IPK_ERR_INVALID_ARG (null handle, unknown path).
 */
enum { IPK_SCORE_AUTO = 0, IPK_SCORE_WIDE = 1, IPK_SCORE_NARROW = 2 };
int ipk_relpos_attn_set_score_path(ipk_relpos_attn_t* h, int32_t path);
int ipk_relpos_attn_score_path(const ipk_relpos_attn_t* h);

/*
 * Position projection kept on the handle (Sec. 3.1: q_P depends only on the
 * sinusoidal table and W_pos, so the paper computes it offline).
 * Projects `pos_table` (DEVICE int8 [2 T_table - 1][d_model], row r = relative
 * position T_table-1-r, 16-byte aligned) once, on `stream`, and keeps the result.
 * Later runs (ipk_relpos_attn_run, ipk_mhsa_residual_run) that pass pos_table = NULL
 * use it for any T <= T_table: the table of a shorter T is rows T_table - T ..
 * T_table + T - 2 of the longer one (each row is a function of its relative position
 * only), so the result is byte for byte that of passing the T-row table.  A run that
 * passes a table still projects it and leaves the kept one unchanged.  Calling this
 * again replaces the kept projection (stream-ordered with the runs on `stream`).
 * The first call allocates device memory for max_T (synchronously).
 * Errors: IPK_ERR_INVALID_ARG (null handle or table, misaligned table, T_table
 * outside [1, max_T]); IPK_ERR_OUT_OF_MEMORY; IPK_ERR_HIP.
 * A later run with pos_table = NULL and no kept projection, or T > T_table, fails
 * with IPK_ERR_INVALID_ARG.
 */
int ipk_relpos_attn_cache_positions(ipk_relpos_attn_t* h, const int8_t* pos_table, int32_t T_table, void* stream);

/*
 * The MHSA module of the Conformer block (Eq. 2) on integer grids:
 *   x  = LN(z1)                     integer LayerNorm (I-BERT, Sec. 3.1) into the block's input grid
 *   y  = the block above on x
 *   z2 = clamp8(RS(m_z z1 + m_y y, 1, shift_r))   residual add, both terms moved to z2's grid
 * LayerNorm of a row z of d_model int8 values:
 *   mu    = floor((2 sum_k z_k + d) / (2 d))           (mean, ties up)
 *   sigma = max(1, floor(sqrt(sum_k (z_k - mu)^2)))    (integer square root)
 *   F     = floor(2^31 / sigma)
 *   u_k   = floor((z_k - mu) F / 2)                    (~ 2^30 (z_k - mu) / sigma)
 *   x_k   = clamp8(floor((u_k ln_mult[k] + ln_bias[k] + 2^(ln_shift-1)) / 2^ln_shift))
 * where ln_mult and ln_bias fold LayerNorm's gamma, beta and the move to the block's
 * input grid into one fixed-point step per channel.
 * Ranges: |ln_mult[k]| < 2^24, |ln_bias[k]| < 2^56, 1 <= ln_shift <= 62;
 * 0 <= m_z, m_y < 2^23; 1 <= shift_r <= 40.
 */
typedef struct ipk_mhsa_residual_desc {
  const int32_t* ln_mult; /* HOST int32 [d_model] */
  const int64_t* ln_bias; /* HOST int64 [d_model] */
  int32_t ln_shift;
  int32_t m_z, m_y, shift_r;
} ipk_mhsa_residual_desc;

/*
 * Attaches (or replaces) the LayerNorm and residual constants of `r` on the handle;
 * the first call allocates the LayerNorm output workspace for (max_batch, max_T).
 * Synchronizes its own copies; the caller may free `r`'s arrays when it returns.
 * Errors: IPK_ERR_INVALID_ARG (null handle/desc/array, a value outside its range);
 * IPK_ERR_OUT_OF_MEMORY; IPK_ERR_HIP.
 */
int ipk_mhsa_residual_set(ipk_relpos_attn_t* h, const ipk_mhsa_residual_desc* r);

/*
 * Runs the MHSA module on `stream`: z2 = z1 + MHSA(LN(z1)) as defined above.
 * z1 DEVICE int8 [B][T][d_model], z2 DEVICE int8 [B][T][d_model], both 16-byte
 * aligned; z2 may be z1 itself (in place) but may not overlap it otherwise.
 * pos_table, lengths, B, T, stream: as for ipk_relpos_attn_run (pos_table may be
 * NULL after ipk_relpos_attn_cache_positions).  Rows t >= L_b of z2 hold the
 * residual of z1 alone (the block's output there is zero).
 * Errors: as ipk_relpos_attn_run, and IPK_ERR_INVALID_ARG when no constants were set.
 * If stage events are pending (ipk_relpos_attn_record_stages), events[0] is stamped
 * when the LayerNorm kernel starts.
 */
int ipk_mhsa_residual_run(ipk_relpos_attn_t* h, const int8_t* z1, const int8_t* pos_table, const int32_t* lengths,
                          int32_t B, int32_t T, int8_t* z2, void* stream);

/*
 * The feed-forward module of the Conformer block (Eq. 1) on integer grids:
 *   x  = LN(z)                                   the LayerNorm above, on ln_mult/ln_bias/ln_shift
 *   h  = clamp8(RS(x W1^T, mult1[c], shift1))    Eq. 7, d_ff outputs per row
 *   q  = -(|h| L + h sw_q1),  L = (min(|h|, sw_qc) - sw_qc)^2 + sw_q1
 *                                                the minimax integer Swish (Sec. 3.2, Eq. 12
 *                                                with Eq. 13's (a*, c*)) on h's grid S:
 *                                                sw_qc = floor(c* / (S/2)),
 *                                                sw_q1 = floor(1 / (a* (S/2)^2)) (negative)
 *   o  = clamp8(RS(q, m_sw, shift_sw))           to W2's input grid
 *   y  = clamp8(RS(o W2^T, mult2[c], shift2))    Eq. 7, d_model outputs per row
 *   z' = clamp8(RS(m_z z + m_y y, 1, shift_r))   the half-step residual (the 0.5 of Eq. 1 in m_y)
 * Shapes: d_model and d_ff multiples of 64, d_model <= 16384, d_ff <= 65536;
 * max_rows >= 1 with max_rows * d_ff < 2^31.
 * Weights (DEVICE, int8, row-major, y = x W^T): w1 [d_ff][d_model], w2 [d_model][d_ff].
 * Multipliers (HOST, int32): mult1 [d_ff], mult2 [d_model], each in [0, 2^23).
 * LayerNorm constants (HOST): as ipk_mhsa_residual_desc.
 * Ranges: shifts in [1, 40] (ln_shift in [1, 62]); 0 <= m_sw, m_z, m_y < 2^23;
 * 0 <= sw_qc < 2^20; |sw_q1| < 2^45; and |q m_sw| + 2^(shift_sw - 1) < 2^62 for every int8 h
 * (IPK_ERR_UNSUPPORTED otherwise).
 */
typedef struct ipk_ffn_desc {
  int32_t d_model, d_ff, max_rows;
  const int8_t *w1, *w2;
  const int32_t *mult1, *mult2;
  int32_t shift1, shift2;
  int32_t sw_qc;
  int64_t sw_q1;
  int32_t m_sw, shift_sw;
  const int32_t* ln_mult;
  const int64_t* ln_bias;
  int32_t ln_shift;
  int32_t m_z, m_y, shift_r;
} ipk_ffn_desc;

typedef struct ipk_ffn ipk_ffn_t;

/* Validates `desc`, allocates the handle and its workspace for max_rows rows and
 * keeps device copies of the weights (in MFMA fragment order), the multipliers and
 * the Swish of every int8 input (a 256-entry table, computed on the device).
 * Synchronizes its own copies.  Returns IPK_OK and sets *out, or a negative status
 * with *out = NULL and nothing leaked. */
int ipk_ffn_create(const ipk_ffn_desc* desc, ipk_ffn_t** out);

/* Runs the module on `stream` over `rows` rows: z DEVICE int8 [rows][d_model] ->
 * z_out DEVICE int8 [rows][d_model], both 16-byte aligned; z_out may be z itself (in
 * place) but may not overlap it otherwise.  Asynchronous; calls on one handle must be
 * ordered on one stream.  Errors: IPK_ERR_INVALID_ARG (null handle or pointer,
 * misalignment, partial overlap, rows outside [1, max_rows]), IPK_ERR_HIP. */
int ipk_ffn_run(ipk_ffn_t* h, const int8_t* z, int32_t rows, int8_t* z_out, void* stream);

/* Copies an intermediate of the last run into `dst` (DEVICE, `bytes` bytes), on
 * `stream`: IPK_FFN_X the LayerNorm output int8 [rows][d_model], IPK_FFN_O the Swish
 * output int8 [rows][d_ff].  Errors: IPK_ERR_INVALID_ARG (no run yet, unknown `which`,
 * bytes too small, null), IPK_ERR_HIP. */
enum { IPK_FFN_X = 0, IPK_FFN_O = 1 };
int ipk_ffn_intermediate(ipk_ffn_t* h, int32_t which, void* dst, int64_t bytes, void* stream);

/* Frees the handle after synchronizing the device; NULL is a no-op. */
int ipk_ffn_destroy(ipk_ffn_t* h);

/*
 * The convolution module of the Conformer block (Eq. 3 and Eq. 5) on integer grids,
 * z' = z + Conv(LN(z)) with Conv = PW2(Swish(BN(DW(GLU(PW1(.)))))):
 *   x  = LN(z)                                      the LayerNorm above
 *   u  = clamp8(RS(x W_pw1^T, mult_pw1[c], shift_pw1))   2 d channels: a = u[:, :d], b = u[:, d:]
 *   g  = clamp8(RS(a s, m_glu, shift_glu)),  s = -(glu_q1 + sgn(b) L_g(b)),
 *        L_g(q) = (min(|q|, glu_qc) - glu_qc)^2 + glu_q1
 *                                                   GLU with the sigmoid (1 + tanh^(x/2)) / 2 of
 *                                                   Eq. 12's polynomial; g = 0 on frames t >= L_b
 *   v  = clamp16(RS(bias_dw[c] + sum_k w_dw[c][k] g[t + k - 4], mult_dw[c], shift_dw))
 *                                                   depthwise convolution over time (9 taps,
 *                                                   zero outside [0, T)) with BatchNorm folded
 *                                                   into w_dw and bias_dw; v on the INT16 grid
 *                                                   of the BatchNorm output ([-32767, 32767])
 *   o  = clamp8(RS(-(|v| L_s(v) + v sw_q1), m_sw, shift_sw)) for t < L_b, else 0,
 *        L_s(q) = (min(|q|, sw_qc) - sw_qc)^2 + sw_q1    Eq. 12's Swish on v's grid
 *   y  = clamp8(RS(o W_pw2^T, mult_pw2[c], shift_pw2))
 *   z' = clamp8(RS(m_z z + m_y y, 1, shift_r))
 * Shapes: d_model a multiple of 64 in [64, 16384]; max_batch in [1, IPK_MAX_BATCH],
 * max_T in [1, IPK_MAX_T] size the workspace.
 * Weights (DEVICE, int8, row-major): w_pw1 [2 d][d], w_dw [d][9], w_pw2 [d][d].
 * Per-channel constants (HOST, int32): mult_pw1 [2 d], bias_dw [d], mult_dw [d], mult_pw2 [d].
 * Ranges: multipliers in [0, 2^23); |bias_dw| < 2^30; shift_pw1, shift_dw, shift_pw2,
 * shift_r in [1, 40]; shift_glu, shift_sw in [1, 62]; 0 <= glu_qc, sw_qc < 2^20;
 * |glu_q1|, |sw_q1| < 2^45 (an int16 grid puts q_1 far beyond 32 bits); and for
 * every int8 a, b: |a s| m_glu + 2^(shift_glu - 1) < 2^62, for every int16 v:
 * |Swish(v)| m_sw + 2^(shift_sw - 1) < 2^62 (IPK_ERR_UNSUPPORTED otherwise).
 * LayerNorm and residual constants as ipk_mhsa_residual_desc.
 */
typedef struct ipk_conv_desc {
  int32_t d_model, max_batch, max_T;
  const int8_t* w_pw1;
  const int32_t* mult_pw1;
  int32_t shift_pw1;
  int32_t glu_qc;
  int64_t glu_q1;
  int32_t m_glu, shift_glu;
  const int8_t* w_dw;
  const int32_t *bias_dw, *mult_dw;
  int32_t shift_dw;
  int32_t sw_qc;
  int64_t sw_q1;
  int32_t m_sw, shift_sw;
  const int8_t* w_pw2;
  const int32_t* mult_pw2;
  int32_t shift_pw2;
  const int32_t* ln_mult;
  const int64_t* ln_bias;
  int32_t ln_shift;
  int32_t m_z, m_y, shift_r;
} ipk_conv_desc;

typedef struct ipk_conv ipk_conv_t;

/* Validates `desc`, allocates the handle and its workspace and keeps device copies of
 * the weights and constants.  Synchronizes its own copies.  Returns IPK_OK and sets
 * *out, or a negative status with *out = NULL and nothing leaked. */
int ipk_conv_create(const ipk_conv_desc* desc, ipk_conv_t** out);

/* Runs the module on `stream`: z DEVICE int8 [B][T][d_model] -> z_out (same layout),
 * both 16-byte aligned; z_out may be z itself but may not overlap it otherwise.
 * lengths: HOST int32 [B] valid frames in [1, T] (NULL: all T; exactly B entries are
 * read), captured at the call.
 * Asynchronous; calls on one handle must be ordered on one stream.
 * Errors: IPK_ERR_INVALID_ARG (null handle or pointer, misalignment, partial overlap,
 * B or T outside the handle's limits, a length outside [1, T]), IPK_ERR_HIP. */
int ipk_conv_run(ipk_conv_t* h, const int8_t* z, const int32_t* lengths, int32_t B, int32_t T, int8_t* z_out,
                 void* stream);

/* Copies an intermediate of the last run into `dst` (DEVICE, `bytes` bytes) on
 * `stream`: IPK_CONV_X the LayerNorm output int8 [B][T][d], IPK_CONV_U PW1's output int8
 * [B][T][2 d], IPK_CONV_V the BatchNorm output int16 [B][T][d], IPK_CONV_O the Swish
 * output int8 [B][T][d].  A run does not store the BatchNorm output (it is consumed in
 * registers); IPK_CONV_V enqueues the middle kernel again on the kept PW1 output, with
 * the int16 store, before the copy.  Errors: IPK_ERR_INVALID_ARG (no run yet, unknown
 * `which`, bytes too small, null), IPK_ERR_HIP. */
enum { IPK_CONV_X = 0, IPK_CONV_U = 1, IPK_CONV_V = 2, IPK_CONV_O = 3 };
int ipk_conv_intermediate(ipk_conv_t* h, int32_t which, void* dst, int64_t bytes, void* stream);

/* Frees the handle after synchronizing the device; NULL is a no-op. */
int ipk_conv_destroy(ipk_conv_t* h);

/*
 * The integer LayerNorm alone (the LN of Eq. 1 - 4, defined above under
 * ipk_mhsa_residual_desc), for the block's final normalization H = LN(...) of Eq. 4.
 * ln_mult HOST int32 [d_model], ln_bias HOST int64 [d_model]; ranges as for the MHSA
 * module: |ln_mult| < 2^24, |ln_bias| < 2^56, ln_shift in [1, 62]; d_model a multiple of
 * 16 in [16, 16384].  create copies them to the device (synchronously).
 */
typedef struct ipk_layernorm_desc {
  int32_t d_model;
  const int32_t* ln_mult;
  const int64_t* ln_bias;
  int32_t ln_shift;
} ipk_layernorm_desc;

typedef struct ipk_layernorm ipk_layernorm_t;

int ipk_layernorm_create(const ipk_layernorm_desc* desc, ipk_layernorm_t** out);

/* x = LN(z) row by row on `stream`: z, x DEVICE int8 [rows][d_model], 16-byte aligned,
 * x may be z itself.  Errors: IPK_ERR_INVALID_ARG (null handle or pointer, misalignment,
 * rows < 1, partial overlap), IPK_ERR_HIP. */
int ipk_layernorm_run(ipk_layernorm_t* h, const int8_t* z, int64_t rows, int8_t* x, void* stream);

/* Frees the handle after synchronizing the device; NULL is a no-op. */
int ipk_layernorm_destroy(ipk_layernorm_t* h);

/* Human-readable name of a status code (static storage). */
const char* ipk_status_string(int status);

/* Text of the last error reported on the calling thread ("" if none). */
const char* ipk_last_error(void);

/* IPK_ABI_VERSION of the loaded library. */
int ipk_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* IPK_H */
