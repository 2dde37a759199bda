/*
 * CPU oracle for the integer-only relative-positional multi-head self-attention
 * block (Sec. 3.1 of "I-Parakeet: Integer-Only Conformer ASR on Mobile NPU").
 *
 * TEST INFRASTRUCTURE.  This file is the slow, plain reference the GPU library is
 * checked against.  Only the test suite, the package's smoke check and the
 * benchmark's CPU-baseline leg may load it; the product never does.  It shares no
 * code, header or constant with the GPU path: its descriptor is declared here.
 *
 * Every quantity is an exact integer held in int64; there is no blocking, fusion
 * or reordering beyond the definitions.  OpenMP only splits independent outer
 * loops (output rows, attention rows) across threads.
 *
 * Readings of points the paper leaves open (the same list is kept with the
 * design notes):
 *  - round-to-nearest in Eq. 7 and Eq. 11 breaks ties upward:
 *      RS(a, m, n) = floor((a*m + 2^(n-1)) / 2^n);
 *  - int8 grids saturate to [-127, 127] (Eq. 6 clips to +-alpha, S = alpha/127);
 *  - the fused score q_s lives on an int8 grid (one INT8 grid per tensor);
 *  - the softmax follows I-BERT: integer exp with a second-order polynomial on
 *    [-ln2, 0] and a right shift by the ln2 quotient, then F = floor(2^32 / sum)
 *    and a = floor(e * F / 2^24), an 8-bit output on the 2^-8 grid; the single
 *    value 256 that this can reach is clamped to 255;
 *  - row r of the position table holds relative position T-1-r, so the relative
 *    shift Phi reads column j-i+T-1 of row i (relative position i-j);
 *  - keys j >= L_b are left out of the softmax; rows i >= L_b output zeros.
 */
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int32_t d_model, n_heads, d_k;
  const int8_t *w_q, *w_k, *w_v, *w_pos, *w_out; /* [d_out][d_in] */
  const int8_t *pos_bias_u, *pos_bias_v;         /* [H][d_k], on Q's grid */
  const int32_t *mult_q, *mult_k, *mult_v, *mult_pos, *mult_out; /* [d] */
  int32_t shift_q, shift_k, shift_v, shift_pos, shift_out;
  int32_t m_c, m_p, shift_s;
  int32_t m_o, shift_o;
  int32_t q_ln2, q_b, q_c;
} oracle_desc;

/* Optional intermediates; every pointer may be NULL. */
typedef struct {
  int8_t *q, *k, *v; /* [B][T][d] */
  int8_t *p;         /* [2T-1][d] */
  int8_t *s;         /* [B][H][T][T]: fused scores of valid (row, key) pairs */
  uint8_t *a;        /* [B][H][T][T]: softmax output of valid pairs */
  int8_t *ctx;       /* [B][T][d] */
} oracle_trace;

/* Threads the parallel loops will use, and a way to change it (timing only). */
int ipk_oracle_num_threads(void) { return omp_get_max_threads(); }
void ipk_oracle_set_num_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }

/* floor(v / 2^n) for n >= 0, written without relying on signed shifts. */
static int64_t floor_div_pow2(int64_t v, int32_t n) {
  int64_t d = (int64_t)1 << n;
  int64_t q = v / d; /* truncates toward zero */
  if ((v % d) != 0 && v < 0) q -= 1;
  return q;
}

/* Eq. 7: round(2^-n * m * a) with ties toward +infinity. */
int64_t ipk_oracle_rs(int64_t a, int64_t m, int32_t n) {
  int64_t half = n > 0 ? ((int64_t)1 << (n - 1)) : 0;
  return floor_div_pow2(a * m + half, n);
}

/* Eq. 6 with b = 8: the symmetric int8 grid stops at +-127. */
int64_t ipk_oracle_clamp8(int64_t v) { return v < -127 ? -127 : (v > 127 ? 127 : v); }

/* Eq. 7: integer linear layer y = W x with INT32-range accumulation and one
 * fixed-point multiplier per output channel (weights are per-channel, Sec. 2.2). */
void ipk_oracle_linear(const int8_t* x, int64_t rows, int32_t d_in, const int8_t* w, int32_t d_out,
                       const int32_t* mult, int32_t shift, int8_t* y) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < rows; ++t) {
    for (int32_t c = 0; c < d_out; ++c) {
      int64_t acc = 0;
      for (int32_t i = 0; i < d_in; ++i) acc += (int64_t)x[t * d_in + i] * (int64_t)w[(int64_t)c * d_in + i];
      y[t * d_out + c] = (int8_t)ipk_oracle_clamp8(ipk_oracle_rs(acc, mult[c], shift));
    }
  }
}

/* Phi for one query row i: out[j] = p[j - i + T - 1], j < T (Sec. 3.1: a pure
 * index map; nothing is computed). */
void ipk_oracle_rel_shift_row(const int64_t* p_row, int32_t i, int32_t T, int64_t* out_row) {
  for (int32_t j = 0; j < T; ++j) out_row[j] = p_row[j - i + T - 1];
}

/* Phi on a whole [T][2T-1] position-score matrix, giving [T][T]. */
void ipk_oracle_rel_shift(const int64_t* p, int32_t T, int64_t* out) {
  for (int32_t i = 0; i < T; ++i) ipk_oracle_rel_shift_row(p + (int64_t)i * (2 * T - 1), i, T, out + (int64_t)i * T);
}

/* Eq. 11: fused content + position requantization of one score. */
int64_t ipk_oracle_fused_score(int64_t c, int64_t p_shifted, int64_t m_c, int64_t m_p, int32_t shift_s) {
  return ipk_oracle_clamp8(ipk_oracle_rs(m_c * c + m_p * p_shifted, 1, shift_s));
}

/* I-BERT integer exp of the non-positive integer -d (real value -d * S):
 * split -d = -z*q_ln2 + r with r in (-q_ln2, 0], evaluate the polynomial
 * (r + q_b)^2 + q_c (on grid a*S^2) and divide by 2^z. */
int64_t ipk_oracle_iexp(int64_t d, int64_t q_ln2, int64_t q_b, int64_t q_c) {
  int64_t z = d / q_ln2; /* d >= 0, q_ln2 >= 1 */
  int64_t r = z * q_ln2 - d;
  int64_t L = (r + q_b) * (r + q_b) + q_c;
  if (z >= 62) return 0;
  return L >> z; /* L >= 0 here, so the shift is a floor division */
}

/* I-BERT integer softmax over n integer scores: max, exp, sum, then the 8-bit
 * normalization a = floor(e * floor(2^32 / sum) / 2^24), clamped to 255. */
void ipk_oracle_softmax_row(const int64_t* s, int32_t n, int64_t q_ln2, int64_t q_b, int64_t q_c, uint8_t* a) {
  int64_t M = s[0];
  for (int32_t j = 1; j < n; ++j) if (s[j] > M) M = s[j];
  int64_t* e = (int64_t*)malloc(sizeof(int64_t) * (size_t)n);
  int64_t sum = 0;
  for (int32_t j = 0; j < n; ++j) { e[j] = ipk_oracle_iexp(M - s[j], q_ln2, q_b, q_c); sum += e[j]; }
  uint64_t F = sum > 0 ? ((uint64_t)1 << 32) / (uint64_t)sum : 0;
  for (int32_t j = 0; j < n; ++j) {
    uint64_t v = ((uint64_t)e[j] * F) >> 24;
    a[j] = (uint8_t)(v > 255 ? 255 : v);
  }
  free(e);
}

/* The whole block: projections (Eq. 7), content and position scores (Eq. 8),
 * Phi, fused requantization (Eq. 11), integer softmax, A V with Eq. 7's requant,
 * and the output projection.  Returns 0, or -1 on an invalid argument. */
int ipk_oracle_relpos_attn(const oracle_desc* D, const int8_t* x, const int8_t* pos_table, const int32_t* lengths,
                           int32_t B, int32_t T, int8_t* y, oracle_trace* tr) {
  if (!D || !x || !pos_table || !y || B < 1 || T < 1) return -1;
  const int32_t d = D->d_model, H = D->n_heads, dk = D->d_k;
  if (d != H * dk || D->q_ln2 < 1 || D->q_b < 0 || D->q_c < 0) return -1;
  if ((int64_t)D->q_b * D->q_b + D->q_c == 0) return -1; /* e(0) must be positive */
  for (int32_t b = 0; b < B; ++b)
    if (lengths && (lengths[b] < 1 || lengths[b] > T)) return -1;
  const int64_t rows = (int64_t)B * T, R = 2 * (int64_t)T - 1;

  int8_t* Q = (int8_t*)malloc((size_t)(rows * d));
  int8_t* K = (int8_t*)malloc((size_t)(rows * d));
  int8_t* V = (int8_t*)malloc((size_t)(rows * d));
  int8_t* P = (int8_t*)malloc((size_t)(R * d));
  int8_t* ctx = (int8_t*)calloc((size_t)(rows * d), 1);
  if (!Q || !K || !V || !P || !ctx) { free(Q); free(K); free(V); free(P); free(ctx); return -2; }

  /* Step 1: projections of every row, padded ones included. */
  ipk_oracle_linear(x, rows, d, D->w_q, d, D->mult_q, D->shift_q, Q);
  ipk_oracle_linear(x, rows, d, D->w_k, d, D->mult_k, D->shift_k, K);
  ipk_oracle_linear(x, rows, d, D->w_v, d, D->mult_v, D->shift_v, V);
  ipk_oracle_linear(pos_table, R, d, D->w_pos, d, D->mult_pos, D->shift_pos, P);

  /* Steps 2-7, one (utterance, head, query row) at a time. */
#pragma omp parallel
  {
    int64_t* c = (int64_t*)malloc(sizeof(int64_t) * (size_t)T);
    int64_t* p = (int64_t*)malloc(sizeof(int64_t) * (size_t)R);
    int64_t* pt = (int64_t*)malloc(sizeof(int64_t) * (size_t)T);
    int64_t* s = (int64_t*)malloc(sizeof(int64_t) * (size_t)T);
    uint8_t* a = (uint8_t*)malloc((size_t)T);
#pragma omp for collapse(3) schedule(dynamic, 4)
    for (int32_t b = 0; b < B; ++b)
      for (int32_t h = 0; h < H; ++h)
        for (int32_t i = 0; i < T; ++i) {
          const int32_t L = lengths ? lengths[b] : T;
          if (i >= L) continue; /* padded query rows stay zero */
          const int8_t* q = Q + ((int64_t)b * T + i) * d + (int64_t)h * dk;
          const int8_t* u = D->pos_bias_u + (int64_t)h * dk;
          const int8_t* v = D->pos_bias_v + (int64_t)h * dk;
          /* Eq. 8, content branch: (q + u) . k_j */
          for (int32_t j = 0; j < T; ++j) {
            const int8_t* kr = K + ((int64_t)b * T + j) * d + (int64_t)h * dk;
            int64_t acc = 0;
            for (int32_t k = 0; k < dk; ++k) acc += ((int64_t)q[k] + u[k]) * (int64_t)kr[k];
            c[j] = acc;
          }
          /* Eq. 8, position branch before Phi: (q + v) . p_r for every relative position */
          for (int64_t r = 0; r < R; ++r) {
            const int8_t* pr = P + r * d + (int64_t)h * dk;
            int64_t acc = 0;
            for (int32_t k = 0; k < dk; ++k) acc += ((int64_t)q[k] + v[k]) * (int64_t)pr[k];
            p[r] = acc;
          }
          ipk_oracle_rel_shift_row(p, i, T, pt);
          /* Eq. 11 on the valid keys, then the integer softmax */
          for (int32_t j = 0; j < L; ++j) s[j] = ipk_oracle_fused_score(c[j], pt[j], D->m_c, D->m_p, D->shift_s);
          ipk_oracle_softmax_row(s, L, D->q_ln2, D->q_b, D->q_c, a);
          if (tr && tr->s)
            for (int32_t j = 0; j < L; ++j) tr->s[(((int64_t)b * H + h) * T + i) * T + j] = (int8_t)s[j];
          if (tr && tr->a)
            for (int32_t j = 0; j < L; ++j) tr->a[(((int64_t)b * H + h) * T + i) * T + j] = a[j];
          /* A V, requantized to the context grid (Eq. 7 with the scalar m_o) */
          for (int32_t k = 0; k < dk; ++k) {
            int64_t acc = 0;
            for (int32_t j = 0; j < L; ++j) acc += (int64_t)a[j] * (int64_t)V[((int64_t)b * T + j) * d + (int64_t)h * dk + k];
            ctx[((int64_t)b * T + i) * d + (int64_t)h * dk + k] =
                (int8_t)ipk_oracle_clamp8(ipk_oracle_rs(acc, D->m_o, D->shift_o));
          }
        }
    free(c); free(p); free(pt); free(s); free(a);
  }

  /* Step 8: output projection of the valid rows; padded rows are zero. */
  memset(y, 0, (size_t)(rows * d));
  for (int32_t b = 0; b < B; ++b) {
    const int32_t L = lengths ? lengths[b] : T;
    ipk_oracle_linear(ctx + (int64_t)b * T * d, L, d, D->w_out, d, D->mult_out, D->shift_out, y + (int64_t)b * T * d);
  }

  if (tr) {
    if (tr->q) memcpy(tr->q, Q, (size_t)(rows * d));
    if (tr->k) memcpy(tr->k, K, (size_t)(rows * d));
    if (tr->v) memcpy(tr->v, V, (size_t)(rows * d));
    if (tr->p) memcpy(tr->p, P, (size_t)(R * d));
    if (tr->ctx) memcpy(tr->ctx, ctx, (size_t)(rows * d));
  }
  free(Q); free(K); free(V); free(P); free(ctx);
  return 0;
}

/* ------------------------------------------------------------------------------
 * The MHSA residual sub-module of Eq. 2: Z2 = Z1 + MHSA(LN(Z1)), on integer grids.
 * The paper takes LayerNorm from I-BERT; the integer steps below are this oracle's
 * reading of it (kept with the design notes):
 *  - mean mu = round(sum / d), ties upward;
 *  - y = z - mu, sigma = floor(sqrt(sum y^2)) by I-BERT's integer Newton iteration
 *    (at least 1);
 *  - F = floor(2^31 / sigma) and u = floor(y F / 2), so u ~ 2^30 (z - mean) / sigma,
 *    i.e. the normalized value (z - mean) / std is u sqrt(d) / 2^30;
 *  - the affine gamma, beta and the move to the MHSA input grid S_x are one
 *    fixed-point step per channel: x = clamp8(floor((u g + c + 2^(n-1)) / 2^n)) with
 *    g = round(2^n sqrt(d) gamma / (2^30 S_x)) and c = round(2^n beta / S_x).
 *  - the residual add requantizes both terms to Z2's grid in one step, as Eq. 11
 *    does for the two score branches: z2 = clamp8(floor((m_z z1 + m_y y + 2^(n-1))
 *    / 2^n)) with m_z = round(2^n S_z1 / S_z2), m_y = round(2^n S_y / S_z2).
 * ------------------------------------------------------------------------------ */

/* floor(a / b) for b > 0 */
static int64_t floor_div(int64_t a, int64_t b) {
  int64_t q = a / b;
  if ((a % b) != 0 && a < 0) q -= 1;
  return q;
}

/* I-BERT's integer square root: floor(sqrt(n)) for n >= 0.  Newton's iteration on
 * integers, x <- floor((x + floor(n / x)) / 2), started at a power of two not below
 * the root, decreases strictly until it reaches the floor of the root. */
int64_t ipk_oracle_isqrt(int64_t n) {
  if (n <= 0) return 0;
  int bits = 0;
  for (int64_t t = n; t > 0; t >>= 1) ++bits;
  int64_t x = (int64_t)1 << ((bits + 1) / 2);
  for (;;) {
    const int64_t nx = (x + n / x) / 2;
    if (nx >= x) return x;
    x = nx;
  }
}

/* Integer LayerNorm of one row of d int8 values (steps as listed above). */
void ipk_oracle_layernorm_row(const int8_t* z, int32_t d, const int32_t* g, const int64_t* c, int32_t shift,
                              int8_t* x) {
  int64_t s = 0;
  for (int32_t k = 0; k < d; ++k) s += z[k];
  const int64_t mu = floor_div(2 * s + d, 2 * (int64_t)d);
  int64_t v = 0;
  for (int32_t k = 0; k < d; ++k) v += (z[k] - mu) * (z[k] - mu);
  int64_t sigma = ipk_oracle_isqrt(v);
  if (sigma < 1) sigma = 1;
  const int64_t F = ((int64_t)1 << 31) / sigma;
  const int64_t half = (int64_t)1 << (shift - 1);
  for (int32_t k = 0; k < d; ++k) {
    const int64_t u = floor_div_pow2((z[k] - mu) * F, 1);
    x[k] = (int8_t)ipk_oracle_clamp8(floor_div_pow2(u * g[k] + c[k] + half, shift));
  }
}

/* Eq. 2's residual add of one element on integer grids. */
int64_t ipk_oracle_residual(int64_t z1, int64_t y, int64_t m_z, int64_t m_y, int32_t shift) {
  return ipk_oracle_clamp8(floor_div_pow2(m_z * z1 + m_y * y + ((int64_t)1 << (shift - 1)), shift));
}

/* The sub-module on [B][T][d]: x = LN(z1) row by row, y = the block on x, z2 =
 * residual(z1, y).  x_out and y_out (may be NULL) receive the intermediates.
 * Returns 0, or -1 on an invalid argument. */
int ipk_oracle_mhsa_residual(const oracle_desc* D, const int32_t* ln_g, const int64_t* ln_c, int32_t ln_shift,
                             int32_t m_z, int32_t m_y, int32_t shift_r, const int8_t* z1, const int8_t* pos_table,
                             const int32_t* lengths, int32_t B, int32_t T, int8_t* z2, int8_t* x_out, int8_t* y_out) {
  if (!D || !ln_g || !ln_c || !z1 || !z2 || B < 1 || T < 1 || ln_shift < 1 || ln_shift > 62 || shift_r < 1 ||
      shift_r > 40)
    return -1;
  const int32_t d = D->d_model;
  const int64_t rows = (int64_t)B * T;
  int8_t* x = (int8_t*)malloc((size_t)(rows * d));
  int8_t* y = (int8_t*)malloc((size_t)(rows * d));
  if (!x || !y) {
    free(x);
    free(y);
    return -1;
  }
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) ipk_oracle_layernorm_row(z1 + r * d, d, ln_g, ln_c, ln_shift, x + r * d);
  const int rc = ipk_oracle_relpos_attn(D, x, pos_table, lengths, B, T, y, NULL);
  if (rc == 0)
    for (int64_t i = 0; i < rows * d; ++i) z2[i] = (int8_t)ipk_oracle_residual(z1[i], y[i], m_z, m_y, shift_r);
  if (rc == 0 && x_out) memcpy(x_out, x, (size_t)(rows * d));
  if (rc == 0 && y_out) memcpy(y_out, y, (size_t)(rows * d));
  free(x);
  free(y);
  return rc;
}

/* ------------------------------------------------------------------------------
 * The feed-forward module of Eq. 1, Z1 = X + 0.5 FFN(LN(X)) with FFN = W2 Swish(W1 .),
 * on integer grids.  Steps (this oracle's reading, kept with the design notes):
 *  - x = LN(z) as above;
 *  - h = clamp8(RS(x W1^T, mult1[c], shift1))            (Eq. 7, per channel, int8);
 *  - the Swish of Sec. 3.2 on h's grid S: with u = x/2 on S_u = S/2, Eq. 12 gives
 *    |tanh^| on the grid a S_u^2 as L = (min(|h|, q_c) - q_c)^2 + q_1 with
 *    q_c = floor(c / S_u) and q_1 = floor(1 / (a S_u^2)), and since
 *    sw^(x) = x (1 + sgn(x) |tanh^|) / 2 = (x + |x| |tanh^|) / 2,
 *    q_sw = -(|h| L + h q_1) on the grid -a S_u^2 S / 2 (positive: a < 0);
 *  - o = clamp8(RS(q_sw, m_sw, shift_sw)), FFN2's int8 input grid;
 *  - y = clamp8(RS(o W2^T, mult2[c], shift2))             (Eq. 7);
 *  - z_out = clamp8(RS(m_z z + m_y y, 1, shift_r)), the 0.5 of Eq. 1 folded into m_y.
 * ------------------------------------------------------------------------------ */

typedef struct {
  int32_t d_model, d_ff;
  const int8_t *w1, *w2;         /* [d_ff][d_model], [d_model][d_ff] */
  const int32_t *mult1, *mult2;  /* [d_ff], [d_model] */
  int32_t shift1, shift2;
  int64_t sw_qc, sw_q1;
  int32_t m_sw, shift_sw;
  const int32_t* ln_mult;
  const int64_t* ln_bias;
  int32_t ln_shift;
  int32_t m_z, m_y, shift_r;
} oracle_ffn_desc;

/* The integer Swish of one value q on its grid (Eq. 12 as described above). */
int64_t ipk_oracle_int_swish(int64_t q, int64_t q_c, int64_t q_1) {
  const int64_t aq = q < 0 ? -q : q;
  const int64_t t = (aq < q_c ? aq : q_c) - q_c;
  const int64_t L = t * t + q_1;
  return -(aq * L + q * q_1);
}

/* The module on `rows` rows of d_model int8 values.  x_out [rows][d_model], h_out and
 * o_out [rows][d_ff], y_out [rows][d_model] receive the intermediates (each may be
 * NULL).  Returns 0, or -1 on an invalid argument. */
int ipk_oracle_ffn_module(const oracle_ffn_desc* D, const int8_t* z, int64_t rows, int8_t* z_out, int8_t* x_out,
                          int8_t* h_out, int8_t* o_out, int8_t* y_out) {
  if (!D || !z || !z_out || rows < 1 || D->d_model < 1 || D->d_ff < 1 || D->ln_shift < 1 || D->ln_shift > 62 ||
      D->shift1 < 1 || D->shift1 > 40 || D->shift2 < 1 || D->shift2 > 40 || D->shift_sw < 1 || D->shift_sw > 40 ||
      D->shift_r < 1 || D->shift_r > 40 || D->sw_qc < 0)
    return -1;
  const int32_t d = D->d_model, f = D->d_ff;
  int8_t* x = (int8_t*)malloc((size_t)(rows * d));
  int8_t* h = (int8_t*)malloc((size_t)(rows * f));
  int8_t* o = (int8_t*)malloc((size_t)(rows * f));
  int8_t* y = (int8_t*)malloc((size_t)(rows * d));
  if (!x || !h || !o || !y) {
    free(x); free(h); free(o); free(y);
    return -1;
  }
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) ipk_oracle_layernorm_row(z + r * d, d, D->ln_mult, D->ln_bias, D->ln_shift, x + r * d);
  ipk_oracle_linear(x, rows, d, D->w1, f, D->mult1, D->shift1, h);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < rows * f; ++i)
    o[i] = (int8_t)ipk_oracle_clamp8(ipk_oracle_rs(ipk_oracle_int_swish(h[i], D->sw_qc, D->sw_q1), D->m_sw, D->shift_sw));
  ipk_oracle_linear(o, rows, f, D->w2, d, D->mult2, D->shift2, y);
  for (int64_t i = 0; i < rows * d; ++i) z_out[i] = (int8_t)ipk_oracle_residual(z[i], y[i], D->m_z, D->m_y, D->shift_r);
  if (x_out) memcpy(x_out, x, (size_t)(rows * d));
  if (h_out) memcpy(h_out, h, (size_t)(rows * f));
  if (o_out) memcpy(o_out, o, (size_t)(rows * f));
  if (y_out) memcpy(y_out, y, (size_t)(rows * d));
  free(x); free(h); free(o); free(y);
  return 0;
}

/* ------------------------------------------------------------------------------
 * The convolution module of Eq. 3 and Eq. 5, Z3 = Z2 + Conv(LN(Z2)) with
 * Conv = PW2(Swish(BN(DW(GLU(PW1(.)))))), on integer grids (this oracle's reading,
 * kept with the design notes):
 *  - x = LN(z) as above;
 *  - u = clamp8(RS(x W_pw1^T, mult_pw1[c], shift_pw1)) over 2 d channels: a = u[:, :d],
 *    b = u[:, d:] (Eq. 7);
 *  - GLU: a * sigmoid(b) with sigmoid(x) = (1 + tanh^(x/2)) / 2 and tanh^ of Eq. 12.
 *    On b's grid S (u = x/2 on S/2), tanh^ = sgn(q) (a* (S/2)^2) L with
 *    L = (min(|q|, q_c) - q_c)^2 + q_1, so sigmoid = -(q_1 + sgn(q) L) on the grid
 *    -a* (S/2)^2 / 2; g = clamp8(RS(a * sigmoid, m_glu, shift_glu)), and g = 0 on
 *    frames t >= L_b (the padding mask before the depthwise convolution);
 *  - DW: depthwise convolution over time, K = 9 taps centred on t (zero outside
 *    [0, T)), BatchNorm folded into its int8 weights and an int32 bias on the
 *    accumulator grid; the result goes to the INT16 grid of the BatchNorm output:
 *    v = clamp16(RS(sum_k w[c][k] g[t + k - 4][c] + bias[c], mult_dw[c], shift_dw));
 *  - Swish of Eq. 12 on the int16 grid as in the feed-forward module, then
 *    o = clamp8(RS(q_sw, m_sw, shift_sw)), o = 0 on frames t >= L_b;
 *  - y = clamp8(RS(o W_pw2^T, mult_pw2[c], shift_pw2)) (Eq. 7);
 *  - z_out = clamp8(RS(m_z z + m_y y, 1, shift_r)).
 * The Swish and GLU products are formed in 128 bits here, so no intermediate can
 * overflow whatever the constants.
 * ------------------------------------------------------------------------------ */

typedef struct {
  int32_t d_model;
  const int8_t* w_pw1; /* [2d][d] */
  const int32_t* mult_pw1;
  int32_t shift_pw1;
  int64_t glu_qc, glu_q1;
  int32_t m_glu, shift_glu;
  const int8_t* w_dw; /* [d][9] */
  const int32_t* bias_dw;
  const int32_t* mult_dw;
  int32_t shift_dw;
  int64_t sw_qc, sw_q1;
  int32_t m_sw, shift_sw;
  const int8_t* w_pw2; /* [d][d] */
  const int32_t* mult_pw2;
  int32_t shift_pw2;
  const int32_t* ln_mult;
  const int64_t* ln_bias;
  int32_t ln_shift;
  int32_t m_z, m_y, shift_r;
} oracle_conv_desc;

/* floor((a m + 2^(n-1)) / 2^n) in 128-bit arithmetic */
static int64_t rs_wide(__int128 a, int64_t m, int32_t n) {
  __int128 v = a * m + ((__int128)1 << (n - 1));
  __int128 d = (__int128)1 << n;
  __int128 q = v / d;
  if (v % d != 0 && v < 0) q -= 1;
  if (q > INT64_MAX / 2) return INT64_MAX / 2;
  if (q < INT64_MIN / 2) return INT64_MIN / 2;
  return (int64_t)q;
}

static int64_t clamp16(int64_t v) { return v < -32767 ? -32767 : (v > 32767 ? 32767 : v); }

/* The sigmoid of GLU on one value q of its grid (as described above). */
int64_t ipk_oracle_int_sigmoid(int64_t q, int64_t q_c, int64_t q_1) {
  const int64_t aq = q < 0 ? -q : q;
  const int64_t t = (aq < q_c ? aq : q_c) - q_c;
  const int64_t L = t * t + q_1;
  const int64_t sg = q > 0 ? 1 : (q < 0 ? -1 : 0);
  return -(q_1 + sg * L);
}

/* The module on [B][T][d_model].  Intermediates (each may be NULL): x_out [B][T][d],
 * u_out [B][T][2d], g_out [B][T][d] (GLU), v_out int16 [B][T][d] (BatchNorm output),
 * o_out [B][T][d] (Swish), y_out [B][T][d].  Returns 0, or -1 on an invalid argument. */
int ipk_oracle_conv_module(const oracle_conv_desc* D, const int8_t* z, const int32_t* lengths, int32_t B, int32_t T,
                           int8_t* z_out, int8_t* x_out, int8_t* u_out, int8_t* g_out, int16_t* v_out, int8_t* o_out,
                           int8_t* y_out) {
  if (!D || !z || !z_out || B < 1 || T < 1 || D->d_model < 1 || D->ln_shift < 1 || D->ln_shift > 62 ||
      D->shift_pw1 < 1 || D->shift_pw1 > 40 || D->shift_glu < 1 || D->shift_glu > 62 || D->shift_dw < 1 ||
      D->shift_dw > 40 || D->shift_sw < 1 || D->shift_sw > 62 || D->shift_pw2 < 1 || D->shift_pw2 > 40 ||
      D->shift_r < 1 || D->shift_r > 40 || D->glu_qc < 0 || D->sw_qc < 0)
    return -1;
  for (int32_t b = 0; b < B; ++b)
    if (lengths && (lengths[b] < 1 || lengths[b] > T)) return -1;
  const int32_t d = D->d_model;
  const int64_t rows = (int64_t)B * T;
  int8_t* x = (int8_t*)malloc((size_t)(rows * d));
  int8_t* u = (int8_t*)malloc((size_t)(rows * 2 * d));
  int8_t* g = (int8_t*)malloc((size_t)(rows * d));
  int16_t* v = (int16_t*)malloc((size_t)(rows * d) * sizeof(int16_t));
  int8_t* o = (int8_t*)malloc((size_t)(rows * d));
  int8_t* y = (int8_t*)malloc((size_t)(rows * d));
  if (!x || !u || !g || !v || !o || !y) {
    free(x); free(u); free(g); free(v); free(o); free(y);
    return -1;
  }
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) ipk_oracle_layernorm_row(z + r * d, d, D->ln_mult, D->ln_bias, D->ln_shift, x + r * d);
  ipk_oracle_linear(x, rows, d, D->w_pw1, 2 * d, D->mult_pw1, D->shift_pw1, u);
  for (int32_t bb = 0; bb < B; ++bb) {
    const int32_t L = lengths ? lengths[bb] : T;
#pragma omp parallel for schedule(static)
    for (int32_t t = 0; t < T; ++t) {
      const int64_t r = (int64_t)bb * T + t;
      for (int32_t c = 0; c < d; ++c) {
        int64_t gv = 0;
        if (t < L) {
          const int64_t sig = ipk_oracle_int_sigmoid(u[r * 2 * d + d + c], D->glu_qc, D->glu_q1);
          gv = ipk_oracle_clamp8(rs_wide((__int128)u[r * 2 * d + c] * sig, D->m_glu, D->shift_glu));
        }
        g[r * d + c] = (int8_t)gv;
      }
    }
#pragma omp parallel for schedule(static)
    for (int32_t t = 0; t < T; ++t) {
      const int64_t r = (int64_t)bb * T + t;
      for (int32_t c = 0; c < d; ++c) {
        int64_t acc = D->bias_dw[c];
        for (int32_t k = 0; k < 9; ++k) {
          const int32_t ts = t + k - 4;
          if (ts >= 0 && ts < T) acc += (int64_t)D->w_dw[c * 9 + k] * g[((int64_t)bb * T + ts) * d + c];
        }
        const int64_t vv = clamp16(ipk_oracle_rs(acc, D->mult_dw[c], D->shift_dw));
        v[r * d + c] = (int16_t)vv;
        int64_t ov = 0;
        if (t < L) ov = ipk_oracle_clamp8(rs_wide(ipk_oracle_int_swish(vv, D->sw_qc, D->sw_q1), D->m_sw, D->shift_sw));
        o[r * d + c] = (int8_t)ov;
      }
    }
  }
  ipk_oracle_linear(o, rows, d, D->w_pw2, d, D->mult_pw2, D->shift_pw2, y);
  for (int64_t i = 0; i < rows * d; ++i) z_out[i] = (int8_t)ipk_oracle_residual(z[i], y[i], D->m_z, D->m_y, D->shift_r);
  if (x_out) memcpy(x_out, x, (size_t)(rows * d));
  if (u_out) memcpy(u_out, u, (size_t)(rows * 2 * d));
  if (g_out) memcpy(g_out, g, (size_t)(rows * d));
  if (v_out) memcpy(v_out, v, (size_t)(rows * d) * sizeof(int16_t));
  if (o_out) memcpy(o_out, o, (size_t)(rows * d));
  if (y_out) memcpy(y_out, y, (size_t)(rows * d));
  free(x); free(u); free(g); free(v); free(o); free(y);
  return 0;
}
