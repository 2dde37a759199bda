// C-ABI entry points of the ipk library: descriptor validation, the handle and its
// workspace, and the per-run launch sequence
//   projections (Q|K|V and the position table) -> rank-1 bias terms and V prefix
//   sums -> attention core -> output projection; for the MHSA module of Eq. 2 an
//   integer LayerNorm first and the residual add in the output projection's epilogue;
//   the feed-forward module of Eq. 1 (LayerNorm, W1 + integer Swish, W2 + residual); and
//   the convolution module of Eq. 5 (LayerNorm, PW1, GLU + depthwise + INT16 BatchNorm
//   + Swish, PW2 + residual).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdlib.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <new>
#include <algorithm>
#include <vector>

#include "../../include/ipk.h"
#include "ipk_internal.h"

using namespace ipk;

struct ipk_relpos_attn {
  int device;
  int d, H, DK, max_B, max_T;
  Weights w;
  Scalars sc;
  Workspace ws;
  std::vector<void*> allocs;
  RunShape last;
  bool has_run;
  bool last_was_residual;
  Workspace last_ws;  // the last run's buffers (ws, the kept table, or the no-allocation array)
  Lengths last_lens;  // the last run's lengths and score constants, for ipk_relpos_attn_repeat_core
  Scalars last_sc;
  bool last_noalloc;  // the last run's workspace was the shared no-allocation array
  hipEvent_t stage_ev[IPK_NUM_STAGES + 1];
  bool stages_pending;
  // projected position table kept by ipk_relpos_attn_cache_positions
  int8_t* pcache;
  int pcache_T;     // table length T_table, 0 when nothing is kept
  int pcache_rows;  // rows per head of pcache
  // LayerNorm and residual constants of the MHSA module
  Residual res;
  bool has_res;
};

static thread_local char g_last_error[512];

static int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
  va_end(ap);
  return status;
}

static bool mult_ok(int64_t m) { return m >= 0 && m < (1 << 23); }
static bool shift_ok(int32_t s) { return s >= 1 && s <= 40; }

static int validate_desc(const ipk_relpos_attn_desc* d) {
  if (!d) return fail(IPK_ERR_INVALID_ARG, "desc is NULL");
  if (d->d_k != 64 && d->d_k != 128) return fail(IPK_ERR_UNSUPPORTED, "d_k=%d: only 64 and 128 are built", d->d_k);
  if (d->n_heads < 1 || d->d_model != d->n_heads * d->d_k)
    return fail(IPK_ERR_INVALID_ARG, "d_model=%d must equal n_heads=%d * d_k=%d", d->d_model, d->n_heads, d->d_k);
  if (d->d_model > 16384) return fail(IPK_ERR_UNSUPPORTED, "d_model=%d above 16384", d->d_model);
  if (d->max_batch < 1 || d->max_batch > IPK_MAX_BATCH)
    return fail(IPK_ERR_INVALID_ARG, "max_batch=%d outside [1, %d]", d->max_batch, IPK_MAX_BATCH);
  if (d->max_T < 1 || d->max_T > IPK_MAX_T)
    return fail(IPK_ERR_INVALID_ARG, "max_T=%d outside [1, %d]", d->max_T, IPK_MAX_T);
  const void* ptrs[] = {d->w_q, d->w_k, d->w_v, d->w_pos, d->w_out, d->pos_bias_u, d->pos_bias_v,
                        d->mult_q, d->mult_k, d->mult_v, d->mult_pos, d->mult_out};
  for (const void* p : ptrs)
    if (!p) return fail(IPK_ERR_INVALID_ARG, "a weight, bias or multiplier pointer is NULL");
  const int32_t* mults[] = {d->mult_q, d->mult_k, d->mult_v, d->mult_pos, d->mult_out};
  const char* names[] = {"mult_q", "mult_k", "mult_v", "mult_pos", "mult_out"};
  for (int t = 0; t < 5; ++t)
    for (int c = 0; c < d->d_model; ++c)
      if (!mult_ok(mults[t][c])) return fail(IPK_ERR_INVALID_ARG, "%s[%d]=%d outside [0, 2^23)", names[t], c, mults[t][c]);
  const int32_t shifts[] = {d->shift_q, d->shift_k, d->shift_v, d->shift_pos, d->shift_out, d->shift_s, d->shift_o};
  for (int32_t s : shifts)
    if (!shift_ok(s)) return fail(IPK_ERR_INVALID_ARG, "a shift (%d) is outside [1, 40]", s);
  if (!mult_ok(d->m_c) || !mult_ok(d->m_p) || !mult_ok(d->m_o))
    return fail(IPK_ERR_INVALID_ARG, "m_c=%d, m_p=%d, m_o=%d must be in [0, 2^23)", d->m_c, d->m_p, d->m_o);
  if (d->q_ln2 < 1 || d->q_b < 0 || d->q_c < 0)
    return fail(IPK_ERR_INVALID_ARG, "softmax constants need q_ln2 >= 1, q_b >= 0, q_c >= 0");
  // the integer-exp polynomial over r in (-q_ln2, 0]
  const int64_t qb = d->q_b, lo = qb - (d->q_ln2 - 1);
  const int64_t sq_max = qb * qb > lo * lo ? qb * qb : lo * lo;
  const int64_t poly_max = sq_max + d->q_c, poly0 = qb * qb + d->q_c;
  if (poly_max >= ((int64_t)1 << 24))
    return fail(IPK_ERR_UNSUPPORTED, "integer-exp polynomial reaches %lld >= 2^24", (long long)poly_max);
  if (poly0 < 256) return fail(IPK_ERR_UNSUPPORTED, "integer exp of 0 is %lld < 2^8", (long long)poly0);
  if ((int64_t)d->max_T * poly_max >= ((int64_t)1 << 32))
    return fail(IPK_ERR_UNSUPPORTED, "max_T * max exp = %lld reaches 2^32", (long long)d->max_T * poly_max);
  if (d->zp_x != 0 || d->zp_y != 0) return fail(IPK_ERR_INVALID_ARG, "zero points must be 0 (symmetric grids)");
  return IPK_OK;
}

// Chooses how the attention core evaluates Eq. 11.  |c|, |p| <= d_k * 255 * 127
// (int8 keys/positions times q + u, q + v with q in [-127, 127] and u, v in
// [-128, 127]); the 32-bit path is used when m_c |c| + m_p |p| plus the rounding and
// code bias stays below 2^31 for every possible score, so its wrap-around arithmetic
// is exact.  force_wide selects the 64-bit path whatever the bound (both are exact and
// give the same bytes).
static void plan_fused_score(Scalars* sc, int d_k, bool force_wide) {
  const int64_t cmax = (int64_t)d_k * 255 * 127;
  const int n = sc->shift_s;
  // 32-bit path: scale the multipliers to a shift of 16 so that the biased code
  // s + 128 = floor((m_c c + m_p p + 2^15 + 128 * 2^16) / 2^16) is byte 2 of the
  // clamped sum; only possible for n <= 16
  bool narrow = n <= 16 && !force_wide;
  int64_t mc = 0, mp = 0;
  const int64_t bias = ((int64_t)1 << 15) + ((int64_t)128 << 16);
  if (narrow) {
    mc = (int64_t)sc->m_c << (16 - n);
    mp = (int64_t)sc->m_p << (16 - n);
    narrow = mc < (1 << 23) && mp < (1 << 23) && (mc + mp) * cmax + bias < ((int64_t)1 << 31);
  }
  sc->fs_wide = !narrow;
  sc->fs_mc24 = narrow ? (int32_t)mc : 0;
  sc->fs_mp24 = narrow ? (int32_t)mp : 0;
  sc->fs_bias32 = (int32_t)bias;
}

static void free_handle(ipk_relpos_attn* h) {
  if (!h) return;
  for (void* p : h->allocs) (void)hipFree(p);
  delete h;
}

// Device allocation recorded on any handle type with an `allocs` list (freed with it).
template <typename H, typename T>
static hipError_t dev_alloc(H* h, T** p, size_t count) {
  void* q = nullptr;
  hipError_t e = hipMalloc(&q, count * sizeof(T) > 0 ? count * sizeof(T) : 1);
  if (e != hipSuccess) return e;
  h->allocs.push_back(q);
  *p = (T*)q;
  return hipSuccess;
}

// Eq. 7 constants of `parts` stacked matrices of N channels each (Requant): the fast
// form when every part's shift is at most 16 and one clamp bound serves every channel,
// the wide form otherwise.  Returns the wide flag; `out` receives the 2 parts N values
// and `clamp` the fast form's bound.
static int build_requant(const int32_t* const* mults, const int32_t* shifts, int parts, int N,
                         std::vector<int32_t>& out, int32_t* clamp) {
  const size_t NT = (size_t)parts * N;
  out.assign(2 * NT, 0);
  *clamp = 0;
  bool fast = true;
  int64_t A = 0, mmax = 0;  // the largest channel bound and multiplier
  for (int p = 0; p < parts && fast; ++p) {
    const int n = shifts[p];
    if (n > 16) {
      fast = false;
      break;
    }
    for (int c = 0; c < N && fast; ++c) {
      const int64_t m1 = (int64_t)mults[p][c] << (16 - n);
      fast = m1 < ((int64_t)1 << 23);
      out[(size_t)p * N + c] = (int32_t)m1;
      if (m1 > 0) {
        const int64_t Ac = (((int64_t)1 << 23) + m1 - 1) / m1 + 1;
        A = Ac > A ? Ac : A;
        mmax = m1 > mmax ? m1 : mmax;
      }
    }
  }
  fast = fast && A < ((int64_t)1 << 23) && A * mmax + (1 << 15) < ((int64_t)1 << 31);
  if (fast) {
    *clamp = (int32_t)A;
    return 0;
  }
  for (int p = 0; p < parts; ++p)
    for (int c = 0; c < N; ++c) {
      out[(size_t)p * N + c] = mults[p][c];
      out[NT + (size_t)p * N + c] = shifts[p];
    }
  return 1;
}

// Builds and uploads a matrix's Eq. 7 constants into a device buffer of the handle.
template <typename H>
static hipError_t upload_requant(H* h, Requant* rq, const int32_t* const* mults, const int32_t* shifts, int parts,
                                 int N) {
  std::vector<int32_t> host;
  rq->wide = build_requant(mults, shifts, parts, N, host, &rq->clamp);
  int32_t* dev = nullptr;
  hipError_t e = dev_alloc(h, &dev, host.size());
  if (e == hipSuccess) e = hipMemcpy(dev, host.data(), host.size() * sizeof(int32_t), hipMemcpyHostToDevice);
  rq->req = dev;
  return e;
}

extern "C" int ipk_relpos_attn_create(const ipk_relpos_attn_desc* desc, ipk_relpos_attn_t** out) {
  g_last_error[0] = 0;
  if (!out) return fail(IPK_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  int st = validate_desc(desc);
  if (st != IPK_OK) return st;
  if (attn_plan(desc->d_k, t_aligned(desc->max_T), 1, desc->max_T).c1.ksplit == 0)
    return fail(IPK_ERR_UNSUPPORTED, "max_T=%d does not fit the on-chip score rows", desc->max_T);

  ipk_relpos_attn* h = new (std::nothrow) ipk_relpos_attn();
  if (!h) return fail(IPK_ERR_OUT_OF_MEMORY, "host allocation failed");
  if (hipGetDevice(&h->device) != hipSuccess) {
    free_handle(h);
    return fail(IPK_ERR_HIP, "hipGetDevice failed");
  }
  h->d = desc->d_model;
  h->H = desc->n_heads;
  h->DK = desc->d_k;
  h->max_B = desc->max_batch;
  h->max_T = desc->max_T;
  h->sc = Scalars{};
  h->sc.m_c = desc->m_c;
  h->sc.m_p = desc->m_p;
  h->sc.shift_s = desc->shift_s;
  h->sc.m_o = desc->m_o;
  h->sc.shift_o = desc->shift_o;
  h->sc.q_ln2 = desc->q_ln2;
  h->sc.q_b = desc->q_b;
  h->sc.q_c = desc->q_c;
  plan_fused_score(&h->sc, desc->d_k, false);
  h->has_run = false;
  h->last_was_residual = false;
  h->last_ws = Workspace{};
  h->last_noalloc = false;
  h->stages_pending = false;
  h->pcache = nullptr;
  h->pcache_T = 0;
  h->pcache_rows = 0;
  h->res = Residual{};
  h->has_res = false;

  const size_t d = h->d, H = h->H, DK = h->DK, Bm = h->max_B;
  const size_t T_al = t_aligned(h->max_T), PR = p_rows((int)T_al);
  hipError_t e = hipSuccess;
  auto chk = [&](hipError_t r) {
    if (e == hipSuccess) e = r;
  };
  chk(dev_alloc(h, &h->w.w_qkv, 3 * d * d));
  chk(dev_alloc(h, &h->w.w_pos, d * d));
  chk(dev_alloc(h, &h->w.w_out, d * d));
  chk(dev_alloc(h, &h->w.u, H * DK));
  chk(dev_alloc(h, &h->w.v, H * DK));
  chk(dev_alloc(h, &h->w.etab, 256));
  chk(dev_alloc(h, &h->ws.q, Bm * H * T_al * DK));
  chk(dev_alloc(h, &h->ws.k, Bm * H * T_al * DK));
  chk(dev_alloc(h, &h->ws.vt, Bm * H * DK * T_al));
  chk(dev_alloc(h, &h->ws.p, H * PR * DK));
  chk(dev_alloc(h, &h->ws.ctx, Bm * (size_t)h->max_T * d));
  if (e != hipSuccess) {
    free_handle(h);
    (void)hipGetLastError();
    return fail(e == hipErrorOutOfMemory ? IPK_ERR_OUT_OF_MEMORY : IPK_ERR_HIP, "device allocation failed: %s",
                hipGetErrorString(e));
  }
  // weights (device to device), multipliers (host to device).  Every weight matrix is
  // kept in MFMA fragment order (the projection kernels stream them straight into
  // registers): each is staged row-major in a temporary buffer and rearranged from
  // there, the stacked Q|K|V in one pass.
  int8_t* stage = nullptr;
  chk(dev_alloc(h, &stage, 3 * d * d));
  chk(hipMemcpy(stage, desc->w_q, d * d, hipMemcpyDefault));
  chk(hipMemcpy(stage + d * d, desc->w_k, d * d, hipMemcpyDefault));
  chk(hipMemcpy(stage + 2 * d * d, desc->w_v, d * d, hipMemcpyDefault));
  chk(pack_weight_fragments(stage, h->w.w_qkv, 3 * (int)d, (int)d, nullptr));
  chk(hipMemcpy(stage, desc->w_pos, d * d, hipMemcpyDefault));
  chk(pack_weight_fragments(stage, h->w.w_pos, (int)d, (int)d, nullptr));
  chk(hipMemcpy(stage, desc->w_out, d * d, hipMemcpyDefault));
  chk(pack_weight_fragments(stage, h->w.w_out, (int)d, (int)d, nullptr));
  chk(hipMemcpy(h->w.u, desc->pos_bias_u, H * DK, hipMemcpyDefault));
  chk(hipMemcpy(h->w.v, desc->pos_bias_v, H * DK, hipMemcpyDefault));
  chk(launch_iexp_table(h->w.etab, desc->q_ln2, desc->q_b, desc->q_c, nullptr));
  // Eq. 7 constants per output channel (integers only)
  {
    const int32_t* mq[3] = {desc->mult_q, desc->mult_k, desc->mult_v};
    const int32_t sq[3] = {desc->shift_q, desc->shift_k, desc->shift_v};
    chk(upload_requant(h, &h->w.rq_qkv, mq, sq, 3, (int)d));
    chk(upload_requant(h, &h->w.rq_pos, &desc->mult_pos, &desc->shift_pos, 1, (int)d));
    chk(upload_requant(h, &h->w.rq_out, &desc->mult_out, &desc->shift_out, 1, (int)d));
  }
  // deterministic contents for the padding rows of the workspace
  chk(hipMemset(h->ws.p, 0, H * PR * DK));
  chk(hipMemset(h->ws.vt, 0, Bm * H * DK * T_al));
  chk(hipMemset(h->ws.k, 0, Bm * H * T_al * DK));
  chk(hipMemset(h->ws.q, 0, Bm * H * T_al * DK));
  chk(hipDeviceSynchronize());
  if (e != hipSuccess) {
    free_handle(h);
    (void)hipGetLastError();
    return fail(IPK_ERR_HIP, "copying the weights failed: %s", hipGetErrorString(e));
  }
  // the staging copy is no longer needed
  h->allocs.erase(std::find(h->allocs.begin(), h->allocs.end(), (void*)stage));
  (void)hipFree(stage);
  *out = h;
  return IPK_OK;
}

// Validates a run's arguments and fills its shape and lengths.
static int validate_run(ipk_relpos_attn* h, const int8_t* x, const int8_t* pos_table, const int32_t* lengths,
                        int32_t B, int32_t T, int8_t* y, RunShape* rs, Lengths* lens) {
  if (((uintptr_t)x | (uintptr_t)pos_table | (uintptr_t)y) & 15)
    return fail(IPK_ERR_INVALID_ARG, "the input, pos_table and output must be 16-byte aligned");
  if (B < 1 || B > h->max_B) return fail(IPK_ERR_INVALID_ARG, "B=%d outside [1, max_batch=%d]", B, h->max_B);
  if (T < 1 || T > h->max_T) return fail(IPK_ERR_INVALID_ARG, "T=%d outside [1, max_T=%d]", T, h->max_T);
  if (!pos_table && T > h->pcache_T)
    return fail(IPK_ERR_INVALID_ARG,
                h->pcache_T ? "pos_table is NULL and the kept projection covers T <= %d only" :
                              "pos_table is NULL and no position projection is kept (T_table %d)",
                h->pcache_T);
  for (int b = 0; b < B; ++b) {
    const int L = lengths ? lengths[b] : T;
    if (L < 1 || L > T) return fail(IPK_ERR_INVALID_ARG, "lengths[%d]=%d outside [1, T=%d]", b, L, T);
    lens->len[b] = L;
  }
  for (int b = B; b < IPK_MAX_BATCH; ++b) lens->len[b] = 0;
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != h->device)
    return fail(IPK_ERR_INVALID_ARG, "the current HIP device (%d) is not the handle's (%d)", cur, h->device);
  *rs = RunShape{B, T, t_aligned(T), h->H, h->DK, h->d, p_base_row(T), p_rows(t_aligned(T))};
  return IPK_OK;
}

// Enqueues a validated run on the buffers of `ws`: LayerNorm (z1 != NULL, the MHSA
// module), projections, attention core, output projection (with the residual add when
// z1 != NULL).  With pos_table NULL the kept projection replaces ws.p.
static int enqueue_run(ipk_relpos_attn* h, RunShape rs, const Lengths& lens, Workspace ws, const int8_t* x,
                       const int8_t* pos_table, int8_t* y, void* stream, const int8_t* z1, bool noalloc) {
  if (!pos_table) {
    // table row r of this T is row r + T_table - T of the kept one, whose relative
    // position 0 sits at a 16-row boundary for every T
    ws.p = h->pcache;
    rs.p_rows = h->pcache_rows;
    rs.p_base = p_base_row(h->pcache_T) + h->pcache_T - rs.T;
  }
  hipStream_t st = (hipStream_t)stream;
  const bool rec = h->stages_pending;
  h->stages_pending = false;
  // stage events ride on the kernel dispatches: event i is stamped when stage i
  // starts, event 3 when the last kernel ends (no separate event packets)
  LaunchEv ev[3];
  if (rec) {
    for (int i = 0; i < 3; ++i) ev[i].start = h->stage_ev[i];
    ev[2].stop = h->stage_ev[3];
  }
  hipError_t e = hipSuccess;
  if (z1) {
    e = launch_layernorm(rs, h->res, z1, ws.xln, st, ev[0]);
    x = ws.xln;
    ev[0] = LaunchEv{};
  }
  if (e == hipSuccess) e = launch_projections(rs, h->w, ws, x, pos_table, st, ev[0]);
  if (e == hipSuccess) e = launch_attention(rs, h->w, h->sc, ws, lens, st, ev[1]);
  if (e == hipSuccess) e = launch_out_projection(rs, h->w, ws, y, st, ev[2], z1 ? &h->res : nullptr, z1);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  h->last = rs;
  h->last_ws = ws;
  h->last_lens = lens;
  h->last_sc = h->sc;
  h->last_noalloc = noalloc;
  h->has_run = true;
  h->last_was_residual = z1 != nullptr;
  return IPK_OK;
}

static int run_on_handle(ipk_relpos_attn* h, const int8_t* x, const int8_t* pos_table, const int32_t* lengths,
                         int32_t B, int32_t T, int8_t* y, void* stream, const int8_t* z1) {
  RunShape rs;
  Lengths lens;
  const int st = validate_run(h, x, pos_table, lengths, B, T, y, &rs, &lens);
  if (st != IPK_OK) return st;
  return enqueue_run(h, rs, lens, h->ws, x, pos_table, y, stream, z1, false);
}

extern "C" int ipk_relpos_attn_run(ipk_relpos_attn_t* h, const int8_t* x, const int8_t* pos_table,
                                   const int32_t* lengths, int32_t B, int32_t T, int8_t* y, void* stream) {
  if (!h) return fail(IPK_ERR_INVALID_ARG, "handle is NULL");
  if (!x || !y) return fail(IPK_ERR_INVALID_ARG, "x and y must be non-NULL");
  return run_on_handle(h, x, pos_table, lengths, B, T, y, stream, nullptr);
}

// Bytes of a run's workspace for (B, T) carved from one block at `base` (each buffer
// at a 256-byte boundary), the projected table only when the run projects one; with
// base = NULL only the size is computed.
static size_t carve_workspace(const RunShape& rs, bool own_p, uint8_t* base, Workspace* ws) {
  size_t off = 0;
  auto take = [&](size_t bytes) {
    uint8_t* p = base ? base + off : nullptr;
    off += (bytes + 255) & ~(size_t)255;
    return p;
  };
  const size_t B = rs.B, H = rs.H, DK = rs.DK, T_al = rs.T_al;
  ws->q = (int8_t*)take(B * H * T_al * DK);
  ws->k = (int8_t*)take(B * H * T_al * DK);
  ws->vt = (int8_t*)take(B * H * DK * T_al);
  ws->p = own_p ? (int8_t*)take(H * (size_t)rs.p_rows * DK) : nullptr;
  ws->ctx = (int8_t*)take(B * (size_t)rs.T * rs.d);
  ws->xln = nullptr;
  return off;
}

extern "C" int ipk_relpos_attn_run_noalloc(ipk_relpos_attn_t* h, const int8_t* x, const int8_t* pos_table,
                                           const int32_t* lengths, int32_t B, int32_t T, int8_t* y, void* stream) {
  if (!h) return fail(IPK_ERR_INVALID_ARG, "handle is NULL");
  if (!x || !y) return fail(IPK_ERR_INVALID_ARG, "x and y must be non-NULL");
  RunShape rs;
  Lengths lens;
  const int st = validate_run(h, x, pos_table, lengths, B, T, y, &rs, &lens);
  if (st != IPK_OK) return st;
  Workspace ws{};
  const size_t need = carve_workspace(rs, pos_table != nullptr, nullptr, &ws);
  if (need > IPK_NOALLOC_SCRATCH_BYTES)
    return fail(IPK_ERR_UNSUPPORTED, "B=%d, T=%d needs %zu bytes of workspace; the no-allocation run holds %zu", B, T,
                need, (size_t)IPK_NOALLOC_SCRATCH_BYTES);
  uint8_t* base = nullptr;
  size_t cap = 0;
  const hipError_t e = noalloc_scratch(&base, &cap);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "looking up the scratch array failed: %s", hipGetErrorString(e));
  carve_workspace(rs, pos_table != nullptr, base, &ws);
  return enqueue_run(h, rs, lens, ws, x, pos_table, y, stream, nullptr, true);
}

extern "C" int ipk_mhsa_residual_run(ipk_relpos_attn_t* h, const int8_t* z1, const int8_t* pos_table,
                                     const int32_t* lengths, int32_t B, int32_t T, int8_t* z2, void* stream) {
  if (!h) return fail(IPK_ERR_INVALID_ARG, "handle is NULL");
  if (!z1 || !z2) return fail(IPK_ERR_INVALID_ARG, "z1 and z2 must be non-NULL");
  if (!h->has_res) return fail(IPK_ERR_INVALID_ARG, "no LayerNorm / residual constants set (ipk_mhsa_residual_set)");
  if (B >= 1 && T >= 1 && z1 != z2) {
    const size_t n = (size_t)B * T * h->d;
    const uintptr_t a = (uintptr_t)z1, b = (uintptr_t)z2;
    if (a < b + n && b < a + n) return fail(IPK_ERR_INVALID_ARG, "z1 and z2 overlap without being equal");
  }
  return run_on_handle(h, z1, pos_table, lengths, B, T, z2, stream, z1);
}

extern "C" int ipk_mhsa_residual_set(ipk_relpos_attn_t* h, const ipk_mhsa_residual_desc* r) {
  if (!h || !r) return fail(IPK_ERR_INVALID_ARG, "handle and desc must be non-NULL");
  if (!r->ln_mult || !r->ln_bias) return fail(IPK_ERR_INVALID_ARG, "ln_mult and ln_bias must be non-NULL");
  if (r->ln_shift < 1 || r->ln_shift > 62) return fail(IPK_ERR_INVALID_ARG, "ln_shift=%d outside [1, 62]", r->ln_shift);
  if (!mult_ok(r->m_z) || !mult_ok(r->m_y))
    return fail(IPK_ERR_INVALID_ARG, "m_z=%d, m_y=%d must be in [0, 2^23)", r->m_z, r->m_y);
  if (!shift_ok(r->shift_r)) return fail(IPK_ERR_INVALID_ARG, "shift_r=%d outside [1, 40]", r->shift_r);
  const int d = h->d;
  std::vector<int64_t> cb(d);
  for (int k = 0; k < d; ++k) {
    if (r->ln_mult[k] <= -(1 << 24) || r->ln_mult[k] >= (1 << 24))
      return fail(IPK_ERR_INVALID_ARG, "ln_mult[%d]=%d outside (-2^24, 2^24)", k, r->ln_mult[k]);
    if (r->ln_bias[k] <= -((int64_t)1 << 56) || r->ln_bias[k] >= ((int64_t)1 << 56))
      return fail(IPK_ERR_INVALID_ARG, "ln_bias[%d] outside (-2^56, 2^56)", k);
    cb[k] = r->ln_bias[k] + ((int64_t)1 << (r->ln_shift - 1));
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != h->device)
    return fail(IPK_ERR_INVALID_ARG, "the current HIP device (%d) is not the handle's (%d)", cur, h->device);
  hipError_t e = hipSuccess;
  auto chk = [&](hipError_t x) {
    if (e == hipSuccess) e = x;
  };
  if (!h->ws.xln) {
    int32_t* g = nullptr;
    int64_t* c = nullptr;
    int8_t* xln = nullptr;
    chk(dev_alloc(h, &g, d));
    chk(dev_alloc(h, &c, d));
    chk(dev_alloc(h, &xln, (size_t)h->max_B * h->max_T * d));
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(e == hipErrorOutOfMemory ? IPK_ERR_OUT_OF_MEMORY : IPK_ERR_HIP, "device allocation failed: %s",
                  hipGetErrorString(e));
    }
    h->res.ln_mult = g;
    h->res.ln_bias = c;
    h->ws.xln = xln;
  }
  // stream-ordered after every run already enqueued on the handle's device
  chk(hipDeviceSynchronize());
  chk(hipMemcpy((void*)h->res.ln_mult, r->ln_mult, d * sizeof(int32_t), hipMemcpyHostToDevice));
  chk(hipMemcpy((void*)h->res.ln_bias, cb.data(), d * sizeof(int64_t), hipMemcpyHostToDevice));
  chk(hipDeviceSynchronize());
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(IPK_ERR_HIP, "copying the LayerNorm constants failed: %s", hipGetErrorString(e));
  }
  h->res.ln_shift = r->ln_shift;
  h->res.m_z = r->m_z;
  h->res.m_y = r->m_y;
  h->res.shift_r = r->shift_r;
  h->has_res = true;
  return IPK_OK;
}

extern "C" int ipk_relpos_attn_cache_positions(ipk_relpos_attn_t* h, const int8_t* pos_table, int32_t T_table,
                                               void* stream) {
  if (!h || !pos_table) return fail(IPK_ERR_INVALID_ARG, "handle and pos_table must be non-NULL");
  if ((uintptr_t)pos_table & 15) return fail(IPK_ERR_INVALID_ARG, "pos_table must be 16-byte aligned");
  if (T_table < 1 || T_table > h->max_T)
    return fail(IPK_ERR_INVALID_ARG, "T_table=%d outside [1, max_T=%d]", T_table, h->max_T);
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != h->device)
    return fail(IPK_ERR_INVALID_ARG, "the current HIP device (%d) is not the handle's (%d)", cur, h->device);
  // rows per head: the table at its 16-aligned base (at most P_PADLO + 15) plus the
  // padding the attention core's windows reach past either end, sized for max_T
  const int rows = P_PADLO + 16 + 2 * t_aligned(h->max_T) + P_PADHI;
  if (!h->pcache) {
    int8_t* p = nullptr;
    hipError_t e = dev_alloc(h, &p, (size_t)h->H * rows * h->DK);
    if (e == hipSuccess) e = hipMemset(p, 0, (size_t)h->H * rows * h->DK);
    if (e != hipSuccess) {
      (void)hipGetLastError();
      return fail(e == hipErrorOutOfMemory ? IPK_ERR_OUT_OF_MEMORY : IPK_ERR_HIP, "device allocation failed: %s",
                  hipGetErrorString(e));
    }
    h->pcache = p;
    h->pcache_rows = rows;
  }
  RunShape rs{1, T_table, t_aligned(T_table), h->H, h->DK, h->d, p_base_row(T_table), rows};
  hipError_t e = launch_pos_projection(rs, h->w, h->pcache, pos_table, (hipStream_t)stream);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  h->pcache_T = T_table;
  return IPK_OK;
}

extern "C" int ipk_relpos_attn_intermediate(ipk_relpos_attn_t* h, int32_t which, void* dst, int64_t bytes,
                                            void* stream) {
  if (!h || !dst) return fail(IPK_ERR_INVALID_ARG, "handle and dst must be non-NULL");
  if (!h->has_run) return fail(IPK_ERR_INVALID_ARG, "no run yet");
  if (which < IPK_INTER_Q || which > IPK_INTER_XLN) return fail(IPK_ERR_INVALID_ARG, "unknown intermediate %d", which);
  if (which == IPK_INTER_XLN && !h->last_was_residual)
    return fail(IPK_ERR_INVALID_ARG, "the last run was not an MHSA module run: no LayerNorm output");
  const RunShape& rs = h->last;
  const int64_t need = (which == IPK_INTER_P ? (int64_t)(2 * rs.T - 1) : (int64_t)rs.B * rs.T) * rs.d;
  if (bytes < need) return fail(IPK_ERR_INVALID_ARG, "dst holds %lld bytes, %lld needed", (long long)bytes, (long long)need);
  hipError_t e = launch_gather_intermediate(rs, h->last_ws, which, (int8_t*)dst, (hipStream_t)stream);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "gather failed: %s", hipGetErrorString(e));
  return IPK_OK;
}

extern "C" int ipk_relpos_attn_record_stages(ipk_relpos_attn_t* h, void* const* events) {
  if (!h) return fail(IPK_ERR_INVALID_ARG, "handle is NULL");
  if (!events) {
    h->stages_pending = false;
    return IPK_OK;
  }
  for (int i = 0; i < IPK_NUM_STAGES + 1; ++i)
    if (!events[i]) return fail(IPK_ERR_INVALID_ARG, "events[%d] is NULL", i);
  for (int i = 0; i < IPK_NUM_STAGES + 1; ++i) h->stage_ev[i] = (hipEvent_t)events[i];
  h->stages_pending = true;
  return IPK_OK;
}

extern "C" int ipk_relpos_attn_repeat_core(ipk_relpos_attn_t* h, int32_t count, void* stream) {
  if (!h) return fail(IPK_ERR_INVALID_ARG, "handle is NULL");
  if (!h->has_run) return fail(IPK_ERR_INVALID_ARG, "no run yet");
  if (h->last_noalloc)
    return fail(IPK_ERR_INVALID_ARG, "the last run worked in the shared no-allocation array, not the handle's workspace");
  if (count < 1 || count > IPK_MAX_REPEAT) return fail(IPK_ERR_INVALID_ARG, "count=%d outside [1, %d]", count, IPK_MAX_REPEAT);
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != h->device)
    return fail(IPK_ERR_INVALID_ARG, "the current HIP device (%d) is not the handle's (%d)", cur, h->device);
  for (int i = 0; i < count; ++i) {
    const hipError_t e = launch_attention(h->last, h->w, h->last_sc, h->last_ws, h->last_lens, (hipStream_t)stream,
                                          LaunchEv{});
    if (e != hipSuccess) return fail(IPK_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  }
  return IPK_OK;
}

extern "C" int ipk_relpos_attn_set_score_path(ipk_relpos_attn_t* h, int32_t path) {
  if (!h) return fail(IPK_ERR_INVALID_ARG, "handle is NULL");
  if (path != IPK_SCORE_AUTO && path != IPK_SCORE_WIDE) return fail(IPK_ERR_INVALID_ARG, "unknown score path %d", path);
  plan_fused_score(&h->sc, h->DK, path == IPK_SCORE_WIDE);
  return IPK_OK;
}

extern "C" int ipk_relpos_attn_score_path(const ipk_relpos_attn_t* h) {
  if (!h) return fail(IPK_ERR_INVALID_ARG, "handle is NULL");
  return h->sc.fs_wide ? IPK_SCORE_WIDE : IPK_SCORE_NARROW;
}

extern "C" int ipk_relpos_attn_destroy(ipk_relpos_attn_t* h) {
  if (!h) return IPK_OK;
  int prev = -1;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(h->device);
  hipError_t e = hipDeviceSynchronize();
  free_handle(h);
  if (prev >= 0) (void)hipSetDevice(prev);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "device error at destroy: %s", hipGetErrorString(e));
  return IPK_OK;
}

// ---------------------------------------------------------------------------
// The feed-forward module of Eq. 1.

struct ipk_ffn {
  int device;
  int d, f, max_rows;
  int8_t *w1, *w2;            // fragment order (wfrag_index)
  Requant rq1, rq2;           // Eq. 7 constants of W1 and W2
  uint8_t* swtab;             // 256 bytes: Swish output of each biased code h + 128
  int8_t *x, *o;              // LayerNorm output [max_rows][d], Swish output [max_rows][f]
  Residual res;
  int last_rows;
  std::vector<void*> allocs;
};

static void free_ffn(ipk_ffn* h) {
  if (!h) return;
  for (void* p : h->allocs) (void)hipFree(p);
  delete h;
}

static int validate_ffn(const ipk_ffn_desc* D) {
  if (!D) return fail(IPK_ERR_INVALID_ARG, "desc is NULL");
  if (D->d_model < 64 || D->d_model % 64 || D->d_model > 16384)
    return fail(IPK_ERR_INVALID_ARG, "d_model=%d must be a multiple of 64 in [64, 16384]", D->d_model);
  if (D->d_ff < 64 || D->d_ff % 64 || D->d_ff > 65536)
    return fail(IPK_ERR_INVALID_ARG, "d_ff=%d must be a multiple of 64 in [64, 65536]", D->d_ff);
  if (D->max_rows < 1 || (int64_t)D->max_rows * D->d_ff >= ((int64_t)1 << 31))
    return fail(IPK_ERR_INVALID_ARG, "max_rows=%d outside [1, 2^31 / d_ff)", D->max_rows);
  if (!D->w1 || !D->w2 || !D->mult1 || !D->mult2 || !D->ln_mult || !D->ln_bias)
    return fail(IPK_ERR_INVALID_ARG, "a weight, multiplier or LayerNorm pointer is NULL");
  for (int c = 0; c < D->d_ff; ++c)
    if (!mult_ok(D->mult1[c])) return fail(IPK_ERR_INVALID_ARG, "mult1[%d]=%d outside [0, 2^23)", c, D->mult1[c]);
  for (int c = 0; c < D->d_model; ++c)
    if (!mult_ok(D->mult2[c])) return fail(IPK_ERR_INVALID_ARG, "mult2[%d]=%d outside [0, 2^23)", c, D->mult2[c]);
  if (!shift_ok(D->shift1) || !shift_ok(D->shift2) || !shift_ok(D->shift_sw) || !shift_ok(D->shift_r))
    return fail(IPK_ERR_INVALID_ARG, "a shift is outside [1, 40]");
  if (D->ln_shift < 1 || D->ln_shift > 62) return fail(IPK_ERR_INVALID_ARG, "ln_shift=%d outside [1, 62]", D->ln_shift);
  if (!mult_ok(D->m_sw) || !mult_ok(D->m_z) || !mult_ok(D->m_y))
    return fail(IPK_ERR_INVALID_ARG, "m_sw, m_z and m_y must be in [0, 2^23)");
  for (int k = 0; k < D->d_model; ++k) {
    if (D->ln_mult[k] <= -(1 << 24) || D->ln_mult[k] >= (1 << 24))
      return fail(IPK_ERR_INVALID_ARG, "ln_mult[%d]=%d outside (-2^24, 2^24)", k, D->ln_mult[k]);
    if (D->ln_bias[k] <= -((int64_t)1 << 56) || D->ln_bias[k] >= ((int64_t)1 << 56))
      return fail(IPK_ERR_INVALID_ARG, "ln_bias[%d] outside (-2^56, 2^56)", k);
  }
  if (D->sw_qc < 0 || D->sw_qc >= (1 << 20)) return fail(IPK_ERR_INVALID_ARG, "sw_qc=%d outside [0, 2^20)", D->sw_qc);
  if (D->sw_q1 <= -((int64_t)1 << 45) || D->sw_q1 >= ((int64_t)1 << 45))
    return fail(IPK_ERR_INVALID_ARG, "sw_q1 outside (-2^45, 2^45)");
  // the Swish table kernel evaluates q m_sw + 2^(n-1) in 64 bits: bound it for every h
  for (int hv = -127; hv <= 127; ++hv) {
    const __int128 ah = hv < 0 ? -hv : hv;
    const __int128 t = (ah < D->sw_qc ? ah : (__int128)D->sw_qc) - D->sw_qc;
    const __int128 L = t * t + D->sw_q1;
    __int128 q = -(ah * L + (__int128)hv * D->sw_q1);
    if (q < 0) q = -q;
    if (q * D->m_sw + ((__int128)1 << (D->shift_sw - 1)) >= ((__int128)1 << 62))
      return fail(IPK_ERR_UNSUPPORTED, "integer Swish times m_sw reaches 2^62 at h=%d", hv);
  }
  return IPK_OK;
}

extern "C" int ipk_ffn_create(const ipk_ffn_desc* desc, ipk_ffn_t** out) {
  g_last_error[0] = 0;
  if (!out) return fail(IPK_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  int st = validate_ffn(desc);
  if (st != IPK_OK) return st;
  ipk_ffn* h = new (std::nothrow) ipk_ffn();
  if (!h) return fail(IPK_ERR_OUT_OF_MEMORY, "host allocation failed");
  if (hipGetDevice(&h->device) != hipSuccess) {
    free_ffn(h);
    return fail(IPK_ERR_HIP, "hipGetDevice failed");
  }
  const size_t d = desc->d_model, f = desc->d_ff, R = desc->max_rows;
  h->d = (int)d;
  h->f = (int)f;
  h->max_rows = (int)R;
  h->last_rows = 0;
  hipError_t e = hipSuccess;
  auto chk = [&](hipError_t r) {
    if (e == hipSuccess) e = r;
  };
  int32_t* g = nullptr;
  int64_t* c = nullptr;
  int8_t* stage = nullptr;
  chk(dev_alloc(h, &h->w1, f * d));
  chk(dev_alloc(h, &h->w2, d * f));
  chk(dev_alloc(h, &h->swtab, 256));
  chk(dev_alloc(h, &h->x, R * d));
  chk(dev_alloc(h, &h->o, R * f));
  chk(dev_alloc(h, &g, d));
  chk(dev_alloc(h, &c, d));
  chk(dev_alloc(h, &stage, f * d));
  if (e != hipSuccess) {
    free_ffn(h);
    (void)hipGetLastError();
    return fail(e == hipErrorOutOfMemory ? IPK_ERR_OUT_OF_MEMORY : IPK_ERR_HIP, "device allocation failed: %s",
                hipGetErrorString(e));
  }
  chk(hipMemcpy(stage, desc->w1, f * d, hipMemcpyDefault));
  chk(pack_weight_fragments(stage, h->w1, (int)f, (int)d, nullptr));
  chk(hipMemcpy(stage, desc->w2, d * f, hipMemcpyDefault));
  chk(pack_weight_fragments(stage, h->w2, (int)d, (int)f, nullptr));
  chk(upload_requant(h, &h->rq1, &desc->mult1, &desc->shift1, 1, (int)f));
  chk(upload_requant(h, &h->rq2, &desc->mult2, &desc->shift2, 1, (int)d));
  std::vector<int64_t> cb(d);
  for (size_t k = 0; k < d; ++k) cb[k] = desc->ln_bias[k] + ((int64_t)1 << (desc->ln_shift - 1));
  chk(hipMemcpy(g, desc->ln_mult, d * sizeof(int32_t), hipMemcpyHostToDevice));
  chk(hipMemcpy(c, cb.data(), d * sizeof(int64_t), hipMemcpyHostToDevice));
  chk(launch_swish_table(h->swtab, desc->sw_qc, desc->sw_q1, desc->m_sw, desc->shift_sw, nullptr));
  chk(hipDeviceSynchronize());
  if (e != hipSuccess) {
    free_ffn(h);
    (void)hipGetLastError();
    return fail(IPK_ERR_HIP, "copying the weights failed: %s", hipGetErrorString(e));
  }
  h->allocs.erase(std::find(h->allocs.begin(), h->allocs.end(), (void*)stage));
  (void)hipFree(stage);
  h->res.ln_mult = g;
  h->res.ln_bias = c;
  h->res.ln_shift = desc->ln_shift;
  h->res.m_z = desc->m_z;
  h->res.m_y = desc->m_y;
  h->res.shift_r = desc->shift_r;
  *out = h;
  return IPK_OK;
}

extern "C" int ipk_ffn_run(ipk_ffn_t* h, const int8_t* z, int32_t rows, int8_t* z_out, void* stream) {
  if (!h) return fail(IPK_ERR_INVALID_ARG, "handle is NULL");
  if (!z || !z_out) return fail(IPK_ERR_INVALID_ARG, "z and z_out must be non-NULL");
  if (((uintptr_t)z | (uintptr_t)z_out) & 15) return fail(IPK_ERR_INVALID_ARG, "z and z_out must be 16-byte aligned");
  if (rows < 1 || rows > h->max_rows) return fail(IPK_ERR_INVALID_ARG, "rows=%d outside [1, max_rows=%d]", rows, h->max_rows);
  if (z != z_out) {
    const size_t n = (size_t)rows * h->d;
    const uintptr_t a = (uintptr_t)z, b = (uintptr_t)z_out;
    if (a < b + n && b < a + n) return fail(IPK_ERR_INVALID_ARG, "z and z_out overlap without being equal");
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != h->device)
    return fail(IPK_ERR_INVALID_ARG, "the current HIP device (%d) is not the handle's (%d)", cur, h->device);
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = launch_layernorm_rows(rows, h->d, h->res, z, h->x, st);
  if (e == hipSuccess) e = launch_ffn_up(h->x, rows, h->d, h->f, h->w1, h->rq1, h->swtab, h->o, st);
  if (e == hipSuccess)
    e = launch_linear_resid(h->o, rows, h->d, h->f, h->w2, h->rq2, z, h->res.m_z, h->res.m_y, h->res.shift_r, z_out,
                            st);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  h->last_rows = rows;
  return IPK_OK;
}

extern "C" int ipk_ffn_intermediate(ipk_ffn_t* h, int32_t which, void* dst, int64_t bytes, void* stream) {
  if (!h || !dst) return fail(IPK_ERR_INVALID_ARG, "handle and dst must be non-NULL");
  if (!h->last_rows) return fail(IPK_ERR_INVALID_ARG, "no run yet");
  if (which != IPK_FFN_X && which != IPK_FFN_O) return fail(IPK_ERR_INVALID_ARG, "unknown intermediate %d", which);
  const int64_t need = (int64_t)h->last_rows * (which == IPK_FFN_X ? h->d : h->f);
  if (bytes < need) return fail(IPK_ERR_INVALID_ARG, "dst holds %lld bytes, %lld needed", (long long)bytes, (long long)need);
  hipError_t e = hipMemcpyAsync(dst, which == IPK_FFN_X ? h->x : h->o, (size_t)need, hipMemcpyDeviceToDevice,
                                (hipStream_t)stream);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "copy failed: %s", hipGetErrorString(e));
  return IPK_OK;
}

extern "C" int ipk_ffn_destroy(ipk_ffn_t* h) {
  if (!h) return IPK_OK;
  int prev = -1;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(h->device);
  hipError_t e = hipDeviceSynchronize();
  free_ffn(h);
  if (prev >= 0) (void)hipSetDevice(prev);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "device error at destroy: %s", hipGetErrorString(e));
  return IPK_OK;
}

// ---------------------------------------------------------------------------
// The convolution module of Eq. 3 and Eq. 5.

struct ipk_conv {
  int device;
  int d, max_B, max_T;
  int8_t *w_pw1, *w_pw2;        // fragment order (wfrag_index)
  Requant rq_pw1, rq_pw2;       // Eq. 7 constants of PW1 and PW2
  ConvMiddle mid;               // depthwise weights and constants (device copies)
  int8_t *x, *u, *o;            // LayerNorm output, PW1 output [.][2 d], Swish output
  int16_t* v;                   // int16 BatchNorm output (written on request only)
  Residual res;
  int last_B, last_T;
  Lengths last_lens;            // the last run's lengths (to recompute v on request)
  std::vector<void*> allocs;
};

static void free_conv(ipk_conv* h) {
  if (!h) return;
  for (void* p : h->allocs) (void)hipFree(p);
  delete h;
}

static __int128 poly_l128(__int128 aq, __int128 q_c, __int128 q_1) {
  const __int128 t = (aq < q_c ? aq : q_c) - q_c;
  return t * t + q_1;
}

static int validate_conv(const ipk_conv_desc* D) {
  if (!D) return fail(IPK_ERR_INVALID_ARG, "desc is NULL");
  if (D->d_model < 64 || D->d_model % 64 || D->d_model > 16384)
    return fail(IPK_ERR_INVALID_ARG, "d_model=%d must be a multiple of 64 in [64, 16384]", D->d_model);
  if (D->max_batch < 1 || D->max_batch > IPK_MAX_BATCH)
    return fail(IPK_ERR_INVALID_ARG, "max_batch=%d outside [1, %d]", D->max_batch, IPK_MAX_BATCH);
  if (D->max_T < 1 || D->max_T > IPK_MAX_T) return fail(IPK_ERR_INVALID_ARG, "max_T=%d outside [1, %d]", D->max_T, IPK_MAX_T);
  if ((int64_t)D->max_batch * D->max_T * 2 * D->d_model >= ((int64_t)1 << 31))
    return fail(IPK_ERR_UNSUPPORTED, "max_batch * max_T * 2 d_model reaches 2^31");
  if (!D->w_pw1 || !D->w_dw || !D->w_pw2 || !D->mult_pw1 || !D->bias_dw || !D->mult_dw || !D->mult_pw2 ||
      !D->ln_mult || !D->ln_bias)
    return fail(IPK_ERR_INVALID_ARG, "a weight, multiplier, bias or LayerNorm pointer is NULL");
  const int d = D->d_model;
  for (int c = 0; c < 2 * d; ++c)
    if (!mult_ok(D->mult_pw1[c])) return fail(IPK_ERR_INVALID_ARG, "mult_pw1[%d]=%d outside [0, 2^23)", c, D->mult_pw1[c]);
  for (int c = 0; c < d; ++c) {
    if (!mult_ok(D->mult_dw[c])) return fail(IPK_ERR_INVALID_ARG, "mult_dw[%d]=%d outside [0, 2^23)", c, D->mult_dw[c]);
    if (!mult_ok(D->mult_pw2[c])) return fail(IPK_ERR_INVALID_ARG, "mult_pw2[%d]=%d outside [0, 2^23)", c, D->mult_pw2[c]);
    if (D->bias_dw[c] <= -(1 << 30) || D->bias_dw[c] >= (1 << 30))
      return fail(IPK_ERR_INVALID_ARG, "bias_dw[%d]=%d outside (-2^30, 2^30)", c, D->bias_dw[c]);
    if (D->ln_mult[c] <= -(1 << 24) || D->ln_mult[c] >= (1 << 24))
      return fail(IPK_ERR_INVALID_ARG, "ln_mult[%d]=%d outside (-2^24, 2^24)", c, D->ln_mult[c]);
    if (D->ln_bias[c] <= -((int64_t)1 << 56) || D->ln_bias[c] >= ((int64_t)1 << 56))
      return fail(IPK_ERR_INVALID_ARG, "ln_bias[%d] outside (-2^56, 2^56)", c);
  }
  if (!shift_ok(D->shift_pw1) || !shift_ok(D->shift_dw) || !shift_ok(D->shift_pw2) || !shift_ok(D->shift_r))
    return fail(IPK_ERR_INVALID_ARG, "shift_pw1, shift_dw, shift_pw2 and shift_r must be in [1, 40]");
  if (D->shift_glu < 1 || D->shift_glu > 62 || D->shift_sw < 1 || D->shift_sw > 62)
    return fail(IPK_ERR_INVALID_ARG, "shift_glu and shift_sw must be in [1, 62]");
  if (D->ln_shift < 1 || D->ln_shift > 62) return fail(IPK_ERR_INVALID_ARG, "ln_shift=%d outside [1, 62]", D->ln_shift);
  if (!mult_ok(D->m_glu) || !mult_ok(D->m_sw) || !mult_ok(D->m_z) || !mult_ok(D->m_y))
    return fail(IPK_ERR_INVALID_ARG, "m_glu, m_sw, m_z and m_y must be in [0, 2^23)");
  if (D->glu_qc < 0 || D->glu_qc >= (1 << 20) || D->sw_qc < 0 || D->sw_qc >= (1 << 20))
    return fail(IPK_ERR_INVALID_ARG, "glu_qc and sw_qc must be in [0, 2^20)");
  const int64_t q1lim = (int64_t)1 << 45;
  if (D->glu_q1 <= -q1lim || D->glu_q1 >= q1lim || D->sw_q1 <= -q1lim || D->sw_q1 >= q1lim)
    return fail(IPK_ERR_INVALID_ARG, "glu_q1 and sw_q1 must be in (-2^45, 2^45)");
  // the kernel's 64-bit products: GLU over every int8 (a, b), Swish over every int16 v
  const __int128 lim = (__int128)1 << 62;
  __int128 smax = 0;
  for (int b = -127; b <= 127; ++b) {
    const __int128 ab = b < 0 ? -b : b, sg = b > 0 ? 1 : (b < 0 ? -1 : 0);
    __int128 sgm = -((__int128)D->glu_q1 + sg * poly_l128(ab, D->glu_qc, D->glu_q1));
    if (sgm < 0) sgm = -sgm;
    if (sgm > smax) smax = sgm;
  }
  if (smax * 128 * D->m_glu + ((__int128)1 << (D->shift_glu - 1)) >= lim)
    return fail(IPK_ERR_UNSUPPORTED, "GLU product times m_glu reaches 2^62");
  for (int vv = -32767; vv <= 32767; ++vv) {
    const __int128 av = vv < 0 ? -vv : vv;
    __int128 q = -(av * poly_l128(av, D->sw_qc, D->sw_q1) + (__int128)vv * D->sw_q1);
    if (q < 0) q = -q;
    if (q * D->m_sw + ((__int128)1 << (D->shift_sw - 1)) >= lim)
      return fail(IPK_ERR_UNSUPPORTED, "Swish of the int16 value %d times m_sw reaches 2^62", vv);
  }
  return IPK_OK;
}

extern "C" int ipk_conv_create(const ipk_conv_desc* desc, ipk_conv_t** out) {
  g_last_error[0] = 0;
  if (!out) return fail(IPK_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  int st = validate_conv(desc);
  if (st != IPK_OK) return st;
  ipk_conv* h = new (std::nothrow) ipk_conv();
  if (!h) return fail(IPK_ERR_OUT_OF_MEMORY, "host allocation failed");
  if (hipGetDevice(&h->device) != hipSuccess) {
    free_conv(h);
    return fail(IPK_ERR_HIP, "hipGetDevice failed");
  }
  const size_t d = desc->d_model, R = (size_t)desc->max_batch * desc->max_T;
  h->d = (int)d;
  h->max_B = desc->max_batch;
  h->max_T = desc->max_T;
  h->last_B = h->last_T = 0;
  hipError_t e = hipSuccess;
  auto chk = [&](hipError_t r) {
    if (e == hipSuccess) e = r;
  };
  int8_t *wdw = nullptr, *stage = nullptr;
  int32_t *bias = nullptr, *mdw = nullptr, *g = nullptr;
  int64_t* c = nullptr;
  chk(dev_alloc(h, &h->w_pw1, 2 * d * d));
  chk(dev_alloc(h, &h->w_pw2, d * d));
  chk(dev_alloc(h, &wdw, d * 9));
  chk(dev_alloc(h, &bias, d));
  chk(dev_alloc(h, &mdw, d));
  chk(dev_alloc(h, &g, d));
  chk(dev_alloc(h, &c, d));
  chk(dev_alloc(h, &h->x, R * d));
  chk(dev_alloc(h, &h->u, R * 2 * d));
  chk(dev_alloc(h, &h->o, R * d));
  chk(dev_alloc(h, &h->v, R * d));
  chk(dev_alloc(h, &stage, 2 * d * d));
  int8_t* sw16 = nullptr;
  chk(dev_alloc(h, &sw16, 65535));
  int8_t* glu = nullptr;
  chk(dev_alloc(h, &glu, 65536));
  if (e != hipSuccess) {
    free_conv(h);
    (void)hipGetLastError();
    return fail(e == hipErrorOutOfMemory ? IPK_ERR_OUT_OF_MEMORY : IPK_ERR_HIP, "device allocation failed: %s",
                hipGetErrorString(e));
  }
  chk(hipMemcpy(stage, desc->w_pw1, 2 * d * d, hipMemcpyDefault));
  chk(pack_weight_fragments(stage, h->w_pw1, 2 * (int)d, (int)d, nullptr));
  chk(hipMemcpy(stage, desc->w_pw2, d * d, hipMemcpyDefault));
  chk(pack_weight_fragments(stage, h->w_pw2, (int)d, (int)d, nullptr));
  chk(hipMemcpy(wdw, desc->w_dw, d * 9, hipMemcpyDefault));
  chk(upload_requant(h, &h->rq_pw1, &desc->mult_pw1, &desc->shift_pw1, 1, 2 * (int)d));
  chk(upload_requant(h, &h->rq_pw2, &desc->mult_pw2, &desc->shift_pw2, 1, (int)d));
  chk(hipMemcpy(bias, desc->bias_dw, d * sizeof(int32_t), hipMemcpyHostToDevice));
  chk(hipMemcpy(mdw, desc->mult_dw, d * sizeof(int32_t), hipMemcpyHostToDevice));
  std::vector<int64_t> cb(d);
  for (size_t k = 0; k < d; ++k) cb[k] = desc->ln_bias[k] + ((int64_t)1 << (desc->ln_shift - 1));
  chk(hipMemcpy(g, desc->ln_mult, d * sizeof(int32_t), hipMemcpyHostToDevice));
  chk(hipMemcpy(c, cb.data(), d * sizeof(int64_t), hipMemcpyHostToDevice));
  chk(launch_swish16_table(sw16, desc->sw_qc, desc->sw_q1, desc->m_sw, desc->shift_sw, nullptr));
  chk(launch_glu_table(glu, desc->glu_qc, desc->glu_q1, desc->m_glu, desc->shift_glu, nullptr));
  chk(hipDeviceSynchronize());
  if (e != hipSuccess) {
    free_conv(h);
    (void)hipGetLastError();
    return fail(IPK_ERR_HIP, "copying the weights failed: %s", hipGetErrorString(e));
  }
  h->allocs.erase(std::find(h->allocs.begin(), h->allocs.end(), (void*)stage));
  (void)hipFree(stage);
  h->mid.w_dw = wdw;
  h->mid.bias_dw = bias;
  h->mid.mult_dw = mdw;
  h->mid.shift_dw = desc->shift_dw;
  h->mid.glu_qc = desc->glu_qc;
  h->mid.glu_q1 = desc->glu_q1;
  h->mid.m_glu = desc->m_glu;
  h->mid.shift_glu = desc->shift_glu;
  h->mid.swtab16 = sw16;
  h->mid.glutab = glu;
  h->res.ln_mult = g;
  h->res.ln_bias = c;
  h->res.ln_shift = desc->ln_shift;
  h->res.m_z = desc->m_z;
  h->res.m_y = desc->m_y;
  h->res.shift_r = desc->shift_r;
  *out = h;
  return IPK_OK;
}

extern "C" int ipk_conv_run(ipk_conv_t* h, const int8_t* z, const int32_t* lengths, int32_t B, int32_t T, int8_t* z_out,
                            void* stream) {
  if (!h) return fail(IPK_ERR_INVALID_ARG, "handle is NULL");
  if (!z || !z_out) return fail(IPK_ERR_INVALID_ARG, "z and z_out must be non-NULL");
  if (((uintptr_t)z | (uintptr_t)z_out) & 15) return fail(IPK_ERR_INVALID_ARG, "z and z_out must be 16-byte aligned");
  if (B < 1 || B > h->max_B) return fail(IPK_ERR_INVALID_ARG, "B=%d outside [1, max_batch=%d]", B, h->max_B);
  if (T < 1 || T > h->max_T) return fail(IPK_ERR_INVALID_ARG, "T=%d outside [1, max_T=%d]", T, h->max_T);
  Lengths lens;
  for (int b = 0; b < B; ++b) {
    const int L = lengths ? lengths[b] : T;
    if (L < 1 || L > T) return fail(IPK_ERR_INVALID_ARG, "lengths[%d]=%d outside [1, T=%d]", b, L, T);
    lens.len[b] = L;
  }
  for (int b = B; b < IPK_MAX_BATCH; ++b) lens.len[b] = 0;
  const size_t n = (size_t)B * T * h->d;
  if (z != z_out) {
    const uintptr_t a = (uintptr_t)z, b = (uintptr_t)z_out;
    if (a < b + n && b < a + n) return fail(IPK_ERR_INVALID_ARG, "z and z_out overlap without being equal");
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != h->device)
    return fail(IPK_ERR_INVALID_ARG, "the current HIP device (%d) is not the handle's (%d)", cur, h->device);
  hipStream_t st = (hipStream_t)stream;
  const int rows = B * T;
  hipError_t e = launch_layernorm_rows(rows, h->d, h->res, z, h->x, st);
  if (e == hipSuccess) e = launch_linear(h->x, rows, h->d, 2 * h->d, h->w_pw1, h->rq_pw1, h->u, st);
  // the int16 BatchNorm output is not stored on a run (ipk_conv_intermediate recomputes it)
  if (e == hipSuccess) e = launch_conv_middle(h->mid, h->u, lens, B, T, h->d, h->o, nullptr, st);
  if (e == hipSuccess)
    e = launch_linear_resid(h->o, rows, h->d, h->d, h->w_pw2, h->rq_pw2, z, h->res.m_z, h->res.m_y,
                            h->res.shift_r, z_out, st);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  h->last_B = B;
  h->last_T = T;
  h->last_lens = lens;
  return IPK_OK;
}

extern "C" int ipk_conv_intermediate(ipk_conv_t* h, int32_t which, void* dst, int64_t bytes, void* stream) {
  if (!h || !dst) return fail(IPK_ERR_INVALID_ARG, "handle and dst must be non-NULL");
  if (!h->last_B) return fail(IPK_ERR_INVALID_ARG, "no run yet");
  const int64_t rows = (int64_t)h->last_B * h->last_T;
  const void* src = nullptr;
  int64_t need = 0;
  switch (which) {
    case IPK_CONV_X: src = h->x; need = rows * h->d; break;
    case IPK_CONV_U: src = h->u; need = rows * 2 * h->d; break;
    case IPK_CONV_V: src = h->v; need = rows * h->d * 2; break;
    case IPK_CONV_O: src = h->o; need = rows * h->d; break;
    default: return fail(IPK_ERR_INVALID_ARG, "unknown intermediate %d", which);
  }
  if (bytes < need) return fail(IPK_ERR_INVALID_ARG, "dst holds %lld bytes, %lld needed", (long long)bytes, (long long)need);
  hipError_t e = hipSuccess;
  if (which == IPK_CONV_V)  // rerun the middle kernel on the kept PW1 output, storing v (o is rewritten unchanged)
    e = launch_conv_middle(h->mid, h->u, h->last_lens, h->last_B, h->last_T, h->d, h->o, h->v, (hipStream_t)stream);
  if (e == hipSuccess) e = hipMemcpyAsync(dst, src, (size_t)need, hipMemcpyDeviceToDevice, (hipStream_t)stream);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "copy failed: %s", hipGetErrorString(e));
  return IPK_OK;
}

extern "C" int ipk_conv_destroy(ipk_conv_t* h) {
  if (!h) return IPK_OK;
  int prev = -1;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(h->device);
  hipError_t e = hipDeviceSynchronize();
  free_conv(h);
  if (prev >= 0) (void)hipSetDevice(prev);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "device error at destroy: %s", hipGetErrorString(e));
  return IPK_OK;
}

// ---------------------------------------------------------------------------
// The integer LayerNorm alone (the final LN of Eq. 4).

struct ipk_layernorm {
  int device, d;
  Residual res;  // only the LayerNorm fields are used
  std::vector<void*> allocs;
};

static void free_ln(ipk_layernorm* h) {
  if (!h) return;
  for (void* p : h->allocs) (void)hipFree(p);
  delete h;
}

extern "C" int ipk_layernorm_create(const ipk_layernorm_desc* desc, ipk_layernorm_t** out) {
  g_last_error[0] = 0;
  if (!out) return fail(IPK_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!desc) return fail(IPK_ERR_INVALID_ARG, "desc is NULL");
  const int d = desc->d_model;
  if (d < 16 || d % 16 || d > 16384) return fail(IPK_ERR_INVALID_ARG, "d_model=%d must be a multiple of 16 in [16, 16384]", d);
  if (!desc->ln_mult || !desc->ln_bias) return fail(IPK_ERR_INVALID_ARG, "ln_mult and ln_bias must be non-NULL");
  if (desc->ln_shift < 1 || desc->ln_shift > 62) return fail(IPK_ERR_INVALID_ARG, "ln_shift=%d outside [1, 62]", desc->ln_shift);
  std::vector<int64_t> cb(d);
  for (int k = 0; k < d; ++k) {
    if (desc->ln_mult[k] <= -(1 << 24) || desc->ln_mult[k] >= (1 << 24))
      return fail(IPK_ERR_INVALID_ARG, "ln_mult[%d]=%d outside (-2^24, 2^24)", k, desc->ln_mult[k]);
    if (desc->ln_bias[k] <= -((int64_t)1 << 56) || desc->ln_bias[k] >= ((int64_t)1 << 56))
      return fail(IPK_ERR_INVALID_ARG, "ln_bias[%d] outside (-2^56, 2^56)", k);
    cb[k] = desc->ln_bias[k] + ((int64_t)1 << (desc->ln_shift - 1));
  }
  ipk_layernorm* h = new (std::nothrow) ipk_layernorm();
  if (!h) return fail(IPK_ERR_OUT_OF_MEMORY, "host allocation failed");
  h->d = d;
  hipError_t e = hipGetDevice(&h->device);
  void *g = nullptr, *c = nullptr;
  if (e == hipSuccess) e = hipMalloc(&g, d * sizeof(int32_t));
  if (e == hipSuccess) h->allocs.push_back(g);
  if (e == hipSuccess) e = hipMalloc(&c, d * sizeof(int64_t));
  if (e == hipSuccess) h->allocs.push_back(c);
  if (e == hipSuccess) e = hipMemcpy(g, desc->ln_mult, d * sizeof(int32_t), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemcpy(c, cb.data(), d * sizeof(int64_t), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    free_ln(h);
    (void)hipGetLastError();
    return fail(e == hipErrorOutOfMemory ? IPK_ERR_OUT_OF_MEMORY : IPK_ERR_HIP, "device setup failed: %s",
                hipGetErrorString(e));
  }
  h->res.ln_mult = (const int32_t*)g;
  h->res.ln_bias = (const int64_t*)c;
  h->res.ln_shift = desc->ln_shift;
  *out = h;
  return IPK_OK;
}

extern "C" int ipk_layernorm_run(ipk_layernorm_t* h, const int8_t* z, int64_t rows, int8_t* x, void* stream) {
  if (!h) return fail(IPK_ERR_INVALID_ARG, "handle is NULL");
  if (!z || !x) return fail(IPK_ERR_INVALID_ARG, "z and x must be non-NULL");
  if (((uintptr_t)z | (uintptr_t)x) & 15) return fail(IPK_ERR_INVALID_ARG, "z and x must be 16-byte aligned");
  if (rows < 1 || rows > ((int64_t)1 << 31) / h->d) return fail(IPK_ERR_INVALID_ARG, "rows=%lld outside [1, 2^31 / d)", (long long)rows);
  if (z != x) {
    const size_t n = (size_t)rows * h->d;
    const uintptr_t a = (uintptr_t)z, b = (uintptr_t)x;
    if (a < b + n && b < a + n) return fail(IPK_ERR_INVALID_ARG, "z and x overlap without being equal");
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != h->device)
    return fail(IPK_ERR_INVALID_ARG, "the current HIP device (%d) is not the handle's (%d)", cur, h->device);
  hipError_t e = launch_layernorm_rows((long)rows, h->d, h->res, z, x, (hipStream_t)stream);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(e));
  return IPK_OK;
}

extern "C" int ipk_layernorm_destroy(ipk_layernorm_t* h) {
  if (!h) return IPK_OK;
  int prev = -1;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(h->device);
  hipError_t e = hipDeviceSynchronize();
  free_ln(h);
  if (prev >= 0) (void)hipSetDevice(prev);
  if (e != hipSuccess) return fail(IPK_ERR_HIP, "device error at destroy: %s", hipGetErrorString(e));
  return IPK_OK;
}

extern "C" const char* ipk_status_string(int status) {
  switch (status) {
    case IPK_OK: return "IPK_OK";
    case IPK_ERR_INVALID_ARG: return "IPK_ERR_INVALID_ARG";
    case IPK_ERR_UNSUPPORTED: return "IPK_ERR_UNSUPPORTED";
    case IPK_ERR_OUT_OF_MEMORY: return "IPK_ERR_OUT_OF_MEMORY";
    case IPK_ERR_HIP: return "IPK_ERR_HIP";
    default: return "IPK_ERR_UNKNOWN";
  }
}

extern "C" const char* ipk_last_error(void) { return g_last_error; }

extern "C" int ipk_abi_version(void) { return IPK_ABI_VERSION; }
