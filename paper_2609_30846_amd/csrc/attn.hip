// Relative-position attention core of the integer MHSA block (Sec. 3.1).
//
// Work split: a workgroup of ATTN_WAVES waves owns (utterance b, head h, WGQ
// consecutive queries).  Each wave owns NTL 16-query MFMA tiles (32 or 48 queries:
// every K, P and V fragment it loads feeds NTL MFMAs, and the loads bound the
// kernel); KSPLIT waves share one set of queries and split its keys: phase 1 in
// 16-key steps, phases 2 and 3 in 64-key chunks (scores are exchanged through LDS in
// between).  The host picks (KSPLIT, NTL) per launch from the LDS the score rows need
// and the rounds of workgroups over the CUs.
//
// Phase 1, per 16-key step, with v_mfma_i32_16x16x64_i8 (queries on MFMA rows):
//  * content   c = Q K^T, accumulator seeded with the rank-1 term u.K_j
//  * position  G = Q P_win^T, seeded with v.P_r, for the 16 table rows that
//              start at relative position j0-i0+T-1 ("hi" window).  The rows
//              just before it ("lo") are the previous step's hi window, and tile t
//              reuses the P fragment tile 0 loaded t steps earlier, so each step
//              loads one new P fragment and runs one new position MFMA pair per
//              tile.
//  * Phi       p_ij = G_i(j-i+T-1) is a rotation by the row index inside each
//              16-lane row group: every source lane picks the window its value
//              belongs to and ds_bpermute moves it to the lane of its key.
//  * Eq. 11    s = clamp8(RS(m_c c + m_p p, 1, n)), exact: in 32-bit
//              integers when the descriptor bounds |m_c c + m_p p| below 2^31,
//              otherwise in float64 (every intermediate is an integer below 2^53).
//              Scores are kept as biased codes s + 128 in [1, 255].
//  * each of the four scores a lane holds (four queries, one key) is stored as
//    one byte of its query's score row (ds_write_b8 of the code's byte; packing
//    and transposing them first cost more than it saved): the int8 score rows of
//    the workgroup stay in LDS, never in HBM.
// Phase 2: row max (shuffles + LDS across the KSPLIT waves), I-BERT integer exp
// of every distance d = max - s from a table, row sums, F = floor(2^32 / sum).
// Phase 3: per-row tables of the softmax code a = min(floor(e F / 2^24), 255),
// stored as a - 128; A.V on MFMA with that signed operand plus the exact
// correction 128 * sum_j V_j over the same keys (per-chunk sums of V, fetched
// with the V fragments; V is streamed in parts of four 16-channel tiles); partial
// contexts of the KSPLIT waves are added with LDS atomics (exact int32) and
// requantized with (m_o, shift_o) by all waves together.
// Both lookup tables are laid out [d][32 banks] in dwords: the exp table holds one
// copy per bank (lane l reads copy l % 32); the code tables hold bytes, row r = 16 tt
// + rr in byte tt of banks rr and rr + 16, and the two half-waves' lanes g = 0, 1 (2,
// 3) read different copies, so a lookup is one multiply-add and one conflict-free
// LDS read.
#include <mutex>
#include <type_traits>
#include <utility>
#include <vector>

#include "ipk_internal.h"

namespace ipk {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef uint16_t us2 __attribute__((ext_vector_type(2)));

struct AttnArgs {
  const int8_t *q, *k, *vt, *p;
  const int8_t *u, *v;  // [H][d_k]
  const int32_t* vsum;
  int8_t* ctx;
  Lengths lens;
  int T, T_al, H, d, p_rows, p_base;
  int nqb;        // query blocks per (utterance, head) of the first segment
  int xcd_group;  // keep each (utterance, head) on one XCD
  // second segment of a two-shape grid: blocks from seg2_block on cover the queries
  // from seg2_q0 on, nqb2 blocks per (utterance, head), with the second shape
  int seg2_block, seg2_q0, nqb2;
  // fused score: narrow path
  int32_t mc24, mp24, bias32, post_shift;
  // fused score: wide path (multipliers scaled by 2^-shift_s)
  double mcd, mpd;
  int32_t m_o, shift_o, q_ln2, q_b, q_c;
};

constexpr int SCORE_PAD = 16;  // bytes added to each LDS score row
constexpr int TAB_DW = 256 * 32;  // dwords of the [d][32 banks] lookup-table region

__device__ __forceinline__ uint32_t iexp_int(int d, int q_ln2, int q_b, int q_c) {
  // I-BERT integer exp of -d: d = z q_ln2 - r with r in (-q_ln2, 0]
  const int z = d / q_ln2;
  const int r = z * q_ln2 - d;
  const int poly = (r + q_b) * (r + q_b) + q_c;  // < 2^24 (checked at create)
  return z >= 32 ? 0u : ((uint32_t)poly >> z);
}

// Low 32 bits of a * b + c for 24-bit signed a, b (v_mad_i32_i24); the addition
// wraps modulo 2^32.
__device__ __forceinline__ int mad_i24(int a, int b, int c) {
  return (int)((uint32_t)__mul24(a, b) + (uint32_t)c);
}

constexpr int ATTN_WAVES = 8;  // waves per workgroup (two per SIMD)
// Share (out of 256) of a SIMD's keys that its older wave takes in phase 1 and in
// phases 2 and 3.  With equal shares the younger wave of a pair ends phase 1 about
// 1.35x and phase 3 about 1.25x later than the older one on the long-form workload;
// these shares (about 65 % and 59 %) measured fastest over the whole kernel.
constexpr int P1_OLDER = 166;
constexpr int P3_OLDER = 150;

template <int S>
using Phase = std::integral_constant<int, S>;

// One workgroup of the core: block `lin` of a segment of nqb query blocks per
// (utterance, head) that starts at query q_base.
template <int DK, int KSPLIT, int NTL, bool WIDE>
__device__ __forceinline__ void attn_block(const AttnArgs& a, unsigned char* smem, const int lin, const int nqb,
                                           const int q_base) {
  constexpr int NQS = ATTN_WAVES / KSPLIT;  // query sets per workgroup
  constexpr int ROWS = 16 * NTL;            // queries per set: NTL 16-query MFMA tiles
  constexpr int WGQ = ROWS * NQS;           // queries per workgroup
  constexpr int NKS = DK / 64;              // MFMA K-steps over d_k
  constexpr int NT = DK / 16;               // 16-channel output tiles of the context
  static_assert(NQS * NTL <= 4, "the code tables hold four 16-row tiles");

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index: uniform, kept in SGPRs
  const int col = lane & 15, g = lane >> 4;
  // Waves w and w + 4 share SIMD w % 4, whose instruction arbiter favours the older
  // one (the lower index): given equal work, the younger wave finishes long after it
  // and runs its tail alone.  The two waves of a SIMD therefore take the same query set
  // and split its keys unevenly, the older one taking the larger share.
  constexpr int HK = KSPLIT > 1 ? KSPLIT / 2 : 1;  // key parts per age class
  const int simd = w & 3, younger = w >> 2;
  const int qset = KSPLIT > 1 ? simd / HK : w;
  const int kpart = KSPLIT > 1 ? younger * HK + simd % HK : 0;
  const int slot = qset * KSPLIT + kpart;  // this wave's row-max and row-sum slot
  // work units [*b, *e) of this wave out of n: every SIMD gets n / HK of them, of
  // which its older wave takes older / 256 (rounded) and its younger wave the rest
  auto split = [&](const int n, const int older, int* b, int* e) {
    if (KSPLIT == 1) {
      *b = 0;
      *e = n;
      return;
    }
    const int pair = kpart % HK;
    const int ps = n * pair / HK, pe = n * (pair + 1) / HK;
    const int mid = ps + ((pe - ps) * older + 128) / 256;
    *b = younger ? mid : ps;
    *e = younger ? pe : mid;
  };
  // Workgroups go round-robin to the 8 XCDs (id % 8); when the (utterance, head)
  // pairs divide evenly, every workgroup of one pair is placed on the same XCD so that
  // its K, P and V stay in that XCD's L2.
  int qb, bhi;
  if (a.xcd_group) {
    const int x = lin & 7, k = lin >> 3, slot = k / nqb;
    qb = k - slot * nqb;
    bhi = x + 8 * slot;
  } else {
    qb = lin % nqb;
    bhi = lin / nqb;
  }
  const int b = bhi / a.H, h = bhi - (bhi / a.H) * a.H;
  const int wg_q0 = q_base + qb * WGQ;
  const int q0 = wg_q0 + ROWS * qset;  // first query of this wave
  const int L = a.lens.len[b];
  const int T = a.T, T_al = a.T_al;
  const int srow = T_al + SCORE_PAD;
  const int nkc = (L + KCHUNK - 1) / KCHUNK;
  int c_begin, c_end;
  split(nkc, P3_OLDER, &c_begin, &c_end);
  // chunks below c_full hold only valid keys; c_full < c_end only when this wave's
  // range holds the chunk with the utterance's last key (an empty range past it too
  // ends at c_full = c_end)
  const int c_full = max(c_begin, min(c_end, L / KCHUNK));
  const bool active = q0 < L;

  // LDS carve-up (the host computes the same sizes)
  constexpr int RSTRIDE = DK + 4;  // dwords per row of the key-split partial sums
  const int s_bytes = WGQ * srow;
  const int red_bytes = KSPLIT > 1 ? NQS * ROWS * RSTRIDE * 4 : 0;
  const int big = ((s_bytes > red_bytes ? s_bytes : red_bytes) + 15) & ~15;
  uint8_t* sbuf = smem;
  int32_t* red = (int32_t*)smem;  // reused once the scores are consumed
  // lookup tables, [d][32 banks] in dwords: first the per-bank copies of the exp
  // table (phase 2), then the code tables (phase 3)
  uint32_t* tab = (uint32_t*)(smem + big);
  uint32_t* etab = tab + TAB_DW;  // the 255 exp values, once
  int32_t* smax = (int32_t*)(etab + 256);
  uint32_t* ssum = (uint32_t*)(smax + ROWS * ATTN_WAVES);
  uint32_t* sF = ssum + ROWS * ATTN_WAVES;

  const size_t bh = (size_t)b * a.H + h;
  const int8_t* Qh = a.q + bh * T_al * DK;
  const int8_t* Kh = a.k + bh * T_al * DK;
  const int8_t* VTh = a.vt + bh * DK * T_al;
  const int8_t* Ph = a.p + (size_t)h * a.p_rows * DK;
  const int32_t* vs = a.vsum + bh * (size_t)(T_al / KCHUNK) * DK;
  uint8_t* my_rows = sbuf + (size_t)(ROWS * qset) * srow;
  // this lane's 16 bytes of a 1 KB operand fragment (stored in lane order)
  const int frag_off = lane * 16;

  constexpr int LOCODE = WIDE ? 1 : (1 << 16);  // code of s = -127 (biased s + 128)
  constexpr int HICODE = WIDE ? 255 : ((255 << 16) | 0xFFFF);

  // ---------------- phase 1: fused scores into LDS, running row max
  int mx[NTL][4];
#pragma unroll
  for (int t = 0; t < NTL; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) mx[t][i] = LOCODE;

  // phase 1 splits the 16-key steps that hold a valid key over the key parts
  const int nst = (L + 15) >> 4;
  int j_begin, j_stop;
  split(nst, P1_OLDER, &j_begin, &j_stop);
  j_begin *= 16;
  j_stop *= 16;
  const int j_full = max(j_begin, min(j_stop, L & ~15));  // steps below this are unmasked
  if (active && j_begin < j_stop) {
    const uint32_t frag = (uint32_t)frag_off;
    v4i qf[NTL][NKS];
#pragma unroll
    for (int t = 0; t < NTL; ++t) {
      // a tile past the padded sequence (last workgroup, T_al not a multiple of the
      // workgroup's queries) re-reads the last tile: its rows are never stored
      const int qrow = min(q0 + 16 * t, T_al - 16);
#pragma unroll
      for (int s = 0; s < NKS; ++s) qf[t][s] = *(const v4i*)(Qh + (size_t)qrow * DK + frag + s * 1024);
    }
    bool take_hi[4];
    int src_addr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int arow = 4 * g + i;
      take_hi[i] = (col + arow) < 16;                    // as a source lane
      src_addr[i] = (g * 16 + ((col - arow) & 15)) * 4;  // as a destination lane
    }
    // a lane's score of query row 4g + i of tile t and key j0 + col is one byte of
    // the row: stored directly, so no packing or transposing is spent on it
    uint8_t* sdst = my_rows + (size_t)(4 * g) * srow + col;

    // K and the position table are streamed with raw buffer loads: the lane's offset in
    // a fragment is fixed and the step's offset is a scalar, so no vector address
    // arithmetic is spent per load.  Table row of (query q0, key j0) is
    // j0 - q0 + T - 1; tile t sits 16 t rows lower.  Every offset stays inside the
    // padded buffers (the table keeps P_PADLO rows below row 0).
    const __amdgpu_buffer_rsrc_t kres =
        __builtin_amdgcn_make_buffer_rsrc((void*)Kh, (short)0, T_al * DK, BUF_WORD3);
    const __amdgpu_buffer_rsrc_t pres =
        __builtin_amdgcn_make_buffer_rsrc((void*)Ph, (short)0, a.p_rows * DK, BUF_WORD3);
    int koff = __builtin_amdgcn_readfirstlane(j_begin * DK);
    int poff = __builtin_amdgcn_readfirstlane((a.p_base + j_begin - q0 + T - 1) * DK);
    auto ldk = [&](int off, int s) { return (v4i)__builtin_amdgcn_raw_buffer_load_b128(kres, frag + s * 1024, off, 0); };
    auto ldp = [&](int off, int s) { return (v4i)__builtin_amdgcn_raw_buffer_load_b128(pres, frag + s * 1024, off, 0); };
    // The rank-1 terms of Eq. 8 come from MFMAs of a 16-row operand whose rows all
    // equal u (v): their products with a K (P) fragment hold u.K_j (v.P_r) in every
    // row, which is the accumulator seed the content (position) MFMAs need.  No load
    // is spent on them.
    v4i uf[NKS], vf[NKS];
#pragma unroll
    for (int s = 0; s < NKS; ++s) {
      uf[s] = *(const v4i*)(a.u + (size_t)h * DK + s * 64 + g * 16);
      vf[s] = *(const v4i*)(a.v + (size_t)h * DK + s * 64 + g * 16);
    }
    auto rank1 = [&](const v4i* vec, const v4i* fr) {
      v4i r = (v4i){0, 0, 0, 0};
#pragma unroll
      for (int s = 0; s < NKS; ++s) r = __builtin_amdgcn_mfma_i32_16x16x64_i8(vec[s], fr[s], r, 0, 0, 0);
      return r;
    };

    // Register rings over the step phase S = (step index) % RING, all indices static
    // (RING = NTL, and 2 for a single tile, so that the current and the next step never
    // share a slot):
    //  pr[u]:    tile 0's hi-window P fragment of the step with phase u; at phase S
    //            tile t uses slot (S - t) mod RING (its window is tile 0's window of t
    //            steps before)
    //  kr[u]:    K fragment of the step with phase u (current, next)
    //  gr[u][t]: position MFMA results (hi windows) of the step with phase u; a
    //            step's lo windows are the previous step's hi windows
    constexpr int RING = NTL > 1 ? NTL : 2;
    v4i pr[RING][NKS], kr[RING][NKS], gr[RING][NTL];
    int bvp[RING];
    auto splat = [](int bb) { return (v4i){bb, bb, bb, bb}; };
    {
      // tile t's hi window of the first step: tile 0's window 16 t rows lower
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
        const int u = (RING - t) % RING;
#pragma unroll
        for (int s = 0; s < NKS; ++s) pr[u][s] = ldp(poff - 16 * t * DK, s);
      }
      // lo windows of the first step: tile t's lo window is tile (t + 1)'s hi window;
      // the last tile's lies one more window lower
      v4i plast[NKS];
#pragma unroll
      for (int s = 0; s < NKS; ++s) plast[s] = ldp(poff - 16 * NTL * DK, s);
#pragma unroll
      for (int t = 0; t < NTL; ++t) bvp[(RING - t) % RING] = rank1(vf, pr[(RING - t) % RING])[0];
      const int bvlast = rank1(vf, plast)[0];
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
        const int u = (RING - t - 1) % RING;  // slot of tile (t + 1)'s hi window
        v4i gacc = splat(t + 1 < NTL ? bvp[u] : bvlast);
#pragma unroll
        for (int s = 0; s < NKS; ++s)
          gacc = __builtin_amdgcn_mfma_i32_16x16x64_i8(qf[t][s], t + 1 < NTL ? pr[u][s] : plast[s], gacc, 0, 0, 0);
        gr[RING - 1][t] = gacc;
      }
    }
#pragma unroll
    for (int s = 0; s < NKS; ++s) kr[0][s] = ldk(koff, s);

    int j0 = j_begin;
    // One 16-key step at phase S: fetches the next step's K and P fragments (the last
    // step re-reads its own rows, in bounds), runs the content and position MFMAs of
    // every tile and turns them into score codes in LDS.
    auto step = [&](auto Sc, const bool masked) {
      constexpr int S = decltype(Sc)::value;
      constexpr int SN = (S + 1) % RING, SP = (S + RING - 1) % RING;
      const int adv = j0 + 16 < j_stop ? 16 * DK : 0;
#pragma unroll
      for (int s = 0; s < NKS; ++s) kr[SN][s] = ldk(koff + adv, s);
      // seeds: u.K_j of this step's keys (shared by the tiles) and, per tile, v.P_r
      // of the tile's window (recomputed rather than kept: the matrix pipe has room,
      // the registers do not)
      const v4i uk = rank1(uf, kr[S]);
      bvp[S] = rank1(vf, pr[S])[0];
      v4i cs[NTL];
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
        cs[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(qf[t][0], kr[S][0], uk, 0, 0, 0);
        gr[S][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(qf[t][0], pr[(S + RING - t) % RING][0],
                                                         splat(bvp[(S + RING - t) % RING]), 0, 0, 0);
      }
#pragma unroll
      for (int s = 1; s < NKS; ++s)
#pragma unroll
        for (int t = 0; t < NTL; ++t) {
          cs[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(qf[t][s], kr[S][s], cs[t], 0, 0, 0);
          gr[S][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(qf[t][s], pr[(S + RING - t) % RING][s], gr[S][t], 0, 0, 0);
        }
      // the last tile's window (slot SN) is consumed: it takes the next step's tile-0 window
#pragma unroll
      for (int s = 0; s < NKS; ++s) pr[SN][s] = ldp(poff + adv, s);
      // cs holds c0 + u.K_j: the addend is the rounding and code bias alone
      const int k1 = a.bias32;
      const double k1d = 128.5;
      const bool key_ok = j0 + col < L;
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int sel = take_hi[i] ? gr[S][t][i] : gr[SP][t][i];
          const int pt = __builtin_amdgcn_ds_bpermute(src_addr[i], sel);
          int v;
          if (WIDE) {
            // truncation equals the floor here: every negative value clamps to code 1
            v = (int)__builtin_fma(a.mcd, (double)cs[t][i], __builtin_fma(a.mpd, (double)pt, k1d));
          } else {
            int x = mad_i24(a.mp24, pt, k1);
            asm("" : "+v"(x));  // opaque to the optimizer (keeps the multiply-adds apart), not a scheduling barrier
            v = mad_i24(a.mc24, cs[t][i], x);
          }
          v = min(max(v, LOCODE), HICODE);
          if (masked && !key_ok) v = LOCODE;
          mx[t][i] = max(mx[t][i], v);
          // the code is bits 0..7 (wide path) or 16..23 (narrow path) of v
          sdst[(size_t)(16 * t + i) * srow + j0] = (uint8_t)(WIDE ? v : (v >> 16));
        }
      }
      koff += 16 * DK;
      poff += 16 * DK;
      j0 += 16;
    };
    // RING unmasked steps per iteration, so that every ring index stays static
    while (j0 + 16 * RING <= j_full) {
      step(Phase<0>{}, false);
      step(Phase<1>{}, false);
      if constexpr (RING > 2) step(Phase<2 % RING>{}, false);
    }
    // the rest (fewer than RING steps below j_full, then the masked ones)
    int ph = 0;
    while (j0 < j_stop) {
      const bool m = j0 + 16 > j_full;
      if (ph == 0)
        step(Phase<0>{}, m);
      else if (ph == 1 || RING == 2)
        step(Phase<1 % RING>{}, m);
      else
        step(Phase<2 % RING>{}, m);
      ph = ph + 1 == RING ? 0 : ph + 1;
    }
  }
  // I-BERT integer exp of every score distance d = M - s in [0, 254] (first read in
  // phase 2, so waves that finish phase 1 early fill it while the others score): once, and
  // in 32 per-bank copies (copy (d + c) % 32 of the pass is written by lane d,
  // which keeps the writes free of bank conflicts)
  {
    const int dd = tid & 255;
    const uint32_t e = dd < 255 ? iexp_int(dd, a.q_ln2, a.q_b, a.q_c) : 0u;
    if (tid < 256) etab[dd] = e;
    for (int c = (tid >> 8) * 16; c < 32; c += 16 * (64 * ATTN_WAVES / 256)) {
#pragma unroll
      for (int k = 0; k < 16; ++k) tab[dd * 32 + ((c + k + dd) & 31)] = e;
    }
  }

  // row max over the 16 key lanes of each row group
#pragma unroll
  for (int t = 0; t < NTL; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int v = mx[t][i];
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) v = max(v, __shfl_xor(v, o));
      mx[t][i] = v;
    }
  if (col == 0) {
#pragma unroll
    for (int t = 0; t < NTL; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) smax[slot * ROWS + 16 * t + 4 * g + i] = WIDE ? mx[t][i] : (mx[t][i] >> 16);
  }
  __syncthreads();

  // phases 2 and 3: lane (g, col) works on query row `col` of each tile and keys
  // g*16 .. g*16+15 of a chunk
  int Mrow[NTL];
  const uint8_t* srd[NTL];
#pragma unroll
  for (int t = 0; t < NTL; ++t) {
    int m = 1;
#pragma unroll
    for (int k2 = 0; k2 < KSPLIT; ++k2) m = max(m, smax[(qset * KSPLIT + k2) * ROWS + 16 * t + col]);
    Mrow[t] = m;
    srd[t] = my_rows + (size_t)(16 * t + col) * srow + g * 16;
  }

  // ---------------- phase 2: row sums of the integer exp
  // lane l reads copy l % 32 of the exp table: e(M - code) at erow[-32 code]
  uint32_t sum[NTL];
#pragma unroll
  for (int t = 0; t < NTL; ++t) sum[t] = 0u;
  if (active) {
    const uint32_t* erow[NTL];
#pragma unroll
    for (int t = 0; t < NTL; ++t) erow[t] = tab + Mrow[t] * 32 + (lane & 31);
    for (int c = c_begin; c < c_full; ++c) {
      // all lookups of the chunk are issued before any is summed (LDS latency
      // overlaps instead of being paid once per four codes)
      v4i sv[NTL];
#pragma unroll
      for (int t = 0; t < NTL; ++t) sv[t] = *(const v4i*)(srd[t] + c * KCHUNK);
      uint32_t ev[NTL][16];
#pragma unroll
      for (int t = 0; t < NTL; ++t)
#pragma unroll
        for (int k = 0; k < 16; ++k)
          ev[t][k] = erow[t][__mul24(-32, (int)(((uint32_t)sv[t][k >> 2] >> (8 * (k & 3))) & 0xff))];
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
        uint32_t acc_e = 0;
#pragma unroll
        for (int k = 0; k < 16; ++k) acc_e += ev[t][k];
        sum[t] += acc_e;
      }
    }
    if (c_full < c_end) {  // the chunk that holds the utterance's last key
      const int c = c_full;
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
        const v4i sv = *(const v4i*)(srd[t] + c * KCHUNK);
#pragma unroll
        for (int by = 0; by < 16; ++by) {
          const bool ok = c * KCHUNK + g * 16 + by < L;
          const int code = ok ? (int)(((uint32_t)sv[by >> 2] >> (8 * (by & 3))) & 0xff) : Mrow[t];
          const uint32_t e = etab[Mrow[t] - code];
          sum[t] += ok ? e : 0u;
        }
      }
    }
  }
#pragma unroll
  for (int t = 0; t < NTL; ++t) {
    sum[t] += __shfl_xor(sum[t], 16);
    sum[t] += __shfl_xor(sum[t], 32);
  }
  if (g == 0) {
#pragma unroll
    for (int t = 0; t < NTL; ++t) ssum[slot * ROWS + 16 * t + col] = sum[t];
  }
  __syncthreads();
  // F = floor(2^32 / sum), one row per thread.  The float64 quotient is correctly
  // rounded, and 2^32 / sum lies at least 1 / sum below the next integer while its
  // rounding error is at most 2^32 / sum * 2^-53, so truncating it gives the floor.
  if (tid < WGQ) {
    const int qs = tid / ROWS, rr = tid - qs * ROWS;
    uint32_t tot = 0;
#pragma unroll
    for (int k2 = 0; k2 < KSPLIT; ++k2) tot += ssum[(qs * KSPLIT + k2) * ROWS + rr];
    sF[tid] = tot ? (uint32_t)(4294967296.0 / (double)tot) : 0u;
  }
  __syncthreads();
  // softmax code tables (over the exp copies, which phase 2 has finished with): the
  // dword of distance d and bank rr + 16 c (c = 0, 1: two copies) holds in byte tt
  // min(floor(e(d) F_r / 2^24), 255) ^ 0x80 of row r = 16 tt + rr, i.e. a - 128.
  // floor(e F / 2^24) is the high word of (e 2^8) F (e < 2^24).  Each dword is
  // computed once and written to both copies.
  for (int idx = tid; idx < TAB_DW / 2; idx += 64 * ATTN_WAVES) {
    const int dd = idx >> 4, rr = idx & 15;
    const uint32_t e8 = etab[dd] << 8;
    uint32_t packed = 0;
#pragma unroll
    for (int tt = 0; tt < NQS * NTL; ++tt) {
      const uint32_t v = __umulhi(e8, sF[16 * tt + rr]);
      packed |= ((v > 255u ? 255u : v) ^ 0x80u) << (8 * tt);
    }
    tab[dd * 32 + rr] = packed;
    tab[dd * 32 + rr + 16] = packed;
  }
  __syncthreads();

  // ---------------- phase 3: A.V on MFMA
  v4i acc[NTL][NT];
#pragma unroll
  for (int t = 0; t < NTL; ++t)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[t][nt] = (v4i){0, 0, 0, 0};
  if (active && c_begin < c_end) {
    // code byte of (row, M - code) at arow[-128 code]: lanes g = 0, 1 (and 2, 3) read
    // the two bank copies of their row, so one read touches 32 distinct banks
    const uint8_t* arow[NTL];
#pragma unroll
    for (int t = 0; t < NTL; ++t)
      arow[t] = (const uint8_t*)tab + (Mrow[t] * 32 + col + 16 * (g & 1)) * 4 + (qset * NTL + t);
    const int vt_off = lane * 16;               // lane's bytes of a 16-channel x 64-key block
    constexpr int CH = 64 * DK;                 // bytes of V^T per 64-key chunk
    // softmax codes (as a - 128) of one chunk of keys for every query tile;
    // all lookups of a chunk are issued before any is packed
    auto codes_full = [&](int c, v4i* af) {
      v4i sv[NTL];
#pragma unroll
      for (int t = 0; t < NTL; ++t) sv[t] = *(const v4i*)(srd[t] + c * KCHUNK);
      // bytes 0 and 2 of a dword are loaded into the two halves of one register, bytes 1
      // and 3 into another (16-bit loads that keep the other half), so one shift-or
      // packs four codes
      us2 ev[NTL][4], od[NTL][4];
#pragma unroll
      for (int t = 0; t < NTL; ++t)
#pragma unroll
        for (int k = 0; k < 16; ++k) {
          const uint16_t v = arow[t][__mul24(-128, (int)(((uint32_t)sv[t][k >> 2] >> (8 * (k & 3))) & 0xff))];
          us2& dst = (k & 1) ? od[t][k >> 2] : ev[t][k >> 2];
          if (k & 2)
            dst.y = v;
          else
            dst.x = v;
        }
#pragma unroll
      for (int t = 0; t < NTL; ++t)
#pragma unroll
        for (int wd = 0; wd < 4; ++wd)
          af[t][wd] = (int)(__builtin_bit_cast(uint32_t, ev[t][wd]) | (__builtin_bit_cast(uint32_t, od[t][wd]) << 8));
    };
    auto codes_tail = [&](int c, v4i* af) {
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
        const v4i sv = *(const v4i*)(srd[t] + c * KCHUNK);
#pragma unroll
        for (int wd = 0; wd < 4; ++wd) {
          uint32_t packed = 0;
#pragma unroll
          for (int by = 0; by < 4; ++by) {
            const bool ok = c * KCHUNK + g * 16 + wd * 4 + by < L;
            const int code = ok ? (int)(((uint32_t)sv[wd] >> (8 * by)) & 0xff) : Mrow[t];
            const uint32_t av = arow[t][-128 * code];
            packed |= (ok ? av : 0x80u) << (8 * by);  // a = 0 for padded keys
          }
          af[t][wd] = (int)packed;
        }
      }
    };
    // V^T operands in parts of NP = 2 channel tiles, each with this lane's V sums over
    // the chunk for channels (hp NP + k) * 16 + col.  One buffer per part of a chunk:
    // a part is refilled with the next chunk's as soon as its MFMAs are issued, so a
    // whole chunk of V is in flight while the current one is multiplied (past the last
    // chunk the loads re-read it: in bounds, unused, and the loads stay unconditional).
    constexpr int NP = 2;
    constexpr int NPART = NT / NP;
    struct VPart {
      v4i v[NP];
      int s[NP];
    };
    auto load_part = [&](int c, int hp, VPart& dst) {
      const int8_t* src = VTh + (size_t)c * CH + hp * NP * 1024 + vt_off;
#pragma unroll
      for (int k = 0; k < NP; ++k) dst.v[k] = *(const v4i*)(src + k * 1024);
      const int2 sv2 = *(const int2*)(vs + ((size_t)c * 16 + col) * NT + hp * NP);
      dst.s[0] = sv2.x;
      dst.s[1] = sv2.y;
    };
    int vacc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) vacc[nt] = 0;
    v4i af[NTL];
    auto mma_part = [&](const int hp, const VPart& vp) {
#pragma unroll
      for (int k = 0; k < NP; ++k) {
#pragma unroll
        for (int t = 0; t < NTL; ++t)
          acc[t][hp * NP + k] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[t], vp.v[k], acc[t][hp * NP + k], 0, 0, 0);
        vacc[hp * NP + k] += vp.s[k];
      }
    };
    const int c_last = c_end - 1;
    VPart pb[NPART];
#pragma unroll
    for (int hp = 0; hp < NPART; ++hp) load_part(c_begin, hp, pb[hp]);
    auto mma_chunk = [&](const int c) {
      const int cn = min(c + 1, c_last);
#pragma unroll
      for (int hp = 0; hp < NPART; ++hp) {
        mma_part(hp, pb[hp]);
        load_part(cn, hp, pb[hp]);
      }
    };
    // the full chunks in a loop of their own (a shared loop body would make every chunk
    // pay the tail's per-key selects), then the chunk with the utterance's last key
    int c = c_begin;
    for (; c < c_full; ++c) {
      codes_full(c, af);
      mma_chunk(c);
    }
    if (c < c_end) {
      codes_tail(c, af);
      mma_chunk(c);
    }
    // exact correction for the -128 offset: + 128 * sum of V over the same keys
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int t = 0; t < NTL; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[t][nt][i] += 128 * vacc[nt];
  }

  // ---------------- combine the key splits, requantize, store
  const int64_t half_o = (int64_t)1 << (a.shift_o - 1);
  auto requant_o = [&](int32_t v) -> int {
    const int64_t r = ((int64_t)v * a.m_o + half_o) >> a.shift_o;
    return r < -127 ? -127 : (r > 127 ? 127 : (int)r);
  };
  if (KSPLIT == 1) {
#pragma unroll
    for (int t = 0; t < NTL; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int qi = q0 + 16 * t + 4 * g + i;
        if (qi >= T) continue;
        int8_t* out = a.ctx + ((size_t)b * T + qi) * a.d + (size_t)h * DK + col;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) out[nt * 16] = (int8_t)(qi < L ? requant_o(acc[t][nt][i]) : 0);
      }
  } else {
    // partial sums of one query set: [ROWS][RSTRIDE] int32; the padding puts rows 4
    // apart into different banks.  The first key split stores, the others add with
    // LDS atomics (exact, order-free).
    int32_t* rq = red + (size_t)qset * ROWS * RSTRIDE;
    __syncthreads();  // every wave is done with the score rows
    if (kpart == 0) {
#pragma unroll
      for (int t = 0; t < NTL; ++t)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int i = 0; i < 4; ++i) rq[(16 * t + 4 * g + i) * RSTRIDE + nt * 16 + col] = acc[t][nt][i];
    }
    __syncthreads();
    if (kpart != 0 && active) {
#pragma unroll
      for (int t = 0; t < NTL; ++t)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
          for (int i = 0; i < 4; ++i) atomicAdd(&rq[(16 * t + 4 * g + i) * RSTRIDE + nt * 16 + col], acc[t][nt][i]);
    }
    __syncthreads();
    // the KSPLIT waves of the set share its rows: items of 4 channels, row-major
    constexpr int IPR = DK / 4;  // items per row
    for (int it = kpart * 64 + lane; it < ROWS * IPR; it += 64 * KSPLIT) {
      const int rr = it / IPR;
      const int ch = (it % IPR) * 4;
      const int qi = q0 + rr;
      if (qi >= T) continue;
      const v4i v = *(const v4i*)(rq + rr * RSTRIDE + ch);
      uint32_t packed = 0;
      if (qi < L) {
#pragma unroll
        for (int e = 0; e < 4; ++e) packed |= ((uint32_t)requant_o(v[e]) & 0xffu) << (8 * e);
      }
      *(uint32_t*)(a.ctx + ((size_t)b * T + qi) * a.d + (size_t)h * DK + ch) = packed;
    }
  }
}

// The core kernel: one workgroup shape (NTL2 == 0), or two shapes in one grid, the
// first one's blocks ahead of the second one's, so that the second shape fills what
// the first leaves of the last round (workgroups start in block order).
template <int DK, int KS1, int NTL1, int KS2, int NTL2, bool WIDE>
__global__ __launch_bounds__(64 * ATTN_WAVES) void relpos_attn_core(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  if constexpr (NTL2 == 0) {
    attn_block<DK, KS1, NTL1, WIDE>(a, smem, blockIdx.x, a.nqb, 0);
  } else {
    if ((int)blockIdx.x < a.seg2_block)
      attn_block<DK, KS1, NTL1, WIDE>(a, smem, blockIdx.x, a.nqb, 0);
    else
      attn_block<DK, KS2, NTL2, WIDE>(a, smem, blockIdx.x - a.seg2_block, a.nqb2, a.seg2_q0);
  }
}

// ---------------------------------------------------------------------------
// Copies a workspace tensor back to the documented [B][T][d] / [2T-1][d] layouts.
struct GatherArgs {
  const int8_t* src;
  int8_t* dst;
  int which, B, T, T_al, H, DK, d, p_rows, p_base;
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
    v = a.src[(size_t)h * a.p_rows * a.DK + frag_index(a.p_base + (int)m, kk, a.DK)];
  } else if (a.which >= 4) {  // the context or the LayerNorm output, [B][T][d]
    v = a.src[idx];
  } else {
    const long b = m / a.T, t = m % a.T;
    const size_t base = ((size_t)b * a.H + h) * a.T_al * a.DK;
    v = a.src[base + (a.which == 2 ? vt_index((int)t, kk, a.DK) : frag_index((int)t, kk, a.DK))];
  }
  a.dst[idx] = v;
}

// ---------------------------------------------------------------------------
size_t attn_lds_bytes(int DK, int ksplit, int ntl, int T_al) {
  const int rows = 16 * ntl, nqs = ATTN_WAVES / ksplit;
  const int wgq = rows * nqs;
  const size_t s_bytes = (size_t)wgq * (T_al + SCORE_PAD);
  const size_t red = ksplit > 1 ? (size_t)nqs * rows * (DK + 4) * 4 : 0;
  const size_t big = ((s_bytes > red ? s_bytes : red) + 15) & ~(size_t)15;
  return big + (size_t)TAB_DW * 4 + 256 * 4 + 2 * (size_t)rows * ATTN_WAVES * 4 + (size_t)wgq * 4;
}

// Workgroup shapes the kernel is built for: (key splits, 16-query tiles per wave).
static const AttnCfg kAttnCfgs[] = {{4, 2}, {8, 2}, {8, 3}};
// One 16-query tile per wave: the smallest score rows, for utterances whose rows do not
// fit any shape above (every K, P and V fragment then feeds a single MFMA)
static const AttnCfg kAttnLong = {8, 1};
constexpr size_t kLdsBudget = 160 * 1024;
constexpr int kNumCUs = 256;

static int wgq_of(const AttnCfg& c) { return 16 * c.ntl * (ATTN_WAVES / c.ksplit); }
static bool fits(const AttnCfg& c, int DK, int T_al) { return attn_lds_bytes(DK, c.ksplit, c.ntl, T_al) <= kLdsBudget; }

// Time of one workgroup, modelled per key of a wave's share as 125 cycles for the K, P
// and V streams (the same for any number of query tiles) plus 29 per 16-query tile
// (score post-processing, exp sums, code lookups, combine), as measured on the
// long-form workload.
static double wg_cost(const AttnCfg& c, int T) { return ((double)T / c.ksplit) * (125.0 + 29.0 * c.ntl); }

// Finishing time of groups of workgroups (count[g] of cost[g] each) started in order on
// the CUs, one workgroup per CU (eight waves of more than 128 VGPRs), each CU taking the
// next workgroup when it is free.  CUs are kept in buckets of equal free time.
static double makespan(const long* count, const double* cost, int ng) {
  struct Bucket {
    double t;
    long n;
  };
  std::vector<Bucket> b{{0.0, (long)kNumCUs}};  // ascending t
  auto insert = [&](Bucket x) {
    size_t i = 0;
    while (i < b.size() && b[i].t < x.t) ++i;
    if (i < b.size() && b[i].t == x.t)
      b[i].n += x.n;
    else
      b.insert(b.begin() + i, x);
  };
  for (int g = 0; g < ng; ++g) {
    long left = count[g];
    while (left > 0) {
      Bucket e = b.front();
      b.erase(b.begin());
      const long take = left < e.n ? left : e.n;
      left -= take;
      if (e.n > take) b.insert(b.begin(), Bucket{e.t, e.n - take});
      insert(Bucket{e.t + cost[g], take});
    }
  }
  return b.back().t;
}

// Plan of one launch: a single workgroup shape, or 48-query workgroups for whole
// rounds followed by 32-query ones for the remaining queries, whichever finishes
// first by the model above.  c1.ksplit == 0 if no shape fits in LDS.
AttnPlan attn_plan(int DK, int T_al, long bh_count, int T) {
  AttnPlan best{};
  double best_t = 0.0;
  auto consider = [&](const AttnPlan& p) {
    const long cnt[2] = {bh_count * p.nqb1, bh_count * p.nqb2};
    const double cst[2] = {wg_cost(p.c1, T), p.c2.ksplit ? wg_cost(p.c2, T) : 0.0};
    const double t = makespan(cnt, cst, p.c2.ksplit ? 2 : 1);
    if (best.c1.ksplit == 0 || t < best_t) {
      best = p;
      best_t = t;
    }
  };
  for (const AttnCfg& c : kAttnCfgs)
    if (fits(c, DK, T_al)) consider(AttnPlan{c, (T + wgq_of(c) - 1) / wgq_of(c), AttnCfg{0, 0}, 0});
  if (best.c1.ksplit == 0 && fits(kAttnLong, DK, T_al))
    return AttnPlan{kAttnLong, (T + wgq_of(kAttnLong) - 1) / wgq_of(kAttnLong), AttnCfg{0, 0}, 0};
  const AttnCfg c1{8, 3}, c2{8, 2};
  if (fits(c1, DK, T_al) && fits(c2, DK, T_al)) {
    const int per_round = (int)(kNumCUs / bh_count);  // blocks per (utterance, head) in one round
    const int n1_all = (T + wgq_of(c1) - 1) / wgq_of(c1);
    for (int n1 = per_round; n1 > 0 && n1 < n1_all; n1 += per_round) {
      const int rest = T - n1 * wgq_of(c1);
      consider(AttnPlan{c1, n1, c2, (rest + wgq_of(c2) - 1) / wgq_of(c2)});
    }
  }
  return best;
}

// Raises a kernel's dynamic-LDS ceiling to the whole budget, once per device (per
// launch the call would cost host time on every run).
static hipError_t allow_full_lds(const void* kernel) {
  static std::mutex mu;
  static std::vector<std::pair<const void*, int>> done;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  for (const auto& d : done)
    if (d.first == kernel && d.second == dev) return hipSuccess;
  e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsBudget);
  if (e == hipSuccess) done.emplace_back(kernel, dev);
  return e;
}

template <int DK, int KS1, int NTL1, int KS2, int NTL2, bool WIDE>
static hipError_t launch_attn_plan(const AttnArgs& args, const AttnPlan& p, int B, int H, int T_al, hipStream_t st,
                                   const LaunchEv& ev) {
  size_t shmem = attn_lds_bytes(DK, KS1, NTL1, T_al);
  if (NTL2) {
    const size_t s2 = attn_lds_bytes(DK, KS2, NTL2, T_al);
    shmem = s2 > shmem ? s2 : shmem;
  }
  hipError_t e = allow_full_lds((const void*)relpos_attn_core<DK, KS1, NTL1, KS2, NTL2, WIDE>);
  if (e != hipSuccess) return e;
  AttnArgs a2 = args;
  a2.nqb = p.nqb1;
  a2.xcd_group = (B * H) % 8 == 0;
  a2.seg2_block = p.nqb1 * B * H;
  a2.seg2_q0 = p.nqb1 * wgq_of(p.c1);
  a2.nqb2 = p.nqb2;
  dim3 grid((p.nqb1 + p.nqb2) * B * H);
  return launch_kernel(relpos_attn_core<DK, KS1, NTL1, KS2, NTL2, WIDE>, grid, dim3(64 * ATTN_WAVES),
                       (uint32_t)shmem, st, ev, a2);
}

template <int DK, bool WIDE>
static hipError_t launch_attn_dk(const AttnArgs& a, const RunShape& rs, hipStream_t st, const LaunchEv& ev) {
  const AttnPlan p = attn_plan(DK, rs.T_al, (long)rs.B * rs.H, rs.T);
  auto is = [](const AttnCfg& c, int ks, int ntl) { return c.ksplit == ks && c.ntl == ntl; };
  if (p.c2.ksplit == 0) {
    if (is(p.c1, 4, 2)) return launch_attn_plan<DK, 4, 2, 0, 0, WIDE>(a, p, rs.B, rs.H, rs.T_al, st, ev);
    if (is(p.c1, 8, 2)) return launch_attn_plan<DK, 8, 2, 0, 0, WIDE>(a, p, rs.B, rs.H, rs.T_al, st, ev);
    if (is(p.c1, 8, 3)) return launch_attn_plan<DK, 8, 3, 0, 0, WIDE>(a, p, rs.B, rs.H, rs.T_al, st, ev);
    if (is(p.c1, 8, 1)) return launch_attn_plan<DK, 8, 1, 0, 0, WIDE>(a, p, rs.B, rs.H, rs.T_al, st, ev);
  } else if (is(p.c1, 8, 3) && is(p.c2, 8, 2)) {
    return launch_attn_plan<DK, 8, 3, 8, 2, WIDE>(a, p, rs.B, rs.H, rs.T_al, st, ev);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_attention(const RunShape& rs, const Weights& w, const Scalars& sc, const Workspace& ws,
                            const Lengths& lens, hipStream_t st, const LaunchEv& ev) {
  AttnArgs a{};
  a.q = ws.q;
  a.k = ws.k;
  a.vt = ws.vt;
  a.p = ws.p;
  a.u = w.u;
  a.v = w.v;
  a.vsum = ws.vsum;
  a.ctx = ws.ctx;
  a.lens = lens;
  a.T = rs.T;
  a.T_al = rs.T_al;
  a.H = rs.H;
  a.d = rs.d;
  a.p_rows = rs.p_rows;
  a.p_base = rs.p_base;
  a.mc24 = sc.fs_mc24;
  a.mp24 = sc.fs_mp24;
  a.bias32 = sc.fs_bias32;
  a.post_shift = sc.fs_post_shift;
  a.mcd = sc.fs_mcd;
  a.mpd = sc.fs_mpd;
  a.m_o = sc.m_o;
  a.shift_o = sc.shift_o;
  a.q_ln2 = sc.q_ln2;
  a.q_b = sc.q_b;
  a.q_c = sc.q_c;
  if (rs.DK == 128) return sc.fs_wide ? launch_attn_dk<128, true>(a, rs, st, ev) : launch_attn_dk<128, false>(a, rs, st, ev);
  if (rs.DK == 64) return sc.fs_wide ? launch_attn_dk<64, true>(a, rs, st, ev) : launch_attn_dk<64, false>(a, rs, st, ev);
  return hipErrorInvalidValue;
}

hipError_t launch_gather_intermediate(const RunShape& rs, const Workspace& ws, int which, int8_t* dst,
                                      hipStream_t st) {
  GatherArgs a{};
  a.src = which == 0 ? ws.q : which == 1 ? ws.k : which == 2 ? ws.vt : which == 3 ? ws.p : which == 4 ? ws.ctx : ws.xln;
  a.dst = dst;
  a.which = which;
  a.B = rs.B;
  a.T = rs.T;
  a.T_al = rs.T_al;
  a.H = rs.H;
  a.DK = rs.DK;
  a.d = rs.d;
  a.p_rows = rs.p_rows;
  a.p_base = rs.p_base;
  const long rows = which == 3 ? (long)(2 * rs.T - 1) : (long)rs.B * rs.T;
  const long total = rows * rs.d;
  hipLaunchKernelGGL(gather_intermediate, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace ipk
