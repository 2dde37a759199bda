// Relative-position attention core of the integer MHSA block (Sec. 3.1).
//
// Work split: a workgroup of ATTN_WAVES waves owns (utterance b, head h, WGQ
// consecutive queries).  Its int8 score rows stay in LDS (never in HBM), laid out in
// 16-key blocks: block j/16 holds the WGQ rows' 16 scores of those keys, 16 bytes per
// row, so the row of query r and key j sits at byte (j/16) WGQ 16 + 16 r + j % 16.
// The host picks the workgroup shape per launch from the LDS the rows need and the
// rounds of workgroups over the CUs.
//
// Phase 1 (scores), per 16-key step, with v_mfma_i32_16x16x64_i8 (queries on MFMA
// rows).  KSPLIT waves share a query set of NTL 16-query tiles (every K and P fragment
// a wave loads feeds NTL MFMAs) and split its keys:
//  * content   c = Q K^T, accumulator seeded with the rank-1 term u.K_j
//  * position  G = Q P_win^T, seeded with v.P_r, for the 16 table rows that start at
//              relative position j0-i0+T-1 ("hi" window).  The rows just before it
//              ("lo") are the previous step's hi window, and tile t reuses the P
//              fragment tile 0 loaded t steps earlier, so each step loads one new P
//              fragment and runs one new position MFMA pair per tile.
//  * Phi       p_ij = G_i(j-i+T-1) is a rotation by the row index inside each 16-lane
//              row group: every source lane picks the window its value belongs to and
//              ds_bpermute moves it to the lane of its key.
//  * Eq. 11    s = clamp8(RS(m_c c + m_p p, 1, n)), exact: in 32-bit integers when
//              the descriptor bounds |m_c c + m_p p| below 2^31, otherwise in 64-bit
//              integers.  Scores are kept as biased codes s + 128 in [1, 255].
//  * each score byte is stored straight into its row's block (one address add per
//    step: the tile and row offsets are instruction immediates).
// Phase 2 (row sums): row max over a row's 16 key lanes (DPP) and over the key splits
// (LDS); every lane then reads 16 scores of one row (16 bytes), forms the four
// distances d = M - s of each dword with one subtraction (every s <= M, so no byte
// borrows), and looks up the I-BERT integer exp of each d in a table with one copy per
// LDS bank; the address of one lookup is a single v_dot4 (base + 128 d).
// Conversion: F = floor(2^32 / sum) per row (integer long division), per-row tables of
// the softmax code a - 128 = min(floor(e F / 2^24), 255) - 128, and every score byte of
// the workgroup replaced in place by its code.  Keys past the utterance take distance
// 255 in both passes: its exp is 0 (left out of the sum) and its code -128 (a = 0).
// Phase 3 (A.V): the waves split the d_k channels (two 16-channel MFMA tiles each) and
// the keys; with the V^T fragment as the A operand and 16 queries' codes (16 bytes of
// one row, read straight from its block) as B, each output lane holds four consecutive
// channels of one query.  The exact correction 128 sum_j V_j for the -128 offset is
// summed from the V fragments themselves (v_dot4 against ones).  The key parts' int32
// partial contexts are added in LDS (exact, order-free) and requantized with
// (m_o, shift_o) in 64-bit integers.
// No floating-point instruction runs in the kernel.
#include <mutex>
#include <type_traits>
#include <utility>
#include <vector>

#include "ipk_internal.h"

namespace ipk {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) uint8_t lds8;
typedef __attribute__((address_space(3))) uint32_t lds32;
typedef __attribute__((address_space(3))) int32_t ldsi32;
typedef __attribute__((address_space(3))) v4i ldsv4;

struct AttnArgs {
  const int8_t *q, *k, *vt, *p;
  const int8_t *u, *v;   // [H][d_k]
  const uint32_t* etab;  // [256]: integer exp of every distance d (0 at d = 255)
  int8_t* ctx;
  Lengths lens;
  int T, T_al, H, d, p_rows, p_base;
  int nqb;        // query blocks per (utterance, head) of the first segment
  DivU dv_nqb, dv_nqb2, dv_H;  // the block decomposition's divisors
  int xcd_group;  // keep each (utterance, head) on one XCD
  // second segment of a two-shape grid: blocks from seg2_block on cover the queries
  // from seg2_q0 on, nqb2 blocks per (utterance, head), with the second shape
  int seg2_block, seg2_q0, nqb2;
  // fused score, 32-bit path: t = mc24 c + mp24 p + bias32, code in bits 16..23
  int32_t mc24, mp24, bias32;
  // fused score, 64-bit path: t = m_c c + m_p p + bias64, code = t >> shift_s
  int32_t m_c, m_p, shift_s;
  int64_t bias64;
  int32_t m_o, shift_o;
};

// Maximum over the 16 lanes of each row (DPP quad_perm [1,0,3,2], quad_perm [2,3,0,1],
// row_half_mirror, row_mirror): every lane ends with its row's maximum, and no LDS
// round trip is spent (a lane shuffle would be a ds_bpermute each step).
__device__ __forceinline__ int row16_max(int v) {
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false));
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false));
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false));
  v = max(v, __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false));
  return v;
}

// Sum of lanes l, l ^ 16, l ^ 32 and l ^ 48 (the same column of the four 16-lane rows)
// in every lane: v_permlane16_swap pairs rows 0/1 and 2/3, v_permlane32_swap the two
// halves.  Integer adds, so the order does not matter.
__device__ __forceinline__ uint32_t col4_sum(uint32_t v) {
  const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = r[0] + r[1];
  const auto h = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return h[0] + h[1];
}

constexpr int TAB_DW = 256 * 32;  // dwords of the [d][32 banks] lookup-table region
constexpr int ATTN_WAVES = 8;     // waves per workgroup (two per SIMD)

// Share (out of 256) of a SIMD's work that its older wave takes in phase 1 and in the
// later phases: the arbiter favours the older wave of a SIMD (the lower index), so with
// equal shares the younger one finishes long after it.
constexpr int P1_OLDER = 166;  // phase 1 (16-key steps)
constexpr int P2_OLDER = 162;  // phase 2 and the conversion (64-key chunks)
constexpr int P3_OLDER = 156;  // phase 3 (64-key chunks)

template <int S>
using Phase = std::integral_constant<int, S>;

// Low 32 bits of a * b + c for 24-bit signed a, b (v_mad_i32_i24); the addition
// wraps modulo 2^32.
__device__ __forceinline__ int mad_i24(int a, int b, int c) {
  return (int)((uint32_t)__mul24(a, b) + (uint32_t)c);
}

// floor(2^32 / D) for 2^8 <= D < 2^32 by binary long division in 32-bit integers:
// floor((2^32 - 1) / D), plus one when D divides 2^32 (a power of two).  Quotient bits
// 31..24 are zero for D >= 2^8, which leaves the remainder 2^8 - 1 after them; each
// further step doubles the remainder and adds the next dividend bit (a one): it stays
// below D after the conditional subtraction, so the wrap-around of 2 r + 1 past 2^32
// cancels in the subtraction.
__device__ __forceinline__ uint32_t floor_2p32_div(uint32_t D) {
  const uint32_t half = D >> 1;  // 2 r + 1 >= D  <=>  r >= floor(D / 2)
  uint32_t r = 255u, q = 0;
#pragma unroll
  for (int i = 23; i >= 0; --i) {
    const bool c = r >= half;
    r = (r << 1) + 1u - (c ? D : 0u);
    q = (q << 1) | (c ? 1u : 0u);
  }
  return q + ((D & (D - 1)) == 0 ? 1u : 0u);
}

// LDS carve-up of one workgroup shape (the host computes the same sizes).
struct AttnLds {
  uint32_t tab, etab, smax, ssum, sF, total;
};
__host__ __device__ constexpr AttnLds attn_lds(int wgq, int rows, int T_al) {
  const uint32_t s = (uint32_t)wgq * (uint32_t)T_al;  // score blocks (a multiple of 16)
  const uint32_t tab = s;
  const uint32_t etab = tab + TAB_DW * 4;
  const uint32_t smax = etab + 256 * 4;
  const uint32_t ssum = smax + (uint32_t)rows * ATTN_WAVES * 4;
  const uint32_t sF = ssum + (uint32_t)rows * ATTN_WAVES * 4;
  return AttnLds{tab, etab, smax, ssum, sF, sF + (uint32_t)wgq * 4};
}

// Work units [*b, *e) of part `part` of 2 hk parts out of n: the parts come in pairs that
// share a SIMD (part p and p + hk, the first one older); each pair gets n / hk of the
// units, of which the older wave takes older / 256 (rounded).
__device__ __forceinline__ void split_pairs(int n, int older, int hk, int part, int* b, int* e) {
  const int pair = part % hk, younger = part / hk;
  const int ps = n * pair / hk, pe = n * (pair + 1) / hk;
  const int mid = ps + ((pe - ps) * older + 128) / 256;
  *b = younger ? mid : ps;
  *e = younger ? pe : mid;
}

// One workgroup of the core: block `lin` of a segment of nqb query blocks per
// (utterance, head) that starts at query q_base.
template <int DK, int KSPLIT, int NTL, bool WIDE>
__device__ __forceinline__ void attn_block(const AttnArgs& a, unsigned char* smem, const int lin, const DivU& dnqb,
                                           const int q_base) {
  const int nqb = (int)dnqb.d;
  constexpr int NQS = ATTN_WAVES / KSPLIT;  // query sets per workgroup
  constexpr int ROWS = 16 * NTL;            // queries per set: NTL 16-query MFMA tiles
  constexpr int WGQ = ROWS * NQS;           // queries per workgroup
  constexpr int NTILES = WGQ / 16;          // 16-query tiles per workgroup
  constexpr int NKS = DK / 64;              // MFMA K-steps over d_k
  constexpr int BLK = WGQ * 16;             // bytes per 16-key block of score rows
  constexpr int AV_NT = DK / 64;            // 16-channel tiles per wave in phase 3
  constexpr int NCG = DK / (16 * AV_NT);    // channel groups of phase 3 (four)
  constexpr int KH = ATTN_WAVES / NCG;      // key parts of phase 3 (two)
  static_assert(NTILES <= 4, "the code tables hold four 16-row tiles");
  static_assert(KH == 2, "phase-3 wave grid");

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index: uniform, kept in SGPRs
  const int col = lane & 15, g = lane >> 4;
  // Waves w and w + 4 share SIMD w % 4.  In phase 1 the two waves of a SIMD take the
  // same query set and split its keys unevenly (the older one the larger share).
  constexpr int HK = KSPLIT > 1 ? KSPLIT / 2 : 1;  // key parts per age class
  const int simd = w & 3, younger = w >> 2;
  const int qset = KSPLIT > 1 ? simd / HK : w;
  const int kpart = KSPLIT > 1 ? younger * HK + simd % HK : 0;
  const int slot = qset * KSPLIT + kpart;  // this wave's row-max and row-sum slot
  auto split = [&](const int n, const int older, int* b, int* e) {
    if (KSPLIT == 1) {
      *b = 0;
      *e = n;
    } else {
      split_pairs(n, older, HK, kpart, b, e);
    }
  };
  // Workgroups go round-robin to the 8 XCDs (id % 8); when the (utterance, head)
  // pairs divide evenly, every workgroup of one pair is placed on the same XCD so that
  // its K, P and V stay in that XCD's L2.
  int qb, bhi;
  if (a.xcd_group) {
    const int x = lin & 7, k = lin >> 3, s = (int)div_u(k, dnqb);
    qb = k - s * nqb;
    bhi = x + 8 * s;
  } else {
    bhi = (int)div_u(lin, dnqb);
    qb = lin - bhi * nqb;
  }
  const int b = (int)div_u(bhi, a.dv_H), h = bhi - b * a.H;
  const int wg_q0 = q_base + qb * WGQ;
  const int q0 = wg_q0 + ROWS * qset;  // first query of this wave's set
  const int L = a.lens.len[b];
  const int T = a.T, T_al = a.T_al;
  if (wg_q0 >= L) {
    // no valid query in this workgroup (a ragged batch): its context rows are zeros,
    // and nothing else of it is needed
    const int tid0 = threadIdx.x;
    constexpr int PIECES = DK / 16;  // 16-byte pieces of one row's head slice
    for (int idx = tid0; idx < WGQ * PIECES; idx += 64 * ATTN_WAVES) {
      const int qi = wg_q0 + idx / PIECES;
      if (qi < T)
        *(v4i*)(a.ctx + ((size_t)b * T + qi) * a.d + (size_t)h * DK + (idx % PIECES) * 16) = (v4i){0, 0, 0, 0};
    }
    return;
  }
  const int nkc = (L + KCHUNK - 1) / KCHUNK;
  int c_begin, c_end;
  split(nkc, P2_OLDER, &c_begin, &c_end);
  // chunks below c_full hold only valid keys; c_full < c_end only when this wave's
  // range holds the chunk with the utterance's last key
  const int c_full = max(c_begin, min(c_end, L / KCHUNK));
  const bool active = q0 < L;

  constexpr AttnLds lay0 = attn_lds(WGQ, ROWS, 0);
  const uint32_t base = (uint32_t)(uintptr_t)(lds8*)smem;
  const uint32_t s_bytes = (uint32_t)WGQ * (uint32_t)T_al;
  const uint32_t TAB = base + s_bytes;                  // [d][32 banks] dwords
  const uint32_t ETAB = TAB + (lay0.etab - lay0.tab);   // the 256 exp values, once
  lds32* tab = (lds32*)(uintptr_t)TAB;
  lds32* etab = (lds32*)(uintptr_t)ETAB;
  ldsi32* smax = (ldsi32*)(uintptr_t)(TAB + (lay0.smax - lay0.tab));
  lds32* ssum = (lds32*)(uintptr_t)(TAB + (lay0.ssum - lay0.tab));
  lds32* sF = (lds32*)(uintptr_t)(TAB + (lay0.sF - lay0.tab));

  const size_t bh = (size_t)b * a.H + h;
  const int8_t* Qh = a.q + bh * T_al * DK;
  const int8_t* Kh = a.k + bh * T_al * DK;
  const int8_t* VTh = a.vt + bh * DK * T_al;
  const int8_t* Ph = a.p + (size_t)h * a.p_rows * DK;
  // this lane's 16 bytes of a 1 KB operand fragment (stored in lane order)
  const int frag_off = lane * 16;

  constexpr int LOCODE = WIDE ? 1 : (1 << 16);  // code of s = -127 (biased s + 128)
  constexpr int HICODE = WIDE ? 255 : ((255 << 16) | 0xFFFF);

  // the integer exp of this thread's distance
  const uint32_t e_mine = a.etab[tid & 255];
  // the integer exp of every distance d in [0, 255): once, and in 32 per-bank copies
  // (copy (d + c) % 32 of pass c is written by the thread of d, which keeps the writes
  // free of bank conflicts).  Phase 1 does not touch the table region, so these stores
  // go out while its first operands load.
  {
    const int dd = tid & 255;
    if (tid < 256) etab[dd] = e_mine;
    for (int c = (tid >> 8) * 16; c < 32; c += 16 * (64 * ATTN_WAVES / 256)) {
#pragma unroll
      for (int k = 0; k < 16; ++k) tab[dd * 32 + ((c + k + dd) & 31)] = e_mine;
    }
  }

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
    // a lane's score of query row 4g + i of tile t and key j0 + col is byte col of that
    // row's 16 bytes in block j0 / 16: the row and tile offsets are immediates
    const uint32_t sdst0 = base + (uint32_t)((ROWS * qset + 4 * g) * 16 + col);

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
    //  bv[u]:    the seed v.P_r of that window (all four rows)
    //  kr[u]:    K fragment of the step with phase u (current, next)
    //  gr[u][t]: position MFMA results (hi windows) of the step with phase u; a
    //            step's lo windows are the previous step's hi windows
    constexpr int RING = NTL > 1 ? NTL : 2;
    v4i pr[RING][NKS], kr[RING][NKS], gr[RING][NTL], bv[RING];
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
      for (int t = 0; t < NTL; ++t) bv[(RING - t) % RING] = rank1(vf, pr[(RING - t) % RING]);
      const v4i bvlast = rank1(vf, plast);
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
        const int u = (RING - t - 1) % RING;  // slot of tile (t + 1)'s hi window
        v4i gacc = t + 1 < NTL ? bv[u] : bvlast;
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
      // seeds: u.K_j of this step's keys (shared by the tiles) and v.P_r of this step's
      // new window (kept with it in the ring)
      const v4i uk = rank1(uf, kr[S]);
      bv[S] = rank1(vf, pr[S]);
      v4i cs[NTL];
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
        cs[t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(qf[t][0], kr[S][0], uk, 0, 0, 0);
        gr[S][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(qf[t][0], pr[(S + RING - t) % RING][0],
                                                         bv[(S + RING - t) % RING], 0, 0, 0);
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
      const bool key_ok = j0 + col < L;
      lds8* sp = (lds8*)(uintptr_t)(sdst0 + (uint32_t)(j0 >> 4) * BLK);
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int sel = take_hi[i] ? gr[S][t][i] : gr[SP][t][i];
          const int pt = __builtin_amdgcn_ds_bpermute(src_addr[i], sel);
          int v;
          if (WIDE) {
            // exact in 64 bits: |m c| + |m p| < 2^47
            const int64_t tt = (int64_t)a.m_c * cs[t][i] + (int64_t)a.m_p * pt + a.bias64;
            const int64_t q = tt >> a.shift_s;
            v = q < 1 ? 1 : (q > 255 ? 255 : (int)q);
          } else {
            // cs holds c0 + u.K_j: the addend is the rounding and code bias alone
            int x = mad_i24(a.mp24, pt, a.bias32);
            asm("" : "+v"(x));  // opaque to the optimizer (keeps the multiply-adds apart), not a scheduling barrier
            v = mad_i24(a.mc24, cs[t][i], x);
            v = min(max(v, LOCODE), HICODE);
          }
          if (masked && !key_ok) v = LOCODE;
          mx[t][i] = max(mx[t][i], v);
          // the code is bits 0..7 (64-bit path) or 16..23 (32-bit path) of v
          sp[(16 * t + i) * 16] = (uint8_t)(WIDE ? v : (v >> 16));
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
    // the rest: fewer than RING steps below j_full, then at most one masked step (j_stop
    // is at most L rounded up to 16, and j_full at least L rounded down), so at most
    // RING steps in straight-line code whose ring phases stay static (a loop over them
    // would move the rings between registers on every pass)
    if (j0 < j_stop) step(Phase<0>{}, j0 + 16 > j_full);
    if (j0 < j_stop) step(Phase<1 % RING>{}, j0 + 16 > j_full);
    if constexpr (RING > 2) {
      if (j0 < j_stop) step(Phase<2 % RING>{}, j0 + 16 > j_full);
    }
  }
  // row max over the 16 key lanes of each row group
#pragma unroll
  for (int t = 0; t < NTL; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) mx[t][i] = row16_max(mx[t][i]);
  if (col == 0) {
#pragma unroll
    for (int t = 0; t < NTL; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) smax[slot * ROWS + 16 * t + 4 * g + i] = WIDE ? mx[t][i] : (mx[t][i] >> 16);
  }
  __syncthreads();

  // phase 2 and the conversion: lane (g, col) works on row 16 t + col of its set and
  // keys 16 g .. 16 g + 15 of a 64-key chunk, 16 bytes at
  // base + (4 c + g) BLK + (ROWS qset + 16 t + col) 16
  uint32_t Mrep[NTL];
#pragma unroll
  for (int t = 0; t < NTL; ++t) {
    int m = 1;
#pragma unroll
    for (int k2 = 0; k2 < KSPLIT; ++k2) m = max(m, smax[(qset * KSPLIT + k2) * ROWS + 16 * t + col]);
    Mrep[t] = (uint32_t)m * 0x01010101u;
  }
  const uint32_t rd0 = base + (uint32_t)(g * BLK + (ROWS * qset + col) * 16);
  // Distances of four keys of the chunk that holds the utterance's last key: keys at or
  // past L get distance 255, whose integer exp is 0 and whose softmax code is -128
  // (a = 0).  A byte past L may exceed M, but its borrow only reaches later keys.
  auto tail_dist = [&](uint32_t dw, int c, int wd) {
    const int nv = L - (c * KCHUNK + g * 16 + 4 * wd);  // valid keys from this dword's first
    return nv >= 4 ? dw : (nv <= 0 ? 0xffffffffu : dw | (0xffffffffu << (8 * nv)));
  };
  auto chunk_ptr = [&](int c, int t) { return (ldsv4*)(uintptr_t)(rd0 + (uint32_t)c * (4 * BLK) + t * 256); };

  // ---------------- phase 2: row sums of the integer exp
  // lane l reads copy l % 32 of the exp table: e(d) at TAB + 4 (l % 32) + 128 d
  uint32_t sum[NTL];
#pragma unroll
  for (int t = 0; t < NTL; ++t) sum[t] = 0u;
  if (active) {
    const uint32_t ebase = TAB + 4u * (uint32_t)(lane & 31);
    auto e_at = [&](uint32_t dw, int k) {
      return *(const lds32*)(uintptr_t)__builtin_amdgcn_udot4(dw, 128u << (8 * k), ebase, false);
    };
    // the next chunk's scores are read while the current chunk's lookups run
    v4i svn[NTL];
    if (c_begin < c_full) {
#pragma unroll
      for (int t = 0; t < NTL; ++t) svn[t] = *chunk_ptr(c_begin, t);
    }
    for (int c = c_begin; c < c_full; ++c) {
      v4i sv[NTL];
      const int cn = min(c + 1, c_full - 1);
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
        sv[t] = svn[t];
        svn[t] = *chunk_ptr(cn, t);
      }
      // all lookups of the chunk are issued before any is summed
      uint32_t ev[NTL][16];
#pragma unroll
      for (int t = 0; t < NTL; ++t)
#pragma unroll
        for (int wd = 0; wd < 4; ++wd) {
          const uint32_t dw = Mrep[t] - (uint32_t)sv[t][wd];  // four distances M - s, no borrows
#pragma unroll
          for (int k = 0; k < 4; ++k) ev[t][4 * wd + k] = e_at(dw, k);
        }
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
        const v4i sv = *chunk_ptr(c, t);
        uint32_t acc_e = 0;
#pragma unroll
        for (int wd = 0; wd < 4; ++wd) {
          const uint32_t dw = tail_dist(Mrep[t] - (uint32_t)sv[wd], c, wd);
#pragma unroll
          for (int k = 0; k < 4; ++k) acc_e += e_at(dw, k);
        }
        sum[t] += acc_e;
      }
    }
  }
#pragma unroll
  for (int t = 0; t < NTL; ++t) sum[t] = col4_sum(sum[t]);
  if (g == 0) {
#pragma unroll
    for (int t = 0; t < NTL; ++t) ssum[slot * ROWS + 16 * t + col] = sum[t];
  }
  __syncthreads();
  // F = floor(2^32 / sum), one row per thread; sum >= e(0) >= 2^8 on every row that has
  // a valid key (rows without one, which are never stored, take F = 0)
  if (tid < WGQ) {
    const int qs = tid / ROWS, rr = tid - qs * ROWS;
    uint32_t tot = 0;
#pragma unroll
    for (int k2 = 0; k2 < KSPLIT; ++k2) tot += ssum[(qs * KSPLIT + k2) * ROWS + rr];
    sF[tid] = tot >= 256 ? floor_2p32_div(tot) : 0u;
  }
  __syncthreads();
  // softmax code tables (over the exp copies, which phase 2 has finished with): the
  // dword of distance d and bank rr + 16 c (c = 0, 1: two copies) holds in byte tt
  // min(floor(e(d) F_r / 2^24), 255) ^ 0x80 of row r = 16 tt + rr, i.e. a - 128.
  // e < 2^24 and F <= 2^24: floor(e F / 2^24) is bits 24..55 of the 48-bit product of
  // the 24-bit multiplies (F = 2^24, when the sum is 2^8, gives e itself).  Each dword
  // is computed once and written to both copies.  The thread's rr is the same on every
  // pass (the stride is a multiple of 16), so its rows' F are read once.
  static_assert((64 * ATTN_WAVES) % 16 == 0, "a thread's rr is fixed across passes");
  uint32_t Fr[NTILES];
#pragma unroll
  for (int tt = 0; tt < NTILES; ++tt) Fr[tt] = sF[16 * tt + (tid & 15)];
  for (int idx = tid; idx < TAB_DW / 2; idx += 64 * ATTN_WAVES) {
    const int dd = idx >> 4, rr = idx & 15;
    const uint32_t e = etab[dd];
    uint32_t packed = 0;
#pragma unroll
    for (int tt = 0; tt < NTILES; ++tt) {
      const uint32_t F = Fr[tt];
      const uint64_t prod = (uint64_t)(e & 0xffffffu) * (uint64_t)(F & 0xffffffu);  // 24-bit operands
      const uint32_t v = F == (1u << 24) ? e : (uint32_t)(prod >> 24);
      packed |= ((v > 255u ? 255u : v) ^ 0x80u) << (8 * tt);
    }
    tab[dd * 32 + rr] = packed;
    tab[dd * 32 + rr + 16] = packed;
  }
  __syncthreads();

  // ---------------- conversion: every score byte of this wave's units replaced by its
  // softmax code a - 128 (lanes g = 0, 1 (and 2, 3) read the two bank copies of their
  // row, so one lookup touches 32 distinct banks)
  if (active) {
    uint32_t cbase[NTL];
#pragma unroll
    for (int t = 0; t < NTL; ++t) cbase[t] = TAB + (uint32_t)((col + 16 * (g & 1)) * 4 + qset * NTL + t);
    auto code_at = [&](uint32_t dw, int k, int t) {
      return (uint32_t) * (const lds8*)(uintptr_t)__builtin_amdgcn_udot4(dw, 128u << (8 * k), cbase[t], false);
    };
    // four codes of one dword: two 16-bit halves (a shift-or each), then one byte
    // permute that takes bytes 0, 1 of each (three instructions per four codes)
    auto codes4 = [&](uint32_t dw, int t) {
      const uint32_t lo = code_at(dw, 0, t) | (code_at(dw, 1, t) << 8);
      const uint32_t hi = code_at(dw, 2, t) | (code_at(dw, 3, t) << 8);
      return (int)__builtin_amdgcn_perm(hi, lo, 0x05040100u);
    };
    // the next chunk is read before the current one is written back (chunks are disjoint)
    v4i svn[NTL];
    if (c_begin < c_full) {
#pragma unroll
      for (int t = 0; t < NTL; ++t) svn[t] = *chunk_ptr(c_begin, t);
    }
    for (int c = c_begin; c < c_full; ++c) {
      v4i sv[NTL];
      const int cn = min(c + 1, c_full - 1);
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
        sv[t] = svn[t];
        svn[t] = *chunk_ptr(cn, t);
      }
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
        v4i out;
#pragma unroll
        for (int wd = 0; wd < 4; ++wd) out[wd] = codes4(Mrep[t] - (uint32_t)sv[t][wd], t);
        *chunk_ptr(c, t) = out;
      }
    }
    if (c_full < c_end) {
      const int c = c_full;
#pragma unroll
      for (int t = 0; t < NTL; ++t) {
        const v4i sv = *chunk_ptr(c, t);
        v4i out;
#pragma unroll
        for (int wd = 0; wd < 4; ++wd) out[wd] = codes4(tail_dist(Mrep[t] - (uint32_t)sv[wd], c, wd), t);
        *chunk_ptr(c, t) = out;
      }
    }
  }
  __syncthreads();

  // ---------------- phase 3: A.V on MFMA, the waves split channels and keys
  const int cg = w % NCG, kh = w / NCG;
  int a_begin, a_end;
  split_pairs(nkc, P3_OLDER, 1, kh, &a_begin, &a_end);
  v4i acc[NTILES][AV_NT];
#pragma unroll
  for (int tt = 0; tt < NTILES; ++tt)
#pragma unroll
    for (int j = 0; j < AV_NT; ++j) acc[tt][j] = (v4i){0, 0, 0, 0};
  const bool wg_active = wg_q0 < L;
  if (wg_active && a_begin < a_end) {
    // V^T fragment of 16 channels x 64 keys (A operand: lane (ch, g) holds keys
    // 16 g .. 16 g + 15 of channel ch); codes of 16 queries x the same keys (B operand:
    // lane (q, g) holds keys 16 g .. of row q), straight from the score blocks
    constexpr int CH = 64 * DK;  // bytes of V^T per 64-key chunk
    const int8_t* vsrc = VTh + (size_t)(cg * AV_NT) * 1024 + frag_off;
    const uint32_t av0 = base + (uint32_t)(g * BLK + col * 16);
    // rings over the chunk phase (chunk - a_begin) % 3, all indices static: V fragments
    // two chunks ahead, codes one chunk ahead (past the last chunk the reads re-read it)
    int vpart[AV_NT];
    v4i vr[3][AV_NT], br[3][NTILES];
    auto ldv = [&](int c, v4i* dst) {
#pragma unroll
      for (int j = 0; j < AV_NT; ++j) dst[j] = *(const v4i*)(vsrc + (size_t)c * CH + j * 1024);
    };
    auto ldc = [&](int c, v4i* dst) {
      const uint32_t cp = av0 + (uint32_t)c * (4 * BLK);
#pragma unroll
      for (int tt = 0; tt < NTILES; ++tt) dst[tt] = *(const ldsv4*)(uintptr_t)(cp + tt * 256);
    };
#pragma unroll
    for (int j = 0; j < AV_NT; ++j) vpart[j] = 0;
    const int c_last = a_end - 1;
    ldv(a_begin, vr[0]);
    ldv(min(a_begin + 1, c_last), vr[1]);
    ldc(a_begin, br[0]);
    int c = a_begin;
    auto avstep = [&](auto Sc) {
      constexpr int S = decltype(Sc)::value;
      ldv(min(c + 2, c_last), vr[(S + 2) % 3]);
      ldc(min(c + 1, c_last), br[(S + 1) % 3]);
#pragma unroll
      for (int j = 0; j < AV_NT; ++j) {
#pragma unroll
        for (int wd = 0; wd < 4; ++wd) vpart[j] = __builtin_amdgcn_sdot4(vr[S][j][wd], 0x01010101, vpart[j], false);
#pragma unroll
        for (int tt = 0; tt < NTILES; ++tt)
          acc[tt][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(vr[S][j], br[S][tt], acc[tt][j], 0, 0, 0);
      }
      ++c;
    };
    while (c + 3 <= a_end) {
      avstep(Phase<0>{});
      avstep(Phase<1>{});
      avstep(Phase<2>{});
    }
    if (c < a_end) avstep(Phase<0>{});
    if (c < a_end) avstep(Phase<1>{});
    // exact correction for the -128 offset: + 128 * sum of V over the same keys.  Lane
    // (ch, g) summed keys 16 g .. of channel ch; the output lane (q, g) needs channels
    // 4 g .. 4 g + 3.
#pragma unroll
    for (int j = 0; j < AV_NT; ++j) {
      const int vs = (int)col4_sum((uint32_t)vpart[j]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int vi = __shfl(vs, 4 * g + i);
#pragma unroll
        for (int tt = 0; tt < NTILES; ++tt) acc[tt][j][i] += 128 * vi;
      }
    }
  }

  // ---------------- combine the two key parts, requantize, store.  The (tile, channel
  // tile) units of a channel group alternate between its two waves: each wave leaves
  // the partial sums of the units it does not own in the table region, as
  // [cg][value][lane] int32, and adds its partner's to the units it owns (exact).
  // The lane's column is read afresh from the lane counter: kept from the start, it
  // was the one value the register allocator spilled to scratch memory.
  int lane_now;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane_now));
  const int col_now = lane_now & 15;
  constexpr int R = NTILES * AV_NT * 4;
  constexpr int NU = NTILES * AV_NT;
  ldsi32* red = (ldsi32*)(uintptr_t)TAB;
#pragma unroll
  for (int u = 0; u < NU; ++u)
    if (u % KH != kh) {
#pragma unroll
      for (int i = 0; i < 4; ++i) red[(cg * R + u * 4 + i) * 64 + lane] = acc[u / AV_NT][u % AV_NT][i];
    }
  __syncthreads();
  // lane (q, g) of unit (tt, j) holds query wg_q0 + 16 tt + q, channels
  // 16 (cg AV_NT + j) + 4 g .. + 3
  const int64_t half_o = (int64_t)1 << (a.shift_o - 1);
  auto requant_o = [&](int32_t v) -> uint32_t {
    const int64_t r = ((int64_t)v * a.m_o + half_o) >> a.shift_o;
    return (uint32_t)(r < -127 ? -127 : (r > 127 ? 127 : (int)r)) & 0xffu;
  };
#pragma unroll
  for (int u = 0; u < NU; ++u) {
    if (u % KH != kh) continue;
    const int tt = u / AV_NT, j = u % AV_NT;
    const int qi = wg_q0 + 16 * tt + col_now;
    if (qi >= T) continue;
    uint32_t packed = 0;
    if (qi < L) {
#pragma unroll
      for (int i = 0; i < 4; ++i) packed |= requant_o(acc[tt][j][i] + red[(cg * R + u * 4 + i) * 64 + lane]) << (8 * i);
    }
    *(uint32_t*)(a.ctx + ((size_t)b * T + qi) * a.d + (size_t)h * DK + (cg * AV_NT + j) * 16 + 4 * g) = packed;
  }
}

// The core kernel: one workgroup shape (NTL2 == 0), or two shapes in one grid, the
// first one's blocks ahead of the second one's, so that the second shape fills what
// the first leaves of the last round (workgroups start in block order).
template <int DK, int KS1, int NTL1, int KS2, int NTL2, bool WIDE>
__global__ __launch_bounds__(64 * ATTN_WAVES) void relpos_attn_core(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  if constexpr (NTL2 == 0) {
    attn_block<DK, KS1, NTL1, WIDE>(a, smem, blockIdx.x, a.dv_nqb, 0);
  } else {
    if ((int)blockIdx.x < a.seg2_block)
      attn_block<DK, KS1, NTL1, WIDE>(a, smem, blockIdx.x, a.dv_nqb, 0);
    else
      attn_block<DK, KS2, NTL2, WIDE>(a, smem, blockIdx.x - a.seg2_block, a.dv_nqb2, a.seg2_q0);
  }
}

// The I-BERT integer exp of every score distance d = M - s in [0, 254] (Sec. 2.2:
// d = z q_ln2 - r with r in (-q_ln2, 0], e = ((r + q_b)^2 + q_c) >> z), and 0 at d = 255,
// which no score reaches; integer arithmetic only.  One thread per d.
__global__ __launch_bounds__(256) void iexp_table(uint32_t* tab, int q_ln2, int q_b, int q_c) {
  const int dd = threadIdx.x;
  uint32_t e = 0;
  if (dd < 255) {
    int z = 0, rem = dd;
    while (rem >= q_ln2) {  // z = floor(d / q_ln2), d <= 254
      rem -= q_ln2;
      ++z;
    }
    const int r = -rem;
    const int poly = (r + q_b) * (r + q_b) + q_c;  // < 2^24 (checked at create)
    e = z >= 32 ? 0u : ((uint32_t)poly >> z);
  }
  tab[dd] = e;
}

hipError_t launch_iexp_table(uint32_t* tab, int q_ln2, int q_b, int q_c, hipStream_t st) {
  hipLaunchKernelGGL(iexp_table, dim3(1), dim3(256), 0, st, tab, q_ln2, q_b, q_c);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Copies a workspace tensor back to the documented [B][T][d] / [2T-1][d] layouts.
struct GatherArgs {
  const int8_t* src;
  int8_t* dst;
  int which, B, T, T_al, H, dks, d, p_rows, p_base;  // d_k = 2^dks
};

// grid: (d / 256 rounded up, rows per utterance, utterances); no division on the device
__global__ __launch_bounds__(256) void gather_intermediate(GatherArgs a) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= a.d) return;
  const int t = blockIdx.y, b = blockIdx.z;
  const int h = c >> a.dks, kk = c & ((1 << a.dks) - 1), DK = 1 << a.dks;
  const size_t idx = ((size_t)b * a.T + t) * a.d + c;
  int8_t v;
  if (a.which == 3) {  // the position table, [2T-1][d]
    v = a.src[(size_t)h * a.p_rows * DK + frag_index(a.p_base + t, kk, DK)];
    a.dst[(size_t)t * a.d + c] = v;
    return;
  }
  if (a.which >= 4) {  // the context or the LayerNorm output, [B][T][d]
    v = a.src[idx];
  } else {
    const size_t base = ((size_t)b * a.H + h) * a.T_al * DK;
    v = a.src[base + (a.which == 2 ? vt_index(t, kk, DK) : frag_index(t, kk, DK))];
  }
  a.dst[idx] = v;
}

// ---------------------------------------------------------------------------
size_t attn_lds_bytes(int DK, int ksplit, int ntl, int T_al) {
  (void)DK;
  const int rows = 16 * ntl, wgq = rows * (ATTN_WAVES / ksplit);
  return attn_lds(wgq, rows, T_al).total;
}

// Workgroup shapes the kernel is built for: (key splits, 16-query tiles per wave).
static const AttnCfg kAttnCfgs[] = {{4, 2}, {8, 2}, {8, 3}};
// One 16-query tile per wave: the smallest score rows, for utterances whose rows do not
// fit any shape above (every K and P fragment then feeds a single MFMA)
static const AttnCfg kAttnLong = {8, 1};
constexpr size_t kLdsBudget = 160 * 1024;
constexpr int kNumCUs = 256;

static int wgq_of(const AttnCfg& c) { return 16 * c.ntl * (ATTN_WAVES / c.ksplit); }
static bool fits(const AttnCfg& c, int DK, int T_al) { return attn_lds_bytes(DK, c.ksplit, c.ntl, T_al) <= kLdsBudget; }

// Time of one workgroup, modelled per key of a wave's share as 125 cycles for the K, P
// and V streams (the same for any number of query tiles) plus 29 per 16-query tile
// (score post-processing, exp sums, code lookups, combine), as measured on the
// long-form workload, plus a fixed ~16 K cycles that do not scale with T (operand
// loads before the first step, the exp and code tables, F, the barriers and the
// combine): at T = 500 a 48-query workgroup lives ~25 K cycles.  Without the fixed
// part, short utterances in large batches took 48-query workgroups in more rounds where
// 64-query ones in fewer finish first (T = 375 x 16 and 500 x 8: 13 - 17 % less time in
// the core, measured).  At T = 2500 the fixed part does not change the plan.
constexpr double kWgFixedCost = 16000.0;
static double wg_cost(const AttnCfg& c, int T) {
  return kWgFixedCost + ((double)T / c.ksplit) * (125.0 + 29.0 * c.ntl);
}

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
  a2.dv_nqb = make_div((uint32_t)p.nqb1);
  a2.dv_nqb2 = make_div((uint32_t)(p.nqb2 > 0 ? p.nqb2 : 1));
  a2.dv_H = make_div((uint32_t)H);
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
  a.etab = w.etab;
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
  a.m_c = sc.m_c;
  a.m_p = sc.m_p;
  a.shift_s = sc.shift_s;
  a.bias64 = ((int64_t)1 << (sc.shift_s - 1)) + ((int64_t)128 << sc.shift_s);
  a.m_o = sc.m_o;
  a.shift_o = sc.shift_o;
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
  a.dks = rs.DK == 128 ? 7 : 6;
  a.d = rs.d;
  a.p_rows = rs.p_rows;
  a.p_base = rs.p_base;
  const dim3 grid((unsigned)((rs.d + 255) / 256), (unsigned)(which == 3 ? 2 * rs.T - 1 : rs.T),
                  (unsigned)(which == 3 ? 1 : rs.B));
  hipLaunchKernelGGL(gather_intermediate, grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace ipk
