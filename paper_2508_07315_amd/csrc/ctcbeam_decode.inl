// Batched CTC beam search, all frames of one utterance per workgroup (gfx950).
// Included by the per-LPT instantiation units (ctcbeam_kernel_lpt*.hip).
//
// Implements the per-frame step of FlexCTC Algorithm 1 (score update with the
// blank/repeat masks, flat TopK over K*(V+1) candidates, threshold pruning,
// LM/boosting state update for emitting labels, beam update, recombination)
// followed by LM.Final and the transcript read-out of the hypothesis trie
// (Sec. III-A).  Scores follow Eq. 1 with the fp32 fold
//   x = s_k + D[c]; x += beta; x += fl(alpha*LM); x += fl(w*BT)
// for emitting labels (neither blank nor a repeat of the beam's last frame
// label).
//
// Design (MI355X, CDNA4): the search is a serial chain over frames, so each
// utterance is one persistent workgroup of 8 wave64 that loops over its own
// frames with no host round trip; the B utterances are independent
// workgroups.  There is no dense contraction: the work is gathers of LM arcs,
// VALU scoring and a selection, bound by dependent latency (LDS round trips,
// cross-lane chains, barriers), so MFMA is not used.
//
// Every wave keeps the whole beam (slot j in lane j: score, last label,
// length, LM/boosting chain headers) in registers and runs the beam update
// itself, so the next frame's fill starts without a hand-off between waves.
// Per-slot state records (transcript hash, LM/boosting states, chains) live
// in LDS, double-buffered by frame.  Per frame (one chunk when K*V fits the
// LDS key rows, e.g. K=8, V=1024), with 4 barriers:
//   F. fill: the explicit continuations of every live beam's LM backoff chain
//      (and its merged boosting continuation list) are cut into tiles of 64
//      that never straddle a (beam, level) run and are dealt to all waves;
//      each lane loads one arc per tile and scatters it into an LDS
//      [beam][token] row: LM entries are 64-bit (generation | order | staging
//      slot : alpha*value) combined with an atomic max, so the highest-order
//      n-gram wins in any order; boosting entries are generation-tagged keys.
//      Entries of older generations read as absent, so the rows are never
//      cleared (except when the 6-bit generation wraps).  For small beams
//      with an LM and no boosting the rows are kept per LM state across
//      frames and only states new to the rows are filled (CACHE); those rows,
//      and the rows of chains of four or more levels, also get the unigram +
//      backoff fold of every token as an order-0 entry.
//   C. candidates: each lane scores its labels for every beam of the chunk in
//      registers (beam data by broadcast LDS reads), resolving the LM value
//      from the row or from the unigram + backoff fold, and publishes the
//      maxima of disjoint (beam row, lane group) candidate groups.
//   T. filter: the K-th largest group maximum (over the frame's chunks so
//      far), and with K live slots the smallest blank score, bound the K-th
//      best candidate from below; candidates at or above the bound (a few on
//      the 3-gram workload) go to a survivor pool in LDS.
//   R. rank: the pool (survivors plus K reserved entries holding the blank
//      candidates, or the best K of earlier chunks) is ranked exactly by
//      (score desc, flat index asc): each wave ranks an eighth of the pool
//      against all of it with ballots.  The owner of each winner builds its
//      successor record from the parent's record (hash of the collapsed
//      transcript, LM/boosting states, chain headers of an emitted token,
//      fetched while the ranking runs).
//   U. update: prune, recombine, take the new beam into registers, plan the
//      next frame's chunks, write back-pointers to HBM.
// Large beams (K*V above the key rows) repeat F/C/T per chunk of beams with
// a running bound and rank the pool only when it fills up or after the last
// chunk.  A survivor pool overflow falls back to an exact extraction.  After the last frame the best beam is traced back through the
// back-pointers staged in LDS.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ctcbeam_internal.h"
#include "ctcbeam_lane.h"

namespace ctcbeam {
namespace detail {


// generation tag in the top 6 bits of LM entry high words and boosting keys
constexpr int kGenShift = 26;
constexpr uint32_t kGenMax = 63u;
constexpr uint32_t kLowMask = (1u << kGenShift) - 1u;
constexpr int kTileUnroll = 8;
// LM target state in a cached row entry (the states are numbered below 2^23)
constexpr uint32_t kTargetMask = (1u << 23) - 1u;

// ---- fp32 log-sum-exp of the log-sum-exp recombination variant ----
// Every step is one IEEE fp32 operation in a fixed order (no contraction), so
// the result is reproducible bit for bit.  exp(d), -80 <= d <= 0: Cody-Waite
// reduction d = k ln2 + r with k = rint(d / ln2) and ln2 split into a 9-bit
// head (k * head is exact) and a tail, the degree-7 Taylor polynomial of e^r
// by Horner, times 2^k built from its exponent bits.
__device__ __forceinline__ float exp32_nonpos(float d) {
  const float k = __builtin_rintf(d * 1.44269504f);
  const float r = (d - k * 0.693359375f) - k * -2.12194440e-4f;
  float q = 1.0f / 5040.0f;
  q = q * r + 1.0f / 720.0f;
  q = q * r + 1.0f / 120.0f;
  q = q * r + 1.0f / 24.0f;
  q = q * r + 1.0f / 6.0f;
  q = q * r + 0.5f;
  q = q * r + 1.0f;
  q = q * r + 1.0f;
  return q * __uint_as_float(static_cast<uint32_t>(static_cast<int>(k) + 127) << 23);
}
// log(1 + e), 2^-24 <= e <= 1: 2 atanh(s) with s = e / (2 + e) <= 1/3, the odd
// series to s^17 by Horner in s^2.
__device__ __forceinline__ float log1p32_unit(float e) {
  const float s = e / (2.0f + e);
  const float z = s * s;
  float q = 1.0f / 17.0f;
  q = q * z + 1.0f / 15.0f;
  q = q * z + 1.0f / 13.0f;
  q = q * z + 1.0f / 11.0f;
  q = q * z + 1.0f / 9.0f;
  q = q * z + 1.0f / 7.0f;
  q = q * z + 1.0f / 5.0f;
  q = q * z + 1.0f / 3.0f;
  q = q * z + 1.0f;
  const float t = s * q;
  return t + t;
}
// log(exp(a) + exp(b))
__device__ __forceinline__ float lse32(float a, float b) {
  const float hi = (a < b) ? b : a;
  const float lo = (a < b) ? a : b;
  if (lo == kNegInf) return hi;
  const float d = lo - hi;
  if (d < -80.0f) return hi;
  const float e = exp32_nonpos(d);
  const float l = (e < 5.9604645e-8f) ? e : log1p32_unit(e);
  return hi + l;
}

// Bitonic sort of (hi, lo, slot) triples, one per lane, ascending over the
// wave (slots are distinct, so the order is total).
template <int k, int jd>
__device__ __forceinline__ void sort3_step(uint32_t& lo, uint32_t& hi, uint32_t& sl, int lane) {
  const uint32_t olo = xor_lane(lo, jd, lane), ohi = xor_lane(hi, jd, lane), osl = xor_lane(sl, jd, lane);
  const bool less = ohi < hi || (ohi == hi && (olo < lo || (olo == lo && osl < sl)));
  // lanes that keep the larger in the descending network keep the smaller here
  const bool take = less == lane_in_here<bitonic_max_lanes(k, jd, 64)>();
  lo = take ? olo : lo;
  hi = take ? ohi : hi;
  sl = take ? osl : sl;
}
template <int k, int jd>
__device__ __forceinline__ void sort3_merge(uint32_t& lo, uint32_t& hi, uint32_t& sl, int lane) {
  sort3_step<k, jd>(lo, hi, sl, lane);
  if constexpr (jd > 1) sort3_merge<k, jd / 2>(lo, hi, sl, lane);
}
template <int k>
__device__ __forceinline__ void sort3_levels(uint32_t& lo, uint32_t& hi, uint32_t& sl, int lane) {
  sort3_merge<k, k / 2>(lo, hi, sl, lane);
  if constexpr (k < 64) sort3_levels<k * 2>(lo, hi, sl, lane);
}
// Recombination of up to 64 slots (lane = slot): sorts the 64-bit keys with
// their slots and flags each slot whose sorted predecessor has the same key,
// i.e. a lower slot with the same transcript.  Dead slots carry all ones and
// are never flagged.  The sorted keys are left in lo / hi (for searches).
__device__ __forceinline__ bool dup_by_sort(uint64_t key, int lane, uint32_t& lo, uint32_t& hi) {
  lo = static_cast<uint32_t>(key);
  hi = static_cast<uint32_t>(key >> 32);
  uint32_t sl = static_cast<uint32_t>(lane);
  sort3_levels<2>(lo, hi, sl, lane);
  const int pa = (lane == 0 ? 63 : lane - 1) << 2;
  const uint32_t plo = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(pa, static_cast<int>(lo)));
  const uint32_t phi = static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(pa, static_cast<int>(hi)));
  const bool d = lane > 0 && plo == lo && phi == hi && (lo & hi) != 0xFFFFFFFFu;
  // back to the slot's lane (the slots are a permutation of the lanes)
  return __builtin_amdgcn_ds_permute(static_cast<int>(sl) << 2, d ? 1 : 0) != 0;
}

// Per-phase clocks (profiling builds, -DCTCBEAM_PHASE_CLOCKS; the macro is in
// ctcbeam_internal.h): each wave adds the s_memtime cycles of every phase of
// every frame (fill, barrier A, candidates, barrier B, filter, barrier C,
// rank, barrier D, the update's remainder; then the frame and chunk counts;
// then, one slot per lane, the update's prune + recombination, new state and
// chunk plan; then the bound, split from the filter) and writes them after the [B, 8] statistics as
// [B, kWaves, kPhaseWords] int64.

// SPL = beam slots per lane: slot j lives in lane j % 64, register set
// j / 64 (SPL = 2 serves beams of 65..128).  SKIP: ranks of chunks before
// the last are skipped while the survivor pool has room (beams above one
// chunk; small beams keep one rank per chunk and the simpler code).
// CACHE (one chunk, one slot per lane, LM without boosting, LM states below
// 2^23): LM key rows are kept per LM state across frames and only the states
// new to the rows are filled; an entry holds its arc's target state.
// REP: the repeat-scoring variant (CTCBEAM_FLAG_REPEAT_SCORE), a kernel of
// its own so that the default kernels carry none of its state.  TREE (beams
// of 33..64): pools of more than 192 entries are reduced to their top 64 by
// a merge tree instead of the block rank (a kernel of its own: the code
// costs the smaller beams' kernels about 3 % through register allocation).
template <int LPT, int NLEV, bool HAS_BT, int SPL, bool SKIP, bool CACHE, bool REP, bool TREE>
__global__ void __launch_bounds__(kThreads) decode_kernel(KernelParams p) {
  constexpr bool HAS_LM = NLEV >= 0;
  constexpr int NL = NLEV > 0 ? NLEV : 0;     // chain levels above the unigram root
  constexpr int NLA = NL > 0 ? NL : 1;        // array extent
  constexpr int NF = NL > 1 ? NL - 1 : 1;     // backoff weights folded into an arc (extent)
  constexpr int KMX = 64 * SPL;               // slot capacity
  // beams (key rows) per chunk; two slots per lane leave LDS for 12 rows of
  // 1024 labels instead of 16
  constexpr int KCR = (SPL == 1 ? 16 : 12) / LPT;
  // LDS scratch carved from one block so the traceback can reuse it:
  // [LM rows: KW x u64][boosting rows: KW x u32][LM targets: kLmStage]
  constexpr int KW = KCR * LPT * kThreads;
  constexpr int kBigWords = 3 * KW + kLmStage;
  constexpr int kOffBtRow = 2 * KW;
  constexpr int kOffTgt = 3 * KW;
  constexpr int NC = KCR * LPT;               // candidates per lane
  // a chunk has at most 64 LM segments (beam, level): one lane each
  constexpr int KSEG = (NL > 0 && KCR * NL > 64) ? 64 / (NL > 0 ? NL : 1) : KCR;
  // without rank skipping the beam fits one chunk of 16 / LPT rows: K <= 8
  // for two or more labels per lane
  constexpr bool kSmallK = SPL == 1 && !SKIP && LPT >= 2;
  // rank skipping means K > 16 / LPT: no beam of at most 8 for LPT <= 2
  constexpr bool kMaySmallK = !SKIP || LPT > 2;
  // LM arc tiles in flight per wave: cached rows fill only the new states
  constexpr int kLmTU = CACHE ? 4 : kTileUnroll;
  // boosting continuation tiles in flight per wave (a few dozen arcs a frame:
  // more tiles only add registers)
  constexpr int kBtTU = 1;
  static_assert(!CACHE || (kSmallK && HAS_LM && NL > 0 && !HAS_BT), "row caching needs one chunk and an LM");
  // The key rows hold the unigram + backoff fold of every token (as order-0
  // entries) with row caching, and for chains of four or more levels with
  // one slot per lane, whose backoff weights would otherwise take KCR x NL
  // registers in the scoring.  Shorter chains, and the many chunks of two
  // slots per lane, fold in the scoring: cheaper than the extra LDS maxima.
  constexpr bool kFoldRows = CACHE || (NL >= 4 && SPL == 1);
  // Fill groups (beams over one chunk, no row cache): the update orders the
  // live beams by LM state and cuts that order into groups of consecutive
  // chunks whose distinct LM states (at most KSEG), boosting lists (at most
  // KCR - 1) and staged arcs (at most kLmStage) fit the rows (a state whose
  // own lists exceed a group is split by list).  A state or list has one row per group,
  // filled at the group's first chunk; the group's other chunks skip the
  // fill and its barrier.  Large beams hold few distinct states and lists
  // (at K = 64 about 10 and 6), so a frame fills about two groups.
  constexpr bool kGroups = !CACHE && SKIP && (HAS_LM || HAS_BT);
  constexpr int kRowWords = kFoldRows ? 4 : 16;  // beam record per live position
  // beam state record (one per slot, double-buffered by frame): score bits,
  // back-pointer, transcript hash (2), length, last label, LM state, then
  // with boosting: boosting state, emitted flag, boosting list
  // begin/count/pot; without: emitted flag; then LM chain begin[NL],
  // count[NL], backoff[NL]; then the fl(alpha*LM) and fl(w*BT) terms the
  // last emitted token received (read by the repeat-scoring variant).  The
  // boosting fields exist (and are accessed) only with boosting.
  constexpr int kRX = 0, kRBp = 1, kRHlo = 2, kRHhi = 3, kRLen = 4, kRLast = 5, kRLms = 6;
  constexpr int kRBts = 7, kRBtb = 9, kRBtc = 10, kRBtp = 11;
  constexpr int kREmit = HAS_BT ? 8 : 7;
  constexpr int kRLvb = HAS_BT ? 12 : 8, kRLvc = kRLvb + NL, kRLvbo = kRLvb + 2 * NL;
  constexpr int kRRal = kRLvb + 3 * NL, kRRwb = kRRal + 1;
  constexpr int RW = ((REP ? kRRwb + 1 : kRRal) + 3) & ~3;
  static_assert(!(REP && CACHE), "the repeat-scoring variant reads uncached rows");

  __shared__ __align__(16) uint32_t s_big[kBigWords];
  // survivor pool: score bits, flat index, LM target (raw), boosting key
  __shared__ uint4 s_pool[kCap];
  static_assert(kCap / 2 <= kThreads, "the fallback reads carried pool entries one per thread");
  // reserved regions (ping-pong): blank candidates, or the best K so far
  __shared__ uint4 s_res[2][KMX];
  // repeat-scoring variant only: the (fl(alpha*LM), fl(w*BT)) terms of the
  // pool entries and of the reserved entries, moved along with them
  __shared__ float2 s_pinc[REP ? kCap : 1];
  __shared__ float2 s_rinc[2][REP ? KMX : 1];
  // beam records by live position: score, last label, slot (and key row),
  // boosting pot, backoff weights unless the rows hold the fold; reused by
  // the epilogue (lengths and ranks, 2 KMX words)
  __shared__ __align__(16) uint32_t s_row[(KMX + 16) * kRowWords];
  // beam state records by slot: [rcur] the current beam, [rcur ^ 1] its successors
  __shared__ __align__(16) uint32_t s_rec[2 * KMX * RW];
  // group maxima of the bound; K <= 8: (row, wave) maxima, then wave maxima
  __shared__ float s_top[kWaves * 8 * SPL + kWaves];
  __shared__ uint64_t s_red[2][kWaves];
  __shared__ int32_t s_nbuf, s_overflow;
  // top 64 of a large pool (one slot per lane, beams over one chunk): the
  // sorted lists of the merge tree (4 + 2 + 1 lists of 64 (lo, hi, source)
  // triples) and the waves' counts of finite entries
  constexpr bool kTreeRank = SPL == 1 && SKIP && TREE;
  __shared__ uint32_t s_srt[kTreeRank ? 7 : 1][3][64];
  __shared__ int32_t s_wcnt[kWaves];
  __shared__ int32_t s_best, s_bestlen;
  __shared__ float s_bestscore;
  // statistics (only with p.stats): alive beam-frames, LM chain states and
  // arcs, boosting chain nodes and arcs, emitting winners
  __shared__ unsigned long long s_st[6];

  uint64_t* const lmrow = reinterpret_cast<uint64_t*>(s_big);
  uint32_t* const btrow = s_big + kOffBtRow;
  uint32_t* const tgt = s_big + kOffTgt;
  // LM target of an uncached row entry (or of a pool entry's raw field): an
  // explicit arc (order >= 1) names its staging slot; a fold entry (order 0)
  // or, in rows without folds, a bare token names the token, whose unigram
  // state has the token's id
  const auto lm_target = [&](uint32_t hi) __attribute__((always_inline)) {
    if constexpr (kFoldRows) return ((hi >> 23) & 7u) != 0u ? tgt[hi & 0xFFFu] : (hi & 0xFFFu);
    else return (hi >> kGenShift) != 0u ? tgt[hi & 0xFFFu] : hi;
  };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: keep it in an SGPR
  const int b = blockIdx.x;
  const int V = p.V, W = V + 1, K = p.K, T = p.T;
  const int kcmax = min(K, KSEG);
  const float alpha = p.alpha, beta = p.beta, boost_w = p.boost_w;
  const uint64_t lmlt = lanemask_lt();
  // repeat-scoring variant: a repeated token gets its LM / boosting terms again
  constexpr bool rep = REP;

  int L = p.lengths[b];
  uint32_t status = 0;
  if (L < 0) { L = 0; status |= 1u; }
  if (L > T) { L = T; status |= 1u; }
  const float* Db = p.logprobs + static_cast<size_t>(b) * T * W;
  int32_t* bpb = p.bp + static_cast<size_t>(b) * T * K;

  // ---- per-lane label constants and the first row ----
  // lane owns labels c = tid + j*512; labels >= V score -inf through rD
  float rD[LPT], rDn[LPT], rP1[LPT];
  uint32_t rRoot[LPT], rcc[LPT];
#pragma unroll
  for (int j = 0; j < LPT; ++j) {
    const int c = tid + j * kThreads;
    const bool ok = c < V;
    rcc[j] = ok ? static_cast<uint32_t>(c) : 0u;
    rP1[j] = (HAS_LM && ok) ? p.lm_unigram[c] : 0.0f;
    rRoot[j] = (HAS_BT && ok) ? p.bt_root_key[c] : 0u;
    rDn[j] = ok ? (L > 0 ? Db[c] : 0.0f) : kNegInf;
    rD[j] = kNegInf;
  }
  float rBlankN = (L > 0 && lane < K) ? Db[V] : 0.0f;
  float rBlank = 0.0f;

  // ---- beam state: slot j = lane + 64 h in register set h, replicated in
  // every wave ----
  const int j = lane;
  float sc[SPL];
  int32_t last[SPL], len[SPL];
  uint32_t lvb[SPL][NLA], lvc[SPL][NLA];
  float lvbo[SPL][NLA];
  uint32_t btb[SPL], btc[SPL];
  int32_t btpot[SPL];
  bool alive[SPL];
  // kGroups: fill group of slot j + 64 h (-1: dead), its LM and boosting
  // rows there and whether the slot fills them; lane q of gch0[h]: the first
  // chunk of group q + 64 h (at most one group per live slot)
  int grp[SPL], lrow_g[SPL], brow_g[SPL], gch0[SPL];
  bool lown[SPL], bown[SPL];
#pragma unroll
  for (int h = 0; h < SPL; ++h) {
    grp[h] = 0;
    lrow_g[h] = 0;
    brow_g[h] = 0;
    gch0[h] = 0;
    lown[h] = bown[h] = h == 0 && j == 0;
  }
  int ngrp = 1;
#pragma unroll
  for (int h = 0; h < SPL; ++h) {
    sc[h] = (h == 0 && j == 0) ? 0.0f : kNegInf;
    last[h] = V;
    len[h] = 0;
#pragma unroll
    for (int l = 0; l < NLA; ++l) {
      lvb[h][l] = 0u;
      lvc[h][l] = 0u;
      lvbo[h][l] = 0.0f;
    }
    btb[h] = 0u;
    btc[h] = 0u;
    btpot[h] = 0;
    alive[h] = h == 0 && j == 0;
  }
#ifdef CTCBEAM_PHASE_CLOCKS
  // profiling builds: the stats buffer takes the phase clocks, and the
  // counters stay off so that the phases time what a plain launch runs
  const bool want_stats = false;
#else
  const bool want_stats = p.stats != nullptr;
#endif
  if (j == 0) {
    if (HAS_LM) {
#pragma unroll
      for (int l = 0; l < NL; ++l) {
        const LmLevel hd = p.lm_states[static_cast<size_t>(p.lm_bos_state) * NL + l];
        lvb[0][l] = hd.begin;
        lvc[0][l] = hd.count;
        lvbo[0][l] = hd.bo;
      }
    }
    if (HAS_BT) {
      const BtNode nd = p.bt_nodes[0];
      btb[0] = nd.list_begin;
      btc[0] = nd.list_count;
      btpot[0] = static_cast<int32_t>(nd.pot & 0xFFu);
    }
  }
  // Row cache (CACHE): lane r < KCR holds the LM state of key row r; lane j
  // the row of slot j and whether slot j fills it in the next frame.  A
  // filled row holds an entry for every token.
  uint32_t rtag = 0xFFFFFFFFu;
  int rowof = 0;
  bool fillrep = false;
  if (CACHE && j == 0 && L > 0) {
    rtag = p.lm_bos_state;
    fillrep = true;
  }
  // beam record of live position lp for slot j + 64 h (written by wave 0 for
  // the live slots); with CACHE the slot field also carries the key row
  // (bits 8..15)
  auto put_row = [&](int lp, int h) __attribute__((always_inline)) {
    uint32_t* rr = s_row + lp * kRowWords;
    const uint32_t zf = static_cast<uint32_t>(j + 64 * h) | (CACHE ? static_cast<uint32_t>(rowof) << 8 : 0u) |
                        (kGroups ? (static_cast<uint32_t>(lrow_g[h]) << 8) | (static_cast<uint32_t>(brow_g[h]) << 16) : 0u);
    *reinterpret_cast<uint4*>(rr) = make_uint4(__float_as_uint(sc[h]), static_cast<uint32_t>(last[h]),
                                               zf, static_cast<uint32_t>(btpot[h]));
#pragma unroll
    for (int l0 = 0; l0 < (kFoldRows ? 0 : NL); l0 += 4) {
      const auto bo_at = [&](int l) __attribute__((always_inline)) { return l < NL ? __float_as_uint(lvbo[h][l < NLA ? l : 0]) : 0u; };
      *reinterpret_cast<uint4*>(rr + 4 + l0) = make_uint4(bo_at(l0), bo_at(l0 + 1), bo_at(l0 + 2), bo_at(l0 + 3));
    }
  };
  // chunk plan: chunk id of each live slot, number of chunks (uniform)
  int cid[SPL];
#pragma unroll
  for (int h = 0; h < SPL; ++h) cid[h] = 0;
  int nch = 1;
  // kGroups: the fill-group plan of the next frame from the new beam (nal:
  // live slots, ac: staged arcs, lk: LM state keys).  LM states are taken in
  // order of their lowest slot; a group takes whole states while its LM rows,
  // staging area and boosting lists have room, and its beams get consecutive
  // live positions, KCR to a chunk (a state whose own lists exceed a group is
  // split by list).  A boosting list is named by its leader, its lowest slot;
  // in a group it gets the rank of its leader among the group's lists as its
  // row, and its lowest member in the group fills the row.  A group holds at
  // most KCR - 1 lists: beams without a list read row KCR - 1, which the
  // group's fill leaves empty.  Sets the live positions lpos, the group
  // fields and chunk ids of the slots, nch, ngrp and gch0.
  const auto plan_groups = [&](const bool (&nal)[SPL], const int32_t (&ac)[SPL], const uint32_t (&lk)[SPL],
                               int (&lpos)[SPL]) __attribute__((always_inline)) {
    const auto any = [&](const uint64_t (&m)[SPL]) __attribute__((always_inline)) {
      bool r = false;
#pragma unroll
      for (int h = 0; h < SPL; ++h) r = r || m[h] != 0ull;
      return r;
    };
    // the register set holding the lowest slot of a non-empty mask
    const auto low_set = [&](const uint64_t (&m)[SPL]) __attribute__((always_inline)) {
      int hs = SPL - 1;
#pragma unroll
      for (int h = SPL - 1; h >= 0; --h) hs = m[h] != 0ull ? h : hs;
      return hs;
    };
    const auto rd64 = [&](uint64_t v, int l) __attribute__((always_inline)) {
      return (static_cast<uint64_t>(rdlane(static_cast<uint32_t>(v >> 32), l)) << 32) |
             rdlane(static_cast<uint32_t>(v), l);
    };
    uint64_t rem[SPL], hbm[SPL];
    bool hasb[SPL], lead[SPL];
    int bl[SPL];             // leader of the slot's boosting list
    uint64_t lmk[SPL][SPL];  // the slots holding the slot's list, by register set
#pragma unroll
    for (int h = 0; h < SPL; ++h) {
      rem[h] = __ballot(nal[h]);
      hasb[h] = HAS_BT && nal[h] && btc[h] != 0u;
      hbm[h] = __ballot(hasb[h]);
      lead[h] = false;
      bl[h] = 0;
#pragma unroll
      for (int hh = 0; hh < SPL; ++hh) lmk[h][hh] = 0ull;
      grp[h] = -1;
      lrow_g[h] = 0;
      brow_g[h] = KCR - 1;
      lown[h] = bown[h] = false;
      cid[h] = -1;
      gch0[h] = 0x7FFFFFFF;
    }
    if constexpr (HAS_BT) {
      // the distinct lists (begin, count): one a pass
      uint64_t brem[SPL];
#pragma unroll
      for (int h = 0; h < SPL; ++h) brem[h] = hbm[h];
      while (any(brem)) {  // uniform
        const int hl = low_set(brem);
        int jl = 0;
        uint32_t b0 = 0u, c0 = 0u;
#pragma unroll
        for (int h = 0; h < SPL; ++h) {
          if (h == hl) {
            jl = static_cast<int>(__builtin_ctzll(brem[h]));
            b0 = rdlane(btb[h], jl);
            c0 = rdlane(btc[h], jl);
          }
        }
        uint64_t m[SPL];
#pragma unroll
        for (int hh = 0; hh < SPL; ++hh) {
          m[hh] = __ballot(hasb[hh] && btb[hh] == b0 && btc[hh] == c0);
          brem[hh] &= ~m[hh];
        }
#pragma unroll
        for (int h = 0; h < SPL; ++h) {
          if ((m[h] >> j) & 1ull) {
            bl[h] = jl + 64 * hl;
#pragma unroll
            for (int hh = 0; hh < SPL; ++hh) lmk[h][hh] = m[hh];
          }
        }
      }
#pragma unroll
      for (int h = 0; h < SPL; ++h) lead[h] = hasb[h] && bl[h] == j + 64 * h;
    }
    int pos = 0, g = -1, chn = 0;
    int g_rows = 0, g_arcs = 0, g_beams = 0;
    uint64_t g_bl[SPL], g_mem[SPL];  // the open group's lists (by leader) and members
#pragma unroll
    for (int h = 0; h < SPL; ++h) g_bl[h] = g_mem[h] = 0ull;
    // the open group's chunks, and its members' boosting rows and fillers
    const auto close_group = [&]() __attribute__((always_inline)) {
      if (g < 0) return;
      chn += (g_beams + KCR - 1) / KCR;
      if constexpr (HAS_BT) {
#pragma unroll
        for (int h = 0; h < SPL; ++h) {
          if (grp[h] == g && hasb[h]) {
            const int L = bl[h];
            int r = 0;
            bool first = true;
#pragma unroll
            for (int hh = 0; hh < SPL; ++hh) {
              const uint64_t lead_below =
                  hh < (L >> 6) ? ~0ull : (hh == (L >> 6) ? ((1ull << (L & 63)) - 1ull) : 0ull);
              r += __popcll(g_bl[hh] & lead_below);
              const uint64_t slot_below = hh < h ? ~0ull : (hh == h ? lmlt : 0ull);
              first = first && (lmk[h][hh] & g_mem[hh] & slot_below) == 0ull;
            }
            brow_g[h] = r;
            bown[h] = first;
          }
        }
      }
    };
    const auto open_group = [&](int a) __attribute__((always_inline)) {
      close_group();
      ++g;
#pragma unroll
      for (int h = 0; h < SPL; ++h) {
        if (h == (g >> 6) && lane == (g & 63)) gch0[h] = chn;
        g_bl[h] = g_mem[h] = 0ull;
      }
      g_rows = 0;
      g_arcs = 0;
      g_beams = 0;
      if (a > kLmStage) status |= 4u;  // a single chain above the staging limit (the builders prevent it)
    };
    // the beams sub join the open group with LM row srow (filled by beam
    // (hs, js) when the row is new) and bring the lists nl
    const auto place = [&](const uint64_t (&sub)[SPL], const uint64_t (&nl)[SPL], int srow, bool newrow, int hs,
                           int js) __attribute__((always_inline)) {
      int before = 0;  // members in the lower register sets
#pragma unroll
      for (int h = 0; h < SPL; ++h) {
        if ((sub[h] >> j) & 1ull) {
          const int inq = before + __popcll(sub[h] & lmlt);
          lpos[h] = pos + inq;
          cid[h] = chn + (g_beams + inq) / KCR;
          grp[h] = g;
          lrow_g[h] = srow;
          lown[h] = newrow && h == hs && j == js;
        }
        before += __popcll(sub[h]);
        g_mem[h] |= sub[h];
        g_bl[h] |= nl[h];
      }
      g_beams += before;
      pos += before;
    };
    while (any(rem)) {  // uniform: one LM state a pass
      const int hs = low_set(rem);
      int js = 0, a = 0;
      uint32_t sk = 0u;
#pragma unroll
      for (int h = 0; h < SPL; ++h) {
        if (h == hs) {
          js = static_cast<int>(__builtin_ctzll(rem[h]));
          sk = rdlane(lk[h], js);
          a = rdlane(ac[h], js);
        }
      }
      uint64_t smem[SPL], sl[SPL];
      int nsl = 0, nu = 0;
#pragma unroll
      for (int h = 0; h < SPL; ++h) {
        smem[h] = __ballot(nal[h] && lk[h] == sk);
        rem[h] &= ~smem[h];
      }
      // the state's lists, by leader
#pragma unroll
      for (int h = 0; h < SPL; ++h) {
        bool pres = false;
#pragma unroll
        for (int hh = 0; hh < SPL; ++hh) pres = pres || (lmk[h][hh] & smem[hh]) != 0ull;
        sl[h] = __ballot(lead[h] && pres);
        nsl += __popcll(sl[h]);
        nu += __popcll(sl[h] | g_bl[h]);
      }
      if (nsl <= KCR - 1) {  // uniform: the whole state joins one group
        if (!(g >= 0 && g_rows < KSEG && g_arcs + a <= kLmStage && nu <= KCR - 1)) open_group(a);
        const int srow = g_rows++;
        g_arcs += a;
        place(smem, sl, srow, true, hs, js);
      } else {
        // the state's lists exceed a group: one list a pass (beams without a
        // list with the lowest slot's pass)
        int srow = -1;
        while (any(smem)) {  // uniform
          const int hb = low_set(smem);
          int jb = 0, L = 0;
          bool lb = false;
#pragma unroll
          for (int h = 0; h < SPL; ++h) {
            if (h == hb) {
              jb = static_cast<int>(__builtin_ctzll(smem[h]));
              lb = ((hbm[h] >> jb) & 1ull) != 0ull;
              L = rdlane(bl[h], jb);
            }
          }
          uint64_t sub[SPL], nl[SPL];
          bool newl = false;
          int nb = 0;
#pragma unroll
          for (int hh = 0; hh < SPL; ++hh) {
            uint64_t mk = 0ull;
#pragma unroll
            for (int h = 0; h < SPL; ++h)
              if (h == hb) mk = rd64(lmk[h][hh], jb);
            sub[hh] = smem[hh] & (lb ? mk : ~hbm[hh]);
            nl[hh] = (lb && hh == (L >> 6)) ? (1ull << (L & 63)) : 0ull;
            newl = newl || (nl[hh] & ~g_bl[hh]) != 0ull;
            nb += __popcll(g_bl[hh]);
          }
          const bool fits = g >= 0 && (srow >= 0 || (g_rows < KSEG && g_arcs + a <= kLmStage)) &&
                            (!newl || nb < KCR - 1);
          if (!fits) {
            open_group(a);
            srow = -1;
          }
          const bool newrow = srow < 0;
          if (newrow) {
            srow = g_rows++;
            g_arcs += a;
          }
          place(sub, nl, srow, newrow, hb, jb);
#pragma unroll
          for (int hh = 0; hh < SPL; ++hh) smem[hh] &= ~sub[hh];
        }
      }
    }
    close_group();
    nch = chn;
    ngrp = g + 1;
  };
  int rcur = 0;  // s_rec buffer holding the current beam
  // record helpers
  auto load_rec = [&](const uint32_t* src, uint32_t (&r)[RW]) {
    src = static_cast<const uint32_t*>(__builtin_assume_aligned(src, 16));
#pragma unroll
    for (int w4 = 0; w4 < RW; w4 += 4) {
      const uint4 v = *reinterpret_cast<const uint4*>(src + w4);
      r[w4] = v.x;
      r[w4 + 1] = v.y;
      r[w4 + 2] = v.z;
      r[w4 + 3] = v.w;
    }
  };
  auto store_rec = [&](uint32_t* dst, const uint32_t (&r)[RW]) {
    dst = static_cast<uint32_t*>(__builtin_assume_aligned(dst, 16));
#pragma unroll
    for (int w4 = 0; w4 < RW; w4 += 4) *reinterpret_cast<uint4*>(dst + w4) = make_uint4(r[w4], r[w4 + 1], r[w4 + 2], r[w4 + 3]);
  };
  // repeat-scoring variant: the terms of an emitted token into its record
  auto put_terms = [&](uint32_t* dst, float2 inc) __attribute__((always_inline)) {
    dst[kRRal] = __float_as_uint(inc.x);
    dst[kRRwb] = __float_as_uint(inc.y);
  };
  // Successor of a selected candidate (flat index idx, resolved LM target,
  // boosting key) from its parent's record.  succ_begin reads the parent and
  // starts the chain-header loads of an emitted token; succ_end builds the
  // record in every lane (branch-free, so the loads stay where they were
  // issued) and the caller stores it for the winners.
  struct Succ {
    uint32_t par, lmt, btk;
    int c;
    bool emit;
    uint32_t r[RW];
    LmLevel hh[NLA];
    BtNode nd;
  };
  auto succ_begin = [&](bool act, uint32_t idx, uint32_t lmt, uint32_t btk, const uint32_t* prec, Succ& sp) __attribute__((always_inline)) {
    sp.par = act ? idx / static_cast<uint32_t>(W) : 0u;
    sp.c = act ? static_cast<int>(idx - sp.par * static_cast<uint32_t>(W)) : V;
    sp.lmt = lmt;
    sp.btk = btk;
    load_rec(prec + sp.par * RW, sp.r);
    sp.emit = act && sp.c != V && sp.c != static_cast<int>(sp.r[kRLast]);
#pragma unroll
    for (int l = 0; l < NL; ++l)
      sp.hh[l] = p.lm_states[static_cast<size_t>(sp.emit ? lmt : p.lm_bos_state) * NL + l];
    sp.nd = BtNode{0u, 0u, 0u, 0u};
    if (HAS_BT) sp.nd = p.bt_nodes[sp.emit ? (btk & kBtChildMask) : 0u];
  };
  auto succ_end = [&](Succ& sp, uint32_t xbits) __attribute__((always_inline)) {
    uint32_t* r = sp.r;
    const bool e = sp.emit;
    uint64_t h = (static_cast<uint64_t>(r[kRHhi]) << 32) | r[kRHlo];
    const uint64_t hm = mix_token(h, static_cast<uint32_t>(sp.c));
    h = e ? hm : h;
    r[kRX] = xbits;
    r[kRBp] = (sp.par << 16) | static_cast<uint32_t>(sp.c);
    r[kRHlo] = static_cast<uint32_t>(h);
    r[kRHhi] = static_cast<uint32_t>(h >> 32);
    r[kRLen] += e ? 1u : 0u;
    r[kRLast] = static_cast<uint32_t>(sp.c);
    if (HAS_LM) r[kRLms] = e ? sp.lmt : r[kRLms];
    if (HAS_BT) r[kRBts] = e ? (sp.btk & kBtChildMask) : r[kRBts];
    r[kREmit] = e ? 1u : 0u;
    if (HAS_BT) {
      r[kRBtb] = e ? sp.nd.list_begin : r[kRBtb];
      r[kRBtc] = e ? sp.nd.list_count : r[kRBtc];
      r[kRBtp] = e ? (sp.nd.pot & 0xFFu) : r[kRBtp];
    }
#pragma unroll
    for (int l = 0; l < NL; ++l) {
      r[kRLvb + l] = e ? sp.hh[l].begin : r[kRLvb + l];
      r[kRLvc + l] = e ? sp.hh[l].count : r[kRLvc + l];
      r[kRLvbo + l] = e ? __float_as_uint(sp.hh[l].bo) : r[kRLvbo + l];
    }
  };

  for (int i = tid; i < kOffTgt; i += kThreads) s_big[i] = 0u;
  for (int i = tid; i < (KMX + 16) * kRowWords; i += kThreads) s_row[i] = 0u;
  if constexpr (REP)
    for (int i = tid; i < 2 * KMX; i += kThreads) s_rinc[i / KMX][i % KMX] = make_float2(0.0f, 0.0f);
  __syncthreads();
  if (tid == 0) {
    put_row(0, 0);
    // record of the initial beam (slot 0)
    uint32_t r[RW];
#pragma unroll
    for (int w = 0; w < RW; ++w) r[w] = 0u;
    r[kRLast] = static_cast<uint32_t>(V);
    r[kRLms] = HAS_LM ? p.lm_bos_state : 0u;
    if (HAS_BT) {
      r[kRBtb] = btb[0];
      r[kRBtc] = btc[0];
      r[kRBtp] = static_cast<uint32_t>(btpot[0]);
    }
#pragma unroll
    for (int l = 0; l < NL; ++l) {
      r[kRLvb + l] = lvb[0][l];
      r[kRLvc + l] = lvc[0][l];
      r[kRLvbo + l] = __float_as_uint(lvbo[0][l]);
    }
    store_rec(s_rec, r);
    s_nbuf = 0;
    s_overflow = 0;
    if (want_stats) {
      // the initial beam's chain is scanned in frame 0
      unsigned long long ns = 0, na = 0;
#pragma unroll
      for (int l = 0; l < NL; ++l) {
        if (L > 0 && (lvc[0][l] & kExists)) {
          ns += 1;
          na += lvc[0][l] & ~kExists;
        }
      }
      s_st[0] = L > 0 ? 1 : 0;
      s_st[1] = ns;
      s_st[2] = na;
      s_st[3] = 0;
      s_st[4] = 0;
      s_st[5] = 0;
    }
  }
  uint32_t gen = 0u;
  int mpar = 0;  // reserved region holding the pool's reserved entries
  __syncthreads();
#ifdef CTCBEAM_PHASE_CLOCKS
  uint64_t ph_acc = 0ull;
  uint64_t ph_t0 = __builtin_amdgcn_s_memtime();
#endif

  for (int t = 0; t < L; ++t) {
    // ---- rotate and prefetch the log-prob row ----
#pragma unroll
    for (int jj = 0; jj < LPT; ++jj) rD[jj] = rDn[jj];
    rBlank = rBlankN;
    if (t + 1 < L) {
      const float* rowp = Db + static_cast<size_t>(t + 1) * W;
#pragma unroll
      for (int jj = 0; jj < LPT; ++jj) {
        const int c = tid + jj * kThreads;
        if (c < V) rDn[jj] = __builtin_nontemporal_load(rowp + c);
      }
      if (lane < K) rBlankN = __builtin_nontemporal_load(rowp + V);
    }
    float tau_run = kNegInf;
    float gacc = kNegInf;  // top 64 group maxima of the frame's chunks so far (K > 8)
    float gacc_hi = kNegInf;  // two slots per lane: positions 64..127 of the top 128
    int nfin = 0;
    // survivors carried in the pool from chunks whose rank was skipped
    int carry = 0;
    int cs = 0;  // live position of the chunk's first beam
    int gi = 0;  // next fill group (kGroups)

    for (int ch = 0; ch < nch; ++ch) {
      // this chunk's beams and their key rows (slot order)
      bool inch[SPL];
      int row[SPL];
      int kc = 0;
      if constexpr (SPL == 1) {
        inch[0] = alive[0] && (cid[0] == ch);
        const uint64_t chmask = __ballot(inch[0]);
        kc = __popcll(chmask);
        row[0] = __popcll(chmask & lmlt);
      } else {
#pragma unroll
        for (int h = 0; h < SPL; ++h) {
          inch[h] = alive[h] && (cid[h] == ch);
          const uint64_t chmask = __ballot(inch[h]);
          row[h] = kc + __popcll(chmask & lmlt);
          kc += __popcll(chmask);
        }
      }

      // ---- F. fill the key rows of this chunk (of its group) ----
      // kGroups: only a group's first chunk fills (uniform)
      bool gfill = !kGroups;
      if constexpr (kGroups) {
#pragma unroll
        for (int h = 0; h < SPL; ++h)
          if (h == (gi >> 6)) gfill = gi < ngrp && ch == rdlane(gch0[h], gi & 63);
      }
      if (gfill) {  // uniform
        if (gen == kGenMax) {
          // rows were last read before the previous filter barrier
          for (int i = tid; i < kOffTgt; i += kThreads) s_big[i] = 0u;
          __syncthreads();
          gen = 0u;
        }
        ++gen;
      }
      const uint32_t genhi = gen << kGenShift;
      if (gfill) {  // uniform
      if (HAS_LM && NL > 0) {
        // Segment table, lane s = segment s: the non-empty (beam, level) arc
        // runs of the chunk, level-major.  The chunk's arcs are numbered by
        // their position in this concatenation, which is also their staging
        // slot.  Fields: arc base, row | level << 8, and the backoff weights
        // an arc of that level adds (bo of the levels above, then zeros).
        int S = 0;
        uint32_t sg_cnt = 0u, sg_base = 0u, sg_rl = 0u;
        float sg_f[NF];
#pragma unroll
        for (int k = 0; k < NF; ++k) sg_f[k] = 0.0f;
#pragma unroll
        for (int l = 0; l < NL; ++l) {
#pragma unroll
          for (int h = 0; h < SPL; ++h) {
            // the beams that fill an LM row (the row's first with fill groups)
            const bool fsel = CACHE ? fillrep : kGroups ? (alive[h] && grp[h] == gi && lown[h]) : inch[h];
            const uint32_t n = fsel ? (lvc[h][l] & ~kExists) : 0u;
            const uint64_t m = __ballot(n != 0u);
            const int nl = __popcll(m);
            if (nl > 0) {  // wave-uniform
              // senders push to their segment lane; the rest to a lane outside
              // [S, S + nl) (S + nl <= 64)
              const int dst = (n != 0u) ? S + __popcll(m & lmlt) : ((S + nl) & 63);
              const int addr = dst << 2;
              const uint32_t r_cnt = static_cast<uint32_t>(__builtin_amdgcn_ds_permute(addr, static_cast<int>(n)));
              const uint32_t r_base =
                  static_cast<uint32_t>(__builtin_amdgcn_ds_permute(addr, static_cast<int>(lvb[h][l])));
              const uint32_t r_rl =
                  static_cast<uint32_t>(__builtin_amdgcn_ds_permute(addr, (CACHE ? rowof : kGroups ? lrow_g[h] : row[h]) | (l << 8)));
              float r_f[NF];
#pragma unroll
              for (int k = 0; k + 1 < NL; ++k) {
                const int lk = l + 1 + k;
                const float fk = lk < NL ? lvbo[h][lk < NLA ? lk : 0] : 0.0f;
                r_f[k] = __int_as_float(__builtin_amdgcn_ds_permute(addr, __float_as_int(fk)));
              }
              if (lane >= S && lane < S + nl) {
                sg_cnt = r_cnt;
                sg_base = r_base;
                sg_rl = r_rl;
#pragma unroll
                for (int k = 0; k + 1 < NL; ++k) sg_f[k] = r_f[k];
              }
              S += nl;
            }
          }
        }
        if constexpr (!CACHE && kFoldRows) {
          // every token of every row of the chunk gets its unigram + backoff
          // fold as an order-0 entry holding the token (its unigram state);
          // the explicit arcs (order >= 1) win the maximum
#pragma unroll
          for (int h = 0; h < SPL; ++h) {
            uint64_t fm = __ballot(kGroups ? (alive[h] && grp[h] == gi && lown[h]) : inch[h]);
            while (fm != 0ull) {  // uniform
              const int jr = static_cast<int>(__builtin_ctzll(fm));
              fm &= fm - 1ull;
              const uint32_t rf = rdlane(static_cast<uint32_t>(kGroups ? lrow_g[h] : row[h]), jr);
              float bo[NLA];
#pragma unroll
              for (int l = 0; l < NL; ++l) bo[l] = rdlane(lvbo[h][l], jr);
#pragma unroll
              for (int jj = 0; jj < LPT; ++jj) {
                if (tid + jj * kThreads < V) {
                  float v = rP1[jj];
#pragma unroll
                  for (int l = 0; l < NL; ++l) v = v + bo[l];
                  const float av = alpha * v;
                  atomicMax(reinterpret_cast<unsigned long long*>(&lmrow[rf * static_cast<uint32_t>(V) + rcc[jj]]),
                            (static_cast<unsigned long long>(genhi | rcc[jj]) << 32) | __float_as_uint(av));
                }
              }
            }
          }
        }
        if constexpr (CACHE) {
          // every token of a new row gets its unigram + backoff fold as an
          // order-0 entry (the explicit arcs, order >= 1, win the maximum),
          // so the scoring reads one entry per token and nothing else
          uint64_t fm = __ballot(fillrep);
          while (fm != 0ull) {  // uniform
            const int jr = static_cast<int>(__builtin_ctzll(fm));
            fm &= fm - 1ull;
            const uint32_t rf = rdlane(static_cast<uint32_t>(rowof), jr);
            float bo[NLA];
#pragma unroll
            for (int l = 0; l < NL; ++l) bo[l] = rdlane(lvbo[0][l], jr);
#pragma unroll
            for (int jj = 0; jj < LPT; ++jj) {
              if (tid + jj * kThreads < V) {
                float v = rP1[jj];
#pragma unroll
                for (int l = 0; l < NL; ++l) v = v + bo[l];
                const float av = alpha * v;
                atomicMax(reinterpret_cast<unsigned long long*>(&lmrow[rf * static_cast<uint32_t>(V) + rcc[jj]]),
                          (static_cast<unsigned long long>(genhi | rcc[jj]) << 32) | __float_as_uint(av));
              }
            }
          }
        }
        // tiles of 64 arcs never straddle segments: a tile's segment is one
        // ballot away and its fields are wave-uniform (readlane)
        if (!CACHE || S > 0) {  // uniform; cached rows often need no fill
        const int sincl = wave_incl_scan(static_cast<int>(sg_cnt), lane);
        const uint32_t sstart = static_cast<uint32_t>(sincl) - sg_cnt;  // staging slot of the first arc
        const int stl = static_cast<int>((sg_cnt + 63u) >> 6);
        const int tincl = wave_incl_scan(stl, lane);
        const int texcl = tincl - stl;
        const int ntile = rdlane(tincl, 63);
        for (int t0 = wave; t0 < ntile; t0 += kWaves * kLmTU) {
          LmArc a[kLmTU];
          uint32_t apos[kLmTU], arl[kLmTU];
          float af[kLmTU][NF];
#pragma unroll
          for (int u = 0; u < kLmTU; ++u) {
            const int tt = t0 + u * kWaves;
            apos[u] = 0xFFFFFFFFu;
            arl[u] = 0u;
            a[u].token = 0xFFFFFFFFu;
            if (tt < ntile) {  // wave-uniform
              const int sg = __popcll(__ballot(tincl <= tt));
              const uint32_t qs = (static_cast<uint32_t>(tt - rdlane(texcl, sg)) << 6) + static_cast<uint32_t>(lane);
              const bool ok = qs < rdlane(sg_cnt, sg);
              apos[u] = ok ? rdlane(sstart, sg) + qs : 0xFFFFFFFFu;
              arl[u] = rdlane(sg_rl, sg);
#pragma unroll
              for (int k = 0; k + 1 < NL; ++k) af[u][k] = rdlane(sg_f[k], sg);
              a[u] = p.lm_arcs[rdlane(sg_base, sg) + (ok ? qs : 0u)];
            }
          }
#pragma unroll
          for (int u = 0; u < kLmTU; ++u) {
            const uint32_t q = apos[u];
            // positions past a segment's arcs (and tiles past the last) skip
            if (q != 0xFFFFFFFFu && a[u].token < static_cast<uint32_t>(V)) {
              float v = a[u].logp;
#pragma unroll
              for (int k = 0; k + 1 < NL; ++k) v = v + af[u][k];
              const float av = alpha * v;
              uint32_t hi = genhi | (((arl[u] >> 8) + 1u) << 23);
              if constexpr (CACHE) {
                hi |= a[u].target;  // below 2^23
              } else {
                tgt[q] = a[u].target;
                hi |= q;
              }
              atomicMax(reinterpret_cast<unsigned long long*>(&lmrow[(arl[u] & 0xFFu) * V + a[u].token]),
                        (static_cast<unsigned long long>(hi) << 32) | __float_as_uint(av));
            }
          }
        }
        }
      }
      if (HAS_BT) {
        // same scheme, one segment per beam (its merged continuation list)
        int S = 0;
        uint32_t bg_cnt = 0u, bg_base = 0u, bg_row = 0u;
#pragma unroll
        for (int h = 0; h < SPL; ++h) {
          // the beams that fill a boosting row (the list's first with fill groups)
          const bool bsel = kGroups ? (alive[h] && grp[h] == gi && bown[h]) : inch[h];
          const uint32_t nb = bsel ? btc[h] : 0u;
          const uint64_t m = __ballot(nb != 0u);
          const int nl = __popcll(m);
          if (nl > 0) {  // wave-uniform
            const int dst = (nb != 0u) ? S + __popcll(m & lmlt) : ((S + nl) & 63);
            const int addr = dst << 2;
            const uint32_t r_cnt = static_cast<uint32_t>(__builtin_amdgcn_ds_permute(addr, static_cast<int>(nb)));
            const uint32_t r_base = static_cast<uint32_t>(__builtin_amdgcn_ds_permute(addr, static_cast<int>(btb[h])));
            const uint32_t r_row = static_cast<uint32_t>(__builtin_amdgcn_ds_permute(addr, kGroups ? brow_g[h] : row[h]));
            if (lane >= S && lane < S + nl) {
              bg_cnt = r_cnt;
              bg_base = r_base;
              bg_row = r_row;
            }
            S += nl;
          }
        }
        if (S > 0) {  // wave-uniform
          const int btl = static_cast<int>((bg_cnt + 63u) >> 6);
          const int tincl = wave_incl_scan(btl, lane);
          const int texcl = tincl - btl;
          const int ntile = rdlane(tincl, 63);
          for (int t0 = wave; t0 < ntile; t0 += kWaves * kBtTU) {
            BtEntry e[kBtTU];
            uint32_t erow[kBtTU];
            bool eok[kBtTU];
#pragma unroll
            for (int u = 0; u < kBtTU; ++u) {
              const int tt = t0 + u * kWaves;
              erow[u] = 0u;
              eok[u] = false;
              e[u].token = 0xFFFFFFFFu;
              if (tt < ntile) {  // wave-uniform
                const int sg = __popcll(__ballot(tincl <= tt));
                const uint32_t qs = (static_cast<uint32_t>(tt - rdlane(texcl, sg)) << 6) + static_cast<uint32_t>(lane);
                eok[u] = qs < rdlane(bg_cnt, sg);
                erow[u] = rdlane(bg_row, sg);
                e[u] = p.bt_list[rdlane(bg_base, sg) + (eok[u] ? qs : 0u)];
              }
            }
#pragma unroll
            for (int u = 0; u < kBtTU; ++u)
              if (eok[u] && e[u].token < static_cast<uint32_t>(V))
                btrow[erow[u] * V + e[u].token] = (e[u].key & kLowMask) | genhi;
          }
        }
      }
      CTCBEAM_PHASE_MARK(0);
      __syncthreads();  // A: rows complete
      CTCBEAM_PHASE_MARK(1);
      if constexpr (kGroups) ++gi;
      }

      // ---- C. candidates ----
      // chunk row i is live position cs + i; its beam record is read with
      // broadcast LDS loads so the scoring is straight-line code
      int kslot[KCR];
      float ksc[KCR];
      int klast[KCR];
      float kbo[KCR][NLA];  // backoff weights (rows without the fold)
      int kpot[KCR];
      // LM key row and boosting row of chunk row i
      uint32_t krow[KCR], kbrow[KCR];
#pragma unroll
      for (int i = 0; i < KCR; ++i) {
        const uint32_t* rr = s_row + (cs + i) * kRowWords;
        const uint4 h0 = *reinterpret_cast<const uint4*>(rr);
        ksc[i] = (i < kc) ? __uint_as_float(h0.x) : kNegInf;
        klast[i] = static_cast<int>(h0.y);
        // (uniform: fill groups keep the fields in scalar registers)
        const uint32_t hz = kGroups ? __builtin_amdgcn_readfirstlane(h0.z) : h0.z;
        kslot[i] = static_cast<int>((CACHE || kGroups) ? (hz & 0xFFu) : hz);
        krow[i] = (CACHE || kGroups) ? ((hz >> 8) & 0xFFu) : static_cast<uint32_t>(i);
        kbrow[i] = kGroups ? ((hz >> 16) & 0xFFu) : static_cast<uint32_t>(i);
        kpot[i] = static_cast<int>(kGroups ? __builtin_amdgcn_readfirstlane(h0.w) : h0.w);
#pragma unroll
        for (int l0 = 0; l0 < (kFoldRows ? 0 : NL); l0 += 4) {
          const uint4 h = *reinterpret_cast<const uint4*>(rr + 4 + l0);
          const uint32_t hv[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (l0 + q < NL) kbo[i][(l0 + q) < NLA ? (l0 + q) : 0] = __uint_as_float(hv[q]);
        }
      }
      float cand[NC];
      // without boosting the LM entries of the candidates fit in registers;
      // with it they are re-read from the rows for the survivors
      constexpr bool kKeepLm = HAS_LM && !HAS_BT;
      uint32_t lhi[kKeepLm ? NC : 1];
      float lmax = kNegInf;
      float rmax[KCR];  // per chunk row: maximum over this lane's labels
      if constexpr (kGroups) {
        // Fill groups: the beams of an LM state are adjacent, so a row in the
        // state of the row before reads the same LM terms, and a row with the
        // same boosting row and pot the same boosting terms; they are kept
        // from that row rather than read and folded again (uniform branches).
        float avk[LPT], bvk[LPT];
        uint32_t lhk[LPT];
#pragma unroll
        for (int jj = 0; jj < LPT; ++jj) {
          avk[jj] = 0.0f;
          bvk[jj] = 0.0f;
          lhk[jj] = 0u;
        }
#pragma unroll
        for (int i = 0; i < KCR; ++i) {
          const bool lm_new = i == 0 || krow[i] != krow[i > 0 ? i - 1 : 0];
          const bool bt_new = i == 0 || kbrow[i] != kbrow[i > 0 ? i - 1 : 0] || kpot[i] != kpot[i > 0 ? i - 1 : 0];
          if (HAS_LM && lm_new) {
#pragma unroll
            for (int jj = 0; jj < LPT; ++jj) {
              // LM entry: the row this beam reads (its state's row in the group)
              const uint32_t el = krow[i] * static_cast<uint32_t>(V) + rcc[jj];
              const uint64_t ent = lmrow[el];
              const uint32_t hi = static_cast<uint32_t>(ent >> 32);
              if constexpr (kFoldRows) {
                // the chunk's rows hold every token: the fold (order 0, the
                // token) or an explicit arc (its staging slot, resolved later)
                avk[jj] = __uint_as_float(static_cast<uint32_t>(ent));
                lhk[jj] = hi;
              } else {
                float v = rP1[jj];
#pragma unroll
                for (int l = 0; l < NL; ++l) v = v + kbo[i][l];
                const bool has = hi >= genhi;
                avk[jj] = has ? __uint_as_float(static_cast<uint32_t>(ent)) : alpha * v;
                // the LM target: an explicit arc's staging slot (resolved
                // later), or the token's unigram state
                lhk[jj] = has ? hi : rcc[jj];
              }
            }
          }
          if (HAS_BT && bt_new) {
#pragma unroll
            for (int jj = 0; jj < LPT; ++jj) {
              const uint32_t be = btrow[kbrow[i] * static_cast<uint32_t>(V) + rcc[jj]];
              const uint32_t bk = (be >= genhi) ? be : rRoot[jj];
              const int pre = static_cast<int>((bk >> 20) & 63u);
              bvk[jj] = boost_w * static_cast<float>(pre - kpot[i]);
            }
          }
#pragma unroll
          for (int jj = 0; jj < LPT; ++jj) {
            const int r = i * LPT + jj;
            const int c = tid + jj * kThreads;
            const float x0 = ksc[i] + rD[jj];
            float x1 = x0 + beta;
            if (HAS_LM) {
              x1 = x1 + avk[jj];
              if constexpr (kKeepLm) lhi[r] = lhk[jj];
            }
            if (HAS_BT) x1 = x1 + bvk[jj];
            const float x = (c != klast[i]) ? x1 : x0;
            cand[r] = x;
            rmax[i] = jj == 0 ? x : fmaxf(rmax[i], x);
          }
          lmax = fmaxf(lmax, rmax[i]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < KCR; ++i) {
#pragma unroll
          for (int jj = 0; jj < LPT; ++jj) {
            const int r = i * LPT + jj;
            const int c = tid + jj * kThreads;
            const uint32_t e = static_cast<uint32_t>(i * V) + rcc[jj];
            // LM entry: the row this beam reads (shared with its state's first beam)
            const uint32_t el = kGroups ? krow[i] * static_cast<uint32_t>(V) + rcc[jj] : e;
            const float x0 = ksc[i] + rD[jj];
            float x1 = x0 + beta;
            if (HAS_LM) {
              if constexpr (CACHE) {
                // a cached row holds every token: the fold or the arc, with
                // the LM target state
                const uint64_t ent = lmrow[krow[i] * static_cast<uint32_t>(V) + rcc[jj]];
                x1 = x1 + __uint_as_float(static_cast<uint32_t>(ent));
                lhi[r] = static_cast<uint32_t>(ent >> 32) & kTargetMask;
              } else if constexpr (kFoldRows) {
                // the chunk's rows hold every token: the fold (order 0, the
                // token) or an explicit arc (its staging slot, resolved later)
                const uint64_t ent = lmrow[el];
                x1 = x1 + __uint_as_float(static_cast<uint32_t>(ent));
                if constexpr (kKeepLm) lhi[r] = static_cast<uint32_t>(ent >> 32);
              } else {
                const uint64_t ent = lmrow[el];
                const uint32_t hi = static_cast<uint32_t>(ent >> 32);
                float v = rP1[jj];
#pragma unroll
                for (int l = 0; l < NL; ++l) v = v + kbo[i][l];
                const bool has = hi >= genhi;
                const float av = has ? __uint_as_float(static_cast<uint32_t>(ent)) : alpha * v;
                x1 = x1 + av;
                // the LM target: an explicit arc's staging slot (resolved
                // later), or the token's unigram state
                if constexpr (kKeepLm) lhi[r] = has ? hi : rcc[jj];
              }
            }
            if (HAS_BT) {
              const uint32_t be = btrow[kGroups ? kbrow[i] * static_cast<uint32_t>(V) + rcc[jj] : e];
              const uint32_t bk = (be >= genhi) ? be : rRoot[jj];
              const int pre = static_cast<int>((bk >> 20) & 63u);
              const float bv = boost_w * static_cast<float>(pre - kpot[i]);
              x1 = x1 + bv;
            }
            const float x = (c != klast[i]) ? x1 : x0;
            cand[r] = x;
            rmax[i] = jj == 0 ? x : fmaxf(rmax[i], x);
          }
          lmax = fmaxf(lmax, rmax[i]);
        }
      }
      if constexpr (rep) {
        // repeat-scoring variant: the repeat of a live row's last label (a
        // token) adds the terms that token got when it was emitted, read
        // from the slot's record; the maxima are taken again
        const uint32_t* prc = s_rec + rcur * (KMX * RW);
        lmax = kNegInf;
#pragma unroll
        for (int i = 0; i < KCR; ++i) {
          const uint32_t* rr = prc + (static_cast<uint32_t>(kslot[i]) & (KMX - 1)) * RW;
          const float ral = __uint_as_float(rr[kRRal]), rwb = __uint_as_float(rr[kRRwb]);
#pragma unroll
          for (int jj = 0; jj < LPT; ++jj) {
            const int r = i * LPT + jj;
            const int c = tid + jj * kThreads;
            if (i < kc && c < V && c == klast[i]) {
              float x = cand[r];
              if (HAS_LM) x = x + ral;
              if (HAS_BT) x = x + rwb;
              cand[r] = x;
            }
            rmax[i] = jj == 0 ? cand[r] : fmaxf(rmax[i], cand[r]);
          }
          lmax = fmaxf(lmax, rmax[i]);
        }
      }
      // The (fl(alpha*LM), fl(w*BT)) terms of candidate (chunk row i, label
      // c) as the scoring formed them, from this chunk's rows, for the
      // repeat-scoring variant (run-time i and c; kc rows of the chunk).
      const auto cand_terms = [&](uint32_t i, uint32_t c, uint32_t row) __attribute__((always_inline)) {
        float av = 0.0f, bv = 0.0f;
        const uint32_t e = i * static_cast<uint32_t>(V) + c;
        const uint32_t* rr = s_row + (static_cast<uint32_t>(cs) + i) * kRowWords;
        if (HAS_LM) {
          if constexpr (CACHE) {
            av = __uint_as_float(static_cast<uint32_t>(lmrow[row * static_cast<uint32_t>(V) + c]));
          } else if constexpr (kFoldRows) {
            const uint32_t el = kGroups ? ((rr[2] >> 8) & 0xFFu) * static_cast<uint32_t>(V) + c : e;
            av = __uint_as_float(static_cast<uint32_t>(lmrow[el]));
          } else {
            const uint32_t el = kGroups ? ((rr[2] >> 8) & 0xFFu) * static_cast<uint32_t>(V) + c : e;
            const uint64_t ent = lmrow[el];
            if (static_cast<uint32_t>(ent >> 32) >= genhi) {
              av = __uint_as_float(static_cast<uint32_t>(ent));
            } else {
              float v = p.lm_unigram[c];
#pragma unroll
              for (int l = 0; l < NL; ++l) v = v + __uint_as_float(rr[4 + l]);
              av = alpha * v;
            }
          }
        }
        if (HAS_BT) {
          const uint32_t be = btrow[kGroups ? ((rr[2] >> 16) & 0xFFu) * static_cast<uint32_t>(V) + c : e];
          const uint32_t bk = (be >= genhi) ? be : p.bt_root_key[c];
          bv = boost_w * static_cast<float>(static_cast<int>((bk >> 20) & 63u) - static_cast<int>(rr[3]));
        }
        return make_float2(av, bv);
      };
      // the same for a candidate of this chunk named by its flat index: its
      // chunk row is the live position of its slot
      const auto terms_of_flat = [&](uint32_t flat) __attribute__((always_inline)) {
        const uint32_t slot = flat / static_cast<uint32_t>(W), c = flat - slot * static_cast<uint32_t>(W);
        uint32_t i = 0u, row = 0u;
#pragma unroll 1
        for (int q = 0; q < kc; ++q) {
          const uint32_t z = s_row[(cs + q) * kRowWords + 2];
          if (((CACHE || kGroups) ? (z & 0xFFu) : z) == slot) {
            i = static_cast<uint32_t>(q);
            row = (z >> 8) & 0xFFu;
          }
        }
        return cand_terms(i, c, row);
      };
      // LM entry (staged, or the token's unigram state) and boosting key of
      // candidate (i, jj), re-read from the rows for the few that are kept
      // rather than held in registers from the scoring
      auto cand_meta = [&](int i, int jj, uint32_t& lraw, uint32_t& bk) __attribute__((always_inline)) {
        const uint32_t e = static_cast<uint32_t>(i * V) + rcc[jj];
        lraw = 0u;
        bk = 0u;
        if (HAS_LM) {
          if constexpr (CACHE) {
            lraw = static_cast<uint32_t>(lmrow[krow[i] * static_cast<uint32_t>(V) + rcc[jj]] >> 32) & kTargetMask;
          } else {
            const uint32_t el = kGroups ? krow[i] * static_cast<uint32_t>(V) + rcc[jj] : e;
            const uint32_t hi = static_cast<uint32_t>(lmrow[el] >> 32);
            lraw = (kFoldRows || hi >= genhi) ? hi : rcc[jj];
          }
        }
        if (HAS_BT) {
          const uint32_t be = btrow[kGroups ? kbrow[i] * static_cast<uint32_t>(V) + rcc[jj] : e];
          bk = (be >= genhi) ? be : rRoot[jj];
        }
      };
      if (SPL == 1 && ch == 0 && wave == 0 && lane < K) {
        // blank candidates of every slot into the reserved region
        const float x = sc[0] + rBlank;
        const bool ok = sc[0] != kNegInf && x != kNegInf;
        s_res[mpar][j] = make_uint4(__float_as_uint(ok ? x : kNegInf),
                                    ok ? static_cast<uint32_t>(j * W + V) : 0xFFFFFFFFu, 0u, 0u);
      } else if (SPL > 1 && ch == 0 && wave == 0) {
#pragma unroll
        for (int h = 0; h < SPL; ++h) {
          const int js = j + 64 * h;
          if (js < K) {
            const float x = sc[h] + rBlank;
            const bool ok = sc[h] != kNegInf && x != kNegInf;
            s_res[mpar][js] = make_uint4(__float_as_uint(ok ? x : kNegInf),
                                         ok ? static_cast<uint32_t>(js * W + V) : 0xFFFFFFFFu, 0u, 0u);
          }
        }
      }
      if (tid == 0 && carry == 0) {
        s_nbuf = 0;  // the previous rank read it before barrier D
        s_overflow = 0;
      }
      // Maxima of disjoint candidate groups are distinct candidates, so the
      // K-th largest of at least K group maxima bounds the K-th best candidate
      // from below.  One slot per lane: groups (row, wave) of this chunk, and
      // for K <= 8 also (row, half of the waves) and the waves; the groups of
      // earlier chunks of the frame still count.  Two slots per lane: 128
      // groups of 4 lanes.
      if (SPL > 1) {
        float g = fmax_sel(lmax, xor_lane(lmax, 1, lane));
        g = fmax_sel(g, xor_lane(g, 2, lane));
        if ((lane & 3) == 3) s_top[wave * 16 + (lane >> 2)] = g;
      } else {
        // The wave maxima of 8 row groups (row i, and i + 8 when a chunk has
        // 16 rows): a transposed reduction halves the groups a lane carries
        // at each of the lane-bit steps 1, 2, 4, leaving lane l with group
        // 4(l&1) + 2(l>>1&1) + (l>>2&1), then reduces over lane bits 3..5.
        // K <= 8 also keeps the 8 wave maxima (the maximum of the 8 row
        // groups below).
        float m8[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          m8[i] = i < KCR ? rmax[i < KCR ? i : 0] : kNegInf;
          if (i + 8 < KCR) m8[i] = fmaxf(m8[i], rmax[i + 8 < KCR ? i + 8 : 0]);
        }
        const bool b0 = lane_in(0xAAAAAAAAAAAAAAAAull), b1 = lane_in(0xCCCCCCCCCCCCCCCCull), b2 = lane_in(kLanesBit2);
        float m4[4], m2[2];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          m4[q] = fmaxf(b0 ? m8[q + 4] : m8[q], xor_lane(b0 ? m8[q] : m8[q + 4], 1, lane));
#pragma unroll
        for (int q = 0; q < 2; ++q)
          m2[q] = fmaxf(b1 ? m4[q + 2] : m4[q], xor_lane(b1 ? m4[q] : m4[q + 2], 2, lane));
        float m1 = fmaxf(b2 ? m2[1] : m2[0], xor_lane(b2 ? m2[0] : m2[1], 4, lane));
        m1 = fmaxf(m1, xor_lane(m1, 8, lane));
        m1 = fmaxf(m1, xor_lane(m1, 16, lane));
        m1 = fmaxf(m1, xor_lane(m1, 32, lane));
        if (lane < 8) s_top[wave * 8 + lane] = m1;
        if (kSmallK || (kMaySmallK && K <= 8)) {
          float wm = fmaxf(m1, xor_lane(m1, 1, lane));
          wm = fmaxf(wm, xor_lane(wm, 2, lane));
          wm = fmaxf(wm, xor_lane(wm, 4, lane));
          if (lane == 0) s_top[kWaves * 8 + wave] = wm;
        }
      }
      // the blank candidates are exact: with K live slots the smallest blank
      // score also bounds the K-th best from below (registers only: small
      // beams take it before the barrier)
      const auto blank_bound = [&]() __attribute__((always_inline)) {
        float tb = (lane < K) ? sc[0] + rBlank : __builtin_huge_valf();
#pragma unroll
        for (int h = 1; h < SPL; ++h)
          if (j + 64 * h < K) tb = fmin_sel(tb, sc[h] + rBlank);
        tb = fmin_sel(tb, xor_lane(tb, 1, lane));
        tb = fmin_sel(tb, xor_lane(tb, 2, lane));
        tb = fmin_sel(tb, xor_lane(tb, 4, lane));
        if (K > 8) tb = fmin_sel(tb, xor_lane(tb, 8, lane));
        if (K > 16) tb = fmin_sel(tb, xor_lane(tb, 16, lane));
        if (K > 32) tb = fmin_sel(tb, xor_lane(tb, 32, lane));
        return rdlane(tb, 0);
      };
      float tblank = 0.0f;
      if constexpr (kSmallK) tblank = blank_bound();
      CTCBEAM_PHASE_MARK(2);
      __syncthreads();  // B: bound inputs, blanks, pool reset
      CTCBEAM_PHASE_MARK(3);

      // ---- T. bound and filter ----
      {
        float tc;
        if (kSmallK || (kMaySmallK && K <= 8)) {
          // two bounds sorted side by side in groups of 16 lanes: lanes 0..15
          // the maxima of (row, half of the waves), lanes 16..23 the wave
          // maxima
          float rw = s_top[lane];  // wave lane >> 3, row slot lane & 7
          const float wm = s_top[kWaves * 8 + (lane & 7)];
          rw = fmaxf(rw, xor_lane(rw, 8, lane));
          rw = fmaxf(rw, xor_lane(rw, 16, lane));  // lanes 0..31: waves 0..3, lanes 32..63: 4..7
          const float oh = xor_lane(rw, 32, lane);
          // plain selects (a nested conditional became branches, with the
          // wave-maxima read moved into one of them)
          float v = kNegInf;
          v = lane_in(0xFF0000ull) ? wm : v;
          v = lane_in(0xFF00ull) ? oh : v;
          v = lane_in(0xFFull) ? rw : v;
          // the K-th largest of each 16-lane row: the largest value with at
          // least K values of its row at or above it
          const float kv = row_max_last(row_ge_count(v) >= static_cast<uint32_t>(K) ? v : kNegInf);
          tc = fmaxf(rdlane(kv, 15), rdlane(kv, 31));
        } else if (SPL == 1) {
          // this chunk's 64 (row group, wave) maxima, sorted ascending, merged
          // into the frame's running top 64 (descending): the elementwise
          // maximum of the two is bitonic and holds the top 64 of the union
          // (without rank skipping each chunk's rank sets tau_run instead)
          // (a chunk none of whose maxima beats the K-th largest so far
          // leaves the top K as it is: no sort)
          const float kth = rdlane(gacc, K - 1);
          if (!SKIP || __ballot(s_top[lane] > kth) != 0ull) {  // uniform
            const float v = -wave_sort_desc<64>(-s_top[lane], lane);
            gacc = bitonic_merge<64, 64, 32>(fmaxf(SKIP ? gacc : kNegInf, v), lane);
          }
          tc = rdlane(gacc, K - 1);
        } else {
          // This chunk's 128 group maxima, sorted ascending, merged into the
          // frame's running top 128 (descending; positions 0..63 in gacc, 64..127
          // in gacc_hi), as for one slot per lane.  The ascending sort runs on
          // the negated values: the halves sorted descending and ascending
          // form a bitonic sequence, merged descending by one exchange
          // between the halves and a 64-lane merge in each.
          const float e0 = wave_sort_desc<64>(-s_top[lane], lane);
          const float f1 = -wave_sort_desc<64>(s_top[64 + lane], lane);
          const float n0 = -bitonic_merge<64, 64, 32>(fmaxf(e0, f1), lane);
          const float n1 = -bitonic_merge<64, 64, 32>(fminf(e0, f1), lane);
          // the elementwise maximum with the descending top 128 is bitonic and
          // holds the top 128 of the union
          const float m0 = fmaxf(gacc, n0), m1 = fmaxf(gacc_hi, n1);
          gacc = bitonic_merge<64, 64, 32>(fmaxf(m0, m1), lane);
          gacc_hi = bitonic_merge<64, 64, 32>(fminf(m0, m1), lane);
          tc = K <= 64 ? rdlane(gacc, K - 1) : rdlane(gacc_hi, K - 65);
        }
        if constexpr (!kSmallK) tblank = blank_bound();
        // an infinite bound admits every finite candidate and no -inf one
        const float tau = fmaxf(fmaxf(fmaxf(tau_run, tc), tblank), -__FLT_MAX__);
        CTCBEAM_PHASE_MARK(14);
        // most waves hold no survivor: their lane maxima say so
        if (__ballot(lmax >= tau) != 0ull) {  // uniform
          uint32_t qmask = 0u;
#pragma unroll
          for (int r = 0; r < NC; ++r) qmask |= (cand[r] >= tau) ? (1u << r) : 0u;
          const int mycnt = __popc(qmask);
          const int incl = wave_incl_scan(mycnt, lane);
          const int wtotal = rdlane(incl, 63);
          int wbase = 0;
          if (lane == 0) wbase = atomicAdd(&s_nbuf, wtotal);
          wbase = __builtin_amdgcn_readfirstlane(wbase);
          int slot = wbase + incl - mycnt;
          // the pool entry of candidate r (LM target: the staged arc's or the
          // token's unigram state; with rank skipping resolved now, as a
          // later chunk reuses the staging area before the rank, otherwise
          // by the rank)
          const auto put = [&](int r, int at) __attribute__((always_inline)) {
            const int i = r / LPT, jj = r % LPT;
            const int c = tid + jj * kThreads;
            uint32_t lraw, bk;
            if constexpr (kKeepLm) {
              lraw = lhi[r];
              bk = 0u;
            } else {
              cand_meta(i, jj, lraw, bk);
            }
            if (HAS_LM && SKIP && !CACHE) lraw = lm_target(lraw);
            s_pool[at] = make_uint4(__float_as_uint(cand[r]), static_cast<uint32_t>(kslot[i] * W + c), lraw, bk);
          };
          if (wbase + wtotal <= kCap) {  // uniform: the wave's range fits
#pragma unroll
            for (int r = 0; r < NC; ++r) {
              if (qmask & (1u << r)) {
                put(r, slot);
                ++slot;
              }
            }
          } else {
#pragma unroll
            for (int r = 0; r < NC; ++r) {
              if (qmask & (1u << r)) {
                if (slot < kCap) put(r, slot);
                else s_overflow = 1;
                ++slot;
              }
            }
          }
        }
      }
      CTCBEAM_PHASE_MARK(4);
      __syncthreads();  // C: pool complete
      CTCBEAM_PHASE_MARK(5);
      if constexpr (rep) {
        // repeat-scoring variant: the terms of this chunk's survivors, while
        // its rows are in place
        const int n = min(s_nbuf, kCap);
        for (int e = carry + tid; e < n; e += kThreads) s_pinc[e] = terms_of_flat(s_pool[e].y);
        __syncthreads();
      }

      // ---- R. exact rank of the pool: reserved region P + survivors ----
      // The best K go to region Q in rank order; after the last chunk the
      // winners' successor records go to s_rec[rcur ^ 1] instead.  Before
      // the last chunk the rank runs only when the pool is more than half
      // full (a quarter with two slots per lane, whose block rank costs the
      // square of the pool; an earlier rank also tightens the bound) or
      // overflowed: otherwise the survivors stay in the pool for the next
      // chunk (with large beams most chunks skip it).
      const bool last_chunk = ch + 1 == nch;
      const int npool = s_nbuf;
      if (SKIP && !last_chunk && !s_overflow && npool <= (SPL > 1 ? kCap / 4 : kCap / 2)) {  // uniform
        carry = npool;
        cs += kc;
        CTCBEAM_PHASE_COUNT(10);  // chunks
        continue;
      }
      {
        const int P = mpar, Q = mpar ^ 1;
        const uint32_t* prec = s_rec + rcur * (KMX * RW);
        uint32_t* nrec = s_rec + (rcur ^ 1) * (KMX * RW);
        if (!s_overflow) {
          CTCBEAM_PHASE_COUNT(15);  // ranks
          const int n = min(s_nbuf, kCap);
          const int N = K + n;
          nfin = 0;
          if (N <= 64) {
            // one entry per lane; this wave ranks (owns) entries wave + 8u
            uint4 eq = make_uint4(__float_as_uint(kNegInf), 0xFFFFFFFFu, 0u, 0u);
            if (lane < N) eq = (lane < K) ? s_res[P][lane] : s_pool[lane - K];
            const float xq = __uint_as_float(eq.x);
            nfin = __popcll(__ballot(xq != kNegInf));
            const bool own = ((lane & (kWaves - 1)) == wave) && xq != kNegInf;
            uint32_t lmt = eq.z;
            if (HAS_LM && !SKIP && !CACHE && lane >= K) lmt = lm_target(lmt);
            Succ sp;
            if (last_chunk) succ_begin(own, eq.y, lmt, eq.w, prec, sp);  // loads overlap the ranking
            int myrank = K;
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              if (u > 0 && u * kWaves >= N) break;  // uniform: no entries left
              const int ql = wave + u * kWaves;
              const float xs = rdlane(xq, ql);
              const uint32_t is = rdlane(eq.y, ql);
              const int rk = __popcll(__ballot(xq > xs || (xq == xs && eq.y < is)));
              myrank = ((lane >> 3) == u) ? rk : myrank;
            }
            if (last_chunk) {
              succ_end(sp, eq.x);
              if (own && myrank < K) {
                store_rec(nrec + myrank * RW, sp.r);
                if (rep && sp.emit) put_terms(nrec + myrank * RW, (lane < K) ? s_rinc[P][lane] : s_pinc[lane - K]);
              }
            } else if (own && myrank < K) {
              s_res[Q][myrank] = make_uint4(eq.x, eq.y, lmt, eq.w);
              if (rep) s_rinc[Q][myrank] = (lane < K) ? s_rinc[P][lane] : s_pinc[lane - K];
            }
          } else if (kTreeRank && N > 192 && N <= kThreads) {
            CTCBEAM_PHASE_COUNT(16);  // merge-tree ranks
            // K <= 64 of 193..512 entries (a few blocks of 64 are cheaper to
            // rank against each other): each wave sorts its 64 entries by
            // (score desc, index asc) as 64-bit keys, then a tree of pairwise
            // merges keeps the top 64 (the 64 largest of two ascending lists
            // are the elementwise maximum of one and the other reversed, a
            // bitonic sequence), instead of ranking every entry against
            // every other
            const int q = tid;
            uint4 eq = make_uint4(__float_as_uint(kNegInf), 0xFFFFFFFFu, 0u, 0u);
            if (q < N) eq = (q < K) ? s_res[P][q] : s_pool[q - K];
            const float xq = __uint_as_float(eq.x);
            const uint64_t key = xq != kNegInf ? order_key(xq, eq.y) : 0ull;
            uint32_t klo = static_cast<uint32_t>(key), khi = static_cast<uint32_t>(key >> 32);
            uint32_t ksl = static_cast<uint32_t>(q);
            sort3_levels<2>(klo, khi, ksl, lane);  // ascending over the wave
            const int wcnt = __popcll(__ballot(xq != kNegInf));
            if (lane == 0) s_wcnt[wave] = wcnt;
            const auto publish = [&](int r) __attribute__((always_inline)) {
              s_srt[r][0][lane] = klo;
              s_srt[r][1][lane] = khi;
              s_srt[r][2][lane] = ksl;
            };
            const auto merge_with = [&](int r) __attribute__((always_inline)) {
              const uint32_t olo = s_srt[r][0][63 - lane], ohi = s_srt[r][1][63 - lane];
              const uint32_t osl = s_srt[r][2][63 - lane];
              const bool gt = ohi > khi || (ohi == khi && (olo > klo || (olo == klo && osl > ksl)));
              klo = gt ? olo : klo;
              khi = gt ? ohi : khi;
              ksl = gt ? osl : ksl;
              sort3_merge<64, 32>(klo, khi, ksl, lane);
            };
            if (wave & 1) publish(wave >> 1);  // waves 1, 3, 5, 7: lists 0..3
            __syncthreads();
            nfin = 0;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) nfin += s_wcnt[w];
            if ((wave & 1) == 0) merge_with(wave >> 1);
            if ((wave & 3) == 2) publish(4 + (wave >> 2));  // waves 2, 6: lists 4, 5
            __syncthreads();
            if ((wave & 3) == 0) merge_with(4 + (wave >> 2));
            if (wave == 4) publish(6);
            __syncthreads();
            if (wave == 0) {
              merge_with(6);
              // lane 63 holds the best entry: rank 63 - lane
              const int rank = 63 - lane;
              if (rank < min(K, nfin)) {
                const uint32_t qq = ksl;
                const uint4 e = (qq < static_cast<uint32_t>(K)) ? s_res[P][qq] : s_pool[qq - K];
                uint32_t lmt = e.z;
                if (HAS_LM && !SKIP && !CACHE && qq >= static_cast<uint32_t>(K)) lmt = lm_target(lmt);
                s_res[Q][rank] = make_uint4(e.x, e.y, lmt, e.w);
                if (rep) s_rinc[Q][rank] = (qq < static_cast<uint32_t>(K)) ? s_rinc[P][qq] : s_pinc[qq - K];
              }
            }
            if (last_chunk) {
              __syncthreads();  // region Q complete
              const bool act = wave == 0 && tid < min(K, nfin);
              uint4 e = make_uint4(__float_as_uint(kNegInf), 0xFFFFFFFFu, 0u, 0u);
              if (act) e = s_res[Q][tid];
              Succ sp;
              succ_begin(act, e.y, e.z, e.w, prec, sp);
              succ_end(sp, e.x);
              if (act) store_rec(nrec + tid * RW, sp.r);
              if (rep && act && sp.emit) put_terms(nrec + tid * RW, s_rinc[Q][tid]);
            }
          } else {
            // blocks of 64 entries: this wave ranks entries qb + (wave + 8u)
            // against every entry, lane f holding entry fb + f
            CTCBEAM_PHASE_COUNT(16);  // block ranks
            for (int qb = 0; qb < N; qb += 64) {
              const int q = qb + lane;
              uint4 eq = make_uint4(__float_as_uint(kNegInf), 0xFFFFFFFFu, 0u, 0u);
              if (q < N) eq = (q < K) ? s_res[P][q] : s_pool[q - K];
              const float xq = __uint_as_float(eq.x);
              nfin += __popcll(__ballot(xq != kNegInf));
              int rk[8];
#pragma unroll
              for (int u = 0; u < 8; ++u) rk[u] = 0;
              for (int fb = 0; fb < N; fb += 64) {
                float xf = xq;
                uint32_t iff = eq.y;
                if (fb != qb) {
                  const int f = fb + lane;
                  uint4 ef = make_uint4(__float_as_uint(kNegInf), 0xFFFFFFFFu, 0u, 0u);
                  if (f < N) ef = (f < K) ? s_res[P][f] : s_pool[f - K];
                  xf = __uint_as_float(ef.x);
                  iff = ef.y;
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                  const int ql = wave + u * kWaves;
                  if (qb + ql < N) {  // wave-uniform
                    const float xs = rdlane(xq, ql);
                    const uint32_t is = rdlane(eq.y, ql);
                    rk[u] += __popcll(__ballot(xf > xs || (xf == xs && iff < is)));
                  }
                }
              }
              // owner lane wave + 8u takes rank u
              int myrank = K;
#pragma unroll
              for (int u = 0; u < 8; ++u) myrank = ((lane >> 3) == u) ? rk[u] : myrank;
              const bool win = (lane & (kWaves - 1)) == wave && myrank < K && xq != kNegInf;
              uint32_t lmt = eq.z;
              if (HAS_LM && !SKIP && !CACHE && win && q >= K) lmt = lm_target(lmt);
              // winners to region Q in rank order (after the last chunk their
              // successor records are built below, in one pass)
              if (win) s_res[Q][myrank] = make_uint4(eq.x, eq.y, lmt, eq.w);
              if (rep && win) s_rinc[Q][myrank] = (q < K) ? s_rinc[P][q] : s_pinc[q - K];
            }
            if (last_chunk) {
              __syncthreads();  // region Q complete
              // rank tid (waves 0 .. SPL-1): the chain-header loads of all
              // winners are in flight together
              const bool act = (SPL > 1 || wave == 0) && tid < min(K, nfin);
              uint4 e = make_uint4(__float_as_uint(kNegInf), 0xFFFFFFFFu, 0u, 0u);
              if (act) e = s_res[Q][tid];
              Succ sp;
              succ_begin(act, e.y, e.z, e.w, prec, sp);
              succ_end(sp, e.x);
              if (act) store_rec(nrec + tid * RW, sp.r);
              if (rep && act && sp.emit) put_terms(nrec + tid * RW, s_rinc[Q][tid]);
            }
          }
        } else {
          CTCBEAM_PHASE_COUNT(17);  // pool overflows (K-step extraction)
          // exact extraction over (reserved region P) U (pool entries carried
          // from earlier chunks) U (this chunk's candidates)
          uint64_t prev = ~0ull;
          int nk = 0;
          for (int it = 0; it < K; ++it) {
            uint64_t best = 0ull;
            int who = -1;  // -1 none, 0 a register candidate, 100+e reserved, 1000+e pool entry
            // the best register candidate's fields, tracked by selects so that
            // no candidate array is indexed at run time
            float wx = kNegInf;
            uint32_t wflat = 0u, wi = 0u, wjj = 0u, wrow = 0u, wbrow = 0u;
#pragma unroll
            for (int r = 0; r < NC; ++r) {
              if (cand[r] != kNegInf) {
                const int i = r / LPT, jj = r % LPT;
                const int c = tid + jj * kThreads;
                const uint32_t flat = static_cast<uint32_t>(kslot[i] * W + c);
                const uint64_t key = order_key(cand[r], flat);
                if (key < prev && key > best) {
                  best = key;
                  who = 0;
                  wx = cand[r];
                  wflat = flat;
                  wi = static_cast<uint32_t>(i);
                  wjj = static_cast<uint32_t>(jj);
                  if constexpr (CACHE || kGroups) wrow = krow[i];
                  if constexpr (kGroups) wbrow = kbrow[i];
                }
              }
            }
            if (tid < K) {
              const uint4 e = s_res[P][tid];
              const float xe = __uint_as_float(e.x);
              if (xe != kNegInf) {
                const uint64_t key = order_key(xe, e.y);
                if (key < prev && key > best) {
                  best = key;
                  who = 100 + tid;
                }
              }
            }
            if (tid < carry) {  // carry <= kCap / 2 <= kThreads
              const uint4 e = s_pool[tid];
              const float xe = __uint_as_float(e.x);
              if (xe != kNegInf) {
                const uint64_t key = order_key(xe, e.y);
                if (key < prev && key > best) {
                  best = key;
                  who = 1000 + tid;
                }
              }
            }
            uint64_t wbest = best;
            for (int off = 1; off < 64; off <<= 1) {
              const uint64_t o = __shfl_xor(wbest, off);
              wbest = o > wbest ? o : wbest;
            }
            if (lane == 0) s_red[it & 1][wave] = wbest;
            __syncthreads();
            uint64_t gbest = s_red[it & 1][0];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) gbest = s_red[it & 1][w] > gbest ? s_red[it & 1][w] : gbest;
            if (gbest == 0ull) break;  // nothing finite left (uniform)
            if (who >= 0 && best == gbest) {
              if (who < 100) {
                // label c = tid + wjj * kThreads of chunk row wi
                const uint32_t c = static_cast<uint32_t>(tid) + wjj * static_cast<uint32_t>(kThreads);
                const uint32_t e = wi * static_cast<uint32_t>(V) + c;
                uint32_t lmt = 0u, bk = 0u;
                if (HAS_LM) {
                  if constexpr (CACHE) {
                    lmt = static_cast<uint32_t>(lmrow[wrow * static_cast<uint32_t>(V) + c] >> 32) & kTargetMask;
                  } else {
                    const uint32_t el = kGroups ? wrow * static_cast<uint32_t>(V) + c : e;
                    const uint32_t hi = static_cast<uint32_t>(lmrow[el] >> 32);
                    lmt = (kFoldRows || hi >= genhi) ? lm_target(hi) : c;
                  }
                }
                if (HAS_BT) {
                  const uint32_t be = btrow[kGroups ? wbrow * static_cast<uint32_t>(V) + c : e];
                  bk = (be >= genhi) ? be : p.bt_root_key[c];
                }
                s_res[Q][it] = make_uint4(__float_as_uint(wx), wflat, lmt, bk);
                // terms taken after the extraction, from this chunk's rows
                if (rep) s_rinc[Q][it] = make_float2(__builtin_nanf(""), 0.0f);
              } else if (who < 1000) {
                s_res[Q][it] = s_res[P][who - 100];
                if (rep) s_rinc[Q][it] = s_rinc[P][who - 100];
              } else {
                s_res[Q][it] = s_pool[who - 1000];
                if (rep) s_rinc[Q][it] = s_pinc[who - 1000];
              }
            }
            prev = gbest;
            ++nk;
          }
          nfin = nk;
          if constexpr (rep) {
            // the terms of the winners taken from this chunk's candidates
            // (the later barriers order them before their readers)
            __syncthreads();
            if (tid < nk && __builtin_isnan(s_rinc[Q][tid].x)) {
              const uint32_t flat = s_res[Q][tid].y;
              // a token (blank winners carry no terms)
              if (flat % static_cast<uint32_t>(W) < static_cast<uint32_t>(V)) s_rinc[Q][tid] = terms_of_flat(flat);
            }
          }
          if (last_chunk) {
            __syncthreads();  // region Q complete
            // rank tid (waves 0 .. SPL-1)
            const bool act = (SPL > 1 || wave == 0) && tid < nk;
            uint4 e = make_uint4(__float_as_uint(kNegInf), 0xFFFFFFFFu, 0u, 0u);
            if (act) e = s_res[Q][tid];
            Succ sp;
            succ_begin(act, e.y, e.z, e.w, prec, sp);
            succ_end(sp, e.x);
            if (act) store_rec(nrec + tid * RW, sp.r);
            if (rep && act && sp.emit) put_terms(nrec + tid * RW, s_rinc[Q][tid]);
          }
        }
        // ranks [nfin, K) hold no candidate (the next chunk reads all K)
        if (!last_chunk && (SPL > 1 || wave == 0) && tid >= nfin && tid < K)
          s_res[Q][tid] = make_uint4(__float_as_uint(kNegInf), 0xFFFFFFFFu, 0u, 0u);
      }
      CTCBEAM_PHASE_MARK(6);
      __syncthreads();  // D: best K of the chunk in region Q
      CTCBEAM_PHASE_MARK(7);
      CTCBEAM_PHASE_COUNT(10);  // chunks
      mpar ^= 1;
      carry = 0;
      if (ch + 1 < nch && nfin >= K) tau_run = fmaxf(tau_run, __uint_as_float(s_res[mpar][K - 1].x));
      cs += kc;
    }

    // The single-slot form (K <= 64) is kept apart from the general one: the
    // general form, instantiated with one slot per lane, changes the register
    // allocation of the frame loop and costs about 2 % at K = 8.
    if constexpr (SPL == 1) {
    // ---- U. prune, recombine, take the new beam (every wave, lane j = slot j) ----
    {
      const int nsel = min(K, nfin);
      const bool valid = j < nsel;
      uint32_t rec[RW];
#pragma unroll
      for (int w = 0; w < RW; ++w) rec[w] = 0u;
      if (valid) load_rec(s_rec + (rcur ^ 1) * (KMX * RW) + j * RW, rec);
      float x = valid ? __uint_as_float(rec[kRX]) : kNegInf;
      // prune (Algorithm 1: below best - theta -> -inf)
      const float best = rdlane(x, 0);
      const float lim = best - p.theta;
      if (valid && x < lim) x = kNegInf;
      const bool emit = valid && rec[kREmit] != 0u;
      const bool emit_fin = x != kNegInf && emit;
      const int32_t nlast = valid ? static_cast<int32_t>(rec[kRLast]) : V;
      const int32_t nlen = static_cast<int32_t>(rec[kRLen]);
      // recombination: same transcript hash, length and ends-in-blank flag as
      // a live lower slot
      const bool alive0 = valid && x != kNegInf;
      const uint32_t meta = (static_cast<uint32_t>(nlen) & 0x3FFFFFFFu) | ((nlast == V ? 1u : 0u) << 30);
      bool dup = false;
      if (K <= 16) {
        // The K slots sit in the first 16-lane row: compare each with the
        // slots below it through row shifts.  The key folds the length and
        // the ends-in-blank flag into the 64-bit transcript hash (a false
        // merge needs a 64-bit collision, as for the hash itself); dead
        // slots use all ones and are never merged into.
        uint64_t key = ((static_cast<uint64_t>(rec[kRHhi]) << 32) | rec[kRHlo]) ^
                       (static_cast<uint64_t>(meta + 1u) * 0xD6E8FEB86659FD93ull);
        if (!alive0) key = ~0ull;
        const uint32_t klo = static_cast<uint32_t>(key), khi = static_cast<uint32_t>(key >> 32);
        dup = (K <= 8 ? recomb_shifts<1, 7>(klo, khi) : recomb_shifts<1, 15>(klo, khi)) && alive0;
      } else {
        // the same key, compared through a sort of all 64 slots
        uint64_t key = ((static_cast<uint64_t>(rec[kRHhi]) << 32) | rec[kRHlo]) ^
                       (static_cast<uint64_t>(meta + 1u) * 0xD6E8FEB86659FD93ull);
        if (!alive0) key = ~0ull;
        uint32_t slo, shi;
        dup = dup_by_sort(key, lane, slo, shi) && alive0;
      }
      if (p.flags & kFlagLogSumExp) {  // uniform
        // Each duplicate, in slot order, is merged into the first live slot
        // of its transcript (a lower slot, which is not a duplicate itself).
        uint64_t dm = __ballot(dup);
        const float xs = x;
        while (dm) {
          const int jj = static_cast<int>(__builtin_ctzll(dm));
          dm &= dm - 1ull;
          const uint32_t hlo = rdlane(rec[kRHlo], jj);
          const uint32_t hhi = rdlane(rec[kRHhi], jj);
          const uint32_t mj = rdlane(meta, jj);
          const uint64_t same = __ballot(alive0 && rec[kRHlo] == hlo && rec[kRHhi] == hhi && meta == mj);
          const int rep = static_cast<int>(__builtin_ctzll(same));  // jj itself matches: same != 0
          const float xj = rdlane(xs, jj);
          if (j == rep && rep != jj) x = lse32(x, xj);
        }
      }
      if (dup) x = kNegInf;
      CTCBEAM_PHASE_MARK(11);
      const bool nalive = alive0 && !dup;
      // back-pointers and beam records from waves 1 and 2: wave 0 carries the
      // frame's longest chain, and a store would hold its next load wait
      // (vmcnt counts stores and loads in issue order)
      if (wave == 1 && j < K) bpb[static_cast<size_t>(t) * K + j] = valid ? static_cast<int32_t>(rec[kRBp]) : -1;
      // new state
      sc[0] = x;
      last[0] = nlast;
      len[0] = nlen;
      alive[0] = nalive;
      int32_t acnt = 0;
#pragma unroll
      for (int l = 0; l < NL; ++l) {
        lvb[0][l] = nalive ? rec[kRLvb + l] : 0u;
        lvc[0][l] = nalive ? rec[kRLvc + l] : 0u;
        lvbo[0][l] = nalive ? __uint_as_float(rec[kRLvbo + l]) : 0.0f;
        acnt += static_cast<int32_t>(lvc[0][l] & ~kExists);
      }
      if (HAS_BT) {
        btb[0] = nalive ? rec[kRBtb] : 0u;
        btc[0] = nalive ? rec[kRBtc] : 0u;
        btpot[0] = nalive ? static_cast<int32_t>(rec[kRBtp]) : 0;
      }
      if (want_stats && wave == 0) {
        // chain work of the next frame (alive beams) and this frame's
        // emitting winners
        uint32_t s_ls = 0u, s_la = 0u, s_bn = 0u, s_ba = 0u;
        const bool counted = t + 1 < L && nalive;
        if (counted) {
#pragma unroll
          for (int l = 0; l < NL; ++l) {
            if (lvc[0][l] & kExists) {
              s_ls += 1u;
              s_la += lvc[0][l] & ~kExists;
            }
          }
          if (HAS_BT) {
            const BtNode pn = p.bt_nodes[rec[kRBts]];
            s_bn = pn.pot >> 8;
            s_ba = pn.chain_arcs;
          }
          atomicAdd(&s_st[0], 1ull);
        }
        if (s_ls) atomicAdd(&s_st[1], static_cast<unsigned long long>(s_ls));
        if (s_la) atomicAdd(&s_st[2], static_cast<unsigned long long>(s_la));
        if (s_bn) atomicAdd(&s_st[3], static_cast<unsigned long long>(s_bn));
        if (s_ba) atomicAdd(&s_st[4], static_cast<unsigned long long>(s_ba));
        if (emit_fin) atomicAdd(&s_st[5], 1ull);
      }
      rcur ^= 1;
      CTCBEAM_PHASE_MARK(12);
      // live positions and beam records for the next frame
      const uint64_t amask = __ballot(nalive);
      const int na = __popcll(amask);
      int lp = __popcll(amask & lmlt);
      if constexpr (CACHE) {
        // Key rows of the new beam: a live slot whose LM state has a row
        // keeps it; each other state takes a row no live slot uses (there are
        // K <= KCR rows) and its first slot fills it in the next frame.  When
        // the next fill wraps the generation every row is cleared, so every
        // state is new.
        // The slots (lanes 0..K-1) meet the row tags (lanes 0..7, rows past
        // KCR empty) through rotations within 16 lanes, lanes 8..15 holding
        // a copy of lanes 0..7.
        const uint32_t st = rec[kRLms];
        if (gen == kGenMax) rtag = 0xFFFFFFFFu;  // the next fill clears every row
        const bool hi8 = lane_in_here<0xFF00FF00FF00FF00ull>();
        const uint32_t rt8 = hi8 ? dpp_row_ror<8>(rtag) : rtag;
        const uint32_t ri8 = static_cast<uint32_t>(lane & 7);
        bool hit = false;
        uint32_t hrow = 0u;
        const auto probe = [&](uint32_t td, uint32_t id) __attribute__((always_inline)) {
          const bool h = st == td;
          hrow = h ? id : hrow;
          hit = hit || h;
        };
        probe(rt8, ri8);
        probe(dpp_row_ror<1>(rt8), dpp_row_ror<1>(ri8));
        probe(dpp_row_ror<2>(rt8), dpp_row_ror<2>(ri8));
        probe(dpp_row_ror<3>(rt8), dpp_row_ror<3>(ri8));
        probe(dpp_row_ror<4>(rt8), dpp_row_ror<4>(ri8));
        probe(dpp_row_ror<5>(rt8), dpp_row_ror<5>(ri8));
        probe(dpp_row_ror<6>(rt8), dpp_row_ror<6>(ri8));
        probe(dpp_row_ror<7>(rt8), dpp_row_ror<7>(ri8));
        hit = hit && nalive;
        if (hit) rowof = static_cast<int>(hrow);
        // rows used by a live slot (slots are lanes 0..7)
        uint32_t ub = hit ? (1u << hrow) : 0u;
        ub |= xor_lane(ub, 1, lane);
        ub |= xor_lane(ub, 2, lane);
        ub |= xor_lane(ub, 4, lane);
        uint32_t used = rdlane(ub, 0);
        bool miss = nalive && !hit;
        fillrep = false;
        uint64_t mm = __ballot(miss);
        while (mm != 0ull) {  // uniform
          const int jm = static_cast<int>(__builtin_ctzll(mm));
          const uint32_t sj = rdlane(st, jm);
          const bool same = miss && st == sj;
          const int r = min(__builtin_ctz(~used), KCR - 1);  // a free row: < KCR
          used |= 1u << r;
          if (lane == r) rtag = sj;
          rowof = same ? r : rowof;
          fillrep = fillrep || j == jm;
          miss = miss && !same;
          mm = __ballot(miss);
        }
      }
      if constexpr (kGroups) {
        const bool nal[1] = {nalive};
        const int32_t ac[1] = {acnt};
        const uint32_t lk[1] = {(HAS_LM && NL > 0 && nalive) ? rec[kRLms] : 0u};  // a unigram LM fills no row
        int lpa[1] = {lp};
        plan_groups(nal, ac, lk, lpa);
        lp = lpa[0];
      }
      CTCBEAM_PHASE_MARK(13);
      if (wave == 2 && nalive) put_row(lp, 0);
      // chunk plan: live slots in slot order, at most kcmax beams and
      // kLmStage staged arcs per chunk (cached rows stage nothing)
      if constexpr (CACHE) {
        nch = na > 0 ? 1 : 0;  // K <= KCR = kcmax, nothing staged
        cid[0] = 0;
      } else if constexpr (kGroups) {
        // planned above
      } else {
      const int ia = wave_incl_scan(acnt, lane);
      const int tota = rdlane(ia, 63);
      if (na <= kcmax && tota <= kLmStage) {
        nch = na > 0 ? 1 : 0;
        cid[0] = 0;
      } else {
        nch = 0;
        cid[0] = -1;
        int start = 0;
        while (start < na) {
          const uint64_t sm = __ballot(nalive && lp == start);
          const int sl = static_cast<int>(__builtin_ctzll(sm));
          const int basea = rdlane(ia - acnt, sl);
          const bool ok = nalive && lp >= start && lp < start + kcmax && (ia - basea) <= kLmStage;
          int cnt = __popcll(__ballot(ok));
          if (cnt == 0) {
            cnt = 1;  // a single chain above the staging limit (the builders prevent it)
            status |= 4u;
          }
          if (nalive && lp >= start && lp < start + cnt) cid[0] = nch;
          ++nch;
          start += cnt;
        }
      }
      }
    }
    } else {
    // ---- U. prune, recombine, take the new beam (every wave; slot
    // j + 64 h in register set h) ----
    {
      const int nsel = min(K, nfin);
      uint32_t rec[SPL][RW];
      float x[SPL];
      bool valid[SPL], alive0[SPL], dup[SPL], emit_fin[SPL];
      int32_t nlast[SPL], nlen[SPL];
      uint32_t meta[SPL];
#pragma unroll
      for (int h = 0; h < SPL; ++h) {
        valid[h] = j + 64 * h < nsel;
#pragma unroll
        for (int w = 0; w < RW; ++w) rec[h][w] = 0u;
        if (valid[h]) load_rec(s_rec + (rcur ^ 1) * (KMX * RW) + (j + 64 * h) * RW, rec[h]);
        x[h] = valid[h] ? __uint_as_float(rec[h][kRX]) : kNegInf;
      }
      // prune (Algorithm 1: below best - theta -> -inf)
      const float best = rdlane(x[0], 0);
      const float lim = best - p.theta;
#pragma unroll
      for (int h = 0; h < SPL; ++h) {
        if (valid[h] && x[h] < lim) x[h] = kNegInf;
        const bool emit = valid[h] && rec[h][kREmit] != 0u;
        emit_fin[h] = x[h] != kNegInf && emit;
        nlast[h] = valid[h] ? static_cast<int32_t>(rec[h][kRLast]) : V;
        nlen[h] = static_cast<int32_t>(rec[h][kRLen]);
        // recombination key: transcript hash, length and ends-in-blank flag
        alive0[h] = valid[h] && x[h] != kNegInf;
        meta[h] = (static_cast<uint32_t>(nlen[h]) & 0x3FFFFFFFu) | ((nlast[h] == V ? 1u : 0u) << 30);
        dup[h] = false;
      }
      if (K <= 16) {
        // The K slots sit in the first 16-lane row: compare each with the
        // slots below it through row shifts.  The key folds the length and
        // the ends-in-blank flag into the 64-bit transcript hash (a false
        // merge needs a 64-bit collision, as for the hash itself); dead
        // slots use all ones and are never merged into.
        uint64_t key = ((static_cast<uint64_t>(rec[0][kRHhi]) << 32) | rec[0][kRHlo]) ^
                       (static_cast<uint64_t>(meta[0] + 1u) * 0xD6E8FEB86659FD93ull);
        if (!alive0[0]) key = ~0ull;
        const uint32_t klo = static_cast<uint32_t>(key), khi = static_cast<uint32_t>(key >> 32);
        dup[0] = (K <= 8 ? recomb_shifts<1, 7>(klo, khi) : recomb_shifts<1, 15>(klo, khi)) && alive0[0];
      } else {
        // Each register set is sorted on its own (its slots are in lane
        // order); a slot of the upper set is also a duplicate when its key
        // occurs among the live keys of the lower set (all lower slots):
        // binary search in the lower set's sorted keys.
        uint64_t key[SPL];
        uint32_t slo[SPL], shi[SPL];
#pragma unroll
        for (int h = 0; h < SPL; ++h) {
          key[h] = ((static_cast<uint64_t>(rec[h][kRHhi]) << 32) | rec[h][kRHlo]) ^
                   (static_cast<uint64_t>(meta[h] + 1u) * 0xD6E8FEB86659FD93ull);
          if (!alive0[h]) key[h] = ~0ull;
          dup[h] = dup_by_sort(key[h], lane, slo[h], shi[h]) && alive0[h];
        }
#pragma unroll
        for (int h = 1; h < SPL; ++h) {
          // position of the first lower key >= key[h]
          int pos = 0;
          const uint64_t kh = key[h];
#pragma unroll
          for (int step = 32; step >= 1; step >>= 1) {
            const int a = (pos + step - 1) << 2;
            const uint64_t v = (static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(a, static_cast<int>(shi[0])))) << 32) |
                               static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(a, static_cast<int>(slo[0])));
            pos += (v < kh) ? step : 0;
          }
          // pos <= 63: the last lower key decides the 64th position
          const uint64_t at = (static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(pos << 2, static_cast<int>(shi[0])))) << 32) |
                              static_cast<uint32_t>(__builtin_amdgcn_ds_bpermute(pos << 2, static_cast<int>(slo[0])));
          dup[h] = dup[h] || (alive0[h] && at == kh);
        }
      }
      if (p.flags & kFlagLogSumExp) {  // uniform
        // Each duplicate, in slot order, is merged into the first live slot
        // of its transcript (a lower slot, which is not a duplicate itself).
        float xs[SPL];
#pragma unroll
        for (int h = 0; h < SPL; ++h) xs[h] = x[h];
#pragma unroll
        for (int hj = 0; hj < SPL; ++hj) {
          uint64_t dm = __ballot(dup[hj]);
          while (dm) {
            const int jj = static_cast<int>(__builtin_ctzll(dm));
            dm &= dm - 1ull;
            const uint32_t hlo = rdlane(rec[hj][kRHlo], jj);
            const uint32_t hhi = rdlane(rec[hj][kRHhi], jj);
            const uint32_t mj = rdlane(meta[hj], jj);
            int rep = -1;  // the duplicate itself matches, so some slot does
#pragma unroll
            for (int h = SPL - 1; h >= 0; --h) {
              const uint64_t same =
                  __ballot(alive0[h] && rec[h][kRHlo] == hlo && rec[h][kRHhi] == hhi && meta[h] == mj);
              if (same) rep = static_cast<int>(__builtin_ctzll(same)) + 64 * h;
            }
            const float xj = rdlane(xs[hj], jj);
#pragma unroll
            for (int h = 0; h < SPL; ++h)
              if (j + 64 * h == rep && rep != jj + 64 * hj) x[h] = lse32(x[h], xj);
          }
        }
      }
      bool nalive[SPL];
      int32_t acnt[SPL];
#pragma unroll
      for (int h = 0; h < SPL; ++h) {
        if (dup[h]) x[h] = kNegInf;
        nalive[h] = alive0[h] && !dup[h];
        const int js = j + 64 * h;
        if (wave == 1 && js < K)
          bpb[static_cast<size_t>(t) * K + js] = valid[h] ? static_cast<int32_t>(rec[h][kRBp]) : -1;
        // new state
        sc[h] = x[h];
        last[h] = nlast[h];
        len[h] = nlen[h];
        alive[h] = nalive[h];
        acnt[h] = 0;
#pragma unroll
        for (int l = 0; l < NL; ++l) {
          lvb[h][l] = nalive[h] ? rec[h][kRLvb + l] : 0u;
          lvc[h][l] = nalive[h] ? rec[h][kRLvc + l] : 0u;
          lvbo[h][l] = nalive[h] ? __uint_as_float(rec[h][kRLvbo + l]) : 0.0f;
          acnt[h] += static_cast<int32_t>(lvc[h][l] & ~kExists);
        }
        if (HAS_BT) {
          btb[h] = nalive[h] ? rec[h][kRBtb] : 0u;
          btc[h] = nalive[h] ? rec[h][kRBtc] : 0u;
          btpot[h] = nalive[h] ? static_cast<int32_t>(rec[h][kRBtp]) : 0;
        }
        if (want_stats && wave == 0) {
          // chain work of the next frame (alive beams) and this frame's
          // emitting winners
          uint32_t s_ls = 0u, s_la = 0u, s_bn = 0u, s_ba = 0u;
          const bool counted = t + 1 < L && nalive[h];
          if (counted) {
#pragma unroll
            for (int l = 0; l < NL; ++l) {
              if (lvc[h][l] & kExists) {
                s_ls += 1u;
                s_la += lvc[h][l] & ~kExists;
              }
            }
            if (HAS_BT) {
              const BtNode pn = p.bt_nodes[rec[h][kRBts]];
              s_bn = pn.pot >> 8;
              s_ba = pn.chain_arcs;
            }
            atomicAdd(&s_st[0], 1ull);
          }
          if (s_ls) atomicAdd(&s_st[1], static_cast<unsigned long long>(s_ls));
          if (s_la) atomicAdd(&s_st[2], static_cast<unsigned long long>(s_la));
          if (s_bn) atomicAdd(&s_st[3], static_cast<unsigned long long>(s_bn));
          if (s_ba) atomicAdd(&s_st[4], static_cast<unsigned long long>(s_ba));
          if (emit_fin[h]) atomicAdd(&s_st[5], 1ull);
        }
      }
      rcur ^= 1;
      // live positions (slot order) and beam records for the next frame;
      // ia = inclusive scan of the staged arcs over the slots
      int lp[SPL], ia[SPL];
      int na = 0, tota = 0;
#pragma unroll
      for (int h = 0; h < SPL; ++h) {
        const uint64_t amask = __ballot(nalive[h]);
        lp[h] = na + __popcll(amask & lmlt);
        na += __popcll(amask);
        if (!kGroups && wave == 2 && nalive[h]) put_row(lp[h], h);
        ia[h] = tota + wave_incl_scan(acnt[h], lane);
        tota = rdlane(ia[h], 63);
      }
      if constexpr (kGroups) {
        uint32_t lk[SPL];
#pragma unroll
        for (int h = 0; h < SPL; ++h) lk[h] = (HAS_LM && NL > 0 && nalive[h]) ? rec[h][kRLms] : 0u;
        plan_groups(nalive, acnt, lk, lp);
#pragma unroll
        for (int h = 0; h < SPL; ++h)
          if (wave == 2 && nalive[h]) put_row(lp[h], h);
      } else if (na <= kcmax && tota <= kLmStage) {
        // chunk plan: live slots in slot order, at most kcmax beams and
        // kLmStage staged arcs per chunk
        nch = na > 0 ? 1 : 0;
#pragma unroll
        for (int h = 0; h < SPL; ++h) cid[h] = 0;
      } else {
        nch = 0;
#pragma unroll
        for (int h = 0; h < SPL; ++h) cid[h] = -1;
        int start = 0;
        while (start < na) {
          // staged arcs before the chunk's first beam (the slot at live
          // position start)
          int basea = 0;
#pragma unroll
          for (int h = SPL - 1; h >= 0; --h) {
            const uint64_t sm = __ballot(nalive[h] && lp[h] == start);
            if (sm) basea = rdlane(ia[h] - acnt[h], static_cast<int>(__builtin_ctzll(sm)));
          }
          int cnt = 0;
#pragma unroll
          for (int h = 0; h < SPL; ++h) {
            const bool ok = nalive[h] && lp[h] >= start && lp[h] < start + kcmax && (ia[h] - basea) <= kLmStage;
            cnt += __popcll(__ballot(ok));
          }
          if (cnt == 0) {
            cnt = 1;  // a single chain above the staging limit (the builders prevent it)
            status |= 4u;
          }
#pragma unroll
          for (int h = 0; h < SPL; ++h)
            if (nalive[h] && lp[h] >= start && lp[h] < start + cnt) cid[h] = nch;
          ++nch;
          start += cnt;
        }
      }
    }
    }
    CTCBEAM_PHASE_MARK(8);
    CTCBEAM_PHASE_COUNT(9);  // frames
  }
#ifdef CTCBEAM_PHASE_CLOCKS
  if (p.stats && lane < kPhaseWords) {
    int64_t* pw = p.stats + static_cast<size_t>(p.B) * 8 + (static_cast<size_t>(b) * kWaves + wave) * kPhaseWords;
    pw[lane] = static_cast<int64_t>(ph_acc);
  }
#endif

  // single-slot and general forms kept apart, as for the beam update
  if constexpr (SPL == 1) {
  // ---- LM.Final, order of the final hypotheses ----
  const bool nbest = p.nbest_scores != nullptr;
  if (wave == 0) {
    float s = sc[0];
    if (HAS_LM && j < K && s != kNegInf) {
      // ln P(</s> | state) through the backoff chain; </s> is the last arc of
      // a state's sorted arcs when present
      float v = p.lm_unigram[V];
      int found = -1;
      float fv = 0.0f;
#pragma unroll
      for (int l = NL - 1; l >= 0; --l) {
        const uint32_t n = lvc[0][l] & ~kExists;
        if (found < 0 && n > 0) {
          const LmArc a = p.lm_arcs[lvb[0][l] + n - 1];
          if (a.token == static_cast<uint32_t>(V)) {
            found = l;
            fv = a.logp;
          }
        }
      }
      if (found >= 0) {
        v = fv;
#pragma unroll
        for (int l = 0; l < NL; ++l)
          if (l > found) v = v + lvbo[0][l];
      } else {
#pragma unroll
        for (int l = 0; l < NL; ++l) v = v + lvbo[0][l];
      }
      const float av = alpha * v;
      s = s + av;
    }
    if (HAS_BT && (p.flags & kFlagBoostRollback) && j < K && s != kNegInf) {
      // the pending boosting of an unfinished phrase is taken back
      const float wb = boost_w * static_cast<float>(-btpot[0]);
      s = s + wb;
    }
    // rank of each slot: final score descending, lowest slot on ties
    const float sj = (j < K) ? s : kNegInf;
    int rank = 0;
    for (int i = 0; i < K; ++i) {
      const float si = rdlane(sj, i);
      rank += (si > sj || (si == sj && i < j)) ? 1 : 0;
    }
    const uint64_t top = __ballot(j < K && rank == 0);
    const int bj = static_cast<int>(__builtin_ctzll(top));  // K >= 1: some slot has rank 0
    const float bs = rdlane(sj, bj);
    const int blen = rdlane(len[0], bj);
    const int nlen = (j < K && sj != kNegInf) ? len[0] : 0;
    if (nbest && j < K) {
      p.nbest_scores[static_cast<size_t>(b) * K + rank] = sj;
      p.nbest_lengths[static_cast<size_t>(b) * K + rank] = nlen;
      s_row[rank] = static_cast<uint32_t>(nlen);  // lengths by rank (the row table is free now)
      s_row[KMX + j] = static_cast<uint32_t>(rank);
    }
    if (lane == 0) {
      s_best = bj;
      s_bestscore = bs;
      s_bestlen = blen;
    }
    if (want_stats && lane == 0) {
      // wave 0 made every update of s_st (LDS operations of one wave complete
      // in order)
      int64_t* so = p.stats + static_cast<size_t>(b) * 8;
      so[0] = L;
#pragma unroll
      for (int q = 0; q < 6; ++q) so[1 + q] = static_cast<int64_t>(s_st[q]);
      so[7] = 0;
    }
  }
  __syncthreads();
  const int best = s_best;
  const float bscore = s_bestscore;
  const bool have = bscore != kNegInf;
  const int nout = have ? s_bestlen : 0;
  int32_t* ot = p.out_tokens ? p.out_tokens + static_cast<size_t>(b) * T : nullptr;
  if (ot)
    for (int tt = nout + tid; tt < T; tt += kThreads) ot[tt] = -1;
  if (tid == 0 && p.out_scores) {
    p.out_scores[b] = bscore;
    if (p.out_lengths) p.out_lengths[b] = nout;
  }
  int32_t* nbt = nbest ? p.nbest_tokens + static_cast<size_t>(b) * K * T : nullptr;
  if (nbest) {
    // padding of every row past its transcript
    for (int r = 0; r < K; ++r) {
      const int n = static_cast<int>(s_row[r]);
      for (int tt = n + tid; tt < T; tt += kThreads) nbt[static_cast<size_t>(r) * T + tt] = -1;
    }
  }

  // ---- traceback through the back-pointers, staged in LDS tiles ----
  // 1-best: lane 0 of wave 0 walks the best slot.  N-best: lane j of wave 0
  // walks slot j (every live slot) and writes the row of its rank.
  // (the LM.Final term is finite, so some slot is live exactly when the best
  // final score is finite)
  const bool walker = (wave == 0) && (nbest ? (j < K && sc[0] != kNegInf) : (lane == 0 && have));
  if (have && L > 0) {
    const int tile_frames = kBigWords / K;
    int jb = nbest ? j : best, cnext = -1;
    int32_t* orow = nullptr;
    int pos = 0;
    if (walker) {
      orow = nbest ? nbt + static_cast<size_t>(s_row[KMX + j]) * T : ot;
      pos = nbest ? len[0] : nout;
    }
    for (int hi = L; hi > 0;) {
      const int lo = hi > tile_frames ? hi - tile_frames : 0;
      __syncthreads();
      const int n = (hi - lo) * K;
      const int32_t* src = bpb + static_cast<size_t>(lo) * K;
      for (int q = tid; q < n; q += kThreads) s_big[q] = static_cast<uint32_t>(src[q]);
      __syncthreads();
      if (walker) {
        for (int tt = hi - 1; tt >= lo; --tt) {
          const uint32_t e = s_big[(tt - lo) * K + jb];
          const int cl = static_cast<int>(e & 0xFFFFu);
          const int par = static_cast<int>(e >> 16);
          if (tt < L - 1 && cnext != V && cnext != cl) {
            if (pos > 0) {
              --pos;
              if (orow) orow[pos] = cnext;
            }
          }
          cnext = cl;
          jb = par;
        }
      }
      hi = lo;
    }
    if (walker) {
      if (cnext != V && cnext >= 0 && pos > 0) {
        --pos;
        if (orow) orow[pos] = cnext;
      }
    }
    if (wave == 0 && __ballot(walker && pos != 0) != 0ull) status |= 2u;
  }
  } else {
  // ---- LM.Final, order of the final hypotheses ----
  const bool nbest = p.nbest_scores != nullptr;
  if (wave == 0) {
    float sj[SPL];
#pragma unroll
    for (int h = 0; h < SPL; ++h) {
      const int js = j + 64 * h;
      float s = sc[h];
      if (HAS_LM && js < K && s != kNegInf) {
        // ln P(</s> | state) through the backoff chain; </s> is the last arc
        // of a state's sorted arcs when present
        float v = p.lm_unigram[V];
        int found = -1;
        float fv = 0.0f;
#pragma unroll
        for (int l = NL - 1; l >= 0; --l) {
          const uint32_t n = lvc[h][l] & ~kExists;
          if (found < 0 && n > 0) {
            const LmArc a = p.lm_arcs[lvb[h][l] + n - 1];
            if (a.token == static_cast<uint32_t>(V)) {
              found = l;
              fv = a.logp;
            }
          }
        }
        if (found >= 0) {
          v = fv;
#pragma unroll
          for (int l = 0; l < NL; ++l)
            if (l > found) v = v + lvbo[h][l];
        } else {
#pragma unroll
          for (int l = 0; l < NL; ++l) v = v + lvbo[h][l];
        }
        const float av = alpha * v;
        s = s + av;
      }
      if (HAS_BT && (p.flags & kFlagBoostRollback) && js < K && s != kNegInf) {
        // the pending boosting of an unfinished phrase is taken back
        const float wb = boost_w * static_cast<float>(-btpot[h]);
        s = s + wb;
      }
      sj[h] = (js < K) ? s : kNegInf;
    }
    // rank of each slot: final score descending, lowest slot on ties
    int rank[SPL];
#pragma unroll
    for (int h = 0; h < SPL; ++h) rank[h] = 0;
    for (int i = 0; i < K; ++i) {
      const float si = (i < 64) ? rdlane(sj[0], i) : rdlane(sj[SPL - 1], i & 63);
#pragma unroll
      for (int h = 0; h < SPL; ++h) rank[h] += (si > sj[h] || (si == sj[h] && i < j + 64 * h)) ? 1 : 0;
    }
    int bj = 0;  // K >= 1: some slot has rank 0
#pragma unroll
    for (int h = SPL - 1; h >= 0; --h) {
      const uint64_t top = __ballot(j + 64 * h < K && rank[h] == 0);
      if (top) bj = static_cast<int>(__builtin_ctzll(top)) + 64 * h;
    }
    const float bs = (bj < 64) ? rdlane(sj[0], bj) : rdlane(sj[SPL - 1], bj & 63);
    const int blen = (bj < 64) ? rdlane(len[0], bj) : rdlane(len[SPL - 1], bj & 63);
#pragma unroll
    for (int h = 0; h < SPL; ++h) {
      const int js = j + 64 * h;
      const int nlen = (js < K && sj[h] != kNegInf) ? len[h] : 0;
      if (nbest && js < K) {
        p.nbest_scores[static_cast<size_t>(b) * K + rank[h]] = sj[h];
        p.nbest_lengths[static_cast<size_t>(b) * K + rank[h]] = nlen;
        s_row[rank[h]] = static_cast<uint32_t>(nlen);  // lengths by rank (the row table is free now)
        s_row[KMX + js] = static_cast<uint32_t>(rank[h]);
      }
    }
    if (lane == 0) {
      s_best = bj;
      s_bestscore = bs;
      s_bestlen = blen;
    }
    if (want_stats && lane == 0) {
      // wave 0 made every update of s_st (LDS operations of one wave complete
      // in order)
      int64_t* so = p.stats + static_cast<size_t>(b) * 8;
      so[0] = L;
#pragma unroll
      for (int q = 0; q < 6; ++q) so[1 + q] = static_cast<int64_t>(s_st[q]);
      so[7] = 0;
    }
  }
  __syncthreads();
  const int best = s_best;
  const float bscore = s_bestscore;
  const bool have = bscore != kNegInf;
  const int nout = have ? s_bestlen : 0;
  int32_t* ot = p.out_tokens ? p.out_tokens + static_cast<size_t>(b) * T : nullptr;
  if (ot)
    for (int tt = nout + tid; tt < T; tt += kThreads) ot[tt] = -1;
  if (tid == 0 && p.out_scores) {
    p.out_scores[b] = bscore;
    if (p.out_lengths) p.out_lengths[b] = nout;
  }
  int32_t* nbt = nbest ? p.nbest_tokens + static_cast<size_t>(b) * K * T : nullptr;
  if (nbest) {
    // padding of every row past its transcript
    for (int r = 0; r < K; ++r) {
      const int n = static_cast<int>(s_row[r]);
      for (int tt = n + tid; tt < T; tt += kThreads) nbt[static_cast<size_t>(r) * T + tt] = -1;
    }
  }

  // ---- traceback through the back-pointers, staged in LDS tiles ----
  // 1-best: lane 0 of wave 0 walks the best slot.  N-best: lane j of wave 0
  // walks slots j + 64 h (every live slot) and writes the rows of their ranks.
  // (the LM.Final term is finite, so some slot is live exactly when the best
  // final score is finite)
  if (have && L > 0) {
    const int tile_frames = kBigWords / K;
    bool walker[SPL];
    int jb[SPL], cnext[SPL], pos[SPL];
    int32_t* orow[SPL];
#pragma unroll
    for (int h = 0; h < SPL; ++h) {
      const int js = j + 64 * h;
      walker[h] = (wave == 0) && (nbest ? (js < K && sc[h] != kNegInf) : (h == 0 && lane == 0));
      jb[h] = nbest ? js : best;
      cnext[h] = -1;
      orow[h] = nullptr;
      pos[h] = 0;
      if (walker[h]) {
        orow[h] = nbest ? nbt + static_cast<size_t>(s_row[KMX + js]) * T : ot;
        pos[h] = nbest ? len[h] : nout;
      }
    }
    for (int hi = L; hi > 0;) {
      const int lo = hi > tile_frames ? hi - tile_frames : 0;
      __syncthreads();
      const int n = (hi - lo) * K;
      const int32_t* src = bpb + static_cast<size_t>(lo) * K;
      for (int q = tid; q < n; q += kThreads) s_big[q] = static_cast<uint32_t>(src[q]);
      __syncthreads();
#pragma unroll
      for (int h = 0; h < SPL; ++h) {
        if (walker[h]) {
          for (int tt = hi - 1; tt >= lo; --tt) {
            const uint32_t e = s_big[(tt - lo) * K + jb[h]];
            const int cl = static_cast<int>(e & 0xFFFFu);
            const int par = static_cast<int>(e >> 16);
            if (tt < L - 1 && cnext[h] != V && cnext[h] != cl) {
              if (pos[h] > 0) {
                --pos[h];
                if (orow[h]) orow[h][pos[h]] = cnext[h];
              }
            }
            cnext[h] = cl;
            jb[h] = par;
          }
        }
      }
      hi = lo;
    }
    bool bad = false;
#pragma unroll
    for (int h = 0; h < SPL; ++h) {
      if (walker[h]) {
        if (cnext[h] != V && cnext[h] >= 0 && pos[h] > 0) {
          --pos[h];
          if (orow[h]) orow[h][pos[h]] = cnext[h];
        }
        bad = bad || pos[h] != 0;
      }
    }
    if (wave == 0 && __ballot(bad) != 0ull) status |= 2u;
  }
  }
  if (tid == 0) {
    p.status[b] = status;
    if (b == 0) write_ws_header(p.ws_header, p.B);
  }
}

template <int LPT, int NLEV, int SPL, bool SKIP, bool REP, bool TREE>
hipError_t launch_tree(const KernelParams& p, hipStream_t s) {
  dim3 grid(p.B), block(kThreads);
  constexpr bool kCacheable = SPL == 1 && !SKIP && LPT >= 2 && NLEV > 0;
  if constexpr (REP) {
    // the repeat-scoring variant reads uncached rows; with neither an LM nor
    // boosting it has nothing to repeat (the caller takes the default kernel)
    if (p.bt_nodes != nullptr) {
      hipLaunchKernelGGL((decode_kernel<LPT, NLEV, true, SPL, SKIP, false, true, TREE>), grid, block, 0, s, p);
    } else {
      if constexpr (NLEV < 0) return hipErrorInvalidValue;
      else hipLaunchKernelGGL((decode_kernel<LPT, NLEV, false, SPL, SKIP, false, true, TREE>), grid, block, 0, s, p);
    }
  } else if (p.bt_nodes != nullptr) {
    hipLaunchKernelGGL((decode_kernel<LPT, NLEV, true, SPL, SKIP, false, false, TREE>), grid, block, 0, s, p);
  } else if (kCacheable && p.lm_states_below_2p23 && !(p.flags & kFlagNoRowCache)) {
    hipLaunchKernelGGL((decode_kernel<LPT, NLEV, false, SPL, SKIP, kCacheable, false, TREE>), grid, block, 0, s, p);
  } else {
    hipLaunchKernelGGL((decode_kernel<LPT, NLEV, false, SPL, SKIP, false, false, TREE>), grid, block, 0, s, p);
  }
  return hipGetLastError();
}

template <int LPT, int NLEV, int SPL, bool SKIP, bool REP>
hipError_t launch_skip(const KernelParams& p, hipStream_t s) {
  // the merge-tree rank for beams of 33..64 over several chunks
  if constexpr (SPL == 1 && SKIP) {
    if (p.K > 32) return launch_tree<LPT, NLEV, SPL, SKIP, REP, true>(p, s);
  }
  return launch_tree<LPT, NLEV, SPL, SKIP, REP, false>(p, s);
}

template <int LPT, int NLEV, int SPL, bool REP>
hipError_t launch_nlev(const KernelParams& p, hipStream_t s) {
  // beams of more than one chunk (16 / LPT rows) skip ranks
  if constexpr (SPL > 1) {
    return launch_skip<LPT, NLEV, SPL, true, REP>(p, s);
  } else {
    if (p.K > 16 / LPT) return launch_skip<LPT, NLEV, SPL, true, REP>(p, s);
    return launch_skip<LPT, NLEV, SPL, false, REP>(p, s);
  }
}

template <int LPT, int SPL, bool REP>
hipError_t launch_spl(const KernelParams& p, hipStream_t s) {
  if (p.lm_states == nullptr && p.lm_arcs == nullptr) return launch_nlev<LPT, -1, SPL, REP>(p, s);
  switch (p.lm_nlev) {
    case 0: return launch_nlev<LPT, 0, SPL, REP>(p, s);
    case 1: return launch_nlev<LPT, 1, SPL, REP>(p, s);
    case 2: return launch_nlev<LPT, 2, SPL, REP>(p, s);
    case 3: return launch_nlev<LPT, 3, SPL, REP>(p, s);
    case 4: return launch_nlev<LPT, 4, SPL, REP>(p, s);
    case 5: return launch_nlev<LPT, 5, SPL, REP>(p, s);
    case 6: return launch_nlev<LPT, 6, SPL, REP>(p, s);
    case 7: return launch_nlev<LPT, 7, SPL, REP>(p, s);
    default: return hipErrorInvalidValue;
  }
}

// beams above 64 take two slots per lane (vocabularies of at most 1024
// tokens; the host rejects the rest)
template <int LPT, bool REP>
hipError_t launch_lpt_impl(const KernelParams& p, hipStream_t s) {
  if constexpr (LPT <= 2) {
    if (p.K > 64) return launch_spl<LPT, 2, REP>(p, s);
  } else {
    if (p.K > 64) return hipErrorInvalidValue;
  }
  return launch_spl<LPT, 1, REP>(p, s);
}

}  // namespace detail
}  // namespace ctcbeam
