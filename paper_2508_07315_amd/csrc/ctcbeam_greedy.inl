// Greedy CTC decoding with n-gram LM shallow fusion and phrase boosting
// (gfx950).  Included by the per-vocabulary instantiation units
// (ctcbeam_greedy_v*.hip).
//
// Greedy decoding with fusion is Algorithm 1 of FlexCTC with a single
// hypothesis (the greedy rows of Table II, Sec. V-A): at every
// frame the one beam is extended by the label with the best Eq. 1 score,
// formed with the same fp32 fold as the beam search,
//   x = s + D[c]; if c emits: x = ((x + beta) + fl(alpha*LM)) + fl(w*BT),
// ties broken towards the lower label index (blank = V last); a frame whose
// best score is -inf ends the hypothesis (empty output, score -inf).
// Pruning and recombination have no effect with one hypothesis.  LM.Final is
// added at the end.
//
// Design: one workgroup of NW wave64 per utterance (one wave up to 1024
// tokens, four above, where a wave alone would score 64 labels per lane; at
// 1024 tokens four waves measured slower: the per-frame exchange costs more
// than the narrower scoring saves).  The fused score of every
// label splits into a part that changes every frame (s + D) and per-label LM
// and boosting terms that change only when a token is emitted (the LM and
// boosting states move only then).  Those terms live in LDS arrays indexed by
// label, rebuilt on emission ("refill"): the unigram + backoff fold for every
// label, then the explicit continuations of the state's backoff chain
// scattered over it in ascending order of context length (the longest context
// wins), then the boosting continuation list over the root keys.
//
// With NW = 4 each wave owns a quarter of the labels and rebuilds only
// their terms: it loads every continuation tile of the chain (the same round
// trips as one wave alone, in parallel) and stores the ones of its labels in
// order, so every entry is written and read by one wave and a refill needs no
// workgroup barrier.  The one exchange per frame is the argmax: each wave
// publishes its best label with that label's successor states and terms, and
// every wave takes the winner after one barrier (double-buffered by frame).
// Log-prob rows are prefetched in batches of frames into registers,
// double-buffered, so the HBM latency is paid once per batch.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ctcbeam_internal.h"

namespace ctcbeam {
namespace greedy {

constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kTiles = 8;  // arc tiles of 64 loaded before their stores

// Order of LDS accesses between lanes of one wave: LDS operations of a wave
// complete in issue order, so a compiler-level fence is all that is needed.
__device__ __forceinline__ void wave_lds_fence() { __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront"); }

template <int CTRL>
__device__ __forceinline__ float dpp_shr(float v, float old) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ int dpp_shr_i(int v, int old) {
  return __builtin_amdgcn_update_dpp(old, v, CTRL, 0xF, 0xF, false);
}

// wave maximum (uniform result); -0 and +0 compare equal
__device__ __forceinline__ float wave_max(float v) {
  const float ni = kNegInf;
  float o;
  o = dpp_shr<0x111>(v, ni); v = (o > v) ? o : v;
  o = dpp_shr<0x112>(v, ni); v = (o > v) ? o : v;
  o = dpp_shr<0x114>(v, ni); v = (o > v) ? o : v;
  o = dpp_shr<0x118>(v, ni); v = (o > v) ? o : v;
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 15));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 31));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 47));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
  const float ab = (b > a) ? b : a, cd = (d > c) ? d : c;
  return (cd > ab) ? cd : ab;
}
// wave minimum of non-negative ints (uniform result)
__device__ __forceinline__ int wave_min(int v) {
  const int big = 0x7FFFFFFF;
  int o;
  o = dpp_shr_i<0x111>(v, big); v = min(v, o);
  o = dpp_shr_i<0x112>(v, big); v = min(v, o);
  o = dpp_shr_i<0x114>(v, big); v = min(v, o);
  o = dpp_shr_i<0x118>(v, big); v = min(v, o);
  const int a = __builtin_amdgcn_readlane(v, 15), b = __builtin_amdgcn_readlane(v, 31);
  const int c = __builtin_amdgcn_readlane(v, 47), d = __builtin_amdgcn_readlane(v, 63);
  return min(min(a, b), min(c, d));
}

// four consecutive fp32 at a 4-byte aligned address (one dwordx4 access)
typedef float f4u __attribute__((ext_vector_type(4), aligned(4)));

// Labels of a thread: threads own runs of 4 consecutive labels, runs of the
// workgroup are 4 * NT labels apart (NT threads), so a frame row is read with
// dwordx4 loads and the LDS arrays with 16-byte accesses.  Wave w owns the
// labels whose position within their run of the workgroup is 256 w .. 256 w
// + 255.
template <int NT>
__device__ __forceinline__ int label_of(int tid, int r) { return 4 * NT * (r >> 2) + 4 * tid + (r & 3); }
template <int NT>
__device__ __forceinline__ int thread_of(int c) { return (c % (4 * NT)) >> 2; }
template <int NT>
__device__ __forceinline__ int wave_of(int c) { return (c % (4 * NT)) >> 8; }

// a wave's best candidate with what the other waves need of it
struct __align__(16) Best {
  float x;       // fused score
  int32_t c;     // label
  uint32_t tg;   // LM state after emitting c
  uint32_t bk;   // boosting key of c
  float av, bv;  // its fl(alpha*LM) and fl(w*BT) terms
  uint32_t pad[2];
};

template <int NW, int NJ, int NLEV, bool HAS_BT, bool REP>
__global__ void __launch_bounds__(64 * NW) greedy_kernel(KernelParams p) {
  static_assert(NJ % 4 == 0, "labels per thread come in runs of 4");
  constexpr int NT = 64 * NW;              // threads
  constexpr bool HAS_LM = NLEV >= 0;
  constexpr int NL = NLEV > 0 ? NLEV : 0;  // chain levels above the unigram root
  constexpr int NLA = NL > 0 ? NL : 1;
  constexpr int NCAP = NT * NJ;            // token capacity
  constexpr int P = NJ >= 16 ? 4 : 8;      // frames per prefetch batch
  // per-label fusion terms of the current state, and the label's successor
  __shared__ __align__(16) float s_av[HAS_LM ? NCAP : 1];       // fl(alpha * LM(c | state))
  __shared__ __align__(16) uint32_t s_tg[HAS_LM ? NCAP : 1];    // LM state after emitting c
  __shared__ __align__(16) float s_p1[HAS_LM ? NCAP : 1];       // unigram ln P(c)
  __shared__ __align__(16) float s_bv[HAS_BT ? NCAP : 1];       // fl(w * BT(c | state))
  __shared__ __align__(16) uint32_t s_bk[HAS_BT ? NCAP : 1];    // boosting key of c
  __shared__ __align__(16) uint32_t s_root[HAS_BT ? NCAP : 1];  // root keys
  // per-frame argmax exchange between the waves (double-buffered)
  __shared__ Best s_best[2][NW];
  // emitted tokens, written to the output 256 at a time by wave 0 (a store
  // per token would hold the wave's next load wait)
  __shared__ int32_t s_tok[256];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int b = blockIdx.x;
  const int V = p.V, W = V + 1, T = p.T;
  const float alpha = p.alpha, beta = p.beta, boost_w = p.boost_w;
  int L = p.lengths[b];
  uint32_t status = 0;
  if (L < 0) { L = 0; status |= 1u; }
  if (L > T) { L = T; status |= 1u; }
  const float* Db = p.logprobs + static_cast<size_t>(b) * T * W;

#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int c = label_of<NT>(tid, j);
    if (HAS_LM) s_p1[c] = c < V ? p.lm_unigram[c] : 0.0f;
    if (HAS_BT) s_root[c] = c < V ? p.bt_root_key[c] : 0u;
  }

  // ---- the hypothesis (uniform over the workgroup) ----
  float s = 0.0f;
  int last = V, nout = 0;
  bool dead = false;
  LmLevel hl[NLA];
#pragma unroll
  for (int l = 0; l < NLA; ++l) hl[l] = LmLevel{0u, 0u, 0.0f};
  int pot = 0;
  // repeat-scoring variant: the terms the last emitted token received
  float ral = 0.0f, rwb = 0.0f;
  // successor states of the last emitted token
  uint32_t nlms = 0u, nbtn = 0u;
  int par = 0;  // exchange buffer of this frame
  int64_t st_ls = 0, st_la = 0, st_bn = 0, st_ba = 0, st_refill = 0, st_live = 0;
  int32_t* ot = p.out_tokens + static_cast<size_t>(b) * T;
  // profiling builds: cycles of scoring, the wave's best, the exchange
  // barrier, the decision, chain headers + fold, continuations, row loads;
  // then frames and refills
#ifdef CTCBEAM_PHASE_CLOCKS
  uint64_t ph_acc = 0ull;
  uint64_t ph_t0 = __builtin_amdgcn_s_memtime();
#endif

  // Rebuild this wave's per-label terms for LM state `lms` and boosting node
  // `btn`: chain headers, the unigram + backoff fold of every label, then the
  // continuations of this wave's labels stored over the fold in ascending
  // order of context length (the longest context wins), and the boosting
  // continuations over the root keys.
  auto refill = [&](uint32_t lms, uint32_t btn) __attribute__((always_inline)) {
    BtNode nd{0u, 0u, 0u, 0u};
    if (HAS_LM) {
#pragma unroll
      for (int l = 0; l < NL; ++l) hl[l] = p.lm_states[static_cast<size_t>(lms) * NL + l];
    }
    if (HAS_BT) nd = p.bt_nodes[btn];
    ++st_refill;
    CTCBEAM_PHASE_COUNT(10);
    if (HAS_LM) {
      // unigram + backoff fold of every label (innermost context first)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int c = label_of<NT>(tid, j);
        float v = s_p1[c];
#pragma unroll
        for (int l = 0; l < NL; ++l) v = v + hl[l].bo;
        s_av[c] = alpha * v;
        s_tg[c] = static_cast<uint32_t>(c);
      }
    }
    if (HAS_BT) {
      pot = static_cast<int>(nd.pot & 0xFFu);
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int c = label_of<NT>(tid, j);
        const uint32_t k = s_root[c];
        s_bk[c] = k;
        s_bv[c] = boost_w * static_cast<float>(static_cast<int>((k >> 20) & 63u) - pot);
      }
    }
    // Explicit continuations, level-major in ascending context length, cut
    // into tiles of 64; a block of kTiles tiles is loaded, then the entries
    // of this wave's labels are stored in order, so a longer context's value
    // overwrites a shorter one's.
    int tl[NLA + 1];  // first tile of each level, then the LM total
    int nt = 0;
#pragma unroll
    for (int l = 0; l < NL; ++l) {
      tl[l] = nt;
      const int n = static_cast<int>(hl[l].count & ~kExists);
      nt += (n + 63) >> 6;
      if (hl[l].count & kExists) ++st_ls;
      st_la += n;
    }
    tl[NL] = nt;
    CTCBEAM_PHASE_MARK(4);
    const int ntb = HAS_BT ? static_cast<int>((nd.list_count + 63u) >> 6) : 0;
    if (HAS_BT) {
      st_bn += nd.pot >> 8;
      st_ba += nd.chain_arcs;
    }
    // labels of this wave (every label with one wave)
    const auto mine = [&](uint32_t c) __attribute__((always_inline)) {
      return NW == 1 || wave_of<NT>(static_cast<int>(c)) == wave;
    };
    wave_lds_fence();
    for (int t0 = 0; t0 < nt + ntb; t0 += kTiles) {
      LmArc a[kTiles];
      BtEntry e[kTiles];
      int lvu[kTiles];
      bool ok[kTiles];
#pragma unroll
      for (int u = 0; u < kTiles; ++u) {
        const int tt = t0 + u;
        ok[u] = false;
        lvu[u] = -1;
        a[u] = LmArc{0.0f, 0u, 0xFFFFFFFFu};
        e[u] = BtEntry{0xFFFFFFFFu, 0u};
        if (HAS_LM && tt < nt) {  // uniform
          // the tile's level by a select chain (constant indices keep the
          // chain headers in registers)
          int lv = 0, t0l = tl[0];
          uint32_t lb = hl[0].begin, lc = hl[0].count & ~kExists;
#pragma unroll
          for (int l = 1; l < NL; ++l) {
            const bool in = tt >= tl[l];
            lv = in ? l : lv;
            t0l = in ? tl[l] : t0l;
            lb = in ? hl[l].begin : lb;
            lc = in ? (hl[l].count & ~kExists) : lc;
          }
          lvu[u] = lv;
          const uint32_t q = static_cast<uint32_t>((tt - t0l) * 64 + lane);
          ok[u] = q < lc;
          a[u] = p.lm_arcs[lb + (ok[u] ? q : 0u)];
        } else if (HAS_BT && tt < nt + ntb) {  // uniform
          const uint32_t q = static_cast<uint32_t>((tt - nt) * 64 + lane);
          ok[u] = q < nd.list_count;
          e[u] = p.bt_list[nd.list_begin + (ok[u] ? q : 0u)];
        }
      }
#pragma unroll
      for (int u = 0; u < kTiles; ++u) {
        if (HAS_LM && lvu[u] >= 0) {  // uniform
          const uint32_t c = a[u].token;
          if (ok[u] && c < static_cast<uint32_t>(V) && mine(c)) {
            // the backoff weights of the longer contexts, which lack this
            // token, in ascending order
            float v = a[u].logp;
#pragma unroll
            for (int l = 1; l < NL; ++l)
              if (l > lvu[u]) v = v + hl[l].bo;
            s_av[c] = alpha * v;
            s_tg[c] = a[u].target;
          }
        } else if (HAS_BT) {
          const uint32_t c = e[u].token;
          if (ok[u] && c < static_cast<uint32_t>(V) && mine(c)) {
            s_bk[c] = e[u].key;
            s_bv[c] = boost_w * static_cast<float>(static_cast<int>((e[u].key >> 20) & 63u) - pot);
          }
        }
      }
    }
    wave_lds_fence();
    CTCBEAM_PHASE_MARK(5);
  };

  // Score one frame; returns true when the winner emits a token (the caller
  // then refills).  Sets `dead` when every candidate is -inf.
  auto step = [&](const float (&d)[NJ], float dbl) -> bool {
    float xb = kNegInf;
    int jb = 0;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int c = label_of<NT>(tid, j);
      const float x0 = s + d[j];
      float x1 = x0 + beta;
      if (HAS_LM) x1 = x1 + s_av[c];
      if (HAS_BT) x1 = x1 + s_bv[c];
      const float x = (c != last) ? x1 : x0;
      if (x > xb) {
        xb = x;
        jb = j;
      }
    }
    if (REP && last != V && tid == thread_of<NT>(last)) {
      // the thread holding the repeated token takes its best again, with the
      // repeat scored x = ((s + D) + fl(alpha*LM)) + fl(w*BT)
      xb = kNegInf;
      jb = 0;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int c = label_of<NT>(tid, j);
        const float x0 = s + d[j];
        float x1 = x0 + beta;
        if (HAS_LM) x1 = x1 + s_av[c];
        if (HAS_BT) x1 = x1 + s_bv[c];
        float xr = x0;
        if (HAS_LM) xr = xr + ral;
        if (HAS_BT) xr = xr + rwb;
        const float x = (c != last) ? x1 : xr;
        if (x > xb) {
          xb = x;
          jb = j;
        }
      }
    }
    CTCBEAM_PHASE_MARK(0);
    // this wave's maximum; its best label (lowest index on ties) and that
    // label's own value (the maximum may differ from it in the sign of a
    // zero) are needed only when a label of this wave can beat the blank,
    // which has the largest index and wins only when strictly better
    const float g = wave_max(xb);
    const float xblank = s + dbl;
    const bool need = !(xblank > g) && g != kNegInf;  // uniform per wave
    int cw = V;
    float xw = kNegInf;
    if (need) {
      const uint64_t m = __ballot(xb == g);
      const int cl = label_of<NT>(tid, jb);
      if (__popcll(m) == 1) {
        cw = __builtin_amdgcn_readlane(cl, static_cast<int>(__builtin_ctzll(m)));
      } else {
        cw = wave_min((xb == g) ? cl : 0x7FFFFFFF);
      }
      // cw < NCAP is a label of this wave
      xw = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(xb), thread_of<NT>(cw) & 63));
    }
    uint32_t tgw = 0u, bkw = 0u;
    float avw = 0.0f, bvw = 0.0f;
    if constexpr (NW > 1) {
      if (lane == 0) {
        // this wave's candidate with its successor states and terms (entries
        // this wave wrote); a wave that cannot beat the blank offers its
        // maximum, which then cannot win either
        Best bw;
        bw.x = need ? xw : g;
        bw.c = need ? cw : 0x7FFFFFFF;
        bw.tg = (HAS_LM && need) ? s_tg[cw] : 0u;
        bw.bk = (HAS_BT && need) ? s_bk[cw] : 0u;
        bw.av = (HAS_LM && need) ? s_av[cw] : 0.0f;
        bw.bv = (HAS_BT && need) ? s_bv[cw] : 0.0f;
        s_best[par][wave] = bw;
      }
      CTCBEAM_PHASE_MARK(1);
      __syncthreads();
      CTCBEAM_PHASE_MARK(2);
      // the largest value, the lowest label on ties
      Best bb = s_best[par][0];
#pragma unroll
      for (int w = 1; w < NW; ++w) {
        const Best o = s_best[par][w];
        if (o.x > bb.x || (o.x == bb.x && o.c < bb.c)) bb = o;
      }
      par ^= 1;
      if (xblank > bb.x || bb.x == kNegInf) {
        cw = V;
        xw = xblank;
      } else {
        xw = bb.x;
        cw = bb.c;
        tgw = bb.tg;
        bkw = bb.bk;
        avw = bb.av;
        bvw = bb.bv;
      }
    } else if (!need) {
      cw = V;
      xw = xblank;
    }
    CTCBEAM_PHASE_COUNT(9);
    if (xw == kNegInf) {
      dead = true;
      return false;
    }
    s = xw;
    ++st_live;
    const bool emit = cw != V && cw != last;
    last = cw;
    if (emit && NW == 1) {
      // one wave: the winner's successor states and terms are its own entries
      tgw = HAS_LM ? s_tg[cw] : 0u;
      bkw = HAS_BT ? s_bk[cw] : 0u;
      avw = HAS_LM ? s_av[cw] : 0.0f;
      bvw = HAS_BT ? s_bv[cw] : 0.0f;
    }
    if (emit) {
      if (tid == 0) s_tok[nout & 255] = cw;
      ++nout;
      if ((nout & 255) == 0 && wave == 0) {  // uniform per wave
        wave_lds_fence();
#pragma unroll
        for (int i = 0; i < 4; ++i) ot[nout - 256 + lane + 64 * i] = s_tok[lane + 64 * i];
        wave_lds_fence();
      }
      nlms = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(tgw)));
      nbtn = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(bkw & kBtChildMask)));
      if (REP) {
        ral = avw;
        rwb = bvw;
      }
    }
    CTCBEAM_PHASE_MARK(3);
    return emit;
  };

  if (L > 0) {
    refill(HAS_LM ? p.lm_bos_state : 0u, 0u);
  } else if (HAS_LM) {
#pragma unroll
    for (int l = 0; l < NL; ++l) hl[l] = p.lm_states[static_cast<size_t>(p.lm_bos_state) * NL + l];
  }

  float qa[P][NJ], qb[P][NJ];
  float ua[P], ub[P];
  auto load_batch = [&](int t0, float (&q)[P][NJ], float (&u)[P]) {
#pragma unroll
    for (int f = 0; f < P; ++f) {
      if (t0 + f < L) {  // uniform
        const float* row = Db + static_cast<size_t>(t0 + f) * W;
#pragma unroll
        for (int j = 0; j < NJ; j += 4) {
          const int c = label_of<NT>(tid, j);
          // uniform per wave: the wave's whole run is in range
          if (4 * NT * (j >> 2) + 256 * wave + 255 < V) {
            const f4u v = __builtin_nontemporal_load(reinterpret_cast<const f4u*>(row + c));
            q[f][j] = v.x;
            q[f][j + 1] = v.y;
            q[f][j + 2] = v.z;
            q[f][j + 3] = v.w;
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) q[f][j + i] = c + i < V ? __builtin_nontemporal_load(row + c + i) : kNegInf;
          }
        }
        u[f] = __builtin_nontemporal_load(row + V);
      }
    }
    CTCBEAM_PHASE_MARK(6);
  };
  // frames t0 .. t0+P-1 from one batch; a refill restarts the unrolled scan
  // after the emitting frame
  auto run_batch = [&](int t0, const float (&q)[P][NJ], const float (&u)[P]) {
    int f0 = 0;
    while (f0 < P && !dead) {
      int fe = P;
#pragma unroll
      for (int f = 0; f < P; ++f) {
        if (f >= f0 && fe == P && !dead && t0 + f < L) {  // uniform
          if (step(q[f], u[f])) fe = f;
        }
      }
      if (fe == P) break;
      refill(nlms, nbtn);
      f0 = fe + 1;
    }
  };

  load_batch(0, qa, ua);
  for (int t0 = 0; t0 < L && !dead; t0 += 2 * P) {
    load_batch(t0 + P, qb, ub);
    run_batch(t0, qa, ua);
    if (dead || t0 + P >= L) break;
    load_batch(t0 + 2 * P, qa, ua);
    run_batch(t0 + P, qb, ub);
  }
  // ---- LM.Final and outputs ----
  if (!dead && HAS_LM) {
    // ln P(</s> | state) through the backoff chain; </s> is the last arc of
    // a state's sorted arcs when present
    float v = p.lm_unigram[V];
    int found = -1;
    float fv = 0.0f;
#pragma unroll
    for (int l = NL - 1; l >= 0; --l) {
      const uint32_t n = hl[l].count & ~kExists;
      if (found < 0 && n > 0) {
        const LmArc a = p.lm_arcs[hl[l].begin + n - 1];
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
        if (l > found) v = v + hl[l].bo;
    } else {
#pragma unroll
      for (int l = 0; l < NL; ++l) v = v + hl[l].bo;
    }
    s = s + alpha * v;
  }
  if (!dead && HAS_BT && (p.flags & kFlagBoostRollback)) {
    // the pending boosting of an unfinished phrase is taken back
    const float wb = boost_w * static_cast<float>(-pot);
    s = s + wb;
  }
  if (dead) {
    s = kNegInf;
    nout = 0;
  }
  if (wave == 0) {
    // the tokens since the last full block, then -1 padding (one wave writes
    // every entry of the row, so the stores of one address keep their order)
    wave_lds_fence();
    const int base = nout & ~255;
    for (int i = lane; i < (nout & 255); i += 64) ot[base + i] = s_tok[i];
    for (int tt = nout + lane; tt < T; tt += 64) ot[tt] = -1;
  }
#ifdef CTCBEAM_PHASE_CLOCKS
  if (p.stats && lane < kPhaseWords) {
    int64_t* pw = p.stats + static_cast<size_t>(p.B) * 8 + (static_cast<size_t>(b) * 8 + wave) * kPhaseWords;
    pw[lane] = static_cast<int64_t>(ph_acc);
  }
#endif
  if (tid == 0) {
    p.out_scores[b] = s;
    if (p.out_lengths) p.out_lengths[b] = nout;
    p.status[b] = status;
    if (b == 0) write_ws_header(p.ws_header, p.B);
    if (p.stats) {
      int64_t* so = p.stats + static_cast<size_t>(b) * 8;
      so[0] = L;
      so[1] = st_live;
      so[2] = st_ls;
      so[3] = st_la;
      so[4] = st_bn;
      so[5] = st_ba;
      so[6] = nout;
      so[7] = st_refill;
    }
  }
}

template <int NW, int NJ, int NLEV, bool REP>
hipError_t launch_greedy_nlev(const KernelParams& p, hipStream_t s) {
  dim3 grid(p.B), block(64 * NW);
  if (p.bt_nodes != nullptr)
    hipLaunchKernelGGL((greedy_kernel<NW, NJ, NLEV, true, REP>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((greedy_kernel<NW, NJ, NLEV, false, REP>), grid, block, 0, s, p);
  return hipGetLastError();
}

template <int NW, int NJ, bool REP>
hipError_t launch_greedy_rep(const KernelParams& p, hipStream_t s) {
  if (p.lm_states == nullptr && p.lm_arcs == nullptr) return launch_greedy_nlev<NW, NJ, -1, REP>(p, s);
  switch (p.lm_nlev) {
    case 0: return launch_greedy_nlev<NW, NJ, 0, REP>(p, s);
    case 1: return launch_greedy_nlev<NW, NJ, 1, REP>(p, s);
    case 2: return launch_greedy_nlev<NW, NJ, 2, REP>(p, s);
    case 3: return launch_greedy_nlev<NW, NJ, 3, REP>(p, s);
    case 4: return launch_greedy_nlev<NW, NJ, 4, REP>(p, s);
    case 5: return launch_greedy_nlev<NW, NJ, 5, REP>(p, s);
    case 6: return launch_greedy_nlev<NW, NJ, 6, REP>(p, s);
    case 7: return launch_greedy_nlev<NW, NJ, 7, REP>(p, s);
    default: return hipErrorInvalidValue;
  }
}

// NW waves of NJ labels per thread; the repeat-scoring variant (with an LM or
// boosting, which it needs to change anything) is a kernel of its own
template <int NW, int NJ>
hipError_t launch_greedy_impl(const KernelParams& p, hipStream_t s) {
  const bool rep = (p.flags & kFlagRepeatScore) &&
                   (p.lm_states != nullptr || p.lm_arcs != nullptr || p.bt_nodes != nullptr);
  return rep ? launch_greedy_rep<NW, NJ, true>(p, s) : launch_greedy_rep<NW, NJ, false>(p, s);
}

}  // namespace greedy
}  // namespace ctcbeam
