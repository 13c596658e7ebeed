// Greedy CTC decoding with n-gram LM shallow fusion and phrase boosting
// (gfx950).  Included by the per-NJ instantiation units
// (ctcbeam_greedy_nj*.hip).
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
// Design: one wave64 per utterance and no workgroup barriers.  The fused
// score of every label splits into a part that changes every frame (s + D)
// and per-label LM and boosting terms that change only when a token is
// emitted (the LM and boosting states move only then).  Those terms live in
// LDS arrays indexed by label, rebuilt on emission ("refill"): the unigram +
// backoff fold for every label, then the explicit continuations of the
// state's backoff chain scattered over it in ascending order of context
// length (the longest context wins), then the boosting continuation list over
// the root keys.  Blank and repeat frames -- most frames of a CTC posterior --
// cost one pass over the labels and a wave reduction.  Log-prob rows are
// prefetched in batches of 64/NJ frames into registers, double-buffered, so
// the HBM latency is paid once per batch.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ctcbeam_internal.h"

namespace ctcbeam {
namespace greedy {

constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kTiles = 8;  // arc tiles of 64 loaded before their stores

// Order of LDS accesses between lanes of the one wave: LDS operations of a
// wave complete in issue order, so a compiler-level fence is all that is
// needed.
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

// Label of a lane's r-th slot: lanes own runs of 4 consecutive labels, runs of
// the wave are 256 labels apart, so a frame row is read with dwordx4 loads
// and the LDS arrays with 16-byte accesses.
__device__ __forceinline__ int label_of(int lane, int r) { return 256 * (r >> 2) + 4 * lane + (r & 3); }
// the lane that owns label c
__device__ __forceinline__ int lane_of(int c) { return (c >> 2) & 63; }

template <int NJ, int NLEV, bool HAS_BT>
__global__ void __launch_bounds__(64) greedy_kernel(KernelParams p) {
  static_assert(NJ % 4 == 0, "labels per lane come in runs of 4");
  constexpr bool HAS_LM = NLEV >= 0;
  constexpr int NL = NLEV > 0 ? NLEV : 0;  // chain levels above the unigram root
  constexpr int NLA = NL > 0 ? NL : 1;
  constexpr int NCAP = 64 * NJ;            // token capacity
  constexpr int P = 64 / NJ;               // frames per prefetch batch
  // per-label fusion terms of the current state, and the label's successor
  __shared__ __align__(16) float s_av[HAS_LM ? NCAP : 1];       // fl(alpha * LM(c | state))
  __shared__ __align__(16) uint32_t s_tg[HAS_LM ? NCAP : 1];    // LM state after emitting c
  __shared__ __align__(16) float s_p1[HAS_LM ? NCAP : 1];       // unigram ln P(c)
  __shared__ __align__(16) float s_bv[HAS_BT ? NCAP : 1];       // fl(w * BT(c | state))
  __shared__ __align__(16) uint32_t s_bk[HAS_BT ? NCAP : 1];    // boosting key of c
  __shared__ __align__(16) uint32_t s_root[HAS_BT ? NCAP : 1];  // root keys

  const int lane = threadIdx.x;
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
    const int c = label_of(lane, j);
    if (HAS_LM) s_p1[c] = c < V ? p.lm_unigram[c] : 0.0f;
    if (HAS_BT) s_root[c] = c < V ? p.bt_root_key[c] : 0u;
  }

  // ---- the hypothesis (wave-uniform) ----
  float s = 0.0f;
  int last = V, nout = 0;
  bool dead = false;
  LmLevel hl[NLA];
#pragma unroll
  for (int l = 0; l < NLA; ++l) hl[l] = LmLevel{0u, 0u, 0.0f};
  int pot = 0;
  int64_t st_ls = 0, st_la = 0, st_bn = 0, st_ba = 0, st_refill = 0, st_live = 0;
  int32_t* ot = p.out_tokens + static_cast<size_t>(b) * T;

  // Rebuild the per-label terms for LM state `lms` and boosting node `btn`.
  auto refill = [&](uint32_t lms, uint32_t btn) __attribute__((always_inline)) {
    BtNode nd{0u, 0u, 0u, 0u};
    if (HAS_LM) {
#pragma unroll
      for (int l = 0; l < NL; ++l) hl[l] = p.lm_states[static_cast<size_t>(lms) * NL + l];
    }
    if (HAS_BT) nd = p.bt_nodes[btn];
    ++st_refill;
    if (HAS_LM) {
      // unigram + backoff fold of every label (innermost context first)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int c = label_of(lane, j);
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
        const int c = label_of(lane, j);
        const uint32_t k = s_root[c];
        s_bk[c] = k;
        s_bv[c] = boost_w * static_cast<float>(static_cast<int>((k >> 20) & 63u) - pot);
      }
    }
    // Explicit continuations, level-major in ascending context length, cut
    // into tiles of 64; a block of kTiles tiles is loaded, then stored in
    // order, so a longer context's value overwrites a shorter one's.
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
    const int ntb = HAS_BT ? static_cast<int>((nd.list_count + 63u) >> 6) : 0;
    if (HAS_BT) {
      st_bn += nd.pot >> 8;
      st_ba += nd.chain_arcs;
    }
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
          if (ok[u] && c < static_cast<uint32_t>(V)) {
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
          if (ok[u] && c < static_cast<uint32_t>(V)) {
            s_bk[c] = e[u].key;
            s_bv[c] = boost_w * static_cast<float>(static_cast<int>((e[u].key >> 20) & 63u) - pot);
          }
        }
      }
    }
    wave_lds_fence();
  };

  // repeat-scoring variant: the terms the last emitted token received
  const bool rep = (HAS_LM || HAS_BT) && (p.flags & kFlagRepeatScore) != 0;
  float ral = 0.0f, rwb = 0.0f;

  // Score one frame; returns true when the winner emits a token (the caller
  // then refills).  Sets `dead` when every candidate is -inf.
  auto step = [&](const float (&d)[NJ], float dbl) -> bool {
    float xb = kNegInf;
    int jb = 0;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int c = label_of(lane, j);
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
    if (rep && last != V && lane == lane_of(last)) {
      // the lane holding the repeated token takes its best again, with the
      // repeat scored x = ((s + D) + fl(alpha*LM)) + fl(w*BT)
      xb = kNegInf;
      jb = 0;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int c = label_of(lane, j);
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
    const float g = wave_max(xb);
    const float xblank = s + dbl;
    int cw;
    float xw;
    if (xblank > g || g == kNegInf) {
      // blank has the largest index: it wins only when strictly better
      cw = V;
      xw = xblank;
    } else {
      const uint64_t m = __ballot(xb == g);
      const int cl = label_of(lane, jb);
      if (__popcll(m) == 1) {
        cw = __builtin_amdgcn_readlane(cl, static_cast<int>(__builtin_ctzll(m)));
      } else {
        cw = wave_min((xb == g) ? cl : 0x7FFFFFFF);
      }
      // the winner's own value (g may differ from it in the sign of a zero)
      xw = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(xb), lane_of(cw)));
    }
    if (xw == kNegInf) {
      dead = true;
      return false;
    }
    s = xw;
    ++st_live;
    const bool emit = cw != V && cw != last;
    last = cw;
    if (emit) {
      if (lane == 0) ot[nout] = cw;
      ++nout;
      if (rep) {
        // read before the refill replaces the per-label terms
        if (HAS_LM) ral = s_av[cw];
        if (HAS_BT) rwb = s_bv[cw];
      }
    }
    return emit;
  };
  // successor states of an emitted token (read before the refill overwrites)
  auto next_states = [&](uint32_t& lms, uint32_t& btn) __attribute__((always_inline)) {
    lms = HAS_LM ? static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(s_tg[last]))) : 0u;
    btn = HAS_BT ? static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(s_bk[last] & kBtChildMask)))
                 : 0u;
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
          const int c = label_of(lane, j);
          if (256 * (j >> 2) + 255 < V) {  // uniform: the whole run of the wave is in range
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
      uint32_t lms, btn;
      next_states(lms, btn);
      refill(lms, btn);
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
  for (int tt = nout + lane; tt < T; tt += 64) ot[tt] = -1;
  if (lane == 0) {
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

template <int NJ, int NLEV>
hipError_t launch_greedy_nlev(const KernelParams& p, hipStream_t s) {
  dim3 grid(p.B), block(64);
  if (p.bt_nodes != nullptr)
    hipLaunchKernelGGL((greedy_kernel<NJ, NLEV, true>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((greedy_kernel<NJ, NLEV, false>), grid, block, 0, s, p);
  return hipGetLastError();
}

template <int NJ>
hipError_t launch_greedy_impl(const KernelParams& p, hipStream_t s) {
  if (p.lm_states == nullptr && p.lm_arcs == nullptr) return launch_greedy_nlev<NJ, -1>(p, s);
  switch (p.lm_nlev) {
    case 0: return launch_greedy_nlev<NJ, 0>(p, s);
    case 1: return launch_greedy_nlev<NJ, 1>(p, s);
    case 2: return launch_greedy_nlev<NJ, 2>(p, s);
    case 3: return launch_greedy_nlev<NJ, 3>(p, s);
    case 4: return launch_greedy_nlev<NJ, 4>(p, s);
    case 5: return launch_greedy_nlev<NJ, 5>(p, s);
    case 6: return launch_greedy_nlev<NJ, 6>(p, s);
    case 7: return launch_greedy_nlev<NJ, 7>(p, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace greedy
}  // namespace ctcbeam
