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
// utterance is one persistent workgroup of 8 wave64 that keeps every beam's
// state in LDS and loops over its own frames with no host round trip.  The
// B utterances are independent workgroups.  There is no dense contraction:
// the work is gathers of LM arcs, VALU scoring and a selection, bound by
// memory latency, LDS traffic and VALU issue, so MFMA is not used.
//
// Per frame (single chunk when K*V fits the LDS key rows, e.g. K=8, V=1024):
//   1. the next frame's log-prob row is prefetched into registers (lane owns
//      labels c = tid + j*512);
//   2. fill: one wave per live beam gathers the explicit continuations of
//      every state of its LM backoff chain (all loads of a beam issued before
//      the first use, so one memory latency covers the chain) and scatters
//      them into an LDS [beam][token] key row with atomicMax on
//      (order << 28 | staging slot): the highest-order n-gram wins with no
//      barrier between orders; boosting continuations (merged per tree state
//      on the host) are stored the same way;
//   3. candidates: each lane scores its labels for every beam in registers,
//      resolving the LM value from the key row or from the unigram + backoff
//      fold (compile-time LM order);
//   4. selection: the K-th largest of 64 lane maxima (each wave sorts its
//      lane maxima in registers, every wave then sorts the union of the waves'
//      top 8) is a lower bound on the K-th best candidate; it filters K*V
//      candidates down to a few dozen survivors in LDS;
//   5. wave 0 sorts the survivors in registers (bitonic, score desc / index
//      asc), prefetching the chain headers of every emitting survivor before
//      the sort, then prunes, advances the beams (hash of the collapsed
//      transcript, LM/boost states), recombines duplicates and builds the next
//      frame's live list; the other waves clear the key rows meanwhile.
//      Back-pointers go to HBM.
// Large beams (K*V above the key rows) run the fill/score/filter per chunk of
// beams with a running bound and compaction.  Rare overflows of the survivor
// buffer fall back to an exact extraction.  After the last frame the best
// beam is traced back through the back-pointers staged in LDS.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ctcbeam_internal.h"

namespace ctcbeam {
namespace detail {

constexpr float kNegInf = -__builtin_huge_valf();

// LDS scratch carved from one block so the traceback can reuse it.
constexpr int kBigWords = 2 * kKeyWords + 3 * kLmStage + kBtStage;
constexpr int kOffLmKey = 0;
constexpr int kOffBtKey = kKeyWords;
constexpr int kOffStV = 2 * kKeyWords;
constexpr int kOffStTgt = kOffStV + kLmStage;
constexpr int kOffStKey = kOffStTgt + kLmStage;
constexpr int kOffBtClr = kOffStKey + kLmStage;
// label survivors may fill the buffer up to kChunkCap; the remaining kMaxK
// entries always take the blank candidates
constexpr int kChunkCap = kCap - kMaxK;
constexpr int kFillUnroll = 16;

__device__ __forceinline__ uint64_t mix_token(uint64_t h, uint32_t c) {
  uint64_t z = h + (static_cast<uint64_t>(c) + 1ull) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Order key: larger is better; (x desc, idx asc); -0 and +0 compare equal.
__device__ __forceinline__ uint64_t order_key(float x, uint32_t idx) {
  const float y = x + 0.0f;
  uint32_t u = __float_as_uint(y);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return (static_cast<uint64_t>(u) << 32) | static_cast<uint64_t>(0xFFFFFFFFu - idx);
}

__device__ __forceinline__ bool beats(float xf, uint32_t if_, float xe, uint32_t ie) {
  return (xf > xe) || (xf == xe && if_ < ie);
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const uint32_t lane = threadIdx.x & 63u;
  return lane == 0 ? 0ull : (~0ull >> (64u - lane));
}

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// ---- cross-lane exchange on gfx950 without the LDS crossbar ----
// DPP row/quad patterns for distances 1..8 and the gfx950 permlane swaps for
// 16 and 32.  update_dpp with bound_ctrl off returns `old` (0) for lanes whose
// source lies outside the row.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ float dpp_movf(float v, float old) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppQuadXor1 = 0xB1;  // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;  // quad_perm [2,3,0,1]
constexpr int kDppRowShl4 = 0x104;
constexpr int kDppRowShr1 = 0x111;
constexpr int kDppRowShr2 = 0x112;
constexpr int kDppRowShr4 = 0x114;
constexpr int kDppRowShr8 = 0x118;
constexpr int kDppRowRor8 = 0x128;

// value of lane (lane ^ j); j must be a compile-time power of two <= 32 after
// unrolling
__device__ __forceinline__ uint32_t xor_lane(uint32_t v, int j, int lane) {
  switch (j) {
    case 1: return dpp_mov<kDppQuadXor1>(v);
    case 2: return dpp_mov<kDppQuadXor2>(v);
    case 4: {
      const uint32_t up = dpp_mov<kDppRowShl4>(v);
      const uint32_t dn = dpp_mov<kDppRowShr4>(v);
      return (lane & 4) ? dn : up;
    }
    case 8: return dpp_mov<kDppRowRor8>(v);
    case 16: {
      const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
      return (lane & 16) ? static_cast<uint32_t>(r[0]) : static_cast<uint32_t>(r[1]);
    }
    default: {
      const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
      return (lane & 32) ? static_cast<uint32_t>(r[0]) : static_cast<uint32_t>(r[1]);
    }
  }
}
__device__ __forceinline__ float xor_lane(float v, int j, int lane) {
  return __uint_as_float(xor_lane(__float_as_uint(v), j, lane));
}
__device__ __forceinline__ int xor_lane(int v, int j, int lane) {
  return static_cast<int>(xor_lane(static_cast<uint32_t>(v), j, lane));
}

// inclusive prefix sum over the wave
__device__ __forceinline__ int wave_incl_scan(int v, int lane) {
  v += static_cast<int>(dpp_mov<kDppRowShr1>(static_cast<uint32_t>(v)));
  v += static_cast<int>(dpp_mov<kDppRowShr2>(static_cast<uint32_t>(v)));
  v += static_cast<int>(dpp_mov<kDppRowShr4>(static_cast<uint32_t>(v)));
  v += static_cast<int>(dpp_mov<kDppRowShr8>(static_cast<uint32_t>(v)));
  const int r0 = __builtin_amdgcn_readlane(v, 15);
  const int r1 = __builtin_amdgcn_readlane(v, 31);
  const int r2 = __builtin_amdgcn_readlane(v, 47);
  v += (lane >= 16 ? r0 : 0) + (lane >= 32 ? r1 : 0) + (lane >= 48 ? r2 : 0);
  return v;
}

// maximum over each 16-lane row, valid in the row's last lane
__device__ __forceinline__ float row_max_last(float v) {
  const float ni = -__builtin_huge_valf();
  v = fmaxf(v, dpp_movf<kDppRowShr1>(v, ni));
  v = fmaxf(v, dpp_movf<kDppRowShr2>(v, ni));
  v = fmaxf(v, dpp_movf<kDppRowShr4>(v, ni));
  v = fmaxf(v, dpp_movf<kDppRowShr8>(v, ni));
  return v;
}

// maximum over each 8-lane group, valid in every lane of the group
__device__ __forceinline__ float group8_max(float v, int lane) {
  v = fmaxf(v, xor_lane(v, 1, lane));
  v = fmaxf(v, xor_lane(v, 2, lane));
  v = fmaxf(v, xor_lane(v, 4, lane));
  return v;
}

// Bitonic sort of one value per lane within groups of N lanes, descending.
template <int N>
__device__ __forceinline__ float wave_sort_desc(float v, int lane) {
#pragma unroll
  for (int k = 2; k <= N; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const float o = xor_lane(v, j, lane);
      const bool desc = (lane & k) == 0 || k == N;
      const bool lower = (lane & j) == 0;
      v = (lower == desc) ? fmaxf(v, o) : fminf(v, o);
    }
  }
  return v;
}

template <int LPT, int NLEV, bool HAS_BT>
__global__ void __launch_bounds__(kThreads) decode_kernel(KernelParams p) {
  constexpr bool HAS_LM = NLEV >= 0;
  constexpr int NL = NLEV > 0 ? NLEV : 0;     // chain levels above the unigram root
  constexpr int NLA = NL > 0 ? NL : 1;        // array extent
  constexpr int KCR = 16 / LPT;               // beams per chunk held in registers

  __shared__ __align__(16) uint32_t s_big[kBigWords];
  // survivor buffer
  __shared__ float s_bx[kCap];
  __shared__ uint32_t s_bi[kCap], s_blm[kCap], s_bbt[kCap];
  // ranked selection (fallback path and large-beam compaction)
  __shared__ float s_nx[kMaxK];
  __shared__ uint32_t s_ni[kMaxK], s_nlm[kMaxK], s_nbt[kMaxK];
  // beams
  __shared__ float s_score[kMaxK];
  __shared__ int32_t s_last[kMaxK], s_len[kMaxK];
  __shared__ uint64_t s_hash[kMaxK];
  __shared__ uint32_t s_lms[kMaxK], s_bts[kMaxK];
  __shared__ uint32_t s_lvb[kMaxK][NLA], s_lvc[kMaxK][NLA];
  __shared__ float s_lvbo[kMaxK][NLA];
  __shared__ uint32_t s_btb[kMaxK], s_btc[kMaxK];
  __shared__ int32_t s_btpot[kMaxK];
  // live list and chunks (positions in the live list)
  __shared__ int32_t s_alive[kMaxK];
  __shared__ int32_t s_hoff[kMaxK + 1], s_boff[kMaxK + 1];
  __shared__ int32_t s_chunk[kMaxK + 1];
  __shared__ int32_t s_nchunk;
  // selection
  __shared__ float s_top[kWaves * 8];
  __shared__ int32_t s_order[kMaxK];
  __shared__ uint64_t s_rkh[kMaxK];
  __shared__ uint32_t s_rkm[kMaxK];
  __shared__ uint64_t s_red[2][kWaves];
  __shared__ int32_t s_nbuf, s_overflow;
  __shared__ int32_t s_best;
  __shared__ float s_bestscore;

  uint32_t* const lmkey = s_big + kOffLmKey;
  uint32_t* const btkey = s_big + kOffBtKey;
  float* const stv = reinterpret_cast<float*>(s_big + kOffStV);
  uint32_t* const sttgt = s_big + kOffStTgt;
  uint32_t* const stkey = s_big + kOffStKey;
  uint32_t* const btclr = s_big + kOffBtClr;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int b = blockIdx.x;
  const int V = p.V, W = V + 1, K = p.K, T = p.T;
  const int kcmax = min(K, KCR);
  const float alpha = p.alpha, beta = p.beta, boost_w = p.boost_w;

  int L = p.lengths[b];
  uint32_t status = 0;
  if (L < 0) { L = 0; status |= 1u; }
  if (L > T) { L = T; status |= 1u; }
  const float* Db = p.logprobs + static_cast<size_t>(b) * T * W;
  int32_t* bpb = p.bp + static_cast<size_t>(b) * T * K;

  // ---- per-lane constants and the first row ----
  float rD[LPT], rDn[LPT], rP1[LPT];
  uint32_t rRoot[LPT];
#pragma unroll
  for (int j = 0; j < LPT; ++j) {
    const int c = tid + j * kThreads;
    const bool ok = c < V;
    rP1[j] = (HAS_LM && ok) ? p.lm_unigram[c] : 0.0f;
    rRoot[j] = (HAS_BT && ok) ? p.bt_root_key[c] : 0u;
    rDn[j] = (ok && L > 0) ? Db[c] : 0.0f;
    rD[j] = 0.0f;
  }
  float rBlankN = (L > 0 && tid < K) ? Db[V] : 0.0f;
  float rBlank = 0.0f;

  // statistics (wave 0, lane = slot)
  int64_t st_alive = 0, st_lms = 0, st_lma = 0, st_btn = 0, st_bta = 0, st_emit = 0;

  // ---- initial beams and their chain headers (wave 0, lane j = slot j) ----
  if (wave == 0) {
    const int j = lane;
    const bool alive = (j == 0);
    int32_t acnt = 0, bcnt = 0;
    if (j < K) {
      s_score[j] = (j == 0) ? 0.0f : kNegInf;
      s_last[j] = V;
      s_len[j] = 0;
      s_hash[j] = 0ull;
      s_lms[j] = HAS_LM ? p.lm_bos_state : 0u;
      s_bts[j] = 0u;
#pragma unroll
      for (int l = 0; l < NLA; ++l) {
        s_lvb[j][l] = 0u;
        s_lvc[j][l] = 0u;
        s_lvbo[j][l] = 0.0f;
      }
      if (HAS_LM && alive) {
#pragma unroll
        for (int l = 0; l < NL; ++l) {
          const LmLevel h = p.lm_states[static_cast<size_t>(p.lm_bos_state) * NL + l];
          s_lvb[j][l] = h.begin;
          s_lvc[j][l] = h.count;
          s_lvbo[j][l] = h.bo;
          acnt += static_cast<int32_t>(h.count & ~kExists);
          if (L > 0 && (h.count & kExists)) {
            st_lms += 1;
            st_lma += h.count & ~kExists;
          }
        }
      }
      if (HAS_BT) {
        const BtNode nd = p.bt_nodes[0];
        s_btb[j] = nd.list_begin;
        s_btc[j] = nd.list_count;
        s_btpot[j] = static_cast<int32_t>(nd.pot & 0xFFu);
        if (alive) bcnt = static_cast<int32_t>(nd.list_count);
      } else {
        s_btpot[j] = 0;
      }
    }
    if (alive && L > 0) st_alive += 1;
    if (j == 0) {
      s_alive[0] = 0;
      s_hoff[0] = 0;
      s_hoff[1] = acnt;
      s_boff[0] = 0;
      s_boff[1] = bcnt;
      s_chunk[0] = 0;
      s_chunk[1] = 1;
      s_nchunk = 1;
      s_nbuf = 0;
      s_overflow = 0;
    }
    if (j < K) {
      s_bx[kChunkCap + j] = kNegInf;
      s_bi[kChunkCap + j] = 0xFFFFFFFFu;
    }
  }
  for (int i = tid; i < kKeyWords; i += kThreads) {
    if (HAS_LM) lmkey[i] = 0u;
    if (HAS_BT) btkey[i] = 0u;
  }
  __syncthreads();

  for (int t = 0; t < L; ++t) {
    // ---- 1. rotate and prefetch the log-prob row ----
#pragma unroll
    for (int j = 0; j < LPT; ++j) rD[j] = rDn[j];
    rBlank = rBlankN;
    if (t + 1 < L) {
      const float* row = Db + static_cast<size_t>(t + 1) * W;
#pragma unroll
      for (int j = 0; j < LPT; ++j) {
        const int c = tid + j * kThreads;
        if (c < V) rDn[j] = __builtin_nontemporal_load(row + c);
      }
      if (tid < K) rBlankN = __builtin_nontemporal_load(row + V);
    }
    // s_nbuf, s_overflow and the reserved blank slots were reset by the
    // previous frame's update (or the initialisation)
    float tau = kNegInf;
    const int nchunk = s_nchunk;

    for (int ch = 0; ch < nchunk; ++ch) {
      const int cs = s_chunk[ch];
      const int kc = s_chunk[ch + 1] - cs;
      const int hbase = s_hoff[cs];
      const int bbase = s_boff[cs];
      const int lm_total = min(s_hoff[cs + kc] - hbase, kLmStage);
      const int bt_total = min(s_boff[cs + kc] - bbase, kBtStage);

      // ---- 2. fill: one wave per beam ----
      for (int i = wave; i < kc; i += kWaves) {
        const int k = s_alive[cs + i];
        const uint32_t rowbase = static_cast<uint32_t>(i) * static_cast<uint32_t>(V);
        if (HAS_LM && NL > 0) {
          const int hoff = s_hoff[cs + i] - hbase;
          uint32_t lb[NLA], lend[NLA];
          float lbo[NLA];
          uint32_t run = 0;
#pragma unroll
          for (int l = 0; l < NL; ++l) {
            lb[l] = s_lvb[k][l];
            run += s_lvc[k][l] & ~kExists;
            lend[l] = run;
            lbo[l] = s_lvbo[k][l];
          }
          const int total = static_cast<int>(run);
          for (int r0 = 0; r0 < total; r0 += 64 * kFillUnroll) {
            LmArc a[kFillUnroll];
            int lv[kFillUnroll];
#pragma unroll
            for (int u = 0; u < kFillUnroll; ++u) {
              lv[u] = -1;
              if (r0 + u * 64 >= total) continue;  // wave-uniform
              const uint32_t q = static_cast<uint32_t>(r0 + u * 64 + lane);
              int l = 0;
              uint32_t start = 0, base = lb[0];
#pragma unroll
              for (int m = 0; m + 1 < NL; ++m) {
                if (q >= lend[m]) {
                  l = m + 1;
                  start = lend[m];
                  base = lb[m + 1];
                }
              }
              const bool ok = q < static_cast<uint32_t>(total);
              lv[u] = ok ? l : -1;
              a[u] = p.lm_arcs[ok ? base + (q - start) : lb[0]];
            }
#pragma unroll
            for (int u = 0; u < kFillUnroll; ++u) {
              if (r0 + u * 64 >= total) continue;  // wave-uniform
              if (lv[u] >= 0) {
                const int q = r0 + u * 64 + lane;
                float v = a[u].logp;
#pragma unroll
                for (int l2 = 1; l2 < NL; ++l2)
                  if (l2 > lv[u]) v = v + lbo[l2];
                const float av = alpha * v;
                const int pos = hoff + q;
                // </s> (token V) is never a frame label; it is read at the end
                const bool tok_ok = a[u].token < static_cast<uint32_t>(V) && pos < kLmStage;
                const uint32_t kidx = rowbase + (tok_ok ? a[u].token : 0u);
                if (pos < kLmStage) {
                  stv[pos] = av;
                  sttgt[pos] = a[u].target;
                  stkey[pos] = kidx;
                }
                if (tok_ok)
                  atomicMax(&lmkey[kidx], (static_cast<uint32_t>(lv[u] + 1) << 28) | static_cast<uint32_t>(pos));
              }
            }
          }
        }
        if (HAS_BT) {
          const int boff = s_boff[cs + i] - bbase;
          const uint32_t lbeg = s_btb[k];
          const int cnt = static_cast<int>(s_btc[k]);
          for (int r0 = 0; r0 < cnt; r0 += 64 * 4) {
            BtEntry e[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int q = r0 + u * 64 + lane;
              e[u] = p.bt_list[lbeg + (q < cnt ? q : 0)];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int q = r0 + u * 64 + lane;
              if (q < cnt && boff + q < kBtStage) {
                const uint32_t kidx = rowbase + e[u].token;
                btkey[kidx] = e[u].key;
                btclr[boff + q] = kidx;
              }
            }
          }
        }
      }
      __syncthreads();
      // stable until the filter below appends (nobody writes s_nbuf between
      // the barrier above and the barrier that follows the bound)
      const int nbuf_before = s_nbuf;

      // ---- 3. candidates ----
      // beam i of the chunk lives in lane i; its data is broadcast per beam
      // with readlane so the scoring below is straight-line code
      const int hrow = lane < kc ? lane : 0;
      const int hk = s_alive[cs + hrow];
      const float hsc = lane < kc ? s_score[hk] : kNegInf;
      const int hlast = s_last[hk];
      float hbo[NLA];
#pragma unroll
      for (int l = 0; l < NL; ++l) hbo[l] = s_lvbo[hk][l];
      const int hpot = HAS_BT ? s_btpot[hk] : 0;
      float cand[16];
      int kslot[KCR];
      float lmax = kNegInf;
#pragma unroll
      for (int i = 0; i < KCR; ++i) {
        kslot[i] = __builtin_amdgcn_readlane(hk, i);
        const float sk = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(hsc), i));
        const int lastk = __builtin_amdgcn_readlane(hlast, i);
        float bo[NLA];
#pragma unroll
        for (int l = 0; l < NL; ++l) bo[l] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(hbo[l]), i));
        const int potk = HAS_BT ? __builtin_amdgcn_readlane(hpot, i) : 0;
#pragma unroll
        for (int j = 0; j < LPT; ++j) {
          const int c = tid + j * kThreads;
          // beams beyond the chunk score -inf (sk = -inf)
          const float x0 = sk + rD[j];
          float x1 = x0 + beta;
          if (HAS_LM) {
            const uint32_t key = lmkey[i * V + c];
            const float sv = stv[key & 0x0FFFFFFFu];
            float v = rP1[j];
#pragma unroll
            for (int l = 0; l < NL; ++l) v = v + bo[l];
            const float av = (key != 0u) ? sv : alpha * v;
            x1 = x1 + av;
          }
          if (HAS_BT) {
            uint32_t bk = btkey[i * V + c];
            bk = (bk != 0u) ? bk : rRoot[j];
            const int pre = static_cast<int>((bk >> 20) & 63u);
            const float bv = boost_w * static_cast<float>(pre - potk);
            x1 = x1 + bv;
          }
          float x = (c != lastk) ? x1 : x0;
          x = (c < V) ? x : kNegInf;
          cand[i * LPT + j] = x;
          lmax = fmaxf(lmax, x);
        }
      }

      // ---- 4a. lower bound on the K-th best ----
      // Maxima of disjoint lane groups are distinct candidates, so the K-th
      // largest of at least K group maxima bounds the K-th best candidate
      // from below.  K <= 32: the 32 rows of 16 lanes; otherwise 64 groups of
      // 8 lanes.
      {
        if (K <= 32) {
          const float g = row_max_last(lmax);
          if ((lane & 15) == 15) s_top[wave * 4 + (lane >> 4)] = g;
        } else {
          const float g = group8_max(lmax, lane);
          if ((lane & 7) == 7) s_top[wave * 8 + (lane >> 3)] = g;
        }
      }
      __syncthreads();
      {
        float tc;
        if (K <= 32) {
          const float v = wave_sort_desc<32>(lane < 32 ? s_top[lane] : kNegInf, lane);
          tc = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), K - 1));
        } else {
          const float v = wave_sort_desc<64>(s_top[lane], lane);
          tc = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), K - 1));
        }
        tau = fmaxf(tau, tc);
      }

      // ---- 4b. filter and append survivors (and, once, the blank candidates) ----
      {
        const bool last_chunk_f = (ch + 1 == nchunk);
        uint32_t qmask = 0u;
#pragma unroll
        for (int r = 0; r < 16; ++r) qmask |= (cand[r] >= tau && cand[r] != kNegInf) ? (1u << r) : 0u;
        const int mycnt = __popc(qmask);
        const int incl = wave_incl_scan(mycnt, lane);
        const int wtotal = __builtin_amdgcn_readlane(incl, 63);
        int wbase = 0;
        if (lane == 0 && wtotal > 0) wbase = atomicAdd(&s_nbuf, wtotal);
        wbase = __builtin_amdgcn_readfirstlane(wbase);
        if (wtotal > 0) {
          int slot = wbase + incl - mycnt;
          uint32_t rem = qmask;
          while (__ballot(rem != 0u)) {  // wave-uniform: max survivors of a lane
            if (rem != 0u) {
              const int r = __builtin_ctz(rem);
              rem &= rem - 1u;
              float x = cand[0];
#pragma unroll
              for (int rr = 1; rr < 16; ++rr) x = (r == rr) ? cand[rr] : x;
              const int i = r / LPT, j = r % LPT;
              const int c = tid + j * kThreads;
              int k = kslot[0];
#pragma unroll
              for (int ii = 1; ii < KCR; ++ii) k = (i == ii) ? kslot[ii] : k;
              uint32_t root = rRoot[0];
#pragma unroll
              for (int jj = 1; jj < LPT; ++jj) root = (j == jj) ? rRoot[jj] : root;
              if (slot < kChunkCap) {
                uint32_t lmt = 0u, bk = 0u;
                if (HAS_LM) {
                  const uint32_t kl = lmkey[i * V + c];
                  // the last chunk leaves the staged target to the selection
                  // (the staging survives until the next fill)
                  lmt = last_chunk_f ? (kl != 0u ? (kl | 0x80000000u) : static_cast<uint32_t>(c))
                                     : (kl != 0u ? sttgt[kl & 0x0FFFFFFFu] : static_cast<uint32_t>(c));
                }
                if (HAS_BT) {
                  const uint32_t kb = btkey[i * V + c];
                  bk = kb != 0u ? kb : root;
                }
                s_bx[slot] = x;
                s_bi[slot] = static_cast<uint32_t>(k * W + c);
                s_blm[slot] = lmt;
                s_bbt[slot] = bk;
              } else {
                s_overflow = 1;
              }
              ++slot;
            }
          }
        }
        if (ch == 0 && tid < K) {
          const float sk = s_score[tid];
          const float x = sk + rBlank;
          if (sk != kNegInf && x != kNegInf && x >= tau) {
            const int bs = kChunkCap + tid;  // reserved blank slots
            s_bx[bs] = x;
            s_bi[bs] = static_cast<uint32_t>(tid * W + V);
            s_blm[bs] = 0u;
            s_bbt[bs] = 0u;
          }
        }
      }
      __syncthreads();

      // ---- 4c. overflow: exact extraction over (buffer before) U (chunk) ----
      if (s_overflow) {
        uint64_t prev = ~0ull;
        int nk = 0;
        for (int it = 0; it < K; ++it) {
          uint64_t best = 0ull;
          int who = -1;  // -1 none, 0..15 register, 100+e buffer
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            if (cand[r] != kNegInf) {
              const int i = r / LPT, j = r % LPT;
              const int c = tid + j * kThreads;
              const int k = s_alive[cs + i];
              const uint64_t key = order_key(cand[r], static_cast<uint32_t>(k * W + c));
              if (key < prev && key > best) { best = key; who = r; }
            }
          }
          for (int e = tid; e < nbuf_before; e += kThreads) {
            const uint64_t key = order_key(s_bx[e], s_bi[e]);
            if (key < prev && key > best) { best = key; who = 100 + e; }
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
              const int r = who;
              const int i = r / LPT, j = r % LPT;
              const int c = tid + j * kThreads;
              const int k = s_alive[cs + i];
              uint32_t lmt = 0u, bk = 0u;
              if (HAS_LM) {
                const uint32_t key = lmkey[i * V + c];
                lmt = (key != 0u) ? sttgt[key & 0x0FFFFFFFu] : static_cast<uint32_t>(c);
              }
              if (HAS_BT) {
                bk = btkey[i * V + c];
                if (bk == 0u) bk = rRoot[j];
              }
              s_nx[it] = cand[r];
              s_ni[it] = static_cast<uint32_t>(k * W + c);
              s_nlm[it] = lmt;
              s_nbt[it] = bk;
            } else {
              const int e = who - 100;
              uint32_t lmt = s_blm[e];
              if (HAS_LM && (lmt & 0x80000000u)) lmt = sttgt[lmt & 0x0FFFFFFFu];
              s_nx[it] = s_bx[e];
              s_ni[it] = s_bi[e];
              s_nlm[it] = lmt;
              s_nbt[it] = s_bbt[e];
            }
          }
          prev = gbest;
          ++nk;
        }
        __syncthreads();
        for (int e = tid; e < nk; e += kThreads) {
          s_bx[e] = s_nx[e];
          s_bi[e] = s_ni[e];
          s_blm[e] = s_nlm[e];
          s_bbt[e] = s_nbt[e];
        }
        if (nk == K) tau = s_nx[K - 1];
        __syncthreads();
        if (tid == 0) {
          s_nbuf = nk;
          s_overflow = 0;
        }
      }

      const bool last_chunk = (ch + 1 == nchunk);
      if (!last_chunk) {
        // ---- clear this chunk's key rows, then compact between chunks ----
        if (HAS_LM)
          for (int q = tid; q < lm_total; q += kThreads) lmkey[stkey[q]] = 0u;
        if (HAS_BT)
          for (int q = tid; q < bt_total; q += kThreads) btkey[btclr[q]] = 0u;
        __syncthreads();
        const int n = min(s_nbuf, kChunkCap);
        if (n > K) {
          for (int e = tid; e < n; e += kThreads) {
            const float xe = s_bx[e];
            const uint32_t ie = s_bi[e];
            int rank = 0;
            for (int f = 0; f < n; ++f) rank += beats(s_bx[f], s_bi[f], xe, ie) ? 1 : 0;
            if (rank < K) {
              s_nx[rank] = xe;
              s_ni[rank] = ie;
              s_nlm[rank] = s_blm[e];
              s_nbt[rank] = s_bbt[e];
            }
          }
          __syncthreads();
          for (int e = tid; e < K; e += kThreads) {
            s_bx[e] = s_nx[e];
            s_bi[e] = s_ni[e];
            s_blm[e] = s_nlm[e];
            s_bbt[e] = s_nbt[e];
          }
          tau = fmaxf(tau, s_nx[K - 1]);
          __syncthreads();
          if (tid == 0) s_nbuf = K;
          __syncthreads();
        }
      } else if (wave != 0) {
        // the key rows are cleared by waves 1..7 while wave 0 selects
        if (HAS_LM)
          for (int q = tid - 64; q < lm_total; q += kThreads - 64) lmkey[stkey[q]] = 0u;
        if (HAS_BT)
          for (int q = tid - 64; q < bt_total; q += kThreads - 64) btkey[btclr[q]] = 0u;
      }
    }

    // ---- 5. selection and beam update ----
    // survivors: s_b*[0, nlab) from the labels, s_b*[kChunkCap, kChunkCap+K) blanks
    const int nlab = min(s_nbuf, kChunkCap);
    const bool small = (nlab + K) <= 64;
    if (!small) {
      // exact ranking in LDS by every thread (large beams, rare otherwise)
      const int n = nlab + K;
      for (int e = tid; e < n; e += kThreads) {
        const int ee = e < nlab ? e : kChunkCap + (e - nlab);
        const float xe = s_bx[ee];
        const uint32_t ie = s_bi[ee];
        if (ie != 0xFFFFFFFFu) {
          int rank = 0;
          for (int f = 0; f < n; ++f) {
            const int ff = f < nlab ? f : kChunkCap + (f - nlab);
            const uint32_t iff = s_bi[ff];
            rank += (iff != 0xFFFFFFFFu && beats(s_bx[ff], iff, xe, ie)) ? 1 : 0;
          }
          if (rank < K) {
            uint32_t lmt = s_blm[ee];
            if (HAS_LM && (lmt & 0x80000000u)) lmt = sttgt[lmt & 0x0FFFFFFFu];
            s_nx[rank] = xe;
            s_ni[rank] = ie;
            s_nlm[rank] = lmt;
            s_nbt[rank] = s_bbt[ee];
          }
        }
      }
      if (tid < K) {
        // count of valid entries decides how many ranks were written
        int cnt = 0;
        for (int f = 0; f < n; ++f) {
          const int ff = f < nlab ? f : kChunkCap + (f - nlab);
          cnt += s_bi[ff] != 0xFFFFFFFFu ? 1 : 0;
        }
        if (tid >= cnt) s_ni[tid] = 0xFFFFFFFFu;
      }
      __syncthreads();
    }
    if (wave == 0) {
      const int j = lane;
      // candidate held by this lane before/after ranking
      float x;
      uint32_t idx;
      int src = lane;
      uint32_t lmt = 0u, btk = 0u;
      LmLevel hh[NLA];
      BtNode nd{0u, 0u, 0u, 0u};
      if (small) {
        // lane e holds survivor e (label survivors, then the blank slots)
        const int n = nlab + K;
        const int ee = j < nlab ? j : (j < n ? kChunkCap + (j - nlab) : -1);
        float xe = kNegInf;
        uint32_t ie = 0xFFFFFFFFu, lmt_e = 0u, btk_e = 0u;
        if (ee >= 0) {
          xe = s_bx[ee];
          ie = s_bi[ee];
          lmt_e = s_blm[ee];
          btk_e = s_bbt[ee];
        }
        const bool valid_e = xe != kNegInf;
        if (HAS_LM && valid_e && (lmt_e & 0x80000000u)) lmt_e = sttgt[lmt_e & 0x0FFFFFFFu];
        // prefetch the chain headers of emitting survivors before ranking
        const uint32_t vpar = valid_e ? ie / static_cast<uint32_t>(W) : 0u;
        const int vc = valid_e ? static_cast<int>(ie - vpar * W) : V;
        const bool vemit = valid_e && vc != V && vc != s_last[vpar];
#pragma unroll
        for (int l = 0; l < NL; ++l) hh[l] = p.lm_states[static_cast<size_t>(vemit ? lmt_e : p.lm_bos_state) * NL + l];
        if (HAS_BT) nd = p.bt_nodes[vemit ? (btk_e & kBtChildMask) : 0u];
        // rank = number of survivors that beat this one (broadcast reads)
        int rank = 0;
        // label survivors, 8 at a time (independent broadcast reads), then blanks
        for (int f0 = 0; f0 < nlab; f0 += 8) {
          float fx[8];
          uint32_t fi[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            fx[u] = s_bx[f0 + u];
            fi[u] = s_bi[f0 + u];
          }
#pragma unroll
          for (int u = 0; u < 8; ++u) rank += (f0 + u < nlab && beats(fx[u], fi[u], xe, ie)) ? 1 : 0;
        }
        for (int f0 = 0; f0 < K; f0 += 8) {
          float fx[8];
          uint32_t fi[8];
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            fx[u] = s_bx[kChunkCap + f0 + u];
            fi[u] = s_bi[kChunkCap + f0 + u];
          }
#pragma unroll
          for (int u = 0; u < 8; ++u) rank += (f0 + u < K && beats(fx[u], fi[u], xe, ie)) ? 1 : 0;
        }
        const int nvalid = __popcll(__ballot(valid_e));
        if (valid_e && rank < K) s_order[rank] = lane;
        wave_sync_lds();
        const int nsel_s = min(nvalid, K);
        src = lane < nsel_s ? s_order[lane] : 0;
        x = __shfl(xe, src);
        idx = __shfl(ie, src);
        lmt = __shfl(lmt_e, src);
        btk = __shfl(btk_e, src);
        if (lane >= nsel_s) {
          x = kNegInf;
          idx = 0xFFFFFFFFu;
        }
#pragma unroll
        for (int l = 0; l < NL; ++l) {
          hh[l].begin = __shfl(hh[l].begin, src);
          hh[l].count = __shfl(hh[l].count, src);
          hh[l].bo = __shfl(hh[l].bo, src);
        }
        if (HAS_BT) {
          nd.list_begin = __shfl(nd.list_begin, src);
          nd.list_count = __shfl(nd.list_count, src);
          nd.pot = __shfl(nd.pot, src);
          nd.chain_arcs = __shfl(nd.chain_arcs, src);
        }
      } else {
        x = j < K ? s_nx[j] : kNegInf;
        idx = j < K ? s_ni[j] : 0xFFFFFFFFu;
        if (idx == 0xFFFFFFFFu) x = kNegInf;
        lmt = j < K ? s_nlm[j] : 0u;
        btk = j < K ? s_nbt[j] : 0u;
        const bool valid = x != kNegInf;
        const uint32_t vpar = valid ? idx / static_cast<uint32_t>(W) : 0u;
        const int vc = valid ? static_cast<int>(idx - vpar * W) : V;
        const bool vemit = valid && vc != V && vc != s_last[vpar];
#pragma unroll
        for (int l = 0; l < NL; ++l) hh[l] = p.lm_states[static_cast<size_t>(vemit ? lmt : p.lm_bos_state) * NL + l];
        if (HAS_BT) nd = p.bt_nodes[vemit ? (btk & kBtChildMask) : 0u];
      }
      // prune (Algorithm 1: below best - theta -> -inf)
      const float best = __shfl(x, 0);
      const float lim = best - p.theta;
      bool valid = (j < K) && (x != kNegInf);
      if (valid && x < lim) x = kNegInf;
      int32_t last = V, len = 0;
      uint64_t hash = 0ull;
      uint32_t lms = 0u, bts = 0u;
      int32_t bpv = -1;
      bool emit = false;
      int par = 0;
      if (valid) {
        par = static_cast<int>(idx / static_cast<uint32_t>(W));
        const int c = static_cast<int>(idx - static_cast<uint32_t>(par) * W);
        const int lastp = s_last[par];
        emit = (c != V) && (c != lastp);
        hash = s_hash[par];
        len = s_len[par];
        lms = s_lms[par];
        bts = s_bts[par];
        if (emit) {
          hash = mix_token(hash, static_cast<uint32_t>(c));
          len += 1;
          if (HAS_LM) lms = lmt;
          if (HAS_BT) bts = btk & kBtChildMask;
        }
        last = c;
        bpv = (par << 16) | c;
      }
      if (x != kNegInf && emit) st_emit += 1;
      // recombination: same transcript hash, length and ends-in-blank flag
      bool alive = valid && (x != kNegInf);
      const int blankend = (last == V) ? 1 : 0;
      const uint32_t meta = (static_cast<uint32_t>(len) & 0x3FFFFFFFu) | (static_cast<uint32_t>(blankend) << 30) |
                            (alive ? 0x80000000u : 0u);
      if (j < K) {
        s_rkh[j] = hash;
        s_rkm[j] = meta;
      }
      wave_sync_lds();
      bool dup = false;
      for (int i0 = 0; i0 < K; i0 += 8) {
        uint32_t mi[8];
        uint64_t hi[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          mi[u] = s_rkm[i0 + u];
          hi[u] = s_rkh[i0 + u];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int i = i0 + u;
          if (i < j && i < K && alive && (mi[u] >> 31) && hi[u] == hash && ((mi[u] ^ meta) & 0x7FFFFFFFu) == 0u)
            dup = true;
        }
      }
      if (dup) x = kNegInf;
      alive = alive && !dup;
      // next chain: prefetched for emitting winners, the parent's otherwise
      uint32_t cb[NLA], cc[NLA];
      float cbo[NLA];
      uint32_t bb = 0u, bc = 0u;
      int32_t bpot = 0;
      if (alive) {
#pragma unroll
        for (int l = 0; l < NL; ++l) {
          cb[l] = emit ? hh[l].begin : s_lvb[par][l];
          cc[l] = emit ? hh[l].count : s_lvc[par][l];
          cbo[l] = emit ? hh[l].bo : s_lvbo[par][l];
        }
        if (HAS_BT) {
          bb = emit ? nd.list_begin : s_btb[par];
          bc = emit ? nd.list_count : s_btc[par];
          bpot = emit ? static_cast<int32_t>(nd.pot & 0xFFu) : s_btpot[par];
        }
      }
      uint32_t chain_nodes = 0u, chain_arcs = 0u;
      if (HAS_BT && alive) {
        // statistics: the parent's record when not emitting
        if (emit) {
          chain_nodes = nd.pot >> 8;
          chain_arcs = nd.chain_arcs;
        }
      }
      wave_sync_lds();  // every lane has read the parents' rows and the survivors
      // reset the survivor buffer for the next frame (visible after the barrier)
      if (lane == 0) {
        s_nbuf = 0;
        s_overflow = 0;
      }
      if (j < K) {
        s_bx[kChunkCap + j] = kNegInf;
        s_bi[kChunkCap + j] = 0xFFFFFFFFu;
      }
      int32_t acnt = 0, bcnt = 0;
      if (j < K) {
        bpb[static_cast<size_t>(t) * K + j] = bpv;
        s_score[j] = x;
        s_last[j] = last;
        s_len[j] = len;
        s_hash[j] = hash;
        s_lms[j] = lms;
        s_bts[j] = bts;
      }
      if (alive) {
#pragma unroll
        for (int l = 0; l < NL; ++l) {
          s_lvb[j][l] = cb[l];
          s_lvc[j][l] = cc[l];
          s_lvbo[j][l] = cbo[l];
          const uint32_t n = cc[l] & ~kExists;
          acnt += static_cast<int32_t>(n);
          if (t + 1 < L && (cc[l] & kExists)) {
            st_lms += 1;
            st_lma += n;
          }
        }
        if (HAS_BT) {
          s_btb[j] = bb;
          s_btc[j] = bc;
          s_btpot[j] = bpot;
          bcnt = static_cast<int32_t>(bc);
        }
        if (t + 1 < L) st_alive += 1;
      }
      // boosting statistics need the node record of inherited states too
      if (HAS_BT && alive && !emit && t + 1 < L && p.stats) {
        const BtNode pn = p.bt_nodes[bts];
        chain_nodes = pn.pot >> 8;
        chain_arcs = pn.chain_arcs;
      }
      if (t + 1 < L) {
        st_btn += chain_nodes;
        st_bta += chain_arcs;
      }
      // live list and chunking (slot order = live order)
      const uint64_t amask = __ballot(alive);
      const int na = __popcll(amask);
      const int apos = __popcll(amask & lanemask_lt());
      const int av = alive ? acnt : 0, bv = alive ? bcnt : 0;
      const int ia_slot = wave_incl_scan(av, lane);
      const int ib_slot = wave_incl_scan(bv, lane);
      if (alive) {
        s_alive[apos] = j;
        s_hoff[apos] = ia_slot - av;
        s_boff[apos] = ib_slot - bv;
      }
      const int tota = __builtin_amdgcn_readlane(ia_slot, 63);
      const int totb = __builtin_amdgcn_readlane(ib_slot, 63);
      if (lane == 0) {
        s_hoff[na] = tota;
        s_boff[na] = totb;
      }
      int nch = 0;
      if (na <= kcmax && tota <= kLmStage && totb <= kBtStage) {
        if (lane == 0) s_chunk[0] = 0;
        nch = na > 0 ? 1 : 0;
      } else {
        wave_sync_lds();
        // inclusive sums by live position
        const int ia = lane < na ? s_hoff[lane + 1] : tota;
        const int ib = lane < na ? s_boff[lane + 1] : totb;
        int start = 0;
        while (start < na) {
          const int basea = start > 0 ? __shfl(ia, start - 1) : 0;
          const int baseb = start > 0 ? __shfl(ib, start - 1) : 0;
          const bool ok = lane >= start && lane < na && lane < start + kcmax &&
                          (ia - basea) <= kLmStage && (ib - baseb) <= kBtStage;
          int cnt = __popcll(__ballot(ok));
          if (cnt == 0) {
            cnt = 1;
            status |= 4u;
          }
          if (lane == 0) s_chunk[nch] = start;
          ++nch;
          start += cnt;
        }
      }
      if (lane == 0) {
        s_chunk[nch] = na;
        s_nchunk = nch;
      }
    }
    __syncthreads();
  }

  // ---- LM.Final, best beam ----
  if (wave == 0) {
    const int j = lane;
    float s = (j < K) ? s_score[j] : kNegInf;
    if (HAS_LM && j < K && s != kNegInf) {
      // ln P(</s> | state) through the backoff chain; </s> is the last arc of
      // a state's sorted arcs when present
      float v = p.lm_unigram[V];
      int found = -1;
      float fv = 0.0f;
#pragma unroll
      for (int l = NL - 1; l >= 0; --l) {
        const uint32_t n = s_lvc[j][l] & ~kExists;
        if (found < 0 && n > 0) {
          const LmArc a = p.lm_arcs[s_lvb[j][l] + n - 1];
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
          if (l > found) v = v + s_lvbo[j][l];
      } else {
#pragma unroll
        for (int l = 0; l < NL; ++l) v = v + s_lvbo[j][l];
      }
      const float av = alpha * v;
      s = s + av;
    }
    // argmax, lowest slot on ties
    float bs = s;
    int bj = (j < K) ? j : 0x7FFF;
    for (int off = 1; off < 64; off <<= 1) {
      const float os = __shfl_xor(bs, off);
      const int oj = __shfl_xor(bj, off);
      if (os > bs || (os == bs && oj < bj)) {
        bs = os;
        bj = oj;
      }
    }
    if (lane == 0) {
      s_best = bj;
      s_bestscore = bs;
    }
    if (p.stats) {
      int64_t a0 = st_alive, a1 = st_lms, a2 = st_lma, a3 = st_btn, a4 = st_bta, a5 = st_emit;
      for (int off = 1; off < 64; off <<= 1) {
        a0 += __shfl_xor(a0, off);
        a1 += __shfl_xor(a1, off);
        a2 += __shfl_xor(a2, off);
        a3 += __shfl_xor(a3, off);
        a4 += __shfl_xor(a4, off);
        a5 += __shfl_xor(a5, off);
      }
      if (lane == 0) {
        int64_t* so = p.stats + static_cast<size_t>(b) * 8;
        so[0] = L;
        so[1] = a0;
        so[2] = a1;
        so[3] = a2;
        so[4] = a3;
        so[5] = a4;
        so[6] = a5;
        so[7] = 0;
      }
    }
  }
  __syncthreads();
  const int best = s_best;
  const float bscore = s_bestscore;
  const bool have = bscore != kNegInf;
  const int nout = have ? s_len[best] : 0;
  int32_t* ot = p.out_tokens + static_cast<size_t>(b) * T;
  for (int t = nout + tid; t < T; t += kThreads) ot[t] = -1;
  if (tid == 0) {
    p.out_scores[b] = bscore;
    if (p.out_lengths) p.out_lengths[b] = nout;
  }

  // ---- traceback through the back-pointers, staged in LDS tiles ----
  if (have && L > 0) {
    const int tile_frames = kBigWords / K;
    int j = best, cnext = -1, pos = nout;
    for (int hi = L; hi > 0;) {
      const int lo = hi > tile_frames ? hi - tile_frames : 0;
      __syncthreads();
      const int n = (hi - lo) * K;
      const int32_t* src = bpb + static_cast<size_t>(lo) * K;
      for (int q = tid; q < n; q += kThreads) s_big[q] = static_cast<uint32_t>(src[q]);
      __syncthreads();
      if (tid == 0) {
        for (int t = hi - 1; t >= lo; --t) {
          const uint32_t e = s_big[(t - lo) * K + j];
          const int c = static_cast<int>(e & 0xFFFFu);
          const int par = static_cast<int>(e >> 16);
          if (t < L - 1 && cnext != V && cnext != c) {
            if (pos > 0) ot[--pos] = cnext;
          }
          cnext = c;
          j = par;
        }
      }
      hi = lo;
    }
    if (tid == 0) {
      if (cnext != V && cnext >= 0 && pos > 0) ot[--pos] = cnext;
      if (pos != 0) status |= 2u;
    }
  }
  if (tid == 0) p.status[b] = status;
}

template <int LPT, int NLEV>
hipError_t launch_nlev(const KernelParams& p, hipStream_t s) {
  dim3 grid(p.B), block(kThreads);
  if (p.bt_nodes != nullptr)
    hipLaunchKernelGGL((decode_kernel<LPT, NLEV, true>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((decode_kernel<LPT, NLEV, false>), grid, block, 0, s, p);
  return hipGetLastError();
}

template <int LPT>
hipError_t launch_lpt_impl(const KernelParams& p, hipStream_t s) {
  if (p.lm_states == nullptr && p.lm_arcs == nullptr) return launch_nlev<LPT, -1>(p, s);
  switch (p.lm_nlev) {
    case 0: return launch_nlev<LPT, 0>(p, s);
    case 1: return launch_nlev<LPT, 1>(p, s);
    case 2: return launch_nlev<LPT, 2>(p, s);
    case 3: return launch_nlev<LPT, 3>(p, s);
    case 4: return launch_nlev<LPT, 4>(p, s);
    case 5: return launch_nlev<LPT, 5>(p, s);
    case 6: return launch_nlev<LPT, 6>(p, s);
    case 7: return launch_nlev<LPT, 7>(p, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace detail
}  // namespace ctcbeam
