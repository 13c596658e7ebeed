// Batched CTC beam search, all frames of one utterance per workgroup (gfx950).
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
// memory latency and LDS traffic, so MFMA is not used.
//
// Per frame:
//   1. the next frame's log-prob row is prefetched into registers (each lane
//      owns the labels c = tid + j*512);
//   2. fill: for every live beam, the explicit continuations of every state of
//      its LM backoff chain are gathered (one wave per beam, loads batched so
//      one memory latency covers a whole chain) and scattered into an LDS
//      [beam][token] key row with atomicMax, so the highest-order explicit
//      n-gram wins without barriers between orders; boosting continuations
//      (pre-merged per tree state on the host) are stored the same way;
//   3. candidates: each lane scores its labels for every beam, resolving the
//      LM value from the key row or from the unigram+backoff fold;
//   4. selection: a lower bound on the K-th best score (min over K lane-group
//      maxima) filters the K*V candidates down to a few dozen, which are
//      ranked exactly by (score desc, index asc); rare overflows fall back to
//      an exact extraction;
//   5. wave 0 prunes, advances the beams (hash of the collapsed transcript,
//      LM/boost states), recombines duplicates and fetches the next states'
//      chain headers; back-pointers go to HBM.
// After the last frame the best beam is traced back through the back-pointers
// (staged in LDS) and written out.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ctcbeam_internal.h"

namespace ctcbeam {
namespace {

constexpr float kNegInf = -__builtin_huge_valf();

// Shared scratch carved from one LDS block so the traceback can reuse it.
constexpr int kBigWords = 2 * kKeyWords + 3 * kLmStage + kBtStage;
constexpr int kOffLmKey = 0;
constexpr int kOffBtKey = kKeyWords;
constexpr int kOffStV = 2 * kKeyWords;
constexpr int kOffStTgt = kOffStV + kLmStage;
constexpr int kOffStKey = kOffStTgt + kLmStage;
constexpr int kOffBtClr = kOffStKey + kLmStage;
// survivors of the label candidates may fill the buffer up to kChunkCap; the
// remaining kMaxK entries always take the K blank candidates
constexpr int kChunkCap = kCap - kMaxK;

__device__ __forceinline__ uint64_t mix_token(uint64_t h, uint32_t c) {
  uint64_t z = h + (static_cast<uint64_t>(c) + 1ull) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Order key: larger is better; (x desc, idx asc); -0 and +0 compare equal.
__device__ __forceinline__ uint64_t order_key(float x, uint32_t idx) {
  float y = x + 0.0f;
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

template <int LPT, bool HAS_LM, bool HAS_BT>
__global__ void __launch_bounds__(kThreads) decode_kernel(KernelParams p) {
  __shared__ __align__(16) uint32_t s_big[kBigWords];
  // candidate buffer
  __shared__ float s_bx[kCap];
  __shared__ uint32_t s_bi[kCap], s_blm[kCap], s_bbt[kCap];
  // selected candidates (rank order)
  __shared__ float s_nx[kMaxK];
  __shared__ uint32_t s_ni[kMaxK], s_nlm[kMaxK], s_nbt[kMaxK];
  // beams
  __shared__ float s_score[kMaxK];
  __shared__ int32_t s_last[kMaxK], s_len[kMaxK];
  __shared__ uint64_t s_hash[kMaxK];
  __shared__ uint32_t s_lms[kMaxK], s_bts[kMaxK];
  __shared__ uint32_t s_lvb[kMaxK][kMaxLev], s_lvc[kMaxK][kMaxLev];
  __shared__ float s_lvbo[kMaxK][kMaxLev];
  __shared__ uint32_t s_btb[kMaxK], s_btc[kMaxK];
  __shared__ int32_t s_btpot[kMaxK];
  // live list and chunks (positions in the live list)
  __shared__ int32_t s_alive[kMaxK];
  __shared__ int32_t s_hoff[kMaxK + 1], s_boff[kMaxK + 1];
  __shared__ int32_t s_chunk[kMaxK + 1];
  __shared__ int32_t s_nalive, s_nchunk;
  // selection
  __shared__ float s_tauw[kWaves];
  __shared__ uint64_t s_red[2][kWaves];
  __shared__ int32_t s_nbuf, s_overflow;
  __shared__ int32_t s_nsel;

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
  const int nlev = HAS_LM ? p.lm_nlev : 0;
  const int kcmax = min(K, 16 / LPT);
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
    const bool alive = (j == 0) && (K > 0);
    int32_t acnt = 0, bcnt = 0;
    if (j < K) {
      s_score[j] = (j == 0) ? 0.0f : kNegInf;
      s_last[j] = V;
      s_len[j] = 0;
      s_hash[j] = 0ull;
      s_lms[j] = HAS_LM ? p.lm_bos_state : 0u;
      s_bts[j] = 0u;
      if (HAS_LM) {
        for (int l = 0; l < kMaxLev; ++l) {
          s_lvb[j][l] = 0u;
          s_lvc[j][l] = 0u;
          s_lvbo[j][l] = 0.0f;
        }
        if (alive) {
          for (int l = 0; l < nlev; ++l) {
            const LmLevel h = p.lm_states[static_cast<size_t>(p.lm_bos_state) * nlev + l];
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
      s_nalive = 1;
      s_hoff[0] = 0;
      s_hoff[1] = acnt;
      s_boff[0] = 0;
      s_boff[1] = bcnt;
      s_chunk[0] = 0;
      s_chunk[1] = 1;
      s_nchunk = 1;
    }
  }
  for (int i = tid; i < kKeyWords; i += kThreads) {
    if (HAS_LM) lmkey[i] = 0u;
    if (HAS_BT) btkey[i] = 0u;
  }
  __syncthreads();

  // group size for the K-th-best lower bound: G >= K groups per wave
  int G = 1;
  while (G < K) G <<= 1;
  if (G > 64) G = 64;
  const int gsz = 64 / G;

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
    if (tid == 0) {
      s_nbuf = 0;
      s_overflow = 0;
    }
    float tau = kNegInf;
    const int nchunk = s_nchunk;

    for (int ch = 0; ch < nchunk; ++ch) {
      const int cs = s_chunk[ch];
      const int kc = s_chunk[ch + 1] - cs;
      const int hbase = s_hoff[cs];
      const int bbase = s_boff[cs];
      const int lm_total = s_hoff[cs + kc] - hbase;
      const int bt_total = s_boff[cs + kc] - bbase;

      // ---- 2. fill: one wave per beam ----
      for (int i = wave; i < kc; i += kWaves) {
        const int k = s_alive[cs + i];
        if (HAS_LM) {
          const int hoff = s_hoff[cs + i] - hbase;
          uint32_t lb[kMaxLev], lend[kMaxLev];
          float lbo[kMaxLev];
          uint32_t run = 0;
#pragma unroll
          for (int l = 0; l < kMaxLev; ++l) {
            if (l < nlev) {
              lb[l] = s_lvb[k][l];
              run += s_lvc[k][l] & ~kExists;
              lbo[l] = s_lvbo[k][l];
            } else {
              lb[l] = 0u;
              lbo[l] = 0.0f;
            }
            lend[l] = run;
          }
          const int total = static_cast<int>(run);
          const uint32_t rowbase = static_cast<uint32_t>(i) * static_cast<uint32_t>(V);
          for (int r0 = 0; r0 < total; r0 += 64 * 8) {
            LmArc a[8];
            int lv[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              const int q = r0 + u * 64 + lane;
              lv[u] = -1;
              if (q < total) {
                int l = 0;
#pragma unroll
                for (int ll = 0; ll < kMaxLev - 1; ++ll)
                  l += (ll < nlev - 1 && static_cast<uint32_t>(q) >= lend[ll]) ? 1 : 0;
                const uint32_t start = (l == 0) ? 0u : lend[l - 1];
                const uint32_t ai = lb[l] + (static_cast<uint32_t>(q) - start);
                a[u] = p.lm_arcs[ai];
                lv[u] = l;
              }
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
              if (lv[u] >= 0) {
                const int q = r0 + u * 64 + lane;
                float v = a[u].logp;
#pragma unroll
                for (int l2 = 1; l2 < kMaxLev; ++l2)
                  if (l2 > lv[u] && l2 < nlev) v = v + lbo[l2];
                const float av = alpha * v;
                const int pos = hoff + q;
                // </s> (token V) is never a frame label; it is only read at the end
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
          const uint32_t rowbase = static_cast<uint32_t>(i) * static_cast<uint32_t>(V);
          for (int r0 = 0; r0 < cnt; r0 += 64 * 4) {
            BtEntry e[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int q = r0 + u * 64 + lane;
              if (q < cnt) e[u] = p.bt_list[lbeg + q];
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
      float cand[16];
      float lmax = kNegInf;
#pragma unroll
      for (int i = 0; i < 16 / LPT; ++i) {
        if (i < kc) {
          const int k = s_alive[cs + i];
          const float sk = s_score[k];
          const int lastk = s_last[k];
          float bo[kMaxLev];
#pragma unroll
          for (int l = 0; l < kMaxLev; ++l) bo[l] = (HAS_LM && l < nlev) ? s_lvbo[k][l] : 0.0f;
          const int potk = HAS_BT ? s_btpot[k] : 0;
#pragma unroll
          for (int j = 0; j < LPT; ++j) {
            const int c = tid + j * kThreads;
            float x = kNegInf;
            if (c < V) {
              x = sk + rD[j];
              if (c != lastk) {
                x = x + beta;
                if (HAS_LM) {
                  const uint32_t key = lmkey[i * V + c];
                  float av;
                  if (key != 0u) {
                    av = stv[key & 0x0FFFFFFFu];
                  } else {
                    float v = rP1[j];
#pragma unroll
                    for (int l = 0; l < kMaxLev; ++l)
                      if (l < nlev) v = v + bo[l];
                    av = alpha * v;
                  }
                  x = x + av;
                }
                if (HAS_BT) {
                  uint32_t bk = btkey[i * V + c];
                  if (bk == 0u) bk = rRoot[j];
                  const int pre = static_cast<int>((bk >> 20) & 63u);
                  const float bv = boost_w * static_cast<float>(pre - potk);
                  x = x + bv;
                }
              }
            }
            cand[i * LPT + j] = x;
            lmax = fmaxf(lmax, x);
          }
        } else {
#pragma unroll
          for (int j = 0; j < LPT; ++j) cand[i * LPT + j] = kNegInf;
        }
      }

      // ---- 4a. lower bound on the K-th best (this chunk alone) ----
      {
        float g = lmax;
        for (int off = 1; off < gsz; off <<= 1) g = fmaxf(g, __shfl_xor(g, off));
        for (int off = gsz; off < 64; off <<= 1) g = fminf(g, __shfl_xor(g, off));
        if (lane == 0) s_tauw[wave] = g;
      }
      __syncthreads();
      {
        float tc = s_tauw[0];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) tc = fmaxf(tc, s_tauw[w]);
        tau = fmaxf(tau, tc);
      }

      // ---- 4b. filter and append survivors ----
      {
        int mycnt = 0;
#pragma unroll
        for (int r = 0; r < 16; ++r) mycnt += (cand[r] >= tau && cand[r] != kNegInf) ? 1 : 0;
        // wave-exclusive prefix of mycnt
        int incl = mycnt;
        for (int off = 1; off < 64; off <<= 1) {
          const int v = __shfl_up(incl, off);
          if (lane >= off) incl += v;
        }
        const int wtotal = __shfl(incl, 63);
        int wbase = 0;
        if (lane == 0 && wtotal > 0) wbase = atomicAdd(&s_nbuf, wtotal);
        wbase = __shfl(wbase, 0);
        int slot = wbase + incl - mycnt;
        if (mycnt > 0) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float x = cand[r];
            if (x >= tau && x != kNegInf) {
              const int i = r / LPT, j = r % LPT;
              const int c = tid + j * kThreads;
              const int k = s_alive[cs + i];
              if (slot < kChunkCap) {
                uint32_t lmt = 0u, bk = 0u;
                if (HAS_LM) {
                  const uint32_t key = lmkey[i * V + c];
                  lmt = (key != 0u) ? sttgt[key & 0x0FFFFFFFu] : static_cast<uint32_t>(c);
                }
                if (HAS_BT) {
                  bk = btkey[i * V + c];
                  if (bk == 0u) bk = rRoot[j];
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
      }
      __syncthreads();

      // ---- 4c. overflow: exact extraction over (buffer before) U (chunk) ----
      if (s_overflow) {
        // keys of buffer entries [0, nbuf_before) and of this lane's candidates
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
              s_nx[it] = s_bx[e];
              s_ni[it] = s_bi[e];
              s_nlm[it] = s_blm[e];
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

      // ---- clear this chunk's key rows ----
      if (HAS_LM)
        for (int q = tid; q < min(lm_total, kLmStage); q += kThreads) lmkey[stkey[q]] = 0u;
      if (HAS_BT)
        for (int q = tid; q < min(bt_total, kBtStage); q += kThreads) btkey[btclr[q]] = 0u;
      __syncthreads();

      // ---- compaction between chunks (large beams) ----
      if (ch + 1 < nchunk) {
        const int n = min(s_nbuf, kCap);
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
      }
    }

    // ---- blank candidates (never scored by LM/boosting) ----
    if (tid < K) {
      const float sk = s_score[tid];
      const float x = sk + rBlank;
      if (sk != kNegInf && x != kNegInf && x >= tau) {
        const int slot = atomicAdd(&s_nbuf, 1);
        s_bx[slot] = x;  // slot < kChunkCap + K <= kCap
        s_bi[slot] = static_cast<uint32_t>(tid * W + V);
        s_blm[slot] = 0u;
        s_bbt[slot] = 0u;
      }
    }
    __syncthreads();

    // ---- 5. exact ranking of the survivors ----
    {
      const int n = min(s_nbuf, kCap);
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
      if (tid == 0) s_nsel = min(n, K);
    }
    __syncthreads();

    // ---- 6. beam update, recombination, next headers (wave 0) ----
    if (wave == 0) {
      const int j = lane;
      const int nsel = s_nsel;
      const float best = nsel > 0 ? s_nx[0] : kNegInf;
      const float lim = best - p.theta;
      float x = kNegInf;
      int32_t last = V, len = 0;
      uint64_t hash = 0ull;
      uint32_t lms = 0u, bts = 0u;
      int32_t bpv = -1;
      bool emit = false;
      if (j < nsel) {
        x = s_nx[j];
        if (x < lim) x = kNegInf;
        const uint32_t idx = s_ni[j];
        const int par = static_cast<int>(idx / static_cast<uint32_t>(W));
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
          if (HAS_LM) lms = s_nlm[j];
          if (HAS_BT) bts = s_nbt[j] & kBtChildMask;
        }
        last = c;
        bpv = (par << 16) | c;
      }
      if (x != kNegInf && emit) st_emit += 1;
      // recombination: same transcript hash, length and ends-in-blank flag
      bool alive = (j < K) && (x != kNegInf);
      const uint32_t hlo = static_cast<uint32_t>(hash), hhi = static_cast<uint32_t>(hash >> 32);
      const int blankend = (last == V) ? 1 : 0;
      bool dup = false;
      for (int i = 0; i < K; ++i) {
        const bool ai = __shfl(alive ? 1 : 0, i) != 0;
        const uint32_t ilo = __shfl(hlo, i), ihi = __shfl(hhi, i);
        const int ilen = __shfl(len, i), iblank = __shfl(blankend, i);
        if (i < j && ai && ilo == hlo && ihi == hhi && ilen == len && iblank == blankend) dup = true;
      }
      if (dup) x = kNegInf;
      alive = alive && !dup;
      if (j < K) {
        bpb[static_cast<size_t>(t) * K + j] = bpv;
        s_score[j] = x;
        s_last[j] = last;
        s_len[j] = len;
        s_hash[j] = hash;
        s_lms[j] = lms;
        s_bts[j] = bts;
      }
      // next chain headers
      int32_t acnt = 0, bcnt = 0;
      if (alive) {
        if (HAS_LM) {
          LmLevel h[kMaxLev];
#pragma unroll
          for (int l = 0; l < kMaxLev; ++l)
            if (l < nlev) h[l] = p.lm_states[static_cast<size_t>(lms) * nlev + l];
#pragma unroll
          for (int l = 0; l < kMaxLev; ++l) {
            if (l < nlev) {
              s_lvb[j][l] = h[l].begin;
              s_lvc[j][l] = h[l].count;
              s_lvbo[j][l] = h[l].bo;
              const uint32_t n = h[l].count & ~kExists;
              acnt += static_cast<int32_t>(n);
              if (t + 1 < L && (h[l].count & kExists)) {
                st_lms += 1;
                st_lma += n;
              }
            }
          }
        }
        if (HAS_BT) {
          const BtNode nd = p.bt_nodes[bts];
          s_btb[j] = nd.list_begin;
          s_btc[j] = nd.list_count;
          s_btpot[j] = static_cast<int32_t>(nd.pot & 0xFFu);
          bcnt = static_cast<int32_t>(nd.list_count);
          if (t + 1 < L) {
            st_btn += nd.pot >> 8;
            st_bta += nd.chain_arcs;
          }
        }
        if (t + 1 < L) st_alive += 1;
      }
      // live list and chunking
      const uint64_t amask = __ballot(alive);
      const int na = __popcll(amask);
      const int apos = __popcll(amask & lanemask_lt());
      if (alive) s_alive[apos] = j;
      // gather (acnt, bcnt) into live order: lane i takes the i-th live slot
      wave_sync_lds();
      const int sl = lane < na ? s_alive[lane] : 0;
      int ai_ = __shfl(acnt, sl);
      int bi_ = __shfl(bcnt, sl);
      if (lane >= na) {
        ai_ = 0;
        bi_ = 0;
      }
      int ia = ai_, ib = bi_;
      for (int off = 1; off < 64; off <<= 1) {
        const int va = __shfl_up(ia, off), vb = __shfl_up(ib, off);
        if (lane >= off) { ia += va; ib += vb; }
      }
      if (lane < na) {
        s_hoff[lane] = ia - ai_;
        s_boff[lane] = ib - bi_;
      }
      const int tota = na > 0 ? __shfl(ia, na > 0 ? na - 1 : 0) : 0;
      const int totb = na > 0 ? __shfl(ib, na > 0 ? na - 1 : 0) : 0;
      if (lane == 0) {
        s_hoff[na] = tota;
        s_boff[na] = totb;
      }
      int start = 0, nch = 0;
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
      if (lane == 0) {
        s_chunk[nch] = na;
        s_nchunk = nch;
        s_nalive = na;
      }
    }
    __syncthreads();
  }

  // ---- LM.Final, best beam ----
  __shared__ int32_t s_best;
  __shared__ float s_bestscore;
  if (wave == 0) {
    const int j = lane;
    float s = (j < K) ? s_score[j] : kNegInf;
    if (HAS_LM && j < K && s != kNegInf) {
      // ln P(</s> | state) through the backoff chain
      float v = p.lm_unigram[V];
      int found = -1;
      float fv = 0.0f;
      for (int l = nlev - 1; l >= 0; --l) {
        const uint32_t n = s_lvc[j][l] & ~kExists;
        if (n > 0) {
          const LmArc a = p.lm_arcs[s_lvb[j][l] + n - 1];
          if (a.token == static_cast<uint32_t>(V)) {
            found = l;
            fv = a.logp;
            break;
          }
        }
      }
      if (found >= 0) {
        v = fv;
        for (int l = found + 1; l < nlev; ++l) v = v + s_lvbo[j][l];
      } else {
        for (int l = 0; l < nlev; ++l) v = v + s_lvbo[j][l];
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

template <int LPT>
hipError_t launch_lpt(const KernelParams& p, hipStream_t s) {
  const bool lm = p.lm_states != nullptr;
  const bool bt = p.bt_nodes != nullptr;
  dim3 grid(p.B), block(kThreads);
  if (lm && bt)
    hipLaunchKernelGGL((decode_kernel<LPT, true, true>), grid, block, 0, s, p);
  else if (lm)
    hipLaunchKernelGGL((decode_kernel<LPT, true, false>), grid, block, 0, s, p);
  else if (bt)
    hipLaunchKernelGGL((decode_kernel<LPT, false, true>), grid, block, 0, s, p);
  else
    hipLaunchKernelGGL((decode_kernel<LPT, false, false>), grid, block, 0, s, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const KernelParams& p, hipStream_t s) {
  if (p.B == 0) return hipSuccess;
  if (p.V <= 512) return launch_lpt<1>(p, s);
  if (p.V <= 1024) return launch_lpt<2>(p, s);
  if (p.V <= 2048) return launch_lpt<4>(p, s);
  return launch_lpt<8>(p, s);
}

}  // namespace ctcbeam
