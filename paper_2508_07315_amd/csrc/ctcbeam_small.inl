// Small-beam decoder: K <= 8 hypotheses, V <= 1024 tokens, no LM and no
// phrase boosting (gfx950).  Included by ctcbeam_small.hip.
//
// Same search as the general decoder (FlexCTC Algorithm 1 with the Eq. 1
// fold x = s_k + D[c], x += beta for emitting labels; TopK by (score desc,
// flat index asc); pruning; recombination; read-out of the hypothesis trie,
// Sec. III-A), laid out for the beam sizes of the paper's main tables
// (K = 4..8) without a language model:
//
// * one workgroup of 4 wave64 per utterance, one wave per SIMD; lane l of
//   wave w scores labels c = 64w + l + 256j, j < 4, for every live beam;
// * the beam itself (scores, last labels, transcript hashes and lengths)
//   lives in registers of wave 0 only (slot k in lane k): the selection and
//   the update run once, in that wave, instead of in every wave.
//
// Per frame: S (all waves) score every candidate in registers and publish
// the maxima of (beam, wave) groups; barrier; F (all waves) take the K-th
// largest group maximum (and, with K live beams, the smallest blank score) as
// a lower bound of the K-th best candidate and write the candidates at or
// above it to per-wave survivor segments; barrier; R (wave 0) ranks the blank
// candidates and the survivors exactly, builds the successors, prunes,
// recombines and writes the back-pointers; barrier.  More than 64 ranked
// entries (mass ties) fall back to an exact K-step extraction over all
// candidates.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ctcbeam_internal.h"
#include "ctcbeam_lane.h"

namespace ctcbeam {
namespace small {

using detail::kNegInf;
using detail::lanemask_lt;
using detail::mix_token;
using detail::order_key;
using detail::rdlane;

constexpr int kST = 256;             // threads: 4 wave64
constexpr int kSW = kST / 64;        // waves
constexpr int kLPL = 4;              // labels per lane
constexpr int kVmax = kST * kLPL;    // 1024 labels (blank handled apart)
constexpr int kKmax = 8;             // beam slots
constexpr int kSeg = 64;             // survivor entries per wave
constexpr int kStage = 2048;         // 64-bit words of the traceback tiles

// value of lane (lane ^ j) for compile-time j, with the lane masks
// materialised where they are used (a frame loop would otherwise keep every
// 64-bit mask live in scalar registers)
template <int J>
__device__ __forceinline__ uint32_t xlane(uint32_t v) {
  if constexpr (J == 1) return detail::dpp_full<detail::kDppQuadXor1>(v);
  else if constexpr (J == 2) return detail::dpp_full<detail::kDppQuadXor2>(v);
  else if constexpr (J == 4) {
    const uint32_t up = detail::dpp_mov<detail::kDppRowShl4>(v);
    const uint32_t dn = detail::dpp_mov<detail::kDppRowShr4>(v);
    return detail::lane_in_here<detail::kLanesBit2>() ? dn : up;
  } else if constexpr (J == 8) return detail::dpp_full<detail::kDppRowRor8>(v);
  else if constexpr (J == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return detail::lane_in_here<detail::kLanesBit4>() ? static_cast<uint32_t>(r[0]) : static_cast<uint32_t>(r[1]);
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return detail::lane_in_here<detail::kLanesBit5>() ? static_cast<uint32_t>(r[0]) : static_cast<uint32_t>(r[1]);
  }
}
template <int J>
__device__ __forceinline__ float xlanef(float v) { return __uint_as_float(xlane<J>(__float_as_uint(v))); }

__global__ void __launch_bounds__(kST) small_kernel(KernelParams p) {
  // back-pointer tiles of the traceback
  __shared__ __align__(16) uint64_t s_big[kStage];

  // this frame's candidates: [live position][thread] -> labels tid + 256 j
  __shared__ __align__(16) float4 s_cand[kKmax * kST];
  __shared__ uint4 s_seg[kSW][kSeg];     // survivors: score bits, flat index, 0, emits
  __shared__ int s_nseg[kSW];
  __shared__ int s_ovf;
  __shared__ float s_gmax[kSW * kKmax];  // (beam, wave) maxima
  // the beam as the scoring sees it, by live position (slot order; dead
  // positions score -inf): score bits, last label, 0, slot * W
  __shared__ uint4 s_beam[2][kKmax];  // [frame & 1] read by frame t
  __shared__ int s_nlive;
  // exact extraction (fallback): winners in rank order; wave maxima
  __shared__ uint4 s_win[kKmax];
  __shared__ __align__(16) uint64_t s_key[64];  // ranked keys (wave 0)
  // the beam's slot records (wave 0 writes them after each update): hash lo,
  // hi, length
  constexpr int kSlotWords = 4;
  __shared__ __align__(16) uint32_t s_slot[kKmax][kSlotWords];
  __shared__ uint64_t s_red[2][kSW];
  __shared__ int s_best, s_bestlen;
  __shared__ float s_bestscore;
  __shared__ int s_nblen[kKmax], s_nbrank[kKmax];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int b = blockIdx.x;
  const int V = p.V, W = V + 1, K = p.K, T = p.T;
  const float beta = p.beta;
  const bool want_stats = p.stats != nullptr;

  int L = p.lengths[b];
  uint32_t status = 0;
  if (L < 0) { L = 0; status |= 1u; }
  if (L > T) { L = T; status |= 1u; }
  const float* Db = p.logprobs + static_cast<size_t>(b) * T * W;
  int32_t* bpb = p.bp + static_cast<size_t>(b) * T * K;

  float rD[kLPL], rDn[kLPL];
#pragma unroll
  for (int j = 0; j < kLPL; ++j) {
    const int c = tid + j * kST;
    rDn[j] = (c < V && L > 0) ? Db[c] : kNegInf;
    rD[j] = kNegInf;
  }

  // ---- the beam (wave 0, slot k in lane k) ----
  float sc = (lane == 0) ? 0.0f : kNegInf;
  int last = V, len = 0;
  uint32_t hlo = 0u, hhi = 0u;

  // counters (wave 0 lanes, summed at the end)
  uint32_t st_alive = 0u, st_emit = 0u;

  if (tid < kKmax) {
    // slot records: slot 0 is the initial (empty) beam, the others never parents
#pragma unroll
    for (int w = 0; w < kSlotWords; ++w) s_slot[tid][w] = 0u;
    s_beam[0][tid] = make_uint4(__float_as_uint(tid == 0 ? 0.0f : kNegInf), static_cast<uint32_t>(V), 0u, 0u);
  }
  if (tid == 0) {
    s_nlive = L > 0 ? 1 : 0;
    s_ovf = 0;
  }
  __syncthreads();

  for (int t = 0; t < L; ++t) {
    const int cb = t & 1;  // double buffers read by this frame
    // labels past V read the row's blank and score -inf (the prefetched
    // values are used only here, a frame after their loads were issued)
#pragma unroll
    for (int j = 0; j < kLPL; ++j) rD[j] = (tid + j * kST < V) ? rDn[j] : kNegInf;
    if (t + 1 < L) {
      const float* rowp = Db + static_cast<size_t>(t + 1) * W;
#pragma unroll
      for (int j = 0; j < kLPL; ++j) rDn[j] = __builtin_nontemporal_load(rowp + min(tid + j * kST, V));
    }
    const float dblank = Db[static_cast<size_t>(t) * W + V];
    const int nlive = __builtin_amdgcn_readfirstlane(s_nlive);

    // ---- S. candidates of every beam position, straight-line ----
    uint4 brec[kKmax];
#pragma unroll
    for (int i = 0; i < kKmax; ++i) brec[i] = s_beam[cb][i];  // broadcast reads
    float cand[kKmax][kLPL];
    float rmax[kKmax];
#pragma unroll
    for (int i = 0; i < kKmax; ++i) {
      const float si = __uint_as_float(brec[i].x);
      const int lasti = static_cast<int>(brec[i].y);
#pragma unroll
      for (int j = 0; j < kLPL; ++j) {
        const int c = tid + j * kST;
        const float x0 = si + rD[j];
        const float x = x0 + beta;
        // the repeat of the beam's last frame label emits nothing
        cand[i][j] = (c == lasti) ? x0 : x;
      }
      rmax[i] = fmaxf(fmaxf(cand[i][0], cand[i][1]), fmaxf(cand[i][2], cand[i][3]));
      s_cand[i * kST + tid] = make_float4(cand[i][0], cand[i][1], cand[i][2], cand[i][3]);
    }
    {
      // wave maxima of the 8 beam groups: a transposed reduction halves the
      // groups a lane carries at lane-bit steps 1, 2, 4, then reduces over
      // lane bits 3..5; lane l ends with group 4(l&1) + 2(l>>1&1) + (l>>2&1)
      const bool b0 = detail::lane_in_here<0xAAAAAAAAAAAAAAAAull>();
      float m4[4], m2[2];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        m4[q] = fmaxf(b0 ? rmax[q + 4] : rmax[q], xlanef<1>(b0 ? rmax[q] : rmax[q + 4]));
      const bool b1 = detail::lane_in_here<0xCCCCCCCCCCCCCCCCull>();
#pragma unroll
      for (int q = 0; q < 2; ++q)
        m2[q] = fmaxf(b1 ? m4[q + 2] : m4[q], xlanef<2>(b1 ? m4[q] : m4[q + 2]));
      const bool b2 = detail::lane_in_here<detail::kLanesBit2>();
      float m1 = fmaxf(b2 ? m2[1] : m2[0], xlanef<4>(b2 ? m2[0] : m2[1]));
      m1 = fmaxf(m1, xlanef<8>(m1));
      m1 = fmaxf(m1, xlanef<16>(m1));
      m1 = fmaxf(m1, xlanef<32>(m1));
      if (lane < kKmax) s_gmax[wave * kKmax + lane] = m1;
    }
    if (tid == 0) s_ovf = 0;
    __syncthreads();  // B1: group maxima, candidates

    // ---- F. bound and survivors ----
    {
      // K-th largest of the (beam, wave) maxima: maxima of disjoint groups
      // are distinct candidates, so at least K candidates reach it
      float g = lane < kSW * kKmax ? s_gmax[lane] : kNegInf;
      g = detail::wave_sort_desc<32>(g, lane);
      float tau = rdlane(g, K - 1);
      if (nlive == K) {
        // the K blank candidates: the K-th best is at least their minimum
        float tb = __builtin_huge_valf();
#pragma unroll
        for (int i = 0; i < kKmax; ++i)
          if (i < K) tb = detail::fmin_sel(tb, __uint_as_float(brec[i].x) + dblank);
        tau = fmaxf(tau, tb);
      }
      // an infinite bound admits every finite candidate and no -inf one
      tau = fmaxf(tau, -__FLT_MAX__);
      uint32_t q = 0u;
#pragma unroll
      for (int i = 0; i < kKmax; ++i) {
        if (__ballot(rmax[i] >= tau) != 0ull) {  // uniform
#pragma unroll
          for (int j = 0; j < kLPL; ++j) q |= (cand[i][j] >= tau) ? (1u << (i * kLPL + j)) : 0u;
        }
      }
      const int cnt = __popc(q);
      const int incl = detail::wave_incl_scan(cnt, lane);
      const int tot = rdlane(incl, 63);
      if (tot > kSeg) {
        if (lane == 0) s_ovf = 1;
      } else {
        int at = incl - cnt;
        for (uint32_t qq = q; qq != 0u; qq &= qq - 1u) {  // a lane's survivors (usually none)
          const int r = __builtin_ctz(qq);
          const int i = r >> 2;
          const uint32_t c = static_cast<uint32_t>(tid + (r & 3) * kST);
          const float x = reinterpret_cast<const float*>(s_cand)[(i * kST + tid) * 4 + (r & 3)];
          const uint4 br = s_beam[cb][i];
          s_seg[wave][at++] = make_uint4(__float_as_uint(x), br.w + c, 0u, c != br.y ? 1u : 0u);
        }
      }
      if (lane == 0) s_nseg[wave] = tot;
    }
    __syncthreads();  // B2: survivors

    // ---- R. exact selection of the K best ----
    const int n0 = s_nseg[0], n1 = s_nseg[1], n2 = s_nseg[2], n3 = s_nseg[3];
    const int N = nlive + n0 + n1 + n2 + n3;
    const bool fallback = s_ovf != 0 || N > 64;  // uniform
    int nfin = 0;
    if (fallback) {
      // K rounds of "best key below the previous one" over every candidate
      // (read back from LDS, rolled loops: a rare path kept small) and the
      // blank candidates (wave 0).  A winner is named by its code: live
      // position << 10 | label.
      uint64_t prev = ~0ull;
      for (int it = 0; it < K; ++it) {
        uint64_t best = 0ull;
        uint32_t wcode = 0u;
#pragma unroll 1
        for (int i = 0; i < kKmax; ++i) {
          const float4 cv = s_cand[i * kST + tid];
          const uint32_t sb = s_beam[cb][i].w;
          const float xs[kLPL] = {cv.x, cv.y, cv.z, cv.w};
#pragma unroll
          for (int j = 0; j < kLPL; ++j) {
            const uint32_t c = static_cast<uint32_t>(tid + j * kST);
            const uint64_t key = xs[j] != kNegInf ? order_key(xs[j], sb + c) : 0ull;
            const bool better = key < prev && key > best;
            best = better ? key : best;
            wcode = better ? ((static_cast<uint32_t>(i) << 10) | c) : wcode;
          }
        }
        if (wave == 0 && lane < nlive) {
          const uint4 br = s_beam[cb][lane];
          const float x = __uint_as_float(br.x) + dblank;
          const uint64_t key = x != kNegInf ? order_key(x, br.w + static_cast<uint32_t>(V)) : 0ull;
          const bool better = key < prev && key > best;
          best = better ? key : best;
          wcode = better ? ((static_cast<uint32_t>(lane) << 10) | 0x8000u) : wcode;  // blank of position lane
        }
        uint64_t wb = best;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const uint64_t o = __shfl_xor(wb, off);
          wb = o > wb ? o : wb;
        }
        if (lane == 0) s_red[it & 1][wave] = wb;
        __syncthreads();
        uint64_t gb = s_red[it & 1][0];
#pragma unroll
        for (int w = 1; w < kSW; ++w) gb = s_red[it & 1][w] > gb ? s_red[it & 1][w] : gb;
        if (gb == 0ull) break;  // nothing finite left (uniform)
        if (best == gb && best != 0ull) {
          const uint32_t i = (wcode >> 10) & 7u;
          const uint4 br = s_beam[cb][i];
          uint4 win;
          if (wcode & 0x8000u) {
            win = make_uint4(__float_as_uint(__uint_as_float(br.x) + dblank), br.w + static_cast<uint32_t>(V), 0u, 0u);
          } else {
            const uint32_t c = wcode & 1023u;
            const float x = reinterpret_cast<const float*>(s_cand)[(i * kST + (c & 255u)) * 4u + (c >> 8)];
            win = make_uint4(__float_as_uint(x), br.w + c, 0u, 0u);
          }
          s_win[it] = win;
        }
        prev = gb;
        ++nfin;
      }
      __syncthreads();  // s_win complete
    }

    if (wave == 0) {
      // ---- entries (normal path): lane l < nlive the blank candidate of live
      // position l, then the four survivor segments ----
      float ex = kNegInf;
      uint32_t eidx = 0xFFFFFFFFu;
      if (!fallback) {
        if (lane < nlive) {
          const uint4 br = s_beam[cb][lane];
          ex = __uint_as_float(br.x) + dblank;
          eidx = br.w + static_cast<uint32_t>(V);
        } else if (lane < N) {
          int e = lane - nlive, w = 0;
          if (e >= n0) { e -= n0; w = 1; if (e >= n1) { e -= n1; w = 2; if (e >= n2) { e -= n2; w = 3; } } }
          const uint4 v = s_seg[w][e];
          ex = __uint_as_float(v.x);
          eidx = v.y;
        }
      } else if (lane < nfin) {
        const uint4 v = s_win[lane];
        ex = __uint_as_float(v.x);
        eidx = v.y;
      }
      const bool evalid = ex != kNegInf;
      // parent slot, label, emission
      const uint32_t epar = evalid ? eidx / static_cast<uint32_t>(W) : 0u;
      const int ec = evalid ? static_cast<int>(eidx - epar * static_cast<uint32_t>(W)) : V;
      const int elast = __builtin_amdgcn_ds_bpermute(static_cast<int>(epar) << 2, last);
      const bool eemit = evalid && ec != V && ec != elast;
      int src = lane;  // entry lane of winner `lane`
      if (!fallback) {
        // rank: the entries' keys counted from broadcast LDS reads, two at a
        // time (lanes past N hold key 0)
        const uint64_t key = evalid ? order_key(ex, eidx) : 0ull;
        s_key[lane] = key;
        int rank = 0;
        const int N2 = (N + 1) >> 1;
#pragma unroll 4
        for (int m2 = 0; m2 < N2; ++m2) {  // uniform trip count
          const ulonglong2 kk = reinterpret_cast<const ulonglong2*>(s_key)[m2];
          rank += (kk.x > key ? 1 : 0) + (kk.y > key ? 1 : 0);
        }
        nfin = min(K, static_cast<int>(__popcll(__ballot(evalid))));
        // winner of rank r learns its entry lane (others write to lane 63,
        // which no winner reads: K <= 8)
        const int dst = (evalid && rank < K) ? rank : 63;
        src = __builtin_amdgcn_ds_permute(dst << 2, lane);
      }
      // cross-lane reads run with every lane active (a source lane that is
      // inactive reads as 0), so none sits in a short-circuit operand
      const bool valid = lane < nfin;
      float x = __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(ex)));
      const int pk = __builtin_amdgcn_ds_bpermute(src << 2, static_cast<int>(epar & 7u) | (ec << 3) | ((eemit ? 1 : 0) << 14));
      const int par = pk & 7;
      const int c = (pk >> 3) & 2047;
      const bool emit = valid && ((pk >> 14) & 1);
      if (!valid) x = kNegInf;

      // counters: the beams entering this frame
      if (want_stats && lane < K && sc != kNegInf) st_alive += 1u;

      // successor of the parent slot (its record, from LDS)
      uint32_t prec[kSlotWords];
#pragma unroll
      for (int w4 = 0; w4 < kSlotWords; w4 += 4) {
        const uint4 v = *reinterpret_cast<const uint4*>(&s_slot[par][w4]);
        prec[w4] = v.x;
        prec[w4 + 1] = v.y;
        prec[w4 + 2] = v.z;
        prec[w4 + 3] = v.w;
      }
      const uint32_t plo = prec[0], phi = prec[1];
      const int plen = static_cast<int>(prec[2]);
      uint64_t h = (static_cast<uint64_t>(phi) << 32) | plo;
      const uint64_t hm = mix_token(h, static_cast<uint32_t>(c));
      h = emit ? hm : h;
      const int nlen = plen + (emit ? 1 : 0);
      const int nlast = valid ? c : V;

      // prune (Algorithm 1: below best - theta -> -inf)
      const float lim = rdlane(x, 0) - p.theta;
      if (valid && x < lim) x = kNegInf;
      if (want_stats && x != kNegInf && emit) st_emit += 1u;
      // recombination: same transcript hash, length and ends-in-blank flag as
      // a live lower slot (slots in lanes 0..7 of one 16-lane row)
      const bool alive0 = valid && x != kNegInf;
      const uint32_t meta = (static_cast<uint32_t>(nlen) & 0x3FFFFFFFu) | ((nlast == V ? 1u : 0u) << 30);
      uint64_t rkey = h ^ (static_cast<uint64_t>(meta + 1u) * 0xD6E8FEB86659FD93ull);
      if (!alive0) rkey = ~0ull;
      const bool dup = detail::recomb_shifts<1, 7>(static_cast<uint32_t>(rkey), static_cast<uint32_t>(rkey >> 32)) && alive0;
      const bool alive = alive0 && !dup;
      if (lane < K) bpb[static_cast<size_t>(t) * K + lane] = valid ? ((par << 16) | c) : -1;

      // the beam after this frame
      sc = alive ? x : kNegInf;
      last = nlast;
      len = nlen;
      hlo = static_cast<uint32_t>(h);
      hhi = static_cast<uint32_t>(h >> 32);
      if (lane < K) *reinterpret_cast<uint4*>(&s_slot[lane][0]) = make_uint4(hlo, hhi, static_cast<uint32_t>(len), 0u);
      const uint64_t am = __ballot(alive && lane < K);
      // the beam as the next frame's scoring sees it (positions past the
      // live slots score -inf)
      const int na = static_cast<int>(__popcll(am));
      if (alive && lane < K) {
        const int lp = static_cast<int>(__popcll(am & lanemask_lt()));
        s_beam[cb ^ 1][lp] = make_uint4(__float_as_uint(sc), static_cast<uint32_t>(last), 0u,
                                        static_cast<uint32_t>(lane * W));
      }
      if (lane >= na && lane < kKmax)
        s_beam[cb ^ 1][lane] = make_uint4(__float_as_uint(kNegInf), static_cast<uint32_t>(V), 0u, 0u);
      if (lane == 0) s_nlive = na;
    }
    __syncthreads();  // B3: beam table
  }

  // ---- the order of the final hypotheses (wave 0) ----
  const bool nbest = p.nbest_scores != nullptr;
  if (wave == 0) {
    const float s = sc;
    const float sj = lane < K ? s : kNegInf;
    // rank: final score descending, lowest slot on ties
    int rank = 0;
    for (int i = 0; i < K; ++i) {
      const float si = rdlane(sj, i);
      rank += (si > sj || (si == sj && i < lane)) ? 1 : 0;
    }
    const int bj = static_cast<int>(__builtin_ctzll(__ballot(lane < K && rank == 0)));
    const int nlen = (lane < K && sj != kNegInf) ? len : 0;
    if (nbest && lane < K) {
      p.nbest_scores[static_cast<size_t>(b) * K + rank] = sj;
      p.nbest_lengths[static_cast<size_t>(b) * K + rank] = nlen;
      s_nblen[rank] = nlen;
      s_nbrank[lane] = rank;
    }
    const float bsc = rdlane(sj, bj);
    const int blen = rdlane(len, bj);
    if (lane == 0) {
      s_best = bj;
      s_bestscore = bsc;
      s_bestlen = blen;
    }
    if (want_stats) {
      uint32_t a0 = st_alive, a3 = st_emit;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        a0 += __shfl_xor(a0, off);
        a3 += __shfl_xor(a3, off);
      }
      if (lane == 0) {
        int64_t* so = p.stats + static_cast<size_t>(b) * 8;
        so[0] = L;
        so[1] = a0;
        so[2] = 0;
        so[3] = 0;
        so[4] = 0;
        so[5] = 0;
        so[6] = a3;
        so[7] = 0;
      }
    }
  }
  __syncthreads();
  const int best = s_best;
  const float bscore = s_bestscore;
  const bool have = bscore != kNegInf;
  const int nout = have ? s_bestlen : 0;
  int32_t* ot = p.out_tokens ? p.out_tokens + static_cast<size_t>(b) * T : nullptr;
  if (ot)
    for (int tt = nout + tid; tt < T; tt += kST) ot[tt] = -1;
  if (tid == 0 && p.out_scores) {
    p.out_scores[b] = bscore;
    if (p.out_lengths) p.out_lengths[b] = nout;
  }
  int32_t* nbt = nbest ? p.nbest_tokens + static_cast<size_t>(b) * K * T : nullptr;
  if (nbest) {
    for (int r = 0; r < K; ++r) {
      const int n = s_nblen[r];
      for (int tt = n + tid; tt < T; tt += kST) nbt[static_cast<size_t>(r) * T + tt] = -1;
    }
  }

  // ---- traceback through the back-pointers, staged in LDS tiles ----
  // 1-best: lane 0 of wave 0 walks the best slot; N-best: lane k of wave 0
  // walks live slot k into the row of its rank
  const bool walker = wave == 0 && (nbest ? (lane < K && sc != kNegInf) : (lane == 0 && have));
  if (have && L > 0) {
    uint32_t* stg = reinterpret_cast<uint32_t*>(s_big);
    const int tile_frames = (kStage * 2) / K;
    int jb = nbest ? lane : best, cnext = -1, pos = 0;
    int32_t* orow = nullptr;
    if (walker) {
      orow = nbest ? nbt + static_cast<size_t>(s_nbrank[lane]) * T : ot;
      pos = nbest ? len : nout;
    }
    for (int hi = L; hi > 0;) {
      const int lo = hi > tile_frames ? hi - tile_frames : 0;
      __syncthreads();
      const int n = (hi - lo) * K;
      const int32_t* src = bpb + static_cast<size_t>(lo) * K;
      for (int q = tid; q < n; q += kST) stg[q] = static_cast<uint32_t>(src[q]);
      __syncthreads();
      if (walker) {
        for (int tt = hi - 1; tt >= lo; --tt) {
          const uint32_t e = stg[(tt - lo) * K + jb];
          const int cl = static_cast<int>(e & 0xFFFFu);
          const int pr = static_cast<int>(e >> 16);
          if (tt < L - 1 && cnext != V && cnext != cl && pos > 0) {
            --pos;
            if (orow) orow[pos] = cnext;
          }
          cnext = cl;
          jb = pr < K ? pr : 0;  // a live slot's ancestors are live: pr < K (else the walk ends unbalanced)
        }
      }
      hi = lo;
    }
    if (walker && cnext != V && cnext >= 0 && pos > 0) {
      --pos;
      if (orow) orow[pos] = cnext;
    }
    if (wave == 0 && __ballot(walker && pos != 0) != 0ull) status |= 2u;
  }
  if (tid == 0) {
    p.status[b] = status;
    if (b == 0) write_ws_header(p.ws_header, p.B);
  }
}

hipError_t launch(const KernelParams& p, hipStream_t s) {
  hipLaunchKernelGGL(small_kernel, dim3(p.B), dim3(kST), 0, s, p);
  return hipGetLastError();
}

}  // namespace small

// The small-beam decoder serves beams of at most 8 without an LM or boosting,
// where it is faster than the general one (1.45 vs 1.72 ms at K = 8 and 1.25
// vs 1.67 ms at K = 4 on 32 utterances of 400 frames, V = 1024).  A form with
// LM rows kept in LDS and the update in one wave lost to the general decoder
// (2.46 vs 2.07 ms on the 3-gram workload at K = 8) and was removed.
bool small_beam_eligible(const KernelParams& p) {
  if (p.bt_nodes != nullptr || p.lm_states != nullptr || p.lm_arcs != nullptr) return false;
  if (p.K > small::kKmax || p.V > small::kVmax) return false;
  return (p.flags & (kFlagNoRowCache | kFlagLogSumExp | kFlagRepeatScore)) == 0;
}

hipError_t launch_small(const KernelParams& p, hipStream_t s) { return small::launch(p, s); }

}  // namespace ctcbeam
