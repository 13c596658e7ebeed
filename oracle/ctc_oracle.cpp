// CPU ORACLE - TEST INFRASTRUCTURE ONLY.
//
// A plain, slow, obviously-correct reference of the batched CTC beam search
// with n-gram LM shallow fusion and phrase boosting (FlexCTC, Algorithm 1 and
// Eq. 1).  Only the test suite, the smoke check and the CPU-baseline leg of
// the benchmark may load it; the product path never does.  It shares no code
// with the HIP implementation.
//
// Arithmetic: IEEE fp32, round-to-nearest-even, no FMA contraction (build with
// -ffp-contract=off), no fast-math.  The paper measures in float32 (Sec. IV-C
// "Metrics"), so fp32 is the method's precision; the fold order of every sum is
// fixed below and the HIP path follows the same order.
//
// Readings of points the paper leaves open (each is also listed in the design
// notes of the repository):
//   * labels 0..V-1 are tokens, V is blank, W = V+1; the flat candidate index
//     is i = k*W + c, so label = i mod W and beam = i div W (Alg. 1, TopK);
//   * the repeat mask compares with the previous *frame* label of the beam,
//     blank included; the initial last label is blank (Alg. 1, masks);
//   * candidate score (Alg. 1 score update, Eq. 1):
//       x = s_k + D_t[c];  if c is neither blank nor a repeat:
//       x = x + beta;  x = x + fl(alpha * LM(k,c));  x = x + fl(w * BT(k,c));
//   * TopK order: score descending, flat index ascending on ties;
//   * threshold pruning: x_j < x_0 - theta  ->  -inf (Alg. 1, pruning);
//   * recombination (Alg. 1 RecombineHypotheses, Sec. III-A): two live
//     hypotheses are the same when their collapsed transcripts are equal and
//     both or neither end in blank; the lower slot (higher score) survives
//     with its own score (max, Viterbi) and dead slots stay in place;
//   * final: alive scores get fl(alpha * LM(k, </s>)) (Alg. 1, LM.Final);
//   * variants (flags; Sec. III-C leaves them open): bit 0 merges recombined
//     hypotheses by log-sum-exp instead of max -- the surviving lower slot
//     takes lse32(own, other) for each later duplicate in slot order, which
//     sums the probability of all alignments of a transcript; bit 1 rolls
//     back the pending boosting of an unfinished phrase at the end of the
//     utterance: after LM.Final, alive scores get fl(w * -pot(q)); bit 2
//     scores repeated emissions with the LM and boosting at every
//     occurrence (Sec. III-C mentions this as a tried alternative): a frame
//     that repeats the beam's last frame label (a token) adds again the
//     fl(alpha * LM) and fl(w * BT) terms that the token received when it was
//     emitted, x = ((s + D[c]) + al) + wb, with no beta and no state change
//     (the LM and boosting states advance once per token of the transcript);
//   * output: best slot, lowest index on ties; if its score is -inf the
//     transcript is empty and the score -inf;
//   * N-best output (all K final hypotheses, the batched-hypotheses result of
//     Alg. 1): the slots ordered by final score descending, lowest slot on
//     ties, each with its transcript; dead slots come last with an empty
//     transcript and score -inf.
//
// LM(k,c): ARPA backoff in natural log (Sec. II "NGPU-LM"; Sec. IV-A builds the
// LM from an ARPA file).  P(c|h) = p(h c) if that n-gram exists, otherwise
// bo(h) + P(c|h minus its oldest symbol), bo(h) = 0 if h is not an entry; the
// base case is the unigram.  Each stored value is fl(double(log10) * ln 10),
// zero canonicalised to +0.  The fp32 sum is formed innermost (shortest
// context) first: inner + bo.
//
// BT(k,c): token-level phrase boosting (Sec. III-B: an Aho-Corasick phrase
// tree whose score is spread over the nodes by depth).  The paper leaves the
// tree's exact rules to the cited GPU-PB work; the definition used here:
//   nodes  = all prefixes of the phrases (root = empty);
//   pot(n) = |n| - (length of the longest whole phrase that is a prefix of n)
//            (tokens matched but not yet banked by a completed phrase);
//   f(n)   = the longest suffix u of n, |u| < |n| and |u| <= pot(n), that is a
//            node; root if none (so a completed phrase restarts at root);
//   step(q, c): q c a node -> (+1, q c); q root -> (0, root);
//               else -> (pot(f(q)) - pot(q)) + step(f(q), c).
// Progress along a phrase earns +1 per token, a mismatch rolls back the
// pending tokens, a completed phrase is banked.  This file evaluates it with
// string operations on a set of prefixes, never with failure arrays.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <set>
#include <string>
#include <thread>
#include <unordered_map>
#include <utility>
#include <vector>

namespace {

const float NEG_INF = -std::numeric_limits<float>::infinity();

std::string key_of(const int32_t* ids, size_t n) {
  return std::string(reinterpret_cast<const char*>(ids), n * sizeof(int32_t));
}
std::string key_of(const std::vector<int32_t>& v) { return key_of(v.data(), v.size()); }

float log10_to_ln(float v) {
  const double LN10 = 2.302585092994045684017991454684364208;
  float f = static_cast<float>(static_cast<double>(v) * LN10);
  if (f == 0.0f) f = 0.0f;  // +0 only
  return f;
}

struct OracleLM {
  int order = 0, V = 0;
  std::unordered_map<std::string, float> prob;  // ln p of every n-gram
  std::unordered_map<std::string, float> bow;   // ln backoff weight of every entry that has one
  std::unordered_map<std::string, int64_t> n_cont;  // explicit continuations per context (instrumentation)

  bool exists(const std::vector<int32_t>& g) const { return prob.count(key_of(g)) != 0; }

  // P(c | h) following the backoff recursion (ARPA semantics).
  float backoff(const std::vector<int32_t>& h, int32_t c) const {
    std::vector<int32_t> g = h;
    g.push_back(c);
    auto it = prob.find(key_of(g));
    if (it != prob.end()) return it->second;
    if (h.empty()) return NEG_INF;  // no unigram: unreachable for valid models
    float b = 0.0f;
    auto ib = bow.find(key_of(h));
    if (ib != bow.end()) b = ib->second;
    std::vector<int32_t> shorter(h.begin() + 1, h.end());
    float inner = backoff(shorter, c);
    return inner + b;
  }

  // Context of a hypothesis: the last min(order-1, |hist|) symbols of <s> y.
  std::vector<int32_t> context(const std::vector<int32_t>& y) const {
    std::vector<int32_t> hist;
    hist.reserve(y.size() + 1);
    hist.push_back(V + 1);
    hist.insert(hist.end(), y.begin(), y.end());
    size_t m = std::min<size_t>(static_cast<size_t>(order - 1), hist.size());
    return std::vector<int32_t>(hist.end() - m, hist.end());
  }

  float score(const std::vector<int32_t>& y, int32_t c) const { return backoff(context(y), c); }

  // Instrumentation: existing suffix contexts of lengths 1..order-1 and their arcs.
  void chain_counts(const std::vector<int32_t>& y, int64_t* states, int64_t* arcs) const {
    std::vector<int32_t> h = context(y);
    for (size_t l = 1; l <= h.size(); ++l) {
      std::vector<int32_t> suf(h.end() - l, h.end());
      std::string k = key_of(suf);
      if (prob.count(k)) {
        *states += 1;
        auto it = n_cont.find(k);
        if (it != n_cont.end()) *arcs += it->second;
      }
    }
  }
};

struct OracleBT {
  int V = 0;
  std::set<std::vector<int32_t>> nodes;    // all non-empty prefixes
  std::set<std::vector<int32_t>> phrases;  // whole phrases
  std::unordered_map<std::string, int64_t> n_children;  // instrumentation

  bool is_node(const std::vector<int32_t>& n) const { return n.empty() || nodes.count(n) != 0; }

  int banked(const std::vector<int32_t>& n) const {
    for (size_t l = n.size(); l >= 1; --l) {
      std::vector<int32_t> p(n.begin(), n.begin() + l);
      if (phrases.count(p)) return static_cast<int>(l);
    }
    return 0;
  }
  int pot(const std::vector<int32_t>& n) const { return static_cast<int>(n.size()) - banked(n); }

  std::vector<int32_t> fail(const std::vector<int32_t>& n) const {
    int lim = std::min(pot(n), static_cast<int>(n.size()) - 1);
    for (int l = lim; l >= 1; --l) {
      std::vector<int32_t> u(n.end() - l, n.end());
      if (nodes.count(u)) return u;
    }
    return {};
  }

  // Returns the score of consuming c in state q; *next receives the new state.
  int step(const std::vector<int32_t>& q, int32_t c, std::vector<int32_t>* next) const {
    std::vector<int32_t> qc = q;
    qc.push_back(c);
    if (nodes.count(qc)) {
      *next = qc;
      return 1;
    }
    if (q.empty()) {
      next->clear();
      return 0;
    }
    std::vector<int32_t> f = fail(q);
    int s = step(f, c, next);
    return (pot(f) - pot(q)) + s;
  }

  void chain_counts(const std::vector<int32_t>& q, int64_t* n_nodes, int64_t* n_arcs) const {
    std::vector<int32_t> x = q;
    while (!x.empty()) {
      *n_nodes += 1;
      auto it = n_children.find(key_of(x));
      if (it != n_children.end()) *n_arcs += it->second;
      x = fail(x);
    }
  }
};

struct Hyp {
  float s = NEG_INF;
  int32_t last = 0;
  float rep_al = 0.0f;      // fl(alpha * LM) and fl(w * BT) received by the
  float rep_wb = 0.0f;      // last emitted token (repeat-scoring variant)
  std::vector<int32_t> y;   // collapsed transcript
  std::vector<int32_t> q;   // boosting-tree state (node string)
};

struct Cand {
  float x;
  int64_t i;
};

// ---- fp32 log-sum-exp, every step an IEEE fp32 operation in a fixed order
// (so that any implementation following the same steps gets the same bits).
// exp: Cody-Waite reduction d = k ln2 + r, k = rint(d / ln2), |r| <= ln2/2,
// with ln2 split into a 9-bit head (k * head exact) and a tail, then the
// degree-7 Taylor polynomial of e^r by Horner, scaled by 2^k.  Valid for
// -80 <= d <= 0 (2^k stays a normal number).
float exp32_nonpos(float d) {
  const float inv_ln2 = 1.44269504f;
  const float ln2_hi = 0.693359375f;
  const float ln2_lo = -2.12194440e-4f;
  const float k = std::nearbyint(d * inv_ln2);
  const float r = (d - k * ln2_hi) - k * ln2_lo;
  float p = 1.0f / 5040.0f;
  p = p * r + 1.0f / 720.0f;
  p = p * r + 1.0f / 120.0f;
  p = p * r + 1.0f / 24.0f;
  p = p * r + 1.0f / 6.0f;
  p = p * r + 0.5f;
  p = p * r + 1.0f;
  p = p * r + 1.0f;
  const int ki = static_cast<int>(k);
  uint32_t bits = static_cast<uint32_t>(ki + 127) << 23;
  float scale;
  std::memcpy(&scale, &bits, sizeof(scale));
  return p * scale;
}

// log(1 + e) for 2^-24 <= e <= 1: with s = e / (2 + e), log(1 + e) =
// 2 atanh(s) = 2 s (1 + s^2/3 + s^4/5 + ... + s^16/17), s <= 1/3.
float log1p32_unit(float e) {
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

// log(exp(a) + exp(b)) in fp32.
float lse32(float a, float b) {
  if (a < b) std::swap(a, b);
  if (b == NEG_INF) return a;
  const float d = b - a;
  if (d < -80.0f) return a;
  const float e = exp32_nonpos(d);
  const float l = (e < 5.9604645e-8f) ? e : log1p32_unit(e);
  return a + l;
}

constexpr int kFlagLogSumExp = 1;
constexpr int kFlagBoostRollback = 2;
constexpr int kFlagRepeatScore = 4;

struct DecodeArgs {
  const float* logprobs;
  const int32_t* lengths;
  int B, T, V, K;
  float alpha, beta, boost_w, theta;
  int flags;
  const OracleLM* lm;
  const OracleBT* bt;
  int32_t* out_tokens;
  int32_t* out_lengths;
  float* out_scores;
  int32_t* out_align;     // [B,T] frame labels of the best path, -1 padded (nullable)
  int32_t* bp_index;      // [B,T,K] flat candidate index of each slot (nullable)
  float* slot_scores;     // [B,T,K] slot scores after recombination (nullable)
  int64_t* counters;      // [B,8] (nullable)
  int32_t* nbest_tokens;  // [B,K,T] -1 padded (nullable: no N-best output)
  int32_t* nbest_lengths; // [B,K]
  float* nbest_scores;    // [B,K]
};

void decode_one(const DecodeArgs& a, int b) {
  const int V = a.V, W = V + 1, K = a.K, T = a.T;
  int L = a.lengths[b];
  if (L < 0) L = 0;
  if (L > T) L = T;
  const float* Db = a.logprobs + static_cast<size_t>(b) * T * W;
  int64_t cnt[8] = {0, 0, 0, 0, 0, 0, 0, 0};

  std::vector<Hyp> hyp(K);
  for (int k = 0; k < K; ++k) hyp[k].last = V;
  hyp[0].s = 0.0f;
  std::vector<std::vector<int32_t>> frame_parent(L, std::vector<int32_t>(K, 0));
  std::vector<std::vector<int32_t>> frame_label(L, std::vector<int32_t>(K, V));

  std::vector<Cand> cand(static_cast<size_t>(K) * W);
  std::vector<float> lmv(W), btv(W);
  std::vector<int32_t> tmp;
  for (int t = 0; t < L; ++t) {
    const float* D = Db + static_cast<size_t>(t) * W;
    cnt[0] += 1;
    // Candidate scores (Alg. 1 score update; Eq. 1).
    for (int k = 0; k < K; ++k) {
      const Hyp& h = hyp[k];
      bool alive = h.s != NEG_INF;
      if (alive) {
        cnt[1] += 1;
        if (a.lm) a.lm->chain_counts(h.y, &cnt[2], &cnt[3]);
        if (a.bt) a.bt->chain_counts(h.q, &cnt[4], &cnt[5]);
      }
      for (int c = 0; c < W; ++c) {
        float x = h.s + D[c];
        bool emit = (c != V) && (c != h.last);
        const bool rep = (a.flags & kFlagRepeatScore) && c != V && c == h.last;
        if (rep && alive) {
          if (a.lm) x = x + h.rep_al;
          if (a.bt) x = x + h.rep_wb;
        }
        if (emit && alive) {
          x = x + a.beta;
          if (a.lm) {
            float l = a.lm->score(h.y, c);
            float al = a.alpha * l;
            x = x + al;
          }
          if (a.bt) {
            int sc = a.bt->step(h.q, c, &tmp);
            float wb = a.boost_w * static_cast<float>(sc);
            x = x + wb;
          }
        }
        // a dead beam stays -inf whatever is added to it
        cand[static_cast<size_t>(k) * W + c] = Cand{x, static_cast<int64_t>(k) * W + c};
      }
    }
    // TopK: score descending, index ascending.
    std::partial_sort(cand.begin(), cand.begin() + K, cand.end(), [](const Cand& p, const Cand& q) {
      if (p.x > q.x) return true;
      if (p.x < q.x) return false;
      return p.i < q.i;
    });
    // Threshold pruning.
    float m = cand[0].x;
    float lim = m - a.theta;
    std::vector<Hyp> nh(K);
    for (int j = 0; j < K; ++j) {
      float x = cand[j].x;
      if (x < lim) x = NEG_INF;
      int p = static_cast<int>(cand[j].i / W);
      int c = static_cast<int>(cand[j].i % W);
      const Hyp& ph = hyp[p];
      bool emit = (c != V) && (c != ph.last);
      Hyp n;
      n.s = x;
      n.last = c;
      n.y = ph.y;
      n.q = ph.q;
      n.rep_al = ph.rep_al;
      n.rep_wb = ph.rep_wb;
      if (emit) {
        if (a.lm) n.rep_al = a.alpha * a.lm->score(ph.y, c);
        n.y.push_back(c);
        if (a.bt) {
          const int sc = a.bt->step(ph.q, c, &tmp);
          n.rep_wb = a.boost_w * static_cast<float>(sc);
          n.q = tmp;
        }
        if (x != NEG_INF) cnt[6] += 1;
      }
      nh[j] = std::move(n);
      frame_parent[t][j] = p;
      frame_label[t][j] = c;
    }
    // Recombination: same collapsed transcript and same ends-in-blank flag;
    // the first live slot of a transcript absorbs the later ones.
    for (int j = 1; j < K; ++j) {
      if (nh[j].s == NEG_INF) continue;
      for (int i = 0; i < j; ++i) {
        if (nh[i].s == NEG_INF) continue;
        if (nh[i].y == nh[j].y && ((nh[i].last == V) == (nh[j].last == V))) {
          if (a.flags & kFlagLogSumExp) nh[i].s = lse32(nh[i].s, nh[j].s);
          nh[j].s = NEG_INF;
          break;
        }
      }
    }
    hyp.swap(nh);
    if (a.bp_index || a.slot_scores) {
      for (int j = 0; j < K; ++j) {
        size_t o = (static_cast<size_t>(b) * T + t) * K + j;
        if (a.bp_index) a.bp_index[o] = frame_parent[t][j] * W + frame_label[t][j];
        if (a.slot_scores) a.slot_scores[o] = hyp[j].s;
      }
    }
  }
  // LM.Final.
  if (a.lm) {
    for (int k = 0; k < K; ++k) {
      if (hyp[k].s == NEG_INF) continue;
      float l = a.lm->score(hyp[k].y, V);
      float al = a.alpha * l;
      hyp[k].s = hyp[k].s + al;
    }
  }
  // End-of-utterance rollback of pending boosting (variant flag).
  if (a.bt && (a.flags & kFlagBoostRollback)) {
    for (int k = 0; k < K; ++k) {
      if (hyp[k].s == NEG_INF) continue;
      float wb = a.boost_w * static_cast<float>(-a.bt->pot(hyp[k].q));
      hyp[k].s = hyp[k].s + wb;
    }
  }
  int best = 0;
  for (int k = 1; k < K; ++k)
    if (hyp[k].s > hyp[best].s) best = k;
  int32_t* ot = a.out_tokens + static_cast<size_t>(b) * T;
  for (int t = 0; t < T; ++t) ot[t] = -1;
  int32_t* oa = a.out_align ? a.out_align + static_cast<size_t>(b) * T : nullptr;
  if (oa)
    for (int t = 0; t < T; ++t) oa[t] = -1;
  float score = hyp[best].s;
  int n_out = 0;
  if (score != NEG_INF) {
    n_out = static_cast<int>(hyp[best].y.size());
    for (int i = 0; i < n_out; ++i) ot[i] = hyp[best].y[i];
    if (oa) {
      int j = best;
      for (int t = L - 1; t >= 0; --t) {
        oa[t] = frame_label[t][j];
        j = frame_parent[t][j];
      }
    }
  }
  a.out_scores[b] = score;
  if (a.out_lengths) a.out_lengths[b] = n_out;
  if (a.nbest_tokens) {
    std::vector<int> order(K);
    for (int k = 0; k < K; ++k) order[k] = k;
    std::stable_sort(order.begin(), order.end(), [&](int p, int q) { return hyp[p].s > hyp[q].s; });
    for (int r = 0; r < K; ++r) {
      const Hyp& h = hyp[order[r]];
      const bool live = h.s != NEG_INF;
      int32_t* nt = a.nbest_tokens + (static_cast<size_t>(b) * K + r) * T;
      for (int t = 0; t < T; ++t) nt[t] = -1;
      const int n = live ? static_cast<int>(h.y.size()) : 0;
      for (int i = 0; i < n; ++i) nt[i] = h.y[i];
      a.nbest_lengths[static_cast<size_t>(b) * K + r] = n;
      a.nbest_scores[static_cast<size_t>(b) * K + r] = h.s;
    }
  }
  if (a.counters)
    for (int i = 0; i < 8; ++i) a.counters[static_cast<size_t>(b) * 8 + i] = cnt[i];
}

}  // namespace

extern "C" {

// n-gram arrays in the layout of the decoder's LM builder: for order m (1-based)
// counts[m-1] entries, ids [counts[m-1] * m] (0..V-1 tokens, V = </s>, V+1 = <s>),
// log10 probabilities, log10 backoff weights (NULL for the top order).
void* oracle_lm_new(int order, int V, const int64_t* counts, const int32_t* const* ids,
                    const float* const* log10_prob, const float* const* log10_bow) {
  if (order < 1 || V < 1) return nullptr;
  OracleLM* lm = new OracleLM();
  lm->order = order;
  lm->V = V;
  for (int m = 1; m <= order; ++m) {
    for (int64_t e = 0; e < counts[m - 1]; ++e) {
      const int32_t* g = ids[m - 1] + e * m;
      for (int j = 0; j < m; ++j) {
        if (g[j] < 0 || g[j] > V + 1) {
          delete lm;
          return nullptr;
        }
      }
      std::string k = key_of(g, m);
      lm->prob[k] = log10_to_ln(log10_prob[m - 1][e]);
      if (m < order && log10_bow && log10_bow[m - 1]) lm->bow[k] = log10_to_ln(log10_bow[m - 1][e]);
      if (m >= 2) lm->n_cont[key_of(g, m - 1)] += 1;
    }
  }
  return lm;
}

void oracle_lm_free(void* lm) { delete static_cast<OracleLM*>(lm); }

// ln P(c | <s> y) for a collapsed transcript y of n tokens.
float oracle_lm_score(const void* lm, const int32_t* y, int n, int c) {
  const OracleLM* p = static_cast<const OracleLM*>(lm);
  std::vector<int32_t> v(y, y + n);
  return p->score(v, c);
}

// ln P(c | h) for an explicit context h (the full recursion, no truncation).
float oracle_lm_backoff(const void* lm, const int32_t* h, int n, int c) {
  const OracleLM* p = static_cast<const OracleLM*>(lm);
  std::vector<int32_t> v(h, h + n);
  return p->backoff(v, c);
}

void* oracle_bt_new(int V, int n_phrases, const int32_t* offsets, const int32_t* tokens) {
  OracleBT* bt = new OracleBT();
  bt->V = V;
  for (int p = 0; p < n_phrases; ++p) {
    int b = offsets[p], e = offsets[p + 1];
    if (e <= b) continue;  // empty phrases are ignored
    std::vector<int32_t> ph(tokens + b, tokens + e);
    for (int32_t t : ph) {
      if (t < 0 || t >= V) {
        delete bt;
        return nullptr;
      }
    }
    bt->phrases.insert(ph);
    for (size_t l = 1; l <= ph.size(); ++l) bt->nodes.insert(std::vector<int32_t>(ph.begin(), ph.begin() + l));
  }
  for (const auto& n : bt->nodes) {
    if (n.size() >= 2) bt->n_children[key_of(n.data(), n.size() - 1)] += 1;
  }
  return bt;
}

void oracle_bt_free(void* bt) { delete static_cast<OracleBT*>(bt); }

// Total boosting score of reading seq[0..n) from the root; the final state is
// written to state (capacity n) and its length to *state_len.
int oracle_bt_run(const void* bt, const int32_t* seq, int n, int32_t* state, int* state_len) {
  const OracleBT* p = static_cast<const OracleBT*>(bt);
  std::vector<int32_t> q, nx;
  int total = 0;
  for (int i = 0; i < n; ++i) {
    total += p->step(q, seq[i], &nx);
    q = nx;
  }
  if (state) std::copy(q.begin(), q.end(), state);
  if (state_len) *state_len = static_cast<int>(q.size());
  return total;
}

// Score of one step from state q (a node string) on token c.
int oracle_bt_step(const void* bt, const int32_t* q, int nq, int c, int32_t* next, int* next_len) {
  const OracleBT* p = static_cast<const OracleBT*>(bt);
  std::vector<int32_t> s(q, q + nq), nx;
  int sc = p->step(s, c, &nx);
  if (next) std::copy(nx.begin(), nx.end(), next);
  if (next_len) *next_len = static_cast<int>(nx.size());
  return sc;
}

int oracle_bt_pot(const void* bt, const int32_t* q, int nq) {
  const OracleBT* p = static_cast<const OracleBT*>(bt);
  return p->pot(std::vector<int32_t>(q, q + nq));
}

// fp32 log-sum-exp of the recombination variant (for its pins).
float oracle_lse32(float a, float b) { return lse32(a, b); }

// Batched beam search over host arrays (same argument meaning as the device
// decoder; theta = +inf disables pruning).  n_threads > 1 spreads utterances
// over std::threads.  Optional outputs (null to skip): the best path's frame
// labels, per-frame back-pointer indices and slot scores, work counters, and
// the N-best list (tokens [B,K,T], lengths [B,K], scores [B,K]).  flags: bit 0
// log-sum-exp recombination, bit 1 end-of-utterance boosting rollback, bit 2
// LM / boosting scores of repeated emissions.
// Returns 0 on success, 1 on invalid arguments.
int oracle_decode(const float* logprobs, const int32_t* lengths, int B, int T, int V, int K,
                  float alpha, float beta, float boost_w, float theta, int flags, const void* lm,
                  const void* bt, int n_threads, int32_t* out_tokens, int32_t* out_lengths, float* out_scores,
                  int32_t* out_align, int32_t* bp_index, float* slot_scores, int64_t* counters,
                  int32_t* nbest_tokens, int32_t* nbest_lengths, float* nbest_scores) {
  if (B < 0 || T < 0 || V < 1 || K < 1 || !out_tokens || !out_scores) return 1;
  if (nbest_tokens && (!nbest_lengths || !nbest_scores)) return 1;
  if (B > 0 && (!logprobs || !lengths)) return 1;
  const OracleLM* plm = static_cast<const OracleLM*>(lm);
  if (plm && plm->V != V) return 1;
  const OracleBT* pbt = static_cast<const OracleBT*>(bt);
  if (pbt && pbt->V != V) return 1;
  DecodeArgs a{logprobs, lengths, B, T, V, K, alpha, beta, boost_w, theta, flags, plm, pbt,
               out_tokens, out_lengths, out_scores, out_align, bp_index, slot_scores, counters,
               nbest_tokens, nbest_lengths, nbest_scores};
  if (n_threads <= 1 || B <= 1) {
    for (int b = 0; b < B; ++b) decode_one(a, b);
    return 0;
  }
  std::vector<std::thread> pool;
  int nt = std::min(n_threads, B);
  for (int w = 0; w < nt; ++w) {
    pool.emplace_back([&a, w, nt, B]() {
      for (int b = w; b < B; b += nt) decode_one(a, b);
    });
  }
  for (auto& th : pool) th.join();
  return 0;
}

}  // extern "C"
