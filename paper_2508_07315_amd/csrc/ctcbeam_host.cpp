// Host side of the ctcbeam C ABI: LM and boosting-tree builders, argument
// checking and the kernel launch.
//
// LM tables (Sec. II "NGPU-LM": a backoff n-gram laid out for batched
// full-vocabulary queries; Sec. IV-A: built from an ARPA file).  Every context
// that is an n-gram entry becomes a state.  A state's arcs are its explicit
// continuations sorted by token, each with the state reached after emitting
// the token (the longest existing suffix of context+token, at most order-1
// words).  A state record stores, for every order of its backoff chain
// (context suffixes of length 1..order-1), the arc range and the backoff
// weight of that suffix, so one gather gives the whole chain.
//
// Boosting tables (Sec. III-B: phrase prefix tree with Aho-Corasick failure
// links, boosting spread over the nodes by depth).  For every tree state the
// continuations of all states on its failure chain (except the root) are
// merged on the host, the deepest owner of a token first, into one list of
// (token, key) pairs; key = (depth(owner)+1) << 26 | (pot(owner)+1) << 20 |
// child.  With the telescoped failure weights pot(f(q)) - pot(q), the score
// of reading token c in state q is (pot(owner)+1) - pot(q) with a continuation
// and -pot(q) without one.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <fstream>
#include <limits>
#include <memory>
#include <new>
#include <sstream>
#include <string>
#include <string_view>
#include <thread>
#include <unordered_map>
#include <vector>

#include "../../include/ctcbeam.h"
#include "ctcbeam_internal.h"

using ctcbeam::BtEntry;
using ctcbeam::BtNode;
using ctcbeam::LmArc;
using ctcbeam::LmLevel;

struct ctcbeam_lm {
  int order = 0, V = 0, nlev = 0;
  int64_t n_states = 0, n_arcs = 0;
  std::vector<LmLevel> states;  // [n_states * nlev]
  std::vector<LmArc> arcs;
  std::vector<float> unigram;   // [V+1]
  LmLevel* d_states = nullptr;
  LmArc* d_arcs = nullptr;
  float* d_unigram = nullptr;
  int device = -1;
};

struct ctcbeam_boost {
  int V = 0;
  std::vector<BtNode> nodes;
  std::vector<BtEntry> list;
  std::vector<uint32_t> root_key;  // [V]
  BtNode* d_nodes = nullptr;
  BtEntry* d_list = nullptr;
  uint32_t* d_root_key = nullptr;
  int device = -1;
};

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

float log10_to_ln(float v) {
  const double LN10 = 2.302585092994045684017991454684364208;
  float f = static_cast<float>(static_cast<double>(v) * LN10);
  if (f == 0.0f) f = 0.0f;  // +0 only
  return f;
}

// Sorted n-gram rows of one order.
// ---- host-side parallelism for the table builders (results do not depend
// on the thread count) ----
int host_threads() {
  const unsigned h = std::thread::hardware_concurrency();
  return static_cast<int>(std::max(1u, std::min(h ? h : 1u, 16u)));
}
// f(begin, end) over contiguous parts of [0, n)
template <class F>
void parallel_for(int64_t n, F&& f, int64_t grain = 65536) {
  const int64_t P = std::min<int64_t>(host_threads(), std::max<int64_t>(1, n / grain));
  if (P <= 1) {
    f(int64_t(0), n);
    return;
  }
  std::vector<std::thread> th;
  for (int64_t t = 0; t < P; ++t) th.emplace_back([&f, n, t, P]() { f(n * t / P, n * (t + 1) / P); });
  for (auto& x : th) x.join();
}
// sort by a total order: parts sorted in parallel, then merged pairwise
template <class T, class Cmp>
void parallel_sort(std::vector<T>& v, Cmp cmp) {
  const int64_t n = static_cast<int64_t>(v.size());
  int64_t P = 1;
  while (P * 2 <= host_threads() && n / (P * 2) >= 65536) P *= 2;
  if (P <= 1) {
    std::sort(v.begin(), v.end(), cmp);
    return;
  }
  std::vector<int64_t> b(P + 1);
  for (int64_t t = 0; t <= P; ++t) b[t] = n * t / P;
  {
    std::vector<std::thread> th;
    for (int64_t t = 0; t < P; ++t) th.emplace_back([&, t]() { std::sort(v.begin() + b[t], v.begin() + b[t + 1], cmp); });
    for (auto& x : th) x.join();
  }
  for (int64_t w = 1; w < P; w *= 2) {
    std::vector<std::thread> th;
    for (int64_t t = 0; t + w < P; t += 2 * w)
      th.emplace_back([&, t, w]() {
        std::inplace_merge(v.begin() + b[t], v.begin() + b[t + w], v.begin() + b[std::min(t + 2 * w, P)], cmp);
      });
    for (auto& x : th) x.join();
  }
}

struct Order {
  int m = 0;
  int64_t n = 0;
  std::vector<int32_t> ids;   // [n*m], rows sorted lexicographically
  std::vector<float> lnp, lnbo;
  std::vector<uint32_t> state;  // state id of each row (contexts), or UINT32_MAX

  const int32_t* row(int64_t i) const { return ids.data() + i * m; }

  // index of the row equal to key[0..m), or -1
  int64_t find(const int32_t* key) const {
    int64_t lo = 0, hi = n;
    while (lo < hi) {
      int64_t mid = (lo + hi) >> 1;
      const int32_t* r = row(mid);
      int cmp = 0;
      for (int j = 0; j < m; ++j) {
        if (r[j] != key[j]) {
          cmp = r[j] < key[j] ? -1 : 1;
          break;
        }
      }
      if (cmp == 0) return mid;
      if (cmp < 0)
        lo = mid + 1;
      else
        hi = mid;
    }
    return -1;
  }
};

int upload(const void* src, size_t bytes, void** dst) {
  size_t n = bytes ? bytes : 16;
  hipError_t e = hipMalloc(dst, n);
  if (e != hipSuccess) {
    *dst = nullptr;
    return e == hipErrorOutOfMemory ? fail(3, "hipMalloc failed: out of device memory")
                                    : fail(4, std::string("hipMalloc: ") + hipGetErrorString(e));
  }
  if (bytes) {
    e = hipMemcpy(*dst, src, bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(4, std::string("hipMemcpy: ") + hipGetErrorString(e));
  }
  return 0;
}

void free_lm_device(ctcbeam_lm* lm) {
  if (lm->d_states) (void)hipFree(lm->d_states);
  if (lm->d_arcs) (void)hipFree(lm->d_arcs);
  if (lm->d_unigram) (void)hipFree(lm->d_unigram);
  lm->d_states = nullptr;
  lm->d_arcs = nullptr;
  lm->d_unigram = nullptr;
}

void free_boost_device(ctcbeam_boost* bt) {
  if (bt->d_nodes) (void)hipFree(bt->d_nodes);
  if (bt->d_list) (void)hipFree(bt->d_list);
  if (bt->d_root_key) (void)hipFree(bt->d_root_key);
  bt->d_nodes = nullptr;
  bt->d_list = nullptr;
  bt->d_root_key = nullptr;
}

int build_lm_tables(int order, int V, const int64_t* counts, const int32_t* const* ngram_ids,
                    const float* const* log10_prob, const float* const* log10_bow,
                    ctcbeam_lm* lm) {
  if (order < 1 || order > CTCBEAM_MAX_ORDER)
    return fail(order < 1 ? 1 : 2, "order must be in 1.." + std::to_string(CTCBEAM_MAX_ORDER));
  if (V < 1) return fail(1, "vocab_size must be >= 1");
  if (V > CTCBEAM_MAX_V) return fail(2, "vocab_size above " + std::to_string(CTCBEAM_MAX_V));
  if (!counts || !ngram_ids || !log10_prob) return fail(1, "null n-gram arrays");
  const int32_t EOS = V, BOS = V + 1;
  std::vector<Order> ord(order + 1);
  for (int m = 1; m <= order; ++m) {
    Order& o = ord[m];
    o.m = m;
    o.n = counts[m - 1];
    if (o.n < 0) return fail(1, "negative n-gram count");
    if (o.n > 0 && (!ngram_ids[m - 1] || !log10_prob[m - 1])) return fail(1, "null array for a non-empty order");
    if (o.n >= (int64_t(1) << 31)) return fail(2, "too many n-grams of one order");
    const int32_t* src = ngram_ids[m - 1];
    std::vector<int64_t> perm(o.n);
    std::atomic<int> bad{0};  // 1 id range, 2 <s> position, 3 </s> position
    parallel_for(o.n, [&](int64_t lo, int64_t hi) {
      for (int64_t i = lo; i < hi; ++i) {
        perm[i] = i;
        const int32_t* r = src + i * m;
        for (int j = 0; j < m; ++j) {
          int e = 0;
          if (r[j] < 0 || r[j] > BOS) e = 1;
          else if (r[j] == BOS && j != 0) e = 2;
          else if (r[j] == EOS && j != m - 1) e = 3;
          if (e) {
            int z = 0;
            bad.compare_exchange_strong(z, e);
          }
        }
      }
    });
    if (bad == 1) return fail(1, "n-gram id out of range");
    if (bad == 2) return fail(1, "<s> may only start an n-gram");
    if (bad == 3) return fail(1, "</s> may only end an n-gram");
    parallel_sort(perm, [src, m](int64_t a, int64_t b) {
      const int32_t* ra = src + a * m;
      const int32_t* rb = src + b * m;
      for (int j = 0; j < m; ++j)
        if (ra[j] != rb[j]) return ra[j] < rb[j];
      return a < b;
    });
    o.ids.resize(static_cast<size_t>(o.n) * m);
    o.lnp.resize(o.n);
    o.lnbo.assign(o.n, 0.0f);
    const float* bo = (m < order && log10_bow) ? log10_bow[m - 1] : nullptr;
    const float* pr = log10_prob[m - 1];
    parallel_for(o.n, [&](int64_t lo, int64_t hi) {
      for (int64_t i = lo; i < hi; ++i) {
        const int64_t s = perm[i];
        std::memcpy(&o.ids[i * m], src + s * m, sizeof(int32_t) * m);
        o.lnp[i] = log10_to_ln(pr[s]);
        if (bo && src[s * m + m - 1] != EOS) o.lnbo[i] = log10_to_ln(bo[s]);
      }
    });
    std::atomic<bool> dup{false};
    parallel_for(o.n, [&](int64_t lo, int64_t hi) {
      for (int64_t i = std::max<int64_t>(lo, 1); i < hi; ++i)
        if (std::memcmp(&o.ids[(i - 1) * m], &o.ids[i * m], sizeof(int32_t) * m) == 0) dup = true;
    });
    if (dup) return fail(1, "duplicate " + std::to_string(m) + "-gram");
  }
  // every token and </s> needs a unigram
  lm->unigram.assign(V + 1, 0.0f);
  for (int32_t c = 0; c <= V; ++c) {
    int64_t r = ord[1].find(&c);
    if (r < 0) return fail(1, "token " + std::to_string(c) + " has no unigram");
    lm->unigram[c] = ord[1].lnp[r];
  }
  // prefix closure
  for (int m = 2; m <= order; ++m) {
    const Order& o = ord[m];
    std::atomic<bool> open{false};
    parallel_for(o.n, [&](int64_t lo, int64_t hi) {
      for (int64_t i = lo; i < hi; ++i) {
        if (i > 0 && std::memcmp(o.row(i - 1), o.row(i), sizeof(int32_t) * (m - 1)) == 0) continue;
        if (ord[m - 1].find(o.row(i)) < 0) open = true;
      }
    });
    if (open) return fail(1, "an " + std::to_string(m) + "-gram's context is not an entry (model not prefix-closed)");
  }
  // states
  const int nlev = order - 1;
  uint32_t next_id = static_cast<uint32_t>(V) + 1;
  for (int m = 1; m <= order; ++m) {
    Order& o = ord[m];
    o.state.assign(o.n, UINT32_MAX);
    if (m == order) continue;
    for (int64_t i = 0; i < o.n; ++i) {
      const int32_t* r = o.row(i);
      if (r[m - 1] == EOS) continue;
      if (m == 1)
        o.state[i] = (r[0] == BOS) ? static_cast<uint32_t>(V) : static_cast<uint32_t>(r[0]);
      else
        o.state[i] = next_id++;
    }
  }
  const int64_t n_states = next_id;
  // arcs: orders 2..order in sorted order; each state's arcs are contiguous
  std::vector<int64_t> arc_off(order + 2, 0);
  for (int m = 2; m <= order; ++m) arc_off[m + 1] = arc_off[m] + ord[m].n;
  const int64_t n_arcs = arc_off[order + 1];
  // state ids stay below 2^31: the kernel tags staged keys with bit 31
  if (n_arcs >= (int64_t(1) << 32) || n_states >= (int64_t(1) << 31))
    return fail(2, "LM too large for the 31-bit state / 32-bit arc indices");
  std::vector<uint32_t> sbeg(n_states, 0), scnt(n_states, 0);
  std::vector<float> sbo(n_states, 0.0f);
  std::vector<uint8_t> sexists(n_states, 0);
  for (int m = 1; m < order; ++m) {
    const Order& o = ord[m];
    for (int64_t i = 0; i < o.n; ++i) {
      if (o.state[i] == UINT32_MAX) continue;
      sbo[o.state[i]] = o.lnbo[i];
      sexists[o.state[i]] = 1;
    }
  }
  lm->arcs.resize(n_arcs);
  for (int m = 2; m <= order; ++m) {
    const Order& o = ord[m];
    const Order& ctx = ord[m - 1];
    // parts start at the first row of a context group, so no group is split
    auto group_start = [&](int64_t i) {
      while (i > 0 && i < o.n && std::memcmp(o.row(i - 1), o.row(i), sizeof(int32_t) * (m - 1)) == 0) ++i;
      return std::min(i, o.n);
    };
    parallel_for(o.n, [&](int64_t lo0, int64_t hi0) {
    const int64_t lo = group_start(lo0), hi = group_start(hi0);
    int64_t i = lo;
    while (i < hi) {
      int64_t j = i + 1;
      while (j < o.n && std::memcmp(o.row(i), o.row(j), sizeof(int32_t) * (m - 1)) == 0) ++j;
      const int64_t ci = ctx.find(o.row(i));
      const uint32_t s = ctx.state[ci];
      sbeg[s] = static_cast<uint32_t>(arc_off[m] + i);
      scnt[s] = static_cast<uint32_t>(j - i);
      for (int64_t r = i; r < j; ++r) {
        const int32_t* g = o.row(r);
        LmArc& a = lm->arcs[arc_off[m] + r];
        a.logp = o.lnp[r];
        a.token = static_cast<uint32_t>(g[m - 1]);
        a.target = UINT32_MAX;
        if (g[m - 1] != EOS) {
          for (int Ls = std::min(order - 1, m); Ls >= 1; --Ls) {
            const int64_t f = ord[Ls].find(g + (m - Ls));
            if (f >= 0 && ord[Ls].state[f] != UINT32_MAX) {
              a.target = ord[Ls].state[f];
              break;
            }
          }
        }
      }
      i = j;
    }
    });
  }
  // chain records
  lm->states.assign(static_cast<size_t>(n_states) * nlev, LmLevel{0, 0, 0.0f});
  std::atomic<uint32_t> max_chain_a{0};
  for (int m = 1; m < order; ++m) {
    const Order& o = ord[m];
    parallel_for(o.n, [&](int64_t lo, int64_t hi) {
    uint32_t part_max = 0;
    for (int64_t i = lo; i < hi; ++i) {
      const uint32_t s = o.state[i];
      if (s == UINT32_MAX) continue;
      const int32_t* h = o.row(i);
      uint32_t chain = 0;
      for (int l = 0; l < nlev && l + 1 <= m; ++l) {
        const int len = l + 1;
        const int64_t f = ord[len].find(h + (m - len));
        if (f < 0 || ord[len].state[f] == UINT32_MAX) continue;
        const uint32_t u = ord[len].state[f];
        LmLevel& rec = lm->states[static_cast<size_t>(s) * nlev + l];
        rec.begin = sbeg[u];
        rec.count = scnt[u] | ctcbeam::kExists;
        rec.bo = sbo[u];
        chain += scnt[u];
      }
      part_max = std::max(part_max, chain);
    }
    uint32_t cur = max_chain_a.load();
    while (part_max > cur && !max_chain_a.compare_exchange_weak(cur, part_max)) {
    }
    });
  }
  const uint32_t max_chain = max_chain_a.load();
  if (max_chain > static_cast<uint32_t>(ctcbeam::kLmStage))
    return fail(2, "a backoff chain holds " + std::to_string(max_chain) +
                       " explicit continuations (limit " + std::to_string(ctcbeam::kLmStage) + ")");
  lm->order = order;
  lm->V = V;
  lm->nlev = nlev;
  lm->n_states = n_states;
  lm->n_arcs = n_arcs;
  return 0;
}

int upload_lm(ctcbeam_lm* lm) {
  int rc;
  if (hipGetDevice(&lm->device) != hipSuccess) return fail(4, "no HIP device");
  if ((rc = upload(lm->states.data(), lm->states.size() * sizeof(LmLevel), reinterpret_cast<void**>(&lm->d_states))))
    return rc;
  if ((rc = upload(lm->arcs.data(), lm->arcs.size() * sizeof(LmArc), reinterpret_cast<void**>(&lm->d_arcs))))
    return rc;
  if ((rc = upload(lm->unigram.data(), lm->unigram.size() * sizeof(float), reinterpret_cast<void**>(&lm->d_unigram))))
    return rc;
  return 0;
}

int build_boost_tables(int V, int n_phrases, const int32_t* offsets, const int32_t* tokens,
                       ctcbeam_boost* bt) {
  if (V < 1) return fail(1, "vocab_size must be >= 1");
  if (V > CTCBEAM_MAX_V) return fail(2, "vocab_size above " + std::to_string(CTCBEAM_MAX_V));
  if (n_phrases < 0) return fail(1, "negative phrase count");
  if (n_phrases > 0 && !offsets) return fail(1, "null offsets");
  struct Node {
    uint32_t parent = 0;
    int32_t token = -1;
    int32_t depth = 0;
    bool phrase = false;
    std::vector<std::pair<int32_t, uint32_t>> kids;
  };
  std::vector<Node> nodes(1);
  std::unordered_map<uint64_t, uint32_t> child;
  auto key = [](uint32_t n, int32_t c) { return (static_cast<uint64_t>(n) << 32) | static_cast<uint32_t>(c); };
  for (int p = 0; p < n_phrases; ++p) {
    const int32_t b = offsets[p], e = offsets[p + 1];
    if (e < b || b < 0) return fail(1, "offsets must be non-decreasing and non-negative");
    if (e > b && !tokens) return fail(1, "null tokens");
    if (e - b > 62) return fail(2, "phrase longer than 62 tokens");
    uint32_t cur = 0;
    for (int32_t i = b; i < e; ++i) {
      const int32_t c = tokens[i];
      if (c < 0 || c >= V) return fail(1, "phrase token out of range");
      auto it = child.find(key(cur, c));
      if (it == child.end()) {
        if (nodes.size() >= (1u << 20) - 1) return fail(2, "more than 2^20-1 boosting tree nodes");
        Node n;
        n.parent = cur;
        n.token = c;
        n.depth = nodes[cur].depth + 1;
        const uint32_t id = static_cast<uint32_t>(nodes.size());
        nodes.push_back(std::move(n));
        nodes[cur].kids.emplace_back(c, id);
        child.emplace(key(cur, c), id);
        cur = id;
      } else {
        cur = it->second;
      }
    }
    if (e > b) nodes[cur].phrase = true;
  }
  const size_t N = nodes.size();
  for (auto& n : nodes) std::sort(n.kids.begin(), n.kids.end());
  // BFS order, banked length, pot, Aho-Corasick failure F, restricted failure f
  std::vector<uint32_t> bfs;
  bfs.reserve(N);
  bfs.push_back(0);
  for (size_t h = 0; h < bfs.size(); ++h)
    for (auto& kc : nodes[bfs[h]].kids) bfs.push_back(kc.second);
  std::vector<int32_t> banked(N, 0), pot(N, 0);
  std::vector<uint32_t> F(N, 0), f(N, 0);
  for (uint32_t u : bfs) {
    if (u == 0) continue;
    const Node& n = nodes[u];
    banked[u] = n.phrase ? n.depth : banked[n.parent];
    pot[u] = n.depth - banked[u];
    if (n.parent == 0) {
      F[u] = 0;
    } else {
      uint32_t x = F[n.parent];
      for (;;) {
        auto it = child.find(key(x, n.token));
        if (it != child.end()) {
          F[u] = it->second;
          break;
        }
        if (x == 0) {
          F[u] = 0;
          break;
        }
        x = F[x];
      }
    }
    uint32_t x = F[u];
    while (x != 0 && nodes[x].depth > pot[u]) x = F[x];
    f[u] = x;
  }
  // merged continuation lists
  bt->nodes.assign(N, BtNode{0, 0, 0, 0});
  bt->list.clear();
  std::vector<uint32_t> seen(V, UINT32_MAX);
  for (uint32_t q = 0; q < N; ++q) {
    const uint32_t begin = static_cast<uint32_t>(bt->list.size());
    uint32_t chain_nodes = 0, chain_arcs = 0;
    for (uint32_t x = q; x != 0; x = f[x]) {
      ++chain_nodes;
      chain_arcs += static_cast<uint32_t>(nodes[x].kids.size());
      for (auto& kc : nodes[x].kids) {
        if (seen[kc.first] == q) continue;
        seen[kc.first] = q;
        const uint32_t k = (static_cast<uint32_t>(nodes[x].depth + 1) << 26) |
                           (static_cast<uint32_t>(pot[x] + 1) << 20) | kc.second;
        bt->list.push_back(BtEntry{static_cast<uint32_t>(kc.first), k});
      }
    }
    // tokens are unique within a merged list, so cnt <= V
    const uint32_t cnt = static_cast<uint32_t>(bt->list.size()) - begin;
    bt->nodes[q] = BtNode{begin, cnt, static_cast<uint32_t>(pot[q]) | (chain_nodes << 8), chain_arcs};
  }
  bt->root_key.assign(V, 0u);
  for (auto& kc : nodes[0].kids) bt->root_key[kc.first] = (1u << 26) | (1u << 20) | kc.second;
  bt->V = V;
  return 0;
}

int upload_boost(ctcbeam_boost* bt) {
  int rc;
  if (hipGetDevice(&bt->device) != hipSuccess) return fail(4, "no HIP device");
  if ((rc = upload(bt->nodes.data(), bt->nodes.size() * sizeof(BtNode), reinterpret_cast<void**>(&bt->d_nodes))))
    return rc;
  if ((rc = upload(bt->list.data(), bt->list.size() * sizeof(BtEntry), reinterpret_cast<void**>(&bt->d_list))))
    return rc;
  if ((rc = upload(bt->root_key.data(), bt->root_key.size() * sizeof(uint32_t),
                   reinterpret_cast<void**>(&bt->d_root_key))))
    return rc;
  return 0;
}

size_t status_bytes(int B) { return (static_cast<size_t>(B) * sizeof(uint32_t) + 255) & ~size_t(255); }

}  // namespace

extern "C" {

const char* ctcbeam_last_error(void) { return g_err.c_str(); }

int ctcbeam_lm_build_host(int order, int vocab_size, const int64_t* counts, const int32_t* const* ngram_ids,
                          const float* const* log10_prob, const float* const* log10_bow, ctcbeam_lm** out) {
  if (!out) return fail(1, "null output handle");
  *out = nullptr;
  std::unique_ptr<ctcbeam_lm> lm;
  try {
    lm.reset(new ctcbeam_lm());
    int rc = build_lm_tables(order, vocab_size, counts, ngram_ids, log10_prob, log10_bow, lm.get());
    if (rc) return rc;
  } catch (const std::bad_alloc&) {
    return fail(3, "host out of memory while building the LM");
  }
  *out = lm.release();
  return 0;
}

int ctcbeam_lm_build(int order, int vocab_size, const int64_t* counts, const int32_t* const* ngram_ids,
                     const float* const* log10_prob, const float* const* log10_bow, ctcbeam_lm** out) {
  int rc = ctcbeam_lm_build_host(order, vocab_size, counts, ngram_ids, log10_prob, log10_bow, out);
  if (rc) return rc;
  rc = upload_lm(*out);
  if (rc) {
    free_lm_device(*out);
    delete *out;
    *out = nullptr;
  }
  return rc;
}

namespace {
int lm_build_arpa(const char* path, int vocab_size, bool device, ctcbeam_lm** out) {
  if (!out) return fail(1, "null output handle");
  *out = nullptr;
  if (!path) return fail(1, "null path");
  if (vocab_size < 1) return fail(1, "vocab_size must be >= 1");
  // the whole file in memory, NUL-terminated
  std::vector<char> buf;
  {
    std::FILE* f = std::fopen(path, "rb");
    if (!f) return fail(1, std::string("cannot open ") + path);
    std::fseek(f, 0, SEEK_END);
    const long sz = std::ftell(f);
    std::fseek(f, 0, SEEK_SET);
    buf.resize(static_cast<size_t>(sz > 0 ? sz : 0) + 1);
    const size_t got = sz > 0 ? std::fread(buf.data(), 1, static_cast<size_t>(sz), f) : 0;
    std::fclose(f);
    buf.resize(got + 1);
    buf[got] = '\0';
  }
  const char* const base = buf.data();
  const char* const fend = base + buf.size() - 1;
  // one line [p, e) without its CR
  auto next_line = [fend](const char* p, const char** e, const char** nxt) {
    const char* q = static_cast<const char*>(std::memchr(p, '\n', static_cast<size_t>(fend - p)));
    const char* le = q ? q : fend;
    *nxt = q ? q + 1 : fend;
    if (le > p && le[-1] == '\r') --le;
    *e = le;
  };
  // pass 1: the data lines of each order, as byte ranges
  std::vector<std::pair<const char*, const char*>> sect;  // by order - 1
  {
    int cur = 0;
    const char* p = base;
    const char* sec_begin = nullptr;
    while (p < fend) {
      const char *e, *nxt;
      next_line(p, &e, &nxt);
      const std::string_view line(p, static_cast<size_t>(e - p));
      if (!line.empty() && line[0] == '\\') {
        if (cur > 0) sect[cur - 1] = {sec_begin, p};
        cur = 0;
        if (line == "\\end\\") break;
        if (line != "\\data\\") {
          const int m = std::atoi(std::string(line.substr(1)).c_str());
          if (m < 1 || m > static_cast<int>(sect.size())) return fail(1, "ARPA section without a header count");
          cur = m;
          sec_begin = nxt;
        }
      } else if (cur == 0 && line.rfind("ngram ", 0) == 0) {
        const int m = std::atoi(std::string(line.substr(6)).c_str());
        if (m < 1 || m > CTCBEAM_MAX_ORDER) return fail(m < 1 ? 1 : 2, "bad ngram order in ARPA header");
        if (static_cast<int>(sect.size()) < m) sect.resize(m, {nullptr, nullptr});
      }
      p = nxt;
    }
    if (cur > 0) sect[cur - 1] = {sec_begin, p};
  }
  auto word_id = [vocab_size](const char* w, size_t n, int32_t* id) {
    if (n == 4 && std::memcmp(w, "</s>", 4) == 0) { *id = vocab_size; return true; }
    if (n == 3 && std::memcmp(w, "<s>", 3) == 0) { *id = vocab_size + 1; return true; }
    if (n == 0 || n > 9) return false;
    int32_t v = 0;
    for (size_t i = 0; i < n; ++i) {
      if (w[i] < '0' || w[i] > '9') return false;
      v = v * 10 + (w[i] - '0');
    }
    if (v >= vocab_size) return false;
    *id = v;
    return true;
  };
  auto is_space = [](char c) { return c == ' ' || c == '\t' || c == '\v' || c == '\f'; };
  // pass 2: each order's lines parsed in parts (split at line starts), then
  // joined in file order
  std::vector<std::vector<int32_t>> ids(sect.size());
  std::vector<std::vector<float>> lp(sect.size()), lb(sect.size());
  for (size_t mi = 0; mi < sect.size(); ++mi) {
    const int cur = static_cast<int>(mi) + 1;
    const char* sb = sect[mi].first;
    const char* se = sect[mi].second;
    if (!sb || se <= sb) continue;
    const int64_t nbytes = se - sb;
    const int P = static_cast<int>(std::min<int64_t>(host_threads(), std::max<int64_t>(1, nbytes / (1 << 20))));
    struct Part {
      std::vector<int32_t> ids;
      std::vector<float> lp, lb;
      const char* bad = nullptr;  // first malformed line
    };
    std::vector<Part> parts(P);
    std::vector<const char*> cut(P + 1);
    cut[0] = sb;
    cut[P] = se;
    for (int t = 1; t < P; ++t) {
      const char* q = sb + nbytes * t / P;
      const char* nl = static_cast<const char*>(std::memchr(q, '\n', static_cast<size_t>(se - q)));
      cut[t] = nl ? nl + 1 : se;
      if (cut[t] < cut[t - 1]) cut[t] = cut[t - 1];
    }
    auto parse = [&](int t) {
      Part& pt = parts[t];
      const char* p = cut[t];
      int32_t g[CTCBEAM_MAX_ORDER];
      const char* tok[CTCBEAM_MAX_ORDER + 2];
      size_t tlen[CTCBEAM_MAX_ORDER + 2];
      while (p < cut[t + 1]) {
        const char *e, *nxt;
        next_line(p, &e, &nxt);
        int nt = 0;
        for (const char* q = p; q < e && nt < cur + 2;) {
          while (q < e && is_space(*q)) ++q;
          if (q >= e) break;
          const char* w = q;
          while (q < e && !is_space(*q)) ++q;
          tok[nt] = w;
          tlen[nt] = static_cast<size_t>(q - w);
          ++nt;
        }
        if (nt == 0) {  // empty line
          p = nxt;
          continue;
        }
        if (nt < cur + 1) {
          if (!pt.bad) pt.bad = p;
          p = nxt;
          continue;
        }
        bool ok = true;
        for (int j = 0; j < cur; ++j) ok = ok && word_id(tok[1 + j], tlen[1 + j], &g[j]);
        if (ok) {  // n-grams with an unknown word are skipped
          pt.ids.insert(pt.ids.end(), g, g + cur);
          pt.lp.push_back(std::strtof(tok[0], nullptr));
          pt.lb.push_back(nt > cur + 1 ? std::strtof(tok[cur + 1], nullptr) : 0.0f);
        }
        p = nxt;
      }
    };
    {
      std::vector<std::thread> th;
      for (int t = 1; t < P; ++t) th.emplace_back(parse, t);
      parse(0);
      for (auto& x : th) x.join();
    }
    for (int t = 0; t < P; ++t) {
      if (parts[t].bad) {
        const char *e, *nxt;
        next_line(parts[t].bad, &e, &nxt);
        return fail(1, "malformed ARPA line: " + std::string(parts[t].bad, static_cast<size_t>(e - parts[t].bad)));
      }
    }
    size_t n = 0;
    for (const Part& pt : parts) n += pt.lp.size();
    ids[mi].reserve(n * cur);
    lp[mi].reserve(n);
    lb[mi].reserve(n);
    for (const Part& pt : parts) {
      ids[mi].insert(ids[mi].end(), pt.ids.begin(), pt.ids.end());
      lp[mi].insert(lp[mi].end(), pt.lp.begin(), pt.lp.end());
      lb[mi].insert(lb[mi].end(), pt.lb.begin(), pt.lb.end());
    }
  }
  const int order = static_cast<int>(ids.size());
  if (order == 0) return fail(1, "no n-grams in ARPA file");
  std::vector<int64_t> counts(order);
  std::vector<const int32_t*> pid(order);
  std::vector<const float*> pp(order), pb(order);
  for (int m = 0; m < order; ++m) {
    counts[m] = static_cast<int64_t>(lp[m].size());
    pid[m] = ids[m].data();
    pp[m] = lp[m].data();
    pb[m] = lb[m].data();
  }
  if (device) return ctcbeam_lm_build(order, vocab_size, counts.data(), pid.data(), pp.data(), pb.data(), out);
  return ctcbeam_lm_build_host(order, vocab_size, counts.data(), pid.data(), pp.data(), pb.data(), out);
}
}  // namespace

int ctcbeam_lm_build_arpa(const char* path, int vocab_size, ctcbeam_lm** out) {
  return lm_build_arpa(path, vocab_size, true, out);
}

int ctcbeam_lm_build_arpa_host(const char* path, int vocab_size, ctcbeam_lm** out) {
  return lm_build_arpa(path, vocab_size, false, out);
}

void ctcbeam_lm_free(ctcbeam_lm* lm) {
  if (!lm) return;
  free_lm_device(lm);
  delete lm;
}

int ctcbeam_boost_build_host(int vocab_size, int n_phrases, const int32_t* offsets, const int32_t* tokens,
                             ctcbeam_boost** out) {
  if (!out) return fail(1, "null output handle");
  *out = nullptr;
  std::unique_ptr<ctcbeam_boost> bt;
  try {
    bt.reset(new ctcbeam_boost());
    int rc = build_boost_tables(vocab_size, n_phrases, offsets, tokens, bt.get());
    if (rc) return rc;
  } catch (const std::bad_alloc&) {
    return fail(3, "host out of memory while building the boosting tree");
  }
  *out = bt.release();
  return 0;
}

int ctcbeam_boost_build(int vocab_size, int n_phrases, const int32_t* offsets, const int32_t* tokens,
                        ctcbeam_boost** out) {
  int rc = ctcbeam_boost_build_host(vocab_size, n_phrases, offsets, tokens, out);
  if (rc) return rc;
  rc = upload_boost(*out);
  if (rc) {
    free_boost_device(*out);
    delete *out;
    *out = nullptr;
  }
  return rc;
}

void ctcbeam_boost_free(ctcbeam_boost* bt) {
  if (!bt) return;
  free_boost_device(bt);
  delete bt;
}

size_t ctcbeam_workspace_bytes(int B, int T, int K) {
  if (B < 0 || T < 0 || K < 0) return 0;
  return ctcbeam::kWsHeaderBytes + status_bytes(B) +
         static_cast<size_t>(B) * static_cast<size_t>(T) * static_cast<size_t>(K) * sizeof(int32_t);
}

static_assert(CTCBEAM_MAX_K == ctcbeam::kMaxK, "beam size limit");
static_assert(CTCBEAM_FLAG_LOGSUMEXP == ctcbeam::kFlagLogSumExp, "flag values");
static_assert(CTCBEAM_FLAG_BOOST_ROLLBACK == ctcbeam::kFlagBoostRollback, "flag values");
static_assert(CTCBEAM_FLAG_NO_ROW_CACHE == ctcbeam::kFlagNoRowCache, "flag values");
static_assert(CTCBEAM_FLAG_REPEAT_SCORE == ctcbeam::kFlagRepeatScore, "flag values");

namespace {

// Shared body of the decode entry points: validation, parameter block and
// launch.  Exactly one output set is given: the 1-best (out_*) or the N-best
// (nbest_*).
int decode_impl(const float* logprobs, const int32_t* lengths, int B, int T, int V, int K, float alpha,
                float beta, float boost_w, const ctcbeam_lm* lm, const ctcbeam_boost* boost, void* workspace,
                size_t workspace_bytes, int32_t* out_tokens, int32_t* out_lengths, float* out_scores,
                int32_t* nbest_tokens, int32_t* nbest_lengths, float* nbest_scores, bool want_nbest,
                bool greedy, hipStream_t stream, const ctcbeam_opts* opts) {
  if (B < 0 || T < 0) return fail(1, "B and T must be >= 0");
  if (V < 1) return fail(1, "V must be >= 1");
  if (V > CTCBEAM_MAX_V) return fail(2, "V above " + std::to_string(CTCBEAM_MAX_V));
  if (K < 1) return fail(1, "K must be >= 1");
  if (K > CTCBEAM_MAX_K) return fail(2, "K above " + std::to_string(CTCBEAM_MAX_K));
  if (!greedy && K > ctcbeam::kMaxKWideV && V > 1024)
    return fail(2, "beams above " + std::to_string(ctcbeam::kMaxKWideV) + " need V <= 1024");
  if (static_cast<int64_t>(T) * (V + 1) >= (int64_t(1) << 40)) return fail(2, "T*(V+1) too large");
  if (lm && lm->V != V) return fail(1, "LM vocabulary size differs from V");
  if (boost && boost->V != V) return fail(1, "boosting tree vocabulary size differs from V");
  if (lm && !lm->d_arcs) return fail(1, "LM handle has no device tables (host-only build)");
  if (boost && !boost->d_nodes) return fail(1, "boosting handle has no device tables (host-only build)");
  const float theta = (opts && !greedy) ? opts->prune_theta : std::numeric_limits<float>::infinity();
  if (std::isnan(theta) || theta < 0.0f) return fail(1, "prune_theta must be >= 0 (or +inf)");
  if (std::isnan(alpha) || std::isnan(beta) || std::isnan(boost_w)) return fail(1, "NaN weight");
  const int flags = opts ? opts->flags : 0;
  if (flags & ~(CTCBEAM_FLAG_LOGSUMEXP | CTCBEAM_FLAG_BOOST_ROLLBACK | CTCBEAM_FLAG_NO_ROW_CACHE |
                CTCBEAM_FLAG_REPEAT_SCORE))
    return fail(1, "unknown flag bits");
  if (B == 0) {
    // nothing to decode; a given workspace records the empty batch
    if (!workspace) return 0;
    if (workspace_bytes < ctcbeam_workspace_bytes(0, 0, 0)) return fail(1, "workspace too small");
    hipError_t e = ctcbeam::launch_ws_header(static_cast<uint32_t*>(workspace), 0, stream);
    if (e != hipSuccess) return fail(4, std::string("kernel launch: ") + hipGetErrorString(e));
    return 0;
  }
  if (!lengths || !workspace || (T > 0 && !logprobs)) return fail(1, "null device pointer");
  if (want_nbest ? (!nbest_lengths || !nbest_scores || (T > 0 && !nbest_tokens))
                 : (!out_scores || (T > 0 && !out_tokens)))
    return fail(1, "null output pointer");
  if (workspace_bytes < ctcbeam_workspace_bytes(B, greedy ? 0 : T, K)) return fail(1, "workspace too small");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(4, "no HIP device");
  if (lm && lm->device != dev) return fail(1, "LM tables live on another device");
  if (boost && boost->device != dev) return fail(1, "boosting tables live on another device");
  ctcbeam::KernelParams p{};
  p.logprobs = logprobs;
  p.lengths = lengths;
  p.B = B;
  p.T = T;
  p.V = V;
  p.K = K;
  p.alpha = alpha;
  p.beta = beta;
  p.boost_w = boost_w;
  p.theta = theta;
  p.flags = greedy ? (flags & ~CTCBEAM_FLAG_LOGSUMEXP) : flags;
  if (lm) {
    p.lm_states = lm->d_states;
    p.lm_arcs = lm->d_arcs;
    p.lm_unigram = lm->d_unigram;
    p.lm_nlev = lm->nlev;
    p.lm_states_below_2p23 = lm->n_states <= (int64_t(1) << 23) ? 1 : 0;
    p.lm_n_states = lm->n_states;
    p.lm_bos_state = static_cast<uint32_t>(V);
  }
  if (boost) {
    p.bt_nodes = boost->d_nodes;
    p.bt_list = boost->d_list;
    p.bt_root_key = boost->d_root_key;
  }
  p.ws_header = static_cast<uint32_t*>(workspace);
  p.status = reinterpret_cast<uint32_t*>(static_cast<char*>(workspace) + ctcbeam::kWsHeaderBytes);
  p.bp = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + ctcbeam::kWsHeaderBytes + status_bytes(B));
  if (want_nbest) {
    p.nbest_tokens = nbest_tokens;  // may be null when T = 0 (empty rows)
    p.nbest_lengths = nbest_lengths;
    p.nbest_scores = nbest_scores;
  } else {
    p.out_tokens = out_tokens;
    p.out_lengths = out_lengths;
    p.out_scores = out_scores;
  }
  p.stats = opts ? opts->stats : nullptr;
  hipError_t e = greedy ? ctcbeam::launch_greedy(p, stream) : ctcbeam::launch_decode(p, stream);
  if (e != hipSuccess) return fail(4, std::string("kernel launch: ") + hipGetErrorString(e));
  return 0;
}

}  // namespace

}  // extern "C"

namespace ctcbeam {
int decode_with_workspace(const float* logprobs, const int32_t* lengths, int B, int T, int V, int K,
                          float alpha, float beta, float boost_w, const ctcbeam_lm* lm,
                          const ctcbeam_boost* boost, void* workspace, size_t workspace_bytes,
                          int32_t* out_tokens, int32_t* out_lengths, float* out_scores,
                          hipStream_t stream, const ctcbeam_opts* opts) {
  return decode_impl(logprobs, lengths, B, T, V, K, alpha, beta, boost_w, lm, boost, workspace, workspace_bytes,
                     out_tokens, out_lengths, out_scores, nullptr, nullptr, nullptr, false, false, stream, opts);
}
int set_last_error(int code, const char* msg) { return fail(code, msg); }
}  // namespace ctcbeam

extern "C" {

int ctcbeam_decode_ex(const float* logprobs, const int32_t* lengths, int B, int T, int V, int K, float alpha,
                      float beta, float boost_w, const ctcbeam_lm* lm, const ctcbeam_boost* boost, void* workspace,
                      size_t workspace_bytes, int32_t* out_tokens, int32_t* out_lengths, float* out_scores,
                      hipStream_t stream, const ctcbeam_opts* opts) {
  return decode_impl(logprobs, lengths, B, T, V, K, alpha, beta, boost_w, lm, boost, workspace, workspace_bytes,
                     out_tokens, out_lengths, out_scores, nullptr, nullptr, nullptr, false, false, stream, opts);
}

int ctcbeam_decode_nbest(const float* logprobs, const int32_t* lengths, int B, int T, int V, int K, float alpha,
                         float beta, float boost_w, const ctcbeam_lm* lm, const ctcbeam_boost* boost,
                         void* workspace, size_t workspace_bytes, int32_t* nbest_tokens, int32_t* nbest_lengths,
                         float* nbest_scores, hipStream_t stream, const ctcbeam_opts* opts) {
  return decode_impl(logprobs, lengths, B, T, V, K, alpha, beta, boost_w, lm, boost, workspace, workspace_bytes,
                     nullptr, nullptr, nullptr, nbest_tokens, nbest_lengths, nbest_scores, true, false, stream, opts);
}

int ctcbeam_greedy_decode(const float* logprobs, const int32_t* lengths, int B, int T, int V, float alpha,
                          float beta, float boost_w, const ctcbeam_lm* lm, const ctcbeam_boost* boost,
                          void* workspace, size_t workspace_bytes, int32_t* out_tokens, int32_t* out_lengths,
                          float* out_scores, hipStream_t stream, const ctcbeam_opts* opts) {
  return decode_impl(logprobs, lengths, B, T, V, 1, alpha, beta, boost_w, lm, boost, workspace, workspace_bytes,
                     out_tokens, out_lengths, out_scores, nullptr, nullptr, nullptr, false, true, stream, opts);
}

int ctcbeam_decode(const float* logprobs, const int32_t* lengths, int B, int T, int V, int K, float alpha,
                   float beta, float boost_w, const ctcbeam_lm* lm, const ctcbeam_boost* boost, void* workspace,
                   size_t workspace_bytes, int32_t* out_tokens, int32_t* out_lengths, float* out_scores,
                   hipStream_t stream) {
  return ctcbeam_decode_ex(logprobs, lengths, B, T, V, K, alpha, beta, boost_w, lm, boost, workspace,
                           workspace_bytes, out_tokens, out_lengths, out_scores, stream, nullptr);
}

int ctcbeam_query_status(const void* workspace, hipStream_t stream, uint32_t* bits) {
  if (!workspace || !bits) return fail(1, "null argument");
  *bits = 0;
  uint32_t hdr[3] = {0u, 0u, 0u};
  hipError_t e = hipMemcpyAsync(hdr, workspace, sizeof(hdr), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return fail(4, std::string("status copy: ") + hipGetErrorString(e));
  if (hdr[0] != ctcbeam::kWsMagic || hdr[2] != ~hdr[1] || hdr[1] > 0x7FFFFFFFu)
    return fail(1, "workspace holds no decode record");
  const int B = static_cast<int>(hdr[1]);
  if (B == 0) return 0;
  std::vector<uint32_t> h(B);
  e = hipMemcpyAsync(h.data(), static_cast<const char*>(workspace) + ctcbeam::kWsHeaderBytes,
                     sizeof(uint32_t) * B, hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return fail(4, std::string("status copy: ") + hipGetErrorString(e));
  for (uint32_t v : h) *bits |= v;
  return 0;
}

int ctcbeam_lm_tables(const ctcbeam_lm* lm, ctcbeam_lm_view* view) {
  if (!lm || !view) return fail(1, "null argument");
  view->order = lm->order;
  view->vocab_size = lm->V;
  view->nlev = lm->nlev;
  view->n_states = lm->n_states;
  view->n_arcs = lm->n_arcs;
  view->states = reinterpret_cast<const uint32_t*>(lm->states.data());
  view->arcs = reinterpret_cast<const uint32_t*>(lm->arcs.data());
  view->unigram = lm->unigram.data();
  return 0;
}

int ctcbeam_boost_tables(const ctcbeam_boost* bt, ctcbeam_boost_view* view) {
  if (!bt || !view) return fail(1, "null argument");
  view->vocab_size = bt->V;
  view->n_nodes = static_cast<int64_t>(bt->nodes.size());
  view->n_list = static_cast<int64_t>(bt->list.size());
  view->nodes = reinterpret_cast<const uint32_t*>(bt->nodes.data());
  view->list = reinterpret_cast<const uint32_t*>(bt->list.data());
  view->root_key = bt->root_key.data();
  return 0;
}

}  // extern "C"
