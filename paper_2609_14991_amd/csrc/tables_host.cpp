// Host-side builders of the n-gram tables and the phrase tree (no GPU calls).
//
// n-gram model (the LM term of Eq. (1), a backoff n-gram over sub-word
// tokens, Sec. III-C): each order is sorted, the closure the backoff
// recursion relies on is checked, the states are numbered canonically (see
// fusion.h) and the model is laid out for the fusion kernels:
//   * dense level-1 rows (one V-wide row per one-token context, already
//     resolved against the unigram row and the context's backoff),
//   * sorted per-order arc arrays for contexts of two or more tokens,
//   * one record per state that inlines its whole backoff chain.
//
// Phrase tree (the boost term of Eq. (1), from a user word list, Sec. III-C).
// Reading used here: a partial match earns token_score per matched token and
// gives it back when the match breaks (potential phi = depth * token_score, 0
// once a phrase is complete), and a completed phrase banks its completion
// bonus; all phrases ending at the current position are credited
// (Aho-Corasick output sets).  Build: trie in BFS order with children by
// ascending token (= the canonical (length, tokens) ids), failure links by
// BFS, output sums along the failure links, then the failure links are
// compiled into per-node transition lists relative to the root's dense row
// so that a kernel resolves any state's full boost row with one node load and
// one list load.
#include "tables_host.h"

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <map>
#include <thread>

namespace fusion {
namespace {

using u128 = unsigned __int128;

int token_bits(int V) {
  int b = 1;
  while ((1 << b) < V + 2) ++b;
  return b;
}

template <class F>
void parallel_for(int64_t n, F &&f) {
  unsigned hw = std::thread::hardware_concurrency();
  int nt = (int)std::min<unsigned>(hw ? hw : 4, 16);
  if (n < (int64_t)1 << 16) nt = 1;
  if (nt <= 1) {
    f((int64_t)0, n);
    return;
  }
  std::vector<std::thread> th;
  for (int i = 0; i < nt; ++i) {
    int64_t a = n * i / nt, b = n * (i + 1) / nt;
    th.emplace_back([&f, a, b] { f(a, b); });
  }
  for (auto &t : th) t.join();
}

struct Order {
  int k = 0;
  int64_t n = 0;
  std::vector<u128> key;     // sorted packed rows
  std::vector<int64_t> src;  // input row of each sorted key (empty: identity)
  int64_t row(int64_t i) const { return src.empty() ? i : src[i]; }
};

}  // namespace

int64_t context_row_min_arcs(int N) {
  const char *env = std::getenv("FUSION_CONTEXT_ROW_MIN_ARCS");
  if (env && *env) {
    char *end = nullptr;
    const long long v = std::strtoll(env, &end, 10);
    if (end && *end == 0 && v >= 0) return (int64_t)v;
  }
  return N > 2 ? 1024 / (N - 2) : INT32_MAX;
}

int build_lm_host(int32_t order, int32_t vocab, int32_t blank_id, const int64_t *count,
                  const int32_t *const *tokens, const float *const *logp, const float *const *backoff,
                  LMHost *out, std::string *why) {
  auto reject = [&](int code, const std::string &msg) {
    *why = msg;
    return code;
  };
  if (order < 2 || order > FUSION_MAX_ORDER)
    return reject(FUSION_E_UNSUPPORTED, "ngram_load: order must be in [2, " + std::to_string(FUSION_MAX_ORDER) + "]");
  if (vocab < 2 || vocab > FUSION_MAX_VOCAB)
    return reject(FUSION_E_UNSUPPORTED, "ngram_load: vocab must be in [2, " + std::to_string(FUSION_MAX_VOCAB) + "]");
  if (blank_id < 0 || blank_id >= vocab) return reject(FUSION_E_ARG, "ngram_load: blank_id out of range");
  if (!count || !tokens || !logp) return reject(FUSION_E_ARG, "ngram_load: NULL table pointer");
  LMHost &d = *out;
  const int N = order, V = vocab, BOS = V, EOS = V + 1;
  const int b = token_bits(V);
  std::vector<Order> ord(N + 1);
  // ---- pack, validate, sort ------------------------------------------------
  for (int k = 1; k <= N; ++k) {
    Order &o = ord[k];
    o.k = k;
    o.n = count[k - 1];
    if (o.n < 0 || o.n > INT32_MAX) return reject(FUSION_E_ARG, "ngram_load: bad count for order " + std::to_string(k));
    if (o.n > 0 && (!tokens[k - 1] || !logp[k - 1]))
      return reject(FUSION_E_ARG, "ngram_load: NULL array for order " + std::to_string(k));
    o.key.resize(o.n);
    const int32_t *tk = tokens[k - 1];
    const float *lp = logp[k - 1];
    const float *bo = (k < N && backoff) ? backoff[k - 1] : nullptr;
    int bad = 0;
    int64_t bad_row = -1;
    for (int64_t i = 0; i < o.n; ++i) {
      u128 key = 0;
      for (int j = 0; j < k; ++j) {
        int32_t t = tk[i * k + j];
        if (t < 0 || t >= V + 2 || t == blank_id) {
          bad = 1;
          bad_row = i;
        }
        key = (key << b) | (u128)(uint32_t)(t & ((1 << b) - 1));
      }
      if (!std::isfinite(lp[i]) || (bo && !std::isfinite(bo[i]))) {
        bad = 2;
        bad_row = i;
      }
      o.key[i] = key;
      if (bad) break;
    }
    if (bad == 1) return reject(FUSION_E_LM_FORMAT, "ngram_load: order " + std::to_string(k) + " row " + std::to_string(bad_row) + ": token out of range or blank");
    if (bad == 2) return reject(FUSION_E_LM_FORMAT, "ngram_load: order " + std::to_string(k) + " row " + std::to_string(bad_row) + ": non-finite value");
    bool sorted = true;
    for (int64_t i = 1; i < o.n && sorted; ++i) sorted = o.key[i - 1] < o.key[i];
    if (!sorted) {
      std::vector<std::pair<u128, int64_t>> kv(o.n);
      for (int64_t i = 0; i < o.n; ++i) kv[i] = {o.key[i], i};
      std::sort(kv.begin(), kv.end());
      o.src.resize(o.n);
      for (int64_t i = 0; i < o.n; ++i) {
        o.key[i] = kv[i].first;
        o.src[i] = kv[i].second;
        if (i > 0 && kv[i - 1].first == kv[i].first)
          return reject(FUSION_E_LM_FORMAT, "ngram_load: duplicate n-gram of order " + std::to_string(k));
      }
    }
  }
  auto tok_of = [&](int k, int64_t i, int j) -> int32_t {  // j-th token of sorted row i
    return (int32_t)((ord[k].key[i] >> (b * (k - 1 - j))) & ((1u << b) - 1));
  };
  auto lp_of = [&](int k, int64_t i) { return logp[k - 1][ord[k].row(i)]; };
  auto bo_of = [&](int k, int64_t i) -> float {
    return (k < N && backoff && backoff[k - 1]) ? backoff[k - 1][ord[k].row(i)] : 0.0f;
  };
  // ---- unigrams ------------------------------------------------------------
  std::vector<float> uni_lp(V + 2, 0.0f), uni_bo(V + 2, 0.0f);
  std::vector<char> present(V + 2, 0);
  for (int64_t i = 0; i < ord[1].n; ++i) {
    int32_t w = tok_of(1, i, 0);
    present[w] = 1;
    uni_lp[w] = lp_of(1, i);
    uni_bo[w] = bo_of(1, i);
  }
  for (int w = 0; w <= BOS; ++w)
    if (w != blank_id && !present[w])
      return reject(FUSION_E_LM_FORMAT, "ngram_load: id " + std::to_string(w) + " has no unigram");
  // ---- prefix closure and arc ranges: ctx k-1 -> [beg, beg+cnt) in order k --
  std::vector<std::vector<int64_t>> arc_beg(N + 1), arc_cnt(N + 1);
  for (int k = 2; k <= N; ++k) {
    const Order &lo = ord[k - 1], &hi = ord[k];
    arc_beg[k - 1].assign(lo.n, 0);
    arc_cnt[k - 1].assign(lo.n, 0);
    int64_t c = 0;
    for (int64_t i = 0; i < hi.n; ++i) {
      u128 pre = hi.key[i] >> b;
      while (c < lo.n && lo.key[c] < pre) ++c;
      if (c >= lo.n || lo.key[c] != pre)
        return reject(FUSION_E_LM_FORMAT, "ngram_load: an order-" + std::to_string(k) + " n-gram lacks its prefix");
      if (arc_cnt[k - 1][c] == 0) arc_beg[k - 1][c] = i;
      ++arc_cnt[k - 1][c];
    }
  }
  // ---- suffix closure: order k row -> index of its (k-1)-token suffix --------
  std::vector<std::vector<int64_t>> sfx(N + 1);
  for (int k = 2; k <= N; ++k) {
    const Order &lo = ord[k - 1], &hi = ord[k];
    sfx[k].assign(hi.n, -1);
    const u128 mask = (((u128)1) << (b * (k - 1))) - 1;
    std::vector<int64_t> &s = sfx[k];
    parallel_for(hi.n, [&](int64_t a, int64_t e) {
      for (int64_t i = a; i < e; ++i) {
        u128 suf = hi.key[i] & mask;
        auto it = std::lower_bound(lo.key.begin(), lo.key.end(), suf);
        if (it != lo.key.end() && *it == suf) s[i] = it - lo.key.begin();
      }
    });
    for (int64_t i = 0; i < hi.n; ++i)
      if (s[i] < 0) return reject(FUSION_E_LM_FORMAT, "ngram_load: an order-" + std::to_string(k) + " n-gram lacks its suffix");
  }
  // ---- state numbering -------------------------------------------------------
  d.N = N;
  d.V = V;
  d.blank = blank_id;
  d.eos_ok = present[EOS];
  d.off[2] = V + 2;
  for (int k = 2; k <= N; ++k) d.off[k + 1] = d.off[k] + ord[k].n;
  d.n_states = d.off[N];
  if (d.n_states > INT32_MAX) return reject(FUSION_E_UNSUPPORTED, "ngram_load: more than 2^31 states");
  for (int k = 1; k <= N; ++k) d.n[k] = ord[k].n;
  d.rec_stride = record_stride(N);
  const int RS = d.rec_stride;
  // ---- dense level-1 rows ----------------------------------------------------
  std::vector<float> &dense = d.dense;
  dense.assign((size_t)(V + 2) * V, 0.0f);
  std::vector<int32_t> dense_next((size_t)(V + 2) * V);  // host only: state after (w, y)
  std::vector<int32_t> &cnt1 = d.cnt1;
  cnt1.assign(V + 2, 0);
  std::vector<int64_t> uni_row(V + 2, -1);
  for (int64_t i = 0; i < ord[1].n; ++i) uni_row[tok_of(1, i, 0)] = i;
  parallel_for(V + 2, [&](int64_t a, int64_t e) {
    for (int64_t w = a; w < e; ++w) {
      float bw = uni_bo[w];
      float *row = dense.data() + w * V;
      int32_t *nrow = dense_next.data() + w * V;
      for (int y = 0; y < V; ++y) {
        row[y] = (y == blank_id) ? 0.0f : uni_lp[y] + bw;
        nrow[y] = y;
      }
      int64_t u = uni_row[w];
      if (u < 0) continue;
      int64_t beg = arc_beg[1][u], n = arc_cnt[1][u];
      cnt1[w] = (int32_t)n;  // every explicit successor, </s> included (the fan-out of the traffic count)
      for (int64_t i = beg; i < beg + n; ++i) {
        int32_t y = tok_of(2, i, 1);
        if (y >= V) continue;
        row[y] = lp_of(2, i);
        nrow[y] = N >= 3 ? (int32_t)(d.off[2] + i) : y;
      }
    }
  });
  // ---- level-1 value of </s> per one-token context (the dense rows hold y < V) ----
  std::vector<float> &eos1 = d.eos1;
  eos1.assign(V + 2, 0.0f);
  if (d.eos_ok) {
    for (int64_t w = 0; w < V + 2; ++w) {
      eos1[w] = uni_lp[EOS] + uni_bo[w];
      const int64_t u = uni_row[w];
      if (u < 0) continue;
      const int64_t beg = arc_beg[1][u], n = arc_cnt[1][u];
      if (n > 0 && tok_of(2, beg + n - 1, 1) == EOS) eos1[w] = lp_of(2, beg + n - 1);  // </s> sorts last
    }
  }
  // ---- arcs of levels 2..N-1 (order L+1 n-grams), one array level by level -----
  int64_t n_arcs = 0;
  for (int L = 2; L <= N - 1; ++L) {
    d.arc_base[L] = n_arcs;
    n_arcs += ord[L + 1].n;
  }
  if (n_arcs > INT32_MAX) return reject(FUSION_E_UNSUPPORTED, "ngram_load: more than 2^31 n-grams of orders 3..N");
  std::vector<I2> &arcs = d.arcs;
  arcs.assign((size_t)n_arcs, I2{0, 0});
  for (int L = 2; L <= N - 1; ++L) {
    const int k = L + 1;
    I2 *A = arcs.data() + d.arc_base[L];
    parallel_for(ord[k].n, [&](int64_t a, int64_t e) {
      for (int64_t i = a; i < e; ++i) {
        float p = lp_of(k, i);
        int32_t bits;
        std::memcpy(&bits, &p, 4);
        A[i] = I2{tok_of(k, i, k - 1), bits};
      }
    });
  }
  // ---- state after an order-N arc --------------------------------------------
  std::vector<int32_t> &top_next = d.top_next;
  top_next.assign(ord[N].n, 0);
  for (int64_t i = 0; i < ord[N].n; ++i)
    top_next[i] = (N - 1 == 1) ? tok_of(N, i, N - 1) : (int32_t)(d.off[N - 1] + sfx[N][i]);
  // ---- contexts that get a context row (more than X successors) -----------
  const int64_t X = context_row_min_arcs(N);
  const int CW = record_ctx_word(N);
  std::vector<std::vector<int32_t>> ctx_of(N);  // [L][i]: row of the order-L context i, or -1
  std::vector<std::pair<int, int64_t>> ctx_list;   // row -> (L, i)
  for (int L = 2; L <= N - 1; ++L) {
    ctx_of[L].assign(ord[L].n, -1);
    for (int64_t i = 0; i < ord[L].n; ++i)
      if (arc_cnt[L][i] > X) {
        ctx_of[L][i] = (int32_t)ctx_list.size();
        ctx_list.push_back({L, i});
      }
  }
  if ((int64_t)ctx_list.size() >= ((int64_t)1 << 28)) return reject(FUSION_E_UNSUPPORTED, "ngram_load: too many context rows");
  d.n_ctx = (int64_t)ctx_list.size();
  // ---- state records (orders 2..N-1) -----------------------------------------
  std::vector<int32_t> &rec = d.rec;
  rec.assign((size_t)(d.n_states - (V + 2)) * RS, 0);
  for (int m = 2; m <= N - 1; ++m) {
    parallel_for(ord[m].n, [&](int64_t a, int64_t e) {
      for (int64_t i = a; i < e; ++i) {
        int32_t *r = rec.data() + (size_t)(d.off[m] - (V + 2) + i) * RS;
        r[0] = tok_of(m, i, m - 1) | (m << 16);
        r[1] = (int32_t)(d.off[m] + i);
        if (m >= 3) {
          const int32_t *sr = rec.data() + (size_t)(d.off[m - 1] - (V + 2) + sfx[m][i]) * RS;
          std::memcpy(r + 2, sr + 2, sizeof(int32_t) * 3 * (m - 2));
        }
        float bo = bo_of(m, i);
        std::memcpy(&r[2 + 3 * (m - 2)], &bo, 4);
        r[2 + 3 * (m - 2) + 1] = (int32_t)(d.arc_base[m] + arc_beg[m][i]);
        r[2 + 3 * (m - 2) + 2] = (int32_t)arc_cnt[m][i];
        // the deepest context row of the chain: this state's own, else its suffix's
        const int32_t cr = ctx_of[m][i];
        if (cr >= 0) r[CW] = (m << 28) | cr;
        else if (m >= 3) r[CW] = rec[(size_t)(d.off[m - 1] - (V + 2) + sfx[m][i]) * RS + CW];
      }
    });
  }
  // ---- context rows: the LM row of each such context and the state after each token --
  // Level by level from the context's last token: row_1 = the dense level-1
  // row; row_j(y) = p*(c_j y) for an arc of c_j, else row_{j-1}(y) + bo(c_j),
  // one fp32 addition (the backoff recursion's order).  The state after y is
  // the arc's state at the longest level with an arc, else the level-1 one.
  d.ctx_lm.assign((size_t)d.n_ctx * V, 0.0f);
  d.ctx_rec.assign((size_t)d.n_ctx * V * RS, 0);
  parallel_for(d.n_ctx, [&](int64_t a, int64_t e) {
    std::vector<float> row(V);
    std::vector<int32_t> nxt(V);
    int64_t idx[FUSION_MAX_ORDER + 1];
    for (int64_t c = a; c < e; ++c) {
      const int L = ctx_list[c].first;
      idx[L] = ctx_list[c].second;
      for (int j = L; j >= 3; --j) idx[j - 1] = sfx[j][idx[j]];
      const int32_t w = tok_of(L, idx[L], L - 1);
      std::memcpy(row.data(), dense.data() + (size_t)w * V, sizeof(float) * V);
      std::memcpy(nxt.data(), dense_next.data() + (size_t)w * V, sizeof(int32_t) * V);
      for (int j = 2; j <= L; ++j) {
        const float bj = bo_of(j, idx[j]);
        for (int y = 0; y < V; ++y) row[y] = row[y] + bj;
        const int64_t beg = arc_beg[j][idx[j]], n = arc_cnt[j][idx[j]];
        for (int64_t u = beg; u < beg + n; ++u) {
          const int32_t y = tok_of(j + 1, u, j);
          if (y >= V) continue;
          row[y] = lp_of(j + 1, u);
          nxt[y] = (j + 1 <= N - 1) ? (int32_t)(d.off[j + 1] + u) : top_next[u];
        }
      }
      std::memcpy(d.ctx_lm.data() + (size_t)c * V, row.data(), sizeof(float) * V);
      for (int y = 0; y < V; ++y) {
        int32_t *r = d.ctx_rec.data() + ((size_t)c * V + y) * RS;
        const int32_t sid = nxt[y];
        if (sid >= V + 2) {
          std::memcpy(r, rec.data() + (size_t)(sid - (V + 2)) * RS, sizeof(int32_t) * RS);
        } else {
          r[0] = sid | (1 << 16);
          r[1] = sid;
        }
      }
    }
  });
  // ---- record of the state after (w, y) for every one-token context w ------
  std::vector<int32_t> &rec_dense = d.rec_dense;
  rec_dense.assign((size_t)(V + 2) * V * RS, 0);
  parallel_for((int64_t)(V + 2) * V, [&](int64_t a, int64_t e) {
    for (int64_t i = a; i < e; ++i) {
      const int32_t sid = dense_next[i];
      int32_t *r = rec_dense.data() + (size_t)i * RS;
      if (sid >= V + 2) {
        std::memcpy(r, rec.data() + (size_t)(sid - (V + 2)) * RS, sizeof(int32_t) * RS);
      } else {
        r[0] = sid | (1 << 16);
        r[1] = sid;
      }
    }
  });
  return FUSION_OK;
}

int build_trie_host(int32_t vocab, int32_t blank_id, int32_t n_phrases, const int32_t *tokens,
                    const int64_t *offsets, const float *completion, float token_score, TrieHost *out,
                    std::string *why) {
  auto reject = [&](int code, const std::string &msg) {
    *why = msg;
    return code;
  };
  if (vocab < 2 || vocab > FUSION_MAX_VOCAB) return reject(FUSION_E_UNSUPPORTED, "boost_build: vocab out of range");
  if (blank_id < 0 || blank_id >= vocab) return reject(FUSION_E_ARG, "boost_build: blank_id out of range");
  if (n_phrases < 0) return reject(FUSION_E_ARG, "boost_build: negative phrase count");
  if (n_phrases > 0 && (!tokens || !offsets)) return reject(FUSION_E_ARG, "boost_build: NULL phrase arrays");
  if (!std::isfinite(token_score)) return reject(FUSION_E_PHRASES, "boost_build: token_score not finite");
  TrieHost &h = *out;
  const int V = vocab;
  // ---- trie of distinct phrases (first occurrence keeps its bonus) ---------
  struct Node {
    std::map<int32_t, int32_t> child;
    int depth = 0;
    int terminal = 0;
    float bonus = 0.0f;
  };
  std::vector<Node> tn(1);
  if (n_phrases > 0 && offsets[0] != 0) return reject(FUSION_E_PHRASES, "boost_build: offsets[0] must be 0");
  for (int32_t i = 0; i < n_phrases; ++i) {
    int64_t a = offsets[i], e = offsets[i + 1];
    if (e - a < 1 || e - a > 255) return reject(FUSION_E_PHRASES, "boost_build: phrase " + std::to_string(i) + " is empty or longer than 255 tokens");
    int32_t u = 0;
    for (int64_t j = a; j < e; ++j) {
      int32_t y = tokens[j];
      if (y < 0 || y >= V || y == blank_id)
        return reject(FUSION_E_PHRASES, "boost_build: phrase " + std::to_string(i) + " has a token out of range or blank");
      auto it = tn[u].child.find(y);
      if (it == tn[u].child.end()) {
        int32_t nid = (int32_t)tn.size();
        int dep = tn[u].depth + 1;
        tn[u].child.emplace(y, nid);
        tn.emplace_back();
        tn.back().depth = dep;
        u = nid;
      } else {
        u = it->second;
      }
    }
    if (!tn[u].terminal) {
      tn[u].terminal = 1;
      tn[u].bonus = completion ? completion[i] : token_score * (float)(e - a);
      if (!std::isfinite(tn[u].bonus)) return reject(FUSION_E_PHRASES, "boost_build: completion bonus not finite");
    }
  }
  // ---- canonical ids: BFS, children by ascending token ----------------------
  const int32_t n = (int32_t)tn.size();
  std::vector<int32_t> order;  // BFS position -> build index
  order.reserve(n);
  order.push_back(0);
  for (size_t h = 0; h < order.size(); ++h)
    for (auto &kv : tn[order[h]].child) order.push_back(kv.second);
  std::vector<int32_t> id(n);
  for (int32_t i = 0; i < n; ++i) id[order[i]] = i;
  // per canonical id: children (token, child id) sorted by token
  std::vector<std::vector<std::pair<int32_t, int32_t>>> kids(n);
  std::vector<int> depth(n), term(n);
  std::vector<float> bonus(n);
  for (int32_t i = 0; i < n; ++i) {
    const Node &nd = tn[order[i]];
    depth[i] = nd.depth;
    term[i] = nd.terminal;
    bonus[i] = nd.bonus;
    for (auto &kv : nd.child) kids[i].push_back({kv.first, id[kv.second]});
  }
  auto child_of = [&](int32_t q, int32_t y) -> int32_t {
    auto &c = kids[q];
    auto it = std::lower_bound(c.begin(), c.end(), std::make_pair(y, INT32_MIN));
    return (it != c.end() && it->first == y) ? it->second : -1;
  };
  // ---- failure links, potentials, output sums (BFS order = id order) -------
  std::vector<int32_t> fail(n, 0);
  std::vector<float> phi(n), outs(n), E(n);
  int max_depth = 0;
  for (int32_t q = 0; q < n; ++q) {
    max_depth = std::max(max_depth, depth[q]);
    for (auto &yc : kids[q]) {
      int32_t y = yc.first, c = yc.second;
      if (q == 0) {
        fail[c] = 0;
        continue;
      }
      int32_t f = fail[q];
      int32_t g = child_of(f, y);
      while (g < 0 && f != 0) {
        f = fail[f];
        g = child_of(f, y);
      }
      fail[c] = g >= 0 ? g : 0;
    }
  }
  for (int32_t q = 0; q < n; ++q) {
    phi[q] = term[q] ? 0.0f : (float)depth[q] * token_score;
    float inherited = q == 0 ? 0.0f : outs[fail[q]];
    outs[q] = term[q] ? bonus[q] + inherited : inherited;
    E[q] = phi[q] + outs[q];
  }
  // ---- transitions that differ from the root's, per node ------------------
  std::vector<std::vector<std::pair<int32_t, int32_t>>> delta(n);
  for (int32_t q = 1; q < n; ++q) {
    const auto &own = kids[q];
    const auto &inh = fail[q] == 0 ? std::vector<std::pair<int32_t, int32_t>>() : delta[fail[q]];
    auto &d = delta[q];
    size_t i = 0, j = 0;
    while (i < own.size() || j < inh.size()) {
      if (j >= inh.size() || (i < own.size() && own[i].first <= inh[j].first)) {
        if (j < inh.size() && inh[j].first == own[i].first) ++j;
        d.push_back(own[i++]);
      } else {
        d.push_back(inh[j++]);
      }
    }
  }
  // ---- device images ---------------------------------------------------------
  std::vector<I4> &node = h.node;
  node.assign(n, I4{0, 0, 0, 0});
  std::vector<I4> &dl = h.delta;
  dl.clear();
  for (int32_t q = 0; q < n; ++q) {
    int32_t pb;
    std::memcpy(&pb, &phi[q], 4);
    node[q] = I4{pb, (int32_t)dl.size(), (int32_t)delta[q].size(), q};
    for (auto &yt : delta[q]) {
      int32_t eb;
      std::memcpy(&eb, &E[yt.second], 4);
      dl.push_back(I4{yt.first, yt.second, eb, 0});
    }
  }
  if (dl.size() > (size_t)INT32_MAX) return reject(FUSION_E_UNSUPPORTED, "boost_build: transition lists too large");
  std::vector<I4> &root_node = h.root_node;
  root_node.assign(V, node[0]);
  std::vector<float> &root_E = h.root_E;
  root_E.assign(V, E[0]);
  for (auto &yc : kids[0]) {
    root_node[yc.first] = node[yc.second];
    root_E[yc.first] = E[yc.second];
  }
  h.n_nodes = n;
  h.V = V;
  h.blank = blank_id;
  h.max_depth = max_depth;
  return FUSION_OK;
}

}  // namespace fusion
