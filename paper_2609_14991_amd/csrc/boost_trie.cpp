// boost_build: a user word list -> device-resident phrase-boosting tree.
//
// The boost term of Eq. (1) comes from a phrase-boosting tree over a user
// word list (Sec. III-C).  Reading used here: a partial match earns
// token_score per matched token and gives it back when the match breaks
// (potential phi = depth * token_score, 0 once a phrase is complete), and a
// completed phrase banks its completion bonus; all phrases ending at the
// current position are credited (Aho-Corasick output sets).
//
// Build: trie in BFS order with children by ascending token (= the canonical
// (length, tokens) ids), failure links by BFS, output sums along the failure
// links, then the failure links are compiled into per-node transition
// lists relative to the root's dense row so that a kernel resolves any
// state's full boost row with one node load and one list load.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <vector>

#include "fusion_internal.h"

extern "C" void boost_free(BoostTrie *t) {
  if (!t) return;
  for (int i = 0; i < t->n_allocs; ++i) (void)hipFree(t->allocs[i]);
  delete t;
}

extern "C" int boost_build(int32_t vocab, int32_t blank_id, int32_t n_phrases, const int32_t *tokens,
                           const int64_t *offsets, const float *completion, float token_score,
                           hipStream_t stream, BoostTrie **out) {
  using fusion::set_error;
  if (!out) return set_error(FUSION_E_ARG, "boost_build: out is NULL");
  *out = nullptr;
  if (vocab < 2 || vocab > FUSION_MAX_VOCAB) return set_error(FUSION_E_UNSUPPORTED, "boost_build: vocab out of range");
  if (blank_id < 0 || blank_id >= vocab) return set_error(FUSION_E_ARG, "boost_build: blank_id out of range");
  if (n_phrases < 0) return set_error(FUSION_E_ARG, "boost_build: negative phrase count");
  if (n_phrases > 0 && (!tokens || !offsets)) return set_error(FUSION_E_ARG, "boost_build: NULL phrase arrays");
  if (!std::isfinite(token_score)) return set_error(FUSION_E_PHRASES, "boost_build: token_score not finite");
  const int V = vocab;
  // ---- trie of distinct phrases (first occurrence keeps its bonus) ---------
  struct Node {
    std::map<int32_t, int32_t> child;
    int depth = 0;
    int terminal = 0;
    float bonus = 0.0f;
  };
  std::vector<Node> tn(1);
  if (n_phrases > 0 && offsets[0] != 0) return set_error(FUSION_E_PHRASES, "boost_build: offsets[0] must be 0");
  for (int32_t i = 0; i < n_phrases; ++i) {
    int64_t a = offsets[i], e = offsets[i + 1];
    if (e - a < 1 || e - a > 255) return set_error(FUSION_E_PHRASES, "boost_build: phrase " + std::to_string(i) + " is empty or longer than 255 tokens");
    int32_t u = 0;
    for (int64_t j = a; j < e; ++j) {
      int32_t y = tokens[j];
      if (y < 0 || y >= V || y == blank_id)
        return set_error(FUSION_E_PHRASES, "boost_build: phrase " + std::to_string(i) + " has a token out of range or blank");
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
      if (!std::isfinite(tn[u].bonus)) return set_error(FUSION_E_PHRASES, "boost_build: completion bonus not finite");
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
  std::vector<int4> node(n);
  std::vector<int4> dl;
  for (int32_t q = 0; q < n; ++q) {
    int32_t pb;
    std::memcpy(&pb, &phi[q], 4);
    node[q] = make_int4(pb, (int32_t)dl.size(), (int32_t)delta[q].size(), q);
    for (auto &yt : delta[q]) {
      int32_t eb;
      std::memcpy(&eb, &E[yt.second], 4);
      dl.push_back(make_int4(yt.first, yt.second, eb, 0));
    }
  }
  if (dl.size() > (size_t)INT32_MAX) return set_error(FUSION_E_UNSUPPORTED, "boost_build: transition lists too large");
  std::vector<int4> root_node(V, node[0]);
  std::vector<float> root_E(V, E[0]);
  for (auto &yc : kids[0]) {
    root_node[yc.first] = node[yc.second];
    root_E[yc.first] = E[yc.second];
  }
  auto *t = new BoostTrie();
  t->dev.n_nodes = n;
  t->dev.V = V;
  t->dev.blank = blank_id;
  t->dev.max_depth = max_depth;
  t->n_delta = (int64_t)dl.size();
  auto put = [&](const void *h, size_t bytes, const void **dst) -> int {
    void *p = nullptr;
    size_t nb = std::max<size_t>(bytes, 16);
    hipError_t e = hipMalloc(&p, nb);
    if (e != hipSuccess) return e == hipErrorOutOfMemory ? set_error(FUSION_E_NOMEM, "device allocation failed") : fusion::hip_error(e, "hipMalloc");
    t->allocs[t->n_allocs++] = p;
    t->device_bytes += (int64_t)nb;
    if (bytes) {
      e = hipMemcpyAsync(p, h, bytes, hipMemcpyHostToDevice, stream);
      if (e != hipSuccess) return fusion::hip_error(e, "hipMemcpyAsync");
    }
    *dst = p;
    return FUSION_OK;
  };
  int rc = put(node.data(), node.size() * sizeof(int4), (const void **)&t->dev.node);
  if (rc == FUSION_OK) rc = put(dl.data(), dl.size() * sizeof(int4), (const void **)&t->dev.delta);
  if (rc == FUSION_OK) rc = put(root_node.data(), root_node.size() * sizeof(int4), (const void **)&t->dev.root_node);
  if (rc == FUSION_OK) rc = put(root_E.data(), root_E.size() * 4, (const void **)&t->dev.root_E);
  if (rc == FUSION_OK) {
    hipError_t e = hipStreamSynchronize(stream);
    if (e != hipSuccess) rc = fusion::hip_error(e, "hipStreamSynchronize");
  }
  if (rc != FUSION_OK) {
    (void)hipStreamSynchronize(stream);
    boost_free(t);
    return rc;
  }
  *out = t;
  return FUSION_OK;
}

extern "C" int boost_info(const BoostTrie *t, int32_t *n_nodes, int32_t *max_depth, int64_t *device_bytes) {
  if (!t) return fusion::set_error(FUSION_E_ARG, "boost_info: NULL handle");
  if (n_nodes) *n_nodes = t->dev.n_nodes;
  if (max_depth) *max_depth = t->dev.max_depth;
  if (device_bytes) *device_bytes = t->device_bytes;
  return FUSION_OK;
}
