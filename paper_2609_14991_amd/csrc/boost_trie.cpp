// boost_build: a user word list -> device-resident phrase-boosting tree.
//
// The boost term of Eq. (1) comes from a phrase-boosting tree over a user
// word list (Sec. III-C).  build_trie_host (tables_host.cpp) builds the tree
// and compiles its failure links into per-node transition lists; this file
// uploads them and owns the device memory.
#include <algorithm>
#include <vector>

#include "fusion_internal.h"
#include "tables_host.h"

extern "C" void boost_free(BoostTrie *t) {
  if (!t) return;
  for (int i = 0; i < t->n_allocs; ++i) (void)hipFree(t->allocs[i]);
  delete t;
}

extern "C" int boost_build(int32_t vocab, int32_t blank_id, int32_t n_phrases, const int32_t *tokens,
                           const int64_t *offsets, const float *completion, float token_score,
                           hipStream_t stream, BoostTrie **out) {
  if (!out) return fusion::set_error(FUSION_E_ARG, "boost_build: out is NULL");
  *out = nullptr;
  fusion::TrieHost h;
  std::string why;
  int rc = fusion::build_trie_host(vocab, blank_id, n_phrases, tokens, offsets, completion, token_score, &h, &why);
  if (rc != FUSION_OK) return fusion::set_error(rc, why);
  auto *t = new BoostTrie();
  t->dev.n_nodes = h.n_nodes;
  t->dev.V = h.V;
  t->dev.blank = h.blank;
  t->dev.max_depth = h.max_depth;
  t->n_delta = (int64_t)h.delta.size();
  auto put = [&](const void *src, size_t bytes, const void **dst) -> int {
    void *p = nullptr;
    size_t nb = std::max<size_t>(bytes, 16);
    hipError_t e = hipMalloc(&p, nb);
    if (e != hipSuccess) return e == hipErrorOutOfMemory ? fusion::set_error(FUSION_E_NOMEM, "device allocation failed") : fusion::hip_error(e, "hipMalloc");
    t->allocs[t->n_allocs++] = p;
    t->device_bytes += (int64_t)nb;
    if (bytes) {
      e = hipMemcpyAsync(p, src, bytes, hipMemcpyHostToDevice, stream);
      if (e != hipSuccess) return fusion::hip_error(e, "hipMemcpyAsync");
    }
    *dst = p;
    return FUSION_OK;
  };
  static_assert(sizeof(fusion::I4) == sizeof(int4), "host and device node layouts differ");
  rc = put(h.node.data(), h.node.size() * sizeof(fusion::I4), (const void **)&t->dev.node);
  if (rc == FUSION_OK) rc = put(h.delta.data(), h.delta.size() * sizeof(fusion::I4), (const void **)&t->dev.delta);
  if (rc == FUSION_OK) rc = put(h.root_node.data(), h.root_node.size() * sizeof(fusion::I4), (const void **)&t->dev.root_node);
  if (rc == FUSION_OK) rc = put(h.root_E.data(), h.root_E.size() * 4, (const void **)&t->dev.root_E);
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
