// Device images of the n-gram tables and the phrase tree, shared by the host
// builders (ngram_tables.cpp, boost_trie.cpp) and the fusion kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "fusion.h"
#include "tables_host.h"

namespace fusion {

// ---------------------------------------------------------------------------
// NgramTables
//
// Level L of a context means its last L tokens: c_1 = the last token, c_m =
// the state itself (m <= N-1).  The LM row of a state sigma is resolved
// bottom-up in the order the backoff recursion fixes:
//   level 1    dense[c_1][y] = p*(c_1 y) if that bigram exists,
//              else uni(y) + bo(c_1)                       (one fp32 add)
//   level L>=2 the arcs of c_L (successors y with p*(c_L y)) override the
//              row; every level above the one an entry came from adds its
//              backoff in increasing L.
// A state record inlines the chain c_2..c_m so that one load resolves it.
// The state reached from one-token context w by token y, when no context of
// two or more tokens has an arc for y, is the bigram (w y) if it exists, else
// the unigram (y); its record is stored again at rec_dense[w * V + y] so a
// kernel reaches it from (w, y) with a single load.
// ---------------------------------------------------------------------------
struct LMDevice {
  const float *dense = nullptr;        // [(V+2) * V]  level-1 row of every one-token context
  const int32_t *rec_dense = nullptr;  // [(V+2) * V * rec_stride]  record of the state after (w, y)
  const int32_t *cnt1 = nullptr;       // [V+2]        explicit bigram successors (</s> included)
  const float *eos1 = nullptr;         // [V+2]        level-1 value of </s>: p*(w </s>), else uni(</s>) + bo(w)
  const int32_t *rec = nullptr;        // [(n_states - (V+2)) * rec_stride] state records
  const int2 *arcs = nullptr;          // (token, logp bits) of the arcs of levels 2..N-1, level by level
  int64_t arc_base[FUSION_MAX_ORDER] = {};  // first arc of level L (arcs of order L+1 n-grams)
  const int32_t *top_next = nullptr;   // [n_N]  state after an order-N arc (index - arc_base[N-1])
  int64_t off[FUSION_MAX_ORDER + 2] = {};   // off[k] = first id of order-k states (k >= 2)
  // context rows (contexts of two or more tokens with many successors):
  const float *ctx_lm = nullptr;       // [n_ctx * V]  lm(y | context), resolved through all its levels
  const int32_t *ctx_rec = nullptr;    // [n_ctx * V * rec_stride]  record of the state after (context, y)
  int64_t n_ctx = 0;
  int64_t n_states = 0;
  int32_t N = 0, V = 0, blank = 0, rec_stride = 0, eos_ok = 0, pad = 0;
};

// (the record layout of a state: record_stride in tables_host.h)

// ---------------------------------------------------------------------------
// BoostTrie
//
// The phrase automaton with its failure links compiled out: the root keeps a
// dense row (target node and entry value E per token); every other node q
// keeps the sorted list of tokens whose transition differs from the root's
// (its own children, then those inherited along its failure chain).
//   delta[i] = (token, target node, E(target) bits, 0)
// boost(y|q) = E(target) - phi(q).
//   node[q]      = (phi(q) bits, first delta entry, delta count, q)
//   root_node[y] = node[root target of y]   (the state after y from the root)
// ---------------------------------------------------------------------------
struct TrieDevice {
  const int4 *node = nullptr;
  const int4 *delta = nullptr;
  const int4 *root_node = nullptr;       // [V]
  const float *root_E = nullptr;         // [V]
  int32_t n_nodes = 0, V = 0, blank = 0, max_depth = 0;
};

}  // namespace fusion

struct NgramTables {
  fusion::LMDevice dev;
  int64_t n[FUSION_MAX_ORDER + 1] = {};
  int64_t device_bytes = 0;
  void *allocs[16] = {};
  int n_allocs = 0;
};

struct BoostTrie {
  fusion::TrieDevice dev;
  int64_t n_delta = 0;
  int64_t device_bytes = 0;
  void *allocs[8] = {};
  int n_allocs = 0;
};

namespace fusion {
// thread-local error text behind fusion_last_error()
int set_error(int code, const std::string &msg);
int hip_error(hipError_t e, const char *what);
// status bits of the end-of-stream kernel, taken and cleared (end_scores.hip)
int end_status_take(int32_t *bits);
}  // namespace fusion
