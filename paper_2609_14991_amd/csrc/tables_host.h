// Host-side construction of the n-gram tables and the phrase tree: the
// validation, canonical numbering and layouts that ngram_load / boost_build
// upload to the device.  Plain C++ with no GPU call, so the builders also
// compile and run in a CPU-only build (the sanitizer test builds them with
// -fsanitize=address,undefined).
#pragma once

#include <climits>
#include <cstdint>
#include <string>
#include <vector>

#include "fusion.h"

namespace fusion {

// layout-compatible with HIP's int2 / int4
struct I2 {
  int32_t x, y;
};
struct I4 {
  int32_t x, y, z, w;
};

// record of a state of order m (int32 words):
//   [0]                     c_1 | (m << 16)
//   [1]                     state id
//   [2 + 3*(L-2) + 0]       bo(c_L) as float bits      (L = 2..m)
//   [2 + 3*(L-2) + 1]       first arc of c_L (index into arcs)
//   [2 + 3*(L-2) + 2]       number of arcs of c_L
//   [record_ctx_word(N)]    deepest level D >= 2 of the chain whose context
//                           has a context row, and that row: D << 28 | row
//                           (0: none)
// (a one-token state w has m = 1 and no level entries)
inline int record_ctx_word(int N) { return 2 + 3 * (N > 2 ? N - 2 : 0); }
inline int record_stride(int N) { return (record_ctx_word(N) + 1 + 3) & ~3; }  // 16-byte records

// A context of L >= 2 tokens gets a context row when it has more than
// context_row_min_arcs(N) explicit successors: then the successors of the
// levels above the deepest such context of any state, at most N-2 levels,
// number at most 1024 in total.  The environment variable
// FUSION_CONTEXT_ROW_MIN_ARCS, read at each load, replaces the threshold
// (tests lower it to give small models context rows).
int64_t context_row_min_arcs(int N);

// The n-gram model laid out for the fusion kernels (see LMDevice for the
// meaning of each array).
struct LMHost {
  int32_t N = 0, V = 0, blank = 0, rec_stride = 0, eos_ok = 0;
  int64_t n_states = 0;
  int64_t off[FUSION_MAX_ORDER + 2] = {};
  int64_t arc_base[FUSION_MAX_ORDER] = {};
  int64_t n[FUSION_MAX_ORDER + 1] = {};
  std::vector<float> dense, eos1;
  std::vector<int32_t> rec_dense, cnt1, rec, top_next;
  std::vector<I2> arcs;
  // context rows: ctx_lm[r * V + y] = lm(y | c) for the r-th context c with a
  // row (the backoff recursion's own fp32 value), ctx_rec[(r * V + y) * RS]
  // the record of the state after (c, y) when no longer context than c has
  // an arc for y
  int64_t n_ctx = 0;
  std::vector<float> ctx_lm;
  std::vector<int32_t> ctx_rec;
};

// ngram_load's arguments (see fusion.h) -> *out; FUSION_OK or an error code
// with the reason in *why
int build_lm_host(int32_t order, int32_t vocab, int32_t blank_id, const int64_t *count,
                  const int32_t *const *tokens, const float *const *logp, const float *const *backoff,
                  LMHost *out, std::string *why);

// The phrase tree with its failure links compiled into per-node transition
// lists (see TrieDevice).
struct TrieHost {
  int32_t n_nodes = 0, V = 0, blank = 0, max_depth = 0;
  std::vector<I4> node, delta, root_node;
  std::vector<float> root_E;
};

// boost_build's arguments (see fusion.h) -> *out; FUSION_OK or an error code
// with the reason in *why
int build_trie_host(int32_t vocab, int32_t blank_id, int32_t n_phrases, const int32_t *tokens,
                    const int64_t *offsets, const float *completion, float token_score, TrieHost *out,
                    std::string *why);

}  // namespace fusion
