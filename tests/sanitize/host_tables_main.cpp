// CPU-only driver of the host table builders (tables_host.cpp), built by
// tests/test_sanitize.py with -fsanitize=address,undefined.  It reads an
// n-gram model and a phrase list in a plain binary form (little-endian; see
// write_case in the test), builds both host layouts and prints their sizes
// and a checksum of every array, or the error code the builders return.
// With a second argument it also writes the state records, the context rows
// and the level-1 next-state records there ("-": not written); with a third,
// the phrase tree's nodes, transition lists, root row and root entry values.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <string>
#include <vector>

#include "tables_host.h"

namespace {

FILE *g_in;

template <class T>
std::vector<T> read_vec(size_t n) {
  std::vector<T> v(n);
  if (n && fread(v.data(), sizeof(T), n, g_in) != n) {
    fprintf(stderr, "short input\n");
    exit(3);
  }
  return v;
}

template <class T>
T read_one() {
  return read_vec<T>(1)[0];
}

// a vector's bytes to f (nothing for an empty one: fwrite takes no null pointer)
template <class T>
void put(FILE *f, const std::vector<T> &v) {
  if (!v.empty()) fwrite(v.data(), sizeof(T), v.size(), f);
}

template <class T>
uint64_t sum_bytes(const std::vector<T> &v) {
  uint64_t h = 1469598103934665603ull;  // FNV-1a over the bytes
  const unsigned char *p = reinterpret_cast<const unsigned char *>(v.data());
  for (size_t i = 0; i < v.size() * sizeof(T); ++i) h = (h ^ p[i]) * 1099511628211ull;
  return h;
}

}  // namespace

int main(int argc, char **argv) {
  if (argc < 2 || argc > 4) return 2;
  g_in = fopen(argv[1], "rb");
  if (!g_in) return 2;
  const int32_t N = read_one<int32_t>(), V = read_one<int32_t>(), blank = read_one<int32_t>();
  std::vector<int64_t> count = read_vec<int64_t>(N);
  std::vector<std::vector<int32_t>> tok(N);
  std::vector<std::vector<float>> lp(N), bo(N);
  std::vector<const int32_t *> tp(N);
  std::vector<const float *> lpp(N), bop(N);
  for (int k = 1; k <= N; ++k) {
    tok[k - 1] = read_vec<int32_t>((size_t)count[k - 1] * k);
    lp[k - 1] = read_vec<float>(count[k - 1]);
    const int32_t has_bo = read_one<int32_t>();
    if (has_bo) bo[k - 1] = read_vec<float>(count[k - 1]);
    tp[k - 1] = tok[k - 1].data();
    lpp[k - 1] = lp[k - 1].data();
    bop[k - 1] = has_bo ? bo[k - 1].data() : nullptr;
  }
  const int32_t n_ph = read_one<int32_t>();
  std::vector<int64_t> offs = read_vec<int64_t>(n_ph + 1);
  std::vector<int32_t> ptok = read_vec<int32_t>(offs[n_ph]);
  const int32_t has_comp = read_one<int32_t>();
  std::vector<float> comp = has_comp ? read_vec<float>(n_ph) : std::vector<float>();
  const float ts = read_one<float>();
  fclose(g_in);

  fusion::LMHost lm;
  std::string why;
  int rc = fusion::build_lm_host(N, V, blank, count.data(), tp.data(), lpp.data(), bop.data(), &lm, &why);
  if (rc != FUSION_OK) {
    printf("lm_error %d %s\n", rc, why.c_str());
  } else {
    printf("lm n_states=%lld rec_stride=%d arcs=%zu dense=%zu rec=%zu rec_dense=%zu top_next=%zu\n",
           (long long)lm.n_states, lm.rec_stride, lm.arcs.size(), lm.dense.size(), lm.rec.size(), lm.rec_dense.size(),
           lm.top_next.size());
    printf("lm_sums %llx %llx %llx %llx %llx %llx %llx\n", (unsigned long long)sum_bytes(lm.dense),
           (unsigned long long)sum_bytes(lm.rec_dense), (unsigned long long)sum_bytes(lm.cnt1),
           (unsigned long long)sum_bytes(lm.eos1), (unsigned long long)sum_bytes(lm.rec),
           (unsigned long long)sum_bytes(lm.arcs), (unsigned long long)sum_bytes(lm.top_next));
    printf("lm_ctx n_ctx=%lld\n", (long long)lm.n_ctx);
    if (argc >= 3 && std::string(argv[2]) != "-") {  // the records and context rows, for the test to check against the oracle
      FILE *f = fopen(argv[2], "wb");
      const int64_t hdr[4] = {lm.rec_stride, lm.n_ctx, (int64_t)lm.rec.size(), (int64_t)lm.rec_dense.size()};
      fwrite(hdr, sizeof hdr, 1, f);
      put(f, lm.rec);
      put(f, lm.ctx_lm);
      put(f, lm.ctx_rec);
      put(f, lm.rec_dense);
      fclose(f);
    }
  }
  fusion::TrieHost tr;
  rc = fusion::build_trie_host(V, blank, n_ph, ptok.data(), offs.data(), has_comp ? comp.data() : nullptr, ts, &tr,
                               &why);
  if (rc != FUSION_OK) {
    printf("trie_error %d %s\n", rc, why.c_str());
  } else {
    printf("trie n_nodes=%d max_depth=%d n_delta=%zu\n", tr.n_nodes, tr.max_depth, tr.delta.size());
    printf("trie_sums %llx %llx %llx %llx\n", (unsigned long long)sum_bytes(tr.node),
           (unsigned long long)sum_bytes(tr.delta), (unsigned long long)sum_bytes(tr.root_node),
           (unsigned long long)sum_bytes(tr.root_E));
    if (argc == 4) {  // the phrase tree, for the test to check against brute force
      FILE *f = fopen(argv[3], "wb");
      const int64_t hdr[4] = {tr.n_nodes, (int64_t)tr.delta.size(), (int64_t)tr.root_node.size(),
                              (int64_t)tr.root_E.size()};
      fwrite(hdr, sizeof hdr, 1, f);
      put(f, tr.node);
      put(f, tr.delta);
      put(f, tr.root_node);
      put(f, tr.root_E);
      fclose(f);
    }
  }
  return 0;
}
