// ngram_load: raw per-order n-gram arrays -> device-resident NgramTables.
//
// The LM term of Eq. (1) is a backoff n-gram over sub-word tokens (Sec. III-C).
// build_lm_host (tables_host.cpp) validates the model, numbers its states and
// lays it out; this file uploads the layout and owns the device memory.
#include <algorithm>
#include <cstring>
#include <vector>

#include "fusion_internal.h"
#include "tables_host.h"

namespace {

struct DeviceUpload {
  NgramTables *t;
  hipStream_t stream;
  // pad: zeroed bytes after the data (the kernels read state records with
  // fixed-size scalar loads that may run past the last record)
  template <class T, class D>
  int put(const std::vector<T> &h, const D **dst, size_t pad = 0) {
    static_assert(sizeof(T) == sizeof(D), "host and device element sizes differ");
    void *p = nullptr;
    const size_t data = h.size() * sizeof(T);
    size_t bytes = std::max<size_t>(data + pad, 16);
    hipError_t e = hipMalloc(&p, bytes);
    if (e != hipSuccess) return e == hipErrorOutOfMemory ? fusion::set_error(FUSION_E_NOMEM, "device allocation failed") : fusion::hip_error(e, "hipMalloc");
    t->allocs[t->n_allocs++] = p;
    t->device_bytes += (int64_t)bytes;
    if (data) {
      e = hipMemcpyAsync(p, h.data(), data, hipMemcpyHostToDevice, stream);
      if (e != hipSuccess) return fusion::hip_error(e, "hipMemcpyAsync");
    }
    if (pad) {
      e = hipMemsetAsync(static_cast<char *>(p) + data, 0, bytes - data, stream);
      if (e != hipSuccess) return fusion::hip_error(e, "hipMemsetAsync");
    }
    *dst = (const D *)p;
    return FUSION_OK;
  }
};

// the kernels read kRecW = 16 words from the start of any record
constexpr size_t kRecordPad = 64;

}  // namespace

extern "C" void ngram_free(NgramTables *lm) {
  if (!lm) return;
  for (int i = 0; i < lm->n_allocs; ++i) (void)hipFree(lm->allocs[i]);
  delete lm;
}

extern "C" int ngram_load(int32_t order, int32_t vocab, int32_t blank_id, const int64_t *count,
                          const int32_t *const *tokens, const float *const *logp,
                          const float *const *backoff, hipStream_t stream, NgramTables **out) {
  if (!out) return fusion::set_error(FUSION_E_ARG, "ngram_load: out is NULL");
  *out = nullptr;
  fusion::LMHost h;
  std::string why;
  int rc = fusion::build_lm_host(order, vocab, blank_id, count, tokens, logp, backoff, &h, &why);
  if (rc != FUSION_OK) return fusion::set_error(rc, why);
  auto *t = new NgramTables();
  fusion::LMDevice &d = t->dev;
  d.N = h.N;
  d.V = h.V;
  d.blank = h.blank;
  d.eos_ok = h.eos_ok;
  d.rec_stride = h.rec_stride;
  d.n_states = h.n_states;
  d.n_ctx = h.n_ctx;
  std::memcpy(d.off, h.off, sizeof d.off);
  std::memcpy(d.arc_base, h.arc_base, sizeof d.arc_base);
  std::memcpy(t->n, h.n, sizeof t->n);
  DeviceUpload up{t, stream};
  if (rc == FUSION_OK) rc = up.put(h.dense, &d.dense);
  if (rc == FUSION_OK) rc = up.put(h.rec_dense, &d.rec_dense, kRecordPad);
  if (rc == FUSION_OK) rc = up.put(h.cnt1, &d.cnt1);
  if (rc == FUSION_OK) rc = up.put(h.eos1, &d.eos1);
  if (rc == FUSION_OK) rc = up.put(h.rec, &d.rec, kRecordPad);
  if (rc == FUSION_OK) rc = up.put(h.arcs, &d.arcs);
  if (rc == FUSION_OK) rc = up.put(h.top_next, &d.top_next);
  if (rc == FUSION_OK) rc = up.put(h.ctx_lm, &d.ctx_lm);
  if (rc == FUSION_OK) rc = up.put(h.ctx_rec, &d.ctx_rec, kRecordPad);
  if (rc == FUSION_OK) {
    hipError_t e = hipStreamSynchronize(stream);
    if (e != hipSuccess) rc = fusion::hip_error(e, "hipStreamSynchronize");
  }
  if (rc != FUSION_OK) {
    (void)hipStreamSynchronize(stream);
    ngram_free(t);
    return rc;
  }
  *out = t;
  return FUSION_OK;
}

extern "C" int ngram_bos_state(const NgramTables *lm, int32_t *state) {
  if (!lm || !state) return fusion::set_error(FUSION_E_ARG, "ngram_bos_state: NULL argument");
  *state = lm->dev.V;
  return FUSION_OK;
}

extern "C" int ngram_info(const NgramTables *lm, int64_t *n_states, int64_t *device_bytes) {
  if (!lm) return fusion::set_error(FUSION_E_ARG, "ngram_info: NULL handle");
  if (n_states) *n_states = lm->dev.n_states;
  if (device_bytes) *device_bytes = lm->device_bytes;
  return FUSION_OK;
}
