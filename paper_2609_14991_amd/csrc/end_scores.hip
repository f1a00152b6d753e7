// End-of-stream scoring: the LM terms of Eq. (1) (Sec. III-C) for the
// end-of-sentence token </s>, added to each hypothesis' running score when its
// stream ends, so that hypotheses are compared on complete sentences.
//
// Per hypothesis and LM i, lm_i(</s> | state) follows the same backoff
// recursion as every other token: the highest level L <= m of the state whose
// context c_L has an explicit </s> arc gives p*, level 1 falls back to the
// stored uni(</s>) + bo(c_1), and the backoffs of the levels above the winner
// are added in increasing level order (fp32, one rounding per addition).
// Since </s> has the largest token id, an explicit </s> arc is always the last
// arc of its context's list.  The weighted terms fl(alpha_i * lm_i) are then
// added to the fp64 score in LM order.  One thread per hypothesis: the call is
// made once per utterance and reads a few words per LM level.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>

#include "fusion_internal.h"

namespace fusion {
namespace {

struct EndParams {
  LMDevice lm[FUSION_MAX_LMS];
  float alpha[FUSION_MAX_LMS];
  const int32_t *lm_state;  // [n_lm][H]
  double *hyp_score;        // [H] or NULL
  double *end_term;         // [H] or NULL
  int32_t *status;          // device word: bit set when a state is invalid
  int32_t n_lm, H;
};

__global__ void __launch_bounds__(256) end_kernel(EndParams p) {
  const int h = blockIdx.x * blockDim.x + threadIdx.x;
  if (h >= p.H) return;
  double term = 0.0;
  bool bad = false;
  for (int i = 0; i < p.n_lm; ++i) {
    const LMDevice &lm = p.lm[i];
    const int V = lm.V;
    const int sig = p.lm_state[(int64_t)i * p.H + h];
    // a state must be a context: not blank, not after </s>, within the table
    if (sig < 0 || sig >= lm.n_states || sig == lm.blank || sig == V + 1) {
      bad = true;
      continue;
    }
    float v;
    if (sig < V + 2) {
      v = lm.eos1[sig];  // one-token context (or <s>)
    } else {
      const int32_t *r = lm.rec + (int64_t)(sig - V - 2) * lm.rec_stride;
      const int m = r[0] >> 16;
      v = lm.eos1[r[0] & 0xFFFF];
      int won = 1;
      for (int L = 2; L <= m; ++L) {
        const int beg = r[3 + 3 * (L - 2)], cnt = r[4 + 3 * (L - 2)];
        if (cnt > 0) {
          const int2 a = lm.arcs[beg + cnt - 1];
          if (a.x == V + 1) {
            v = __int_as_float(a.y);
            won = L;
          }
        }
      }
      for (int L = won + 1; L <= m; ++L) v = v + __int_as_float(r[2 + 3 * (L - 2)]);
    }
    const float t = p.alpha[i] * v;
    term = term + (double)t;
    if (p.hyp_score) p.hyp_score[h] = p.hyp_score[h] + (double)t;
  }
  if (p.end_term) p.end_term[h] = term;
  if (bad) atomicOr(p.status, FUSION_STATUS_BAD_LM_STATE);
}

__device__ int32_t g_end_status;

}  // namespace

// the status bits of the end-of-stream kernel, cleared (fusion_device_status
// merges them with the fusion kernels' own)
int end_status_take(int32_t *bits) {
  int32_t v = 0, zero = 0;
  hipError_t e = hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_end_status), sizeof(int32_t), 0, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_error(e, "hipMemcpyFromSymbol");
  e = hipMemcpyToSymbol(HIP_SYMBOL(g_end_status), &zero, sizeof(int32_t), 0, hipMemcpyHostToDevice);
  if (e != hipSuccess) return hip_error(e, "hipMemcpyToSymbol");
  *bits = v;
  return FUSION_OK;
}

}  // namespace fusion

using namespace fusion;

extern "C" int fusion_end_scores(const NgramTables *const *lms, const float *alphas, int32_t n_lm,
                                 const int32_t *lm_state, int32_t H, double *hyp_score, double *end_term,
                                 hipStream_t stream) {
  if (n_lm < 1 || n_lm > FUSION_MAX_LMS) return set_error(FUSION_E_ARG, "n_lm out of range");
  if (!lms || !alphas) return set_error(FUSION_E_ARG, "NULL LM list or weights");
  if (H < 0 || H > (1 << 24)) return set_error(FUSION_E_ARG, "H out of range");
  EndParams p;
  std::memset(&p, 0, sizeof p);
  for (int i = 0; i < n_lm; ++i) {
    if (!lms[i]) return set_error(FUSION_E_ARG, "NULL n-gram tables");
    if (!std::isfinite(alphas[i])) return set_error(FUSION_E_ARG, "non-finite fusion weight");
    if (!lms[i]->dev.eos_ok) return set_error(FUSION_E_UNSUPPORTED, "an LM has no </s> unigram");
    if (i > 0 && lms[i]->dev.V != lms[0]->dev.V) return set_error(FUSION_E_ARG, "LMs of different vocabularies");
    p.lm[i] = lms[i]->dev;
    p.alpha[i] = alphas[i];
  }
  if (H == 0) return FUSION_OK;
  if (!lm_state || (!hyp_score && !end_term)) return set_error(FUSION_E_ARG, "NULL state or output buffer");
  void *st = nullptr;
  hipError_t e = hipGetSymbolAddress(&st, HIP_SYMBOL(g_end_status));
  if (e != hipSuccess) return hip_error(e, "hipGetSymbolAddress");
  p.lm_state = lm_state;
  p.hyp_score = hyp_score;
  p.end_term = end_term;
  p.status = reinterpret_cast<int32_t *>(st);
  p.n_lm = n_lm;
  p.H = H;
  hipLaunchKernelGGL(end_kernel, dim3((H + 255) / 256), dim3(256), 0, stream, p);
  e = hipGetLastError();
  return e == hipSuccess ? FUSION_OK : hip_error(e, "end-of-stream kernel launch");
}
