// Fusion step kernels for gfx950 and the C ABI entry points fusion_step /
// fusion_run (Eq. (1) of the paper, Sec. III-C, with greedy or top-k
// selection and a frame-synchronous beam).
//
// Work mapping.  A workgroup owns one stream; each hypothesis of the stream
// is processed by a slot of 4 wavefronts (256 lanes).  Lane g of a slot owns
// the tokens y = (c * 256 + g) * 4 + j (j < 4, c < NC), so every logits /
// dense-row read is a coalesced 16-byte-per-lane strip, and the owned
// values stay in registers for the whole step.  Up to 4 slots run side by
// side (1024 lanes), so a beam of 4 is one workgroup.
//
// Per hypothesis and frame (all steps below are the method's, in order):
//   1  row statistics (online max / sum-exp, raw argmax) from the logits;
//   2  LM context chain from one state record (backoffs and arc ranges of
//      every level), the level-1 dense row of the last token;
//   3  LDS scatter of the explicit arcs of levels 2..m, level by level, each
//      already summed with the backoffs above its level (the addition order
//      of the backoff recursion), and of the phrase transitions of the state;
//   4  key = (x + lambda*lm) + beta*boost per owned token, top-k per lane,
//      top-k per wave by shuffles, top-k of the slot from the 4 wave lists;
//   5  next LM / phrase state of each candidate from the winning entry;
//   6  beam: per stream the best B of B*k candidates by fp64 running score.
// No MFMA: this is a gather/scan with ~10 flops per score, bound by memory.
#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>

#include "fusion_internal.h"

namespace fusion {

static thread_local std::string t_err;

int set_error(int code, const std::string &msg) {
  t_err = msg;
  return code;
}

int hip_error(hipError_t e, const char *what) {
  return set_error(FUSION_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

namespace {

constexpr int kSlotLanes = 256;
constexpr int kWavesPerSlot = 4;
constexpr int kMaxSlots = 4;
constexpr int kMaxWaves = kMaxSlots * kWavesPerSlot;
constexpr int kMaxB = FUSION_MAX_BEAM;
constexpr int kMaxLevels = FUSION_MAX_ORDER;  // levels 2..N-1 < 8

__device__ int g_status;

struct Params {
  LMDevice lm;
  TrieDevice tr;
  const float *logits;
  int32_t *lm_state;
  int32_t *boost_state;
  double *hyp_score;
  int32_t *tokens;
  int32_t *parents;
  float *fused;
  int64_t *traffic;
  float *scores;       // fusion_step outputs [H, k]
  int32_t *next_lm;
  int32_t *next_boost;
  int32_t T, S, B, V, k, blank, mode, has_trie, step_mode, Vp, slots, pad;
  float lam, beta;
};

__device__ __forceinline__ bool before(float ka, int ya, float kb, int yb) {
  return ka > kb || (ka == kb && ya < yb);
}

__device__ __forceinline__ float as_float(int v) { return __int_as_float(v); }

__device__ __forceinline__ unsigned long long umin64(unsigned long long a, unsigned long long b) {
  return a < b ? a : b;
}

template <int KM>
__device__ __forceinline__ void topk_insert(float (&lk)[KM], int (&ly)[KM], float key, int y) {
  if (!before(key, y, lk[KM - 1], ly[KM - 1])) return;
  lk[KM - 1] = key;
  ly[KM - 1] = y;
#pragma unroll
  for (int i = KM - 1; i > 0; --i) {
    if (before(lk[i], ly[i], lk[i - 1], ly[i - 1])) {
      float tk = lk[i];
      lk[i] = lk[i - 1];
      lk[i - 1] = tk;
      int ty = ly[i];
      ly[i] = ly[i - 1];
      ly[i - 1] = ty;
    }
  }
}

template <int NC, int KM, bool AL>
__global__ void __launch_bounds__(NC >= 8 ? 512 : 1024) fusion_kernel(Params p) {
  extern __shared__ __align__(16) unsigned char dyn[];
  __shared__ float s_pm[kMaxWaves], s_ps[kMaxWaves], s_pax[kMaxWaves];
  __shared__ int s_paid[kMaxWaves];
  __shared__ float s_wk[kMaxWaves][KM];
  __shared__ int s_wy[kMaxWaves][KM];
  __shared__ float s_cf[kMaxB][KM];
  __shared__ int s_cy[kMaxB][KM], s_cl[kMaxB][KM], s_cq[kMaxB][KM], s_cn[kMaxB];
  __shared__ int s_lm[kMaxB], s_q[kMaxB], s_c1[kMaxB];
  __shared__ double s_sc[kMaxB];
  __shared__ int n_lm[kMaxB], n_q[kMaxB], n_c1[kMaxB];
  __shared__ double n_sc[kMaxB];
  __shared__ unsigned long long s_bytes, s_steps;
  __shared__ const int2 *s_arcs[kMaxLevels];  // arcs of level L
  __shared__ long long s_sbase[kMaxLevels];   // state id of the first arc of level L (< 0: top level)

  const LMDevice &lm = p.lm;
  const TrieDevice &tr = p.tr;
  const int tid = threadIdx.x;
  const int slot = tid >> 8;
  const int g = tid & (kSlotLanes - 1);
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int wslot = (tid >> 6) & (kWavesPerSlot - 1);
  const int B = p.B, V = p.V, blank = p.blank, K = p.k;
  const int s = blockIdx.x;
  const int H = p.S * B;
  const int N = lm.N;
  float *lmval = reinterpret_cast<float *>(dyn) + (size_t)slot * p.Vp;
  uint32_t *win = reinterpret_cast<uint32_t *>(reinterpret_cast<float *>(dyn) + (size_t)p.slots * p.Vp) +
                  (size_t)slot * p.Vp;
  uint16_t *win16 = reinterpret_cast<uint16_t *>(win);
  float *rootE = reinterpret_cast<float *>(dyn) + (size_t)2 * p.slots * p.Vp;  // shared by the slots

  // ---- initial states --------------------------------------------------------
  if (tid < B) {
    const int h = s * B + tid;
    int sig = p.lm_state[h];
    s_lm[tid] = sig;
    s_q[tid] = p.has_trie ? p.boost_state[h] : 0;
    s_sc[tid] = (B > 1) ? p.hyp_score[h] : 0.0;
    int c1 = -1;
    if (sig >= 0 && sig < lm.n_states) c1 = sig < V + 2 ? sig : (lm.rec[(int64_t)(sig - V - 2) * lm.rec_stride] & 0xFFFF);
    s_c1[tid] = c1;
  }
  if (tid == 0) {
    s_bytes = 0;
    s_steps = 0;
  }
  if (tid < kMaxLevels) {
    s_arcs[tid] = lm.arcs[tid];
    s_sbase[tid] = (tid >= 2 && tid + 1 <= N - 1) ? lm.off[tid + 1] : -1;
  }
  // phrase entry values of the root row (state independent), one copy per workgroup
  for (int y = tid; y < p.Vp; y += blockDim.x) rootE[y] = (p.has_trie && y < V) ? tr.root_E[y] : 0.0f;
  __syncthreads();

  for (int t = 0; t < p.T; ++t) {
    for (int b0 = 0; b0 < B; b0 += p.slots) {
      const int b = b0 + slot;
      const bool act = b < B && (B == 1 || s_sc[b] > -INFINITY);
      const int sig = act ? __builtin_amdgcn_readfirstlane(s_lm[b]) : 0;
      const int q = act ? __builtin_amdgcn_readfirstlane(s_q[b]) : 0;
      const int c1 = act ? __builtin_amdgcn_readfirstlane(s_c1[b]) : 0;
      const bool ok_lm = act && sig >= 0 && sig < lm.n_states && sig != blank && (sig != V + 1 || lm.eos_ok) && c1 >= 0;
      const bool ok_q = !p.has_trie || (q >= 0 && q < tr.n_nodes);
      const bool ok = ok_lm && ok_q;
      // ---- state record: backoff chain of the context ---------------------
      int m = 1;
      float bo[kMaxLevels];
      int beg[kMaxLevels], cnt[kMaxLevels];
#pragma unroll
      for (int L = 0; L < kMaxLevels; ++L) {
        bo[L] = 0.0f;
        beg[L] = 0;
        cnt[L] = 0;
      }
      if (ok && sig >= V + 2) {
        const int32_t *r = lm.rec + (int64_t)(sig - V - 2) * lm.rec_stride;
        m = __builtin_amdgcn_readfirstlane(r[0] >> 16);
#pragma unroll
        for (int L = 2; L < kMaxLevels; ++L)
          if (L <= m) {
            bo[L] = as_float(__builtin_amdgcn_readfirstlane(r[1 + 3 * (L - 2)]));
            beg[L] = __builtin_amdgcn_readfirstlane(r[2 + 3 * (L - 2)]);
            cnt[L] = __builtin_amdgcn_readfirstlane(r[3 + 3 * (L - 2)]);
          }
      }
      float phiq = 0.0f;
      int dbeg = 0, dcnt = 0;
      if (ok && p.has_trie) {
        int4 nd = tr.node[q];
        phiq = as_float(__builtin_amdgcn_readfirstlane(nd.x));
        dbeg = __builtin_amdgcn_readfirstlane(nd.y);
        dcnt = __builtin_amdgcn_readfirstlane(nd.z);
      }
      // ---- logits row and level-1 dense row --------------------------------
      const int64_t rowoff = ((int64_t)t * H + (int64_t)s * B + b) * V;
      const float *xrow = p.logits + rowoff;
      const float *drow = lm.dense + (int64_t)(c1 < 0 ? 0 : c1) * V;
      float xv[NC][4], dv[NC][4];
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int y0 = (c * kSlotLanes + g) * 4;
        if (AL) {
          float4 xx = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
          float4 dd = make_float4(0.f, 0.f, 0.f, 0.f);
          if (act && y0 < V) xx = *reinterpret_cast<const float4 *>(xrow + y0);
          if (ok && y0 < V) dd = *reinterpret_cast<const float4 *>(drow + y0);
          xv[c][0] = xx.x; xv[c][1] = xx.y; xv[c][2] = xx.z; xv[c][3] = xx.w;
          dv[c][0] = dd.x; dv[c][1] = dd.y; dv[c][2] = dd.z; dv[c][3] = dd.w;
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            xv[c][j] = (act && y0 + j < V) ? xrow[y0 + j] : -INFINITY;
            dv[c][j] = (ok && y0 + j < V) ? drow[y0 + j] : 0.0f;
          }
        }
        *reinterpret_cast<uint4 *>(win + y0) = make_uint4(0u, 0u, 0u, 0u);
      }
      // ---- row statistics: online max / sum-exp and raw argmax --------------
      float lmx = -INFINITY;
      float ax = -INFINITY;
      int aid = INT_MAX;
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int y = (c * kSlotLanes + g) * 4 + j;
          const float x = xv[c][j];
          if (y < V) {
            lmx = fmaxf(lmx, x);
            if (x > ax) {
              ax = x;
              aid = y;
            }
          }
        }
      float lsum = 0.0f;
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int y = (c * kSlotLanes + g) * 4 + j;
          if (y < V && lmx > -INFINITY) lsum += expf(xv[c][j] - lmx);
        }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        float om = __shfl_xor(lmx, off);
        float os = __shfl_xor(lsum, off);
        float oax = __shfl_xor(ax, off);
        int oaid = __shfl_xor(aid, off);
        float nm = fmaxf(lmx, om);
        float a = (lmx > -INFINITY) ? lsum * expf(lmx - nm) : 0.0f;
        float bb = (om > -INFINITY) ? os * expf(om - nm) : 0.0f;
        lmx = nm;
        lsum = a + bb;
        if (oax > ax || (oax == ax && oaid < aid)) {
          ax = oax;
          aid = oaid;
        }
      }
      if (lane == 0) {
        s_pm[wave] = lmx;
        s_ps[wave] = lsum;
        s_pax[wave] = ax;
        s_paid[wave] = aid;
      }
      __syncthreads();
      // ---- scatter: phrase transitions, then LM arcs level by level ---------
      if (ok && p.has_trie) {
        for (int j = g; j < dcnt; j += kSlotLanes) {
          const int y = tr.delta[dbeg + j].x;
          win16[2 * y + 1] = (uint16_t)(j + 1);
        }
      }
      const int nphase = N - 2 > 1 ? N - 2 : 1;
      for (int ph = 0; ph < nphase; ++ph) {
        const int L = ph + 2;
        if (ok && L <= m) {
          int bL = 0, cL = 0;
#pragma unroll
          for (int L2 = 2; L2 < kMaxLevels; ++L2)
            if (L2 == L) {
              bL = beg[L2];
              cL = cnt[L2];
            }
          const int2 *A = s_arcs[L] + bL;
          for (int j = g; j < cL; j += kSlotLanes) {
            const int2 a = A[j];
            const int y = a.x;
            if (y < V) {
              float v = as_float(a.y);
#pragma unroll
              for (int L2 = 3; L2 < kMaxLevels; ++L2)
                if (L2 > L && L2 <= m) v = v + bo[L2];
              lmval[y] = v;
              win16[2 * y] = (uint16_t)((L << 13) | j);
            }
          }
        }
        __syncthreads();
      }
      // ---- keys, fused row, per-lane top-k ------------------------------------
      float M = -INFINITY;
      float amx = -INFINITY;
      int am = INT_MAX;
#pragma unroll
      for (int w = 0; w < kWavesPerSlot; ++w) M = fmaxf(M, s_pm[slot * kWavesPerSlot + w]);
      float Ssum = 0.0f;
#pragma unroll
      for (int w = 0; w < kWavesPerSlot; ++w) {
        const int i = slot * kWavesPerSlot + w;
        if (s_pm[i] > -INFINITY) Ssum += s_ps[i] * expf(s_pm[i] - M);
        if (s_pax[i] > amx || (s_pax[i] == amx && s_paid[i] < am)) {
          amx = s_pax[i];
          am = s_paid[i];
        }
      }
      const float lse = M + logf(Ssum);
      const bool blank_by_am = (p.mode == FUSION_BLANK_AM) && am == blank;
      float lk[KM];
      int ly[KM];
#pragma unroll
      for (int i = 0; i < KM; ++i) {
        lk[i] = -INFINITY;
        ly[i] = INT_MAX;
      }
      if (ok && (!blank_by_am || p.fused)) {
        float *frow = p.fused ? p.fused + rowoff : nullptr;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          const int y0 = (c * kSlotLanes + g) * 4;
          const uint4 w4 = *reinterpret_cast<const uint4 *>(win + y0);
          const uint32_t ww[4] = {w4.x, w4.y, w4.z, w4.w};
          float kk[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int y = y0 + j;
            const float x = xv[c][j];
            float key = x;
            if (y != blank) {
              const uint32_t lo = ww[j] & 0xFFFFu, hi = ww[j] >> 16;
              float lmv;
              if (lo) {
                lmv = lmval[y];
              } else {
                lmv = dv[c][j];
#pragma unroll
                for (int L2 = 2; L2 < kMaxLevels; ++L2)
                  if (L2 <= m) lmv = lmv + bo[L2];
              }
              float bst = 0.0f;
              if (p.has_trie) {
                const float e = hi ? as_float(tr.delta[dbeg + (int)hi - 1].z) : rootE[y];
                bst = e - phiq;
              }
              const float a1 = p.lam * lmv;
              const float a2 = x + a1;
              const float a3 = p.beta * bst;
              key = a2 + a3;
            }
            kk[j] = key;
            if (y < V && (p.mode == FUSION_BLANK_COMPETE || y != blank)) topk_insert<KM>(lk, ly, key, y);
          }
          if (frow) {
            if (AL) {
              if (y0 < V) *reinterpret_cast<float4 *>(frow + y0) = make_float4(kk[0] - lse, kk[1] - lse, kk[2] - lse, kk[3] - lse);
            } else {
#pragma unroll
              for (int j = 0; j < 4; ++j)
                if (y0 + j < V) frow[y0 + j] = kk[j] - lse;
            }
          }
        }
      }
      // ---- wave top-k by shuffles ---------------------------------------------
      for (int j = 0; j < K; ++j) {
        float bk = lk[0];
        int by = ly[0];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
          const float ok2 = __shfl_xor(bk, off);
          const int oy = __shfl_xor(by, off);
          if (before(ok2, oy, bk, by)) {
            bk = ok2;
            by = oy;
          }
        }
        if (by != INT_MAX && ly[0] == by) {
#pragma unroll
          for (int i = 0; i < KM - 1; ++i) {
            lk[i] = lk[i + 1];
            ly[i] = ly[i + 1];
          }
          lk[KM - 1] = -INFINITY;
          ly[KM - 1] = INT_MAX;
        }
        if (lane == 0) {
          s_wk[wave][j] = bk;
          s_wy[wave][j] = by;
        }
      }
      __syncthreads();
      // ---- slot top-k from the 4 wave lists, next states ------------------------
      if (act && wslot == 0) {
        if (!ok || blank_by_am) {
          if (lane == 0) {
            const float xb = xrow[blank];
            s_cy[b][0] = blank;
            s_cf[b][0] = xb - lse;
            s_cl[b][0] = sig;
            s_cq[b][0] = q;
            s_cn[b] = 1;
            if (!ok) atomicOr(&g_status, (ok_lm ? 0 : FUSION_STATUS_BAD_LM_STATE) | (ok_q ? 0 : FUSION_STATUS_BAD_BOOST_STATE));
          }
        } else {
          const int ne = kWavesPerSlot * K;
          float ek = -INFINITY;
          int ey = INT_MAX;
          if (lane < ne) {
            ek = s_wk[slot * kWavesPerSlot + lane / K][lane % K];
            ey = s_wy[slot * kWavesPerSlot + lane / K][lane % K];
          }
          int rank = 0, nvalid = 0;
          for (int i = 0; i < ne; ++i) {
            const float ok2 = s_wk[slot * kWavesPerSlot + i / K][i % K];
            const int oy = s_wy[slot * kWavesPerSlot + i / K][i % K];
            if (oy != INT_MAX) {
              ++nvalid;
              if (before(ok2, oy, ek, ey)) ++rank;
            }
          }
          if (lane < ne && ey != INT_MAX && rank < K) {
            const int y = ey;
            int nl = sig, nq = q;
            if (y != blank) {
              const uint32_t w = win[y];
              const uint32_t lo = w & 0xFFFFu, hi = w >> 16;
              if (lo) {
                const int L = (int)(lo >> 13), j = (int)(lo & 0x1FFFu);
                int bL = 0;
#pragma unroll
                for (int L2 = 2; L2 < kMaxLevels; ++L2)
                  if (L2 == L) bL = beg[L2];
                const int64_t a = (int64_t)bL + j;
                const long long sb = s_sbase[L];
                nl = sb >= 0 ? (int)(sb + a) : lm.top_next[a];
              } else {
                nl = lm.dense_next[(int64_t)c1 * V + y];
              }
              nq = p.has_trie ? (hi ? tr.delta[dbeg + (int)hi - 1].y : tr.root_target[y]) : 0;
            }
            s_cy[b][rank] = y;
            s_cf[b][rank] = ek - lse;
            s_cl[b][rank] = nl;
            s_cq[b][rank] = nq;
          }
          if (lane == 0) s_cn[b] = nvalid < K ? nvalid : K;
        }
        if (p.traffic && lane == 0) {
          unsigned long long by = 4ull * V;  // logits row
          if (ok) {
            const unsigned long long dense_row = 4ull * V;
            by += umin64(8ull * (unsigned long long)lm.cnt1[c1], dense_row);
#pragma unroll
            for (int L2 = 2; L2 < kMaxLevels; ++L2)
              if (L2 <= m) by += umin64(8ull * (unsigned long long)cnt[L2], dense_row) + 12ull;
            if (m >= 2) by += 4ull;
            if (p.has_trie) by += 16ull + 16ull * (unsigned long long)dcnt;
          }
          by += (B > 1) ? 8ull : 4ull;
          if (p.fused) by += 4ull * V;
          atomicAdd(&s_bytes, by);
          atomicAdd(&s_steps, 1ull);
        }
      } else if (wslot == 0 && lane == 0 && b < B) {
        s_cn[b] = 0;
      }
      __syncthreads();
    }
    // ---- selection across the stream ---------------------------------------------
    if (p.step_mode) {
      // fusion_step: B == 1, every candidate of the hypothesis is an output
      if (tid < K) {
        const int h = s;
        const int n = s_cn[0];
        const int64_t o = (int64_t)h * K + tid;
        p.tokens[o] = tid < n ? s_cy[0][tid] : -1;
        p.scores[o] = tid < n ? s_cf[0][tid] : -INFINITY;
        p.next_lm[o] = tid < n ? s_cl[0][tid] : s_lm[0];
        p.next_boost[o] = tid < n ? s_cq[0][tid] : s_q[0];
      }
    } else if (B == 1) {
      if (tid == 0) {
        const int y = s_cy[0][0];
        p.tokens[(int64_t)t * H + s] = y;
        n_lm[0] = s_cl[0][0];
        n_q[0] = s_cq[0][0];
        n_c1[0] = y != blank ? y : s_c1[0];
        n_sc[0] = 0.0;
      }
    } else if (wave == 0) {
      // beam: rank the live candidates by (score desc, parent asc, rank asc)
      const int ncand = B * K;
      int live = 0;
      for (int i0 = 0; i0 < ncand; i0 += 64) {
        const int i = i0 + lane;
        bool valid = false;
        double sc = -INFINITY;
        int bi = 0, ji = 0;
        if (i < ncand) {
          bi = i / K;
          ji = i % K;
          valid = ji < s_cn[bi];
          if (valid) sc = s_sc[bi] + (double)s_cf[bi][ji];
        }
        int rank = 0;
        if (valid) {
          for (int i2 = 0; i2 < ncand; ++i2) {
            const int b2 = i2 / K, j2 = i2 % K;
            if (j2 >= s_cn[b2]) continue;
            const double sc2 = s_sc[b2] + (double)s_cf[b2][j2];
            if (sc2 > sc || (sc2 == sc && (b2 < bi || (b2 == bi && j2 < ji)))) ++rank;
          }
          if (rank < B) {
            const int y = s_cy[bi][ji];
            n_lm[rank] = s_cl[bi][ji];
            n_q[rank] = s_cq[bi][ji];
            n_c1[rank] = y != blank ? y : s_c1[bi];
            n_sc[rank] = sc;
            const int64_t o = (int64_t)t * H + (int64_t)s * B + rank;
            p.tokens[o] = y;
            p.parents[o] = bi;
          }
        }
        live += __popcll(__ballot(valid));
      }
      for (int i = live + lane; i < B; i += 64) {
        n_lm[i] = s_lm[i];
        n_q[i] = s_q[i];
        n_c1[i] = s_c1[i];
        n_sc[i] = -INFINITY;
        const int64_t o = (int64_t)t * H + (int64_t)s * B + i;
        p.tokens[o] = -1;
        p.parents[o] = -1;
      }
    }
    __syncthreads();
    if (!p.step_mode && tid < B) {
      s_lm[tid] = n_lm[tid];
      s_q[tid] = n_q[tid];
      s_c1[tid] = n_c1[tid];
      s_sc[tid] = n_sc[tid];
    }
    __syncthreads();
  }
  // ---- final states ------------------------------------------------------------------
  if (!p.step_mode && tid < B) {
    const int h = s * B + tid;
    p.lm_state[h] = s_lm[tid];
    if (p.has_trie) p.boost_state[h] = s_q[tid];
    if (B > 1) p.hyp_score[h] = s_sc[tid];
  }
  if (p.traffic && tid == 0) {
    unsigned long long extra = (s == 0 && p.has_trie) ? 4ull * V * (unsigned long long)p.T : 0ull;
    atomicAdd(reinterpret_cast<unsigned long long *>(p.traffic), s_bytes + extra);
    atomicAdd(reinterpret_cast<unsigned long long *>(p.traffic) + 1, s_steps);
  }
}

// ---------------------------------------------------------------------------
// launch
// ---------------------------------------------------------------------------
typedef void (*KernelFn)(Params);

template <int NC, int KM>
KernelFn pick_al(bool al) {
  return al ? fusion_kernel<NC, KM, true> : fusion_kernel<NC, KM, false>;
}
template <int NC>
KernelFn pick_k(int km, bool al) {
  return km == 1 ? pick_al<NC, 1>(al) : km == 4 ? pick_al<NC, 4>(al) : pick_al<NC, 8>(al);
}
KernelFn pick(int nc, int km, bool al) {
  switch (nc) {
    case 1: return pick_k<1>(km, al);
    case 2: return pick_k<2>(km, al);
    case 4: return pick_k<4>(km, al);
    default: return pick_k<8>(km, al);
  }
}

struct DeviceLimits {
  int lds_per_block = 0;
  bool ok = false;
};

DeviceLimits device_limits() {
  static std::mutex mu;
  static DeviceLimits cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return {};
  std::lock_guard<std::mutex> lk(mu);
  if (!cache[dev].ok) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) return {};
    cache[dev].lds_per_block = v;
    cache[dev].ok = true;
  }
  return cache[dev];
}

int launch(Params &p, int grid, hipStream_t stream) {
  const int nc_need = (p.V + 1023) / 1024;
  const int nc = nc_need <= 1 ? 1 : nc_need <= 2 ? 2 : nc_need <= 4 ? 4 : 8;
  const int km = p.k <= 1 ? 1 : p.k <= 4 ? 4 : 8;
  const bool al = (p.V % 4 == 0) && ((uintptr_t)p.logits % 16 == 0) && (!p.fused || (uintptr_t)p.fused % 16 == 0);
  KernelFn fn = pick(nc, km, al);
  hipFuncAttributes attr;
  hipError_t e = hipFuncGetAttributes(&attr, reinterpret_cast<const void *>(fn));
  if (e != hipSuccess) return hip_error(e, "hipFuncGetAttributes");
  DeviceLimits lim = device_limits();
  if (!lim.ok) return set_error(FUSION_E_HIP, "cannot query the device's LDS size");
  p.Vp = nc * 1024;
  const size_t per_slot = (size_t)8 * p.Vp;
  const size_t fixed = (size_t)4 * p.Vp;  // root row
  const long lds_avail = (long)lim.lds_per_block - (long)attr.sharedSizeBytes - (long)fixed;
  int slots = (int)std::min<size_t>((size_t)kMaxSlots, lds_avail > 0 ? (size_t)lds_avail / per_slot : 0);
  if (nc >= 8) slots = std::min(slots, 2);
  slots = std::min(slots, p.B);
  if (slots < 1) return set_error(FUSION_E_UNSUPPORTED, "vocabulary too large for the device's LDS");
  p.slots = slots;
  const size_t dyn = per_slot * slots + fixed;
  e = hipFuncSetAttribute(reinterpret_cast<const void *>(fn), hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
  if (e != hipSuccess) return hip_error(e, "hipFuncSetAttribute");
  hipLaunchKernelGGL(fn, dim3(grid), dim3(slots * kSlotLanes), dyn, stream, p);
  e = hipGetLastError();
  if (e != hipSuccess) return hip_error(e, "fusion kernel launch");
  return FUSION_OK;
}

int check_common(const NgramTables *lm, const BoostTrie *trie, const float *logits, int32_t V,
                 int32_t k, int32_t blank_id, int32_t blank_mode, float lambda, float beta) {
  if (!lm) return set_error(FUSION_E_ARG, "NULL n-gram tables");
  if (!logits) return set_error(FUSION_E_ARG, "NULL logits");
  if (V != lm->dev.V) return set_error(FUSION_E_ARG, "V does not match the n-gram tables");
  if (blank_id != lm->dev.blank) return set_error(FUSION_E_ARG, "blank_id does not match the n-gram tables");
  if (trie && (trie->dev.V != V || trie->dev.blank != blank_id))
    return set_error(FUSION_E_ARG, "phrase tree built for another vocabulary or blank");
  if (k < 1 || k > FUSION_MAX_K || k > V) return set_error(FUSION_E_ARG, "k out of range");
  if (blank_mode != FUSION_BLANK_AM && blank_mode != FUSION_BLANK_COMPETE) return set_error(FUSION_E_ARG, "unknown blank_mode");
  if (blank_mode == FUSION_BLANK_AM && k != 1) return set_error(FUSION_E_ARG, "FUSION_BLANK_AM needs k == 1");
  if (!std::isfinite(lambda) || !std::isfinite(beta)) return set_error(FUSION_E_ARG, "non-finite fusion weight");
  return FUSION_OK;
}

Params make_params(const NgramTables *lm, const BoostTrie *trie) {
  Params p;
  std::memset(&p, 0, sizeof p);
  p.lm = lm->dev;
  if (trie) p.tr = trie->dev;
  p.has_trie = trie != nullptr;
  return p;
}

}  // namespace
}  // namespace fusion

using namespace fusion;

extern "C" const char *fusion_last_error(void) { return t_err.c_str(); }

extern "C" int fusion_device_status(hipStream_t stream, int32_t *code) {
  if (!code) return set_error(FUSION_E_ARG, "NULL code");
  hipError_t e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_error(e, "hipStreamSynchronize");
  int v = 0;
  e = hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_status), sizeof(int), 0, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_error(e, "hipMemcpyFromSymbol");
  int zero = 0;
  e = hipMemcpyToSymbol(HIP_SYMBOL(g_status), &zero, sizeof(int), 0, hipMemcpyHostToDevice);
  if (e != hipSuccess) return hip_error(e, "hipMemcpyToSymbol");
  *code = v;
  return FUSION_OK;
}

extern "C" int fusion_step(const NgramTables *lm, const BoostTrie *trie, const float *logits,
                           const int32_t *lm_state, const int32_t *boost_state, int32_t H, int32_t V,
                           float lambda, float beta, int32_t blank_id, int32_t k, int32_t blank_mode,
                           float *fused, int32_t *tokens, float *scores, int32_t *next_lm,
                           int32_t *next_boost, hipStream_t stream) {
  int rc = check_common(lm, trie, logits, V, k, blank_id, blank_mode, lambda, beta);
  if (rc != FUSION_OK) return rc;
  if (H < 1 || H > (1 << 24)) return set_error(FUSION_E_ARG, "H out of range");
  if (!lm_state || !tokens || !scores || !next_lm || !next_boost || (trie && !boost_state))
    return set_error(FUSION_E_ARG, "NULL state or output buffer");
  Params p = make_params(lm, trie);
  p.logits = logits;
  p.lm_state = const_cast<int32_t *>(lm_state);
  p.boost_state = const_cast<int32_t *>(boost_state);
  p.tokens = tokens;
  p.scores = scores;
  p.next_lm = next_lm;
  p.next_boost = next_boost;
  p.fused = fused;
  p.T = 1;
  p.S = H;
  p.B = 1;
  p.V = V;
  p.k = k;
  p.blank = blank_id;
  p.mode = blank_mode;
  p.step_mode = 1;
  p.lam = lambda;
  p.beta = beta;
  return launch(p, H, stream);
}

extern "C" int fusion_run(const NgramTables *lm, const BoostTrie *trie, const float *logits, int32_t T,
                          int32_t S, int32_t B, int32_t V, int32_t k, float lambda, float beta,
                          int32_t blank_id, int32_t blank_mode, int32_t *lm_state, int32_t *boost_state,
                          double *hyp_score, int32_t *tokens, int32_t *parents, float *fused,
                          int64_t *traffic, hipStream_t stream) {
  int rc = check_common(lm, trie, logits, V, k, blank_id, blank_mode, lambda, beta);
  if (rc != FUSION_OK) return rc;
  if (T < 0 || S < 1 || B < 1 || B > FUSION_MAX_BEAM) return set_error(FUSION_E_ARG, "T, S or B out of range");
  if ((int64_t)S * B > (1 << 24)) return set_error(FUSION_E_ARG, "too many hypotheses");
  if (B == 1 && k != 1) return set_error(FUSION_E_ARG, "greedy decoding (B == 1) needs k == 1");
  if (B > 1 && blank_mode != FUSION_BLANK_COMPETE) return set_error(FUSION_E_ARG, "beam decoding needs FUSION_BLANK_COMPETE");
  if (!lm_state || !tokens || (trie && !boost_state)) return set_error(FUSION_E_ARG, "NULL state or output buffer");
  if (B > 1 && (!hyp_score || !parents)) return set_error(FUSION_E_ARG, "beam decoding needs hyp_score and parents");
  if (T == 0) return FUSION_OK;
  Params p = make_params(lm, trie);
  p.logits = logits;
  p.lm_state = lm_state;
  p.boost_state = boost_state;
  p.hyp_score = hyp_score;
  p.tokens = tokens;
  p.parents = parents;
  p.fused = fused;
  p.traffic = traffic;
  p.T = T;
  p.S = S;
  p.B = B;
  p.V = V;
  p.k = k;
  p.blank = blank_id;
  p.mode = blank_mode;
  p.step_mode = 0;
  p.lam = lambda;
  p.beta = beta;
  return launch(p, S, stream);
}
