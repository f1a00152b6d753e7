// Fusion step kernels for gfx950 and the C ABI entry points fusion_step /
// fusion_run: Eq. (1) of the paper (Sec. III-C) with greedy or top-k
// selection and a frame-synchronous beam.
//
// Work mapping.  One workgroup per hypothesis (W = 64, 256 or 1024 lanes),
// so a 64 x 4 beam keeps all 256 CUs busy.  Lane g owns the tokens
// y = (c * W + g) * 4 + j (j < 4, c < NC): every logits row read is a
// coalesced 16-byte strip per lane held in registers; the level-1 dense LM row
// goes straight from HBM into the workgroup's LDS row (global_load_lds), where
// the arcs of the longer contexts are then scattered.
//
// Per frame and hypothesis, the method's steps in order:
//   1  one load brings the state record (the whole backoff chain: backoffs and
//      arc ranges of every context level) and the phrase node; the logits row
//      and the dense row are issued alongside;
//   2  one load brings the arcs of all levels (flattened) and the phrase
//      transitions of the state; meanwhile the row statistics are reduced
//      (online max / sum-exp, raw argmax);
//   3  the arcs are scattered into LDS level by level, each summed with the
//      backoffs above its level (the addition order of the backoff
//      recursion), and the phrase transitions with their entry values;
//   4  key = (x + lambda*lm) + beta*boost per owned token, top-k per lane, per
//      wave (shuffles) and per hypothesis; each candidate carries where its
//      next LM / phrase state comes from, so no further lookup is needed;
//   5  beam: the B workgroups of a stream publish their candidates, meet at a
//      per-stream counter, and each ranks all B*k candidates (fp64 running
//      score) to take its own new hypothesis.
// No MFMA: ~10 flops per score over gathered data.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

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

constexpr int kMaxWaves = 16;
constexpr int kMaxLevels = FUSION_MAX_ORDER;  // context levels 1..N-1 <= 5
constexpr int kAux = 256;                     // LDS side tables: phrase transitions, top-level next states
constexpr int kRecW = 16;                     // words read per state record: record_stride(FUSION_MAX_ORDER)
constexpr int kSpinLimit = 1 << 21;           // bounded wait at the beam rendezvous (polls, each waiting
                                              // for its loads: about a second)

__device__ int g_status;
__device__ __align__(64) int32_t g_zero_words[16];  // never written: the record and node of "no state"

// Beam exchange memory of fusion_run_lms_noalloc, one copy per GPU, held until
// the process ends.  Host code never passes this name to a kernel: it is a
// host-side stand-in, not a device address.  The device address comes from
// hipGetSymbolAddress (static_scratch below) and is what the kernels receive.
constexpr size_t kStaticScratchBytes = FUSION_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned long long scratch[kStaticScratchBytes / sizeof(unsigned long long)];

struct Params {
  LMDevice lm[FUSION_MAX_LMS];  // the n_lm models of Eq. (1), each with its own weight lam[i]
  TrieDevice tr;
  const float *logits;
  int32_t *lm_state;
  int32_t *boost_state;
  double *hyp_score;
  int32_t *tokens;
  int32_t *parents;
  float *fused;
  int64_t *traffic;
  float *scores;  // fusion_step outputs [H, k]
  int32_t *next_lm;
  int32_t *next_boost;
  unsigned long long *xchg;  // beam exchange [S][2][B][k] candidate records of four tagged words
  unsigned long long *hist;  // recombination: [H] in/out history hashes (0: derive from the initial states) or NULL
  unsigned *tickets;         // beam: arrival counters, one per blockIdx class (8 with xcd_map, else 1)
  // t_base: the number of frames decoded by earlier calls of a frame loop that
  // keeps the exchange between calls (its records are tagged by global frame)
  int32_t T, S, B, V, k, blank, mode, has_trie, step_mode, s_off, xcd_map, n_lm, recombine, t_base;
  float lam[FUSION_MAX_LMS], beta;
};

// The kernel's argument block (its one argument, a Params, at offset 0) through an
// address the compiler cannot see through: a field read from it is read where it
// is used.  For pointers that only rare paths of the frame loop need; read as
// plain arguments, they are hoisted out of the loop and hold scalar registers
// across it (pushing other values into spill slots)
__device__ __forceinline__ const __attribute__((address_space(4))) Params &args_here() {
  const __attribute__((address_space(4))) char *kb =
      (const __attribute__((address_space(4))) char *)__builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(kb));
  return *(const __attribute__((address_space(4))) Params *)kb;
}
__device__ __forceinline__ bool before(float ka, int ya, float kb, int yb) {
  return ka > kb || (ka == kb && ya < yb);
}
__device__ __forceinline__ float as_float(int v) { return __int_as_float(v); }
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
// the splitmix64 finalizer: a 64-bit mix for the beam's history hashes
__device__ __forceinline__ unsigned long long mix64(unsigned long long z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
// log(exp(a) + exp(b)) in fp64.  Not inlined: the merges that call it are rare,
// and inlined, the constants of its exp and log1p would stay in vector
// registers across the whole frame loop of the recombining kernel
__device__ __attribute__((noinline)) double log_add(double a, double b) {
  const double m = a > b ? a : b, d = a > b ? b - a : a - b;
  return m + log1p(exp(d));
}
__device__ __forceinline__ unsigned long long umin64(unsigned long long a, unsigned long long b) {
  return a < b ? a : b;
}

// raw buffer access to one V-wide row: a 4-SGPR descriptor and a per-lane
// byte offset; reads past the row return 0
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t row_rsrc(const float *base, int n) {
  // every field uniform (a descriptor the compiler cannot prove uniform costs a
  // readfirstlane loop around each access)
  const unsigned long long v = reinterpret_cast<unsigned long long>(base);
  const unsigned lo = (unsigned)__builtin_amdgcn_readfirstlane((int)(unsigned)v);
  const unsigned hi = (unsigned)__builtin_amdgcn_readfirstlane((int)(unsigned)(v >> 32));
  float *ub = reinterpret_cast<float *>(((unsigned long long)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, (short)0, __builtin_amdgcn_readfirstlane(n * 4), 0x00020000);
}
__device__ __forceinline__ float4 row_load4(rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ float row_load1(rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}
__device__ __forceinline__ void row_store4(rsrc_t r, float4 v, int voff, int soff) {
  typedef int v4i __attribute__((ext_vector_type(4)));
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4i, v), r, voff, soff, 0);
}
__device__ __forceinline__ void row_store1(rsrc_t r, float v, int voff, int soff) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), r, voff, soff, 0);
}
typedef __attribute__((address_space(3))) void *lds_ptr_t;

// record words: [0] c_1 | m << 16, [1] state id, [2 + 3(L-2) + {0,1,2}] = (bo, first arc, arcs) of level L
__device__ __forceinline__ constexpr int rec_bo_word(int L) { return 2 + 3 * (L - 2); }
__device__ __forceinline__ constexpr int rec_beg_word(int L) { return 3 + 3 * (L - 2); }
__device__ __forceinline__ constexpr int rec_cnt_word(int L) { return 4 + 3 * (L - 2); }
// the record word naming the chain's context row (record_ctx_word)
__device__ __forceinline__ constexpr int rec_ctx_word(int N) { return 2 + 3 * (N > 2 ? N - 2 : 0); }

// ---- wave-level reductions with DPP moves (no LDS) ------------------------------
// rows of 16 lanes: quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror,
// row_mirror; then row_bcast:15 (rows 1, 3) and row_bcast:31 (rows 2, 3) carry
// the row results to lane 63
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_f(float ident, float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(ident), __float_as_int(v), CTRL, ROWS, 0xF, false));
}
__device__ __forceinline__ float row_max(float v) {
  v = fmaxf(v, dpp_f<0xB1, 0xF>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x4E, 0xF>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x141, 0xF>(-INFINITY, v));
  return fmaxf(v, dpp_f<0x140, 0xF>(-INFINITY, v));
}
__device__ __forceinline__ float row_sum(float v) {
  v = v + dpp_f<0xB1, 0xF>(0.0f, v);
  v = v + dpp_f<0x4E, 0xF>(0.0f, v);
  v = v + dpp_f<0x141, 0xF>(0.0f, v);
  return v + dpp_f<0x140, 0xF>(0.0f, v);
}
// uniform maximum over the wave (-0 and +0 may come out either way)
__device__ __forceinline__ float wave_max_f(float v) {
  v = row_max(v);
  v = fmaxf(v, dpp_f<0x142, 0xA>(-INFINITY, v));
  v = fmaxf(v, dpp_f<0x143, 0xC>(-INFINITY, v));
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
// uniform sum over the wave
__device__ __forceinline__ float wave_sum(float v) {
  v = row_sum(v);
  v = v + dpp_f<0x142, 0xA>(0.0f, v);
  v = v + dpp_f<0x143, 0xC>(0.0f, v);
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
// order-preserving map of non-NaN floats onto int32 (x + 0.0 first folds -0
// into +0, so equal floats map to equal ints); an involution
__device__ __forceinline__ int ord_key(float x) {
  const int b = __float_as_int(x + 0.0f);
  return b ^ ((b >> 31) & 0x7FFFFFFF);
}
__device__ __forceinline__ float key_of(int i) { return __int_as_float(i ^ ((i >> 31) & 0x7FFFFFFF)); }
// (order-preserving key image, token id) as one unsigned 64-bit value, larger
// for a higher key and, at equal keys, for a lower id
__device__ __forceinline__ unsigned long long sel_order(int key, int y) {
  return ((unsigned long long)((uint32_t)key ^ 0x80000000u) << 32) | (unsigned long long)(~(uint32_t)y);
}
// the key of a composite's upper half
__device__ __forceinline__ int sel_key(int hi) { return (int)((uint32_t)hi ^ 0x80000000u); }
// uniform maximum of an int over the wave (identity INT_MIN)
template <int CTRL, int ROWS>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(INT_MIN, v, CTRL, ROWS, 0xF, false);
}
// maximum of an int over each 16-lane row, in every lane of the row
__device__ __forceinline__ int row_max_i(int v) {
  v = max(v, dpp_i<0xB1, 0xF>(v));
  v = max(v, dpp_i<0x4E, 0xF>(v));
  v = max(v, dpp_i<0x141, 0xF>(v));
  return max(v, dpp_i<0x140, 0xF>(v));
}
__device__ __forceinline__ int wave_max_i(int v) {
  v = max(v, dpp_i<0xB1, 0xF>(v));
  v = max(v, dpp_i<0x4E, 0xF>(v));
  v = max(v, dpp_i<0x141, 0xF>(v));
  v = max(v, dpp_i<0x140, 0xF>(v));
  v = max(v, dpp_i<0x142, 0xA>(v));
  v = max(v, dpp_i<0x143, 0xC>(v));
  return __builtin_amdgcn_readlane(v, 63);
}
// e^x through the hardware base-2 exponential (about 1e-6 relative error near
// the arguments used here, x <= 0)
__device__ __forceinline__ float exp_fast(float x) { return __builtin_amdgcn_exp2f(x * 1.4426950408889634f); }

// every lane of each 16-lane row ends with the row's best (key desc, id asc)
template <int CTRL>
__device__ __forceinline__ void dpp_best(float &k, int &y) {
  const float k2 = dpp_f<CTRL, 0xF>(-INFINITY, k);
  const int y2 = __builtin_amdgcn_update_dpp(INT_MAX, y, CTRL, 0xF, 0xF, false);
  if (before(k2, y2, k, y)) {
    k = k2;
    y = y2;
  }
}
__device__ __forceinline__ void row_best(float &k, int &y) {
  dpp_best<0xB1>(k, y);
  dpp_best<0x4E>(k, y);
  dpp_best<0x141>(k, y);
  dpp_best<0x140>(k, y);
}

// Barrier for data exchanged through LDS alone: waits for this wave's LDS
// operations but not for its vector-memory loads in flight (the next frame's
// logits).  __syncthreads would wait for those too (its release fence waits for
// every outstanding vector-memory operation).
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// hypothesis state carried between frames (LDS, written by one lane)
template <int NL>
struct HypState {
  // per LM: where the next state comes from (an id; -1: reached from c1p by
  // token y; -(r + 2): reached from the context of context row r by token y),
  // the parent's c_1, the last token of the context (-1: from the record), the
  // id of the state scored this frame
  int lmsrc[NL], c1p[NL], c1[NL], cur_lm[NL];
  int qsrc, y, fl;  // phrase source, token; flags 1 alive, 2 invalid
  int cur_q;        // phrase state scored this frame
  double S;         // running beam score
  unsigned long long hist;  // 48-bit hash of the history (initial states, emitted tokens): recombination
};


// MODE: what a launch computes (the code of the other modes is compiled out)
// (kModeBeamRC: beam with recombination of equal histories)
constexpr int kModeStep = 0, kModeGreedy = 1, kModeBeam = 2, kModeBeamRC = 3;

template <int W, int NC, int KM, bool AL, int MODE, int NL>
__global__ void __launch_bounds__(W) fusion_kernel(Params p) {
  constexpr int NW = W / 64;
  constexpr int Vp = NC * 4 * W;
  constexpr int kUA = W >= 1024 ? 1 : 4;  // arcs per lane fetched in the second hop
  constexpr int kUD = W >= 1024 ? 1 : 2;  // phrase transitions per lane fetched in the second hop
  constexpr bool CTX = NC == 1;  // context rows used (an 8192-wide row pair would not fit the LDS)
  extern __shared__ __align__(16) unsigned char dyn[];
  // LDS rows, one entry per token: per LM, the dense level-1 row and the winning
  // explicit arc (stamp << 48 | level << 45 | offset << 32 | value bits, kept by
  // an atomic max, so the highest level wins whatever the order of the writes);
  // the phrase transition overriding the root's (stamp << 16 | transition + 1).
  // The stamp is the frame's (t mod 2^15) + 1: entries of earlier frames compare
  // lower and read as absent, so no per-frame clearing is needed.  Row NL of
  // lmval holds the first LM's context row when its state has one: the LM row of
  // the deepest context of the chain with many successors, already resolved
  // through every level up to that context
  // With one LM the phrase term reads erow: per token the entry value E of the
  // phrase state after it, the root's unless this frame's phrase state
  // overrides the token.  Each lane puts its tokens back to the root's values
  // right after reading them, and the scatter writes the overrides.
  constexpr bool ER = NL == 1 && NC == 1;  // (8192-wide rows: no room in the LDS)
  constexpr int kRows = NL + (CTX ? 1 : 0);
  float *lmval = reinterpret_cast<float *>(dyn);                                                  // [kRows][Vp]
  unsigned long long *arcw = reinterpret_cast<unsigned long long *>(dyn + 4 * kRows * Vp);        // [NL][Vp]
  uint32_t *ptag = reinterpret_cast<uint32_t *>(dyn + (4 * kRows + 8 * NL) * Vp);
  float *erow = reinterpret_cast<float *>(dyn + (4 * kRows + 8 * NL + 4) * Vp);                   // [Vp] if ER
  float *sE = reinterpret_cast<float *>(dyn + (4 * kRows + 8 * NL + 4 + (ER ? 4 : 0)) * Vp);  // sE[j + 1]: entry value of transition j
  int *sDT = reinterpret_cast<int *>(sE + kAux + 4);
  int *sTN = sDT + kAux;  // [NL][kAux]
  __shared__ float s_pm[kMaxWaves], s_ps[kMaxWaves];
  __shared__ int s_paid[kMaxWaves];
  __shared__ float s_lse;  // the current frame's log-sum-exp of the logits row
  __shared__ int s_am;     // and the lowest id holding its maximum
  __shared__ int s_nstat;  // waves done with the next frame's strip statistics
  __shared__ int w_key[kMaxWaves][KM];  // order-preserving images of the keys (ord_key)
  __shared__ int w_y[kMaxWaves][KM];
  // each wave's best key with its wave index, and the hypothesis' listed entries
  // (compacted) and top K, all as sel_order composites (KM > 1)
  __shared__ __align__(16) unsigned long long s_wmax[kMaxWaves];
  __shared__ __align__(16) unsigned long long s_sel[16];
  __shared__ unsigned long long s_win[KM];
  __shared__ HypState<NL> hs;
  // beam rendezvous staging (wave 0): candidate records (the second LM's source
  // and c_1 in s_xb), parent flags, totals
  __shared__ int4 s_xa[FUSION_MAX_BEAM * FUSION_MAX_K];
  __shared__ int2 s_xb[NL > 1 ? FUSION_MAX_BEAM * FUSION_MAX_K : 1];
  __shared__ int s_xf[FUSION_MAX_BEAM * FUSION_MAX_K];
  __shared__ __align__(16) double s_tot[FUSION_MAX_BEAM * FUSION_MAX_K];
  // recombination: history hash after each candidate, merged totals
  __shared__ unsigned long long s_hh[MODE == kModeBeamRC ? FUSION_MAX_BEAM * FUSION_MAX_K : 1];
  __shared__ double s_mt[MODE == kModeBeamRC ? FUSION_MAX_BEAM * FUSION_MAX_K : 1];
  __shared__ long long s_sbase[NL][kMaxLevels];  // state id of arc index i of level L < N-1: s_sbase[L] + i
  __shared__ int s_lbeg[NL][kMaxLevels];  // first arc of each level of the current state
  __shared__ int s_cfg[2];  // V, blank: re-read each frame so per-token masks stay inside the loop
  __shared__ int s_ticket;  // beam: this workgroup's arrival ticket
  __shared__ unsigned long long s_bytes, s_steps;

  const LMDevice *lms = p.lm;
  const TrieDevice &tr = p.tr;
  const int g = threadIdx.x;
  // this lane's entries of the arc and phrase rows back to 0 (absent)
  auto clear_rows = [&]() {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int y0 = (c * W + g) * 4;
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        *reinterpret_cast<uint4 *>(arcw + i * Vp + y0) = make_uint4(0u, 0u, 0u, 0u);
        *reinterpret_cast<uint4 *>(arcw + i * Vp + y0 + 2) = make_uint4(0u, 0u, 0u, 0u);
      }
      *reinterpret_cast<uint4 *>(ptag + y0) = make_uint4(0u, 0u, 0u, 0u);
    }
  };
  const int wave = g >> 6;
  const int lane = g & 63;
  constexpr bool BEAM = MODE == kModeBeam || MODE == kModeBeamRC;
  constexpr bool RC = MODE == kModeBeamRC;
  const int B = BEAM ? p.B : 1, K = p.k;
  int Nl[NL], RSl[NL];  // order and record stride of each LM
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    Nl[i] = lms[i].N;
    RSl[i] = lms[i].rec_stride;
  }
  // workgroup -> (stream, hypothesis); with xcd_map the B workgroups of a stream
  // share blockIdx mod 8, i.e. one XCD and its L2, for the per-frame exchange.
  // A beam takes its index r within that class from an arrival counter: the
  // workgroups that have started always hold the first tickets of each class,
  // so every stream but the last one started in a class is complete and runs
  // to its end, freeing room for the rest.  The beam therefore needs no
  // co-residency guarantee (no cooperative launch), only room for the
  // incomplete streams beside one complete one (checked at launch)
  int sl, b;
  {
    const int x = blockIdx.x;
    int r = p.xcd_map ? x >> 3 : x;
    if constexpr (BEAM) {
      const int n_cls = p.xcd_map ? (int)(gridDim.x >> 3) : (int)gridDim.x;
      if (g == 0) {
        unsigned *ctr = p.tickets + (p.xcd_map ? (x & 7) : 0);
        const int tk = (int)atomicAdd(ctr, 1u);
        // the class's last ticket leaves the counter at 0 for the next launch
        if (tk == n_cls - 1) atomicExch(ctr, 0u);
        s_ticket = tk;
      }
      __syncthreads();
      r = s_ticket;
      if (r >= n_cls) {  // counters not reset since an earlier launch: no slot for this workgroup
        if (g == 0) atomicOr(&g_status, FUSION_STATUS_SYNC_TIMEOUT);
        return;
      }
    }
    if (p.xcd_map) {
      sl = (x & 7) + 8 * (r / B);
      b = r % B;
    } else {
      sl = r / B;
      b = r % B;
    }
  }
  const int s = sl + p.s_off;
  const int H = p.S * B;
  const int h = s * B + b;

  // ---- prologue ------------------------------------------------------------------
  if (g < kMaxLevels) {
#pragma unroll
    for (int i = 0; i < NL; ++i)
      s_sbase[i][g] = (g >= 2 && g + 1 <= Nl[i] - 1) ? lms[i].off[g + 1] - lms[i].arc_base[g] : 0;
  }
  if (g == 0) {
    s_cfg[0] = p.V;
    s_cfg[1] = p.blank;
    s_bytes = 0;
    s_steps = 0;
    const int V = p.V, blank = p.blank;
    const int q = p.has_trie ? p.boost_state[h] : 0;
    const double sc = BEAM ? p.hyp_score[h] : 0.0;
    bool ok_lm = true;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int sig = p.lm_state[(int64_t)i * H + h];  // [n_lm][H]
      const bool ok_i = sig >= 0 && sig < lms[i].n_states && sig != blank && (sig != V + 1 || lms[i].eos_ok);
      ok_lm = ok_lm && ok_i;
      hs.lmsrc[i] = sig;
      hs.c1p[i] = -1;
      // c_1, the last token of the state: the state itself below V + 2, else
      // from its record (so that every frame knows c_1 before its record arrives)
      hs.c1[i] = !ok_i ? -1 : sig < V + 2 ? sig : (lms[i].rec[(int64_t)(sig - V - 2) * lms[i].rec_stride] & 0xFFFF);
      hs.cur_lm[i] = sig;
    }
    const bool ok_q = !p.has_trie || (q >= 0 && q < tr.n_nodes);
    const bool alive = !BEAM || sc > -INFINITY;
    hs.qsrc = q;
    hs.y = -1;
    hs.fl = (alive ? 1 : 0) | ((ok_lm && ok_q) ? 0 : 2);
    hs.cur_q = q;
    hs.S = sc;
    if constexpr (RC) {
      // the history carried from an earlier call, else one that starts at the
      // slot's initial states (never 0, which marks the start of a stream)
      unsigned long long hh = p.hist ? (p.hist[h] & ((1ull << 48) - 1)) : 0ull;
      if (hh == 0ull) {
        hh = mix64(0x243F6A8885A308D3ull ^ (unsigned long long)(unsigned)q);
#pragma unroll
        for (int i = 0; i < NL; ++i) hh = mix64(hh ^ ((unsigned long long)(unsigned)hs.lmsrc[i] << (8 * i + 1)));
        hh &= (1ull << 48) - 1;
        hh = hh ? hh : 1ull;
      }
      hs.hist = hh;
    }
    if (alive && !(ok_lm && ok_q))
      atomicOr(&g_status, (ok_lm ? 0 : FUSION_STATUS_BAD_LM_STATE) | (ok_q ? 0 : FUSION_STATUS_BAD_BOOST_STATE));
  }
  float rE[NC][4];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int y0 = (c * W + g) * 4;
#pragma unroll
    for (int j = 0; j < 4; ++j) rE[c][j] = (p.has_trie && y0 + j < p.V) ? tr.root_E[y0 + j] : 0.0f;
    if (ER) *reinterpret_cast<float4 *>(erow + y0) = make_float4(rE[c][0], rE[c][1], rE[c][2], rE[c][3]);
  }
  clear_rows();
  __syncthreads();

  // logits strip of this lane, raw (masked per frame): frame t+1's strip is
  // fetched during frame t, so it is in registers when t+1 begins
  const int voff = g * 16;
  float xraw[NC][4];
  float xraw0[NC][4];  // wave 1: wave 0's strip too, for its row statistics
  auto fetch_strip = [&](const rsrc_t &xr, float (&dst)[NC][4], int off) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      if (AL) {
        const float4 xx = row_load4(xr, off, c * W * 16);
        dst[c][0] = xx.x; dst[c][1] = xx.y; dst[c][2] = xx.z; dst[c][3] = xx.w;
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) dst[c][j] = row_load1(xr, off + 4 * j, c * W * 16);
      }
    }
  };
  // the logits row of this hypothesis at the frame being fetched; it advances by
  // one frame (H rows) per fetch and stays on the last frame
  const float *xrow = p.logits + (int64_t)h * p.V;
  const int64_t xstride = (int64_t)H * p.V;
  auto fetch_logits = [&]() {
    const rsrc_t xr = row_rsrc(xrow, p.V);
    fetch_strip(xr, xraw, voff);
    if (NW > 1 && wave == 1) fetch_strip(xr, xraw0, lane * 16);
  };
  fetch_logits();
  // row statistics of the logits of strip sw (the 64-lane strip of wave sw) held
  // in xs: strip max, sum of exp below it, lowest id holding the max (only the
  // acoustic blank decision needs it).  They depend on the logits alone, so those
  // of frame t+1 are computed in frame t by the waves that are otherwise idle
  // while wave 0 ends the frame (wave 1 takes wave 0's strip); frame 0's here
  auto row_stats = [&](const float (&xs)[NC][4], int sw, int V) {
    float xv[NC][4];  // tokens >= V: -inf
    float lmx = -INFINITY;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        xv[c][j] = (c * W + sw * 64 + lane) * 4 + j < V ? xs[c][j] : -INFINITY;
        lmx = fmaxf(lmx, xv[c][j]);
      }
    const float mw = wave_max_f(lmx);
    float lsum = 0.0f;
    if (mw > -INFINITY) {
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int j = 0; j < 4; ++j) lsum += (xv[c][j] > -INFINITY) ? exp_fast(xv[c][j] - mw) : 0.0f;
    }
    const float ssum = wave_sum(lsum);
    int aid = INT_MAX;
    if (p.mode == FUSION_BLANK_AM && mw > -INFINITY) {
#pragma unroll
      for (int c = NC - 1; c >= 0; --c) {
        unsigned long long mj[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) mj[j] = __ballot(xv[c][j] == mw && (c * W + sw * 64 + lane) * 4 + j < V);
        const unsigned long long any = mj[0] | mj[1] | mj[2] | mj[3];
        if (any) {
          const int src = __ffsll((long long)any) - 1;
          int jj = 3;
#pragma unroll
          for (int j = 2; j >= 0; --j) jj = ((mj[j] >> src) & 1ull) ? j : jj;
          aid = (c * W + sw * 64 + src) * 4 + jj;
        }
      }
    }
    if (lane == 0) {
      s_pm[sw] = mw;
      s_ps[sw] = ssum;
      s_paid[sw] = aid;
    }
  };
  // the strip statistics of all NW waves combined into s_lse / s_am (one wave)
  auto combine_stats = [&]() {
    const bool wl = lane < NW;
    const float pm = wl ? s_pm[lane] : -INFINITY;
    const float M = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(row_max(pm)), 0));
    const float term = (wl && pm > -INFINITY) ? s_ps[lane] * exp_fast(pm - M) : 0.0f;
    const float lse = M + logf(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(row_sum(term)), 0)));
    float ak = pm;
    int ay = wl ? s_paid[lane] : INT_MAX;
    row_best(ak, ay);
    if (lane == 0) {
      s_lse = lse;
      s_am = ay;
    }
  };
  // a V-wide fp32 row straight from HBM into an LDS row (this wave's strips)
  auto load_row = [&](const float *drow, float *row, int V) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int wbase = c * W + wave * 64;  // first 4-token strip of this wave
      if (AL) {
        const int y0 = (wbase + lane) * 4;
        __builtin_amdgcn_global_load_lds(drow + (y0 < V ? y0 : 0), (lds_ptr_t)(row + wbase * 4), 16, 0, 0);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int y = wbase * 4 + j * 64 + lane;
          __builtin_amdgcn_global_load_lds(drow + (y < V ? y : 0), (lds_ptr_t)(row + wbase * 4 + j * 64), 4, 0, 0);
        }
      }
    }
  };
  row_stats(xraw, wave, p.V);
  if (g == 0) s_nstat = 0;
  __syncthreads();
  if (wave == NW - 1) combine_stats();
  __syncthreads();

  bool aborted = false;  // after one failed rendezvous this workgroup stops waiting
  for (int t = 0; t < p.T; ++t) {
    const int V = uni(s_cfg[0]), blank = uni(s_cfg[1]);
    const int fl = uni(hs.fl);
    const bool act = (fl & 1) != 0;
    const bool inv = act && (fl & 2) != 0;
    const bool ok = act && !inv;
    // stamps repeat every 2^15 frames: the rows are cleared before they would
    // (the previous frame's last reads of them precede its final barrier)
    const uint32_t stamp = (uint32_t)(t & 0x7FFF) + 1u;
    if (stamp == 1u && t > 0) {
      clear_rows();
      __syncthreads();
    }
    const int qsrc = uni(hs.qsrc), yin = uni(hs.y);
    int lmsrc[NL], c1[NL];
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      lmsrc[i] = uni(hs.lmsrc[i]);
      c1[i] = uni(hs.c1[i]);
    }
    // ---- hop 1: state records, phrase node, dense level-1 rows ------------------
    const int32_t *rp[NL];
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      rp[i] = nullptr;
      if (ok) {
        if (lmsrc[i] < -1) rp[i] = lms[i].ctx_rec + ((int64_t)(-lmsrc[i] - 2) * V + yin) * RSl[i];
        else if (lmsrc[i] < 0) rp[i] = lms[i].rec_dense + ((int64_t)uni(hs.c1p[i]) * V + yin) * RSl[i];
        else if (lmsrc[i] >= V + 2) rp[i] = lms[i].rec + (int64_t)(lmsrc[i] - V - 2) * RSl[i];
      }
    }
    const int4 *np = nullptr;
    if (ok && p.has_trie) np = qsrc < 0 ? tr.root_node + yin : tr.node + qsrc;
    const int64_t rowoff = ((int64_t)t * H + h) * V;
    // this frame's logits (fetched during the previous frame); waited for here,
    // before this frame's loads are issued
#pragma unroll
    for (int c = 0; c < NC; ++c) asm volatile("" ::"v"(xraw[c][0]), "v"(xraw[c][1]), "v"(xraw[c][2]), "v"(xraw[c][3]));
    float xv[NC][4];
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int j = 0; j < 4; ++j) xv[c][j] = (act && (c * W + g) * 4 + j < V) ? xraw[c][j] : -INFINITY;
    // the state records and the phrase node with scalar loads (uniform addresses):
    // kRecW words per record (the record arrays carry a tail pad so that reading
    // past a short record stays inside them); "no record" / "no node" read the
    // zero words
    int rec[NL][kRecW];
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const __attribute__((address_space(4))) int32_t *r =
          (const __attribute__((address_space(4))) int32_t *)(rp[i] ? rp[i] : g_zero_words);
#pragma unroll
      for (int w = 0; w < kRecW; ++w) rec[i][w] = r[w];
    }
    const __attribute__((address_space(4))) int32_t *nq =
        (const __attribute__((address_space(4))) int32_t *)(np ? reinterpret_cast<const int32_t *>(np) : g_zero_words);
    const int node[4] = {nq[0], nq[1], nq[2], nq[3]};
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      // level-1 dense row straight into the LM's LDS row.  Issued
      // unconditionally (row 0 stands in when the hypothesis has no keys to
      // compute this frame), so that only the records are waited for before the
      // second hop
      load_row(lms[i].dense + (int64_t)(ok ? c1[i] : 0) * V, lmval + i * Vp, V);
    }
    if (NW == 1 && t > 0) {  // a single wave has no idle helper
      row_stats(xraw, 0, V);
      combine_stats();
    }
    // ---- decode the records ---------------------------------------------------------
    const float phiq = as_float(node[0]);
    const int dbeg = node[1];
    const int dcnt = node[2];
    const int qid = np ? node[3] : qsrc;
    // per LM: order m of the state, its id; backoffs, first arcs and arc counts of
    // levels 2..m.  The first LM's context row (level D >= 2 of the chain, row r)
    // replaces the levels up to D: only the arcs of the levels above D are fetched
    // (lcnt 0 for the others).  Further LMs fetch the arcs of every level
    int m[NL], sid[NL], total_arcs[NL], Dc = 0, crow = 0;
    float bo[NL][kMaxLevels];
    int lcnt[NL][kMaxLevels], lbeg[NL][kMaxLevels];
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      m[i] = rp[i] ? (rec[i][0] >> 16) : 1;
      sid[i] = rp[i] ? rec[i][1] : lmsrc[i];
      int Di = 0;
      if (CTX && i == 0 && rp[0]) {
        const int n0 = Nl[0];
        const int cw = n0 == 3 ? rec[0][rec_ctx_word(3)] : n0 == 4 ? rec[0][rec_ctx_word(4)]
                     : n0 == 5 ? rec[0][rec_ctx_word(5)] : n0 == 6 ? rec[0][rec_ctx_word(6)] : 0;
        Dc = Di = (int)((unsigned)cw >> 28);
        crow = cw & 0x0FFFFFFF;
      }
      total_arcs[i] = 0;
      // levels above m are absent: backoff 0 and no arcs (their record words
      // hold zeros or, at level N, the context-row word)
#pragma unroll
      for (int L = 2; L < kMaxLevels; ++L) {
        const bool lv = L <= m[i];
        bo[i][L] = lv ? as_float(rec[i][rec_bo_word(L)]) : 0.0f;
        lcnt[i][L] = (lv && L > Di) ? rec[i][rec_cnt_word(L)] : 0;
        lbeg[i][L] = lv ? rec[i][rec_beg_word(L)] : 0;
        total_arcs[i] += lcnt[i][L];
      }
    }
    if (CTX && ok && Dc >= 2) load_row(lms[0].ctx_lm + (int64_t)crow * V, lmval + NL * Vp, V);
    // ---- hop 2: first arcs of levels 2..m (flattened) and first phrase transitions --
    int2 ab[NL][kUA];
    int at[NL][kUA], tn[NL][kUA];  // at = level << 16 | offset within the level
#pragma unroll
    for (int i = 0; i < NL; ++i) {
#pragma unroll
      for (int u = 0; u < kUA; ++u) {
        int f = u * W + g;
        ab[i][u] = make_int2(INT_MAX, 0);
        at[i][u] = 0;
        tn[i][u] = 0;
        // the level of flattened arc f against the (uniform) starts of the levels:
        // the last level that starts at or before f; then f's offset within it
        int L = 2, bL = lbeg[i][2], fo = f, e = 0;
#pragma unroll
        for (int L2 = 3; L2 < kMaxLevels; ++L2) {
          e += lcnt[i][L2 - 1];  // first flattened index of level L2
          const bool past = f >= e && L2 <= m[i];
          L = past ? L2 : L;
          bL = past ? lbeg[i][L2] : bL;
          fo = past ? f - e : fo;
        }
        f = fo;
        if (u * W + g < total_arcs[i]) {
          at[i][u] = (L << 16) | f;
          ab[i][u] = lms[i].arcs[bL + f];
          if (L == Nl[i] - 1 && f < kAux) tn[i][u] = lms[i].top_next[bL + f - lms[i].arc_base[Nl[i] - 1]];
        }
      }
    }
    int4 dd[kUD];
#pragma unroll
    for (int u = 0; u < kUD; ++u) {
      const int j = u * W + g;
      dd[u] = make_int4(INT_MAX, 0, 0, 0);
      if (j < dcnt) dd[u] = tr.delta[dbeg + j];
    }
    if (ok && g == 0) {
      hs.cur_q = qid;
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        hs.cur_lm[i] = sid[i];
        hs.c1[i] = c1[i];
#pragma unroll
        for (int L = 2; L < kMaxLevels; ++L) s_lbeg[i][L] = lbeg[i][L];
      }
    }
    // ---- scatter (no ordering between levels: see arcw) ----------------------------
    // an arc of level L is stored summed with the backoffs of levels L+1.., the
    // addition order of the backoff recursion
    auto put_arc = [&](int i, int L, int j, int2 a, int tnext) {
      const int y = a.x;
      if (y < V) {
        float v = as_float(a.y);
#pragma unroll
        for (int L2 = 3; L2 < kMaxLevels; ++L2) {
          if (L2 > m[i]) break;  // uniform: the levels above m back off by nothing
          v = v + (L2 > L ? bo[i][L2] : 0.0f);
        }
        const uint32_t tag = (stamp << 16) | (uint32_t)((L << 13) | j);
        __hip_atomic_fetch_max(arcw + i * Vp + y, ((unsigned long long)tag << 32) | (unsigned long long)__float_as_uint(v),
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        if (L == Nl[i] - 1 && j < kAux) sTN[i * kAux + j] = tnext;
      }
    };
    if (ok) {
#pragma unroll
      for (int u = 0; u < kUD; ++u) {
        const int j = u * W + g;
        if (j < dcnt) {
          ptag[dd[u].x] = (stamp << 16) | (uint32_t)(j + 1);
          if (ER) erow[dd[u].x] = as_float(dd[u].z);
          if (j < kAux) {
            sE[j + 1] = as_float(dd[u].z);
            sDT[j] = dd[u].y;
          }
        }
      }
      for (int j = kUD * W + g; j < dcnt; j += W) {
        const int4 e = tr.delta[dbeg + j];
        ptag[e.x] = (stamp << 16) | (uint32_t)(j + 1);
        if (ER) erow[e.x] = as_float(e.z);
        if (j < kAux) {
          sE[j + 1] = as_float(e.z);
          sDT[j] = e.y;
        }
      }
#pragma unroll
      for (int i = 0; i < NL; ++i)
#pragma unroll
        for (int u = 0; u < kUA; ++u)
          if (at[i][u] != 0) put_arc(i, at[i][u] >> 16, at[i][u] & 0xFFFF, ab[i][u], tn[i][u]);
      // arcs beyond the first kUA * W of the flattened levels
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        const int N = Nl[i];
        int covered = kUA * W;
#pragma unroll
        for (int L = 2; L < kMaxLevels; ++L) {
          if (L > m[i]) break;  // uniform
          const int bL = lbeg[i][L], cL = lcnt[i][L];
          const int done = min(cL, max(0, covered));
          covered -= cL;
          const int2 *A = lms[i].arcs + bL;
          for (int j0 = done; j0 < cL; j0 += 4 * W) {
            int2 a4[4];
            int t4[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int j = j0 + u * W + g;
              a4[u] = j < cL ? A[j] : make_int2(INT_MAX, 0);
              t4[u] = (L == N - 1 && j < cL && j < kAux) ? lms[i].top_next[bL + j - lms[i].arc_base[N - 1]] : 0;
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int j = j0 + u * W + g;
              if (j < cL) put_arc(i, L, j, a4[u], t4[u]);
            }
          }
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0);  // the dense rows have landed in LDS
    __syncthreads();
    // ---- the row statistics of this frame ---------------------------------------------
    // the log-sum-exp is needed by wave 0 (selected scores, beam totals) and, for
    // fused rows, by every wave; the acoustic argmax (mode A) by every wave
    const float lse = __int_as_float(uni(__float_as_int(s_lse)));
    const int am = uni(s_am);
    // ---- keys and the fused row ------------------------------------------------------
    const bool blank_only = inv || (p.mode == FUSION_BLANK_AM && am == blank);
    const bool want_keys = ok && (!blank_only || p.fused);
    const bool compete = p.mode == FUSION_BLANK_COMPETE;
    const bool write_fused = p.fused != nullptr && ok;
    float kk[NC][4];
    bool cd[NC][4];  // token (c, j) of this lane is a candidate
    // which tokens compete this frame (uniform): blank in blank-only frames or
    // when it competes, the others unless the frame is blank-only
    const bool take_blank = act & (blank_only | compete);
    const bool take_other = act & !blank_only;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int y0 = (c * W + g) * 4;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        // bitwise logic on lane masks: no per-token branches
        const int y = y0 + j;
        const bool is_blank = y == blank;
        cd[c][j] = (y < V) & ((is_blank & take_blank) | (!is_blank & take_other));
        kk[c][j] = xv[c][j];
      }
      if (want_keys) {
        uint32_t aw[NL][4], av[NL][4];  // tag and value halves of the arc entries
        float lv[NL][4];                // dense rows
#pragma unroll
        for (int i = 0; i < NL; ++i) {
          const uint4 a01 = *reinterpret_cast<const uint4 *>(arcw + i * Vp + y0);
          const uint4 a23 = *reinterpret_cast<const uint4 *>(arcw + i * Vp + y0 + 2);
          const float4 l4 = *reinterpret_cast<const float4 *>(lmval + (CTX && i == 0 && Dc >= 2 ? NL : i) * Vp + y0);
          aw[i][0] = a01.y; aw[i][1] = a01.w; aw[i][2] = a23.y; aw[i][3] = a23.w;
          av[i][0] = a01.x; av[i][1] = a01.z; av[i][2] = a23.x; av[i][3] = a23.z;
          lv[i][0] = l4.x; lv[i][1] = l4.y; lv[i][2] = l4.z; lv[i][3] = l4.w;
        }
        float eh[4];
        uint32_t hi[4];
        if constexpr (ER) {
          const float4 ev4 = *reinterpret_cast<const float4 *>(erow + y0);
          eh[0] = ev4.x; eh[1] = ev4.y; eh[2] = ev4.z; eh[3] = ev4.w;
        } else {
          // transition + 1 of this frame's phrase entry, 0 if none
          const uint4 p4 = *reinterpret_cast<const uint4 *>(ptag + y0);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const uint32_t pw = j == 0 ? p4.x : j == 1 ? p4.y : j == 2 ? p4.z : p4.w;
            hi[j] = (pw >> 16) == stamp ? (pw & 0xFFFFu) : 0u;
          }
          // the phrase entry values: the LDS copy of the state's first kAux transitions
          // (read for every token, index 0 when unused, so that no per-token branch
          // guards the read), the delta table beyond them only for a state with more
#pragma unroll
          for (int j = 0; j < 4; ++j) eh[j] = sE[min((int)hi[j], kAux)];
          asm volatile("" ::"v"(eh[0]), "v"(eh[1]), "v"(eh[2]), "v"(eh[3]));
          if (dcnt > kAux) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
              if (hi[j] > (uint32_t)kAux) eh[j] = as_float(tr.delta[dbeg + (int)hi[j] - 1].z);
          }
        }
        // per LM, the dense row (the first LM's context row when it has one) plus
        // the backoffs of the levels above it up to m, in increasing order (the
        // levels above m back off by 0)
        float dres[NL][4];
#pragma unroll
        for (int i = 0; i < NL; ++i) {
#pragma unroll
          for (int j = 0; j < 4; ++j) dres[i][j] = lv[i][j];
          const int from = (CTX && i == 0 && Dc >= 2) ? Dc + 1 : 2;
#pragma unroll
          for (int L2 = 2; L2 < kMaxLevels; ++L2) {
            if (L2 > m[i]) break;  // uniform
            if (L2 >= from) {
#pragma unroll
              for (int j = 0; j < 4; ++j) dres[i][j] = dres[i][j] + bo[i][L2];
            }
          }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int y = y0 + j;
          const float x = xv[c][j];
          // the LM terms in model order: u = (x + a_1 lm_1) + a_2 lm_2 ..., each LM
          // its winning arc of this frame if there is one, else its backed-off
          // dense row
          float u = x;
#pragma unroll
          for (int i = 0; i < NL; ++i) {
            const float lmv = (aw[i][j] >> 16) == stamp ? __uint_as_float(av[i][j]) : dres[i][j];
            const float a1 = p.lam[i] * lmv;
            u = u + a1;
          }
          // phrases: the transition's entry value if this state overrides y, else the
          // root's (with no phrase tree both are 0 and so is phi)
          const float e = ER ? eh[j] : (hi[j] ? eh[j] : rE[c][j]);
          const float bst = e - phiq;
          const float a3 = p.beta * ((ER || p.has_trie) ? bst : 0.0f);
          kk[c][j] = (y == blank) ? x : u + a3;
        }
      }
      // this lane's entry values back to the root's for the next frame (read above)
      if (ER) *reinterpret_cast<float4 *>(erow + y0) = make_float4(rE[c][0], rE[c][1], rE[c][2], rE[c][3]);
      if (write_fused && y0 < V) {
        const rsrc_t fr = row_rsrc(args_here().fused + rowoff, V);
        if (AL) {
          row_store4(fr, make_float4(kk[c][0] - lse, kk[c][1] - lse, kk[c][2] - lse, kk[c][3] - lse), voff, c * W * 16);
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j)
            if (y0 + j < V) row_store1(fr, kk[c][j] - lse, voff + 4 * j, c * W * 16);
        }
      }
    }
    // the next frame's logits strip: fetched here, in a compute-bound phase, rather
    // than beside the frame-start loads, whose burst sets the start of the frame.
    // Unconditional (the last frame fetches its own row again): a conditional
    // fetch would make the compiler wait for it where the branches join
    if (t + 1 < p.T) xrow += xstride;
    fetch_logits();
    // ---- the wave's top-k: per round the wave maximum of the remaining keys, then
    // the lowest id holding it (ties to the lowest id).  Keys compete as
    // order-preserving ints; tokens that are not candidates or are already taken
    // hold INT_MIN, below every key including -inf.  The per-round work stays in
    // the vector units (the scalar unit is shared by all the waves of the CU):
    // each lane finds its own first token holding the maximum, the compare mask
    // is the ballot, the winning lane removes its token, and lane r keeps round
    // r's entry until the list is written at the end.
    {
      int sk[NC][4];
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int o = ord_key(kk[c][j]);
          sk[c][j] = cd[c][j] ? o : INT_MIN;
        }
      // With K > 1 the rounds below run only in a wave that holds more than K
      // keys at or above tau, the K-th largest of the NW wave maxima: those
      // maxima are K distinct tokens with keys >= tau, so no key below tau is
      // among the hypothesis' top K.  A wave with at most K such keys writes
      // them straight into its list (any order: the hypothesis' top-k ranks
      // by key, then id).
      bool listed = false;
      if constexpr (KM > 1) {
        int lb = INT_MIN;
#pragma unroll
        for (int c = 0; c < NC; ++c) lb = max(lb, max(max(sk[c][0], sk[c][1]), max(sk[c][2], sk[c][3])));
        const int mw = wave_max_i(lb);
        if (lane == 0) s_wmax[wave] = sel_order(mw, wave);
        lds_barrier();
        int tau = INT_MIN;
        if (NW >= K) {
          // the K-th largest of the NW maxima (counted with multiplicity): lane
          // l < NW ranks maximum l among all of them (ties by wave index) and the
          // lane of rank K-1 holds it
          const unsigned long long mine = s_wmax[lane < NW ? lane : 0];
          int r = 0;
#pragma unroll
          for (int w2 = 0; w2 < NW; ++w2) r += (int)(s_wmax[w2] > mine);
          const unsigned long long at = __ballot(lane < NW && r == K - 1);
          tau = sel_key(__builtin_amdgcn_readlane((int)(mine >> 32), __ffsll((long long)at) - 1));
        }
        // survivors: keys >= tau, never a non-candidate (INT_MIN; every real key,
        // -inf included, maps above it)
        const int thr = max(tau, INT_MIN + 1);
        unsigned long long sb[NC][4];
        int n = 0;
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            sb[c][j] = __ballot(sk[c][j] >= thr);
            n += __popcll(sb[c][j]);
          }
        if (n <= K) {
          int base = 0;
#pragma unroll
          for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              if (sk[c][j] >= thr) {
                const int slot = base + __builtin_amdgcn_mbcnt_hi((uint32_t)(sb[c][j] >> 32),
                                                                  __builtin_amdgcn_mbcnt_lo((uint32_t)sb[c][j], 0u));
                w_key[wave][slot] = sk[c][j];
                w_y[wave][slot] = (c * W + wave * 64 + lane) * 4 + j;
              }
              base += __popcll(sb[c][j]);
            }
          if (lane >= n && lane < K) {
            w_key[wave][lane] = INT_MIN;
            w_y[wave][lane] = INT_MAX;
          }
          listed = true;
        } else {
#pragma unroll
          for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int j = 0; j < 4; ++j) sk[c][j] = sk[c][j] >= thr ? sk[c][j] : INT_MIN;
        }
      }
      int rk = INT_MIN, ry = INT_MAX;  // lane r: entry r of the wave's list
      for (int r = 0; r < (listed ? 0 : K); ++r) {
        int lbc[NC];
        int lb = INT_MIN;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          lbc[c] = max(max(sk[c][0], sk[c][1]), max(sk[c][2], sk[c][3]));
          lb = max(lb, lbc[c]);
        }
        const int M = wave_max_i(lb);
        if (M == INT_MIN) break;
        // lowest strip, then lowest lane, then lowest position holding M
        int src = -1, wc = 0;
#pragma unroll
        for (int c = NC - 1; c >= 0; --c) {
          const unsigned long long has = __ballot(lbc[c] == M);
          if (has) {
            src = __ffsll((long long)has) - 1;
            wc = c;
          }
        }
        int jm = 3;  // this lane's first position holding M in strip wc
#pragma unroll
        for (int c = 0; c < NC; ++c)
          if (c == wc) {
            jm = sk[c][2] == M ? 2 : jm;
            jm = sk[c][1] == M ? 1 : jm;
            jm = sk[c][0] == M ? 0 : jm;
          }
        const int wy = (wc * W + wave * 64 + src) * 4 + __builtin_amdgcn_readlane(jm, src);
        const int kill = lane == src ? wc * 4 + jm : -1;
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
          for (int j = 0; j < 4; ++j) sk[c][j] = kill == c * 4 + j ? INT_MIN : sk[c][j];
        rk = lane == r ? M : rk;
        ry = lane == r ? wy : ry;
      }
      if (!listed && lane < K) {
        w_key[wave][lane] = rk;
        w_y[wave][lane] = ry;
      }
    }
    if (p.traffic && act && g == 0) {
      // the frame's algorithmic bytes: the logits row; per LM the level-1 row and,
      // for every level of the state's chain, its arc list (at most a row) and
      // 12 bytes of record, plus 8 for a chain of two or more levels; the phrase
      // node and its delta list.  Recomputed here from the frame's sources, which
      // the hypothesis state holds until the install, so that the decode keeps
      // no value alive for a count that only the counting launch takes
      const __attribute__((address_space(4))) Params &pk = args_here();
      unsigned long long by = 4ull * V;
      if (ok) {
        const unsigned long long row = 4ull * V;
        const int y = hs.y;
#pragma unroll
        for (int i = 0; i < NL; ++i) {
          const int rs = pk.lm[i].rec_stride;
          by += umin64(8ull * (unsigned long long)pk.lm[i].cnt1[hs.c1[i]], row);
          const int src = hs.lmsrc[i];
          const int32_t *r = src < -1  ? pk.lm[i].ctx_rec + ((int64_t)(-src - 2) * V + y) * rs
                             : src < 0 ? pk.lm[i].rec_dense + ((int64_t)hs.c1p[i] * V + y) * rs
                             : src >= V + 2 ? pk.lm[i].rec + (int64_t)(src - V - 2) * rs
                                            : nullptr;
          const int mi = r ? (r[0] >> 16) : 1;
          for (int L = 2; L < kMaxLevels; ++L)
            if (L <= mi) by += umin64(8ull * (unsigned long long)(unsigned)r[rec_cnt_word(L)], row) + 12ull;
          if (mi >= 2) by += 8ull;
        }
        if (pk.has_trie) {
          const int q = hs.qsrc;
          const int4 nd = q < 0 ? pk.tr.root_node[y] : pk.tr.node[q];
          by += 16ull + 16ull * (unsigned long long)nd.z;
        }
      }
      by += BEAM ? 8ull : 4ull;
      if (p.fused) by += 4ull * V;
      s_bytes += by;
      s_steps += 1ull;
    }
    lds_barrier();
    // the next frame's row statistics, by the waves other than wave 0; the last of
    // them to finish combines them (ahead of the frame's end, off wave 0's path)
    if (NW > 1 && wave != 0 && t + 1 < p.T) {
      row_stats(xraw, wave, V);
      if (wave == 1) row_stats(xraw0, 0, V);
      int done = 0;
      if (lane == 0) done = __hip_atomic_fetch_add(&s_nstat, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_WORKGROUP);
      if (uni(done) == NW - 2) {
        combine_stats();
        if (lane == 0) s_nstat = 0;
      }
    }
    // ---- the hypothesis' top-k (wave 0): the K-entry lists of the NW waves spread
    // over the lanes (entry j of wave w is element e = j*NW + w, lane e % 64, slot
    // e / 64); K rounds of a wave maximum, ties to the lowest id -------------------
    if (wave == 0) {
      constexpr int kSlots = (kMaxWaves * KM + 63) / 64;
      int ek[kSlots], ey[kSlots];
#pragma unroll
      for (int q = 0; q < kSlots; ++q) {
        const int e = q * 64 + lane;
        const int w = e % NW, j = e / NW;
        ey[q] = j < K ? w_y[w][j] : INT_MAX;
        ek[q] = (j < K && ey[q] != INT_MAX) ? w_key[w][j] : INT_MIN;
      }
      // candidate j ends in lane j
      int ck = INT_MIN, cy = INT_MAX;
      bool picked = false;
      if constexpr (kSlots == 1 && KM > 1) {
        // at most 16 listed entries (the usual case after the wave-level
        // narrowing): compact them into LDS, let each count the entries ahead
        // of it (key desc, then id asc) in registers, and place it by that rank
        const bool valid = ek[0] != INT_MIN;
        const unsigned long long vb = __ballot(valid);
        const int n = __popcll(vb);
        if (n <= 16) {
          const int pos = __builtin_amdgcn_mbcnt_hi((uint32_t)(vb >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)vb, 0u));
          // an entry is ahead of another exactly when its composite is larger;
          // padding (0) is never ahead of a listed entry (every key is above INT_MIN)
          if (valid) s_sel[pos] = sel_order(ek[0], ey[0]);
          if (lane >= n && lane < 16) s_sel[lane] = 0ull;
          // one wave: its LDS operations complete in order
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
          unsigned long long cv[16];
#pragma unroll
          for (int q = 0; q < 16; q += 2) {
            const ulonglong2 d = *reinterpret_cast<const ulonglong2 *>(&s_sel[q]);
            cv[q] = d.x;
            cv[q + 1] = d.y;
          }
          const unsigned long long me = s_sel[lane & 15];
          int r = 0;
#pragma unroll
          for (int q = 0; q < 16; ++q) r += (int)(cv[q] > me);
          if (lane < n && r < K) s_win[r] = me;
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
          const int nk = min(n, K);
          const unsigned long long wv = s_win[lane < nk ? lane : 0];
          if (lane < nk) {
            ck = sel_key((int)(wv >> 32));
            cy = (int)~(uint32_t)wv;
          }
          picked = true;
        }
      }
      for (int j = 0; j < (picked ? 0 : K); ++j) {
        int v = ek[0];
#pragma unroll
        for (int q = 1; q < kSlots; ++q) v = max(v, ek[q]);
        const int M = wave_max_i(v);
        if (M == INT_MIN) break;
        int by = INT_MAX, bl = 0, bq = 0;
#pragma unroll
        for (int q = 0; q < kSlots; ++q) {
          for (unsigned long long own = __ballot(ek[q] == M); own; own &= own - 1) {
            const int l = __ffsll((long long)own) - 1;
            const int yl = __builtin_amdgcn_readlane(ey[q], l);
            if (yl < by) {
              by = yl;
              bl = l;
              bq = q;
            }
          }
        }
        if (lane == j) {
          ck = M;
          cy = by;
        }
#pragma unroll
        for (int q = 0; q < kSlots; ++q)
          if (q == bq && lane == bl) ek[q] = INT_MIN;
      }
      // each candidate lane resolves where its next state comes from (see HypState)
      const float cf = cy != INT_MAX ? key_of(ck) - lse : -INFINITY;
      int cl[NL], cq = qid;
#pragma unroll
      for (int i = 0; i < NL; ++i) cl[i] = sid[i];
      if (cy != INT_MAX && cy != blank) {
        // the token's LDS entries of this frame: per LM the winner's level /
        // offset, the phrase transition
#pragma unroll
        for (int i = 0; i < NL; ++i) {
          const uint32_t aw = (uint32_t)(arcw[i * Vp + cy] >> 32);
          const uint32_t lo = (aw >> 16) == stamp ? (aw & 0xFFFFu) : 0u;
          // -1: the state after (c_1, y) (rec_dense); -(r + 2): the state after
          // (context of row r, y) (ctx_rec)
          cl[i] = (CTX && i == 0 && Dc >= 2) ? -(crow + 2) : -1;
          if (lo) {
            const int L = (int)(lo >> 13), jj = (int)(lo & 0x1FFFu), N = Nl[i];
            const int bL = s_lbeg[i][L];
            cl[i] = L < N - 1 ? (int)(s_sbase[i][L] + bL + jj)
                              : (jj < kAux ? sTN[i * kAux + jj] : lms[i].top_next[bL + jj - lms[i].arc_base[N - 1]]);
          }
        }
        const uint32_t pw = ptag[cy];
        const uint32_t hi = (pw >> 16) == stamp ? (pw & 0xFFFFu) : 0u;
        cq = -1;
        if (hi) {
          // LDS copy for the first kAux transitions, the table beyond; the table is
          // read through a global-space pointer so the two loads stay distinct
          // (a merged load would take the slower generic-address path)
          const int4 __attribute__((address_space(1))) *gdelta =
              (const int4 __attribute__((address_space(1))) *)tr.delta;
          cq = (int)hi - 1 < kAux ? sDT[hi - 1] : gdelta[dbeg + (int)hi - 1].y;
        }
        if (!p.has_trie) cq = 0;
      }
      if (MODE == kModeStep) {
        if (lane < K) {
          const int64_t o = (int64_t)h * K + lane;
          if (cy == INT_MAX) {
            p.tokens[o] = -1;
            p.scores[o] = -INFINITY;
#pragma unroll
            for (int i = 0; i < NL; ++i) p.next_lm[(int64_t)i * H * K + o] = hs.cur_lm[i];  // [n_lm][H][k]
            p.next_boost[o] = hs.cur_q;
          } else {
            int q = cq;
#pragma unroll
            for (int i = 0; i < NL; ++i) {
              int l = cl[i];
              if (!inv && l < -1) l = lms[i].ctx_rec[((int64_t)(-l - 2) * V + cy) * RSl[i] + 1];
              else if (!inv && l < 0) l = lms[i].rec_dense[((int64_t)hs.c1[i] * V + cy) * RSl[i] + 1];
              p.next_lm[(int64_t)i * H * K + o] = l;
            }
            if (!inv && q < 0) q = tr.root_node[cy].w;
            p.tokens[o] = cy;
            p.scores[o] = cf;
            p.next_boost[o] = q;
          }
        }
      } else if (MODE == kModeGreedy) {
        if (lane == 0) {
          p.tokens[(int64_t)t * H + h] = cy;
#pragma unroll
          for (int i = 0; i < NL; ++i) {
            const int c1p = hs.c1[i];
            hs.lmsrc[i] = cl[i];
            hs.c1p[i] = c1p;
            hs.c1[i] = cy != blank ? cy : c1p;
          }
          hs.qsrc = cq;
          hs.y = cy;
        }
      } else {
        // ---- beam: publish this hypothesis' candidates, meet the stream, rank all ----
        // A candidate record is XW = 4 + NL 64-bit words, each carrying the frame
        // tag in its top 16 bits over 48 bits of payload: the total score S_b +
        // fused (fp64), the first LM's and the phrase source, the token, the
        // parent's c_1 (first LM) and flags, for a second LM its source and the
        // parent's c_1, and (recombination only) the hash of the history the
        // candidate reaches.  Words are written and read as relaxed agent-scope
        // atomics, so a reader that sees the current tag in all words holds the
        // whole record: polling the records is the rendezvous (no counter, no
        // fence).  Frames alternate between two buffers; a writer can be at most
        // one frame ahead of any reader of its stream, so it never overwrites a
        // buffer that is still being read.
        constexpr int XW = 3 + NL + (RC ? 1 : 0);
        // tags run 1..65535 over the global frame index (0 marks a cleared record);
        // a record left in a buffer is from two frames back, so never current
        const int tg = p.t_base + t;
        unsigned long long *xs = p.xchg + ((size_t)sl * 2 + (tg & 1)) * (size_t)B * K * XW;
        const unsigned long long tag = (unsigned long long)(tg % 65535 + 1) << 48;
        constexpr unsigned long long kPay = (1ull << 48) - 1;
        if (lane < K) {
          const bool has = act && cy != INT_MAX;
          const double tot = has ? hs.S + (double)cf : -INFINITY;
          const unsigned long long tb = (unsigned long long)__double_as_longlong(tot);
          unsigned long long w[XW];
          w[0] = (tb & kPay) | tag;
          w[1] = (tb >> 48) | ((unsigned long long)(unsigned)cl[0] << 16) | tag;
          w[2] = (unsigned long long)(unsigned)cq | ((unsigned long long)(has ? cy + 1 : 0) << 32) | tag;
          w[3] = (unsigned long long)((hs.c1[0] + 1) & 0xFFFF) | ((unsigned long long)(hs.fl & 0xFF) << 16) | tag;
          if constexpr (NL > 1)
            w[4] = (unsigned long long)(unsigned)cl[1] | ((unsigned long long)((hs.c1[1] + 1) & 0xFFFF) << 32) | tag;
          if constexpr (RC) {
            // the history after the candidate: blank emits nothing (a hash is
            // never 0, which marks the start of a stream in the carried buffer)
            const unsigned long long hist = hs.hist;
            const unsigned long long hn = mix64(hist ^ (0x632BE59BD9B4E019ull * (unsigned long long)(cy + 1))) & kPay;
            w[XW - 1] = ((!has || cy == blank) ? hist : (hn ? hn : 1ull)) | tag;
          }
#pragma unroll
          for (int q = 0; q < XW; ++q)
            __hip_atomic_store(xs + (b * K + lane) * XW + q, w[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        // every workgroup of the stream ranks the same B*k candidates by (total
        // desc, parent asc, rank asc), i.e. candidate order breaks ties; slot b
        // takes rank b.  The totals are staged in LDS (NaN: no candidate, never
        // ahead of anything) and each lane counts the candidates ahead of its own.
        const int nc = B * K;
        for (int i0 = 0; i0 < nc; i0 += 64) {
          const int i = i0 + lane;
          unsigned long long w[XW];
#pragma unroll
          for (int q = 0; q < XW; ++q) w[q] = 0ull;
          bool cur = i >= nc;
          for (int spins = 0;; ++spins) {
            if (i < nc) {
#pragma unroll
              for (int q = 0; q < XW; ++q) w[q] = __hip_atomic_load(xs + i * XW + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              cur = true;
#pragma unroll
              for (int q = 0; q < XW; ++q) cur = cur && (w[q] & ~kPay) == tag;
            }
            if (__ballot(!cur) == 0ull || aborted) break;
            if (spins >= kSpinLimit) {
              if (lane == 0) atomicOr(&g_status, FUSION_STATUS_SYNC_TIMEOUT);
              aborted = true;
              break;
            }
          }
          if (i < nc) {
            const int y1 = (int)((w[2] >> 32) & 0xFFFF);
            const bool valid = cur && y1 != 0;
            s_xa[i] = make_int4(y1 - 1, (int)(unsigned)((w[1] >> 16) & 0xFFFFFFFFull), (int)(unsigned)(w[2] & 0xFFFFFFFFull),
                                (int)(w[3] & 0xFFFF) - 1);
            s_xf[i] = (int)((w[3] >> 16) & 0xFF);
            if constexpr (NL > 1)
              s_xb[i] = make_int2((int)(unsigned)(w[4] & 0xFFFFFFFFull), (int)((w[4] >> 32) & 0xFFFF) - 1);
            if constexpr (RC) s_hh[i] = w[XW - 1] & kPay;
            s_tot[i] = valid ? __longlong_as_double((long long)((w[0] & kPay) | ((w[1] & 0xFFFF) << 48)))
                             : __longlong_as_double(0x7FF8000000000000ll);
          } else if (i < 16) {
            s_tot[i] = __longlong_as_double(0x7FF8000000000000ll);  // unused: never ahead
          }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        if constexpr (RC) {
          // recombination: candidates that reach the same history (equal hash)
          // merge into the first of them in candidate order, with the log-sum
          // of their totals folded in that order; the others leave the ranking
          if (nc <= 64) {
            // one candidate per lane, every other candidate's total and hash
            // read from its lane (readlane), not from LDS
            const double ti = lane < nc ? s_tot[lane] : __longlong_as_double(0x7FF8000000000000ll);
            const unsigned long long hi = lane < nc ? s_hh[lane] : 0ull;
            const long long tb = __double_as_longlong(ti);
            int first = -1;
            double acc = 0.0;
            for (int j = 0; j < nc; ++j) {
              const double tj = __longlong_as_double(
                  ((long long)(unsigned)__builtin_amdgcn_readlane((int)(tb >> 32), j) << 32) |
                  (long long)(unsigned)__builtin_amdgcn_readlane((int)tb, j));
              const unsigned long long hj =
                  ((unsigned long long)(unsigned)__builtin_amdgcn_readlane((int)(hi >> 32), j) << 32) |
                  (unsigned long long)(unsigned)__builtin_amdgcn_readlane((int)hi, j);
              if (ti == ti && tj == tj && hj == hi) {
                if (first < 0) {
                  first = j;
                  acc = tj;
                } else {
                  acc = log_add(acc, tj);
                }
              }
            }
            // every lane has read its own entry before any lane writes
            if (lane < nc) s_tot[lane] = (ti == ti && first == lane) ? acc : __longlong_as_double(0x7FF8000000000000ll);
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
          } else {
#pragma unroll 1
            for (int i = lane; i < nc; i += 64) {
              double m = __longlong_as_double(0x7FF8000000000000ll);
              const double ti = s_tot[i];
              if (ti == ti) {
                const unsigned long long hi = s_hh[i];
                int first = -1;
                double acc = 0.0;
#pragma unroll 1
                for (int j = 0; j < nc; ++j) {
                  const double tj = s_tot[j];
                  if (tj == tj && s_hh[j] == hi) {
                    if (first < 0) {
                      first = j;
                      acc = tj;
                    } else {
                      acc = log_add(acc, tj);
                    }
                  }
                }
                if (first == i) m = acc;
              }
              s_mt[i] = m;
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
#pragma unroll 1
            for (int i = lane; i < nc; i += 64) s_tot[i] = s_mt[i];
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
          }
        }
        int wi = -1;
        bool ranked = false;
        if (nc <= 16) {
          // up to 16 candidates (B * k <= 16; entries nc..15 hold NaN): every
          // lane loads all totals at once (eight 16-byte reads) and counts
          // those ahead of its own in registers; equal totals need the
          // candidate-order rule and take the general count below
          double tv[16];
#pragma unroll
          for (int q = 0; q < 16; q += 2) {
            const double2 d = *reinterpret_cast<const double2 *>(&s_tot[q]);
            tv[q] = d.x;
            tv[q + 1] = d.y;
          }
          const double ti = s_tot[lane & 15];
          int gt = 0, eq = 0;
#pragma unroll
          for (int q = 0; q < 16; ++q) {
            gt += (int)(tv[q] > ti);
            eq += (int)(tv[q] == ti);
          }
          const bool live = lane < nc && ti == ti;
          if (__ballot(live && eq > 1) == 0ull) {
            if (live && gt == b) wi = lane;
            ranked = true;
          }
        }
        for (int i = (ranked ? 64 : 0) + lane; i < nc; i += 64) {
          const double ti = s_tot[i];
          if (ti == ti) {
            int r = 0;
#pragma unroll 16
            for (int j = 0; j < nc; ++j) {
              const double tj = s_tot[j];
              r += (tj > ti || (tj == ti && j < i)) ? 1 : 0;
            }
            if (r == b) wi = i;
          }
        }
        const int64_t o = (int64_t)t * H + h;
        if (wi >= 0) {
          // the lane holding the slot's candidate installs it
          const int4 a = s_xa[wi];
          const int xf = s_xf[wi];
          const double tot = s_tot[wi];
          int2 xb = make_int2(0, 0);
          if constexpr (NL > 1) xb = s_xb[wi];
          const int y = a.x;
          int src[NL], c1p[NL];
          src[0] = a.y;
          c1p[0] = a.w;
          if constexpr (NL > 1) {
            src[1] = xb.x;
            c1p[1] = xb.y;
          }
#pragma unroll
          for (int i = 0; i < NL; ++i) {
            hs.lmsrc[i] = src[i];
            hs.c1p[i] = c1p[i];
            hs.c1[i] = y != blank ? y : c1p[i];
          }
          hs.qsrc = a.z;
          hs.y = y;
          hs.fl = 1 | (xf & 2);
          if constexpr (RC) hs.hist = s_hh[wi];
          hs.S = tot;
          p.tokens[o] = y;
          p.parents[o] = wi / K;
        }
        if (__ballot(wi >= 0) == 0ull && lane == 0) {
          // no candidate reaches this slot: the hypothesis is dead and keeps its state
#pragma unroll
          for (int i = 0; i < NL; ++i) {
            hs.lmsrc[i] = hs.cur_lm[i];
            hs.c1p[i] = -1;
          }
          hs.qsrc = hs.cur_q;
          hs.y = -1;
          hs.fl = 0;
          hs.S = -INFINITY;
          p.tokens[o] = -1;
          p.parents[o] = -1;
        }
      }
    }
    lds_barrier();
  }
  // ---- final state ----------------------------------------------------------------
  if (MODE != kModeStep && g == 0) {
    const int V = p.V;
    int nq = hs.qsrc;
    const int y = hs.y;
    // a negative source means "reached by token y" only for valid hypotheses
    // that made a transition; an invalid hypothesis keeps its raw ids
    const bool moved = (hs.fl & 2) == 0 && y >= 0 && y != p.blank;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      int nl = hs.lmsrc[i];
      if (moved && nl < -1) nl = lms[i].ctx_rec[((int64_t)(-nl - 2) * V + y) * RSl[i] + 1];
      else if (moved && nl < 0) nl = lms[i].rec_dense[((int64_t)hs.c1p[i] * V + y) * RSl[i] + 1];
      p.lm_state[(int64_t)i * H + h] = nl;
    }
    if (moved && nq < 0) nq = tr.root_node[y].w;
    if (p.has_trie) p.boost_state[h] = nq;
    if (BEAM) p.hyp_score[h] = hs.S;
    if constexpr (RC) {
      if (p.hist) p.hist[h] = hs.hist;
    }
  }
  if (p.traffic && g == 0) {
    const unsigned long long extra = (h == 0 && p.has_trie) ? 4ull * p.V * (unsigned long long)p.T : 0ull;
    atomicAdd(reinterpret_cast<unsigned long long *>(p.traffic), s_bytes + extra);
    atomicAdd(reinterpret_cast<unsigned long long *>(p.traffic) + 1, s_steps);
  }
}

__global__ void zero_ints(int *p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

// ---------------------------------------------------------------------------
// launch
// ---------------------------------------------------------------------------
typedef void (*KernelFn)(Params);

template <int W, int NC, int KM, bool AL, int NL>
KernelFn pick_mode(int mode) {
  if constexpr (KM == 1) {
    if (mode == kModeGreedy) return fusion_kernel<W, NC, KM, AL, kModeGreedy, NL>;
  }
  if (mode == kModeBeamRC) return fusion_kernel<W, NC, KM, AL, kModeBeamRC, NL>;
  return mode == kModeStep ? fusion_kernel<W, NC, KM, AL, kModeStep, NL> : fusion_kernel<W, NC, KM, AL, kModeBeam, NL>;
}
template <int W, int NC, int KM, int NL>
KernelFn pick_al(bool al, int mode) {
  return al ? pick_mode<W, NC, KM, true, NL>(mode) : pick_mode<W, NC, KM, false, NL>(mode);
}
template <int W, int NC, int NL>
KernelFn pick_k(int km, bool al, int mode) {
  return km == 1 ? pick_al<W, NC, 1, NL>(al, mode) : km == 4 ? pick_al<W, NC, 4, NL>(al, mode) : pick_al<W, NC, 8, NL>(al, mode);
}

struct Shape {
  int W, NC, Vp;
};

// lanes per hypothesis and 4-token strips per lane for a vocabulary
Shape shape_for(int V) {
  if (V <= 256) return {64, 1, 256};
  if (V <= 1024) return {256, 1, 1024};
  if (V <= 4096) return {1024, 1, 4096};
  return {1024, 2, 8192};
}

// two LMs are compiled for vocabularies up to 4096 (two LMs at 8192 need more
// LDS than a workgroup has)
KernelFn pick(const Shape &sh, int km, bool al, int mode, int n_lm) {
  if (n_lm == 2) {
    if (sh.W == 64) return pick_k<64, 1, 2>(km, al, mode);
    if (sh.W == 256) return pick_k<256, 1, 2>(km, al, mode);
    if (sh.NC == 1) return pick_k<1024, 1, 2>(km, al, mode);
    return nullptr;
  }
  if (sh.W == 64) return pick_k<64, 1, 1>(km, al, mode);
  if (sh.W == 256) return pick_k<256, 1, 1>(km, al, mode);
  if (sh.NC == 1) return pick_k<1024, 1, 1>(km, al, mode);
  return pick_k<1024, 2, 1>(km, al, mode);
}

// dynamic LDS of a launch: per LM the dense row and the arc entries, the first
// LM's context row (rows of at most 4096 tokens), the phrase entries, with one LM
// the phrase entry values (rows of at most 4096 tokens), the phrase side tables
// and per LM the top-level next states
size_t dyn_lds_bytes(int Vp, int n_lm) {
  return (size_t)Vp * (12 * n_lm + 4 + (Vp <= 4096 ? 4 : 0) + (n_lm == 1 && Vp <= 4096 ? 4 : 0)) +
         (size_t)4 * (kAux * (2 + n_lm) + 4);
}

struct DeviceInfo {
  int lds_per_block = 0, cus = 0;
  bool ok = false;
};

DeviceInfo device_info() {
  static std::mutex mu;
  static DeviceInfo cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return {};
  std::lock_guard<std::mutex> lk(mu);
  if (!cache[dev].ok) {
    int v = 0, c = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) return {};
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return {};
    cache[dev].lds_per_block = v;
    cache[dev].cus = c;
    cache[dev].ok = true;
  }
  return cache[dev];
}

// The device address of this GPU's static scratch array, looked up once per
// device (with that device current) and kept; nullptr after a failed lookup.
int static_scratch(unsigned long long **out) {
  static std::mutex mu;
  static unsigned long long *ptr[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_error(e, "hipGetDevice");
  if (dev < 0 || dev >= 64) return set_error(FUSION_E_UNSUPPORTED, "device index beyond 63");
  std::lock_guard<std::mutex> lk(mu);
  if (!ptr[dev]) {
    void *a = nullptr;
    e = hipGetSymbolAddress(&a, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_error(e, "hipGetSymbolAddress(scratch)");
    ptr[dev] = reinterpret_cast<unsigned long long *>(a);
  }
  *out = ptr[dev];
  return FUSION_OK;
}

// Per device and kernel: its static LDS, resident workgroups per CU at the
// launch's dynamic LDS, and whether that dynamic LDS has been granted; looked up
// once (the dynamic LDS of a kernel is fixed by its template shape)
struct KernelInfo {
  const void *fn = nullptr;
  int dev = -1;
  size_t static_lds = 0;
  int per_cu = 0;
};

int kernel_info(KernelFn fn, int W, size_t dyn, int lds_per_block, KernelInfo *out) {
  static std::mutex mu;
  static std::vector<KernelInfo> cache;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_error(e, "hipGetDevice");
  const void *f = reinterpret_cast<const void *>(fn);
  std::lock_guard<std::mutex> lk(mu);
  for (const KernelInfo &ki : cache)
    if (ki.fn == f && ki.dev == dev) {
      *out = ki;
      return FUSION_OK;
    }
  KernelInfo ki;
  ki.fn = f;
  ki.dev = dev;
  hipFuncAttributes attr;
  e = hipFuncGetAttributes(&attr, f);
  if (e != hipSuccess) return hip_error(e, "hipFuncGetAttributes");
  ki.static_lds = attr.sharedSizeBytes;
  if (dyn + ki.static_lds > (size_t)lds_per_block)
    return set_error(FUSION_E_UNSUPPORTED, "vocabulary too large for the device's LDS");
  e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
  if (e != hipSuccess) return hip_error(e, "hipFuncSetAttribute");
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&ki.per_cu, f, W, dyn);
  if (e != hipSuccess) return hip_error(e, "hipOccupancyMaxActiveBlocksPerMultiprocessor");
  cache.push_back(ki);
  *out = ki;
  return FUSION_OK;
}

// fixed: caller-provided exchange memory of fixed_words 64-bit words (no
// allocation); nullptr: the exchange is allocated stream-ordered per call.
// keep_exchange: the call continues a frame loop whose earlier calls used the
// same exchange with p.t_base counting their frames, so its records need no
// reset (only when one launch holds every stream; otherwise it is reset anyway)
int launch(Params &p, int n_hyp, hipStream_t stream, unsigned long long *fixed = nullptr, size_t fixed_words = 0,
           bool keep_exchange = false) {
  const Shape sh = shape_for(p.V);
  const int km = p.k <= 1 ? 1 : p.k <= 4 ? 4 : 8;
  const bool al = (p.V % 4 == 0) && ((uintptr_t)p.logits % 16 == 0) && (!p.fused || (uintptr_t)p.fused % 16 == 0);
  const int mode = p.step_mode ? kModeStep : p.B == 1 ? kModeGreedy : p.recombine ? kModeBeamRC : kModeBeam;
  KernelFn fn = pick(sh, km, al, mode, p.n_lm);
  if (!fn) return set_error(FUSION_E_UNSUPPORTED, "two LMs need V <= 4096");
  const DeviceInfo di = device_info();
  if (!di.ok) return set_error(FUSION_E_HIP, "cannot query the device");
  const size_t dyn = dyn_lds_bytes(sh.Vp, p.n_lm);
  KernelInfo ki;
  int rc0 = kernel_info(fn, sh.W, dyn, di.lds_per_block, &ki);
  if (rc0 != FUSION_OK) return rc0;
  hipError_t e = hipSuccess;
  p.s_off = 0;
  p.xcd_map = 0;
  if (p.B == 1 || p.step_mode) {
    hipLaunchKernelGGL(fn, dim3(n_hyp), dim3(sh.W), dyn, stream, p);
    e = hipGetLastError();
    return e == hipSuccess ? FUSION_OK : hip_error(e, "fusion kernel launch");
  }
  // beam: a stream's workgroups meet every frame.  They take their slots from
  // arrival counters (see the kernel), which keeps a launch free of deadlock
  // even when other work holds part of the device, provided the incomplete
  // streams (one per blockIdx class, at most 8 x (B - 1) workgroups) cannot
  // fill it.  A launch holds no more streams than fit at once, so that no
  // workgroup waits at a rendezvous for a sibling that has yet to start behind
  // whole streams (the wait is bounded); further streams run in further launches
  const long resident = (long)ki.per_cu * di.cus;
  if (resident <= 8L * (p.B - 1)) return set_error(FUSION_E_UNSUPPORTED, "a beam does not fit on the device");
  // exchange records: 2 buffers x B x k candidates x (3 + n_lm (+1 recombining)) words per
  // stream, then the 8 arrival counters (4 words)
  const size_t stream_words = (size_t)2 * p.B * p.k * (3 + p.n_lm + (p.recombine ? 1 : 0));
  constexpr size_t kTicketWords = 4;
  int s_batch = (int)std::min<long>(p.S, resident / p.B);
  if (fixed) {
    if (stream_words + kTicketWords > fixed_words)
      return set_error(FUSION_E_UNSUPPORTED, "one stream's beam exchange exceeds the static scratch");
    s_batch = (int)std::min<size_t>((size_t)s_batch, (fixed_words - kTicketWords) / stream_words);
  }
  if (s_batch >= 8) s_batch -= s_batch % 8;
  const size_t xwords = (size_t)s_batch * stream_words + kTicketWords;
  void *xbuf = fixed;
  if (!fixed) {
    e = hipMallocAsync(&xbuf, xwords * sizeof(unsigned long long), stream);
    if (e != hipSuccess) return hip_error(e, "hipMallocAsync");
  }
  p.xchg = reinterpret_cast<unsigned long long *>(xbuf);
  p.tickets = reinterpret_cast<unsigned *>(p.xchg + (size_t)s_batch * stream_words);
  int rc = FUSION_OK;
  for (int s0 = 0; s0 < p.S && rc == FUSION_OK; s0 += s_batch) {
    const int ns = std::min(s_batch, p.S - s0);
    // tag 0 (no frame uses it) everywhere and the counters at 0, so that neither
    // uninitialised memory nor an earlier batch's records can pass for the
    // current frame's (a frame loop that keeps the exchange relies on its
    // global frame numbers and on the counters resetting themselves)
    if (!(keep_exchange && s_batch >= p.S)) {
      const int n_ints = (int)(xwords * 2);
      hipLaunchKernelGGL(zero_ints, dim3(std::min(64, (n_ints + 255) / 256)), dim3(256), 0, stream,
                         reinterpret_cast<int *>(xbuf), n_ints);
      e = hipGetLastError();
      if (e != hipSuccess) {
        rc = hip_error(e, "exchange reset launch");
        break;
      }
    }
    Params q = p;
    q.s_off = s0;
    q.xcd_map = (ns % 8 == 0) ? 1 : 0;
    hipLaunchKernelGGL(fn, dim3(ns * p.B), dim3(sh.W), dyn, stream, q);
    e = hipGetLastError();
    if (e != hipSuccess) rc = hip_error(e, "fusion kernel launch");
  }
  if (!fixed) {
    hipError_t e2 = hipFreeAsync(xbuf, stream);
    if (rc == FUSION_OK && e2 != hipSuccess) rc = hip_error(e2, "hipFreeAsync");
  }
  return rc;
}

int check_common(const NgramTables *const *lms, const float *alphas, int32_t n_lm, const BoostTrie *trie,
                 const float *logits, int32_t V, int32_t k, int32_t blank_id, int32_t blank_mode, float beta,
                 bool need_logits = true) {
  if (n_lm < 1 || n_lm > FUSION_MAX_LMS) return set_error(FUSION_E_ARG, "n_lm out of range");
  if (!lms || !alphas) return set_error(FUSION_E_ARG, "NULL LM list or weights");
  for (int i = 0; i < n_lm; ++i) {
    if (!lms[i]) return set_error(FUSION_E_ARG, "NULL n-gram tables");
    if (V != lms[i]->dev.V) return set_error(FUSION_E_ARG, "V does not match the n-gram tables");
    if (blank_id != lms[i]->dev.blank) return set_error(FUSION_E_ARG, "blank_id does not match the n-gram tables");
    if (!std::isfinite(alphas[i])) return set_error(FUSION_E_ARG, "non-finite fusion weight");
  }
  if (need_logits && !logits) return set_error(FUSION_E_ARG, "NULL logits");
  if (trie && (trie->dev.V != V || trie->dev.blank != blank_id))
    return set_error(FUSION_E_ARG, "phrase tree built for another vocabulary or blank");
  if (k < 1 || k > FUSION_MAX_K || k > V) return set_error(FUSION_E_ARG, "k out of range");
  if (blank_mode != FUSION_BLANK_AM && blank_mode != FUSION_BLANK_COMPETE) return set_error(FUSION_E_ARG, "unknown blank_mode");
  if (blank_mode == FUSION_BLANK_AM && k != 1) return set_error(FUSION_E_ARG, "FUSION_BLANK_AM needs k == 1");
  if (!std::isfinite(beta)) return set_error(FUSION_E_ARG, "non-finite fusion weight");
  return FUSION_OK;
}

Params make_params(const NgramTables *const *lms, const float *alphas, int32_t n_lm, const BoostTrie *trie) {
  Params p;
  std::memset(&p, 0, sizeof p);
  for (int i = 0; i < n_lm; ++i) {
    p.lm[i] = lms[i]->dev;
    p.lam[i] = alphas[i];
  }
  p.n_lm = n_lm;
  if (trie) p.tr = trie->dev;
  p.has_trie = trie != nullptr;
  return p;
}

int step_impl(const NgramTables *const *lms, const float *alphas, int32_t n_lm, const BoostTrie *trie,
              const float *logits, const int32_t *lm_state, const int32_t *boost_state, int32_t H, int32_t V,
              float beta, int32_t blank_id, int32_t k, int32_t blank_mode, float *fused, int32_t *tokens,
              float *scores, int32_t *next_lm, int32_t *next_boost, hipStream_t stream) {
  int rc = check_common(lms, alphas, n_lm, trie, logits, V, k, blank_id, blank_mode, beta, H != 0);
  if (rc != FUSION_OK) return rc;
  if (H < 0 || H > (1 << 24)) return set_error(FUSION_E_ARG, "H out of range");
  if (H == 0) return FUSION_OK;  // no hypotheses: no buffer is read or written
  if (!lm_state || !tokens || !scores || !next_lm || !next_boost || (trie && !boost_state))
    return set_error(FUSION_E_ARG, "NULL state or output buffer");
  Params p = make_params(lms, alphas, n_lm, trie);
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
  p.beta = beta;
  return launch(p, H, stream);
}

int run_impl(const NgramTables *const *lms, const float *alphas, int32_t n_lm, const BoostTrie *trie,
             const float *logits, int32_t T, int32_t S, int32_t B, int32_t V, int32_t k, float beta,
             int32_t blank_id, int32_t blank_mode, int32_t *lm_state, int32_t *boost_state, double *hyp_score,
             int32_t *tokens, int32_t *parents, float *fused, int64_t *traffic, int32_t flags, uint64_t *hist,
             hipStream_t stream, bool no_alloc = false, unsigned long long *xbuf = nullptr, size_t xbuf_words = 0,
             int32_t t_base = 0) {
  int rc = check_common(lms, alphas, n_lm, trie, logits, V, k, blank_id, blank_mode, beta, T != 0 && S != 0);
  if (rc != FUSION_OK) return rc;
  if (T < 0 || S < 0 || B < 1 || B > FUSION_MAX_BEAM) return set_error(FUSION_E_ARG, "T, S or B out of range");
  if ((int64_t)S * B > (1 << 24)) return set_error(FUSION_E_ARG, "too many hypotheses");
  if (B == 1 && k != 1) return set_error(FUSION_E_ARG, "greedy decoding (B == 1) needs k == 1");
  if (B > 1 && blank_mode != FUSION_BLANK_COMPETE) return set_error(FUSION_E_ARG, "beam decoding needs FUSION_BLANK_COMPETE");
  if (flags & ~FUSION_RUN_RECOMBINE) return set_error(FUSION_E_ARG, "unknown flags");
  if (T == 0 || S == 0) return FUSION_OK;  // nothing to decode: no buffer is read or written
  if (!lm_state || !tokens || (trie && !boost_state)) return set_error(FUSION_E_ARG, "NULL state or output buffer");
  if (B > 1 && (!hyp_score || !parents)) return set_error(FUSION_E_ARG, "beam decoding needs hyp_score and parents");
  Params p = make_params(lms, alphas, n_lm, trie);
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
  p.beta = beta;
  p.recombine = (flags & FUSION_RUN_RECOMBINE) && B > 1;
  p.hist = p.recombine ? reinterpret_cast<unsigned long long *>(hist) : nullptr;
  p.t_base = t_base;
  if (xbuf) return launch(p, S * B, stream, xbuf, xbuf_words, t_base > 0);
  if (no_alloc) {
    unsigned long long *xs = nullptr;
    rc = static_scratch(&xs);
    if (rc != FUSION_OK) return rc;
    return launch(p, S * B, stream, xs, kStaticScratchBytes / sizeof(unsigned long long));
  }
  return launch(p, S * B, stream);
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
  int32_t end_bits = 0;
  const int rc = end_status_take(&end_bits);
  if (rc != FUSION_OK) return rc;
  *code = v | end_bits;
  return FUSION_OK;
}

extern "C" int fusion_step(const NgramTables *lm, const BoostTrie *trie, const float *logits,
                           const int32_t *lm_state, const int32_t *boost_state, int32_t H, int32_t V,
                           float lambda, float beta, int32_t blank_id, int32_t k, int32_t blank_mode,
                           float *fused, int32_t *tokens, float *scores, int32_t *next_lm,
                           int32_t *next_boost, hipStream_t stream) {
  return step_impl(&lm, &lambda, 1, trie, logits, lm_state, boost_state, H, V, beta, blank_id, k, blank_mode,
                   fused, tokens, scores, next_lm, next_boost, stream);
}

extern "C" int fusion_step_lms(const NgramTables *const *lms, const float *alphas, int32_t n_lm,
                               const BoostTrie *trie, const float *logits, const int32_t *lm_state,
                               const int32_t *boost_state, int32_t H, int32_t V, float beta, int32_t blank_id,
                               int32_t k, int32_t blank_mode, float *fused, int32_t *tokens, float *scores,
                               int32_t *next_lm, int32_t *next_boost, hipStream_t stream) {
  return step_impl(lms, alphas, n_lm, trie, logits, lm_state, boost_state, H, V, beta, blank_id, k, blank_mode,
                   fused, tokens, scores, next_lm, next_boost, stream);
}

extern "C" int fusion_run(const NgramTables *lm, const BoostTrie *trie, const float *logits, int32_t T,
                          int32_t S, int32_t B, int32_t V, int32_t k, float lambda, float beta,
                          int32_t blank_id, int32_t blank_mode, int32_t *lm_state, int32_t *boost_state,
                          double *hyp_score, int32_t *tokens, int32_t *parents, float *fused,
                          int64_t *traffic, hipStream_t stream) {
  return run_impl(&lm, &lambda, 1, trie, logits, T, S, B, V, k, beta, blank_id, blank_mode, lm_state,
                  boost_state, hyp_score, tokens, parents, fused, traffic, 0, nullptr, stream);
}

extern "C" int fusion_run_lms(const NgramTables *const *lms, const float *alphas, int32_t n_lm,
                              const BoostTrie *trie, const float *logits, int32_t T, int32_t S, int32_t B,
                              int32_t V, int32_t k, float beta, int32_t blank_id, int32_t blank_mode,
                              int32_t *lm_state, int32_t *boost_state, double *hyp_score, int32_t *tokens,
                              int32_t *parents, float *fused, int64_t *traffic, int32_t flags,
                              uint64_t *hist, hipStream_t stream) {
  return run_impl(lms, alphas, n_lm, trie, logits, T, S, B, V, k, beta, blank_id, blank_mode, lm_state,
                  boost_state, hyp_score, tokens, parents, fused, traffic, flags, hist, stream);
}

extern "C" int fusion_run_lms_noalloc(const NgramTables *const *lms, const float *alphas, int32_t n_lm,
                                      const BoostTrie *trie, const float *logits, int32_t T, int32_t S,
                                      int32_t B, int32_t V, int32_t k, float beta, int32_t blank_id,
                                      int32_t blank_mode, int32_t *lm_state, int32_t *boost_state,
                                      double *hyp_score, int32_t *tokens, int32_t *parents, float *fused,
                                      int64_t *traffic, int32_t flags, uint64_t *hist, hipStream_t stream) {
  return run_impl(lms, alphas, n_lm, trie, logits, T, S, B, V, k, beta, blank_id, blank_mode, lm_state,
                  boost_state, hyp_score, tokens, parents, fused, traffic, flags, hist, stream, true);
}

extern "C" int fusion_run_projected(const NgramTables *const *lms, const float *alphas, int32_t n_lm,
                                    const BoostTrie *trie, const uint16_t *A, const uint16_t *W, const float *bias,
                                    int32_t K, float *logits, int32_t chunk, int32_t T, int32_t S, int32_t B,
                                    int32_t V, int32_t k,
                                    float beta, int32_t blank_id, int32_t blank_mode, int32_t *lm_state,
                                    int32_t *boost_state, double *hyp_score, int32_t *tokens, int32_t *parents,
                                    int32_t flags, uint64_t *hist, hipStream_t stream) {
  int rc = check_common(lms, alphas, n_lm, trie, nullptr, V, k, blank_id, blank_mode, beta, false);
  if (rc != FUSION_OK) return rc;
  if (T < 0 || S < 0 || B < 1 || B > FUSION_MAX_BEAM) return set_error(FUSION_E_ARG, "T, S or B out of range");
  if ((int64_t)S * B > (1 << 24)) return set_error(FUSION_E_ARG, "too many hypotheses");
  if (chunk < 1) return set_error(FUSION_E_ARG, "chunk must be at least 1");
  if (T == 0 || S == 0) return FUSION_OK;
  if (!A || !W || !logits) return set_error(FUSION_E_ARG, "NULL joint states, weight or logits workspace");
  const int64_t H = (int64_t)S * B;
  const int32_t C = std::min(chunk, T);
  if ((int64_t)C * H > INT32_MAX) return set_error(FUSION_E_ARG, "chunk * H exceeds the projection's row count");
  // the beam's exchange records, allocated once for all chunks (every stream at once)
  unsigned long long *xbuf = nullptr;
  size_t xwords = 0;
  if (B > 1) {
    // every stream's records and the arrival counters (4 words)
    xwords = (size_t)S * 2 * B * k * (3 + n_lm + ((flags & FUSION_RUN_RECOMBINE) ? 1 : 0)) + 4;
    hipError_t e = hipMallocAsync(reinterpret_cast<void **>(&xbuf), xwords * sizeof(unsigned long long), stream);
    if (e != hipSuccess) return hip_error(e, "hipMallocAsync");
  }
  for (int32_t t = 0; t < T && rc == FUSION_OK; t += C) {
    const int32_t n = std::min(C, T - t);
    // the chunk's logits of all H hypotheses from their joint hidden states
    rc = joint_project(A + (size_t)t * H * K, W, bias, (int32_t)(n * H), V, K, logits, stream);
    if (rc != FUSION_OK) break;
    rc = run_impl(lms, alphas, n_lm, trie, logits, n, S, B, V, k, beta, blank_id, blank_mode, lm_state, boost_state,
                  hyp_score, tokens + (size_t)t * H, parents ? parents + (size_t)t * H : nullptr, nullptr, nullptr,
                  flags, hist, stream, false, xbuf, xwords, t);
  }
  if (xbuf) {
    const hipError_t e = hipFreeAsync(xbuf, stream);
    if (rc == FUSION_OK && e != hipSuccess) rc = hip_error(e, "hipFreeAsync");
  }
  return rc;
}
