// Output projection of the Transducer joint network on MFMA: the logits that
// the acoustic term of Eq. (1) (Sec. III-C) is computed from, for a batch of
// hypothesis-frames at once:
//
//   out[m, n] = sum_k A[m, k] * W[n, k] + bias[n]      (bf16 inputs, fp32 accumulate)
//
// A is [M, K] and W is [N, K], both row-major bf16 (W in the usual layout of a
// linear layer's weight), so both MFMA operands are contiguous along K.
//
// Tiling for gfx950: a workgroup of WM x WN waves computes a (16 TM WM) x
// (16 TN WN) output tile, each wave (16 TM) x (16 TN) as a TM x TN grid of
// v_mfma_f32_16x16x32_bf16 tiles (4 TM TN fp32 accumulators per lane); the
// larger the wave's tile, the fewer LDS bytes each multiply-accumulate reads.
// K advances in stages of BK, double-buffered in LDS (rows padded by 16
// bytes); every lane fetches its 16-byte strips of A and W two stages ahead
// into one of two register sets, so a load has two stages of MFMAs to arrive
// in.  The logits leave with streaming (non-temporal) stores.  Tiles are
// assigned per XCD (see the kernel) so that each XCD's L2 serves a row band of
// A to the column tiles of its half and keeps half of W.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "fusion_internal.h"

namespace fusion {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));


__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

// kWM x kWN waves, each a (16 kTM) x (16 kTN) output tile; K stages of kBK
template <int kWM, int kWN, int kBK, int kTM, int kTN>
__global__ void __launch_bounds__(64 * kWM * kWN) joint_proj_kernel(const uint16_t *__restrict__ A,
                                                                     const uint16_t *__restrict__ W,
                                                                     const float *__restrict__ bias, int M, int N,
                                                                     int K, int n_col_tiles, int xcd_map, int vec_out,
                                                                     float *__restrict__ out) {
  constexpr int kRM = 16 * kTM, kRN = 16 * kTN;  // rows and columns of a wave's tile
  constexpr int kBM = kRM * kWM, kBN = kRN * kWN;
  constexpr int kLd = kBK + 8;  // bf16 per LDS row (16-byte pad)
  constexpr int kThreads = 64 * kWM * kWN;
  constexpr int kStripsA = kBM * kBK / 8 / kThreads;  // 16-byte strips per thread and stage
  constexpr int kStripsW = kBN * kBK / 8 / kThreads;
  constexpr int kChunks = kBK / 8;                     // strips per row
  // one LDS block: the double-buffered operand stages, reused by the epilogue
  __shared__ __align__(16) uint16_t smem[2 * (kBM + kBN) * kLd];
  uint16_t(*sA)[kBM * kLd] = reinterpret_cast<uint16_t(*)[kBM * kLd]>(smem);
  uint16_t(*sW)[kBN * kLd] = reinterpret_cast<uint16_t(*)[kBN * kLd]>(smem + 2 * kBM * kLd);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  // tile of this workgroup.  With xcd_map (row tiles a multiple of 4, column
  // tiles even) workgroup w runs on XCD w % 8 under the hardware's round-robin,
  // and XCD x takes the row tiles = x % 4 (mod 4) against column half x / 4: a
  // row band of A is fetched by two XCDs instead of eight and each XCD's L2
  // keeps half of W.  Otherwise tiles go column-fastest.
  int tr, tc;
  if (xcd_map) {
    const int x = blockIdx.x & 7, i = blockIdx.x >> 3;
    const int half = n_col_tiles >> 1;
    tr = (i / half) * 4 + (x & 3);
    tc = (x >> 2) * half + i % half;
  } else {
    tr = blockIdx.x / n_col_tiles;
    tc = blockIdx.x % n_col_tiles;
  }
  const int bn = tc * kBN, bm = tr * kBM;
  const int wm = (wave / kWN) * kRM, wn = (wave % kWN) * kRN;

  // reads past a row range or past K return zeros (buffer range check)
  const __amdgpu_buffer_rsrc_t ra = rsrc(A, (uint32_t)((int64_t)M * K * 2));
  const __amdgpu_buffer_rsrc_t rw = rsrc(W, (uint32_t)((int64_t)N * K * 2));
  // strip c = tid + kThreads * i of a stage: row c / kChunks, K offset (c % kChunks) * 8
  auto fetch = [&](int k0, i32x4 (&ga)[kStripsA], i32x4 (&gw)[kStripsW]) {
#pragma unroll
    for (int i = 0; i < kStripsA; ++i) {
      const int c = tid + kThreads * i;
      const int k = k0 + (c % kChunks) * 8, m = bm + c / kChunks;
      const uint32_t oa = (m < M && k < K) ? (uint32_t)(((int64_t)m * K + k) * 2) : 0xFFFFFFF0u;
      ga[i] = __builtin_amdgcn_raw_buffer_load_b128(ra, oa, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < kStripsW; ++i) {
      const int c = tid + kThreads * i;
      const int k = k0 + (c % kChunks) * 8, n = bn + c / kChunks;
      const uint32_t ow = (n < N && k < K) ? (uint32_t)(((int64_t)n * K + k) * 2) : 0xFFFFFFF0u;
      gw[i] = __builtin_amdgcn_raw_buffer_load_b128(rw, ow, 0, 0);
    }
  };
  auto stash = [&](int buf, const i32x4 (&ga)[kStripsA], const i32x4 (&gw)[kStripsW]) {
#pragma unroll
    for (int i = 0; i < kStripsA; ++i) {
      const int c = tid + kThreads * i;
      *reinterpret_cast<i32x4 *>(&sA[buf][(c / kChunks) * kLd + (c % kChunks) * 8]) = ga[i];
    }
#pragma unroll
    for (int i = 0; i < kStripsW; ++i) {
      const int c = tid + kThreads * i;
      *reinterpret_cast<i32x4 *>(&sW[buf][(c / kChunks) * kLd + (c % kChunks) * 8]) = gw[i];
    }
  };

  f32x4 acc[kTM][kTN];
#pragma unroll
  for (int i = 0; i < kTM; ++i)
#pragma unroll
    for (int j = 0; j < kTN; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  // K stages: stage s sits in LDS buffer s & 1 while it feeds the MFMAs; its
  // global loads were issued two stages earlier into register set s & 1, so
  // each load has two stages' compute to arrive in
  const int nk = (K + kBK - 1) / kBK;
  i32x4 ga[2][kStripsA], gw[2][kStripsW];
  fetch(0, ga[0], gw[0]);
  stash(0, ga[0], gw[0]);
  if (nk > 1) fetch(kBK, ga[1], gw[1]);
  __syncthreads();
  // fragment of a 16 x 32 operand tile: lane l holds row l % 16, K elements 8 * (l / 16) .. + 7
  const int fr = lane & 15, fk = (lane >> 4) * 8;
  auto stage = [&](int kt, auto set) {
    constexpr int S = decltype(set)::value;  // = kt & 1
    if (kt + 2 < nk) fetch((kt + 2) * kBK, ga[S], gw[S]);  // set S held stage kt, already in LDS
#pragma unroll
    for (int ks = 0; ks < kBK; ks += 32) {
      bf16x8 fa[kTM], fw[kTN];
#pragma unroll
      for (int i = 0; i < kTM; ++i) fa[i] = *reinterpret_cast<const bf16x8 *>(&sA[S][(wm + i * 16 + fr) * kLd + ks + fk]);
#pragma unroll
      for (int j = 0; j < kTN; ++j) fw[j] = *reinterpret_cast<const bf16x8 *>(&sW[S][(wn + j * 16 + fr) * kLd + ks + fk]);
#pragma unroll
      for (int i = 0; i < kTM; ++i)
#pragma unroll
        for (int j = 0; j < kTN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fw[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) stash(S ^ 1, ga[S ^ 1], gw[S ^ 1]);
    __syncthreads();
  };
  for (int kt = 0; kt < nk; kt += 2) {
    stage(kt, std::integral_constant<int, 0>{});
    if (kt + 1 < nk) stage(kt + 1, std::integral_constant<int, 1>{});
  }

  // accumulator of a 16 x 16 tile: lane l holds column l % 16, rows 4 * (l / 16) .. + 3
  if (vec_out) {
    // each 16-row slab of the wave's tile goes through the wave's own LDS area
    // (the operand buffers are free after the last stage) and leaves as whole
    // rows: 16 lanes store a row segment of 64 floats with 16-byte stores
    constexpr int kSlabLd = kRN + 4;
    float *slab = reinterpret_cast<float *>(smem) + wave * 16 * kSlabLd;
    static_assert(sizeof(smem) >= sizeof(float) * 16 * kSlabLd * kWM * kWN, "LDS too small for the epilogue");
    static_assert(kRN % 64 == 0, "the epilogue stores 64-column segments");
    float bv[kTN];
#pragma unroll
    for (int j = 0; j < kTN; ++j) {
      const int n = bn + wn + j * 16 + (lane & 15);
      bv[j] = (bias && n < N) ? bias[n] : 0.0f;
    }
#pragma unroll
    for (int i = 0; i < kTM; ++i) {
#pragma unroll
      for (int j = 0; j < kTN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) slab[((lane >> 4) * 4 + r) * kSlabLd + j * 16 + (lane & 15)] = acc[i][j][r] + bv[j];
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int sg = 0; sg < kRN / 64; ++sg) {
        const int cn = bn + wn + sg * 64 + (lane & 15) * 4;  // first of the 4 columns this lane stores
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = q * 4 + (lane >> 4);
          const f32x4 v = *reinterpret_cast<const f32x4 *>(&slab[row * kSlabLd + sg * 64 + (lane & 15) * 4]);
          const int m = bm + wm + i * 16 + row;
          // streaming stores: the logits are not read back by this kernel
          if (m < M && cn < N) __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(&out[(int64_t)m * N + cn]));
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  } else {
#pragma unroll
    for (int j = 0; j < kTN; ++j) {
      const int n = bn + wn + j * 16 + (lane & 15);
      if (n >= N) continue;
      const float bv = bias ? bias[n] : 0.0f;
#pragma unroll
      for (int i = 0; i < kTM; ++i) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = bm + wm + i * 16 + (lane >> 4) * 4 + r;
          if (m < M) out[(int64_t)m * N + n] = acc[i][j][r] + bv;
        }
      }
    }
  }
}

// a launch shape of joint_proj_kernel
template <int WM_, int WN_, int BK_, int TM_, int TN_>
struct ProjCfg {
  static constexpr int WM = WM_, WN = WN_, BK = BK_, TM = TM_, TN = TN_;
};

}  // namespace
}  // namespace fusion

using namespace fusion;

extern "C" int joint_project(const uint16_t *A, const uint16_t *W, const float *bias, int32_t M, int32_t N,
                             int32_t K, float *out, hipStream_t stream) {
  if (M < 0 || N < 1 || K < 8) return set_error(FUSION_E_ARG, "M, N or K out of range");
  if (K % 8 != 0) return set_error(FUSION_E_UNSUPPORTED, "K must be a multiple of 8");
  if ((int64_t)M * K * 2 > 0x7FFFFFF0ll || (int64_t)N * K * 2 > 0x7FFFFFF0ll)
    return set_error(FUSION_E_UNSUPPORTED, "operand larger than 2 GiB: split the call along M");
  if (M == 0) return FUSION_OK;
  if (!A || !W || !out) return set_error(FUSION_E_ARG, "NULL operand");
  if (((uintptr_t)A | (uintptr_t)W) % 16 != 0) return set_error(FUSION_E_ARG, "A and W must be 16-byte aligned");
  // whole 16-byte row segments when every row starts 16-byte aligned
  const int vec_out = (N % 4 == 0 && (uintptr_t)out % 16 == 0) ? 1 : 0;
  auto go = [&](auto cfg) -> int {
    using C = decltype(cfg);
    constexpr int BM = 16 * C::TM * C::WM, BN = 16 * C::TN * C::WN;
    const int nct = (N + BN - 1) / BN, nrt = (M + BM - 1) / BM;
    if ((int64_t)nct * nrt > 0x7FFFFFFFll) return set_error(FUSION_E_UNSUPPORTED, "too many tiles");
    const int xcd_map = (nrt % 4 == 0 && nct % 2 == 0) ? 1 : 0;
    hipLaunchKernelGGL((joint_proj_kernel<C::WM, C::WN, C::BK, C::TM, C::TN>), dim3(nct * nrt), dim3(64 * C::WM * C::WN),
                       0, stream, A, W, bias, M, N, K, nct, xcd_map, vec_out, out);
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? FUSION_OK : hip_error(e, "joint projection launch");
  };
  // large batches (all frames at once): 256 x 256 tiles, 8 waves of 128 x 64;
  // one frame's hypotheses (M of a few hundred): 64 x 64 tiles, 4 waves of 16 x
  // 64, so that the launch still spreads over the CUs.  K stages of 32.
  return M <= 4096 ? go(ProjCfg<4, 1, 64, 1, 4>{}) : go(ProjCfg<2, 4, 32, 8, 4>{});
}
