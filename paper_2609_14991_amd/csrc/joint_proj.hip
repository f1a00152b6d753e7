// Output projection of the Transducer joint network on MFMA: the logits that
// the acoustic term of Eq. (1) (Sec. III-C) is computed from, for a batch of
// hypothesis-frames at once:
//
//   out[m, n] = sum_k A[m, k] * W[n, k] + bias[n]      (bf16 inputs, fp32 accumulate)
//
// A is [M, K] and W is [N, K], both row-major bf16 (W in the usual layout of a
// linear layer's weight), so both MFMA operands are contiguous along K.
//
// Tiling for gfx950: a 256-lane workgroup computes a 128 x 128 output tile as
// 4 waves of 64 x 64, each a 4 x 4 grid of v_mfma_f32_16x16x32_bf16 tiles
// (64 fp32 accumulators per lane).  K advances in stages of 32: every lane
// fetches two 16-byte strips of A and two of W per stage into registers while
// the previous stage, double-buffered in LDS (rows padded by 16 bytes), feeds
// the MFMAs.  Tiles are numbered column-fastest, so with the hardware's
// round-robin of workgroups over the 8 XCDs each XCD's L2 holds a quarter of W.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "fusion_internal.h"

namespace fusion {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int kBM = 128, kBN = 128, kBK = 32;
constexpr int kLd = kBK + 8;  // bf16 per LDS row: 80 bytes

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

__global__ void __launch_bounds__(256) joint_proj_kernel(const uint16_t *__restrict__ A,
                                                          const uint16_t *__restrict__ W,
                                                          const float *__restrict__ bias, int M, int N, int K,
                                                          int n_col_tiles, float *__restrict__ out) {
  __shared__ __align__(16) uint16_t sA[2][kBM * kLd];
  __shared__ __align__(16) uint16_t sW[2][kBN * kLd];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int tile = blockIdx.x;
  const int bn = (tile % n_col_tiles) * kBN, bm = (tile / n_col_tiles) * kBM;
  const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;

  // reads past a row range or past K return zeros (buffer range check)
  const __amdgpu_buffer_rsrc_t ra = rsrc(A, (uint32_t)((int64_t)M * K * 2));
  const __amdgpu_buffer_rsrc_t rw = rsrc(W, (uint32_t)((int64_t)N * K * 2));
  // strip c = tid + 256 * i (i < 2) of a 128 x 32 stage: row c >> 2, K offset (c & 3) * 8
  int arow[2], kc[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = tid + 256 * i;
    arow[i] = c >> 2;
    kc[i] = (c & 3) * 8;
  }
  auto fetch = [&](int k0, i32x4 (&ga)[2], i32x4 (&gw)[2]) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int k = k0 + kc[i];
      const int m = bm + arow[i], n = bn + arow[i];
      const uint32_t oa = (m < M && k < K) ? (uint32_t)(((int64_t)m * K + k) * 2) : 0xFFFFFFF0u;
      const uint32_t ow = (n < N && k < K) ? (uint32_t)(((int64_t)n * K + k) * 2) : 0xFFFFFFF0u;
      ga[i] = __builtin_amdgcn_raw_buffer_load_b128(ra, oa, 0, 0);
      gw[i] = __builtin_amdgcn_raw_buffer_load_b128(rw, ow, 0, 0);
    }
  };
  auto stash = [&](int buf, const i32x4 (&ga)[2], const i32x4 (&gw)[2]) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      *reinterpret_cast<i32x4 *>(&sA[buf][arow[i] * kLd + kc[i]]) = ga[i];
      *reinterpret_cast<i32x4 *>(&sW[buf][arow[i] * kLd + kc[i]]) = gw[i];
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

  const int nk = (K + kBK - 1) / kBK;
  {
    i32x4 ga[2], gw[2];
    fetch(0, ga, gw);
    stash(0, ga, gw);
  }
  __syncthreads();
  // fragment of a 16 x 32 operand tile: lane l holds row l % 16, K elements 8 * (l / 16) .. + 7
  const int fr = lane & 15, fk = (lane >> 4) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    i32x4 ga[2], gw[2];
    const bool more = kt + 1 < nk;
    if (more) fetch((kt + 1) * kBK, ga, gw);
    bf16x8 fa[4], fw[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      fa[i] = *reinterpret_cast<const bf16x8 *>(&sA[buf][(wm + i * 16 + fr) * kLd + fk]);
      fw[i] = *reinterpret_cast<const bf16x8 *>(&sW[buf][(wn + i * 16 + fr) * kLd + fk]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i], fw[j], acc[i][j], 0, 0, 0);
    if (more) stash(buf ^ 1, ga, gw);
    __syncthreads();
  }

  // accumulator of a 16 x 16 tile: lane l holds column l % 16, rows 4 * (l / 16) .. + 3
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = bn + wn + j * 16 + (lane & 15);
    if (n >= N) continue;
    const float bv = bias ? bias[n] : 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = bm + wm + i * 16 + (lane >> 4) * 4 + r;
        if (m < M) out[(int64_t)m * N + n] = acc[i][j][r] + bv;
      }
    }
  }
}

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
  const int nct = (N + kBN - 1) / kBN, nrt = (M + kBM - 1) / kBM;
  if ((int64_t)nct * nrt > 0x7FFFFFFFll) return set_error(FUSION_E_UNSUPPORTED, "too many tiles");
  hipLaunchKernelGGL(joint_proj_kernel, dim3(nct * nrt), dim3(256), 0, stream, A, W, bias, M, N, K, nct, out);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? FUSION_OK : hip_error(e, "joint projection launch");
}
