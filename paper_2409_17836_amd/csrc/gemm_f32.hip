// float32 matrix product for float32 decoders: C = A[M, K] * B[N, K]^T with
// the same fused epilogues as the bf16 kernel.  A plain LDS-tiled FMA kernel
// (64 x 64 tile, 256 threads, 4 x 4 outputs per thread); every output is a
// sequential k-ordered FMA chain, so results do not depend on M or on other
// rows (a decoding step runs it on one row per window and gets the same
// values).  Used for the small float32 model, where the work is latency-bound.
#include "epilogue.h"

namespace lmgc {
namespace {

constexpr int TM = 64, TN = 64, TK = 16;

template <int KIND>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A,
                                                       const float* __restrict__ Bw, int M, int K,
                                                       EpiArgs e) {
  __shared__ float As[TK][TM + 4];
  __shared__ float Bs[TK][TN + 4];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * TM, n0 = blockIdx.x * TN;
  // loader: row tid/4, k offset (tid%4)*4
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  const float* pa = A + (int64_t)min(m0 + lr, M - 1) * K + lk;
  const float* pb = Bw + (int64_t)(n0 + lr) * K + lk;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; i++)
#pragma unroll
    for (int j = 0; j < 4; j++) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < K; k0 += TK) {
    const float4 va = *reinterpret_cast<const float4*>(pa + k0);
    const float4 vb = *reinterpret_cast<const float4*>(pb + k0);
    As[lk + 0][lr] = va.x;
    As[lk + 1][lr] = va.y;
    As[lk + 2][lr] = va.z;
    As[lk + 3][lr] = va.w;
    Bs[lk + 0][lr] = vb.x;
    Bs[lk + 1][lr] = vb.y;
    Bs[lk + 2][lr] = vb.z;
    Bs[lk + 3][lr] = vb.w;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < TK; k++) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; i++) a[i] = As[k][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; j++) b[j] = Bs[k][tx + 16 * j];
#pragma unroll
      for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  if constexpr (KIND == EPI_HEAD) {
    // the tile is one 64-column group; the 16 threads of a row (tx = lane & 15
    // of one wave) hold its columns tx + 16 j
    bool ok[4];
    int aidx[4];
#pragma unroll
    for (int j = 0; j < 4; j++) {
      ok[j] = n0 + tx + 16 * j < e.N;
      aidx[j] = ok[j] ? alpha_index(e, n0 + tx + 16 * j) : -1;
    }
    const bool any_alpha = __any(aidx[0] >= 0 || aidx[1] >= 0 || aidx[2] >= 0 || aidx[3] >= 0);
    float z[4][4];
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
      for (int j = 0; j < 4; j++) z[i][j] = ok[j] ? acc[i][j] : -INFINITY;
    head_rows4(e, z, aidx, any_alpha, m0 + ty * 4, M, blockIdx.x, tx);
    return;
  }
  // thread columns tx + 16 j: pairs (tx, tx + 32) and (tx + 16, tx + 48)
  using E = Epi<float, KIND, 0>;
  const ColInfo ci0 = E::column(e, n0 + tx), ci1 = E::column(e, n0 + tx + 16);
  const int W = e.W > 0 ? e.W : 1;
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int row = m0 + ty * 4 + i;
    if (row >= M) continue;
    const int b = e.step ? row : row / W, pos = e.step ? e.dpos : row - b * W;
    E::row(e, ci0, n0 + tx, row, b, pos, acc[i][0], acc[i][2]);
    E::row(e, ci1, n0 + tx + 16, row, b, pos, acc[i][1], acc[i][3]);
  }
}

}  // namespace

hipError_t launch_gemm_f32(const float* A, const float* B, int M, int N_pad, int K,
                           const EpiArgs& e, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (K % TK != 0 || N_pad % TN != 0) return hipErrorInvalidValue;
  const dim3 grid(N_pad / TN, (M + TM - 1) / TM), block(256);
  switch (e.kind) {
    case EPI_STORE_F32:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE_F32>, grid, block, 0, s, A, B, M, K, e);
      break;
    case EPI_RESID:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_RESID>, grid, block, 0, s, A, B, M, K, e);
      break;
    case EPI_QKV_ROPE:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_QKV_ROPE>, grid, block, 0, s, A, B, M, K, e);
      break;
    case EPI_QKV_BIAS:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_QKV_BIAS>, grid, block, 0, s, A, B, M, K, e);
      break;
    case EPI_SWIGLU:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_SWIGLU>, grid, block, 0, s, A, B, M, K, e);
      break;
    case EPI_BIAS_GELU:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_BIAS_GELU>, grid, block, 0, s, A, B, M, K, e);
      break;
    case EPI_HEAD:
      hipLaunchKernelGGL(gemm_f32_kernel<EPI_HEAD>, grid, block, 0, s, A, B, M, K, e);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace lmgc
