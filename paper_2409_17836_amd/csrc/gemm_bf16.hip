// bf16 matrix product on CDNA4 matrix cores: C[M, N] = A[M, K] * B[N, K]^T
// with float32 accumulation, followed by a fused epilogue (epilogue.h).
//
// Both operands are K-contiguous (activations row-major, weights [out, in]).
// Tile: 256 x 256 output per 256-thread workgroup, four 64-wide waves in a
// 2 x 2 grid, each wave 128 x 128 = 4 x 4 blocks of v_mfma_f32_32x32x16_bf16.
// K advances in steps of 64 through a double-buffered LDS stage (2 x 64 KB)
// filled by direct global->LDS loads (no staging registers); 16-byte LDS
// chunks are XOR-swizzled by (row & 7) so that the eight rows a group of
// lanes reads in one ds_read_b128 fall in distinct banks.  Each stage lives
// in its own __shared__ array so the compiler can tell the in-flight loads
// of one stage from the reads of the other.
//
// Determinism: every output element is the same fixed sequence of MFMA
// accumulations over k regardless of M, of the tile it sits in, and of the
// values of other rows, so the LM's per-position tables do not depend on the
// batch or window length (lossless decoding relies on this).
//
// Workgroup -> tile order: the hardware deals workgroups to the 8 XCDs
// round-robin; ids are remapped so each XCD walks a contiguous range of a
// row-grouped tile order (4 row-tiles per group), which keeps the A and B
// panels the ~32 co-resident workgroups of an XCD share in that XCD's L2.
#include "epilogue.h"

namespace lmgc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kThreads = 256;
constexpr int kGroupM = 4;
constexpr int kXcds = 8;

__device__ inline int swz(int row, int chunk) { return row * 8 + (chunk ^ (row & 7)); }

__device__ inline bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ inline bool map_tile(int bid, int nblocks, int ntm, int ntn, int& tm, int& tn) {
  const int total = ntm * ntn;
  const int per = nblocks / kXcds;  // nblocks is a multiple of kXcds
  const int t = (bid % kXcds) * per + bid / kXcds;
  if (t >= total) return false;
  const int in_group = kGroupM * ntn;
  const int g = t / in_group;
  const int first = g * kGroupM;
  const int gs = min(ntm - first, kGroupM);
  const int r = t - g * in_group;
  tm = first + r % gs;
  tn = r / gs;
  return true;
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

template <int KIND>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ Bw, int M, int K, int ntm,
    int ntn, EpiArgs e) {
  __shared__ uint4 sA0[BM * 8], sB0[BN * 8], sA1[BM * 8], sB1[BN * 8];  // 4 x 32 KB

  int tm, tn;
  if (!map_tile(blockIdx.x, gridDim.x, ntm, ntn, tm, tn)) return;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Direct global->LDS loads (16 B per lane): load i of wave w fills LDS rows
  // (w*8 + i)*8 .. +8; lane l lands at row +l/8, physical chunk l%8, so it
  // fetches logical chunk (l%8) ^ (l/8): the swizzle is applied on the
  // global side.
  const int lr = lane >> 3;
  const int lc = (lane & 7) ^ lr;
  const uint16_t* ga[8];
  const uint16_t* gb[8];
#pragma unroll
  for (int i = 0; i < 8; i++) {
    const int row = (wave * 8 + i) * 8 + lr;
    ga[i] = A + (int64_t)min(m0 + row, M - 1) * K + lc * 8;
    gb[i] = Bw + (int64_t)(n0 + row) * K + lc * 8;
  }

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; i++)
#pragma unroll
    for (int j = 0; j < 4; j++) acc[i][j] = f32x16{};

  const int arow0 = wm * 128 + (lane & 31);
  const int brow0 = wn * 128 + (lane & 31);
  const int khalf = lane >> 5;

  auto load = [&](uint4* sa, uint4* sb, int k0) {
#pragma unroll
    for (int i = 0; i < 8; i++) {
      const int blk = (wave * 8 + i) * 64;
      __builtin_amdgcn_global_load_lds((const void*)(ga[i] + k0), (lds_ptr_t)(sa + blk), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)(gb[i] + k0), (lds_ptr_t)(sb + blk), 16, 0, 0);
    }
  };
  auto compute = [&](const uint4* sa, const uint4* sb) {
#pragma unroll
    for (int ks = 0; ks < BK / 16; ks++) {
      const int ch = ks * 2 + khalf;
      bf16x8 af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; i++) af[i] = as_bf16x8(sa[swz(arow0 + 32 * i, ch)]);
#pragma unroll
      for (int j = 0; j < 4; j++) bf[j] = as_bf16x8(sb[swz(brow0 + 32 * j, ch)]);
#pragma unroll
      for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
  };

  const int nk = K / BK;
  load(sA0, sB0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  int kt = 0;
  for (; kt + 2 <= nk; kt += 2) {
    load(sA1, sB1, (kt + 1) * BK);
    __builtin_amdgcn_sched_barrier(0);
    compute(sA0, sB0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (kt + 2 < nk) load(sA0, sB0, (kt + 2) * BK);
    __builtin_amdgcn_sched_barrier(0);
    compute(sA1, sB1);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }
  if (kt < nk) compute(sA0, sB0);

  // Epilogue: lane holds column (lane & 31) of each 32x32 block and rows
  // 8 (r / 4) + 4 (lane / 32) + r % 4; blocks j and j + 1 give the pair
  // (col, col + 32).
  const int rbase = m0 + wm * 128 + 4 * khalf;
  const int cbase = n0 + wn * 128 + (lane & 31);
#pragma unroll
  for (int i = 0; i < 4; i++) {
#pragma unroll
    for (int r = 0; r < 16; r++) {
      const int row = rbase + 32 * i + 8 * (r >> 2) + (r & 3);
      if (row < M) {
        epi_pair<uint16_t, KIND>(e, row, cbase, acc[i][0][r], acc[i][1][r]);
        epi_pair<uint16_t, KIND>(e, row, cbase + 64, acc[i][2][r], acc[i][3][r]);
      }
    }
  }
}

}  // namespace

hipError_t launch_gemm_bf16(const uint16_t* A, const uint16_t* B, int M, int N_pad, int K,
                            const EpiArgs& e, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (K % BK != 0 || N_pad % BN != 0) return hipErrorInvalidValue;
  const int ntm = (M + BM - 1) / BM, ntn = N_pad / BN;
  const int total = ntm * ntn;
  const int nblocks = (total + kXcds - 1) / kXcds * kXcds;
  const dim3 grid(nblocks), block(kThreads);
  switch (e.kind) {
    case EPI_STORE_F32:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_STORE_F32>, grid, block, 0, s, A, B, M, K, ntm, ntn, e);
      break;
    case EPI_RESID:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_RESID>, grid, block, 0, s, A, B, M, K, ntm, ntn, e);
      break;
    case EPI_QKV_ROPE:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_QKV_ROPE>, grid, block, 0, s, A, B, M, K, ntm, ntn, e);
      break;
    case EPI_QKV_BIAS:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_QKV_BIAS>, grid, block, 0, s, A, B, M, K, ntm, ntn, e);
      break;
    case EPI_SWIGLU:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_SWIGLU>, grid, block, 0, s, A, B, M, K, ntm, ntn, e);
      break;
    case EPI_BIAS_GELU:
      hipLaunchKernelGGL(gemm_bf16_kernel<EPI_BIAS_GELU>, grid, block, 0, s, A, B, M, K, ntm, ntn, e);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace lmgc
