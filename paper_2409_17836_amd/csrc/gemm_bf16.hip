// bf16 matrix product on CDNA4 matrix cores: C[M, N] = A[M, K] * B[N, K]^T
// with float32 accumulation, followed by a fused epilogue (epilogue.h).
//
// Both operands are K-contiguous (activations row-major, weights [out, in]).
// Tile: 256 x 256 output per 512-thread workgroup: eight 64-wide waves, two
// per SIMD so that one wave's LDS reads and waits overlap the other's matrix
// instructions; wave (wm, wn) owns rows wm*128 .. +128 and columns
// wn*64 .. +64 as 8 x 4 blocks of v_mfma_f32_16x16x32_bf16.
// K advances in steps of 64 through a double-buffered LDS stage (2 x 64 KB)
// filled by direct global->LDS loads (no staging registers).  A 256 x 64
// operand tile is stored as rows of eight 16-byte chunks; chunk c of row r
// sits at slot c ^ ((r >> 1) & 7): the 16 lanes that one ds_read_b128 cycle
// serves read 16 consecutive rows, and the swizzle gives every (row parity,
// slot) pair once, i.e. all 64 banks.  Each stage lives in its own
// __shared__ array so the compiler can tell the in-flight loads of one stage
// from the reads of the other.
//
// Determinism: every output element is the same fixed sequence of MFMA
// accumulations over k regardless of M, of the tile it sits in, and of the
// values of other rows, so the LM's per-position tables do not depend on the
// batch or window length (lossless decoding relies on this).
//
// Workgroup -> tile order: the hardware deals workgroups to the 8 XCDs
// round-robin; ids are remapped so each XCD walks a contiguous range of a
// row-grouped tile order (8 row-tiles per group), which keeps the A and B
// panels the co-resident workgroups of an XCD share in that XCD's L2.
#include "epilogue.h"

namespace lmgc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kThreads = 512;
constexpr int kGroupM = 8;
constexpr int kXcds = 8;

__device__ inline int slot(int row, int chunk) { return row * 8 + (chunk ^ ((row >> 1) & 7)); }

__device__ inline bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

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

template <int KIND, int HD>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ Bw, int M, int K, int ntm,
    int ntn, EpiArgs e) {
  __shared__ u32x4 sA0[BM * 8], sB0[BN * 8], sA1[BM * 8], sB1[BN * 8];  // 4 x 32 KB

  int tm, tn;
  if (!map_tile(blockIdx.x, gridDim.x, ntm, ntn, tm, tn)) return;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;

  // Direct global->LDS loads (16 B per lane): load i of wave w fills LDS rows
  // (w*4 + i)*8 .. +8; lane l lands at row +l/8, slot l%8, so it fetches the
  // logical chunk that the swizzle puts there.
  const uint16_t* ga[4];
  const uint16_t* gb[4];
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int row = (wave * 4 + i) * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ ((row >> 1) & 7);
    ga[i] = A + (int64_t)min(m0 + row, M - 1) * K + lc * 8;
    gb[i] = Bw + (int64_t)(n0 + row) * K + lc * 8;
  }

  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; i++)
#pragma unroll
    for (int j = 0; j < 4; j++) acc[i][j] = f32x4{};

  // MFMA operands: lane l supplies row (l & 15) of a 16-row block and the
  // 8 k-values of chunk (l >> 4) of the 32-wide k step.
  const int arow0 = wm * 128 + (lane & 15), brow0 = wn * 64 + (lane & 15), kq = lane >> 4;

  auto load = [&](u32x4* sa, u32x4* sb, int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int blk = (wave * 4 + i) * 64;
      __builtin_amdgcn_global_load_lds((const void*)(ga[i] + k0), (lds_ptr_t)(sa + blk), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((const void*)(gb[i] + k0), (lds_ptr_t)(sb + blk), 16, 0, 0);
    }
  };
  auto compute = [&](const u32x4* sa, const u32x4* sb) __attribute__((always_inline)) {
#pragma unroll
    for (int ks = 0; ks < BK / 32; ks++) {
      const int ch = ks * 4 + kq;
      bf16x8 af[8], bf[4];
#pragma unroll
      for (int i = 0; i < 8; i++) af[i] = as_bf16x8(sa[slot(arow0 + 16 * i, ch)]);
#pragma unroll
      for (int j = 0; j < 4; j++) bf[j] = as_bf16x8(sb[slot(brow0 + 16 * j, ch)]);
#pragma unroll
      for (int i = 0; i < 8; i++)
#pragma unroll
        for (int j = 0; j < 4; j++)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
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

  // Epilogue.  16 x 16 block layout: lane holds column (lane & 15) and rows
  // 4 (lane >> 4) + r, r = 0..3.  Blocks j and j + 2 give the column pair
  // (col, col + 32).  Rows 4 (lane >> 4) + 0..3 never straddle a window
  // (W is a multiple of 8).
  using E = Epi<uint16_t, KIND, HD>;
  const int c0 = n0 + wn * 64 + (lane & 15);
  const ColInfo ci0 = E::column(e, c0), ci1 = E::column(e, c0 + 16);
  const int W = e.W > 0 ? e.W : 1;
#pragma unroll
  for (int i = 0; i < 8; i++) {
    const int r0 = m0 + wm * 128 + 16 * i + 4 * kq;
    const int b = r0 / W, p0 = r0 - b * W;
    const float a0[4] = {acc[i][0][0], acc[i][0][1], acc[i][0][2], acc[i][0][3]};
    const float a2[4] = {acc[i][2][0], acc[i][2][1], acc[i][2][2], acc[i][2][3]};
    const float a1[4] = {acc[i][1][0], acc[i][1][1], acc[i][1][2], acc[i][1][3]};
    const float a3[4] = {acc[i][3][0], acc[i][3][1], acc[i][3][2], acc[i][3][3]};
    E::rows4(e, ci0, c0, r0, M, b, p0, a0, a2);
    E::rows4(e, ci1, c0 + 16, r0, M, b, p0, a1, a3);
  }
}

template <int HD>
hipError_t launch_kind(const uint16_t* A, const uint16_t* B, int M, int K, int ntm, int ntn,
                       const EpiArgs& e, hipStream_t s) {
  const int total = ntm * ntn;
  const dim3 grid((total + kXcds - 1) / kXcds * kXcds), block(kThreads);
  switch (e.kind) {
    case EPI_STORE_F32:
      hipLaunchKernelGGL((gemm_bf16_kernel<EPI_STORE_F32, HD>), grid, block, 0, s, A, B, M, K, ntm, ntn, e);
      break;
    case EPI_RESID:
      hipLaunchKernelGGL((gemm_bf16_kernel<EPI_RESID, HD>), grid, block, 0, s, A, B, M, K, ntm, ntn, e);
      break;
    case EPI_QKV_ROPE:
      hipLaunchKernelGGL((gemm_bf16_kernel<EPI_QKV_ROPE, HD>), grid, block, 0, s, A, B, M, K, ntm, ntn, e);
      break;
    case EPI_QKV_BIAS:
      hipLaunchKernelGGL((gemm_bf16_kernel<EPI_QKV_BIAS, HD>), grid, block, 0, s, A, B, M, K, ntm, ntn, e);
      break;
    case EPI_SWIGLU:
      hipLaunchKernelGGL((gemm_bf16_kernel<EPI_SWIGLU, HD>), grid, block, 0, s, A, B, M, K, ntm, ntn, e);
      break;
    case EPI_BIAS_GELU:
      hipLaunchKernelGGL((gemm_bf16_kernel<EPI_BIAS_GELU, HD>), grid, block, 0, s, A, B, M, K, ntm, ntn, e);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16(const uint16_t* A, const uint16_t* B, int M, int N_pad, int K,
                            const EpiArgs& e, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (K % BK != 0 || N_pad % BN != 0) return hipErrorInvalidValue;
  const int ntm = (M + BM - 1) / BM, ntn = N_pad / BN;
  const bool qkv = e.kind == EPI_QKV_ROPE || e.kind == EPI_QKV_BIAS;
  if (qkv && e.hd == 128) return launch_kind<128>(A, B, M, K, ntm, ntn, e, s);
  if (qkv && e.hd == 64) return launch_kind<64>(A, B, M, K, ntm, ntn, e, s);
  if (qkv) return hipErrorInvalidValue;
  return launch_kind<0>(A, B, M, K, ntm, ntn, e, s);
}

}  // namespace lmgc
