// Row-wise kernels of the decoder: embedding with the BOS shift, RMSNorm /
// LayerNorm, the kernel that turns the LM head's partials into log-sum-exp
// and integer tables, and the row gather used to repack weights.  All are
// HBM-bound; each uses one
// 64-wide wavefront per row with fixed-order (butterfly) reductions, so every
// row's result is a bitwise function of that row alone.
#include <math.h>

#include "common.h"

namespace lmgc {
namespace {

constexpr int kWave = 64;

struct AlphaIds {
  int32_t v[LMGC_NALPHA_MAX];
};

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

__device__ inline float load_param(const void* p, int i, int dtype) {
  return dtype == LMGC_DTYPE_BF16 ? bf16_to_f32(((const uint16_t*)p)[i]) : ((const float*)p)[i];
}

// ------------------------------------------------------------------ embed
// h[b*W + j, :] = E[x] (+ P[j]) with x = BOS for j = 0, else tokens[b, j-1];
// a decoding step (dpos >= 0): h[b, :] for position dpos, x = BOS for
// dpos = 0, else tokens[b].
__global__ void embed_kernel(const int32_t* __restrict__ tokens, int B, int W, int bos,
                             const void* __restrict__ E, const void* __restrict__ P, int d,
                             int V, int dtype, int dpos, float* __restrict__ h) {
  const int64_t row = (int64_t)blockIdx.x * 4 + threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (row >= (dpos >= 0 ? (int64_t)B : (int64_t)B * W)) return;
  const int j = dpos >= 0 ? dpos : (int)(row % W);
  const int prev = j == 0 ? bos : (dpos >= 0 ? tokens[row] : tokens[row - 1]);
  const int x = min(max(prev, 0), V - 1);
  float* out = h + row * d;
  for (int c = lane * 4; c < d; c += kWave * 4) {
    float4 v;
    v.x = load_param(E, x * d + c + 0, dtype);
    v.y = load_param(E, x * d + c + 1, dtype);
    v.z = load_param(E, x * d + c + 2, dtype);
    v.w = load_param(E, x * d + c + 3, dtype);
    if (P) {
      v.x += load_param(P, j * d + c + 0, dtype);
      v.y += load_param(P, j * d + c + 1, dtype);
      v.z += load_param(P, j * d + c + 2, dtype);
      v.w += load_param(P, j * d + c + 3, dtype);
    }
    *reinterpret_cast<float4*>(out + c) = v;
  }
}

// ------------------------------------------------------------------- norms
// One wave per row; lane l keeps elements l, l+64, ... in registers (general
// case: any d that is a multiple of 64, float32 or bf16 output).
template <int MAXV>
__global__ __launch_bounds__(256) void norm_kernel(const float* __restrict__ h, int M, int d,
                                                   const void* __restrict__ g,
                                                   const void* __restrict__ b, int layernorm,
                                                   float eps, int dtype, void* __restrict__ y) {
  const int64_t row = (int64_t)blockIdx.x * 4 + threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (row >= M) return;
  const float* x = h + row * d;
  float v[MAXV];
  const int nv = d / kWave;
#pragma unroll
  for (int i = 0; i < MAXV; i++)
    if (i < nv) v[i] = x[i * kWave + lane];
  float mean = 0.f;
  if (layernorm) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < MAXV; i++)
      if (i < nv) s += v[i];
    mean = wave_sum(s) / (float)d;
  }
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < MAXV; i++) {
    if (i < nv) {
      const float a = v[i] - mean;
      ss += a * a;
    }
  }
  const float r = 1.0f / sqrtf(wave_sum(ss) / (float)d + eps);
#pragma unroll
  for (int i = 0; i < MAXV; i++) {
    if (i >= nv) continue;
    const int c = i * kWave + lane;
    float t = (v[i] - mean) * r * load_param(g, c, dtype);
    if (layernorm) t += load_param(b, c, dtype);
    if (dtype == LMGC_DTYPE_BF16)
      ((__bf16*)y)[row * d + c] = (__bf16)t;
    else
      ((float*)y)[row * d + c] = t;
  }
}

// bf16 output, d = 256 * NV4: lane l keeps the float4 chunks l, l+64, ... of
// the row (1 KB per wave load), writes four bf16 per store and reads the
// gains (and biases) four at a time.
template <int NV4>
__global__ void norm_bf16x4_kernel(const float* __restrict__ h, int M, const uint16_t* __restrict__ g,
                                   const uint16_t* __restrict__ b, int layernorm, float eps,
                                   __bf16* __restrict__ y) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  constexpr int d = NV4 * 4 * kWave;
  const int64_t row = (int64_t)blockIdx.x * 4 + threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (row >= M) return;
  const float4* x = reinterpret_cast<const float4*>(h + row * d);
  float4 v[NV4];
#pragma unroll
  for (int i = 0; i < NV4; i++) {
    // the residual stream is read once here: non-temporal loads keep it from
    // displacing the matrix kernels' operands in the caches (norm 10.0 ->
    // 8.4 ms per 7B step)
    typedef float f4v __attribute__((ext_vector_type(4)));
    const f4v t = __builtin_nontemporal_load(reinterpret_cast<const f4v*>(x) + i * kWave + lane);
    v[i] = make_float4(t[0], t[1], t[2], t[3]);
  }
  float mean = 0.f;
  if (layernorm) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NV4; i++) s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
    mean = wave_sum(s) / (float)d;
  }
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < NV4; i++) {
    const float a0 = v[i].x - mean, a1 = v[i].y - mean, a2 = v[i].z - mean, a3 = v[i].w - mean;
    ss += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
  }
  const float r = 1.0f / sqrtf(wave_sum(ss) / (float)d + eps);
  bf16x4* out = reinterpret_cast<bf16x4*>(y + row * d);
#pragma unroll
  for (int i = 0; i < NV4; i++) {
    const int c4 = i * kWave + lane;
    const uint2 gg = reinterpret_cast<const uint2*>(g)[c4];
    float t0 = (v[i].x - mean) * r * bf16_to_f32(gg.x & 0xFFFF);
    float t1 = (v[i].y - mean) * r * bf16_to_f32(gg.x >> 16);
    float t2 = (v[i].z - mean) * r * bf16_to_f32(gg.y & 0xFFFF);
    float t3 = (v[i].w - mean) * r * bf16_to_f32(gg.y >> 16);
    if (layernorm) {
      const uint2 bb = reinterpret_cast<const uint2*>(b)[c4];
      t0 += bf16_to_f32(bb.x & 0xFFFF);
      t1 += bf16_to_f32(bb.x >> 16);
      t2 += bf16_to_f32(bb.y & 0xFFFF);
      t3 += bf16_to_f32(bb.y >> 16);
    }
    out[c4] = bf16x4{(__bf16)t0, (__bf16)t1, (__bf16)t2, (__bf16)t3};
  }
}

// ------------------------------------------------------------ LSE + table
// log-sum-exp merge of (m, s) with (mo, so): the larger maximum stays, the
// other sum is rescaled; an empty side (m = -inf, s = 0) adds nothing.
__device__ inline void lse_merge(float& m, float& s, float mo, float so) {
  const float mn = fmaxf(m, mo);
  if (mn == -INFINITY) return;
  const float a = (m == -INFINITY) ? 0.f : s * expf(m - mn);
  const float c = (mo == -INFINITY) ? 0.f : so * expf(mo - mn);
  s = a + c;  // commutative: both sides of a butterfly get the same bits
  m = mn;
}

// One wave per row.  Full-vocabulary tables: the row's head partials (one
// (max, sum-exp) per 64-column group, written by the head GEMM's epilogue)
// are merged lane-locally in group order (lane l: groups l, l + 64, ...),
// then across the wave by a fixed butterfly; LSE = max + log(sum).
// renorm: the log-sum-exp runs over the NA alphabet logits alone.  Then the
// NA alphabet log-probabilities z_a - LSE and their integer table of NA + 2
// entries (quantised in double; escape bin NA; renorm: the largest frequency
// takes total - sum and the escape bin is empty).
template <int NA>
__global__ void head_tables_kernel(const float2* __restrict__ part, int ngroups,
                                   const float* __restrict__ za, int ld_za, int M, uint32_t total,
                                   int renorm, uint32_t* __restrict__ cdf, float* __restrict__ logp) {
  constexpr int NS = NA + 1;  // coder bins incl. escape
  const uint32_t spread = renorm ? total - NA : total - NS;
  const int64_t alpha_total = renorm ? (int64_t)total : (int64_t)total - 1;
  const int64_t row = (int64_t)blockIdx.x * 4 + threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  if (row >= M) return;
  const float* zr = za + row * (int64_t)ld_za;
  float m = -INFINITY, s = 0.f;
  if (renorm) {
    if (lane < NA) {
      m = zr[lane];
      s = 1.f;
    }
  } else {
    const float2* pr = part + row * (int64_t)ngroups;
    // (unrolled so that several loads are in flight: the few rows of a
    // decoding step are bound by load latency; the order of the merges is
    // unchanged)
#pragma unroll 4
    for (int g = lane; g < ngroups; g += kWave) {
      const float2 p = pr[g];
      lse_merge(m, s, p.x, p.y);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float mo = __shfl_xor(m, o, kWave);
    const float so = __shfl_xor(s, o, kWave);
    lse_merge(m, s, mo, so);
  }
  const float lse = m + logf(s);
  uint32_t f = 0;
  if (lane < NA) {
    const float lp = zr[lane] - lse;
    const double p = exp((double)lp);
    f = 1u + (uint32_t)floor(p * (double)spread);
    if (logp) logp[row * NA + lane] = lp;
  }
  uint32_t fa[NA];
  int64_t S = 0;
#pragma unroll
  for (int a = 0; a < NA; a++) {
    fa[a] = (uint32_t)__shfl((int)f, a, kWave);
    S += fa[a];
  }
  if (S > alpha_total || (renorm && S < alpha_total)) {
    int big = 0;
#pragma unroll
    for (int a = 1; a < NA; a++)
      if (fa[a] > fa[big]) big = a;
    const int64_t adj = alpha_total - S;
#pragma unroll
    for (int a = 0; a < NA; a++)
      if (a == big) fa[a] = (uint32_t)((int64_t)fa[a] + adj);
    S = alpha_total;
  }
  if (lane <= NS) {
    uint32_t c = 0;
#pragma unroll
    for (int a = 0; a < NA; a++)
      if (a < lane) c += fa[a];
    if (lane == NS) c = total;
    cdf[row * (NS + 1) + lane] = c;
  }
}

// Rows of the LM head for the alphabet tokens: dst row r (r < na) = head row
// ids[r]; rows na..gridDim.x-1 are zero.  One block per row.
// bf16: head and tile in MFMA blocks; one thread per 16-byte piece (8
// values of one row) of the tile.
__global__ void alpha_head_blocked_kernel(const uint4* __restrict__ head, AlphaIds ids, int na, int rows,
                                          int cols, uint4* __restrict__ dst) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int pieces = cols / 8;
  if (t >= (int64_t)rows * pieces) return;
  const int r = (int)(t / pieces), q = (int)(t - (int64_t)r * pieces);
  const int64_t di = blocked_index(r, 8 * q, cols) / 8;
  if (r >= na) {
    dst[di] = make_uint4(0u, 0u, 0u, 0u);
    return;
  }
  dst[di] = head[blocked_index(ids.v[r], 8 * q, cols) / 8];
}

__global__ void alpha_head_kernel(const uint32_t* __restrict__ head, AlphaIds ids, int na, int words,
                                  uint32_t* __restrict__ dst) {
  const int r = blockIdx.x;
  uint32_t* out = dst + (int64_t)r * words;
  if (r >= na) {
    for (int c = threadIdx.x; c < words; c += blockDim.x) out[c] = 0u;
    return;
  }
  const uint32_t* src = head + (int64_t)ids.v[r] * words;
  for (int c = threadIdx.x; c < words; c += blockDim.x) out[c] = src[c];
}

// ------------------------------------------------------------------ gather
// bf16 rows into MFMA blocks: one thread per 16-byte piece of an output row.
__global__ void gather_rows_blocked_kernel(GatherSrcs srcs, const int32_t* __restrict__ idx, int rows,
                                           int cols, uint4* __restrict__ dst) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int pieces = cols / 8;
  if (t >= (int64_t)rows * pieces) return;
  const int r = (int)(t / pieces), q = (int)(t - (int64_t)r * pieces);
  const int64_t di = blocked_index(r, 8 * q, cols) / 8;
  const int32_t id = idx ? idx[r] : r;
  if (id < 0) {
    dst[di] = make_uint4(0u, 0u, 0u, 0u);
    return;
  }
  const uint4* src = (const uint4*)srcs.p[id >> 28] + (int64_t)(id & 0x0fffffff) * pieces;
  dst[di] = src[q];
}

__global__ void gather_rows_kernel(GatherSrcs srcs, const int32_t* __restrict__ idx, int rows,
                                   int words, uint32_t* __restrict__ dst) {
  const int r = blockIdx.x;
  if (r >= rows) return;
  const int32_t id = idx[r];
  uint32_t* out = dst + (int64_t)r * words;
  if (id < 0) {
    for (int c = threadIdx.x; c < words; c += blockDim.x) out[c] = 0u;
    return;
  }
  const uint32_t* src = (const uint32_t*)srcs.p[id >> 28] + (int64_t)(id & 0x0fffffff) * words;
  for (int c = threadIdx.x; c < words; c += blockDim.x) out[c] = src[c];
}

}  // namespace

hipError_t launch_embed(const int32_t* tokens, int B, int W, int bos_id, const void* tok_emb,
                        const void* pos_emb, int d, int vocab, int dtype, int dpos, float* h,
                        hipStream_t s) {
  const int64_t rows = dpos >= 0 ? (int64_t)B : (int64_t)B * W;
  hipLaunchKernelGGL(embed_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, tokens,
                     B, W, bos_id, tok_emb, pos_emb, d, vocab, dtype, dpos, h);
  return hipGetLastError();
}

hipError_t launch_norm(const float* h, int M, int d, const void* gain, const void* bias,
                       int layernorm, float eps, int dtype, void* y, hipStream_t s) {
  const dim3 grid((unsigned)((M + 3) / 4));
  if (d % kWave != 0 || d > 8192) return hipErrorInvalidValue;
  if (dtype == LMGC_DTYPE_BF16 && d % 256 == 0) {
    const uint16_t* g16 = (const uint16_t*)gain;
    const uint16_t* b16 = (const uint16_t*)bias;
    __bf16* yb = (__bf16*)y;
    switch (d / 256) {
      case 2:
        hipLaunchKernelGGL(norm_bf16x4_kernel<2>, grid, dim3(256), 0, s, h, M, g16, b16, layernorm, eps, yb);
        return hipGetLastError();
      case 3:
        hipLaunchKernelGGL(norm_bf16x4_kernel<3>, grid, dim3(256), 0, s, h, M, g16, b16, layernorm, eps, yb);
        return hipGetLastError();
      case 4:
        hipLaunchKernelGGL(norm_bf16x4_kernel<4>, grid, dim3(256), 0, s, h, M, g16, b16, layernorm, eps, yb);
        return hipGetLastError();
      case 8:
        hipLaunchKernelGGL(norm_bf16x4_kernel<8>, grid, dim3(256), 0, s, h, M, g16, b16, layernorm, eps, yb);
        return hipGetLastError();
      case 16:
        hipLaunchKernelGGL(norm_bf16x4_kernel<16>, grid, dim3(256), 0, s, h, M, g16, b16, layernorm, eps, yb);
        return hipGetLastError();
      default:
        break;  // the general kernel below
    }
  }
  if (d <= 1024)
    hipLaunchKernelGGL(norm_kernel<16>, grid, dim3(256), 0, s, h, M, d, gain, bias, layernorm,
                       eps, dtype, y);
  else if (d <= 4096)
    hipLaunchKernelGGL(norm_kernel<64>, grid, dim3(256), 0, s, h, M, d, gain, bias, layernorm,
                       eps, dtype, y);
  else
    hipLaunchKernelGGL(norm_kernel<128>, grid, dim3(256), 0, s, h, M, d, gain, bias, layernorm,
                       eps, dtype, y);
  return hipGetLastError();
}

hipError_t launch_head_tables(const float2* part, int ngroups, const float* za, int ld_za, int M,
                              int n_alpha, uint32_t total, int renorm, uint32_t* cdf, float* logp,
                              hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (n_alpha != LMGC_NALPHA && n_alpha != LMGC_NALPHA_MAX) return hipErrorInvalidValue;
  if (ld_za < n_alpha || (!renorm && (!part || ngroups <= 0))) return hipErrorInvalidValue;
  const dim3 grid((unsigned)((M + 3) / 4)), block(256);
  if (n_alpha == LMGC_NALPHA)
    hipLaunchKernelGGL(head_tables_kernel<LMGC_NALPHA>, grid, block, 0, s, part, ngroups, za, ld_za, M, total,
                       renorm, cdf, logp);
  else
    hipLaunchKernelGGL(head_tables_kernel<LMGC_NALPHA_MAX>, grid, block, 0, s, part, ngroups, za, ld_za, M,
                       total, renorm, cdf, logp);
  return hipGetLastError();
}

hipError_t launch_alpha_head(const void* head, const int32_t* alpha_ids, int n_alpha, int rows, int cols,
                             int elem_bytes, void* dst, hipStream_t s) {
  AlphaIds ids = {};
  if (n_alpha < 1 || n_alpha > LMGC_NALPHA_MAX || rows < n_alpha || (cols * elem_bytes) % 4)
    return hipErrorInvalidValue;
  for (int a = 0; a < n_alpha; a++) ids.v[a] = alpha_ids[a];
  if (elem_bytes == 2) {
    if (rows % 16 || cols % 32) return hipErrorInvalidValue;
    const int64_t n = (int64_t)rows * (cols / 8);
    hipLaunchKernelGGL(alpha_head_blocked_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const uint4*)head, ids, n_alpha, rows, cols, (uint4*)dst);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(alpha_head_kernel, dim3((unsigned)rows), dim3(256), 0, s, (const uint32_t*)head, ids, n_alpha,
                     cols * elem_bytes / 4, (uint32_t*)dst);
  return hipGetLastError();
}

hipError_t launch_gather_rows_blocked(GatherSrcs srcs, const int32_t* idx, int rows, int cols,
                                      void* dst, hipStream_t s) {
  if (rows % 16 || cols % 32) return hipErrorInvalidValue;
  const int64_t n = (int64_t)rows * (cols / 8);
  hipLaunchKernelGGL(gather_rows_blocked_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, srcs, idx,
                     rows, cols, (uint4*)dst);
  return hipGetLastError();
}

hipError_t launch_gather_rows(GatherSrcs srcs, const int32_t* idx, int rows, int cols,
                              int elem_bytes, void* dst, hipStream_t s) {
  const int words = cols * elem_bytes / 4;
  hipLaunchKernelGGL(gather_rows_kernel, dim3((unsigned)rows), dim3(256), 0, s, srcs, idx, rows,
                     words, (uint32_t*)dst);
  return hipGetLastError();
}

}  // namespace lmgc
