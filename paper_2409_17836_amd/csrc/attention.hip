// Causal self-attention of the decoder (softmax(q.k / sqrt(hd)) v over keys
// <= query), tiled through LDS with an online softmax so the W x W score
// matrix never exists (the FlashAttention idea the paper lists as a
// throughput lever in its discussion section).
//
// bf16 kernel (CDNA4 matrix cores).  A workgroup of four 64-wide waves owns
// 128 queries of one (window, head); each wave 32 queries.  Key/value tiles
// of 64 keys are staged in LDS.  The wave computes S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16, so each lane holds one query's scores in its own
// registers: the row max / row sum need one cross-lane exchange (lane ^ 32)
// instead of a 32-lane reduction.  The K rows are fed to the MFMA in a
// permuted order so that the score registers are, without any shuffle, the
// B operand of O^T += V^T P^T; V is transposed on its way into LDS.  The
// next K/V tile is fetched into registers while the current one is in use.
// Softmax statistics are float32 in base 2; P is rounded to bf16 for the
// second product; O is normalised at the end.
//
// Determinism / prefix invariance: a query's key tiles are processed in a
// fixed order that depends only on the query's 128-query block; masked keys
// contribute exact zeros.  So each output row is a bitwise function of the
// keys/values at positions <= its own, independent of W and of other windows.
#include <math.h>

#include "common.h"

namespace lmgc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Swizzle of the 16-byte chunks of a K row so that the 8 rows one group of
// lanes reads together (keys {0-3, 8-11} + 16 j and {4-7, 12-15} + 16 j)
// fall in distinct bank groups.
__device__ inline int kswz(int key) { return (key & 3) | ((key >> 1) & 4); }

// key held by score register r of a lane in half h (see the S^T layout).
__device__ inline int key_of_reg(int r, int h) { return r < 8 ? 8 * h + r : 16 + 8 * h + (r - 8); }

__device__ inline uint32_t word_of(const u32x4& v, int w) { return v[w]; }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ inline uint32_t pack2(float a, float b) {
  const bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

template <int HD>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(const uint16_t* __restrict__ q,
                                                           const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ v,
                                                           uint16_t* __restrict__ o, int Hq,
                                                           int Hkv, int W, float sl2) {
  constexpr int BQ = 128, BKV = 64, KCH = HD / 8, NKS = HD / 16, NOB = HD / 32;
  // per thread and tile: K chunks (16 B) and V key pairs x 8 dims
  constexpr int NKL = BKV * KCH / 256;       // K chunks per thread
  constexpr int NVL = (BKV / 2) * KCH / 256;  // V (key pair, dim chunk) units per thread
  __shared__ u32x4 sK[BKV * KCH];
  __shared__ u32x4 sV[HD * 8];  // V^T: [dim][64 keys], 16-byte chunks swizzled by dim

  const int nqb = (W + BQ - 1) / BQ;
  const int qb = nqb - 1 - (int)blockIdx.x;  // longest blocks first
  const int h = blockIdx.y, b = blockIdx.z;
  const int kvh = h * Hkv / Hq;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int half = lane >> 5, c32 = lane & 31;
  const int q0 = qb * BQ + wave * 32;
  const int myq = q0 + c32;

  const uint16_t* Qp = q + (int64_t)(b * Hq + h) * W * HD;
  const uint16_t* Kp = k + (int64_t)(b * Hkv + kvh) * W * HD;
  const uint16_t* Vp = v + (int64_t)(b * Hkv + kvh) * W * HD;

  bf16x8 qf[NKS];
  {
    const int qr = min(myq, W - 1);
#pragma unroll
    for (int ks = 0; ks < NKS; ks++)
      qf[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(Qp + (int64_t)qr * HD + 16 * ks + 8 * half));
  }
  f32x16 oacc[NOB];
#pragma unroll
  for (int i = 0; i < NOB; i++) oacc[i] = f32x16{};
  float m_i = -INFINITY, l_i = 0.f;

  // MFMA row rho = 8a + 4g + c (a = rho/8, g = (rho/4)&1, c = rho&3) takes key
  // 16 (a/2) + 8 g + 4 (a&1) + c of its 32-key block.
  const int pa = c32 >> 3, pg = (c32 >> 2) & 1, pc = c32 & 3;
  const int kperm = 16 * (pa >> 1) + 8 * pg + 4 * (pa & 1) + pc;

  // register staging of one K/V tile (loaded one tile ahead)
  u32x4 rk[NKL], rv[NVL][2];
  auto gload = [&](int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NKL; i++) {
      const int c = tid + 256 * i, key = c / KCH, ch = c % KCH;
      rk[i] = *reinterpret_cast<const u32x4*>(Kp + (int64_t)min(k0 + key, W - 1) * HD + ch * 8);
    }
#pragma unroll
    for (int i = 0; i < NVL; i++) {
      const int u = tid + 256 * i, kp = u & 31, ch = u >> 5;
#pragma unroll
      for (int e = 0; e < 2; e++) {
        const int key = k0 + 2 * kp + e;
        rv[i][e] = key < W ? *reinterpret_cast<const u32x4*>(Vp + (int64_t)key * HD + ch * 8)
                           : u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto lstore = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NKL; i++) {
      const int c = tid + 256 * i, key = c / KCH, ch = c % KCH;
      sK[key * KCH + (ch ^ kswz(key))] = rk[i];
    }
    // V^T: word (dim, key pair) <- (V[2kp][dim], V[2kp+1][dim])
    uint32_t* sv = reinterpret_cast<uint32_t*>(sV);
#pragma unroll
    for (int i = 0; i < NVL; i++) {
      const int u = tid + 256 * i, kp = u & 31, ch = u >> 5;
#pragma unroll
      for (int e = 0; e < 8; e++) {
        const int d = ch * 8 + e;
        const uint32_t wa = word_of(rv[i][0], e >> 1), wb = word_of(rv[i][1], e >> 1);
        const uint32_t lo = (e & 1) ? (wa >> 16) : (wa & 0xffffu);
        const uint32_t hi = (e & 1) ? (wb >> 16) : (wb & 0xffffu);
        const int kc = kp >> 2;  // 16-byte chunk of the 64-key row
        sv[(d * 8 + (kc ^ (d & 7))) * 4 + (kp & 3)] = lo | (hi << 16);
      }
    }
  };

  const int kend = min(W, qb * BQ + BQ);
  const int ntiles = (kend + BKV - 1) / BKV;
  gload(0);
  for (int t = 0; t < ntiles; t++) {
    const int k0 = t * BKV;
    __syncthreads();  // every wave is done with the previous tile
    lstore();
    __syncthreads();
    if (t + 1 < ntiles) gload(k0 + BKV);  // in flight during this tile's math
    if (k0 > q0 + 31) continue;           // tile entirely after this wave's queries

    f32x16 s0 = f32x16{}, s1 = f32x16{};
#pragma unroll
    for (int ks = 0; ks < NKS; ks++) {
      const int ch = 2 * ks + half;
      const int key0 = kperm, key1 = 32 + kperm;
      const bf16x8 ka = as_bf16x8(sK[key0 * KCH + (ch ^ kswz(key0))]);
      const bf16x8 kb = as_bf16x8(sK[key1 * KCH + (ch ^ kswz(key1))]);
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[ks], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb, qf[ks], s1, 0, 0, 0);
    }
    float mx = -INFINITY;
    const bool diag = k0 + BKV - 1 > q0;  // some key of the tile may lie after a query
#pragma unroll
    for (int r = 0; r < 16; r++) {
      const int key = k0 + key_of_reg(r, half);
      s0[r] = (!diag || key <= myq) ? s0[r] * sl2 : -INFINITY;
      s1[r] = (!diag || key + 32 <= myq) ? s1[r] * sl2 : -INFINITY;
      mx = fmaxf(mx, fmaxf(s0[r], s1[r]));
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mnew = fmaxf(m_i, mx);
    const float alpha = __builtin_amdgcn_exp2f(m_i - mnew);
    float ls = 0.f;
#pragma unroll
    for (int r = 0; r < 16; r++) {
      s0[r] = __builtin_amdgcn_exp2f(s0[r] - mnew);
      s1[r] = __builtin_amdgcn_exp2f(s1[r] - mnew);
      ls += s0[r] + s1[r];
    }
    ls += __shfl_xor(ls, 32, 64);
    l_i = l_i * alpha + ls;
    m_i = mnew;
#pragma unroll
    for (int i = 0; i < NOB; i++) oacc[i] *= alpha;

    bf16x8 pf[4];
#pragma unroll
    for (int kk = 0; kk < 4; kk++) {
      const f32x16& sv = (kk < 2) ? s0 : s1;
      const int r0 = (kk & 1) * 8;
      const u32x4 u = {pack2(sv[r0 + 0], sv[r0 + 1]), pack2(sv[r0 + 2], sv[r0 + 3]),
                       pack2(sv[r0 + 4], sv[r0 + 5]), pack2(sv[r0 + 6], sv[r0 + 7])};
      pf[kk] = as_bf16x8(u);
    }
#pragma unroll
    for (int i = 0; i < NOB; i++) {
      const int d = i * 32 + c32;
#pragma unroll
      for (int kk = 0; kk < 4; kk++) {
        const bf16x8 va = as_bf16x8(sV[d * 8 + ((2 * kk + half) ^ (d & 7))]);
        oacc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pf[kk], oacc[i], 0, 0, 0);
      }
    }
  }

  if (myq < W) {
    const float inv = 1.0f / l_i;
    uint16_t* orow = o + ((int64_t)b * W + myq) * (int64_t)(Hq * HD) + h * HD;
#pragma unroll
    for (int i = 0; i < NOB; i++) {
#pragma unroll
      for (int a = 0; a < 4; a++) {
        const int d = i * 32 + 8 * a + 4 * half;
        uint2 u;
        u.x = pack2(oacc[i][4 * a + 0] * inv, oacc[i][4 * a + 1] * inv);
        u.y = pack2(oacc[i][4 * a + 2] * inv, oacc[i][4 * a + 3] * inv);
        *reinterpret_cast<uint2*>(orow + d) = u;
      }
    }
  }
}

// float32 attention for float32 decoders: one thread per query, keys in
// order through 64-key LDS tiles, online softmax per key.
template <int HD>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ q,
                                                      const float* __restrict__ k,
                                                      const float* __restrict__ v,
                                                      float* __restrict__ o, int Hq, int Hkv,
                                                      int W, float scale) {
  __shared__ float sK[64][HD + 1];
  __shared__ float sV[64][HD + 1];
  const int h = blockIdx.y, b = blockIdx.z;
  const int kvh = h * Hkv / Hq;
  const int myq = blockIdx.x * 64 + threadIdx.x;
  const float* Qp = q + (int64_t)(b * Hq + h) * W * HD;
  const float* Kp = k + (int64_t)(b * Hkv + kvh) * W * HD;
  const float* Vp = v + (int64_t)(b * Hkv + kvh) * W * HD;
  float qv[HD], acc[HD];
  const int qr = min(myq, W - 1);
#pragma unroll
  for (int i = 0; i < HD; i++) {
    qv[i] = Qp[(int64_t)qr * HD + i];
    acc[i] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const int kend = min(W, (int)blockIdx.x * 64 + 64);
  for (int k0 = 0; k0 < kend; k0 += 64) {
    __syncthreads();
    for (int c = threadIdx.x; c < 64 * HD; c += 64) {
      const int key = c / HD, i = c % HD;
      const int kk = min(k0 + key, W - 1);
      sK[key][i] = Kp[(int64_t)kk * HD + i];
      sV[key][i] = Vp[(int64_t)kk * HD + i];
    }
    __syncthreads();
    for (int j = 0; j < 64; j++) {
      const int key = k0 + j;
      if (key > myq || key >= W) break;
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < HD; i++) s = fmaf(qv[i], sK[j][i], s);
      s *= scale;
      const float mn = fmaxf(m, s);
      const float corr = expf(m - mn);
      const float p = expf(s - mn);
      l = l * corr + p;
#pragma unroll
      for (int i = 0; i < HD; i++) acc[i] = acc[i] * corr + p * sV[j][i];
      m = mn;
    }
  }
  if (myq < W) {
    float* orow = o + ((int64_t)b * W + myq) * (int64_t)(Hq * HD) + h * HD;
#pragma unroll
    for (int i = 0; i < HD; i++) orow[i] = acc[i] / l;
  }
}

}  // namespace

hipError_t launch_attention_bf16(const uint16_t* q, const uint16_t* k, const uint16_t* v,
                                 uint16_t* o, int B, int Hq, int Hkv, int W, int hd,
                                 hipStream_t s) {
  if (B <= 0 || W <= 0) return hipSuccess;
  const dim3 grid((W + 127) / 128, Hq, B), block(256);
  const float sl2 = (float)(1.4426950408889634 / sqrt((double)hd));
  if (hd == 128)
    hipLaunchKernelGGL(attn_bf16_kernel<128>, grid, block, 0, s, q, k, v, o, Hq, Hkv, W, sl2);
  else if (hd == 64)
    hipLaunchKernelGGL(attn_bf16_kernel<64>, grid, block, 0, s, q, k, v, o, Hq, Hkv, W, sl2);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attention_f32(const float* q, const float* k, const float* v, float* o, int B,
                                int Hq, int Hkv, int W, int hd, hipStream_t s) {
  if (B <= 0 || W <= 0) return hipSuccess;
  const dim3 grid((W + 63) / 64, Hq, B), block(64);
  const float scale = (float)(1.0 / sqrt((double)hd));
  switch (hd) {
    case 16:
      hipLaunchKernelGGL(attn_f32_kernel<16>, grid, block, 0, s, q, k, v, o, Hq, Hkv, W, scale);
      break;
    case 32:
      hipLaunchKernelGGL(attn_f32_kernel<32>, grid, block, 0, s, q, k, v, o, Hq, Hkv, W, scale);
      break;
    case 48:
      hipLaunchKernelGGL(attn_f32_kernel<48>, grid, block, 0, s, q, k, v, o, Hq, Hkv, W, scale);
      break;
    case 64:
      hipLaunchKernelGGL(attn_f32_kernel<64>, grid, block, 0, s, q, k, v, o, Hq, Hkv, W, scale);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace lmgc
