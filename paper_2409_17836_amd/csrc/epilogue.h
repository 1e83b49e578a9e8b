// Fused epilogues of the decoder's matrix products.  Both GEMM kernels hand
// their accumulators over in column pairs (col, col + 32) with col % 64 < 32;
// the weights are repacked so that each pair is what a fused op needs:
//   - q/k projections: the two halves of a RoPE rotation pair (i, i + hd/2);
//   - gate/up projection: gate and up of the same FFN feature;
//   - everything else: two independent columns.
#pragma once

#include <math.h>

#include "common.h"

namespace lmgc {

template <typename T>
__device__ inline void store_act(void* p, int64_t i, float v);
template <>
__device__ inline void store_act<uint16_t>(void* p, int64_t i, float v) {
  ((uint16_t*)p)[i] = f32_to_bf16(v);
}
template <>
__device__ inline void store_act<float>(void* p, int64_t i, float v) {
  ((float*)p)[i] = v;
}

// Parameters (biases) are stored in the model dtype, like the activations.
template <typename T>
__device__ inline float load_par(const void* p, int i);
template <>
__device__ inline float load_par<uint16_t>(const void* p, int i) {
  return bf16_to_f32(((const uint16_t*)p)[i]);
}
template <>
__device__ inline float load_par<float>(const void* p, int i) {
  return ((const float*)p)[i];
}

__device__ inline float silu_f(float x) { return x / (1.0f + expf(-x)); }

__device__ inline float gelu_tanh_f(float x) {
  const float k0 = 0.7978845608028654f;  // sqrt(2/pi)
  return 0.5f * x * (1.0f + tanhf(k0 * (x + 0.044715f * x * x * x)));
}

// Where a column of the fused QKV output goes: segment (0 q, 1 k, 2 v), head, dim.
// q and k columns of a 64-column group g hold rotation pairs g*32 .. g*32+31:
// column g*64 + t is dim i of pair P = g*32 + t, column g*64 + 32 + t its
// partner dim i + hd/2 (head = P / (hd/2), i = P % (hd/2)).
__device__ inline void qkv_rope_target(int col, int Hq, int Hkv, int hd, int& seg, int& head,
                                       int& i) {
  const int segq = Hq * hd, segk = Hkv * hd;
  int cc = col;
  seg = 0;
  if (cc >= segq) {
    cc -= segq;
    seg = 1;
    if (cc >= segk) {
      cc -= segk;
      seg = 2;
    }
  }
  if (seg == 2) {  // v: natural order
    head = cc / hd;
    i = cc % hd;
    return;
  }
  const int P = (cc >> 6) * 32 + (cc & 31);
  head = P / (hd / 2);
  i = P % (hd / 2);
}

template <typename T, int KIND>
__device__ inline void epi_pair(const EpiArgs& e, int row, int col, float vlo, float vhi) {
  if (KIND != EPI_STORE_F32 && col + 32 >= e.N + 32) return;  // padded columns
  if (KIND == EPI_STORE_F32) {
    float* c = e.c + (int64_t)row * e.ldc;
    if (col < e.N) c[col] = vlo;
    if (col + 32 < e.N) c[col + 32] = vhi;
  } else if (KIND == EPI_RESID) {
    float* c = e.c + (int64_t)row * e.ldc;
    if (e.bias) {
      vlo += load_par<T>(e.bias, col);
      vhi += load_par<T>(e.bias, col + 32);
    }
    c[col] += vlo;
    c[col + 32] += vhi;
  } else if (KIND == EPI_SWIGLU) {
    const int f = (col >> 6) * 32 + (col & 31);
    store_act<T>(e.out, (int64_t)row * e.ld_out + f, silu_f(vlo) * vhi);
  } else if (KIND == EPI_BIAS_GELU) {
    const int64_t base = (int64_t)row * e.ld_out;
    store_act<T>(e.out, base + col, gelu_tanh_f(vlo + load_par<T>(e.bias, col)));
    store_act<T>(e.out, base + col + 32, gelu_tanh_f(vhi + load_par<T>(e.bias, col + 32)));
  } else if (KIND == EPI_QKV_ROPE) {
    const int b = row / e.W, pos = row - b * e.W;
    int seg, head, i;
    qkv_rope_target(col, e.Hq, e.Hkv, e.hd, seg, head, i);
    if (seg < 2) {
      const float2 cs = e.rope[pos * (e.hd / 2) + i];
      const float lo = vlo * cs.x - vhi * cs.y;
      const float hi = vhi * cs.x + vlo * cs.y;
      const int H = seg == 0 ? e.Hq : e.Hkv;
      void* dst = seg == 0 ? e.q : e.k;
      const int64_t base = (((int64_t)b * H + head) * e.W + pos) * e.hd;
      store_act<T>(dst, base + i, lo);
      store_act<T>(dst, base + i + e.hd / 2, hi);
    } else {
      int seg2, head2, i2;
      qkv_rope_target(col + 32, e.Hq, e.Hkv, e.hd, seg2, head2, i2);
      if (sizeof(T) == 2) {  // v stored transposed: [B, Hkv, hd, W]
        store_act<T>(e.v, (((int64_t)b * e.Hkv + head) * e.hd + i) * e.W + pos, vlo);
        store_act<T>(e.v, (((int64_t)b * e.Hkv + head2) * e.hd + i2) * e.W + pos, vhi);
      } else {
        store_act<T>(e.v, (((int64_t)b * e.Hkv + head) * e.W + pos) * e.hd + i, vlo);
        store_act<T>(e.v, (((int64_t)b * e.Hkv + head2) * e.W + pos) * e.hd + i2, vhi);
      }
    }
  } else if (KIND == EPI_QKV_BIAS) {
    const int b = row / e.W, pos = row - b * e.W;
    const int d = e.Hq * e.hd;
#pragma unroll
    for (int t = 0; t < 2; t++) {
      const int cc = col + 32 * t;
      const float v = (t ? vhi : vlo) + load_par<T>(e.bias, cc);
      const int seg = cc / d, r = cc - seg * d, head = r / e.hd, i = r % e.hd;
      if (seg < 2) {
        void* dst = seg == 0 ? e.q : e.k;
        store_act<T>(dst, (((int64_t)b * e.Hq + head) * e.W + pos) * e.hd + i, v);
      } else if (sizeof(T) == 2) {
        store_act<T>(e.v, (((int64_t)b * e.Hq + head) * e.hd + i) * e.W + pos, v);
      } else {
        store_act<T>(e.v, (((int64_t)b * e.Hq + head) * e.W + pos) * e.hd + i, v);
      }
    }
  }
}

}  // namespace lmgc
