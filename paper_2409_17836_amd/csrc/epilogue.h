// Fused epilogues of the decoder's matrix products.  Both GEMM kernels hand
// their accumulators over in column pairs (col, col + 32) with col % 64 < 32;
// the weights are repacked so that each pair is what a fused op needs:
//   - q/k projections: the two halves of a RoPE rotation pair (i, i + hd/2);
//   - gate/up projection: gate and up of the same FFN feature;
//   - everything else: two independent columns.
// Per-column decoding (which of q/k/v, head, dim, bias) is done once per
// column pair (Epi::column); the per-row part (Epi::row) only needs the
// window index b and position pos of the row.  bf16 models store V
// transposed ([B, Hkv, hd, W]) for the attention kernel; Epi::rows4 writes
// four consecutive positions of a V column as one 8-byte store.
#pragma once

#include <math.h>

#include "common.h"

namespace lmgc {

template <typename T>
__device__ inline void store_act(void* p, int64_t i, float v);
template <>
__device__ inline void store_act<uint16_t>(void* p, int64_t i, float v) {
  ((__bf16*)p)[i] = (__bf16)v;  // round to nearest even (v_cvt_pk_bf16_f32)
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

// silu(x) = x / (1 + e^-x) in float32 with the hardware exp2 and reciprocal
// (about 1 ulp each).
__device__ inline float silu_f(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * x));
}

// The tanh form of GELU, 0.5 x (1 + tanh(u)) with u = sqrt(2/pi) (x +
// 0.044715 x^3), evaluated as the identical x / (1 + e^(-2u)): one hardware
// exp2 and one reciprocal instead of a tanh routine (the epilogue runs with
// one wave per SIMD, where long dependent sequences are not hidden).  e^(-2u)
// overflows to inf for large negative x, giving x * 0.
__device__ inline float gelu_tanh_f(float x) {
  const float k2 = -2.0f * 0.7978845608028654f * 1.4426950408889634f;  // -2 sqrt(2/pi) log2(e)
  const float inner = __builtin_fmaf(0.044715f * x * x, x, x);  // explicit fusion, as in rope_rot
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(k2 * inner));
}

// The per-element arithmetic of the residual add and the RoPE rotation, in
// one place: the tiled and the one-row kernels must give the same bits.
// Products that meet an addition are fused explicitly: left to the
// compiler, a sum of two products may be contracted around either product
// depending on the surrounding code, which changes the rounding between
// the two kernels.
__device__ inline float resid_add(float old, float v, float bias) { return old + (v + bias); }
__device__ inline void rope_rot(float vlo, float vhi, float c, float s, float& lo, float& hi) {
  lo = __builtin_fmaf(vlo, c, -(vhi * s));
  hi = __builtin_fmaf(vhi, c, vlo * s);
}

// ------------------------------------------------------------- LM head
// The head never stores its logits.  For every row and group of 64 columns
// it writes the log-sum-exp partial (max m, sum of exp(z - m)) and the
// logits of the alphabet columns; launch_head_tables merges the partials.
// In all three matrix kernels (tiled bf16, decoding-step bf16, float32) a
// group's 64 values of one row sit in one row of 16 lanes (lanes 16 k ..
// 16 k + 15) of a wave, lane t holding columns t + 16 j, j = 0..3, so one
// function reduces them for all three and the encoder's and decoder's
// tables agree bit for bit.
constexpr float kLog2e = 1.4426950408889634f;

// One DPP exchange within each row of 16 lanes (row_mirror: lane l <-> 15 -
// l; row_half_mirror: l <-> 7 - l in each half; quad_perm 1,0,3,2 / 2,3,0,1:
// l <-> l ^ 1 / l ^ 2).  Every lane has a source, so no lane keeps `old`.
constexpr int kDppRowMirror = 0x140, kDppRowHalfMirror = 0x141, kDppXor1 = 0xB1, kDppXor2 = 0x4E;
template <int CTRL>
__device__ inline float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// z[j]: column t + 16 j of the group (-inf past the vocabulary).  The max
// over the group, then exp(z - max) summed lane-locally in j order and over
// the 16 lanes of the row by four DPP exchanges (partners 15 - l, then 7 - l
// within each half, then l ^ 1, l ^ 2).  Each exchange pairs lanes whose
// values are already equal group-wise, and + and max are commutative, so all
// 16 lanes end with the same bits.  A group of -inf only (columns past the
// vocabulary) gives (-inf, 0): its reference is taken as 0 so every exp is
// exp(-inf) = 0.  Every lane of the wave must call it (DPP reads the other
// lanes).
__device__ inline float2 group_lse_part(const float z[4]) {
  float m = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
  m = fmaxf(m, dpp_f<kDppRowMirror>(m));
  m = fmaxf(m, dpp_f<kDppRowHalfMirror>(m));
  m = fmaxf(m, dpp_f<kDppXor1>(m));
  m = fmaxf(m, dpp_f<kDppXor2>(m));
  const float ref = m == -INFINITY ? 0.f : m;
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; j++) s += __builtin_amdgcn_exp2f((z[j] - ref) * kLog2e);
  s += dpp_f<kDppRowMirror>(s);
  s += dpp_f<kDppRowHalfMirror>(s);
  s += dpp_f<kDppXor1>(s);
  s += dpp_f<kDppXor2>(s);
  return make_float2(m, s);
}

// Alphabet index of a (valid) head column, or -1.
__device__ inline int alpha_index(const EpiArgs& e, int col) {
  int a = -1;
#pragma unroll
  for (int t = 0; t < LMGC_NALPHA_MAX; t++)
    if (t < e.n_alpha && e.alpha_ids[t] == col) a = t;
  return a;
}

// Four consecutive rows row0 .. row0 + 3 of the head epilogue: z[r][j] and
// aidx[j] for the lane's columns t + 16 j of group g; lane16 = t.  Rows at or
// past M are not stored.  Lanes t < 4 of each 16-lane group store the
// partial of row row0 + t (all 16 lanes hold it).  any_alpha (the same in
// every lane of the wave): some lane of the wave has an alphabet column.
__device__ inline void head_rows4(const EpiArgs& e, const float z[4][4], const int aidx[4],
                                  bool any_alpha, int64_t row0, int64_t M, int g, int lane16) {
  float2 p[4];
#pragma unroll
  for (int r = 0; r < 4; r++) p[r] = group_lse_part(z[r]);
  if (e.part) {
    // selected component by component from scalars: a select between the
    // float2 elements themselves became a lane-indexed load from a
    // stack copy of p
    const float m0 = p[0].x, m1 = p[1].x, m2 = p[2].x, m3 = p[3].x;
    const float s0 = p[0].y, s1 = p[1].y, s2 = p[2].y, s3 = p[3].y;
    const float vm = lane16 == 0 ? m0 : lane16 == 1 ? m1 : lane16 == 2 ? m2 : m3;
    const float vs = lane16 == 0 ? s0 : lane16 == 1 ? s1 : lane16 == 2 ? s2 : s3;
    if (lane16 < 4 && row0 + lane16 < M) e.part[(row0 + lane16) * e.ngroups + g] = make_float2(vm, vs);
  }
  if (any_alpha) {
#pragma unroll
    for (int j = 0; j < 4; j++)
#pragma unroll
      for (int r = 0; r < 4; r++)
        if (aidx[j] >= 0 && row0 + r < M) e.za[(row0 + r) * e.ld_za + aidx[j]] = z[r][j];
  }
}

// Column info of one (col, col + 32) pair.
struct ColInfo {
  int seg, head, i;     // QKV target of col: segment (0 q, 1 k, 2 v), head, dim
  int seg2, head2, i2;  // QKV target of col + 32 (v and unrotated layouts)
  float blo, bhi;       // biases of col and col + 32 (0 if none)
  bool valid;
};

// HD = head dim when known at compile time (0: read e.hd).
template <typename T, int KIND, int HD>
struct Epi {
  __device__ static inline int hdim(const EpiArgs& e) { return HD ? HD : e.hd; }

  __device__ static inline ColInfo column(const EpiArgs& e, int col) {
    ColInfo c;
    c.valid = col < e.N;
    c.seg = c.head = c.i = c.seg2 = c.head2 = c.i2 = 0;
    c.blo = c.bhi = 0.f;
    if (!c.valid) return c;
    const int h = hdim(e);
    if ((KIND == EPI_RESID || KIND == EPI_BIAS_GELU || KIND == EPI_QKV_BIAS) && e.bias) {
      c.blo = load_par<T>(e.bias, col);
      c.bhi = load_par<T>(e.bias, col + 32);
    }
    if (KIND == EPI_QKV_ROPE) {
      const int segq = e.Hq * h, segk = e.Hkv * h;
      int cc = col;
      if (cc >= segq) {
        cc -= segq;
        c.seg = 1;
        if (cc >= segk) {
          cc -= segk;
          c.seg = 2;
        }
      }
      if (c.seg == 2) {  // v: natural order, the pair is (cc, cc + 32)
        c.head = cc / h;
        c.i = cc % h;
        c.head2 = (cc + 32) / h;
        c.i2 = (cc + 32) % h;
      } else {  // 64-column group g holds rotation pairs g*32 .. g*32+31
        const int P = (cc >> 6) * 32 + (cc & 31);
        c.head = P / (h / 2);
        c.i = P % (h / 2);
      }
    } else if (KIND == EPI_QKV_BIAS) {
      const int d = e.Hq * h;
      c.seg = col / d;
      const int r = col - c.seg * d;
      c.head = r / h;
      c.i = r % h;
      c.seg2 = (col + 32) / d;
      const int r2 = col + 32 - c.seg2 * d;
      c.head2 = r2 / h;
      c.i2 = r2 % h;
    }
    return c;
  }

  __device__ static inline void row(const EpiArgs& e, const ColInfo& c, int col, int rw, int b,
                                    int pos, float vlo, float vhi) {
    if (c.valid) row_in(e, c, col, rw, b, pos, vlo, vhi);
  }

  // row() for a column known to be valid
  __device__ static inline void row_in(const EpiArgs& e, const ColInfo& c, int col, int rw, int b,
                                       int pos, float vlo, float vhi) {
    const int h = hdim(e);
    if (KIND == EPI_STORE_F32) {
      float* p = e.c + (int64_t)rw * e.ldc;
      p[col] = vlo;
      if (col + 32 < e.N) p[col + 32] = vhi;
    } else if (KIND == EPI_RESID) {
      float* p = e.c + (int64_t)rw * e.ldc;
      p[col] = resid_add(p[col], vlo, c.blo);
      p[col + 32] = resid_add(p[col + 32], vhi, c.bhi);
    } else if (KIND == EPI_SWIGLU) {
      const int f = (col >> 6) * 32 + (col & 31);
      store_act<T>(e.out, (int64_t)rw * e.ld_out + f, silu_f(vlo) * vhi);
    } else if (KIND == EPI_BIAS_GELU) {
      const int64_t base = (int64_t)rw * e.ld_out;
      store_act<T>(e.out, base + col, gelu_tanh_f(vlo + c.blo));
      store_act<T>(e.out, base + col + 32, gelu_tanh_f(vhi + c.bhi));
    } else if (KIND == EPI_QKV_ROPE) {
      if (c.seg < 2) {
        const float2 cs = e.rope[pos * (h / 2) + c.i];
        store_qk(e, c, b, pos, vlo, vhi, cs.x, cs.y);
      } else {
        store_act<T>(e.v, vidx(e, b, e.Hkv, c.head, c.i, pos), vlo);
        store_act<T>(e.v, vidx(e, b, e.Hkv, c.head2, c.i2, pos), vhi);
      }
    } else if (KIND == EPI_QKV_BIAS) {
      const float v1 = vlo + c.blo, v2 = vhi + c.bhi;
      if (c.seg == 2) store_act<T>(e.v, vidx(e, b, e.Hq, c.head, c.i, pos), v1);
      else store_act<T>(c.seg ? e.k : e.q, (((int64_t)b * e.Hq + c.head) * e.W + pos) * h + c.i, v1);
      if (c.seg2 == 2) store_act<T>(e.v, vidx(e, b, e.Hq, c.head2, c.i2, pos), v2);
      else store_act<T>(c.seg2 ? e.k : e.q, (((int64_t)b * e.Hq + c.head2) * e.W + pos) * h + c.i2, v2);
    }
  }

  // Element index of (window b, kv head, dim i, position pos) of V.
  __device__ static inline int64_t vidx(const EpiArgs& e, int b, int H, int head, int i, int pos) {
    const int h = hdim(e);
    return sizeof(T) == 2 ? (((int64_t)b * H + head) * h + i) * e.W + pos
                          : (((int64_t)b * H + head) * e.W + pos) * h + i;
  }

  // What the epilogue of rows rw0 .. rw0+3 reads before it writes: the
  // residual values (RESID) or the RoPE cos/sin of the q/k rotation
  // (QKV_ROPE).  A load cannot move above an earlier store that may alias
  // it, so the tiled kernel issues these loads for its next row block before
  // the stores of the current one.
  struct Pre4 {
    float x[4], y[4];
  };
  // FULL: the caller knows every row and column of its tile is in range.
  template <bool FULL>
  __device__ static inline Pre4 pre4(const EpiArgs& e, const ColInfo& c, int col, int rw0, int M, int p0) {
    Pre4 q;
#pragma unroll
    for (int r = 0; r < 4; r++) q.x[r] = q.y[r] = 0.f;
    if (!FULL && !c.valid) return q;
    if (KIND == EPI_RESID) {
#pragma unroll
      for (int r = 0; r < 4; r++)
        if (FULL || rw0 + r < M) {
          const float* p = e.c + (int64_t)(rw0 + r) * e.ldc;
          q.x[r] = p[col];
          q.y[r] = p[col + 32];
        }
    } else if (KIND == EPI_QKV_ROPE) {
      if (c.seg < 2) {
        const int h = hdim(e);
#pragma unroll
        for (int r = 0; r < 4; r++)
          if (FULL || rw0 + r < M) {
            const float2 cs = e.rope[(p0 + r) * (h / 2) + c.i];
            q.x[r] = cs.x;
            q.y[r] = cs.y;
          }
      }
    }
    return q;
  }

  // Rows rw0 .. rw0+3 (positions p0 .. p0+3 of window b; p0 % 4 == 0), with
  // the values pre4 loaded for them.
  template <bool FULL>
  __device__ static inline void rows4(const EpiArgs& e, const ColInfo& c, int col, int rw0, int M,
                                      int b, int p0, const float* lo, const float* hi, const Pre4& q) {
    if (!FULL && !c.valid) return;
    if (KIND == EPI_RESID) {
#pragma unroll
      for (int r = 0; r < 4; r++)
        if (FULL || rw0 + r < M) {
          float* p = e.c + (int64_t)(rw0 + r) * e.ldc;
          p[col] = resid_add(q.x[r], lo[r], c.blo);
          p[col + 32] = resid_add(q.y[r], hi[r], c.bhi);
        }
      return;
    }
    if (KIND == EPI_QKV_ROPE && c.seg < 2) {
#pragma unroll
      for (int r = 0; r < 4; r++)
        if (FULL || rw0 + r < M) store_qk(e, c, b, p0 + r, lo[r], hi[r], q.x[r], q.y[r]);
      return;
    }
    constexpr bool qkv = KIND == EPI_QKV_ROPE || KIND == EPI_QKV_BIAS;
    if (qkv && sizeof(T) == 2 && (FULL || rw0 + 3 < M) && (c.seg == 2 || c.seg2 == 2)) {
      const int H = KIND == EPI_QKV_ROPE ? e.Hkv : e.Hq;
      const float bl = KIND == EPI_QKV_BIAS ? c.blo : 0.f, bh = KIND == EPI_QKV_BIAS ? c.bhi : 0.f;
      if (c.seg == 2) {
        store4(e.v, vidx(e, b, H, c.head, c.i, p0), lo[0] + bl, lo[1] + bl, lo[2] + bl, lo[3] + bl);
      } else {
        for (int r = 0; r < 4; r++) row_one(e, c, col, rw0 + r, b, p0 + r, lo[r], true);
      }
      if (c.seg2 == 2 || (KIND == EPI_QKV_ROPE && c.seg == 2)) {
        store4(e.v, vidx(e, b, H, c.head2, c.i2, p0), hi[0] + bh, hi[1] + bh, hi[2] + bh, hi[3] + bh);
      } else {
        for (int r = 0; r < 4; r++) row_one(e, c, col, rw0 + r, b, p0 + r, hi[r], false);
      }
      return;
    }
#pragma unroll
    for (int r = 0; r < 4; r++)
      if (FULL || rw0 + r < M) row_in(e, c, col, rw0 + r, b, p0 + r, lo[r], hi[r]);
  }

 private:
  // RoPE-rotated q or k pair (dims i and i + hd/2 of the head) of one row
  __device__ static inline void store_qk(const EpiArgs& e, const ColInfo& c, int b, int pos, float vlo,
                                         float vhi, float cs, float sn) {
    const int h = hdim(e);
    float lo, hi;
    rope_rot(vlo, vhi, cs, sn, lo, hi);
    const int H = c.seg == 0 ? e.Hq : e.Hkv;
    void* dst = c.seg == 0 ? e.q : e.k;
    const int64_t base = (((int64_t)b * H + c.head) * e.W + pos) * h;
    store_act<T>(dst, base + c.i, lo);
    store_act<T>(dst, base + c.i + h / 2, hi);
  }
  // four consecutive bf16 values, 8-byte aligned
  __device__ static inline void store4(void* p, int64_t idx, float a, float b, float c, float d) {
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    const bf16x4 v = {(__bf16)a, (__bf16)b, (__bf16)c, (__bf16)d};
    *reinterpret_cast<bf16x4*>((uint16_t*)p + idx) = v;
  }
  // one half (col or col + 32) of a QKV_BIAS pair whose other half is V
  __device__ static inline void row_one(const EpiArgs& e, const ColInfo& c, int col, int rw, int b,
                                        int pos, float v, bool first) {
    const int h = hdim(e);
    const int seg = first ? c.seg : c.seg2, head = first ? c.head : c.head2, i = first ? c.i : c.i2;
    const float bias = first ? c.blo : c.bhi;
    store_act<T>(seg ? e.k : e.q, (((int64_t)b * e.Hq + head) * e.W + pos) * h + i, v + bias);
    (void)col;
    (void)rw;
  }
};

}  // namespace lmgc
