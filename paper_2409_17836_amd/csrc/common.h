// Internal declarations shared by the liblmgc translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/lmgc.h"

namespace lmgc {

// ------------------------------------------------------------ bf16 helpers
__host__ __device__ inline float bf16_to_f32(uint16_t b) {
  union { uint32_t u; float f; } v;
  v.u = (uint32_t)b << 16;
  return v.f;
}

// Round to nearest even; NaN stays NaN.
__host__ __device__ inline uint16_t f32_to_bf16(float f) {
  union { uint32_t u; float f; } v;
  v.f = f;
  uint32_t u = v.u;
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// ------------------------------------------------------- epilogue selectors
// What the matrix-product kernels do with each output pair (col, col + 32).
enum EpiKind : int {
  EPI_STORE_F32 = 0,   // C[row, col] = v                          (float)
  EPI_RESID = 1,       // h[row, col] += v (+ bias[col])            (float)
  EPI_QKV_ROPE = 2,    // RoPE on q/k pairs, scatter to q, k, v      (act)
  EPI_QKV_BIAS = 3,    // + bias, scatter to q, k, v (no RoPE)       (act)
  EPI_SWIGLU = 4,      // out[row, f] = silu(gate) * up              (act)
  EPI_BIAS_GELU = 5,   // out[row, col] = gelu_tanh(v + bias[col])   (act)
  EPI_HEAD = 6,        // LM head: per-(row, 64-column group) max and
                       // sum of exp, and the alphabet columns' logits (float)
};

// Arguments of every epilogue (unused fields ignored).
struct EpiArgs {
  int kind;
  int M, N;            // valid output extent (N = real columns)
  // EPI_STORE_F32 / EPI_RESID
  float* c;            // [M, ldc]
  int ldc;
  const void* bias;    // [N] model dtype, nullable
  // attention layout scatter: q [B,Hq,W,hd], k [B,Hkv,W,hd]; v [B,Hkv,hd,W]
  // (transposed) for bf16 models, [B,Hkv,W,hd] for f32 models
  void* q;
  void* k;
  void* v;
  int W, Hq, Hkv, hd;
  const float2* rope;  // [max_pos, hd/2] (cos, sin)
  // row -> (window, position): step == 0 (the zero-initialised default): row
  // r is position r % W of window r / W (a batch of whole windows); step != 0:
  // row r is window r at position dpos (one decoding step)
  int step, dpos;
  // SWIGLU / GELU output
  void* out;           // [M, ld_out]
  int ld_out;
  // HEAD: za[row, a] = logit of column alpha_ids[a] (a < n_alpha); part[row,
  // g] = (max, sum of exp(z - max)) over the valid columns of group g
  // (columns 64 g .. 64 g + 63), nullable; ngroups = padded N / 64
  float* za;
  int ld_za;
  float2* part;
  int ngroups;
  int n_alpha;
  int alpha_ids[LMGC_NALPHA_MAX];
};

// ------------------------------------------------------------ launchers
// All launchers return hipError_t of the launch.
hipError_t launch_serialize(const void* values, int64_t n_values, const lmgc_serial_params& p,
                            int64_t first_window, int64_t n_windows, int32_t* tokens,
                            uint8_t* sym, hipStream_t s);

// Token ids outside [0, vocab) are clamped (callers validate them).
// dpos < 0: rows b*W + j of B whole windows (token of row j is BOS for j = 0,
// else tokens[b, j-1]); dpos >= 0: row b is window b at position dpos, whose
// input token is BOS for dpos = 0, else tokens[b].
hipError_t launch_embed(const int32_t* tokens, int B, int W, int bos_id, const void* tok_emb,
                        const void* pos_emb, int d, int vocab, int dtype, int dpos, float* h,
                        hipStream_t s);

// y = norm(h) (rms if ln_bias == nullptr && !layernorm) in model dtype.
hipError_t launch_norm(const float* h, int M, int d, const void* gain, const void* bias,
                       int layernorm, float eps, int dtype, void* y, hipStream_t s);

// Weight matrices of bf16 models are stored in MFMA blocks: for B [N, K]
// (N % 16 == 0, K % 32 == 0), block (n / 16, k / 32) holds 16 rows x 32 k as
// 1 KB in the order the 64 lanes of a 16x16x32 MFMA take their B operand:
// element (n, k) sits at block ((n/16) * (K/32) + k/32), lane
// (n % 16) + 16 * ((k % 32) / 8), position k % 8.  Blocks of one 16-row
// group are consecutive, so a tile of rows n0 .. n0+255 starts at n0 * K, as
// in row-major order.
__host__ __device__ inline int64_t blocked_index(int64_t n, int64_t k, int64_t K) {
  return ((n >> 4) * (K >> 5) + (k >> 5)) * 512 + ((n & 15) + 16 * ((k & 31) >> 3)) * 8 + (k & 7);
}

// blocked_b: B in MFMA blocks (the model's weights) or row-major [N, K] (only
// for the float32 store, the exposed operator).
hipError_t launch_gemm_bf16(const uint16_t* A, const uint16_t* B, int M, int N_pad, int K,
                            const EpiArgs& e, hipStream_t s, bool blocked_b = true);
hipError_t launch_gemm_f32(const float* A, const float* B, int M, int N_pad, int K,
                           const EpiArgs& e, hipStream_t s);
// Decoding step: M <= 32 rows, each output element accumulated exactly as
// launch_gemm_bf16 accumulates it (same MFMA, operand layout and k order);
// B in MFMA blocks.
hipError_t launch_gemm_bf16_rows(const uint16_t* A, const uint16_t* B, int M, int N_pad, int K,
                                 const EpiArgs& e, hipStream_t s);

// dq < 0: all queries of B windows, o [B*W, Hq*hd].  dq >= 0: only query dq
// of each window (same per-query arithmetic), o [B, Hq*hd].
hipError_t launch_attention_bf16(const uint16_t* q, const uint16_t* k, const uint16_t* vt,
                                 uint16_t* o, int B, int Hq, int Hkv, int W, int hd, int dq,
                                 hipStream_t s);
hipError_t launch_attention_f32(const float* q, const float* k, const float* v, float* o,
                                int B, int Hq, int Hkv, int W, int hd, int dq, hipStream_t s);

// The LM head's tables from what its EPI_HEAD epilogue wrote: the partials
// part [M, ngroups] merge, in a fixed order, into the row's log-sum-exp over
// the whole vocabulary; za [M, ld_za] holds the n_alpha (17 or 18) alphabet
// logits.  -> cdf [M, A + 2], logp [M, A] (nullable).  renorm: the tables
// are renormalised over the alphabet (the log-sum-exp runs over za alone,
// part is not read); otherwise full-vocabulary tables with an escape bin.
hipError_t launch_head_tables(const float2* part, int ngroups, const float* za, int ld_za, int M,
                              int n_alpha, uint32_t total, int renorm, uint32_t* cdf, float* logp,
                              hipStream_t s);

// dst [rows, cols]: row r < n_alpha = head row alpha_ids[r] (host array),
// the remaining rows zero.  Rows are cols * elem_bytes bytes (multiple of 4).
// elem_bytes == 2: head and dst are in MFMA blocks (rows % 16 == 0).
hipError_t launch_alpha_head(const void* head, const int32_t* alpha_ids, int n_alpha, int rows, int cols,
                             int elem_bytes, void* dst, hipStream_t s);

// Lossy steps (lossy.hip).  The workspace holds the top-k select state, the
// per-chunk tie counts and the min/max partials; its size does not depend on n.
struct LossyMinMax {
  float mn, mx;
  uint32_t nonfinite;  // values that are NaN or infinite
  uint32_t pad;
};
size_t lossy_workspace_bytes();
hipError_t launch_sparsify_topk(const float* v, int64_t n, int64_t k, float* out, void* ws, hipStream_t s);
// Writes the vector's LossyMinMax to res (device memory, e.g. lossy_minmax_slot(ws)).
hipError_t launch_minmax(const float* v, int64_t n, void* ws, LossyMinMax* res, hipStream_t s);
LossyMinMax* lossy_minmax_slot(void* ws);
// Address (on the current device) and size of the library-owned device
// scratch that lmgc_sparsify_topk_noalloc uses in place of a workspace.
hipError_t lossy_scratch(void** ptr, size_t* bytes);
hipError_t launch_quantize_linear(const float* v, int64_t n, int bits, float mn, float mx, void* idx,
                                  hipStream_t s);
hipError_t launch_sign_pack(const float* v, int64_t n, uint8_t* out, hipStream_t s);

// dst[r, :] = srcs.p[idx[r] >> 28][(idx[r] & 0x0fffffff), :] for r < rows;
// idx[r] == -1 gives a zero row.  Rows are cols * elem_bytes bytes (multiple of 4).
struct GatherSrcs {
  const void* p[4];
};
hipError_t launch_gather_rows(GatherSrcs srcs, const int32_t* idx, int rows, int cols,
                              int elem_bytes, void* dst, hipStream_t s);
// The same gather of bf16 rows, written in MFMA blocks (rows % 16 == 0,
// cols % 32 == 0); idx == nullptr: row r of srcs.p[0] (no reordering).
hipError_t launch_gather_rows_blocked(GatherSrcs srcs, const int32_t* idx, int rows, int cols,
                                      void* dst, hipStream_t s);

}  // namespace lmgc
