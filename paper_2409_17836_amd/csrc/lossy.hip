// The lossy steps LM-GC is composed with (Sec. 5.4, "Compatibility"):
// top-k sparsification by magnitude, linear quantisation to n-bit indices
// (Eq. 4) and SignSGD sign bits.  All three are streaming passes over a
// float32 vector and bound by HBM bandwidth.
//
// Top-k is a radix select on the magnitude key (the IEEE bits with the sign
// cleared, an unsigned integer whose order is the order of |v| for numbers):
// four passes build a 256-bin histogram of one key byte among the keys that
// match the bytes chosen so far, and a one-block kernel picks the next byte,
// so the threshold key T and the number of keys equal to T that are kept
// never leave the device.  Keys above T are kept; among keys equal to T the
// lowest indices are kept, which needs the count of such keys before each
// element: a per-chunk count, then an ordered pass per chunk with a block
// scan.
#include <mutex>

#include "common.h"

namespace lmgc {
namespace {

constexpr int kThreads = 256;
constexpr int kGridStride = 1024;       // blocks of the grid-stride passes
constexpr int kMaxChunks = 2048;        // ordered chunks of the write pass
constexpr int kTile = kThreads * 4;     // elements per block iteration

struct TopkState {
  uint32_t prefix;  // key bytes chosen so far
  uint32_t mask;    // which bits of prefix are chosen
  uint32_t need;    // keys still to keep among those matching prefix
  uint32_t pad;
};

__device__ inline uint32_t mag_key(float x) { return __float_as_uint(x) & 0x7FFFFFFFu; }

// Four consecutive elements starting at i (a multiple of 4); lanes past n
// read as +0 and are marked invalid through `valid` (number of valid lanes).
__device__ inline float4 load4(const float* __restrict__ v, int64_t i, int64_t n, int& valid) {
  if (i + 4 <= n) {
    valid = 4;
    return *reinterpret_cast<const float4*>(v + i);
  }
  float t[4] = {0.f, 0.f, 0.f, 0.f};
  valid = (int)(n > i ? n - i : 0);
  for (int e = 0; e < valid; e++) t[e] = v[i + e];
  return make_float4(t[0], t[1], t[2], t[3]);
}

__device__ inline void store4(float* __restrict__ o, int64_t i, int valid, float4 x) {
  if (valid == 4) {
    *reinterpret_cast<float4*>(o + i) = x;
  } else {
    const float t[4] = {x.x, x.y, x.z, x.w};
    for (int e = 0; e < valid; e++) o[i + e] = t[e];
  }
}

// ------------------------------------------------------------------ top-k
__global__ void topk_init_kernel(TopkState* st, uint32_t* hist, uint32_t k) {
  hist[threadIdx.x] = 0;
  if (threadIdx.x == 0) *st = TopkState{0u, 0u, k, 0u};
}

__global__ __launch_bounds__(kThreads) void topk_hist_kernel(const float* __restrict__ v, int64_t n,
                                                             const TopkState* __restrict__ st,
                                                             uint32_t* __restrict__ hist, int shift) {
  __shared__ uint32_t lh[256];
  lh[threadIdx.x] = 0;
  __syncthreads();
  const uint32_t prefix = st->prefix, mask = st->mask;
  const int64_t stride = (int64_t)gridDim.x * kThreads * 4;
  for (int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * 4; i < n; i += stride) {
    int valid;
    const float4 x = load4(v, i, n, valid);
    const float t[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < 4; e++) {
      const uint32_t key = mag_key(t[e]);
      if (e < valid && (key & mask) == prefix) atomicAdd(&lh[(key >> shift) & 0xFFu], 1u);
    }
  }
  __syncthreads();
  const uint32_t c = lh[threadIdx.x];
  if (c) atomicAdd(&hist[threadIdx.x], c);
}

// One block of 256: bin b of the byte at `shift` is chosen so that fewer than
// `need` matching keys lie in bins above b and at least `need` in bins >= b.
// The histogram is cleared for the next pass.
__global__ __launch_bounds__(kThreads) void topk_select_kernel(TopkState* st, uint32_t* hist, int shift) {
  __shared__ uint32_t suf[257];
  const int t = threadIdx.x;
  suf[t] = hist[t];
  hist[t] = 0;
  if (t == 0) suf[256] = 0;
  __syncthreads();
  // inclusive suffix sums: suf[t] = sum of bins t..255
  for (int d = 1; d < 256; d <<= 1) {
    const uint32_t add = (t + d < 256) ? suf[t + d] : 0u;
    __syncthreads();
    suf[t] += add;
    __syncthreads();
  }
  const uint32_t need = st->need;
  __syncthreads();
  if (suf[t] >= need && suf[t + 1] < need) {
    st->prefix |= (uint32_t)t << shift;
    st->mask |= 0xFFu << shift;
    st->need = need - suf[t + 1];
  }
}

// Per chunk: how many keys equal the threshold.
__global__ __launch_bounds__(kThreads) void topk_tie_count_kernel(const float* __restrict__ v, int64_t n,
                                                                  int64_t chunk,
                                                                  const TopkState* __restrict__ st,
                                                                  uint32_t* __restrict__ ties) {
  __shared__ uint32_t wsum[kThreads / 64];
  const uint32_t T = st->prefix;
  const int64_t c0 = (int64_t)blockIdx.x * chunk;
  const int64_t c1 = c0 + chunk < n ? c0 + chunk : n;
  uint32_t cnt = 0;
  for (int64_t i = c0 + threadIdx.x * 4; i < c1; i += kTile) {
    int valid;
    const float4 x = load4(v, i, c1, valid);
    const float t[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < 4; e++) cnt += (e < valid && mag_key(t[e]) == T) ? 1u : 0u;
  }
  for (int d = 32; d >= 1; d >>= 1) cnt += __shfl_xor(cnt, d);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t s = 0;
    for (int w = 0; w < kThreads / 64; w++) s += wsum[w];
    ties[blockIdx.x] = s;
  }
}

// Ordered pass over one chunk: keep keys above T, and keys equal to T whose
// rank among equal keys (in index order) is below `need`.
__global__ __launch_bounds__(kThreads) void topk_write_kernel(const float* v, int64_t n, int64_t chunk,
                                                              const TopkState* __restrict__ st,
                                                              const uint32_t* __restrict__ ties,
                                                              float* out) {
  __shared__ uint32_t wtot[2][kThreads / 64];
  __shared__ uint32_t base_sh;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t T = st->prefix, need = st->need;
  // equal keys in the chunks before this one
  uint32_t before = 0;
  for (int b = threadIdx.x; b < (int)blockIdx.x; b += kThreads) before += ties[b];
  for (int d = 32; d >= 1; d >>= 1) before += __shfl_xor(before, d);
  if (lane == 0) wtot[0][wave] = before;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t s = 0;
    for (int w = 0; w < kThreads / 64; w++) s += wtot[0][w];
    base_sh = s;
  }
  __syncthreads();
  uint32_t running = base_sh;
  const int64_t c0 = (int64_t)blockIdx.x * chunk;
  const int64_t c1 = c0 + chunk < n ? c0 + chunk : n;
  int buf = 1;
  for (int64_t i0 = c0; i0 < c1; i0 += kTile) {
    const int64_t i = i0 + threadIdx.x * 4;
    int valid;
    const float4 x = load4(v, i, c1, valid);
    float t[4] = {x.x, x.y, x.z, x.w};
    uint32_t key[4], eq = 0;
#pragma unroll
    for (int e = 0; e < 4; e++) {
      key[e] = mag_key(t[e]);
      eq += (e < valid && key[e] == T) ? 1u : 0u;
    }
    // inclusive scan of eq over the wave, then over the waves
    uint32_t inc = eq;
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t y = __shfl_up(inc, d);
      if (lane >= d) inc += y;
    }
    if (lane == 63) wtot[buf][wave] = inc;
    __syncthreads();
    uint32_t woff = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; w++) {
      const uint32_t s = wtot[buf][w];
      woff += (w < wave) ? s : 0u;
      tot += s;
    }
    uint32_t rank = running + woff + inc - eq;  // equal keys before this thread's first element
#pragma unroll
    for (int e = 0; e < 4; e++) {
      bool keep = e < valid && key[e] > T;
      if (e < valid && key[e] == T) {
        keep = rank < need;
        rank++;
      }
      if (!keep) t[e] = 0.0f;
    }
    if (valid > 0) store4(out, i, valid, make_float4(t[0], t[1], t[2], t[3]));
    running += tot;
    buf ^= 1;  // the next tile writes the other buffer; this one is read by all before then
  }
}

__global__ void fill_zero_kernel(float* __restrict__ out, int64_t n) {
  const int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * 4;
  if (i < n) {
    const int valid = (int)(i + 4 <= n ? 4 : n - i);
    store4(out, i, valid, make_float4(0.f, 0.f, 0.f, 0.f));
  }
}

// ----------------------------------------------------------- quantisation
__global__ __launch_bounds__(kThreads) void minmax_kernel(const float* __restrict__ v, int64_t n,
                                                          LossyMinMax* __restrict__ part) {
  __shared__ LossyMinMax ws[kThreads / 64];
  float mn = INFINITY, mx = -INFINITY;
  uint32_t bad = 0;
  const int64_t stride = (int64_t)gridDim.x * kThreads * 4;
  for (int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * 4; i < n; i += stride) {
    int valid;
    const float4 x = load4(v, i, n, valid);
    const float t[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < 4; e++) {
      if (e < valid) {
        bad += isfinite(t[e]) ? 0u : 1u;
        mn = fminf(mn, t[e]);
        mx = fmaxf(mx, t[e]);
      }
    }
  }
  for (int d = 32; d >= 1; d >>= 1) {
    mn = fminf(mn, __shfl_xor(mn, d));
    mx = fmaxf(mx, __shfl_xor(mx, d));
    bad += __shfl_xor(bad, d);
  }
  if ((threadIdx.x & 63) == 0) ws[threadIdx.x >> 6] = LossyMinMax{mn, mx, bad, 0u};
  __syncthreads();
  if (threadIdx.x == 0) {
    LossyMinMax r = ws[0];
    for (int w = 1; w < kThreads / 64; w++) {
      r.mn = fminf(r.mn, ws[w].mn);
      r.mx = fmaxf(r.mx, ws[w].mx);
      r.nonfinite += ws[w].nonfinite;
    }
    part[blockIdx.x] = r;
  }
}

__global__ __launch_bounds__(kThreads) void minmax_final_kernel(const LossyMinMax* __restrict__ part, int nparts,
                                                                LossyMinMax* __restrict__ res) {
  __shared__ LossyMinMax ws[kThreads / 64];
  float mn = INFINITY, mx = -INFINITY;
  uint32_t bad = 0;
  for (int b = threadIdx.x; b < nparts; b += kThreads) {
    mn = fminf(mn, part[b].mn);
    mx = fmaxf(mx, part[b].mx);
    bad += part[b].nonfinite;
  }
  for (int d = 32; d >= 1; d >>= 1) {
    mn = fminf(mn, __shfl_xor(mn, d));
    mx = fmaxf(mx, __shfl_xor(mx, d));
    bad += __shfl_xor(bad, d);
  }
  if ((threadIdx.x & 63) == 0) ws[threadIdx.x >> 6] = LossyMinMax{mn, mx, bad, 0u};
  __syncthreads();
  if (threadIdx.x == 0) {
    LossyMinMax r = ws[0];
    for (int w = 1; w < kThreads / 64; w++) {
      r.mn = fminf(r.mn, ws[w].mn);
      r.mx = fmaxf(r.mx, ws[w].mx);
      r.nonfinite += ws[w].nonfinite;
    }
    *res = r;
  }
}

// Eq. 4 in float32: one rounding per operation, no contraction, round half
// to even.  span = max - min > 0; every index lands in [0, levels].
__device__ inline uint32_t eq4_index(float x, float mn, float span, float levels) {
#pragma clang fp contract(off)
  const float t = (x - mn) / span;
  return (uint32_t)__builtin_rintf(t * levels);
}

template <typename IdxT>
__global__ __launch_bounds__(kThreads) void quantize_kernel(const float* __restrict__ v, int64_t n, float mn,
                                                            float mx, float levels, IdxT* __restrict__ idx) {
  const int64_t i = ((int64_t)blockIdx.x * kThreads + threadIdx.x) * 4;
  if (i >= n) return;
  int valid;
  const float4 x = load4(v, i, n, valid);
  const float span = mx - mn;
  const float t[4] = {x.x, x.y, x.z, x.w};
  uint32_t q[4];
#pragma unroll
  for (int e = 0; e < 4; e++) q[e] = mx > mn ? eq4_index(t[e], mn, span, levels) : 0u;
  if (valid == 4) {
    if constexpr (sizeof(IdxT) == 1) {
      *reinterpret_cast<uint32_t*>(idx + i) = q[0] | (q[1] << 8) | (q[2] << 16) | (q[3] << 24);
    } else {
      *reinterpret_cast<uint2*>(idx + i) = make_uint2(q[0] | (q[1] << 16), q[2] | (q[3] << 16));
    }
  } else {
    for (int e = 0; e < valid; e++) idx[i + e] = (IdxT)q[e];
  }
}

// ------------------------------------------------------------------- signs
// Thread j packs values 8j..8j+7 into byte j, the first value in bit 7.
__global__ __launch_bounds__(kThreads) void sign_pack_kernel(const float* __restrict__ v, int64_t n,
                                                             uint8_t* __restrict__ out) {
  const int64_t j = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t i = j * 8;
  if (i >= n) return;
  int va, vb;
  const float4 a = load4(v, i, n, va);
  const float4 b = load4(v, i + 4, n, vb);
  const float t[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
  uint32_t byte = 0;
#pragma unroll
  for (int e = 0; e < 8; e++) {
    const uint32_t s = (e < va + vb) ? (__float_as_uint(t[e]) >> 31) : 0u;
    byte |= s << (7 - e);
  }
  out[j] = (uint8_t)byte;
}

inline unsigned blocks_for(int64_t n, int64_t per_block) { return (unsigned)((n + per_block - 1) / per_block); }

}  // namespace

// ------------------------------------------------------------- launchers
size_t lossy_workspace_bytes() {
  return sizeof(TopkState) + 256 * sizeof(uint32_t) + kMaxChunks * sizeof(uint32_t) +
         (kGridStride + 1) * sizeof(LossyMinMax);
}

int64_t topk_chunk(int64_t n) {
  // a multiple of the tile, so that only the vector's last float4 can be partial
  const int64_t per = (n + kMaxChunks - 1) / kMaxChunks;
  const int64_t c = (per + kTile - 1) / kTile * kTile;
  return c > kTile ? c : kTile;
}

hipError_t launch_sparsify_topk(const float* v, int64_t n, int64_t k, float* out, void* ws, hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (k <= 0) {
    hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks_for(n, kTile)), dim3(kThreads), 0, s, out, n);
    return hipGetLastError();
  }
  if (k > n) k = n;
  uint8_t* w = (uint8_t*)ws;
  TopkState* st = (TopkState*)w;
  uint32_t* hist = (uint32_t*)(w + sizeof(TopkState));
  uint32_t* ties = hist + 256;
  hipLaunchKernelGGL(topk_init_kernel, dim3(1), dim3(256), 0, s, st, hist, (uint32_t)k);
  const unsigned g = std::min<unsigned>(kGridStride, blocks_for(n, kTile));
  for (int shift = 24; shift >= 0; shift -= 8) {
    hipLaunchKernelGGL(topk_hist_kernel, dim3(g), dim3(kThreads), 0, s, v, n, (const TopkState*)st, hist,
                       shift);
    hipLaunchKernelGGL(topk_select_kernel, dim3(1), dim3(kThreads), 0, s, st, hist, shift);
  }
  const int64_t chunk = topk_chunk(n);
  const unsigned nchunks = blocks_for(n, chunk);
  hipLaunchKernelGGL(topk_tie_count_kernel, dim3(nchunks), dim3(kThreads), 0, s, v, n, chunk,
                     (const TopkState*)st, ties);
  hipLaunchKernelGGL(topk_write_kernel, dim3(nchunks), dim3(kThreads), 0, s, v, n, chunk, (const TopkState*)st,
                     (const uint32_t*)ties, out);
  return hipGetLastError();
}

hipError_t launch_minmax(const float* v, int64_t n, void* ws, LossyMinMax* res, hipStream_t s) {
  uint8_t* w = (uint8_t*)ws + sizeof(TopkState) + 256 * sizeof(uint32_t) + kMaxChunks * sizeof(uint32_t);
  LossyMinMax* part = (LossyMinMax*)w;
  const unsigned g = std::max(1u, std::min<unsigned>(kGridStride, blocks_for(n, kTile)));
  hipLaunchKernelGGL(minmax_kernel, dim3(g), dim3(kThreads), 0, s, v, n, part);
  hipLaunchKernelGGL(minmax_final_kernel, dim3(1), dim3(kThreads), 0, s, (const LossyMinMax*)part, (int)g, res);
  return hipGetLastError();
}

// ------------------------------------------------ library-owned scratch
// The scratch of lmgc_sparsify_topk_noalloc: a file-scope device array, one
// copy on every GPU the library runs on, held from module load until the
// process ends.  In host code `scratch` names a host-side stand-in, not a
// device address; the current device's copy is found with
// hipGetSymbolAddress (once per device, then cached) and only that address
// reaches the kernels.  The top-k kernels clear what must start at zero
// (state and histogram) themselves and write every tie count before reading
// it, so what an earlier call left there does not matter; calls that overlap
// on one GPU (two streams at once) race on it.
constexpr size_t kScratchBytes = 32768;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

hipError_t lossy_scratch(void** ptr, size_t* bytes) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  *bytes = kScratchBytes;
  return hipSuccess;
}

LossyMinMax* lossy_minmax_slot(void* ws) {
  return (LossyMinMax*)((uint8_t*)ws + sizeof(TopkState) + 256 * sizeof(uint32_t) +
                        kMaxChunks * sizeof(uint32_t) + kGridStride * sizeof(LossyMinMax));
}

hipError_t launch_quantize_linear(const float* v, int64_t n, int bits, float mn, float mx, void* idx,
                                  hipStream_t s) {
  if (n == 0) return hipSuccess;
  const float levels = (float)((1u << bits) - 1u);
  if (bits <= 8)
    hipLaunchKernelGGL(quantize_kernel<uint8_t>, dim3(blocks_for(n, kTile)), dim3(kThreads), 0, s, v, n, mn, mx,
                       levels, (uint8_t*)idx);
  else
    hipLaunchKernelGGL(quantize_kernel<uint16_t>, dim3(blocks_for(n, kTile)), dim3(kThreads), 0, s, v, n, mn, mx,
                       levels, (uint16_t*)idx);
  return hipGetLastError();
}

hipError_t launch_sign_pack(const float* v, int64_t n, uint8_t* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const int64_t nbytes = (n + 7) / 8;
  hipLaunchKernelGGL(sign_pack_kernel, dim3(blocks_for(nbytes, kThreads)), dim3(kThreads), 0, s, v, n, out);
  return hipGetLastError();
}

}  // namespace lmgc
