// Serialisation kernel: values -> hex-digit + separator token windows
// (Sec. 4, "Serialization").  Each thread produces four consecutive tokens of
// the window range and stores them with one 16-byte and one 4-byte store;
// the value bytes it needs are read through the cache (nine tokens share
// one float32).  The work is HBM-bound: 4/9 B read and 5 B written per token
// (one separator token; 4/10 B and 5 B with two).
#include "common.h"

namespace lmgc {
namespace {

struct SerialDev {
  int64_t n_values, n_tokens, nbytes;
  int32_t bpv, bpg, msb_first, W;
  int32_t pad_id, nsep, sep[2];  // separator tokens after each group (bins 16, 17)
  int32_t hex[16];
};

__device__ inline void token_at(const uint8_t* __restrict__ vals, const SerialDev& p, int64_t t,
                                int32_t& tok, uint8_t& sym) {
  if (t >= p.n_tokens) {
    tok = p.pad_id;
    sym = 255;
    return;
  }
  int64_t byte;
  int sep = -1, low = 0;
  if (p.bpg > 0) {
    const int64_t G = 2 * (int64_t)p.bpg + p.nsep;  // a full group's tokens
    const int64_t g = t / G;
    const int32_t r = (int32_t)(t - g * G);
    const int64_t b0 = g * p.bpg;
    const int64_t left = p.nbytes - b0;
    const int32_t nb = left < p.bpg ? (int32_t)left : p.bpg;
    if (r >= 2 * nb) {
      sep = r - 2 * nb;  // 0 or 1
      byte = 0;
    } else {
      byte = b0 + (r >> 1);
      low = r & 1;
    }
  } else {
    byte = t >> 1;
    low = (int)(t & 1);
  }
  if (sep >= 0) {
    tok = p.sep[sep];
    sym = (uint8_t)(16 + sep);
    return;
  }
  const int64_t i = byte / p.bpv;
  const int32_t k = (int32_t)(byte - i * p.bpv);
  const int32_t mem = p.msb_first ? (p.bpv - 1 - k) : k;
  const uint8_t b = vals[i * p.bpv + mem];
  const int nib = low ? (b & 15) : (b >> 4);
  tok = p.hex[nib];
  sym = (uint8_t)nib;
}

__global__ void serialize_kernel(const uint8_t* __restrict__ vals, SerialDev p, int64_t t0,
                                 int64_t n_local, int32_t* __restrict__ tokens,
                                 uint8_t* __restrict__ sym) {
  const int64_t base = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (base >= n_local) return;
  int32_t tk[4];
  uint8_t sy[4];
#pragma unroll
  for (int e = 0; e < 4; e++) {
    if (base + e < n_local) token_at(vals, p, t0 + base + e, tk[e], sy[e]);
  }
  if (base + 4 <= n_local) {
    *reinterpret_cast<int4*>(tokens + base) = make_int4(tk[0], tk[1], tk[2], tk[3]);
    if (sym) {
      uint32_t packed = (uint32_t)sy[0] | ((uint32_t)sy[1] << 8) | ((uint32_t)sy[2] << 16) |
                        ((uint32_t)sy[3] << 24);
      *reinterpret_cast<uint32_t*>(sym + base) = packed;
    }
  } else {
    for (int e = 0; e < 4 && base + e < n_local; e++) {
      tokens[base + e] = tk[e];
      if (sym) sym[base + e] = sy[e];
    }
  }
}

}  // namespace

hipError_t launch_serialize(const void* values, int64_t n_values, const lmgc_serial_params& sp,
                            int64_t first_window, int64_t n_windows, int32_t* tokens,
                            uint8_t* sym, hipStream_t s) {
  SerialDev p;
  p.n_values = n_values;
  p.bpv = sp.bytes_per_value;
  p.bpg = sp.bytes_per_group;
  p.msb_first = sp.msb_first;
  p.W = sp.window;
  p.pad_id = sp.pad_id;
  p.nsep = sp.sep2_id >= 0 ? 2 : 1;
  p.sep[0] = sp.sep_id;
  p.sep[1] = sp.sep2_id;
  for (int i = 0; i < 16; i++) p.hex[i] = sp.hex_ids[i];
  p.nbytes = n_values * (int64_t)sp.bytes_per_value;
  p.n_tokens = 2 * p.nbytes + (sp.bytes_per_group > 0
                                   ? (p.nbytes + sp.bytes_per_group - 1) / sp.bytes_per_group * p.nsep
                                   : 0);
  const int64_t t0 = first_window * sp.window;
  const int64_t n_local = n_windows * sp.window;
  if (n_local == 0) return hipSuccess;
  const int threads = 256;
  const int64_t nthreads = (n_local + 3) / 4;
  const int64_t blocks = (nthreads + threads - 1) / threads;
  if (blocks > INT32_MAX) return hipErrorInvalidValue;
  hipLaunchKernelGGL(serialize_kernel, dim3((unsigned)blocks), dim3(threads), 0, s,
                     (const uint8_t*)values, p, t0, n_local, tokens, sym);
  return hipGetLastError();
}

}  // namespace lmgc
