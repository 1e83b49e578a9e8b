// Causal self-attention of the decoder (softmax(q.k / sqrt(hd)) v over keys
// <= query), tiled through LDS with an online softmax so the W x W score
// matrix never exists (the FlashAttention idea the paper lists as a
// throughput lever in its discussion section).
//
// bf16 kernel (CDNA4 matrix cores).  A workgroup of four 64-wide waves owns
// 128 queries of one (window, head); each wave 32 queries.  Tiles of 64 keys
// of K [key][dim] and of V^T [dim][key] (the QKV projection writes V
// transposed) go to LDS with direct global->LDS loads into two buffers each,
// K one tile ahead of V, with one barrier per tile; each buffer is its own
// __shared__ array so the compiler can tell the in-flight loads of one buffer
// from the reads of the other.  Each wave issues the S MFMAs of the next tile
// before the softmax of the current one, so the exponentials overlap matrix
// work.  The wave
// computes S^T = K Q^T with v_mfma_f32_32x32x16_bf16, so each lane holds one
// query's scores in its own registers: the row max / row sum need one
// cross-lane exchange (lane ^ 32) instead of a 32-lane reduction.  The K rows
// are fed to the MFMA in a permuted order so that the score registers are,
// without any shuffle, the B operand of O^T += V^T P^T.  Softmax statistics
// are float32 in base 2 (the 1/sqrt(hd) scale folded into the exponent); a
// query's reference maximum moves, and O is rescaled, only when a score
// exceeds it by more than 2^8 in probability; P is rounded to bf16 for the
// second product and the row sums are taken over the rounded P (v_dot2 with
// ones); O is normalised at the end.
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
typedef __attribute__((address_space(3))) void* lds_ptr_t;

__device__ inline bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// LDS swizzles.  One ds_read_b128 cycle serves 16 lanes (64 banks x 4 B =
// 256 B), so the 16 rows such a group reads must land on 16 distinct
// 16-byte slots modulo 256 B.
//  - K tile [key][hd], rows of hd*2 bytes: the S^T operand lanes 0..15 read
//    keys {0-3, 8-11, 4-7, 12-15} (+16): for hd = 128 (256-byte rows) the
//    slot is chunk ^ (key & 15); for hd = 64 (128-byte rows) rows of equal
//    parity share a half, so the slot is chunk ^ ((key >> 1) & 7).
//  - V^T tile [dim][64 keys], 128-byte rows: slot = chunk ^ ((dim >> 1) & 7).
template <int HD>
__device__ inline int kswz(int key) { return HD == 128 ? (key & 15) : ((key >> 1) & 7); }
__device__ inline int vswz(int d) { return (d >> 1) & 7; }

// Raw buffer resource (gfx9 layout: stride 0, dword 3 = 0x00020000) over
// `bytes` bytes at p.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}

// key held by score register r of a lane in half h (see the S^T layout).
__device__ inline int key_of_reg(int r, int h) { return r < 8 ? 8 * h + r : 16 + 8 * h + (r - 8); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two floats -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ inline uint32_t pack2(float a, float b) {
  const bf16x2 v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

constexpr float kLazy = 8.0f;  // log2 headroom of the lazily moved softmax reference

// Item k of an XCD's range [r0, r1) of (head, query block) items (item u:
// head u / nqb, block nqb - 1 - u % nqb, so a head's blocks come longest
// first).  The long blocks (block >= S) keep that head-major order, which
// keeps a head's K/V in the XCD's L2 while its blocks run; the short ones
// (block < S) follow, longest first across the range's heads, so the
// range ends with short items and no CU waits long on the last ones.
__device__ inline bool xcd_item(int k, int r0, int r1, int nqb, int S, int& h, int& qb) {
  if (k >= r1 - r0) return false;
  const int h0 = r0 / nqb, h1 = (r1 - 1) / nqb;
  for (int hh = h0; hh <= h1; hh++) {
    const int ja = hh == h0 ? r0 - hh * nqb : 0;
    const int jb = hh == h1 ? r1 - hh * nqb : nqb;
    const int nl = max(0, min(jb, nqb - S) - ja);  // long items of this head
    if (k < nl) {
      h = hh;
      qb = nqb - 1 - (ja + k);
      return true;
    }
    k -= nl;
  }
  for (int j = nqb - S; j < nqb; j++)
    for (int hh = h0; hh <= h1; hh++) {
      const int ja = hh == h0 ? r0 - hh * nqb : 0;
      const int jb = hh == h1 ? r1 - hh * nqb : nqb;
      if (j < ja || j >= jb) continue;
      if (k == 0) {
        h = hh;
        qb = nqb - 1 - j;
        return true;
      }
      k--;
    }
  return false;
}

// DQM: decoding-step mode (only query dq of each window; see below).
template <int HD, bool DQM>
__global__ __launch_bounds__(256, 2) void attn_bf16_kernel(const uint16_t* __restrict__ q,
                                                           const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ vt,
                                                           uint16_t* __restrict__ o, int Hq,
                                                           int Hkv, int W, float sl2, int dq) {
  constexpr int BQ = 128, BKV = 64, KCH = HD / 8, NKS = HD / 16, NOB = HD / 32;
  constexpr int KROWS = 1024 / (HD * 2);          // K rows per 1 KB direct load
  constexpr int NKL = BKV * HD * 2 / 1024 / 4;    // direct K loads per wave and tile
  // two LDS buffers: tile t+1 is filled while tile t is read
  __shared__ u32x4 sK0[BKV * KCH], sK1[BKV * KCH];
  __shared__ u32x4 sV0[HD * 8], sV1[HD * 8];  // V^T: [dim][64 keys]

  const int nqb = (W + BQ - 1) / BQ;
  int qb, h;
  const int b = blockIdx.z;
  if (DQM) {
    // a decoding step runs only the block of position dq
    qb = dq / BQ;
    h = blockIdx.y;
  } else {
    // Workgroup x of window b runs on XCD x % 8 (gridDim.x is a multiple of
    // 8).  Each XCD gets a contiguous range of the window's (head, query
    // block) items, so all blocks of a head read its K and V through one L2
    // (spread over the eight L2s, the K/V tiles came from HBM); the order
    // within the range is xcd_item's.
    const int per = gridDim.x / 8, x = (int)blockIdx.x % 8;
    const int r0 = x * per, r1 = min(r0 + per, nqb * Hq);
    if (!xcd_item((int)blockIdx.x / 8, r0, r1, nqb, nqb / 4, h, qb)) return;
  }
  const int kvh = h * Hkv / Hq;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, c32 = lane & 31;
  // A decoding step needs only query dq.  Every wave then takes the 32
  // queries of dq's wave (the same scores and softmax, bit for bit, in each)
  // and accumulates one of the NOB 32-dim blocks of P V (wave w: block w, in
  // oacc[0]; waves past NOB only load), so a tile's critical path is one
  // wave's S MFMAs and softmax plus a quarter of the P V MFMAs.  Each block's
  // chain is the one the whole-window pass runs for that query.
  const int q0 = DQM ? (dq / 32) * 32 : qb * BQ + wave * 32;
  const int myq = q0 + c32;
  const bool computes = !DQM || wave < NOB;
  constexpr int NACC = DQM ? 1 : NOB;  // accumulated output blocks
  // dims of accumulated block i
  auto oblk = [&](int i) __attribute__((always_inline)) { return DQM ? wave : i; };

  const uint16_t* Qp = q + (int64_t)(b * Hq + h) * W * HD;
  const uint16_t* Kp = k + (int64_t)(b * Hkv + kvh) * W * HD;
  const uint16_t* Vp = vt + (int64_t)(b * Hkv + kvh) * HD * W;

  bf16x8 qf[NKS];
  {
    const int qr = min(myq, W - 1);
#pragma unroll
    for (int ks = 0; ks < NKS; ks++)
      qf[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(Qp + (int64_t)qr * HD + 16 * ks + 8 * half));
  }
  f32x16 oacc[NACC];
#pragma unroll
  for (int i = 0; i < NACC; i++) oacc[i] = f32x16{};
  float m_i = -INFINITY, l_i = 0.f;
  const float lazy = kLazy / sl2;

  // MFMA row rho = 8a + 4g + c (a = rho/8, g = (rho/4)&1, c = rho&3) takes key
  // 16 (a/2) + 8 g + 4 (a&1) + c of its 32-key block.
  const int pa = c32 >> 3, pg = (c32 >> 2) & 1, pc = c32 & 3;
  const int kperm = 16 * (pa >> 1) + 8 * pg + 4 * (pa & 1) + pc;

  // K: direct global->LDS loads.  Load i of wave w covers tile rows
  // (w*NKL + i)*KROWS .. +KROWS; lane l lands at row +l/KCH, slot l%KCH and
  // fetches the chunk the swizzle puts there.
  auto kload = [&](u32x4* sKb, int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NKL; i++) {
      const int key = (wave * NKL + i) * KROWS + lane / KCH;
      const int ch = (lane % KCH) ^ kswz<HD>(key);
      const uint16_t* src = Kp + (int64_t)min(k0 + key, W - 1) * HD + ch * 8;
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (lds_ptr_t)(sKb + (wave * NKL + i) * 64), 16, 0, 0);
    }
  };
  // V^T direct loads: HD rows (dims) x 128 B per tile = HD/8 wave loads;
  // load i of wave w covers rows (w*NVD + i)*8 .. +8, lane l -> row +l/8, slot
  // l%8.  W % 8 == 0, so an 8-key chunk lies wholly before or after the end
  // of the window; chunks after it re-read the last chunk (finite values
  // that meet probability exactly 0) so that no load leaves the row.
  constexpr int NVD = HD * 128 / 1024 / 4;
  auto vtload = [&](u32x4* sVb, int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NVD; i++) {
      const int d = (wave * NVD + i) * 8 + lane / 8;
      const int ch = (lane % 8) ^ vswz(d);
      const uint16_t* src = Vp + (int64_t)d * W + min(k0 + ch * 8, W - 8);
      __builtin_amdgcn_global_load_lds((const void*)src,
                                       (lds_ptr_t)(sVb + (wave * NVD + i) * 64), 16, 0, 0);
    }
  };
  // Full tiles (k0 + BKV <= W) load through buffer resources over this
  // (window, kv head)'s K and V^T, with lane offsets fixed for the whole loop
  // and the tile's offset in a scalar; a ragged last tile takes the clamped
  // loads above.
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(Kp, W * HD * 2);
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(Vp, HD * W * 2);
  // (fixed array sizes: with sizes that depend on HD the host compilation
  // pass silently dropped this kernel's launch stub)
  static_assert(NKL <= 4 && NVD <= 4, "offset arrays hold four loads");
  int kvo[4], vvo[4];
#pragma unroll
  for (int i = 0; i < NKL; i++) {
    const int key = (wave * NKL + i) * KROWS + lane / KCH;
    kvo[i] = (key * HD + ((lane % KCH) ^ kswz<HD>(key)) * 8) * 2;
  }
#pragma unroll
  for (int i = 0; i < NVD; i++) {
    const int d = (wave * NVD + i) * 8 + lane / 8;
    vvo[i] = (d * W + ((lane % 8) ^ vswz(d)) * 8) * 2;
  }
  auto kload_full = [&](u32x4* sKb, int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NKL; i++)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_ptr_t)(sKb + (wave * NKL + i) * 64), 16,
                                               kvo[i], k0 * HD * 2, 0, 0);
  };
  auto vtload_full = [&](u32x4* sVb, int k0) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NVD; i++)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_ptr_t)(sVb + (wave * NVD + i) * 64), 16,
                                               vvo[i], k0 * 2, 0, 0);
  };
  auto kload_any = [&](u32x4* sKb, int k0) __attribute__((always_inline)) {
    if (k0 + BKV <= W) kload_full(sKb, k0);
    else kload(sKb, k0);
  };
  auto vtload_any = [&](u32x4* sVb, int k0) __attribute__((always_inline)) {
    if (k0 + BKV <= W) vtload_full(sVb, k0);
    else vtload(sVb, k0);
  };
  const int kend = min(W, qb * BQ + BQ);
  const int ntiles = (kend + BKV - 1) / BKV;
  // S^T of key tile t (64 keys, two 32-key blocks) from the K tile in sKc.
  auto qk = [&](const u32x4* sKc, f32x16& s0, f32x16& s1) __attribute__((always_inline)) {
    s0 = f32x16{};
    s1 = f32x16{};
#pragma unroll
    for (int ks = 0; ks < NKS; ks++) {
      const int ch = 2 * ks + half;
      const int key0 = kperm, key1 = 32 + kperm;
      const bf16x8 ka = as_bf16x8(sKc[key0 * KCH + (ch ^ kswz<HD>(key0))]);
      const bf16x8 kb = as_bf16x8(sKc[key1 * KCH + (ch ^ kswz<HD>(key1))]);
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[ks], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb, qf[ks], s1, 0, 0, 0);
    }
  };
  // softmax of tile t's scores (masking, lazy reference, exponentials, row
  // sums) and O^T += V^T P^T with the V^T tile in sVc
  auto softmax_pv = [&](int t, f32x16& s0, f32x16& s1, const u32x4* sVc)
      __attribute__((always_inline)) {
    const int k0 = t * BKV;
    // scores stay unscaled: p = 2^(s*sl2 - m*sl2) with m the reference maximum
    float mx = -INFINITY;
    const bool diag = k0 + BKV - 1 > q0;  // some key of the tile may lie after a query
    if (diag) {
#pragma unroll
      for (int r = 0; r < 16; r++) {
        const int key = k0 + key_of_reg(r, half);
        if (key > myq) s0[r] = -INFINITY;
        if (key + 32 > myq) s1[r] = -INFINITY;
      }
    }
#pragma unroll
    for (int r = 0; r < 16; r++) mx = fmaxf(fmaxf(mx, s0[r]), s1[r]);  // v_max3
    // Lazy rescaling: a query's reference point m_i moves only when one of
    // its scores exceeds it by more than kLazy/sl2 (probabilities stay below
    // 2^kLazy), and then to the maximum over both lane halves; both halves
    // hold the same m_i.  A wave-wide ballot finds out whether any lane needs
    // this; only then are the halves' maxima exchanged.  Either way a query
    // rescales exactly when its own maximum passes the threshold.
    if (__ballot(mx > m_i + lazy)) {
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      if (mx > m_i + lazy) {
        const float alpha = __builtin_amdgcn_exp2f((m_i - mx) * sl2);
        l_i *= alpha;
#pragma unroll
        for (int i = 0; i < NACC; i++) oacc[i] *= alpha;
        m_i = mx;
      }
    }
    const float nms = -m_i * sl2;
#pragma unroll
    for (int r = 0; r < 16; r++) {
      s0[r] = __builtin_amdgcn_exp2f(fmaf(s0[r], sl2, nms));
      s1[r] = __builtin_amdgcn_exp2f(fmaf(s1[r], sl2, nms));
    }
    // P rounded to bf16; the row sum is taken over these rounded values (the
    // ones P V uses), two per v_dot2 against (1, 1), over this half's keys
    // (the halves are added at the end)
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    bf16x8 pf[4];
#pragma unroll
    for (int kk = 0; kk < 4; kk++) {
      const f32x16& sv = (kk < 2) ? s0 : s1;
      const int r0 = (kk & 1) * 8;
      // (the dot2 operands are the packed words themselves: reading them back
      // out of the u32x4 below made this compiler feed element 0 to all four)
      const uint32_t w0 = pack2(sv[r0 + 0], sv[r0 + 1]), w1 = pack2(sv[r0 + 2], sv[r0 + 3]);
      const uint32_t w2 = pack2(sv[r0 + 4], sv[r0 + 5]), w3 = pack2(sv[r0 + 6], sv[r0 + 7]);
      l_i = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w0), ones, l_i, false);
      l_i = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w1), ones, l_i, false);
      l_i = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w2), ones, l_i, false);
      l_i = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w3), ones, l_i, false);
      const u32x4 u = {w0, w1, w2, w3};
      pf[kk] = as_bf16x8(u);
    }
    // k-step outer: the NOB accumulations of a step are independent chains
#pragma unroll
    for (int kk = 0; kk < 4; kk++) {
      bf16x8 va[NACC];
#pragma unroll
      for (int i = 0; i < NACC; i++) {
        const int d = oblk(i) * 32 + c32;
        va[i] = as_bf16x8(sVc[d * 8 + ((2 * kk + half) ^ vswz(d))]);
      }
#pragma unroll
      for (int i = 0; i < NACC; i++)
        oacc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[i], pf[kk], oacc[i], 0, 0, 0);
    }
  };
  // Software pipeline, one step per key tile t: K runs one tile ahead of V.
  // At step t, K(t+1) and V(t) are in LDS; the wave issues the S MFMAs of tile
  // t+1 first, so the matrix cores work on them while it does the softmax of
  // tile t (whose scores it computed in the previous step), then the P V
  // MFMAs of tile t.  Meanwhile K(t+2) and V(t+1) stream into the buffers of
  // K(t) and V(t-1), which every wave finished with before the step's barrier.
  // A tile lying entirely after the wave's 32 queries is skipped.
  const int tlast = min(ntiles - 1, (q0 + 31) / BKV);  // last tile this wave needs
  f32x16 sa0, sa1, sb0, sb1;                          // scores of two tiles in flight
  auto step = [&](int t, f32x16& c0, f32x16& c1, f32x16& n0, f32x16& n1, const u32x4* sKn,
                  const u32x4* sVc, u32x4* sKf, u32x4* sVf) __attribute__((always_inline)) {
    __syncthreads();
    if (t + 2 < ntiles) kload_any(sKf, (t + 2) * BKV);
    if (t + 1 < ntiles) vtload_any(sVf, (t + 1) * BKV);
    __builtin_amdgcn_sched_barrier(0);
    if (computes && t + 1 <= tlast) qk(sKn, n0, n1);
    if (computes && t <= tlast) softmax_pv(t, c0, c1, sVc);
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  };
  kload_any(sK0, 0);
  vtload_any(sV0, 0);
  if (ntiles > 1) kload_any(sK1, BKV);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (computes) qk(sK0, sa0, sa1);
  int t = 0;
  for (; t + 2 <= ntiles; t += 2) {
    step(t, sa0, sa1, sb0, sb1, sK1, sV0, sK0, sV1);
    step(t + 1, sb0, sb1, sa0, sa1, sK0, sV1, sK1, sV0);
  }
  if (t < ntiles) step(t, sa0, sa1, sb0, sb1, sK1, sV0, sK0, sV1);

  l_i += __shfl_xor(l_i, 32, 64);
  if (DQM ? myq == dq && computes : myq < W) {
    const float inv = 1.0f / l_i;
    uint16_t* orow = o + ((int64_t)b * (DQM ? 1 : W) + (DQM ? 0 : myq)) * (int64_t)(Hq * HD) + h * HD;
#pragma unroll
    for (int i = 0; i < NACC; i++) {
#pragma unroll
      for (int a = 0; a < 4; a++) {
        const int d = oblk(i) * 32 + 8 * a + 4 * half;
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
                                                      int W, float scale, int dq) {
  __shared__ float sK[64][HD + 1];
  __shared__ float sV[64][HD + 1];
  const int h = blockIdx.y, b = blockIdx.z;
  const int kvh = h * Hkv / Hq;
  const int qblk = dq >= 0 ? dq / 64 : (int)blockIdx.x;  // a decoding step: dq's block only
  const int myq = qblk * 64 + threadIdx.x;
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
  const int kend = min(W, qblk * 64 + 64);
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
  if (dq >= 0 ? myq == dq : myq < W) {
    float* orow = o + ((int64_t)b * (dq >= 0 ? 1 : W) + (dq >= 0 ? 0 : myq)) * (int64_t)(Hq * HD) + h * HD;
#pragma unroll
    for (int i = 0; i < HD; i++) orow[i] = acc[i] / l;
  }
}

}  // namespace

hipError_t launch_attention_bf16(const uint16_t* q, const uint16_t* k, const uint16_t* vt,
                                 uint16_t* o, int B, int Hq, int Hkv, int W, int hd, int dq,
                                 hipStream_t s) {
  if (B <= 0 || W <= 0) return hipSuccess;
  if (W % 8 || dq >= W) return hipErrorInvalidValue;
  const int items = (W + 127) / 128 * Hq;  // (head, 128-query block) items per window
  const dim3 grid = dq >= 0 ? dim3(1, Hq, B) : dim3((items + 7) / 8 * 8, 1, B), block(256);
  const float sl2 = (float)(1.4426950408889634 / sqrt((double)hd));
  if (hd == 128 && dq >= 0)
    hipLaunchKernelGGL((attn_bf16_kernel<128, true>), grid, block, 0, s, q, k, vt, o, Hq, Hkv, W, sl2, dq);
  else if (hd == 128)
    hipLaunchKernelGGL((attn_bf16_kernel<128, false>), grid, block, 0, s, q, k, vt, o, Hq, Hkv, W, sl2, dq);
  else if (hd == 64 && dq >= 0)
    hipLaunchKernelGGL((attn_bf16_kernel<64, true>), grid, block, 0, s, q, k, vt, o, Hq, Hkv, W, sl2, dq);
  else if (hd == 64)
    hipLaunchKernelGGL((attn_bf16_kernel<64, false>), grid, block, 0, s, q, k, vt, o, Hq, Hkv, W, sl2, dq);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}


hipError_t launch_attention_f32(const float* q, const float* k, const float* v, float* o, int B,
                                int Hq, int Hkv, int W, int hd, int dq, hipStream_t s) {
  if (B <= 0 || W <= 0) return hipSuccess;
  if (dq >= W) return hipErrorInvalidValue;
  const dim3 grid(dq >= 0 ? 1 : (W + 63) / 64, Hq, B), block(64);
  const float scale = (float)(1.0 / sqrt((double)hd));
  switch (hd) {
    case 16:
      hipLaunchKernelGGL(attn_f32_kernel<16>, grid, block, 0, s, q, k, v, o, Hq, Hkv, W, scale, dq);
      break;
    case 32:
      hipLaunchKernelGGL(attn_f32_kernel<32>, grid, block, 0, s, q, k, v, o, Hq, Hkv, W, scale, dq);
      break;
    case 48:
      hipLaunchKernelGGL(attn_f32_kernel<48>, grid, block, 0, s, q, k, v, o, Hq, Hkv, W, scale, dq);
      break;
    case 64:
      hipLaunchKernelGGL(attn_f32_kernel<64>, grid, block, 0, s, q, k, v, o, Hq, Hkv, W, scale, dq);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace lmgc
