// bf16 matrix product on CDNA4 matrix cores: C[M, N] = A[M, K] * B[N, K]^T
// with float32 accumulation, followed by a fused epilogue (epilogue.h).
//
// Both operands are K-contiguous: activations row-major, weights [out, in]
// in MFMA blocks (BLKB; common.h: 16 rows x 32 k per 1 KB in the order the
// lanes take their operand) or row-major (the exposed float32-store product).
// Tile: 256 x 256 output per 256-thread workgroup: four 64-wide waves, one
// per SIMD; wave (wm, wn) owns rows wm*128 .. +128 and columns wn*128 .. +128
// as 8 x 8 blocks of v_mfma_f32_16x16x32_bf16.  The 256 accumulator
// registers of a lane live in the AGPR file: the MFMAs are issued as inline
// assembly with the accumulator as an AGPR operand, which keeps the
// compiler from shuttling accumulators between the two register files.
// A 128 x 128 wave tile reads a third fewer LDS bytes per flop than 128 x 64.
//
// Operand pipeline.  K advances in stages of 64 (two 32-wide k-steps).
// Stages go to LDS with buffer loads straight into LDS (no staging
// registers): one operand through a ring of three 32 KB buffers, the other
// through two (5 x 32 KB = the whole 160 KB LDS).  The ring holds A by
// default and B when RB is set: the longer prefetch goes to the operand
// whose panels miss L2 more often.  A wide weight matrix (N >= 2K: gate/up,
// QKV, LM head) has new B panels for every wave of tiles, while an XCD's A
// panels repeat; for a narrow one (the N = d products that add into the
// residual) B stays cached and A streams.
//
// Schedule of stage s (one wave; every memory operation sits between two
// MFMAs, in this order):
//  - k-step 0: 64 MFMAs on fragments already in registers; after every
//    fourth, one LDS read of k-step 1's fragments; after every eighth, one
//    load of the ring operand of stage s + 2 (into the ring buffer stage
//    s - 1 used);
//  - k-step 1: 32 MFMAs; then the wave waits for its own loads of stage
//    s + 1 and for its LDS reads, and the workgroup meets at a barrier,
//    which makes stage s + 1 visible and ends every read of stage s;
//  - the last 32 MFMAs; the first 16 of them carry the LDS reads of stage
//    s + 1's first k-step (done before the stage ends) and the loads of the
//    double-buffered operand of stage s + 2 (into the buffer stage s has
//    just released).
// So the matrix cores have work queued on both sides of the barrier, and the
// loads of one operand have a stage, the other's a stage and a half, to
// arrive.
//
// A row-major 256 x 64 operand tile is stored as rows of eight 16-byte
// chunks; chunk c of row r sits at slot c ^ ((r >> 1) & 7): the 16 lanes that
// one ds_read_b128 cycle serves read 16 consecutive rows, and the swizzle
// gives every (row parity, slot) pair once, i.e. all 64 banks.  A blocked B
// tile is its 32 blocks copied as they are: lane l reads 16 bytes at 16 l of
// a block, conflict-free without a swizzle.  The buffer resources are per
// tile with the tile's valid rows as their size: rows past M read as zero
// (and only feed outputs that are never stored).
//
// Determinism: every output element is the same fixed sequence of MFMA
// accumulations over k regardless of M, of the tile it sits in, and of the
// values of other rows, so the LM's per-position tables do not depend on the
// batch or window length (lossless decoding relies on this).
//
// Workgroup -> tile order: the hardware deals workgroups to the 8 XCDs
// round-robin; ids are remapped so each XCD walks a contiguous range of a
// row-grouped tile order (4 row tiles per group, 8 when the ring holds B),
// which keeps the A and B panels the co-resident workgroups of an XCD share
// in that XCD's L2.
#include "epilogue.h"

namespace lmgc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kThreads = 256;
// row tiles per group of the tile order: 4 when the ring holds A, 8 when it
// holds B (measured best at the 7B shape)
constexpr int kGroupM = 4, kGroupMB = 8;
constexpr int kXcds = 8;
// MFMAs of a stage that follow its barrier
constexpr int kAfterBarrier = 32;
// s_waitcnt immediates: vmcnt(n) with expcnt and lgkmcnt at their maxima
// (vmcnt bits 3:0 and 15:14), and lgkmcnt(0) alone
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | 0xF70; }
constexpr int kLgkm0 = 0xC07F;

__device__ inline int slot(int row, int chunk) { return row * 8 + (chunk ^ ((row >> 1) & 7)); }

__device__ inline bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

template <int GM>
__device__ inline bool map_tile(int bid, int nblocks, int ntm, int ntn, int& tm, int& tn) {
  const int total = ntm * ntn;
  const int per = nblocks / kXcds;  // nblocks is a multiple of kXcds
  const int t = (bid % kXcds) * per + bid / kXcds;
  if (t >= total) return false;
  const int in_group = GM * ntn;
  const int g = t / in_group;
  const int first = g * GM;
  const int gs = min(ntm - first, GM);
  const int r = t - g * in_group;
  tm = first + r % gs;
  tn = r / gs;
  return true;
}

// Raw buffer resource (gfx9 layout: stride 0, dword 3 = 0x00020000) over
// `bytes` bytes at p; loads at offsets >= bytes return zero.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* p, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, bytes, 0x00020000);
}

template <int KIND, int HD, bool RB, bool BLKB>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_kernel(
    const uint16_t* __restrict__ A, const uint16_t* __restrict__ Bw, int M, int K, int ntm,
    int ntn, EpiArgs e) {
  // sR*: the ring of three (A, or B if RB); sD*: the double buffer
  __shared__ u32x4 sR0[BM * 8], sR1[BM * 8], sR2[BM * 8];  // 3 x 32 KB
  __shared__ u32x4 sD0[BN * 8], sD1[BN * 8];               // 2 x 32 KB

  int tm, tn;
  if (!map_tile<RB ? kGroupMB : kGroupM>(blockIdx.x, gridDim.x, ntm, ntn, tm, tn)) return;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A + (int64_t)m0 * K, min(M - m0, BM) * K * 2);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(Bw + (int64_t)n0 * K, BN * K * 2);
  // A stage of one operand is 32 loads of 1 KB; wave w issues q = 8 w + i.
  // Row-major: load q fills LDS rows 8q .. 8q + 7; lane l lands at row
  // 8q + l/8, slot l%8 (the hardware writes lane l at base + 16 l), so it
  // fetches the logical chunk the swizzle puts there.  The row is part of the
  // lane offset (for the bounds check), the stage's k offset is scalar.
  // BLKB: a stage's B tile is 32 blocks of 1 KB (16 row groups x two 32-wide
  // k chunks); load q copies block q = 16 kc + j (row group j, chunk kc of
  // the stage) to the same place in LDS, where lane l's 16 bytes are already
  // its MFMA operand.
  int voffa[8], voffb[8];
#pragma unroll
  for (int i = 0; i < 8; i++) {
    const int q = wave * 8 + i;
    const int row = q * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ ((row >> 1) & 7);
    voffa[i] = (row * K + lc * 8) * 2;
    const int kc = q >> 4, j = q & 15;
    voffb[i] = BLKB ? ((j * (K / 32) + kc) * 1024 + lane * 16) : voffa[i];
  }

  // zeroed through empty asm statements, so that the zeros are in the AGPRs
  // before the first (inline) MFMA in program order
  f32x4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; i++)
#pragma unroll
    for (int j = 0; j < 8; j++) asm volatile("" : "=a"(acc[i][j]) : "0"(f32x4{}));

  // MFMA operands: lane l supplies row (l & 15) of a 16-row block and the
  // 8 k-values of chunk (l >> 4) of the 32-wide k-step.
  const int arow0 = wm * 128 + (lane & 15), brow0 = wn * 128 + (lane & 15), kq = lane >> 4;

  auto ldA = [&](u32x4* sa, int i, int k0) __attribute__((always_inline)) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr_t)(sa + (wave * 8 + i) * 64), 16, voffa[i],
                                             k0 * 2, 0, 0);
  };
  auto ldB = [&](u32x4* sb, int i, int k0) __attribute__((always_inline)) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_ptr_t)(sb + (wave * 8 + i) * 64), 16, voffb[i],
                                             BLKB ? k0 * 32 : k0 * 2, 0, 0);
  };
  auto ld_r = [&](u32x4* buf, int i, int k0) __attribute__((always_inline)) {
    if (RB) ldB(buf, i, k0);
    else ldA(buf, i, k0);
  };
  auto ld_d = [&](u32x4* buf, int i, int k0) __attribute__((always_inline)) {
    if (RB) ldA(buf, i, k0);
    else ldB(buf, i, k0);
  };
  // Fragments of a k-step: fa/fb for k-step 0 of a stage, ga/gb for k-step 1.
  // Read r of a k-step: the eight B fragments first (the first eight MFMAs
  // need all of them), then the A fragments.
  bf16x8 fa[8], fb[8], ga[8], gb[8];
  auto rd = [&](bf16x8* xa, bf16x8* xb, const u32x4* sa, const u32x4* sb, int ks, int r)
      __attribute__((always_inline)) {
    const int ch = ks * 4 + kq;
    if (r < 8)
      xb[r] = as_bf16x8(BLKB ? sb[(ks * 16 + wn * 8 + r) * 64 + lane] : sb[slot(brow0 + 16 * r, ch)]);
    else
      xa[r - 8] = as_bf16x8(sa[slot(arow0 + 16 * (r - 8), ch)]);
  };
  // MFMA n of a k-step: block (n / 8, n % 8)
  auto mma = [&](const bf16x8* xa, const bf16x8* xb, int n) __attribute__((always_inline)) {
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0"
                 : "+a"(acc[n >> 3][n & 7])
                 : "v"(xa[n >> 3]), "v"(xb[n & 7]));
  };
  auto barrier = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };

  // One stage on buffers (sa, sb); (na, nb) are the next stage's.  NEXT: a
  // next stage exists (barrier, its first reads); LOADS: stage s + 2 exists
  // and is loaded (the ring operand into lr, the double-buffered one into
  // ldb, both at k offset k2).
  auto stage = [&](auto next_tag, auto loads_tag, const u32x4* sa, const u32x4* sb, const u32x4* na,
                   const u32x4* nb, u32x4* lr, u32x4* ldb, int k2) __attribute__((always_inline)) {
    constexpr bool NEXT = decltype(next_tag)::value, LOADS = decltype(loads_tag)::value;
#pragma unroll
    for (int n = 0; n < 64; n++) {
      mma(fa, fb, n);
      if ((n & 3) == 3) rd(ga, gb, sa, sb, 1, n >> 2);
      if (LOADS && (n & 7) == 7) ld_r(lr, n >> 3, k2);
    }
#pragma unroll
    for (int n = 0; n < 64 - kAfterBarrier; n++) mma(ga, gb, n);
    if constexpr (NEXT) {
      // loads in flight, oldest first: R(s+1), D(s+1), then R(s+2) if
      // LOADS; stage s + 1 needs the first two
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(LOADS ? 8 : 0));
      __builtin_amdgcn_s_waitcnt(kLgkm0);
      barrier();
#pragma unroll
      for (int n = 64 - kAfterBarrier; n < 64; n++) {
        const int r = n - (64 - kAfterBarrier);
        mma(ga, gb, n);
        if (r < 16) rd(fa, fb, na, nb, 0, r);
        if (LOADS && r < 16 && (r & 1) == 0) ld_d(ldb, r >> 1, k2);
      }
    } else {
#pragma unroll
      for (int n = 64 - kAfterBarrier; n < 64; n++) mma(ga, gb, n);
    }
  };
  // Stage s reads ring buffer s % 3 and double buffer s % 2; it loads R(s+2)
  // into ring buffer (s + 2) % 3 and D(s+2) into double buffer s % 2.  The
  // prologue loads stages 0 and 1.
  const int nk = K / BK;
#pragma unroll
  for (int i = 0; i < 8; i++) ld_r(sR0, i, 0);
#pragma unroll
  for (int i = 0; i < 8; i++) ld_d(sD0, i, 0);
  if (nk > 1) {
#pragma unroll
    for (int i = 0; i < 8; i++) ld_r(sR1, i, BK);
#pragma unroll
    for (int i = 0; i < 8; i++) ld_d(sD1, i, BK);
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(16));
  } else {
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  }
  barrier();
  // rotating buffer roles: cr/nr/lr the ring buffers of stages s, s + 1 and
  // s + 2; cd/nd the double buffers of stages s and s + 1
  u32x4 *cr = sR0, *nr = sR1, *lr = sR2, *cd = sD0, *nd = sD1;
#define LMGC_A(R, D) (RB ? (D) : (R))
#define LMGC_B(R, D) (RB ? (R) : (D))
#pragma unroll
  for (int r = 0; r < 16; r++) rd(fa, fb, LMGC_A(cr, cd), LMGC_B(cr, cd), 0, r);
  auto rotate = [&]() __attribute__((always_inline)) {
    u32x4* t = cr;
    cr = nr;
    nr = lr;
    lr = t;
    t = cd;
    cd = nd;
    nd = t;
  };
  int s = 0;
  for (; s + 2 < nk; s++) {
    stage(std::true_type{}, std::true_type{}, LMGC_A(cr, cd), LMGC_B(cr, cd), LMGC_A(nr, nd),
          LMGC_B(nr, nd), lr, cd, (s + 2) * BK);
    rotate();
  }
  if (s + 1 < nk) {
    stage(std::true_type{}, std::false_type{}, LMGC_A(cr, cd), LMGC_B(cr, cd), LMGC_A(nr, nd),
          LMGC_B(nr, nd), lr, cd, 0);
    rotate();
  }
  stage(std::false_type{}, std::false_type{}, LMGC_A(cr, cd), LMGC_B(cr, cd), LMGC_A(nr, nd),
        LMGC_B(nr, nd), lr, cd, 0);
#undef LMGC_A
#undef LMGC_B
  // The compiler does not know the inline MFMAs write the accumulators, so
  // it cannot space their first reads: 32 wait states cover the longest
  // MFMA-write -> VALU-read distance.
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
#pragma unroll
  for (int i = 0; i < 8; i++)
#pragma unroll
    for (int j = 0; j < 8; j++) asm volatile("" : "+a"(acc[i][j]));

  // Epilogue, one 64-column half of the wave's tile at a time: half h holds
  // blocks acc[.][4h .. 4h + 3], columns n0 + 128 wn + 64 h + 16 j + (lane &
  // 15).  16 x 16 block layout: lane holds column (lane & 15) and rows
  // 4 (lane >> 4) + r, r = 0..3.  Blocks j and j + 2 of a half give the
  // column pair (col, col + 32).  Rows 4 (lane >> 4) + 0..3 never straddle a
  // window (W is a multiple of 8).
  // The reads an epilogue needs (residual, RoPE table) for row block i + 1
  // are issued before the stores of block i.  Whole tiles (all but the
  // ragged edges) take a path without row and column checks, so the
  // epilogue stays one basic block.
  using E = Epi<uint16_t, KIND, HD>;
  using Pre4 = typename E::Pre4;
  const int W = e.W > 0 ? e.W : 1;
  constexpr bool kQkv = KIND == EPI_QKV_ROPE || KIND == EPI_QKV_BIAS;
  constexpr bool kStaged = KIND == EPI_RESID;
  // V columns of a whole tile (bf16 QKV): a half's 128 rows x 64 columns go
  // through LDS, transposed, so that each V^T row (a dim of a head) is
  // written as 16-byte pieces of 8 consecutive positions.  The region of
  // (wave, half) is 16 KB of the operand buffers: 64 rows (columns) of 128
  // positions, 16-byte chunks swizzled by chunk ^ (row & 15).  Needs
  // W % 128 == 0 so the rows lie in one window.
  auto v_transposed = [&](auto h_tag, const ColInfo& ci0, const ColInfo& ci1, int cw)
      __attribute__((always_inline)) {
    constexpr int H = decltype(h_tag)::value;
    u32x4* reg = (wave == 0 ? sR0 : wave == 1 ? sR1 : wave == 2 ? sR2 : sD0) + H * 1024;
    char* regb = reinterpret_cast<char*>(reg);
    const float bl0 = KIND == EPI_QKV_BIAS ? ci0.blo : 0.f, bh0 = KIND == EPI_QKV_BIAS ? ci0.bhi : 0.f;
    const float bl1 = KIND == EPI_QKV_BIAS ? ci1.blo : 0.f, bh1 = KIND == EPI_QKV_BIAS ? ci1.bhi : 0.f;
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
#pragma unroll
    for (int i = 0; i < 8; i++)
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const int kap = (lane & 15) + 16 * j, rho = 16 * i + 4 * kq;
        const float bias = j == 0 ? bl0 : j == 1 ? bl1 : j == 2 ? bh0 : bh1;
        const f32x4 a = acc[i][4 * H + j];
        const bf16x4 val = {(__bf16)(a[0] + bias), (__bf16)(a[1] + bias), (__bf16)(a[2] + bias),
                            (__bf16)(a[3] + bias)};
        const int off = kap * 256 + (((rho >> 3) ^ (kap & 15)) << 4) + (rho & 7) * 2;
        *reinterpret_cast<bf16x4*>(regb + off) = val;
      }
    const int Hv = KIND == EPI_QKV_ROPE ? e.Hkv : e.Hq;
    const int h = HD ? HD : e.hd;
    const int row0 = m0 + wm * 128, b = row0 / W, pos0 = row0 - b * W;
    // first V column: after q and k (Hq and Hkv heads for RoPE models,
    // Hq and Hq for GPT-2's fused projection)
    const int vcol0 = cw - (KIND == EPI_QKV_ROPE ? e.Hq + e.Hkv : 2 * e.Hq) * h;
#pragma unroll
    for (int t = 0; t < 16; t++) {
      const int c = lane + 64 * t, kap = c >> 4, ch = c & 15;
      const u32x4 val = reg[kap * 16 + (ch ^ (kap & 15))];
      const int cc = vcol0 + kap, head = cc / h, dim = cc - head * h;
      uint16_t* dst = (uint16_t*)e.v + (((int64_t)b * Hv + head) * h + dim) * W + pos0 + ch * 8;
      *reinterpret_cast<u32x4*>(dst) = val;
    }
  };
  // q and k columns of a whole tile (bf16 QKV, W % 128 == 0, head dim 64 or
  // 128): the wave's 128 columns are whole heads of one segment (one head of
  // 128 dims, or two of 64) and its 128 rows consecutive positions of one
  // window, so its output is one (hd 128) or two (hd 64) contiguous blocks
  // of 128 positions x hd in the [B, H, W, hd] layout.  The rotated (or
  // biased) bf16 values go to the wave's 32 KB of the operand buffers in
  // that layout, 16-byte chunks of a row swizzled by chunk ^ swz(row), and
  // are then read back and stored as 16-byte pieces: each store instruction
  // writes 1 KB of consecutive memory (instead of 4 rows x 32 bytes of
  // 2-byte pieces).  Values and rounding are those of Epi::rows4.
  auto qk_staged = [&](int head0, int seg) __attribute__((always_inline)) {
    constexpr int h = HD == 64 ? 64 : 128;
    constexpr int RC = h / 8;  // 16-byte chunks per row
    u32x4* reg = wave == 0 ? sR0 : wave == 1 ? sR1 : wave == 2 ? sR2 : sD0;
    char* regb = reinterpret_cast<char*>(reg);
    auto swz = [](int row) __attribute__((always_inline)) { return (2 * (row >> 2)) & (RC - 1); };
    auto put = [&](int blk, int row, int dim, float v) __attribute__((always_inline)) {
      const int off = (blk * 128 + row) * (RC * 16) + (((dim >> 3) ^ swz(row)) << 4) + (dim & 7) * 2;
      *reinterpret_cast<__bf16*>(regb + off) = (__bf16)v;  // round to nearest even
    };
    const int cw0 = n0 + wn * 128;
    const int row0 = m0 + wm * 128, b = row0 / W, pos0 = row0 - b * W;
    ColInfo ci[2][2];
#pragma unroll
    for (int H = 0; H < 2; H++)
#pragma unroll
      for (int jp = 0; jp < 2; jp++) ci[H][jp] = E::column(e, cw0 + 64 * H + 16 * jp + (lane & 15));
    Pre4 q[2][2];
#pragma unroll
    for (int H = 0; H < 2; H++)
#pragma unroll
      for (int jp = 0; jp < 2; jp++)
        q[H][jp] = E::template pre4<true>(e, ci[H][jp], cw0 + 64 * H + 16 * jp + (lane & 15),
                                          row0 + 4 * kq, M, pos0 + 4 * kq);
#pragma unroll
    for (int i = 0; i < 8; i++) {
      Pre4 nq[2][2];
#pragma unroll
      for (int H = 0; H < 2; H++)
#pragma unroll
        for (int jp = 0; jp < 2; jp++) {
          nq[H][jp] = q[H][jp];
          if (i + 1 < 8)
            nq[H][jp] = E::template pre4<true>(e, ci[H][jp], cw0 + 64 * H + 16 * jp + (lane & 15),
                                               row0 + 16 * (i + 1) + 4 * kq, M,
                                               pos0 + 16 * (i + 1) + 4 * kq);
        }
#pragma unroll
      for (int H = 0; H < 2; H++)
#pragma unroll
        for (int jp = 0; jp < 2; jp++) {
          const ColInfo& c = ci[H][jp];
          const f32x4 xl = acc[i][4 * H + jp], xh = acc[i][4 * H + jp + 2];
#pragma unroll
          for (int r = 0; r < 4; r++) {
            const int row = 16 * i + 4 * kq + r;
            if constexpr (KIND == EPI_QKV_ROPE) {
              float lo, hi;
              rope_rot(xl[r], xh[r], q[H][jp].x[r], q[H][jp].y[r], lo, hi);
              put(c.head - head0, row, c.i, lo);
              put(c.head - head0, row, c.i + h / 2, hi);
            } else {
              put(c.head - head0, row, c.i, xl[r] + c.blo);
              put(c.head2 - head0, row, c.i2, xh[r] + c.bhi);
            }
          }
        }
#pragma unroll
      for (int H = 0; H < 2; H++)
#pragma unroll
        for (int jp = 0; jp < 2; jp++) q[H][jp] = nq[H][jp];
    }
    const int Hs = KIND == EPI_QKV_ROPE && seg == 1 ? e.Hkv : e.Hq;
    uint16_t* base = (uint16_t*)(seg == 0 ? e.q : e.k);
#pragma unroll
    for (int t = 0; t < 32; t++) {
      const int c = lane + 64 * t, blk = c / (128 * RC), rem = c - blk * (128 * RC);
      const int row = rem / RC, ch = rem - row * RC;
      const u32x4 val = reg[(blk * 128 + row) * RC + (ch ^ swz(row))];
      uint16_t* dst = base + ((((int64_t)b * Hs + head0 + blk) * W + pos0 + row) * h + ch * 8);
      *reinterpret_cast<u32x4*>(dst) = val;
    }
  };
  // residual add of a whole tile: the float32 accumulators of one 64-column
  // half at a time go to the wave's LDS region as [row][64] (16-byte chunks
  // swizzled by chunk ^ 4 ((row >> 2) & 3)); each lane then reads 4
  // consecutive columns of a row back and adds them to the residual stream
  // with 16-byte loads and stores (4 rows x 256 B per instruction), in the
  // arithmetic of Epi::row_in.  The residual rows are loaded in batches of 8
  // loads per lane, three batches ahead of the one being added, so the loads
  // of the second half are in flight while the first half is stored.
  auto resid_staged = [&]() __attribute__((always_inline)) {
    u32x4* reg = wave == 0 ? sR0 : wave == 1 ? sR1 : wave == 2 ? sR2 : sD0;
    float* regf = reinterpret_cast<float*>(reg);
    auto swz = [](int row) __attribute__((always_inline)) { return (4 * (row >> 2)) & 15; };
    const int row0 = m0 + wm * 128, ch = lane & 15;
    // the residual rows through a buffer resource over the wave's 128 rows:
    // lane offset (row lane / 16, columns 4 ch ..), row 4 t a scalar offset
    const __amdgpu_buffer_rsrc_t rc =
        make_rsrc(e.c + (int64_t)row0 * e.ldc + n0 + wn * 128, 128 * e.ldc * 4);
    const int vo0 = ((lane >> 4) * e.ldc + 4 * ch) * 4;
    float bs[2][4];
#pragma unroll
    for (int H = 0; H < 2; H++)
#pragma unroll
      for (int u = 0; u < 4; u++)
        bs[H][u] = e.bias ? load_par<uint16_t>(e.bias, n0 + wn * 128 + 64 * H + 4 * ch + u) : 0.f;
    // batch q: half q / 4, loads t = 8 (q % 4) .. + 8 of that half
    u32x4 x[8][8];
    auto load_batch = [&](int q) __attribute__((always_inline)) {
#pragma unroll
      for (int u = 0; u < 8; u++)
        x[q][u] = __builtin_amdgcn_raw_buffer_load_b128(rc, vo0 + 256 * (q >> 2),
                                                        16 * (8 * (q & 3) + u) * e.ldc, 0);
    };
    auto to_lds = [&](int H) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < 8; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) {
          const f32x4 a = acc[i][4 * H + j];
          const int cc = 16 * j + (lane & 15);
#pragma unroll
          for (int r = 0; r < 4; r++) {
            const int row = 16 * i + 4 * kq + r;
            regf[row * 64 + (((cc >> 2) ^ swz(row)) << 2) + (cc & 3)] = a[r];
          }
        }
    };
    auto add_batch = [&](int q) __attribute__((always_inline)) {
      const int H = q >> 2;
#pragma unroll
      for (int u = 0; u < 8; u++) {
        const int t = 8 * (q & 3) + u, row = 4 * t + (lane >> 4);
        const f32x4 a = reinterpret_cast<const f32x4*>(reg)[row * 16 + (ch ^ swz(row))];
        const f32x4 xo = __builtin_bit_cast(f32x4, x[q][u]);
        f32x4 y;
#pragma unroll
        for (int k = 0; k < 4; k++) y[k] = resid_add(xo[k], a[k], bs[H][k]);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, y), rc, vo0 + 256 * H,
                                               16 * t * e.ldc, 0);
      }
    };
    load_batch(0);
    load_batch(1);
    load_batch(2);
    to_lds(0);
#pragma unroll
    for (int q = 0; q < 8; q++) {
      if (q == 4) to_lds(1);  // after the first half's reads, in LDS order
      add_batch(q);
      if (q + 3 < 8) load_batch(q + 3);
    }
  };
  auto half = [&](auto h_tag, auto full_tag) __attribute__((always_inline)) {
    constexpr int H = decltype(h_tag)::value;
    constexpr bool FULL = decltype(full_tag)::value;
    const int cw = n0 + wn * 128 + 64 * H;  // first column of the half
    const int c0 = cw + (lane & 15);
    if constexpr (KIND == EPI_HEAD) {
      // the half's 64 columns are group cw / 64; lane holds columns c0 + 16 j
      // of rows 4 kq + r of every 16-row block
      const int g = cw >> 6;
      bool ok[4];
      int aidx[4];
#pragma unroll
      for (int j = 0; j < 4; j++) {
        ok[j] = c0 + 16 * j < e.N;
        aidx[j] = ok[j] ? alpha_index(e, c0 + 16 * j) : -1;
      }
      const bool any_alpha = __any(aidx[0] >= 0 || aidx[1] >= 0 || aidx[2] >= 0 || aidx[3] >= 0);
#pragma unroll
      for (int i = 0; i < 8; i++) {
        float z[4][4];
#pragma unroll
        for (int r = 0; r < 4; r++)
#pragma unroll
          for (int j = 0; j < 4; j++) z[r][j] = ok[j] ? acc[i][4 * H + j][r] : -INFINITY;
        head_rows4(e, z, aidx, any_alpha, m0 + wm * 128 + 16 * i + 4 * kq, M, g, lane & 15);
      }
    } else {
      ColInfo ci0 = E::column(e, c0), ci1 = E::column(e, c0 + 16);
      if constexpr (kQkv) {
        // bf16 models have head_dim 64 or 128, so q, k and v and every head
        // are whole 64-column groups: a half's columns share segment and
        // head.  Saying so turns the epilogue's q/k/v branches into scalar
        // ones.
        auto uniform = [](ColInfo& c) __attribute__((always_inline)) {
          c.valid = __builtin_amdgcn_readfirstlane((int)c.valid) != 0;
          c.seg = __builtin_amdgcn_readfirstlane(c.seg);
          c.seg2 = __builtin_amdgcn_readfirstlane(c.seg2);
          c.head = __builtin_amdgcn_readfirstlane(c.head);
          c.head2 = __builtin_amdgcn_readfirstlane(c.head2);
        };
        uniform(ci0);
        uniform(ci1);
        if constexpr (FULL) {
          if (W % 128 == 0 && ci0.seg == 2) {
            v_transposed(h_tag, ci0, ci1, cw);
            return;
          }
        }
      }
      const int rb = m0 + wm * 128 + 4 * kq;
      Pre4 q0 = E::template pre4<FULL>(e, ci0, c0, rb, M, rb % W);
      Pre4 q1 = E::template pre4<FULL>(e, ci1, c0 + 16, rb, M, rb % W);
#pragma unroll
      for (int i = 0; i < 8; i++) {
        const int r0 = rb + 16 * i;
        const int b = r0 / W, p0 = r0 - b * W;
        Pre4 n0q = q0, n1q = q1;
        if (i + 1 < 8) {
          const int r1 = r0 + 16, p1 = r1 % W;
          n0q = E::template pre4<FULL>(e, ci0, c0, r1, M, p1);
          n1q = E::template pre4<FULL>(e, ci1, c0 + 16, r1, M, p1);
        }
        const f32x4 x0 = acc[i][4 * H + 0], x1 = acc[i][4 * H + 1];
        const f32x4 x2 = acc[i][4 * H + 2], x3 = acc[i][4 * H + 3];
        const float a0[4] = {x0[0], x0[1], x0[2], x0[3]};
        const float a2[4] = {x2[0], x2[1], x2[2], x2[3]};
        const float a1[4] = {x1[0], x1[1], x1[2], x1[3]};
        const float a3[4] = {x3[0], x3[1], x3[2], x3[3]};
        E::template rows4<FULL>(e, ci0, c0, r0, M, b, p0, a0, a2, q0);
        E::template rows4<FULL>(e, ci1, c0 + 16, r0, M, b, p0, a1, a3, q1);
        q0 = n0q;
        q1 = n1q;
      }
    }
  };
  auto epilogue = [&](auto full_tag) __attribute__((always_inline)) {
    constexpr bool FULL = decltype(full_tag)::value;
    // the V halves reuse the operand buffers: every wave has finished
    // reading them
    if constexpr (FULL && kStaged) {
      // the LDS regions still hold operands other waves may be reading
      barrier();
      resid_staged();
      return;
    }
    if constexpr (FULL && kQkv) {
      if (W % 128 == 0) {
        barrier();
        if constexpr (HD == 64 || HD == 128) {
          // segment and head of the wave's first and last 64 columns
          const ColInfo c0 = E::column(e, n0 + wn * 128), c1 = E::column(e, n0 + wn * 128 + 64);
          const int s0 = __builtin_amdgcn_readfirstlane(c0.seg);
          const int s1 = __builtin_amdgcn_readfirstlane(c1.seg);
          if (s0 < 2 && s1 == s0) {
            qk_staged(__builtin_amdgcn_readfirstlane(c0.head), s0);
            return;
          }
        }
      }
    }
    half(std::integral_constant<int, 0>{}, full_tag);
    half(std::integral_constant<int, 1>{}, full_tag);
  };
  bool full = m0 + BM <= M && n0 + BN <= e.N;
  if constexpr (kStaged) {
    // the staged residual add moves 16-byte pieces of rows; other tiles take
    // the checked path (kernel arguments: the same for every wave)
    full = full && (reinterpret_cast<uintptr_t>(e.c) & 15) == 0 && e.ldc % 4 == 0;
  }
  if (full) epilogue(std::true_type{});
  else epilogue(std::false_type{});
}

// Decoding step (M <= 32 rows: one row per window).  Every wave accumulates
// one 16-column block for NRB blocks of 16 rows (NRB = 1 for M <= 16, else
// 2; both row blocks take the same weight fragment) and runs, for every
// output element, the same chain as gemm_bf16_kernel: 16x16x32 bf16 MFMAs
// over the 32-wide k chunks in increasing order, lane l holding row (l & 15)
// of its row block and k values 8*(l >> 4) .. +8 of a chunk.  So a row's
// outputs equal, bit for bit, what the tiled kernel gives that row in a batch
// of whole windows.  Operands come straight from global memory (the step
// streams the weights once), kRowsPf chunks ahead (fewer with two row
// blocks, for registers).  The step is bound by how many weight bytes each
// wave has in flight, so the waves are spread over as many CUs as the
// epilogue allows.  NWR waves per workgroup:
//  - 4: 64 columns; waves 2 and 3 hand their accumulators to waves 0 and 1
//    through LDS, which run the epilogue on the (col, col + 32) pairs (QKV:
//    the RoPE pairs and the transposed V stores);
//  - 2: the two blocks c and c + 32 of one pair (gate/up, GELU, float32
//    store);
//  - 1: one block, for the residual add, which pairs nothing (N = d = 4096 has
//    only 256 blocks: one wave on each CU instead of 64 four-wave groups).
constexpr int kRowsPf = 16;
constexpr int kRowsMax = 32;

template <int KIND, int HD, int NWR, int NRB>
__global__ __launch_bounds__(64 * NWR) void gemm_bf16_rows_kernel(const uint16_t* __restrict__ A,
                                                                  const uint16_t* __restrict__ Bw,
                                                                  int M, int K, EpiArgs e) {
  constexpr int PF = NRB == 1 ? kRowsPf : 12;  // chunks in flight
  // accumulators handed over: to the pair's first block (QKV: waves 2, 3 to
  // 0, 1), or all to wave 0 (HEAD: waves 1..3, the group's blocks j = 1..3)
  __shared__ f32x4 part[NWR == 4 ? 3 : 1][NRB][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int c;  // this wave's block
  if (NWR == 4) c = blockIdx.x * 64 + wave * 16;
  else if (NWR == 2) c = (blockIdx.x >> 1) * 64 + (blockIdx.x & 1) * 16 + wave * 32;
  else c = blockIdx.x * 16;
  const int r = lane & 15, kq = lane >> 4;
  // rows past M re-read row M - 1; they only feed outputs that are not stored
  const u32x4* pa[NRB];
#pragma unroll
  for (int rb = 0; rb < NRB; rb++)
    pa[rb] = reinterpret_cast<const u32x4*>(A + (int64_t)min(16 * rb + r, M - 1) * K + kq * 8);
  // B in MFMA blocks: the wave's 16 rows are one contiguous stream of 1 KB
  // blocks, lane l's 16 bytes at 16 l of each
  const int nkc = K / 32;  // A chunk kc starts at u32x4 index 4 * kc
  const u32x4* pb = reinterpret_cast<const u32x4*>(Bw) + (int64_t)(c / 16) * nkc * 64 + lane;
  f32x4 acc[NRB];
#pragma unroll
  for (int rb = 0; rb < NRB; rb++) acc[rb] = f32x4{};
  u32x4 fa[PF][NRB], fb[PF];
  auto fetch = [&](int u, int kc) __attribute__((always_inline)) {
#pragma unroll
    for (int rb = 0; rb < NRB; rb++) fa[u][rb] = pa[rb][4 * kc];
    fb[u] = pb[(int64_t)kc * 64];
  };
  auto mma = [&](int u) __attribute__((always_inline)) {
#pragma unroll
    for (int rb = 0; rb < NRB; rb++)
      acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(fa[u][rb]), as_bf16x8(fb[u]), acc[rb], 0, 0, 0);
  };
  // chunk kc lives in slot kc % PF.  The steady loop consumes and refills
  // every slot without conditions (so the loads' wait counts stay exact);
  // the last chunks drain afterwards.
  if (nkc >= PF) {
#pragma unroll
    for (int u = 0; u < PF; u++) fetch(u, u);
    int kc0 = 0;
    for (; kc0 + 2 * PF <= nkc; kc0 += PF) {
#pragma unroll
      for (int u = 0; u < PF; u++) {
        mma(u);
        fetch(u, kc0 + PF + u);
      }
    }
    const int rest = nkc - kc0 - PF;  // chunks after the loaded ones, < PF
#pragma unroll
    for (int u = 0; u < PF; u++) {
      mma(u);
      if (u < rest) fetch(u, kc0 + PF + u);
    }
#pragma unroll
    for (int u = 0; u < PF; u++)
      if (u < rest) mma(u);
  } else {
    for (int kc = 0; kc < nkc; kc++) {
      fetch(0, kc);
      mma(0);
    }
  }
  // lane holds column c + (lane & 15) and rows 16 rb + 4 kq + i
  using E = Epi<uint16_t, KIND, HD>;
  const int col = c + r;
  if constexpr (NWR == 1) {
    static_assert(KIND == EPI_RESID, "single blocks only for the residual add");
    if (col >= e.N) return;
    const float bias = e.bias ? load_par<uint16_t>(e.bias, col) : 0.f;
#pragma unroll
    for (int rb = 0; rb < NRB; rb++)
#pragma unroll
      for (int i = 0; i < 4; i++) {
        const int row = 16 * rb + 4 * kq + i;
        if (row < M) {
          float* p = e.c + (int64_t)row * e.ldc;
          p[col] = resid_add(p[col], acc[rb][i], bias);
        }
      }
  } else if constexpr (KIND == EPI_HEAD) {
    static_assert(NWR == 4, "the head's groups are 64 columns: four waves");
#pragma unroll
    for (int rb = 0; rb < NRB; rb++)
      if (wave > 0) part[wave - 1][rb][lane] = acc[rb];
    __syncthreads();
    if (wave > 0) return;
    bool ok[4];
    int aidx[4];
#pragma unroll
    for (int j = 0; j < 4; j++) {
      ok[j] = col + 16 * j < e.N;
      aidx[j] = ok[j] ? alpha_index(e, col + 16 * j) : -1;
    }
    const bool any_alpha = __any(aidx[0] >= 0 || aidx[1] >= 0 || aidx[2] >= 0 || aidx[3] >= 0);
#pragma unroll
    for (int rb = 0; rb < NRB; rb++) {
      f32x4 blk[4];
      blk[0] = acc[rb];
#pragma unroll
      for (int j = 1; j < 4; j++) blk[j] = part[j - 1][rb][lane];
      float z[4][4];
#pragma unroll
      for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) z[i][j] = ok[j] ? blk[j][i] : -INFINITY;
      head_rows4(e, z, aidx, any_alpha, 16 * rb + 4 * kq, M, blockIdx.x, r);
    }
  } else {
    constexpr int NH = NWR / 2;  // the second half of the waves hand over
#pragma unroll
    for (int rb = 0; rb < NRB; rb++)
      if (wave >= NH) part[wave - NH][rb][lane] = acc[rb];
    __syncthreads();
    if (wave >= NH) return;
    const ColInfo ci = E::column(e, col);
#pragma unroll
    for (int rb = 0; rb < NRB; rb++) {
      const f32x4 hi = part[wave][rb][lane];  // block c + 32, same lane layout
#pragma unroll
      for (int i = 0; i < 4; i++) {
        const int row = 16 * rb + 4 * kq + i;
        if (row < M) E::row(e, ci, col, row, row, e.dpos, acc[rb][i], hi[i]);
      }
    }
  }
}

template <int KIND, int HD, int NRB>
hipError_t launch_rows_nrb(const uint16_t* A, const uint16_t* B, int M, int N_pad, int K,
                           const EpiArgs& e, hipStream_t s) {
  if constexpr (KIND == EPI_RESID) {
    hipLaunchKernelGGL((gemm_bf16_rows_kernel<KIND, HD, 1, NRB>), dim3(N_pad / 16), dim3(64), 0, s, A, B, M, K, e);
  } else if constexpr (KIND == EPI_QKV_ROPE || KIND == EPI_QKV_BIAS || KIND == EPI_HEAD) {
    hipLaunchKernelGGL((gemm_bf16_rows_kernel<KIND, HD, 4, NRB>), dim3(N_pad / 64), dim3(256), 0, s, A, B, M, K, e);
  } else {
    hipLaunchKernelGGL((gemm_bf16_rows_kernel<KIND, HD, 2, NRB>), dim3(N_pad / 32), dim3(128), 0, s, A, B, M, K, e);
  }
  return hipGetLastError();
}

template <int KIND, int HD>
hipError_t launch_rows_one(const uint16_t* A, const uint16_t* B, int M, int N_pad, int K,
                           const EpiArgs& e, hipStream_t s) {
  return M <= 16 ? launch_rows_nrb<KIND, HD, 1>(A, B, M, N_pad, K, e, s)
                 : launch_rows_nrb<KIND, HD, 2>(A, B, M, N_pad, K, e, s);
}

// HD != 0: the QKV kinds of a bf16 model with that head dim; HD == 0: the rest.
template <int HD>
hipError_t launch_rows_kind(const uint16_t* A, const uint16_t* B, int M, int N_pad, int K,
                            const EpiArgs& e, hipStream_t s) {
  if constexpr (HD != 0) {
    switch (e.kind) {
      case EPI_QKV_ROPE:
        return launch_rows_one<EPI_QKV_ROPE, HD>(A, B, M, N_pad, K, e, s);
      case EPI_QKV_BIAS:
        return launch_rows_one<EPI_QKV_BIAS, HD>(A, B, M, N_pad, K, e, s);
      default:
        return hipErrorInvalidValue;
    }
  } else {
    switch (e.kind) {
      case EPI_HEAD:
        return launch_rows_one<EPI_HEAD, 0>(A, B, M, N_pad, K, e, s);
      case EPI_RESID:
        return launch_rows_one<EPI_RESID, 0>(A, B, M, N_pad, K, e, s);
      case EPI_SWIGLU:
        return launch_rows_one<EPI_SWIGLU, 0>(A, B, M, N_pad, K, e, s);
      case EPI_BIAS_GELU:
        return launch_rows_one<EPI_BIAS_GELU, 0>(A, B, M, N_pad, K, e, s);
      default:
        return hipErrorInvalidValue;
    }
  }
}

template <int KIND, int HD, bool BLKB>
hipError_t launch_one(const uint16_t* A, const uint16_t* B, int M, int K, int ntm, int ntn, bool rb,
                      const EpiArgs& e, hipStream_t s) {
  const int total = ntm * ntn;
  const dim3 grid((total + kXcds - 1) / kXcds * kXcds), block(kThreads);
  if constexpr (KIND == EPI_RESID) {
    (void)rb;  // the residual products (N = d) keep the ring on A
    hipLaunchKernelGGL((gemm_bf16_kernel<KIND, HD, false, BLKB>), grid, block, 0, s, A, B, M, K, ntm, ntn, e);
  } else {
    if (rb)
      hipLaunchKernelGGL((gemm_bf16_kernel<KIND, HD, true, BLKB>), grid, block, 0, s, A, B, M, K, ntm, ntn, e);
    else
      hipLaunchKernelGGL((gemm_bf16_kernel<KIND, HD, false, BLKB>), grid, block, 0, s, A, B, M, K, ntm, ntn, e);
  }
  return hipGetLastError();
}

// HD != 0: the QKV kinds of a bf16 model with that head dim; HD == 0: the rest.
// Row-major B (blocked == false) only for the float32 store.
template <int HD>
hipError_t launch_kind(const uint16_t* A, const uint16_t* B, int M, int K, int ntm, int ntn,
                       const EpiArgs& e, hipStream_t s, bool blocked) {
  const bool rb = (int64_t)ntn * BN >= 2 * (int64_t)K;  // wide weight matrix: the ring holds B
  if constexpr (HD != 0) {
    if (!blocked) return hipErrorInvalidValue;
    switch (e.kind) {
      case EPI_QKV_ROPE:
        return launch_one<EPI_QKV_ROPE, HD, true>(A, B, M, K, ntm, ntn, rb, e, s);
      case EPI_QKV_BIAS:
        return launch_one<EPI_QKV_BIAS, HD, true>(A, B, M, K, ntm, ntn, rb, e, s);
      default:
        return hipErrorInvalidValue;
    }
  } else {
    if (!blocked) {
      if (e.kind != EPI_STORE_F32) return hipErrorInvalidValue;
      return launch_one<EPI_STORE_F32, 0, false>(A, B, M, K, ntm, ntn, rb, e, s);
    }
    switch (e.kind) {
      case EPI_STORE_F32:
        return launch_one<EPI_STORE_F32, 0, true>(A, B, M, K, ntm, ntn, rb, e, s);
      case EPI_HEAD:
        return launch_one<EPI_HEAD, 0, true>(A, B, M, K, ntm, ntn, rb, e, s);
      case EPI_RESID:
        return launch_one<EPI_RESID, 0, true>(A, B, M, K, ntm, ntn, rb, e, s);
      case EPI_SWIGLU:
        return launch_one<EPI_SWIGLU, 0, true>(A, B, M, K, ntm, ntn, rb, e, s);
      case EPI_BIAS_GELU:
        return launch_one<EPI_BIAS_GELU, 0, true>(A, B, M, K, ntm, ntn, rb, e, s);
      default:
        return hipErrorInvalidValue;
    }
  }
}

}  // namespace

hipError_t launch_gemm_bf16_rows(const uint16_t* A, const uint16_t* B, int M, int N_pad, int K,
                                 const EpiArgs& e, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (M > kRowsMax || !e.step || K % BK != 0 || N_pad % BN != 0) return hipErrorInvalidValue;
  const bool qkv = e.kind == EPI_QKV_ROPE || e.kind == EPI_QKV_BIAS;
  if (qkv && e.hd == 128) return launch_rows_kind<128>(A, B, M, N_pad, K, e, s);
  if (qkv && e.hd == 64) return launch_rows_kind<64>(A, B, M, N_pad, K, e, s);
  if (qkv) return hipErrorInvalidValue;
  return launch_rows_kind<0>(A, B, M, N_pad, K, e, s);
}

hipError_t launch_gemm_bf16(const uint16_t* A, const uint16_t* B, int M, int N_pad, int K,
                            const EpiArgs& e, hipStream_t s, bool blocked_b) {
  if (M <= 0) return hipSuccess;
  if (e.step || K % BK != 0 || N_pad % BN != 0) return hipErrorInvalidValue;
  const int ntm = (M + BM - 1) / BM, ntn = N_pad / BN;
  const bool qkv = e.kind == EPI_QKV_ROPE || e.kind == EPI_QKV_BIAS;
  if (qkv && e.hd == 128) return launch_kind<128>(A, B, M, K, ntm, ntn, e, s, blocked_b);
  if (qkv && e.hd == 64) return launch_kind<64>(A, B, M, K, ntm, ntn, e, s, blocked_b);
  if (qkv) return hipErrorInvalidValue;
  return launch_kind<0>(A, B, M, K, ntm, ntn, e, s, blocked_b);
}

}  // namespace lmgc
