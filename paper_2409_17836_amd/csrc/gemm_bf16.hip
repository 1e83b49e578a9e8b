// bf16 matrix product on CDNA4 matrix cores: C[M, N] = A[M, K] * B[N, K]^T
// with float32 accumulation, followed by a fused epilogue (epilogue.h).
//
// Both operands are K-contiguous: activations row-major, weights [out, in]
// in MFMA blocks (BLKB; common.h: 16 rows x 32 k per 1 KB in the order the
// lanes take their operand) or row-major (the exposed float32-store product).
// Tile: 256 x 256 output per 512-thread workgroup: eight 64-wide waves, two
// per SIMD so that one wave's LDS reads and waits overlap the other's matrix
// instructions; wave (wm, wn) owns rows wm*128 .. +128 and columns
// wn*64 .. +64 as 8 x 4 blocks of v_mfma_f32_16x16x32_bf16.
//
// Operand pipeline.  K advances in stages of 64.  Stages go to LDS with
// buffer loads straight into LDS (no staging registers): one operand through
// a ring of three 32 KB buffers, loaded two stages ahead, the other through
// two, loaded one stage ahead (5 x 32 KB = the whole 160 KB LDS).  The ring
// holds A by default and B when RB is set: the deeper prefetch goes to the
// operand whose panels miss L2 more often.  A wide weight matrix (N >= 2K:
// gate/up, QKV, LM head) has new B panels for every wave of tiles, while an
// XCD's A panels repeat; for a narrow one (the N = d products that add into
// the residual) B stays cached and A streams.  A wave's eight loads of a
// stage are spread through its MFMA stream (one after every four MFMAs, three
// when the ring holds B) instead of being issued in one burst after the
// barrier: all workgroups
// bursting at once queue in L2 and roughly double the load latency.  Each
// buffer is its own __shared__ array, so the compiler can tell the in-flight
// loads of one buffer from the reads of another.  The buffer resources are
// per tile with the tile's valid rows as their size: rows past M read as
// zero (and only feed outputs that are never stored).
//
// A row-major 256 x 64 operand tile is stored as rows of eight 16-byte
// chunks; chunk c of row r sits at slot c ^ ((r >> 1) & 7): the 16 lanes that
// one ds_read_b128 cycle serves read 16 consecutive rows, and the swizzle
// gives every (row parity, slot) pair once, i.e. all 64 banks.  A blocked B
// tile is its 32 blocks copied as they are: lane l reads 16 bytes at 16 l of
// a block, conflict-free without a swizzle.
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
constexpr int kThreads = 512;
// row tiles per group of the tile order: 4 when the ring holds A, 8 when it
// holds B (measured best at the 7B shape)
constexpr int kGroupM = 4, kGroupMB = 8;
constexpr int kXcds = 8;
// MFMAs between two operand loads of a wave (ring on A / ring on B)
constexpr int kLoadEvery = 4, kLoadEveryB = 3;
// s_waitcnt immediates (vmcnt in bits 3:0, expcnt and lgkmcnt left at their maxima)
constexpr int kVmcnt0 = 0xF70, kVmcnt4 = 0xF74;

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
  const int wm = wave >> 2, wn = wave & 3;

  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A + (int64_t)m0 * K, min(M - m0, BM) * K * 2);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(Bw + (int64_t)n0 * K, BN * K * 2);
  // Load i of wave w fills LDS rows (w*4 + i)*8 .. +8 of a stage; lane l lands
  // at row +l/8, slot l%8 (the hardware writes lane l at base + 16 l), so it
  // fetches the logical chunk the swizzle puts there.  The row is part of the
  // lane offset (for the bounds check), the stage's k offset is scalar.
  int voff[4];
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int row = (wave * 4 + i) * 8 + (lane >> 3);
    const int lc = (lane & 7) ^ ((row >> 1) & 7);
    voff[i] = (row * K + lc * 8) * 2;
  }
  // BLKB: B in MFMA blocks.  A stage's B tile is 32 blocks of 1 KB (16 row
  // groups x two 32-wide k chunks); load i of wave w copies block w*4 + i =
  // 16 kc + j (row group j, chunk kc of the stage) to the same place in LDS,
  // where lane l's 16 bytes are already its MFMA operand: no swizzle.
  int voffb[4];
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int blk = wave * 4 + i, kc = blk >> 4, j = blk & 15;
    voffb[i] = BLKB ? ((j * (K / 32) + kc) * 1024 + lane * 16) : voff[i];
  }

  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; i++)
#pragma unroll
    for (int j = 0; j < 4; j++) acc[i][j] = f32x4{};

  // MFMA operands: lane l supplies row (l & 15) of a 16-row block and the
  // 8 k-values of chunk (l >> 4) of the 32-wide k step.
  const int arow0 = wm * 128 + (lane & 15), brow0 = wn * 64 + (lane & 15), kq = lane >> 4;

  auto ldA = [&](u32x4* sa, int i, int k0) __attribute__((always_inline)) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr_t)(sa + (wave * 4 + i) * 64), 16, voff[i],
                                             k0 * 2, 0, 0);
  };
  auto ldB = [&](u32x4* sb, int i, int k0) __attribute__((always_inline)) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_ptr_t)(sb + (wave * 4 + i) * 64), 16, voffb[i],
                                             BLKB ? k0 * 32 : k0 * 2, 0, 0);
  };
  // One stage from ring buffer sr and double buffer sd.  The double-buffered
  // operand of stage kd goes to nd and the ring operand of stage kr to nr
  // (negative: no load), one load after every kLoadEvery (kLoadEveryB) MFMAs.
  auto ld_r = [&](u32x4* buf, int i, int k0) __attribute__((always_inline)) {
    if (RB) ldB(buf, i, k0);
    else ldA(buf, i, k0);
  };
  auto ld_d = [&](u32x4* buf, int i, int k0) __attribute__((always_inline)) {
    if (RB) ldA(buf, i, k0);
    else ldB(buf, i, k0);
  };
  auto compute = [&](const u32x4* sr, const u32x4* sd, u32x4* nr, int kr, u32x4* nd, int kd)
      __attribute__((always_inline)) {
    const u32x4* sa = RB ? sd : sr;
    const u32x4* sb = RB ? sr : sd;
    int issued = 0, nm = 0;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ks++) {
      const int ch = ks * 4 + kq;
      bf16x8 af[8], bf[4];
#pragma unroll
      for (int i = 0; i < 8; i++) af[i] = as_bf16x8(sa[slot(arow0 + 16 * i, ch)]);
#pragma unroll
      for (int j = 0; j < 4; j++)
        bf[j] = as_bf16x8(BLKB ? sb[(ks * 16 + wn * 4 + j) * 64 + lane] : sb[slot(brow0 + 16 * j, ch)]);
#pragma unroll
      for (int i = 0; i < 8; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
          if (++nm % (RB ? kLoadEveryB : kLoadEvery) == 0 && issued < 8) {
            __builtin_amdgcn_sched_barrier(0);
            if (issued < 4) {
              if (kd >= 0) ld_d(nd, issued, kd);
            } else {
              if (kr >= 0) ld_r(nr, issued - 4, kr);
            }
            __builtin_amdgcn_sched_barrier(0);
            issued++;
          }
        }
    }
  };
  auto barrier = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };

  // Stage t reads ring buffer t % 3 and double buffer t % 2.  During stage t
  // a wave loads D(t+1) (into the double buffer stage t-1 used) and R(t+2)
  // (into the ring buffer of stage t-1), in that order; at the start of stage
  // t its loads in flight are, oldest first, R(t), D(t), R(t+1), so vmcnt(4)
  // leaves only R(t+1) outstanding.  The barrier then makes every wave's part
  // of stage t visible, and ends every wave's reads of stage t-1.
  auto full = [&](int t, const u32x4* cr, const u32x4* cd, u32x4* nd, u32x4* nr)
      __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(kVmcnt4);
    barrier();
    compute(cr, cd, nr, (t + 2) * BK, nd, (t + 1) * BK);
  };
  const int nk = K / BK;
  auto tail = [&](int t, const u32x4* cr, const u32x4* cd, u32x4* nd, u32x4* nr)
      __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(kVmcnt0);
    barrier();
    compute(cr, cd, nr, t + 2 < nk ? (t + 2) * BK : -1, nd, t + 1 < nk ? (t + 1) * BK : -1);
  };
#pragma unroll
  for (int i = 0; i < 4; i++) ld_r(sR0, i, 0);
#pragma unroll
  for (int i = 0; i < 4; i++) ld_d(sD0, i, 0);
  if (nk > 1) {
#pragma unroll
    for (int i = 0; i < 4; i++) ld_r(sR1, i, BK);
  }
  // buffers repeat every 6 stages; the loop runs while all six steps and the
  // loads they issue are in range, the rest (at most 7 stages) is predicated
  int t = 0;
  for (; t + 8 <= nk; t += 6) {
    full(t + 0, sR0, sD0, sD1, sR2);
    full(t + 1, sR1, sD1, sD0, sR0);
    full(t + 2, sR2, sD0, sD1, sR1);
    full(t + 3, sR0, sD1, sD0, sR2);
    full(t + 4, sR1, sD0, sD1, sR0);
    full(t + 5, sR2, sD1, sD0, sR1);
  }
  if (t + 0 < nk) tail(t + 0, sR0, sD0, sD1, sR2);
  if (t + 1 < nk) tail(t + 1, sR1, sD1, sD0, sR0);
  if (t + 2 < nk) tail(t + 2, sR2, sD0, sD1, sR1);
  if (t + 3 < nk) tail(t + 3, sR0, sD1, sD0, sR2);
  if (t + 4 < nk) tail(t + 4, sR1, sD0, sD1, sR0);
  if (t + 5 < nk) tail(t + 5, sR2, sD1, sD0, sR1);
  if (t + 6 < nk) tail(t + 6, sR0, sD0, sD1, sR2);

  // Epilogue.  16 x 16 block layout: lane holds column (lane & 15) and rows
  // 4 (lane >> 4) + r, r = 0..3.  Blocks j and j + 2 give the column pair
  // (col, col + 32).  Rows 4 (lane >> 4) + 0..3 never straddle a window
  // (W is a multiple of 8).
  // The reads an epilogue needs (residual, RoPE table) for row block i + 1
  // are issued before the stores of block i.  Whole tiles (all but the
  // ragged edges) take a path without row and column checks, so the
  // epilogue stays one basic block.
  using E = Epi<uint16_t, KIND, HD>;
  using Pre4 = typename E::Pre4;
  const int c0 = n0 + wn * 64 + (lane & 15);
  if constexpr (KIND == EPI_HEAD) {
    // the wave's 64 columns are group (n0 + 64 wn) / 64; lane holds columns
    // c0 + 16 j of rows 4 kq + r of every 16-row block
    const int g = (n0 + wn * 64) >> 6;
    bool ok[4];
    int aidx[4];
#pragma unroll
    for (int j = 0; j < 4; j++) {
      ok[j] = c0 + 16 * j < e.N;
      aidx[j] = ok[j] ? alpha_index(e, c0 + 16 * j) : -1;
    }
#pragma unroll
    for (int i = 0; i < 8; i++)
#pragma unroll
      for (int r = 0; r < 4; r++) {
        const int row = m0 + wm * 128 + 16 * i + 4 * kq + r;
        float z[4];
#pragma unroll
        for (int j = 0; j < 4; j++) z[j] = ok[j] ? acc[i][j][r] : -INFINITY;
        head_row(e, z, aidx, row, row < M, g, lane & 15);
      }
    return;
  }
  ColInfo ci0 = E::column(e, c0), ci1 = E::column(e, c0 + 16);
  if (KIND == EPI_QKV_ROPE || KIND == EPI_QKV_BIAS) {
    // bf16 models have head_dim 64 or 128, so q, k and v and every head are
    // whole 64-column groups: a wave's columns share segment and head.
    // Saying so turns the epilogue's q/k/v branches into scalar ones.
    auto uniform = [](ColInfo& c) __attribute__((always_inline)) {
      c.valid = __builtin_amdgcn_readfirstlane((int)c.valid) != 0;
      c.seg = __builtin_amdgcn_readfirstlane(c.seg);
      c.seg2 = __builtin_amdgcn_readfirstlane(c.seg2);
      c.head = __builtin_amdgcn_readfirstlane(c.head);
      c.head2 = __builtin_amdgcn_readfirstlane(c.head2);
    };
    uniform(ci0);
    uniform(ci1);
  }
  const int W = e.W > 0 ? e.W : 1;
  // V columns of a whole tile (bf16 QKV): the wave's 128 rows x 64 columns
  // go through LDS, transposed, so that each V^T row (a dim of a head) is
  // written as 16-byte pieces of 8 consecutive positions.  A wave's region
  // is 16 KB: 64 rows (columns) of 128 positions, 16-byte chunks swizzled by
  // chunk ^ (row & 15).  Needs W % 128 == 0 so the rows lie in one window.
  auto v_transposed = [&]() __attribute__((always_inline)) {
    u32x4* reg = (wave < 2 ? sR0 : wave < 4 ? sR1 : wave < 6 ? sR2 : sD0) + (wave & 1) * 1024;
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
        const bf16x4 val = {(__bf16)(acc[i][j][0] + bias), (__bf16)(acc[i][j][1] + bias),
                            (__bf16)(acc[i][j][2] + bias), (__bf16)(acc[i][j][3] + bias)};
        const int off = kap * 256 + (((rho >> 3) ^ (kap & 15)) << 4) + (rho & 7) * 2;
        *reinterpret_cast<bf16x4*>(regb + off) = val;
      }
    const int H = KIND == EPI_QKV_ROPE ? e.Hkv : e.Hq;
    const int h = HD ? HD : e.hd;
    const int row0 = m0 + wm * 128, b = row0 / W, pos0 = row0 - b * W;
    // first V column: after q and k (Hq and Hkv heads for RoPE models,
    // Hq and Hq for GPT-2's fused projection)
    const int vcol0 = n0 + wn * 64 - (KIND == EPI_QKV_ROPE ? e.Hq + e.Hkv : 2 * e.Hq) * h;
#pragma unroll
    for (int t = 0; t < 16; t++) {
      const int c = lane + 64 * t, kap = c >> 4, ch = c & 15;
      const u32x4 val = reg[kap * 16 + (ch ^ (kap & 15))];
      const int cc = vcol0 + kap, head = cc / h, dim = cc - head * h;
      uint16_t* dst = (uint16_t*)e.v + (((int64_t)b * H + head) * h + dim) * W + pos0 + ch * 8;
      *reinterpret_cast<u32x4*>(dst) = val;
    }
  };
  auto epilogue = [&](auto full_tag) __attribute__((always_inline)) {
    constexpr bool FULL = decltype(full_tag)::value;
    if constexpr (FULL && (KIND == EPI_QKV_ROPE || KIND == EPI_QKV_BIAS)) {
      if (W % 128 == 0) {
        barrier();  // every wave has finished reading the operand buffers
        if (ci0.seg == 2) {
          v_transposed();
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
      const float a0[4] = {acc[i][0][0], acc[i][0][1], acc[i][0][2], acc[i][0][3]};
      const float a2[4] = {acc[i][2][0], acc[i][2][1], acc[i][2][2], acc[i][2][3]};
      const float a1[4] = {acc[i][1][0], acc[i][1][1], acc[i][1][2], acc[i][1][3]};
      const float a3[4] = {acc[i][3][0], acc[i][3][1], acc[i][3][2], acc[i][3][3]};
      E::template rows4<FULL>(e, ci0, c0, r0, M, b, p0, a0, a2, q0);
      E::template rows4<FULL>(e, ci1, c0 + 16, r0, M, b, p0, a1, a3, q1);
      q0 = n0q;
      q1 = n1q;
    }
  };
  if (m0 + BM <= M && n0 + BN <= e.N) epilogue(std::true_type{});
  else epilogue(std::false_type{});
}

// Decoding step (M <= 16 rows: one row per window).  Every wave accumulates
// one 16-column block and runs, for every output element, the same chain as
// gemm_bf16_kernel: 16x16x32 bf16 MFMAs over the 32-wide k chunks in
// increasing order, lane l holding row (l & 15) and k values 8*(l >> 4) .. +8
// of a chunk.  So a row's outputs equal, bit for bit, what the tiled kernel
// gives that row in a batch of whole windows.  Operands come straight from
// global memory (the step streams the weights once), kRowsPf chunks ahead.
// The step is bound by how many weight bytes each wave has in flight, so the
// waves are spread over as many CUs as the epilogue allows.  NWR waves per
// workgroup:
//  - 4: 64 columns; waves 2 and 3 hand their accumulators to waves 0 and 1
//    through LDS, which run the epilogue on the (col, col + 32) pairs (QKV:
//    the RoPE pairs and the transposed V stores);
//  - 2: the two blocks c and c + 32 of one pair (gate/up, GELU, float32
//    store);
//  - 1: one block, for the residual add, which pairs nothing (N = d = 4096 has
//    only 256 blocks: one wave on each CU instead of 64 four-wave groups).
constexpr int kRowsPf = 16;

template <int KIND, int HD, int NWR>
__global__ __launch_bounds__(64 * NWR) void gemm_bf16_rows_kernel(const uint16_t* __restrict__ A,
                                                                  const uint16_t* __restrict__ Bw,
                                                                  int M, int K, EpiArgs e) {
  // accumulators handed over: to the pair's first block (QKV: waves 2, 3 to
  // 0, 1), or all to wave 0 (HEAD: waves 1..3, the group's blocks j = 1..3)
  __shared__ f32x4 part[NWR == 4 ? 3 : 1][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int c;  // this wave's block
  if (NWR == 4) c = blockIdx.x * 64 + wave * 16;
  else if (NWR == 2) c = (blockIdx.x >> 1) * 64 + (blockIdx.x & 1) * 16 + wave * 32;
  else c = blockIdx.x * 16;
  const int r = lane & 15, kq = lane >> 4;
  // rows past M re-read row M - 1; they only feed outputs that are not stored
  const u32x4* pa = reinterpret_cast<const u32x4*>(A + (int64_t)min(r, M - 1) * K + kq * 8);
  // B in MFMA blocks: the wave's 16 rows are one contiguous stream of 1 KB
  // blocks, lane l's 16 bytes at 16 l of each
  const int nkc = K / 32;  // A chunk kc starts at u32x4 index 4 * kc
  const u32x4* pb = reinterpret_cast<const u32x4*>(Bw) + (int64_t)(c / 16) * nkc * 64 + lane;
  f32x4 acc = f32x4{};
  u32x4 fa[kRowsPf], fb[kRowsPf];
  auto fetch = [&](int u, int kc) __attribute__((always_inline)) {
    fa[u] = pa[4 * kc];
    fb[u] = pb[(int64_t)kc * 64];
  };
  auto mma = [&](int u) __attribute__((always_inline)) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(fa[u]), as_bf16x8(fb[u]), acc, 0, 0, 0);
  };
  // chunk kc lives in slot kc % kRowsPf.  The steady loop consumes and
  // refills every slot without conditions (so the loads' wait counts stay
  // exact); the last chunks drain afterwards.
  if (nkc >= kRowsPf) {
#pragma unroll
    for (int u = 0; u < kRowsPf; u++) fetch(u, u);
    int kc0 = 0;
    for (; kc0 + 2 * kRowsPf <= nkc; kc0 += kRowsPf) {
#pragma unroll
      for (int u = 0; u < kRowsPf; u++) {
        mma(u);
        fetch(u, kc0 + kRowsPf + u);
      }
    }
    const int rest = nkc - kc0 - kRowsPf;  // chunks after the loaded ones, < kRowsPf
#pragma unroll
    for (int u = 0; u < kRowsPf; u++) {
      mma(u);
      if (u < rest) fetch(u, kc0 + kRowsPf + u);
    }
#pragma unroll
    for (int u = 0; u < kRowsPf; u++)
      if (u < rest) mma(u);
  } else {
    for (int kc = 0; kc < nkc; kc++) {
      fetch(0, kc);
      mma(0);
    }
  }
  // lane holds column c + (lane & 15) and rows 4 kq + i
  using E = Epi<uint16_t, KIND, HD>;
  const int col = c + r;
  if constexpr (NWR == 1) {
    static_assert(KIND == EPI_RESID, "single blocks only for the residual add");
    if (col >= e.N) return;
    const float bias = e.bias ? load_par<uint16_t>(e.bias, col) : 0.f;
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int row = 4 * kq + i;
      if (row < M) {
        float* p = e.c + (int64_t)row * e.ldc;
        p[col] = resid_add(p[col], acc[i], bias);
      }
    }
  } else if constexpr (KIND == EPI_HEAD) {
    static_assert(NWR == 4, "the head's groups are 64 columns: four waves");
    if (wave > 0) part[wave - 1][lane] = acc;
    __syncthreads();
    if (wave > 0) return;
    f32x4 blk[4];
    blk[0] = acc;
#pragma unroll
    for (int j = 1; j < 4; j++) blk[j] = part[j - 1][lane];
    bool ok[4];
    int aidx[4];
#pragma unroll
    for (int j = 0; j < 4; j++) {
      ok[j] = col + 16 * j < e.N;
      aidx[j] = ok[j] ? alpha_index(e, col + 16 * j) : -1;
    }
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int row = 4 * kq + i;
      float z[4];
#pragma unroll
      for (int j = 0; j < 4; j++) z[j] = ok[j] ? blk[j][i] : -INFINITY;
      head_row(e, z, aidx, row, row < M, blockIdx.x, r);
    }
  } else {
    constexpr int NH = NWR / 2;  // the second half of the waves hand over
    if (wave >= NH) part[wave - NH][lane] = acc;
    __syncthreads();
    if (wave >= NH) return;
    const f32x4 hi = part[wave][lane];  // block c + 32, same lane layout
    const ColInfo ci = E::column(e, col);
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const int row = 4 * kq + i;
      if (row < M) E::row(e, ci, col, row, row, e.dpos, acc[i], hi[i]);
    }
  }
}

template <int KIND, int HD>
hipError_t launch_rows_one(const uint16_t* A, const uint16_t* B, int M, int N_pad, int K,
                           const EpiArgs& e, hipStream_t s) {
  if constexpr (KIND == EPI_RESID) {
    hipLaunchKernelGGL((gemm_bf16_rows_kernel<KIND, HD, 1>), dim3(N_pad / 16), dim3(64), 0, s, A, B, M, K, e);
  } else if constexpr (KIND == EPI_QKV_ROPE || KIND == EPI_QKV_BIAS || KIND == EPI_HEAD) {
    hipLaunchKernelGGL((gemm_bf16_rows_kernel<KIND, HD, 4>), dim3(N_pad / 64), dim3(256), 0, s, A, B, M, K, e);
  } else {
    hipLaunchKernelGGL((gemm_bf16_rows_kernel<KIND, HD, 2>), dim3(N_pad / 32), dim3(128), 0, s, A, B, M, K, e);
  }
  return hipGetLastError();
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
  if (M > 16 || !e.step || K % BK != 0 || N_pad % BN != 0) return hipErrorInvalidValue;
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
