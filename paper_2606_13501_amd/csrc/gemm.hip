// Projections of the DiT block: out = epilogue(A . W^T + bias).
//
// bf16: a 256x256 (or 256x192) output tile per 256-thread workgroup on the
// gfx950 matrix cores (v_mfma_f32_32x32x16_bf16), fp32 accumulation.  Each of
// the 4 waves (one per SIMD) owns a 128x128 (128x96) sub-tile whose
// accumulators (256 or 192 registers) live in the accumulation registers.  The K loop runs in steps of 64: a
// step's operand tiles are 256 rows x 128 B, i.e. whole cache lines per row.
// LDS double-buffers two steps (2 x 64 KiB); two register stages carry the
// next two steps from global memory, so a load has about two steps of MFMA
// work to land.  Global loads, LDS stores and fragment reads are spread
// evenly between the MFMAs (the memory pipeline never sees a burst that
// would stall MFMA issue).  The 16-byte chunks of each 128-byte LDS row are
// XOR-swizzled so fragment reads are free of bank conflicts.  The kernel
// computes C^T blocks (W as the MFMA A operand) so that every lane ends up
// holding four consecutive output columns of one row, stored as one 8-byte
// write with the fused epilogue (bias, GELU-tanh, residual, gated residual).
// Workgroups are rastered in groups of 2 tile rows per XCD so the tiles
// resident on one XCD share A and W panels in its L2.
//
// fp32: a plain 64x64 LDS-tiled FMA kernel for the small exact configuration.
#include <atomic>

#include "common.hpp"
#include "kernels.hpp"

namespace dit {

namespace {

constexpr int BM = 256, BK = 64;               // tile rows, K step (columns: 256 or 192)
constexpr int kWaves = 4;                           // 2 x 2 waves, each a 128 x 128 sub-tile
constexpr int kThreads = 64 * kWaves;
constexpr int kStages = 2;                          // LDS double buffer
constexpr int kRowBytes = BK * 2;                   // 128 B: one full cache line per tile row
constexpr int kTileBytes = BM * kRowBytes;          // one operand tile of one step (32 KiB)
constexpr int kStageBytes = 2 * kTileBytes;         // A tile + W tile
constexpr int kLoads = kTileBytes / 1024 / kWaves;  // 1 KiB loads per wave, operand and step (8)
constexpr int kEpiBytes = 32 * 256;                 // per wave: 32 rows x 64 fp32 (epilogue window)
constexpr int kGroupM = 2;                          // tile rows per raster group
constexpr int kGroupMFew = 8;                       // the same, at most kFewTileRows tile rows
constexpr int kFewTileRows = 16;
constexpr int kXcds = 8;                            // gfx950: 8 XCDs, workgroups dispatched round-robin

// gelu_tanh(z) = z (1 + tanh u) / 2 = z / (1 + e^(-2u)), u = sqrt(2/pi) (z + 0.044715 z^3)
__device__ __forceinline__ float gelu_tanh(float z) {
  const float k0 = 0.7978845608028654f;  // sqrt(2/pi)
  const float k1 = 0.044715f;
  const float u = k0 * fmaf(k1 * z, z * z, z);
  const float e = __builtin_amdgcn_exp2f(-2.0f * 1.4426950408889634f * u);   // inf for u << 0: z / inf = 0
  return z * __builtin_amdgcn_rcpf(1.0f + e);
}

// Tile sequence of a workgroup.  Each XCD owns a contiguous range of logical
// tiles (the dispatcher places workgroup b on XCD b mod 8); the workgroups of
// one XCD take its tiles round-robin, so at any time they work on adjacent
// tiles.  Logical tiles are rastered in groups of group_m tile rows, so the
// tiles resident on one XCD share A and W panels in its L2.  Two tile rows per
// group measured best at 75,600 rows (1-2.5% over 4, 8 and 16): the weights
// of one GEMM (at most 157 MB) stay in the 256 MB MALL, so reuse of the
// activation rows is what saves memory traffic.  With at most 16 tile rows
// (4,096 rows: one to three rounds of tiles), groups of 8 rows: an XCD's 32
// resident tiles then cover 8 x 4 tiles instead of 2 x 16 and read a quarter
// of the W columns per step.  Measured in alternating order on one box at
// 4,096 rows: 0.2-0.8% faster with D = 3,072 (output, up and down
// projections), the same on the QKV shape.
struct TileSeq {
  int first, stride, count;   // logical tiles first + stride * it, it < count
  int tiles_m, tiles_n, group_m;
  __device__ void coords(int it, int& tm, int& tn) const {
    const int t = first + stride * it;
    const int width = group_m * tiles_n;
    const int group = t / width;
    const int first_m = group * group_m;
    const int gsize = min(tiles_m - first_m, group_m);
    const int r = t - group * width;
    tm = first_m + r % gsize;
    tn = r / gsize;
  }
};

__device__ __forceinline__ TileSeq tile_seq(int b, int nb, int tiles_m, int tiles_n, int group_m) {
  const int tiles = tiles_m * tiles_n;
  const int per_xcd = (tiles + kXcds - 1) / kXcds;
  const int x = b % kXcds, slot = b / kXcds, wgs = nb / kXcds;
  const int lo = x * per_xcd, hi = min(tiles, lo + per_xcd);
  TileSeq q;
  q.first = lo + slot;
  q.stride = wgs;
  q.count = q.first < hi ? (hi - q.first + wgs - 1) / wgs : 0;
  q.tiles_m = tiles_m;
  q.tiles_n = tiles_n;
  q.group_m = group_m;
  return q;
}

// 16-byte chunk swizzle of a 128-byte LDS row: a fragment read touches 16
// consecutive rows at one logical chunk; rows 2t and 2t + 1 lie in different
// halves of a 256-byte bank window and the physical chunk c ^ t differs
// between the 8 values of t, so the 16 reads hit 16 distinct bank groups.
__device__ __forceinline__ int row_swizzle(int r) { return (r >> 1) & 7; }

// Raw buffer descriptor over `bytes` bytes from `base`.  The hardware's range
// check covers the lane offset only (not the scalar offset), so a load
// returns zeros where its lane offset is past the end; the loads below carry
// every row offset in the lane offset.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const uint32_t n = bytes > 0xFFFFFFFFll ? 0xFFFFFFFFu : (uint32_t)(bytes < 0 ? 0 : bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}

// The same descriptor as a plain vector (operand of the LDS-direct load).
__device__ __forceinline__ u32x4 make_desc(const void* base, int64_t bytes) {
  const uint32_t n = bytes > 0xFFFFFFFFll ? 0xFFFFFFFFu : (uint32_t)(bytes < 0 ? 0 : bytes);
  const uint64_t p = (uint64_t)base;
  return u32x4{(uint32_t)p, (uint32_t)(p >> 32) & 0xFFFFu, n, 0x00020000u};
}

// 16 bytes per lane from global memory straight into LDS: lane i writes LDS
// bytes lds + 16 i .. +15.  Inline assembly, so the compiler does not make
// later LDS reads wait for it; completion is waited for by hand.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void load_lds16(const u32x4& desc, int voff, int soff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :: "s"(lds), "v"(voff), "s"(desc), "s"(soff) : "m0");
}
#pragma clang diagnostic pop

// SEQ: the workgroup runs a sequence of tiles (K / 64 even and >= 6);
// otherwise one tile per workgroup and any K / 64.
template <int EPI, bool SEQ, int BNT>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_nt(
    const bf16* __restrict__ A, int64_t lda, const bf16* __restrict__ W, int64_t ldw,
    const bf16* __restrict__ bias, bf16* __restrict__ C, int64_t ldc, const bf16* R, int64_t ldr,
    const float* __restrict__ gate, int64_t gate_stride, ReqTable req, int M, int N, int K,
    int tiles_m, int tiles_n, int group_m, int plane_cols, int64_t plane_skip) {
  constexpr int WN = BNT / 2;                    // columns of a wave's sub-tile
  constexpr int NI = WN / 32;                    // its W blocks of 32 columns (4 or 3)
  constexpr int kTileW = BNT * kRowBytes;        // the W tile of one step
  constexpr int kStage = kTileBytes + kTileW;    // A tile, then W tile
  constexpr int kLW = kTileW / 1024 / kWaves;    // 1 KiB W loads per wave and step (8 or 6)
  __shared__ __attribute__((aligned(1024))) char smem[kStages * kStage + kWaves * kEpiBytes];

  const TileSeq seq = tile_seq(blockIdx.x, gridDim.x, tiles_m, tiles_n, group_m);
  if (seq.count == 0) return;
  int tm, tn;
  seq.coords(0, tm, tn);
  int m0 = tm * BM, n0 = tn * BNT;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  // ---- global -> registers -> LDS.  A step's operand tile is 32 pieces of
  // 1 KiB (8 rows x 128 B); wave w moves pieces q = 8 w .. 8 w + 7 of A and
  // of W.  Lane i of piece q holds row 8 q + i / 8, logical chunk
  // (i % 8) ^ row_swizzle(row), and stores it at LDS byte q * 1024 + 16 i,
  // i.e. physical chunk i % 8 of that row.
  auto a_rs = make_rsrc(A + (int64_t)m0 * lda, ((int64_t)(M - m0 - 1) * lda + K) * 2);
  auto w_rs = make_rsrc(W + (int64_t)n0 * ldw, ((int64_t)(N - n0 - 1) * ldw + K) * 2);
  // Row 8 q + i / 8 has row_swizzle = 4 (q % 2) + i / 16, so the lane part of
  // a load's offset is one of two values per operand (by the parity of q)
  // plus 8 q rows, a uniform value.
  int a_vo[2], w_vo[2];
#pragma unroll
  for (int par = 0; par < 2; ++par) {
    const int c = (lane & 7) ^ (4 * par + (lane >> 4));
    a_vo[par] = (lane >> 3) * (int)lda * 2 + c * 16;
    w_vo[par] = (lane >> 3) * (int)ldw * 2 + c * 16;
  }
  // A load's lane offset is its row inside the tile (piece row 8 q plus the
  // lane's row i / 8) and its chunk; the scalar offset is the K step only.
  // The descriptor's range check sees the whole row offset, so rows past the
  // end of the operand (a ragged last tile) read as zeros and no load leaves
  // the operand.  The piece part 8 q rows is uniform (a scalar added per
  // load).  Steps past the last K step (prologue loads of a short K) reload
  // the last one.
  auto a_po = [&](int u) { return (kLoads * wave + u) * 16 * (int)lda; };   // 8 q rows, in bytes
  auto w_po = [&](int u) { return (kLW * wave + u) * 16 * (int)ldw; };
  auto k_off = [&](int step) { return min(step, K / BK - 1) * BK * 2; };
  struct Stage { u32x4 a[kLoads], w[kLW]; };   // one step of this wave's pieces
  auto gload = [&](Stage& r, int step) {
    const int soff = k_off(step);
#pragma unroll
    for (int u = 0; u < kLoads; ++u) {
      r.a[u] = __builtin_amdgcn_raw_buffer_load_b128(a_rs, a_vo[u & 1] + a_po(u), soff, 0);
      if (u < kLW) r.w[u] = __builtin_amdgcn_raw_buffer_load_b128(w_rs, w_vo[u & 1] + w_po(u), soff, 0);
    }
  };
  // LDS homes of this wave's pieces in the slot of `step`: A piece u, W piece u
  auto a_home = [&](int step) { return smem + (step % kStages) * kStage + kLoads * wave * 1024 + lane * 16; };
  auto w_home = [&](int step) {
    return smem + (step % kStages) * kStage + kTileBytes + kLW * wave * 1024 + lane * 16;
  };
  auto sstore = [&](const Stage& r, int step) {
    char* const sa = a_home(step);
    char* const sw = w_home(step);
#pragma unroll
    for (int u = 0; u < kLoads; ++u) {
      *reinterpret_cast<u32x4*>(sa + u * 1024) = r.a[u];
      if (u < kLW) *reinterpret_cast<u32x4*>(sw + u * 1024) = r.w[u];
    }
  };

  // ---- fragment reads: row base + 32 b + (lane & 31), logical chunk 2 kk + (lane >> 5)
  const int fr = lane & 31;
  const int fh = lane >> 5;
  const int sw = row_swizzle(fr);   // == row_swizzle(base + 32 b + fr)
  int fo_a[4], fo_w[4];             // + 32 * kRowBytes b
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    fo_a[kk] = (wm * 128 + fr) * kRowBytes + (((2 * kk + fh) ^ sw) << 4);
    fo_w[kk] = kTileBytes + (wn * WN + fr) * kRowBytes + (((2 * kk + fh) ^ sw) << 4);
  }
  struct Frags { bf16x8 w[NI], a[4]; };
  auto read = [&](Frags& f, int step, int kk) {
    const char* st = smem + (step % kStages) * kStage;
#pragma unroll
    for (int i = 0; i < NI; ++i) f.w[i] = *reinterpret_cast<const bf16x8*>(st + fo_w[kk] + i * 32 * kRowBytes);
#pragma unroll
    for (int j = 0; j < 4; ++j) f.a[j] = *reinterpret_cast<const bf16x8*>(st + fo_a[kk] + j * 32 * kRowBytes);
  };

  // acc[i][j]: W block i (NI x 32 columns of the wave), A block j (4 x 32 rows)
  f32x16 acc[NI][4];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};
  auto mma = [&](const Frags& f) {
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.w[i], f.a[j], acc[i][j], 0, 0, 0);
  };
  const int KT = K / BK;
  // Per K quarter: 16 MFMAs, the 8 fragment reads of the next quarter, and
  // (when a register stage is being cycled) 4 LDS stores + 4 global loads.
  // The reads go first, one per MFMA over the first half, so each has most
  // of a quarter to land; the stores and loads are spread over the second
  // half.  (Measured at 720p against reads, stores and loads interleaved
  // evenly: QKV 8.85 against 9.16 ms; reads two per MFMA or loads before
  // stores were no better.)  With 3 W blocks per wave: 12 MFMAs, 7 reads, up
  // to 4 stores and 4 loads per quarter, in the same order.  Each quarter is
  // closed by a scheduling fence (below), so the compiler cannot sink the
  // next quarter's reads next to the MFMAs that consume them.
  auto pattern = [] {
    if constexpr (NI == 4) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {   // the next quarter's 8 reads, one per MFMA of the first half
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {   // stores and loads over the second half
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 7; ++i) {   // the next quarter's 7 reads, one per MFMA
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {   // stores and loads over the remaining MFMAs
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      }
    }
  };


  // items u0 .. u0 + 3 of a register stage (items 0-7: A pieces, 8-15: W
  // pieces): store each into the LDS slot of step st_step, then reload it
  // with step ld_step (each part only when asked for)
  auto io4 = [&](Stage& R, int u0, int st_step, int ld_step, bool do_store, bool do_load) {
    char* const sa = a_home(st_step);
    char* const sw = w_home(st_step);
    const int soff = ld_step * BK * 2;   // loads are asked for only while ld_step < K / 64
#pragma unroll
    for (int u = u0; u < u0 + 4; ++u) {
      const int p = u & 7;
      if (u < 8) {
        if (do_store) *reinterpret_cast<u32x4*>(sa + p * 1024) = R.a[p];
        if (do_load) R.a[p] = __builtin_amdgcn_raw_buffer_load_b128(a_rs, a_vo[p & 1] + a_po(p), soff, 0);
      } else if (p < kLW) {
        if (do_store) *reinterpret_cast<u32x4*>(sw + p * 1024) = R.w[p];
        if (do_load) R.w[p] = __builtin_amdgcn_raw_buffer_load_b128(w_rs, w_vo[p & 1] + w_po(p), soff, 0);
      }
    }
  };

  // Pipeline.  LDS holds two steps (slots s % 2); each register stage holds
  // one step in flight.  At the barrier in the middle of step s (before its
  // last K quarter) every wave has finished reading slot s % 2, and the
  // stores of step s + 1 into the other slot are complete.  From there the
  // register stage of step s + 2 drains into slot s % 2 and refills with
  // step s + 4, spread over the last quarter of step s and the first three
  // of step s + 1; so a global load has about two steps to land.  Step s
  // (f0 holds its quarter 0 on entry), with P the stage of window s - 1 and
  // Q the stage of window s:
  //   read q1 -> f1 | MFMAs f0 | P items 4-7      (store s + 1, load s + 3)
  //   read q2 -> f0 | MFMAs f1 | P items 8-11
  //   read q3 -> f1 | MFMAs f0 | P items 12-15
  //   barrier
  //   read q0 of s + 1 -> f0 | MFMAs f1 | Q items 0-3  (store s + 2, load s + 4)
  // A workgroup runs a sequence of tiles.  The two LDS slots of a tile's
  // last two steps are free after their mid-step barriers; the next tile's
  // steps 0 and 1 are loaded straight into them from there (LDS-direct
  // loads), so that tile starts without waiting for memory.  The last steps
  // load nothing into the register stages, which are therefore free during
  // the epilogue.  (With an odd step count the host gives every workgroup a
  // single tile.)
  const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)smem;
  u32x4 nad{}, nwd{};   // the next tile's A and W
  bool has_next = false;
  auto dma_step = [&](int step) {   // step 0 or 1 of the next tile into slot `step` (K / 64 >= 6 here)
    const uint32_t sa = lds_base + step * kStage + kLoads * wave * 1024;
    const uint32_t sw = lds_base + step * kStage + kTileBytes + kLW * wave * 1024;
    const int soff = step * BK * 2;
#pragma unroll
    for (int u = 0; u < kLoads; ++u) {
      load_lds16(nad, a_vo[u & 1] + a_po(u), soff, sa + u * 1024);
      if (u < kLW) load_lds16(nwd, w_vo[u & 1] + w_po(u), soff, sw + u * 1024);
    }
  };
  Stage r0, r1;
  Frags f0, f1;
  // Step s: P drains step s + 1 (stP) and reloads with s + 3 (ldP), Q drains
  // step s + 2 (stQ) and reloads with s + 4 (ldQ); `dma` >= 0 loads step dma
  // of the next tile into slot dma after the barrier.  At the call sites the
  // flags are constants wherever possible, so the compiler knows exactly
  // which loads are in flight and derives exact wait counts.
  auto step = [&](int s, Stage& P, Stage& Q, bool first, bool stP, bool ldP, bool stQ, bool ldQ, int dma) {
    read(f1, s, 1);
    mma(f0);
    if (!first) io4(P, 4, s + 1, s + 3, stP, ldP);
    pattern();
    __builtin_amdgcn_sched_barrier(0);   // the quarter's reads stay in the quarter
    read(f0, s, 2);
    mma(f1);
    if (!first) io4(P, 8, s + 1, s + 3, stP, ldP);
    pattern();
    __builtin_amdgcn_sched_barrier(0);   // the quarter's reads stay in the quarter
    read(f1, s, 3);
    mma(f0);
    if (!first) io4(P, 12, s + 1, s + 3, stP, ldP);
    pattern();
    __builtin_amdgcn_sched_barrier(0);   // the quarter's reads stay in the quarter
    __syncthreads();
    if (dma >= 0) dma_step(dma);
    read(f0, s + 1, 0);   // after the last step: a harmless read of the idle slot
    mma(f1);
    io4(Q, 0, s + 2, s + 4, stQ, ldQ);
    pattern();
    __builtin_amdgcn_sched_barrier(0);   // the quarter's reads stay in the quarter
  };
  // first tile: slots 0 and 1 get steps 0 and 1 through the register stages
  // (with fewer K steps, steps past the end reload the last one; they fill
  // slots and registers that are never consumed)
  gload(r0, 0);
  gload(r1, 1);
  sstore(r0, 0);
  sstore(r1, 1);
  for (int it = 0;; ++it) {
    has_next = SEQ && it + 1 < seq.count;
    int tm1 = 0, tn1 = 0;
    if (has_next) {
      seq.coords(it + 1, tm1, tn1);
      nad = make_desc(A + (int64_t)tm1 * BM * lda, ((int64_t)(M - tm1 * BM - 1) * lda + K) * 2);
      nwd = make_desc(W + (int64_t)tn1 * BNT * ldw, ((int64_t)(N - tn1 * BNT - 1) * ldw + K) * 2);
    }
    // r0 / r1 carry steps 2 / 3; keep the two register stages' loads in this
    // order (as in the loop), so the wait counts the compiler derives inside
    // the loop stay exact
    __builtin_amdgcn_sched_barrier(0);
    gload(r0, 2);
    __builtin_amdgcn_sched_barrier(0);
    gload(r1, 3);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    read(f0, 0, 0);
    // an even step uses (P, Q) = (r1, r0), an odd one (r0, r1); window -1
    // (step 1 into slot 1) is already in LDS
    if constexpr (SEQ) {
      step(0, r1, r0, true, false, false, true, true, -1);
      int s = 1;
      for (; s + 5 < KT; s += 2) {
        step(s, r0, r1, false, true, true, true, true, -1);
        step(s + 1, r1, r0, false, true, true, true, true, -1);
      }
      // s = KT - 5: the last five steps, loads stop at step KT - 1
      step(s, r0, r1, false, true, true, true, true, -1);
      step(s + 1, r1, r0, false, true, true, true, false, -1);
      step(s + 2, r0, r1, false, true, false, true, false, -1);
      step(s + 3, r1, r0, false, true, false, false, false, has_next ? 0 : -1);
      step(s + 4, r0, r1, false, false, false, false, false, has_next ? 1 : -1);
    } else {   // any step count, a single tile
      step(0, r1, r0, true, false, false, 2 < KT, 4 < KT, -1);
      for (int s = 1; s < KT; s += 2) {
        step(s, r0, r1, false, s + 1 < KT, s + 3 < KT, s + 2 < KT, s + 4 < KT, -1);
        if (s + 1 < KT) step(s + 1, r1, r0, false, s + 2 < KT, s + 4 < KT, s + 3 < KT, s + 5 < KT, -1);
      }
    }
    if (has_next) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // the next tile's steps 0 and 1

  // Epilogue through a wave-private LDS window of 32 rows x 64 columns
  // (fp32): acc[i][j][4 g + e] = C[m][n] with m = m0 + wm*128 + 32j + fr and
  // n = n0 + wn*128 + 32i + 8g + 4fh + e.  Each round writes two column
  // blocks of one row block as the MFMAs left them (a lane: 4 consecutive
  // columns of one row) and reads them back row-contiguously, so each
  // global access of a wave covers whole 128-byte row segments.  16-byte
  // chunk c of window row r sits at physical chunk c ^ (r % 16): both the
  // writes and the reads are free of bank conflicts.  One wave's LDS
  // operations complete in order, so the window needs no barrier.
  // The residual rows of two row blocks (and the gate row of each block,
  // when all its rows belong to one request) are loaded before any of their
  // outputs is computed, so the epilogue waits for memory twice per tile;
  // the register stages are free here.  C may alias R: every element is
  // read before it is written, by the same lane.
  char* const ew = smem + kStages * kStage + wave * kEpiBytes;
  const int er = lane >> 4, ec = lane & 15;   // read role: rows er + 4 k, chunk ec
  float bsum[2][4];
  int64_t c_off[2];   // output plane of the lane's 4 columns (planes: column n in plane n / plane_cols)
#pragma unroll
  for (int ih = 0; ih < 2; ++ih) {
    const int n = n0 + wn * WN + 64 * ih + 4 * ec;
    c_off[ih] = plane_cols > 0 ? (int64_t)(n / plane_cols) * plane_skip : 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) bsum[ih][e] = 0.f;
    if (bias && n < N && 64 * ih + 4 * ec < WN) {
      const bf16x4 bv = *reinterpret_cast<const bf16x4*>(bias + n);
#pragma unroll
      for (int e = 0; e < 4; ++e) bsum[ih][e] = (float)bv[e];
    }
  }
#pragma unroll
  for (int hj = 0; hj < 2; ++hj) {
    constexpr bool kRes = EPI == DIT_EPI_RESIDUAL || EPI == DIT_EPI_GATED_RESIDUAL;
    bf16x4 rv[2][2][8];
    f32x4 gv[2][2];
    bool g_one[2];
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int mb = m0 + wm * 128 + 32 * (2 * hj + jj);   // first row of the block
      if (EPI == DIT_EPI_GATED_RESIDUAL) {
        const int r_lo = find_req(req.cu, req.n_req, min(mb, M - 1));
        const int r_hi = find_req(req.cu, req.n_req, min(mb + 31, M - 1));
        g_one[jj] = r_lo == r_hi;
#pragma unroll
        for (int ih = 0; ih < 2; ++ih) {
          const int n = n0 + wn * WN + 64 * ih + 4 * ec;
          gv[jj][ih] = f32x4{};
          if (g_one[jj] && n < N && 64 * ih + 4 * ec < WN)
            gv[jj][ih] = *reinterpret_cast<const f32x4*>(gate + (int64_t)r_lo * gate_stride + n);
        }
      }
      if (kRes) {
#pragma unroll
        for (int ih = 0; ih < 2; ++ih) {
          const int n = n0 + wn * WN + 64 * ih + 4 * ec;
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            const int m = mb + 4 * k + er;
            rv[jj][ih][k] = bf16x4{};
            if (m < M && n < N && 64 * ih + 4 * ec < WN)
              rv[jj][ih][k] = *reinterpret_cast<const bf16x4*>(R + (int64_t)m * ldr + n);
          }
        }
      }
    }
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int j = 2 * hj + jj;
#pragma unroll
      for (int ih = 0; ih < 2; ++ih) {
#pragma unroll
        for (int ii = 0; ii < 2; ++ii) {
          if (2 * ih + ii >= NI) continue;   // 3 W blocks: the last round holds one block (32 columns)
#pragma unroll
          for (int gq = 0; gq < 4; ++gq) {
            const f32x4 v = {acc[2 * ih + ii][j][4 * gq], acc[2 * ih + ii][j][4 * gq + 1],
                             acc[2 * ih + ii][j][4 * gq + 2], acc[2 * ih + ii][j][4 * gq + 3]};
            const int c = 8 * ii + 2 * gq + fh;
            *reinterpret_cast<f32x4*>(ew + fr * 256 + ((c ^ (fr & 15)) << 4)) = v;
          }
        }
        const int n = n0 + wn * WN + 64 * ih + 4 * ec;
        if (n >= N || 64 * ih + 4 * ec >= WN) continue;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const int r = 4 * k + er;
          const f32x4 zv = *reinterpret_cast<const f32x4*>(ew + r * 256 + ((ec ^ (r & 15)) << 4));
          const int m = m0 + wm * 128 + 32 * j + r;
          if (m >= M) continue;
          float z[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) z[e] = zv[e] + bsum[ih][e];
          if (EPI == DIT_EPI_GELU_TANH) {
#pragma unroll
            for (int e = 0; e < 4; ++e) z[e] = gelu_tanh(z[e]);
          } else if (EPI == DIT_EPI_GATED_RESIDUAL) {
            f32x4 g4 = gv[jj][ih];
            if (!g_one[jj])   // the block spans a request boundary
              g4 = *reinterpret_cast<const f32x4*>(gate + (int64_t)find_req(req.cu, req.n_req, m) * gate_stride + n);
#pragma unroll
            for (int e = 0; e < 4; ++e) z[e] = (float)rv[jj][ih][k][e] + g4[e] * z[e];
          } else if (EPI == DIT_EPI_RESIDUAL) {
#pragma unroll
            for (int e = 0; e < 4; ++e) z[e] = (float)rv[jj][ih][k][e] + z[e];
          }
          bf16x4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = (bf16)z[e];
          *reinterpret_cast<bf16x4*>(C + c_off[ih] + (int64_t)m * ldc + n) = o;
        }
      }
    }
  }
    if (!has_next) break;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};
    m0 = tm1 * BM;
    n0 = tn1 * BNT;
    a_rs = make_rsrc(A + (int64_t)m0 * lda, ((int64_t)(M - m0 - 1) * lda + K) * 2);
    w_rs = make_rsrc(W + (int64_t)n0 * ldw, ((int64_t)(N - n0 - 1) * ldw + K) * 2);
  }
}

// ----------------------------------------------------------------- fp32

constexpr int FT = 64;   // fp32 tile
constexpr int FK = 16;

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_nt(
    const float* __restrict__ A, int64_t lda, const float* __restrict__ W, int64_t ldw,
    const float* __restrict__ bias, float* C, int64_t ldc, const float* R, int64_t ldr,
    const float* __restrict__ gate, int64_t gate_stride, ReqTable req, int M, int N, int K, int plane_cols,
    int64_t plane_skip) {
  __shared__ float As[FK][FT + 1];
  __shared__ float Ws[FK][FT + 1];
  const int m0 = blockIdx.y * FT, n0 = blockIdx.x * FT;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += FK) {
    for (int i = threadIdx.x; i < FT * FK; i += 256) {
      int r = i / FK, kk = i % FK;
      int am = m0 + r, wn = n0 + r, k = k0 + kk;
      As[kk][r] = (am < M && k < K) ? A[(int64_t)am * lda + k] : 0.f;
      Ws[kk][r] = (wn < N && k < K) ? W[(int64_t)wn * ldw + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < FK; ++kk) {
      float a[4], w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        a[e] = As[kk][ty * 4 + e];
        w[e] = Ws[kk][tx * 4 + e];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], w[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    int m = m0 + ty * 4 + i;
    if (m >= M) continue;
    const float* g = nullptr;
    if (EPI == DIT_EPI_GATED_RESIDUAL) g = gate + (int64_t)find_req(req.cu, req.n_req, m) * gate_stride;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int n = n0 + tx * 4 + j;
      if (n >= N) continue;
      float z = acc[i][j] + (bias ? bias[n] : 0.f);
      if (EPI == DIT_EPI_GELU_TANH) z = gelu_tanh(z);
      else if (EPI == DIT_EPI_RESIDUAL) z = R[(int64_t)m * ldr + n] + z;
      else if (EPI == DIT_EPI_GATED_RESIDUAL) z = R[(int64_t)m * ldr + n] + g[n] * z;
      C[(plane_cols > 0 ? (int64_t)(n / plane_cols) * plane_skip : 0) + (int64_t)m * ldc + n] = z;
    }
  }
}


std::atomic<int> g_tile_n{0};   // forced output tile width (0: chosen per shape)

template <int EPI, int BNT>
hipError_t launch_bf16_tiles(const LinearArgs& p, int tiles_m, int tiles_n, hipStream_t s) {
  const int tiles = tiles_m * tiles_n;
  int grid = (tiles + kXcds - 1) / kXcds * kXcds;   // one tile per workgroup
  const int kt = p.K / BK;
  const int group_m = tiles_m <= kFewTileRows ? kGroupMFew : kGroupM;
  if (kt % 2 == 0 && kt >= 6) {
    // one workgroup per compute unit, each running a sequence of tiles
    const int resident = cu_count() / kXcds * kXcds;
    if (resident >= kXcds && grid > resident) grid = resident;
    gemm_bf16_nt<EPI, true, BNT><<<grid, kThreads, 0, s>>>(
        (const bf16*)p.a, p.lda, (const bf16*)p.w, p.ldw, (const bf16*)p.bias, (bf16*)p.out, p.ldo,
        (const bf16*)p.res, p.ldr, p.gate, p.gate_stride, p.req, (int)p.M, p.N, p.K, tiles_m, tiles_n,
        group_m, p.plane_cols, p.plane_stride - p.plane_cols);
  } else {
    gemm_bf16_nt<EPI, false, BNT><<<grid, kThreads, 0, s>>>(
        (const bf16*)p.a, p.lda, (const bf16*)p.w, p.ldw, (const bf16*)p.bias, (bf16*)p.out, p.ldo,
        (const bf16*)p.res, p.ldr, p.gate, p.gate_stride, p.req, (int)p.M, p.N, p.K, tiles_m, tiles_n,
        group_m, p.plane_cols, p.plane_stride - p.plane_cols);
  }
  return hipGetLastError();
}

// Output tiles are 256 x 256, or 256 x 192 where that needs fewer rounds of
// tiles over the compute units: with few tiles the last round leaves compute
// units idle (4,096 rows x 3,072 columns: 192 tiles of 256 x 256 on 256 CUs,
// but exactly 256 of 256 x 192).  A round of narrow tiles is costed at
// 192 / 256 of a wide one, plus 8% (7 fragment reads per 12 MFMAs instead of
// 8 per 16).
template <int EPI>
hipError_t launch_bf16(const LinearArgs& p, hipStream_t s) {
  const int tiles_m = (int)((p.M + BM - 1) / BM);
  const int cus = cu_count();
  auto rounds = [&](int bn) { return ((int64_t)tiles_m * ((p.N + bn - 1) / bn) + cus - 1) / cus; };
  int bn = g_tile_n.load(std::memory_order_relaxed);
  if (bn != 192 && bn != 256) bn = rounds(192) * 192 * 108 < rounds(256) * 256 * 100 ? 192 : 256;
  if (bn == 192) return launch_bf16_tiles<EPI, 192>(p, tiles_m, (p.N + 191) / 192, s);
  return launch_bf16_tiles<EPI, 256>(p, tiles_m, (p.N + 255) / 256, s);
}

template <int EPI>
hipError_t launch_f32(const LinearArgs& p, hipStream_t s) {
  dim3 grid((p.N + FT - 1) / FT, (unsigned)((p.M + FT - 1) / FT));
  gemm_f32_nt<EPI><<<grid, 256, 0, s>>>(
      (const float*)p.a, p.lda, (const float*)p.w, p.ldw, (const float*)p.bias, (float*)p.out, p.ldo,
      (const float*)p.res, p.ldr, p.gate, p.gate_stride, p.req, (int)p.M, p.N, p.K, p.plane_cols,
      p.plane_stride - p.plane_cols);
  return hipGetLastError();
}

}  // namespace

// Compute units of the current device (cached per device).
int cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

void set_gemm_tile_n(int bn) { g_tile_n.store(bn, std::memory_order_relaxed); }

hipError_t launch_linear(const LinearArgs& p, hipStream_t s) {
  if (p.M == 0) return hipSuccess;
  if (p.dtype == DIT_BF16) {
    switch (p.epi) {
      case DIT_EPI_NONE: return launch_bf16<DIT_EPI_NONE>(p, s);
      case DIT_EPI_GELU_TANH: return launch_bf16<DIT_EPI_GELU_TANH>(p, s);
      case DIT_EPI_RESIDUAL: return launch_bf16<DIT_EPI_RESIDUAL>(p, s);
      default: return launch_bf16<DIT_EPI_GATED_RESIDUAL>(p, s);
    }
  }
  switch (p.epi) {
    case DIT_EPI_NONE: return launch_f32<DIT_EPI_NONE>(p, s);
    case DIT_EPI_GELU_TANH: return launch_f32<DIT_EPI_GELU_TANH>(p, s);
    case DIT_EPI_RESIDUAL: return launch_f32<DIT_EPI_RESIDUAL>(p, s);
    default: return launch_f32<DIT_EPI_GATED_RESIDUAL>(p, s);
  }
}

}  // namespace dit
