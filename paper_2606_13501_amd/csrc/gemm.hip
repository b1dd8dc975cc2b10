// Projections of the DiT block: out = epilogue(A . W^T + bias).
//
// bf16: a 256x256 output tile per 256-thread workgroup on the gfx950 matrix
// cores (v_mfma_f32_32x32x16_bf16), fp32 accumulation.  Each of the 4 waves
// (one per SIMD) owns a 128x128 sub-tile whose accumulators (256 registers)
// live in the accumulation registers.  The K loop runs in steps of 64: a
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
// Workgroups are rastered in groups of 4 tile rows per XCD so the tiles
// resident on one XCD share A and W panels in its L2.
//
// fp32: a plain 64x64 LDS-tiled FMA kernel for the small exact configuration.
#include "common.hpp"
#include "kernels.hpp"

namespace dit {

namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kWaves = 4;                           // 2 x 2 waves, each a 128 x 128 sub-tile
constexpr int kThreads = 64 * kWaves;
constexpr int kStages = 2;                          // LDS double buffer
constexpr int kRowBytes = BK * 2;                   // 128 B: one full cache line per tile row
constexpr int kTileBytes = BM * kRowBytes;          // one operand tile of one step (32 KiB)
constexpr int kStageBytes = 2 * kTileBytes;         // A tile + W tile
constexpr int kLoads = kTileBytes / 1024 / kWaves;  // 1 KiB loads per wave, operand and step (8)
constexpr int kEpiBytes = 32 * 256;                 // per wave: 32 rows x 64 fp32 (epilogue window)
constexpr int kGroupM = 4;                          // tile rows per raster group
constexpr int kXcds = 8;                            // gfx950: 8 XCDs, workgroups dispatched round-robin

// gelu_tanh(z) = z (1 + tanh u) / 2 = z / (1 + e^(-2u)), u = sqrt(2/pi) (z + 0.044715 z^3)
__device__ __forceinline__ float gelu_tanh(float z) {
  const float k0 = 0.7978845608028654f;  // sqrt(2/pi)
  const float k1 = 0.044715f;
  const float u = k0 * fmaf(k1 * z, z * z, z);
  const float e = __builtin_amdgcn_exp2f(-2.0f * 1.4426950408889634f * u);   // inf for u << 0: z / inf = 0
  return z * __builtin_amdgcn_rcpf(1.0f + e);
}

// Logical tile of hardware workgroup b: each XCD gets a contiguous range of
// logical tiles, and tiles are rastered in groups of kGroupM tile rows so the
// workgroups resident on one XCD share A and W panels in its L2.
__device__ __forceinline__ bool tile_of(int b, int nb, int tiles_m, int tiles_n, int& tm, int& tn) {
  int per_xcd = nb / kXcds;
  int t = (b % kXcds) * per_xcd + b / kXcds;
  if (t >= tiles_m * tiles_n) return false;
  int width = kGroupM * tiles_n;
  int group = t / width;
  int first_m = group * kGroupM;
  int gsize = min(tiles_m - first_m, kGroupM);
  int r = t - group * width;
  tm = first_m + r % gsize;
  tn = r / gsize;
  return true;
}

// 16-byte chunk swizzle of a 128-byte LDS row: a fragment read touches 16
// consecutive rows at one logical chunk; rows 2t and 2t + 1 lie in different
// halves of a 256-byte bank window and the physical chunk c ^ t differs
// between the 8 values of t, so the 16 reads hit 16 distinct bank groups.
__device__ __forceinline__ int row_swizzle(int r) { return (r >> 1) & 7; }

// Raw buffer descriptor over `bytes` bytes from `base`: loads past the end
// return zeros, which covers the ragged last tile without clamping.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const uint32_t n = bytes > 0xFFFFFFFFll ? 0xFFFFFFFFu : (uint32_t)(bytes < 0 ? 0 : bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}

template <int EPI>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_nt(
    const bf16* __restrict__ A, int64_t lda, const bf16* __restrict__ W, int64_t ldw,
    const bf16* __restrict__ bias, bf16* __restrict__ C, int64_t ldc, const bf16* R, int64_t ldr,
    const float* __restrict__ gate, int64_t gate_stride, ReqTable req, int M, int N, int K,
    int tiles_m, int tiles_n) {
  __shared__ __attribute__((aligned(1024))) char smem[kStages * kStageBytes + kWaves * kEpiBytes];

  int tm, tn;
  if (!tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn)) return;
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  // ---- global -> registers -> LDS.  A step's operand tile is 32 pieces of
  // 1 KiB (8 rows x 128 B); wave w moves pieces q = 8 w .. 8 w + 7 of A and
  // of W.  Lane i of piece q holds row 8 q + i / 8, logical chunk
  // (i % 8) ^ row_swizzle(row), and stores it at LDS byte q * 1024 + 16 i,
  // i.e. physical chunk i % 8 of that row.
  const auto a_rs = make_rsrc(A + (int64_t)m0 * lda, ((int64_t)(M - m0 - 1) * lda + K) * 2);
  const auto w_rs = make_rsrc(W + (int64_t)n0 * ldw, ((int64_t)(N - n0 - 1) * ldw + K) * 2);
  int a_voff[kLoads], w_voff[kLoads];
#pragma unroll
  for (int u = 0; u < kLoads; ++u) {
    const int q = kLoads * wave + u;
    const int r = 8 * q + (lane >> 3);
    const int c = (lane & 7) ^ row_swizzle(r);
    a_voff[u] = r * (int)lda * 2 + c * 16;
    w_voff[u] = r * (int)ldw * 2 + c * 16;
  }
  struct Stage { u32x4 a[kLoads], w[kLoads]; };   // one step of this wave's pieces
  auto gload = [&](Stage& r, int step) {
    const int soff = step * BK * 2;
#pragma unroll
    for (int u = 0; u < kLoads; ++u) {
      r.a[u] = __builtin_amdgcn_raw_buffer_load_b128(a_rs, a_voff[u], soff, 0);
      r.w[u] = __builtin_amdgcn_raw_buffer_load_b128(w_rs, w_voff[u], soff, 0);
    }
  };
  auto sstore = [&](const Stage& r, int step) {
    char* st = smem + (step % kStages) * kStageBytes + kLoads * wave * 1024 + lane * 16;
#pragma unroll
    for (int u = 0; u < kLoads; ++u) {
      *reinterpret_cast<u32x4*>(st + u * 1024) = r.a[u];
      *reinterpret_cast<u32x4*>(st + kTileBytes + u * 1024) = r.w[u];
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
    fo_w[kk] = kTileBytes + (wn * 128 + fr) * kRowBytes + (((2 * kk + fh) ^ sw) << 4);
  }
  struct Frags { bf16x8 w[4], a[4]; };
  auto read = [&](Frags& f, int step, int kk) {
    const char* st = smem + (step % kStages) * kStageBytes;
#pragma unroll
    for (int i = 0; i < 4; ++i) f.w[i] = *reinterpret_cast<const bf16x8*>(st + fo_w[kk] + i * 32 * kRowBytes);
#pragma unroll
    for (int j = 0; j < 4; ++j) f.a[j] = *reinterpret_cast<const bf16x8*>(st + fo_a[kk] + j * 32 * kRowBytes);
  };

  // acc[i][j]: W block i (4 x 32 columns of the wave), A block j (4 x 32 rows)
  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};
  auto mma = [&](const Frags& f) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.w[i], f.a[j], acc[i][j], 0, 0, 0);
  };
  const int KT = K / BK;
  // Per K quarter: 16 MFMAs, 8 fragment reads, and (when a register stage
  // is being cycled) 4 LDS stores + 4 global loads, spread evenly: per 4
  // MFMAs 2 reads, 1 store and 1 load.  An even stream of global loads keeps
  // the memory pipeline busy without bursts that would stall MFMA issue.
  auto pattern = [] {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
  };
  // items u0 .. u0 + 3 of a register stage (items 0-7: A pieces, 8-15: W
  // pieces): store each into the LDS slot of step st_step, then reload it
  // with step ld_step (skipped past the last step when `guard`)
  auto io4 = [&](Stage& R, int u0, int st_step, int ld_step, bool guard) {
    char* st = smem + (st_step % kStages) * kStageBytes + kLoads * wave * 1024 + lane * 16;
    const int soff = ld_step * BK * 2;
#pragma unroll
    for (int u = u0; u < u0 + 4; ++u) {
      const int p = u & 7;
      u32x4& v = u < 8 ? R.a[p] : R.w[p];
      if (!guard || st_step < KT) *reinterpret_cast<u32x4*>(st + (u < 8 ? 0 : kTileBytes) + p * 1024) = v;
      if (!guard || ld_step < KT)
        v = __builtin_amdgcn_raw_buffer_load_b128(u < 8 ? a_rs : w_rs, u < 8 ? a_voff[p] : w_voff[p], soff, 0);
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
  Stage r0, r1;
  // prologue: slots 0 and 1 hold steps 0 and 1, r0 / r1 carry steps 2 / 3
  // (steps past the end load zeros or bytes of later rows; they fill slots
  // and registers that are never consumed)
  gload(r0, 0);
  gload(r1, 1);
  sstore(r0, 0);
  sstore(r1, 1);
  // keep the two register stages' loads in this order (as in the loop), so
  // the wait counts the compiler derives inside the loop stay exact
  __builtin_amdgcn_sched_barrier(0);
  gload(r0, 2);
  __builtin_amdgcn_sched_barrier(0);
  gload(r1, 3);
  __builtin_amdgcn_sched_barrier(0);
  __syncthreads();
  Frags f0, f1;
  read(f0, 0, 0);

  auto step = [&](int s, Stage& P, Stage& Q, bool guard, bool first) {
    read(f1, s, 1);
    mma(f0);
    if (!first) io4(P, 4, s + 1, s + 3, guard);
    pattern();
    read(f0, s, 2);
    mma(f1);
    if (!first) io4(P, 8, s + 1, s + 3, guard);
    pattern();
    read(f1, s, 3);
    mma(f0);
    if (!first) io4(P, 12, s + 1, s + 3, guard);
    pattern();
    __syncthreads();
    read(f0, s + 1, 0);   // after the last step: a harmless read of the idle slot
    mma(f1);
    io4(Q, 0, s + 2, s + 4, guard);
    pattern();
  };
  step(0, r1, r0, true, true);   // window -1 (step 1 into slot 1) was the prologue
  int s = 1;
  for (; s + 5 < KT; s += 2) {
    step(s, r0, r1, false, false);
    step(s + 1, r1, r0, false, false);
  }
  for (; s < KT; s += 2) {
    step(s, r0, r1, true, false);
    if (s + 1 < KT) step(s + 1, r1, r0, true, false);
  }

  // Epilogue through a wave-private LDS window of 32 rows x 64 columns
  // (fp32): acc[i][j][4 g + e] = C[m][n] with m = m0 + wm*128 + 32j + fr and
  // n = n0 + wn*128 + 32i + 8g + 4fh + e.  Each round writes two column
  // blocks of one row block as the MFMAs left them (a lane: 4 consecutive
  // columns of one row) and reads them back row-contiguously, so each
  // global access of a wave covers whole 128-byte row segments.  16-byte
  // chunk c of window row r sits at physical chunk c ^ (r % 16): both the
  // writes and the reads are free of bank conflicts.  One wave's LDS
  // operations complete in order, so the window needs no barrier.
  char* const ew = smem + kStages * kStageBytes + wave * kEpiBytes;
  const int er = lane >> 4, ec = lane & 15;   // read role: rows er + 4 k, chunk ec
#pragma unroll
  for (int j = 0; j < 4; ++j) {
#pragma unroll
    for (int ih = 0; ih < 2; ++ih) {
#pragma unroll
      for (int ii = 0; ii < 2; ++ii)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
          const f32x4 v = {acc[2 * ih + ii][j][4 * gq], acc[2 * ih + ii][j][4 * gq + 1],
                           acc[2 * ih + ii][j][4 * gq + 2], acc[2 * ih + ii][j][4 * gq + 3]};
          const int c = 8 * ii + 2 * gq + fh;
          *reinterpret_cast<f32x4*>(ew + fr * 256 + ((c ^ (fr & 15)) << 4)) = v;
        }
      // all of a round's loads are issued before its first store: C may
      // alias R, so no load could be moved above an earlier store
      const int n = n0 + wn * 128 + 64 * ih + 4 * ec;
      const bool n_ok = n < N;
      float bsum[4] = {0.f, 0.f, 0.f, 0.f};
      if (bias && n_ok) {
        const bf16x4 bv = *reinterpret_cast<const bf16x4*>(bias + n);
#pragma unroll
        for (int e = 0; e < 4; ++e) bsum[e] = (float)bv[e];
      }
      f32x4 zv[8];
      bf16x4 rv[8];
      f32x4 gv[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int r = 4 * k + er;
        zv[k] = *reinterpret_cast<const f32x4*>(ew + r * 256 + ((ec ^ (r & 15)) << 4));
        const int m = m0 + wm * 128 + 32 * j + r;
        if (EPI == DIT_EPI_RESIDUAL || EPI == DIT_EPI_GATED_RESIDUAL) {
          rv[k] = bf16x4{};
          if (m < M && n_ok) rv[k] = *reinterpret_cast<const bf16x4*>(R + (int64_t)m * ldr + n);
        }
        if (EPI == DIT_EPI_GATED_RESIDUAL) {
          gv[k] = f32x4{};
          if (m < M && n_ok)
            gv[k] = *reinterpret_cast<const f32x4*>(gate + (int64_t)find_req(req.cu, req.n_req, m) * gate_stride + n);
        }
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int m = m0 + wm * 128 + 32 * j + 4 * k + er;
        if (m >= M || !n_ok) continue;
        float z[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) z[e] = zv[k][e] + bsum[e];
        if (EPI == DIT_EPI_GELU_TANH) {
#pragma unroll
          for (int e = 0; e < 4; ++e) z[e] = gelu_tanh(z[e]);
        } else if (EPI == DIT_EPI_GATED_RESIDUAL) {
#pragma unroll
          for (int e = 0; e < 4; ++e) z[e] = (float)rv[k][e] + gv[k][e] * z[e];
        } else if (EPI == DIT_EPI_RESIDUAL) {
#pragma unroll
          for (int e = 0; e < 4; ++e) z[e] = (float)rv[k][e] + z[e];
        }
        bf16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (bf16)z[e];
        *reinterpret_cast<bf16x4*>(C + (int64_t)m * ldc + n) = o;
      }
    }
  }
}

// ----------------------------------------------------------------- fp32

constexpr int FT = 64;   // fp32 tile
constexpr int FK = 16;

template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_nt(
    const float* __restrict__ A, int64_t lda, const float* __restrict__ W, int64_t ldw,
    const float* __restrict__ bias, float* C, int64_t ldc, const float* R, int64_t ldr,
    const float* __restrict__ gate, int64_t gate_stride, ReqTable req, int M, int N, int K) {
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
      C[(int64_t)m * ldc + n] = z;
    }
  }
}

template <int EPI>
hipError_t launch_bf16(const LinearArgs& p, hipStream_t s) {
  int tiles_m = (int)((p.M + BM - 1) / BM);
  int tiles_n = (p.N + BN - 1) / BN;
  int tiles = tiles_m * tiles_n;
  int grid = (tiles + kXcds - 1) / kXcds * kXcds;
  gemm_bf16_nt<EPI><<<grid, kThreads, 0, s>>>(
      (const bf16*)p.a, p.lda, (const bf16*)p.w, p.ldw, (const bf16*)p.bias, (bf16*)p.out, p.ldo,
      (const bf16*)p.res, p.ldr, p.gate, p.gate_stride, p.req, (int)p.M, p.N, p.K, tiles_m, tiles_n);
  return hipGetLastError();
}

template <int EPI>
hipError_t launch_f32(const LinearArgs& p, hipStream_t s) {
  dim3 grid((p.N + FT - 1) / FT, (unsigned)((p.M + FT - 1) / FT));
  gemm_f32_nt<EPI><<<grid, 256, 0, s>>>(
      (const float*)p.a, p.lda, (const float*)p.w, p.ldw, (const float*)p.bias, (float*)p.out, p.ldo,
      (const float*)p.res, p.ldr, p.gate, p.gate_stride, p.req, (int)p.M, p.N, p.K);
  return hipGetLastError();
}

}  // namespace

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
