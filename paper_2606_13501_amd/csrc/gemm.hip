// Projections of the DiT block: out = epilogue(A . W^T + bias).
//
// bf16: a 256x256x64 tile per 256-thread workgroup on the gfx950 matrix cores
// (v_mfma_f32_32x32x16_bf16), fp32 accumulation, operands staged through LDS
// (two stages, XOR-swizzled 16-byte chunks so the fragment reads are free of
// bank conflicts).  Each wave owns a 128x128 sub-tile (4x4 MFMA blocks).  The
// kernel computes C^T blocks (W as the MFMA A operand) so that every lane ends
// up holding four consecutive output columns of one row, which are stored as a
// single 8-byte write together with the fused epilogue.
//
// fp32: a plain 64x64 LDS-tiled FMA kernel for the small exact configuration.
#include "common.hpp"
#include "kernels.hpp"

namespace dit {

namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int kThreads = 256;
constexpr int kTileBytes = BM * BK * 2;       // one operand tile, bytes
constexpr int kStageBytes = 2 * kTileBytes;   // A tile + W tile
constexpr int kGroupM = 8;                    // tile rows per raster group
constexpr int kXcds = 8;                      // gfx950: 8 XCDs, workgroups dispatched round-robin

__device__ __forceinline__ float gelu_tanh(float z) {
  const float k0 = 0.7978845608028654f;  // sqrt(2/pi)
  const float k1 = 0.044715f;
  float u = k0 * (z + k1 * z * z * z);
  return 0.5f * z * (1.0f + tanhf(u));
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

// Raw buffer resource over `bytes` bytes from `base`: loads past the end
// return zeros, which covers the ragged last tile without clamping.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  uint32_t n = bytes > 0xFFFFFFFFll ? 0xFFFFFFFFu : (uint32_t)(bytes < 0 ? 0 : bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}

template <int EPI>
__global__ __launch_bounds__(kThreads, 1) void gemm_bf16_nt(
    const bf16* __restrict__ A, int64_t lda, const bf16* __restrict__ W, int64_t ldw,
    const bf16* __restrict__ bias, bf16* __restrict__ C, int64_t ldc, const bf16* R, int64_t ldr,
    const float* __restrict__ gate, int64_t gate_stride, ReqTable req, int M, int N, int K,
    int tiles_m, int tiles_n) {
  __shared__ __attribute__((aligned(16))) char smem[2 * kStageBytes];

  int tm, tn;
  if (!tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn)) return;
  const int m0 = tm * BM, n0 = tn * BN;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // global -> register staging: chunk (row lrow + 32 i, 16-byte column lkc)
  const int lrow = tid >> 3;
  const int lkc = tid & 7;
  // ranges end at the last element of the operand's last row (row stride may exceed K)
  const __amdgpu_buffer_rsrc_t ra_rs = make_rsrc(A + (int64_t)m0 * lda, ((int64_t)(M - m0 - 1) * lda + K) * 2);
  const __amdgpu_buffer_rsrc_t rw_rs = make_rsrc(W + (int64_t)n0 * ldw, ((int64_t)(N - n0 - 1) * ldw + K) * 2);
  const int va = lrow * (int)lda * 2 + lkc * 16;
  const int vw = lrow * (int)ldw * 2 + lkc * 16;
  const int sa = 32 * (int)lda * 2;   // byte step between the thread's rows
  const int sw = 32 * (int)ldw * 2;
  const int st_off = lrow * 128 + ((lkc ^ (lrow & 7)) << 4);   // + 4096 i

  u32x4 ra[8], rw[8];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      ra[i] = __builtin_amdgcn_raw_buffer_load_b128(ra_rs, va, i * sa + k0 * 2, 0);
      rw[i] = __builtin_amdgcn_raw_buffer_load_b128(rw_rs, vw, i * sw + k0 * 2, 0);
    }
  };
  auto sstore = [&](int stage) {
    char* as = smem + stage * kStageBytes;
    char* ws = as + kTileBytes;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      *reinterpret_cast<u32x4*>(as + st_off + 4096 * i) = ra[i];
      *reinterpret_cast<u32x4*>(ws + st_off + 4096 * i) = rw[i];
    }
  };

  // fragment reads: row = base + 32 b + (lane & 31), 16-byte column 2 kk + (lane >> 5)
  const int fr = lane & 31;
  const int fh = lane >> 5;
  const int sw_x = fh ^ (fr & 7);
  int fo_w[4], fo_a[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    fo_w[kk] = (wn * 128 + fr) * 128 + (((2 * kk) ^ sw_x) << 4);
    fo_a[kk] = (wm * 128 + fr) * 128 + (((2 * kk) ^ sw_x) << 4);
  }

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};

  const int KT = K / BK;
  gload(0);
  sstore(0);
  __syncthreads();

  // Loop body is one basic block: the last iteration loads and stores one
  // unused stage (loads past the operand return zeros or in-range data), so
  // the instruction interleave below applies to every iteration.
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    gload((kt + 1) * BK);
    const char* as = smem + cur * kStageBytes;
    const char* ws = as + kTileBytes;
    // fragments of step kk+1 are read while the MFMAs of step kk run
    bf16x8 fw[2][4], fa[2][4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      fw[0][b] = *reinterpret_cast<const bf16x8*>(ws + fo_w[0] + b * 4096);
      fa[0][b] = *reinterpret_cast<const bf16x8*>(as + fo_a[0] + b * 4096);
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int c = kk & 1;
      if (kk + 1 < 4) {
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          fw[c ^ 1][b] = *reinterpret_cast<const bf16x8*>(ws + fo_w[kk + 1] + b * 4096);
          fa[c ^ 1][b] = *reinterpret_cast<const bf16x8*>(as + fo_a[kk + 1] + b * 4096);
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[c][i], fa[c][j], acc[i][j], 0, 0, 0);
    }
    sstore(cur ^ 1);
    // interleave: global loads and fragment reads between the MFMAs
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);   // frags of step 0
#pragma unroll
    for (int kk = 0; kk < 3; ++kk) {
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (kk < 2) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
    }
    __syncthreads();
  }

  // epilogue: acc[i][j][4g+e] = C[m][n] with m = m0 + wm*128 + 32j + (lane&31),
  // n = n0 + wn*128 + 32i + 8g + 4*(lane>>5) + e
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int m = m0 + wm * 128 + 32 * j + fr;
    if (m >= M) continue;
    const float* g = nullptr;
    if (EPI == DIT_EPI_GATED_RESIDUAL) g = gate + (int64_t)find_req(req.cu, req.n_req, m) * gate_stride;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int n = n0 + wn * 128 + 32 * i + 8 * gq + 4 * fh;
        if (n >= N) continue;
        float z[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) z[e] = acc[i][j][4 * gq + e];
        if (bias) {
          bf16x4 bv = *reinterpret_cast<const bf16x4*>(bias + n);
#pragma unroll
          for (int e = 0; e < 4; ++e) z[e] += (float)bv[e];
        }
        if (EPI == DIT_EPI_GELU_TANH) {
#pragma unroll
          for (int e = 0; e < 4; ++e) z[e] = gelu_tanh(z[e]);
        } else if (EPI == DIT_EPI_RESIDUAL || EPI == DIT_EPI_GATED_RESIDUAL) {
          bf16x4 rv = *reinterpret_cast<const bf16x4*>(R + (int64_t)m * ldr + n);
          if (EPI == DIT_EPI_GATED_RESIDUAL) {
            f32x4 gv = *reinterpret_cast<const f32x4*>(g + n);
#pragma unroll
            for (int e = 0; e < 4; ++e) z[e] = (float)rv[e] + gv[e] * z[e];
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) z[e] = (float)rv[e] + z[e];
          }
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
