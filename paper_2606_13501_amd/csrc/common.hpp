// Shared device helpers for the gfx950 kernels of the DiT block library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dit_block.h"

namespace dit {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// Per-request metadata of a packed batch, passed by value in kernel arguments.
struct ReqTable {
  int n_req;
  int cu[DIT_MAX_REQ + 1];
};

struct RopeTable {
  int n_req;
  int cu[DIT_MAX_REQ + 1];
  int grid_hw[DIT_MAX_REQ];   // H*W of the request's token grid
  int grid_w[DIT_MAX_REQ];    // W
  int grid_h[DIT_MAX_REQ];    // H
  int offset[DIT_MAX_REQ];    // flattened grid index of the first row
};

// Geometry of the packed latent of a denoising step: request r's fp32 latent
// [C, F*pt, H*ph, W*pw] occupies elements lat_off[r]..lat_off[r+1]; its tokens
// are rows row0[r].. of the token matrix in (f, h, w) order.  The latent
// kernels work in tiles of up to `wt` consecutive tokens of one (f, h) token
// row; request r owns tiles tile_off[r]..tile_off[r+1].
struct LatentTable {
  int n_req;
  int C, pt, ph, pw;
  int wt;
  int64_t lat_off[DIT_MAX_REQ + 1];
  int tile_off[DIT_MAX_REQ + 1];
  int row0[DIT_MAX_REQ];
  int grid_h[DIT_MAX_REQ];
  int grid_w[DIT_MAX_REQ];
};

__device__ __forceinline__ float bf2f(bf16 v) { return (float)v; }
__device__ __forceinline__ bf16 f2bf(float v) { return (bf16)v; }

template <typename T> __device__ __forceinline__ float to_f(T v);
template <> __device__ __forceinline__ float to_f<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f<bf16>(bf16 v) { return (float)v; }

template <typename T> __device__ __forceinline__ T from_f(float v);
template <> __device__ __forceinline__ float from_f<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f<bf16>(float v) { return (bf16)v; }

// Request owning global row `row` (rows of request r are cu[r]..cu[r+1]).
__device__ __forceinline__ int find_req(const int* cu, int n_req, int row) {
  int lo = 0, hi = n_req - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

}  // namespace dit
