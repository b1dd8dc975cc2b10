// Latent <-> token kernels of the denoising step: patchify (fp32 latent ->
// patch vectors in the compute dtype) and unpatchify fused with the
// flow-matching Euler update (latent_out = latent + dt * velocity).
//
// Both kernels walk the latent in its own channel-major order, so the fp32
// latent (the larger side: 4 bytes per value against 2 for bf16 tokens) is read
// and written with consecutive lanes on consecutive addresses; the token side
// is gathered or scattered and stays in L2 (a token row of P values is touched
// by pt*ph rows of pw adjacent latent values each).
#include "common.hpp"
#include "kernels.hpp"

namespace dit {

namespace {

// Position of latent element `idx` (global over all requests): its request,
// token row and patch-vector column.
__device__ __forceinline__ void latent_coords(const LatentTable& tab, int64_t idx, int* req, int64_t* row,
                                              int* col) {
  int lo = 0, hi = tab.n_req - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (tab.lat_off[mid] <= idx) lo = mid; else hi = mid - 1;
  }
  const int r = lo;
  const int gh = tab.grid_h[r], gw = tab.grid_w[r];
  const int64_t lw = (int64_t)gw * tab.pw, lh = (int64_t)gh * tab.ph;
  const int64_t plane = (tab.lat_off[r + 1] - tab.lat_off[r]) / tab.C;   // F*pt * H*ph * W*pw
  const int64_t e = idx - tab.lat_off[r];
  const int c = (int)(e / plane);
  const int64_t rem = e - (int64_t)c * plane;
  const int64_t x = rem % lw;
  const int64_t y = (rem / lw) % lh;
  const int64_t z = rem / (lw * lh);
  const int64_t f = z / tab.pt, h = y / tab.ph, w = x / tab.pw;
  const int i = (int)(z - f * tab.pt), j = (int)(y - h * tab.ph), k = (int)(x - w * tab.pw);
  *req = r;
  *row = tab.row0[r] + (f * gh + h) * gw + w;
  *col = ((c * tab.pt + i) * tab.ph + j) * tab.pw + k;
}

template <typename T>
__global__ __launch_bounds__(256) void patchify_kernel(const float* __restrict__ latent, T* __restrict__ tokens,
                                                      LatentTable tab) {
  const int64_t n = tab.lat_off[tab.n_req];
  const int P = tab.C * tab.pt * tab.ph * tab.pw;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n;
       idx += (int64_t)gridDim.x * blockDim.x) {
    int r, col;
    int64_t row;
    latent_coords(tab, idx, &r, &row, &col);
    tokens[row * P + col] = from_f<T>(latent[idx]);
  }
}

// latent and out may be the same buffer: each element is read, then written, by one thread.
template <typename T>
__global__ __launch_bounds__(256) void unpatchify_euler_kernel(const float* latent, const T* __restrict__ v,
                                                              const float* __restrict__ dt, float* out,
                                                              LatentTable tab) {
  const int64_t n = tab.lat_off[tab.n_req];
  const int P = tab.C * tab.pt * tab.ph * tab.pw;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n;
       idx += (int64_t)gridDim.x * blockDim.x) {
    int r, col;
    int64_t row;
    latent_coords(tab, idx, &r, &row, &col);
    out[idx] = fmaf(dt[r], to_f<T>(v[row * P + col]), latent[idx]);
  }
}

unsigned latent_grid(int64_t n) {
  const int64_t blocks = (n + 255) / 256;
  return (unsigned)(blocks < 8192 ? (blocks > 0 ? blocks : 1) : 8192);
}

}  // namespace

hipError_t launch_patchify(const LatentArgs& p, hipStream_t s) {
  const int64_t n = p.tab.lat_off[p.tab.n_req];
  if (n == 0) return hipSuccess;
  if (p.dtype == DIT_BF16)
    patchify_kernel<bf16><<<latent_grid(n), 256, 0, s>>>(p.latent, (bf16*)p.tokens, p.tab);
  else
    patchify_kernel<float><<<latent_grid(n), 256, 0, s>>>(p.latent, (float*)p.tokens, p.tab);
  return hipGetLastError();
}

hipError_t launch_unpatchify_euler(const LatentArgs& p, hipStream_t s) {
  const int64_t n = p.tab.lat_off[p.tab.n_req];
  if (n == 0) return hipSuccess;
  if (p.dtype == DIT_BF16)
    unpatchify_euler_kernel<bf16><<<latent_grid(n), 256, 0, s>>>(p.latent, (const bf16*)p.tokens, p.dt,
                                                                p.latent_out, p.tab);
  else
    unpatchify_euler_kernel<float><<<latent_grid(n), 256, 0, s>>>(p.latent, (const float*)p.tokens, p.dt,
                                                                 p.latent_out, p.tab);
  return hipGetLastError();
}

}  // namespace dit
