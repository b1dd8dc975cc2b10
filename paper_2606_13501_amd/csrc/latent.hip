// Latent <-> token kernels of the denoising step: patchify (fp32 latent ->
// patch vectors in the compute dtype) and unpatchify fused with the
// flow-matching Euler update (latent_out = latent + dt * velocity).
//
// One workgroup moves one tile: up to `wt` consecutive tokens (f, h, w0..) of
// one request.  Their patch vectors are one contiguous run of the token
// matrix, and their latent values are C*pt*ph runs of wt*pw consecutive
// values, one per (c, i, j).  The tile is transposed through LDS so that both
// sides are read and written with consecutive lanes on consecutive addresses;
// LDS rows are padded to P + 1 floats so that the pw-strided accesses of the
// latent side fall into different banks.
#include "common.hpp"
#include "kernels.hpp"

namespace dit {

namespace {

struct Tile {
  int r, f, h, w0, wn;   // request, token row (f, h), first token and token count
};

__device__ __forceinline__ Tile decode_tile(const LatentTable& tab, int b) {
  int lo = 0, hi = tab.n_req - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (tab.tile_off[mid] <= b) lo = mid; else hi = mid - 1;
  }
  Tile t;
  t.r = lo;
  const int gh = tab.grid_h[lo], gw = tab.grid_w[lo];
  const int nwc = (gw + tab.wt - 1) / tab.wt;
  const int lt = b - tab.tile_off[lo];
  const int wc = lt % nwc, fh = lt / nwc;
  t.h = fh % gh;
  t.f = fh / gh;
  t.w0 = wc * tab.wt;
  t.wn = min(tab.wt, gw - t.w0);
  return t;
}

// Offset (within the request's latent) of value xx of the run of (c, i, j) =
// seg in tile t: ((c*Fl + f*pt + i)*Hl + h*ph + j)*Wl + w0*pw + xx.
__device__ __forceinline__ int64_t run_offset(const LatentTable& tab, const Tile& t, int seg, int64_t Fl,
                                              int64_t Hl, int64_t Wl) {
  const int j = seg % tab.ph, ci = seg / tab.ph;
  const int i = ci % tab.pt, c = ci / tab.pt;
  return (((int64_t)c * Fl + (int64_t)t.f * tab.pt + i) * Hl + (int64_t)t.h * tab.ph + j) * Wl +
         (int64_t)t.w0 * tab.pw;
}

template <typename T> struct Pair;
template <> struct Pair<bf16> { typedef bf16x2 type; };
template <> struct Pair<float> { typedef f32x2 type; };

template <typename T>
__global__ __launch_bounds__(256) void patchify_kernel(const float* __restrict__ latent, T* __restrict__ tokens,
                                                      LatentTable tab) {
  extern __shared__ float lds[];
  const Tile t = decode_tile(tab, blockIdx.x);
  const int pw = tab.pw, P = tab.C * tab.pt * tab.ph * pw, LP = P + 1;
  const int gw = tab.grid_w[t.r], gh = tab.grid_h[t.r];
  const int64_t Wl = (int64_t)gw * pw, Hl = (int64_t)gh * tab.ph;
  const int64_t Fl = (tab.lat_off[t.r + 1] - tab.lat_off[t.r]) / ((int64_t)tab.C * Hl * Wl);
  const float* src = latent + tab.lat_off[t.r];
  const int run = t.wn * pw, n = tab.C * tab.pt * tab.ph * run;
  for (int e = threadIdx.x; e < n; e += 256) {
    const int seg = e / run, xx = e - seg * run;
    const int w = xx / pw, k = xx - w * pw;
    lds[w * LP + seg * pw + k] = src[run_offset(tab, t, seg, Fl, Hl, Wl) + xx];
  }
  __syncthreads();
  typedef typename Pair<T>::type V;
  T* dst = tokens + ((int64_t)tab.row0[t.r] + ((int64_t)t.f * gh + t.h) * gw + t.w0) * P;
  for (int e = 2 * threadIdx.x; e < t.wn * P; e += 512) {   // P is even: a pair never straddles two tokens
    const int w = e / P, col = e - w * P;
    V v;
    v[0] = from_f<T>(lds[w * LP + col]);
    v[1] = from_f<T>(lds[w * LP + col + 1]);
    *reinterpret_cast<V*>(dst + e) = v;
  }
}

// latent and out may be the same buffer: each value is read, then written, by one thread.
template <typename T>
__global__ __launch_bounds__(256) void unpatchify_euler_kernel(const float* latent, const T* __restrict__ v,
                                                              const float* __restrict__ dt, float* out,
                                                              LatentTable tab) {
  extern __shared__ float lds[];
  const Tile t = decode_tile(tab, blockIdx.x);
  const int pw = tab.pw, P = tab.C * tab.pt * tab.ph * pw, LP = P + 1;
  const int gw = tab.grid_w[t.r], gh = tab.grid_h[t.r];
  typedef typename Pair<T>::type V;
  const T* vs = v + ((int64_t)tab.row0[t.r] + ((int64_t)t.f * gh + t.h) * gw + t.w0) * P;
  for (int e = 2 * threadIdx.x; e < t.wn * P; e += 512) {
    const int w = e / P, col = e - w * P;
    const V x = *reinterpret_cast<const V*>(vs + e);
    lds[w * LP + col] = to_f<T>(x[0]);
    lds[w * LP + col + 1] = to_f<T>(x[1]);
  }
  __syncthreads();
  const int64_t Wl = (int64_t)gw * pw, Hl = (int64_t)gh * tab.ph;
  const int64_t Fl = (tab.lat_off[t.r + 1] - tab.lat_off[t.r]) / ((int64_t)tab.C * Hl * Wl);
  const float d = dt[t.r];
  const float* src = latent + tab.lat_off[t.r];
  float* dst = out + tab.lat_off[t.r];
  const int run = t.wn * pw, n = tab.C * tab.pt * tab.ph * run;
  for (int e = threadIdx.x; e < n; e += 256) {
    const int seg = e / run, xx = e - seg * run;
    const int w = xx / pw, k = xx - w * pw;
    const int64_t o = run_offset(tab, t, seg, Fl, Hl, Wl) + xx;
    dst[o] = fmaf(d, lds[w * LP + seg * pw + k], src[o]);
  }
}

}  // namespace

size_t latent_tile_lds_bytes(const LatentTable& tab) {
  return (size_t)tab.wt * (tab.C * tab.pt * tab.ph * tab.pw + 1) * sizeof(float);
}

hipError_t launch_patchify(const LatentArgs& p, hipStream_t s) {
  const int tiles = p.tab.tile_off[p.tab.n_req];
  if (tiles == 0) return hipSuccess;
  const size_t lds = latent_tile_lds_bytes(p.tab);
  if (p.dtype == DIT_BF16)
    patchify_kernel<bf16><<<tiles, 256, lds, s>>>(p.latent, (bf16*)p.tokens, p.tab);
  else
    patchify_kernel<float><<<tiles, 256, lds, s>>>(p.latent, (float*)p.tokens, p.tab);
  return hipGetLastError();
}

hipError_t launch_unpatchify_euler(const LatentArgs& p, hipStream_t s) {
  const int tiles = p.tab.tile_off[p.tab.n_req];
  if (tiles == 0) return hipSuccess;
  const size_t lds = latent_tile_lds_bytes(p.tab);
  if (p.dtype == DIT_BF16)
    unpatchify_euler_kernel<bf16><<<tiles, 256, lds, s>>>(p.latent, (const bf16*)p.tokens, p.dt, p.latent_out,
                                                          p.tab);
  else
    unpatchify_euler_kernel<float><<<tiles, 256, lds, s>>>(p.latent, (const float*)p.tokens, p.dt, p.latent_out,
                                                           p.tab);
  return hipGetLastError();
}

}  // namespace dit
