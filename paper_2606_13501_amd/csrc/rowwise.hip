// Memory-bound kernels of the DiT block: LayerNorm with adaLN modulation or a
// shared affine, per-head RMSNorm with sectioned rotary embedding on q and k,
// the standalone gated residual, and the timestep-conditioning chain
// (sinusoid -> Linear-SiLU -> Linear-SiLU -> Linear to the modulation vectors).
//
// Every kernel moves 16-byte vectors per lane with consecutive lanes on
// consecutive addresses; a row is held in registers between its statistics
// pass and its output pass so it is read from HBM exactly once.  The rows are
// streamed with non-temporal loads and stores (each byte is touched once, so
// keeping it in the caches only displaces other data): measured +4-7% on the
// LayerNorm and gated-residual kernels at 75,600 x 5,120.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace dit {

namespace {

template <typename T> struct Vec16;
template <> struct Vec16<bf16> { typedef bf16x8 type; static constexpr int n = 8; };
template <> struct Vec16<float> { typedef f32x4 type; static constexpr int n = 4; };

// ------------------------------------------------------------ LayerNorm
// out = (x - mean) / sqrt(var + eps) * mul + add, one wave per row.
//   modulate: mul = 1 + scale[req], add = shift[req] (fp32 vectors)
//   affine:   mul = gamma, add = beta (dtype vectors)
// NVL = 16-byte vectors per lane, a compile-time count so the row is held in
// exactly as many registers as it needs (occupancy hides the HBM latency).

// Mean and 1 / sqrt(var + eps) of the wave's row v (NVL vectors per lane).
// The squares are accumulated with explicit fused multiply-adds, so every
// kernel that calls this rounds the statistics the same way.
template <typename T, int NVL, typename V>
__device__ __forceinline__ void row_stats(const V (&v)[NVL], int lane, int nv, int hidden, float eps, float& mean,
                                          float& rstd) {
  constexpr int VN = Vec16<T>::n;
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < NVL; ++i)
#pragma unroll
    for (int e = 0; e < VN; ++e) sum += to_f<T>(v[i][e]);
  mean = wave_sum(sum) / hidden;
  float sq = 0.f;
#pragma unroll
  for (int i = 0; i < NVL; ++i) {
    if (lane + 64 * i < nv) {
#pragma unroll
      for (int e = 0; e < VN; ++e) {
        const float d = to_f<T>(v[i][e]) - mean;
        sq = fmaf(d, d, sq);
      }
    }
  }
  rstd = rsqrtf(wave_sum(sq) / hidden + eps);
}

template <typename T, int NVL>
__global__ __launch_bounds__(256) void layer_norm_affine_kernel(
    const T* __restrict__ x, T* __restrict__ out, int64_t n_rows, int hidden, float eps,
    const T* __restrict__ gamma, const T* __restrict__ beta) {
  typedef typename Vec16<T>::type V;
  constexpr int VN = Vec16<T>::n;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  const int nv = hidden / VN;
  const T* xr = x + row * hidden;
  V v[NVL];
#pragma unroll
  for (int i = 0; i < NVL; ++i) {
    const int c = lane + 64 * i;
    v[i] = c < nv ? __builtin_nontemporal_load(reinterpret_cast<const V*>(xr + c * VN)) : V{};
  }
  float mean, rstd;
  row_stats<T, NVL>(v, lane, nv, hidden, eps, mean, rstd);
  T* orow = out + row * hidden;
#pragma unroll
  for (int i = 0; i < NVL; ++i) {
    const int c = lane + 64 * i;
    if (c < nv) {
      const V g = *reinterpret_cast<const V*>(gamma + c * VN);
      const V b = *reinterpret_cast<const V*>(beta + c * VN);
      V o;
#pragma unroll
      for (int e = 0; e < VN; ++e)
        o[e] = from_f<T>(fmaf((to_f<T>(v[i][e]) - mean) * rstd, to_f<T>(g[e]), to_f<T>(b[e])));
      __builtin_nontemporal_store(o, reinterpret_cast<V*>(orow + c * VN));
    }
  }
}

// Modulated LayerNorm, WAVES rows per workgroup.  When all of them belong to
// one request (every workgroup but those across a request boundary), the
// request's 1 + scale and shift are first staged in LDS as fp32 (8 bytes per
// column), so they are read from L2 once per workgroup rather than once per
// row: at 75,600 x 5,120 the per-row reads were 40 KB of L2 traffic for
// every 10 KB row, and staging took the kernel from 70% to 75% of the HBM
// peak.  The other workgroups read the vectors of each row's request
// directly; both paths round identically.  The row is loaded after the
// staging: issued before it, the row loads held the staged reads back
// behind them and the kernel ran 20% slower.
template <typename T, int NVL, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void layer_norm_mod_kernel(
    const T* __restrict__ x, T* __restrict__ out, int64_t n_rows, int hidden, float eps,
    const float* __restrict__ shift, const float* __restrict__ scale, int64_t mod_stride, ReqTable req) {
  typedef typename Vec16<T>::type V;
  constexpr int VN = Vec16<T>::n;
  // hidden / 4 vectors of 1 + scale, then hidden / 4 of shift.  Source vector
  // j = G c + g (G = VN / 4 per 16-byte row vector c) is kept at g nv + c, so
  // the 64 lanes of a read, and of a staging write, touch 64 consecutive
  // vectors (no bank conflicts).
  constexpr int G = VN / 4;
  extern __shared__ f32x4 smod[];
  const int lane = threadIdx.x & 63;
  const int64_t r0 = (int64_t)blockIdx.x * WAVES;
  const int64_t row = r0 + (threadIdx.x >> 6);
  const int ra = find_req(req.cu, req.n_req, (int)r0);
  const bool staged = ra == find_req(req.cu, req.n_req, (int)(min(r0 + WAVES, n_rows) - 1));
  const int nv = hidden / VN, h4 = hidden / 4;
  if (staged) {   // uniform over the workgroup
    const f32x4* sc = reinterpret_cast<const f32x4*>(scale + (int64_t)ra * mod_stride);
    const f32x4* sh = reinterpret_cast<const f32x4*>(shift + (int64_t)ra * mod_stride);
    for (int at = threadIdx.x; at < h4; at += WAVES * 64) {   // consecutive LDS writes
      const int i = G * (at % nv) + at / nv;
      f32x4 m = sc[i];
#pragma unroll
      for (int u = 0; u < 4; ++u) m[u] = 1.0f + m[u];
      smod[at] = m;
      smod[h4 + at] = sh[i];
    }
    __syncthreads();
  }
  if (row >= n_rows) return;
  V v[NVL];
  {
    const T* xr = x + row * hidden;
#pragma unroll
    for (int i = 0; i < NVL; ++i) {
      const int c = lane + 64 * i;
      v[i] = c < nv ? __builtin_nontemporal_load(reinterpret_cast<const V*>(xr + c * VN)) : V{};
    }
  }
  float mean, rstd;
  row_stats<T, NVL>(v, lane, nv, hidden, eps, mean, rstd);
  const int r = staged ? ra : find_req(req.cu, req.n_req, (int)row);
  const f32x4* sc = reinterpret_cast<const f32x4*>(scale + (int64_t)r * mod_stride);
  const f32x4* sh = reinterpret_cast<const f32x4*>(shift + (int64_t)r * mod_stride);
  T* orow = out + row * hidden;
  auto emit = [&](auto&& mul_add) {
#pragma unroll
    for (int i = 0; i < NVL; ++i) {
      const int c = lane + 64 * i;
      if (c < nv) {
        V o;
#pragma unroll
        for (int e = 0; e < VN; e += 4) {
          f32x4 m4, a4;
          mul_add((c * VN + e) / 4, m4, a4);
#pragma unroll
          for (int u = 0; u < 4; ++u)
            o[e + u] = from_f<T>(fmaf((to_f<T>(v[i][e + u]) - mean) * rstd, m4[u], a4[u]));
        }
        __builtin_nontemporal_store(o, reinterpret_cast<V*>(orow + c * VN));
      }
    }
  };
  if (staged) {
    emit([&](int j, f32x4& m4, f32x4& a4) {
      const int at = (j % G) * nv + j / G;
      m4 = smod[at];
      a4 = smod[h4 + at];
    });
  } else {
    emit([&](int j, f32x4& m4, f32x4& a4) {
      m4 = sc[j];
      a4 = sh[j];
#pragma unroll
      for (int u = 0; u < 4; ++u) m4[u] = 1.0f + m4[u];
    });
  }
}

// ---------------------------------------------------- QK RMSNorm + rotary
// One wave per row, four rows per 256-thread block.  A head of head_dim
// values is LPH = head_dim / VN consecutive lanes (LPH divides 64), so every
// vector a lane touches sits at the same offset inside its head: the lane
// needs the same VN/2 rotary pairs and the same gain vector for all of them.
// Lane j computes the cos/sin of pair j (in double) and the lanes gather
// theirs by shuffles; a head's RMS statistic is a shuffle reduction over its
// LPH lanes.  q and k vectors of a pass (NV per lane each) are all loaded
// before any is computed on.
template <typename T, int NV>
__global__ __launch_bounds__(256) void qk_norm_rope_kernel(
    T* q, T* k, int64_t row_stride, int64_t n_rows, int n_heads, int head_dim, const T* __restrict__ g_q,
    const T* __restrict__ g_k, float eps, int rope, int sec0, int sec1, int sec2, float theta,
    RopeTable tab) {
  typedef typename Vec16<T>::type V;
  constexpr int VN = Vec16<T>::n;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  const int lph = head_dim / VN;
  const int hc = lane % lph;          // chunk index inside the head
  const int cpt = n_heads * lph;      // vectors per tensor
  T* base_ptr[2] = {q + row * row_stride, k ? k + row * row_stride : nullptr};
  const T* gain[2] = {g_q, g_k};
  float cr[VN / 2], sr[VN / 2];
  if (rope) {
    float cj = 1.f, sj = 0.f;
    const int j = lane;
    if (j < head_dim / 2) {
      const int r = find_req(tab.cu, tab.n_req, (int)row);
      const int g = tab.offset[r] + (int)row - tab.cu[r];
      const int pt = g / tab.grid_hw[r];
      const int ph = (g / tab.grid_w[r]) % tab.grid_h[r];
      const int pw = g % tab.grid_w[r];
      // pair j -> (section, index inside the section)
      int p, js, ds;
      if (j < sec0 / 2) { p = pt; js = j; ds = sec0; }
      else if (j < (sec0 + sec1) / 2) { p = ph; js = j - sec0 / 2; ds = sec1; }
      else { p = pw; js = j - (sec0 + sec1) / 2; ds = sec2; }
      const double ang = (double)p * exp(-2.0 * js / ds * log((double)theta));
      double sn, cn;
      sincos(ang, &sn, &cn);
      cj = (float)cn;
      sj = (float)sn;
    }
#pragma unroll
    for (int u = 0; u < VN / 2; ++u) {
      cr[u] = __shfl(cj, hc * (VN / 2) + u, 64);
      sr[u] = __shfl(sj, hc * (VN / 2) + u, 64);
    }
  }
  const int n_t = k ? 2 : 1;
  for (int b0 = 0; b0 < cpt; b0 += 64 * NV) {
    V v[2][NV];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int c = b0 + lane + 64 * i;
        v[t][i] = t < n_t && c < cpt ? __builtin_nontemporal_load(reinterpret_cast<const V*>(base_ptr[t] + (int64_t)c * VN)) : V{};
      }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      if (t >= n_t) break;
      V g{};
      if (gain[t]) g = *reinterpret_cast<const V*>(gain[t] + hc * VN);
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        if (b0 + 64 * i >= cpt) break;   // wave-uniform
        const int c = b0 + lane + 64 * i;
        float f[VN];
#pragma unroll
        for (int e = 0; e < VN; ++e) f[e] = to_f<T>(v[t][i][e]);
        if (gain[t]) {
          float sq = 0.f;
#pragma unroll
          for (int e = 0; e < VN; ++e) sq += f[e] * f[e];
          for (int o = lph / 2; o > 0; o >>= 1) sq += __shfl_xor(sq, o, 64);
          const float rs = rsqrtf(sq / head_dim + eps);
#pragma unroll
          for (int e = 0; e < VN; ++e) f[e] = f[e] * rs * to_f<T>(g[e]);
        }
        if (rope) {
#pragma unroll
          for (int u = 0; u < VN / 2; ++u) {
            const float a = f[2 * u], bb = f[2 * u + 1];
            f[2 * u] = a * cr[u] - bb * sr[u];
            f[2 * u + 1] = a * sr[u] + bb * cr[u];
          }
        }
        if (c < cpt) {
          V o;
#pragma unroll
          for (int e = 0; e < VN; ++e) o[e] = from_f<T>(f[e]);
          __builtin_nontemporal_store(o, reinterpret_cast<V*>(base_ptr[t] + (int64_t)c * VN));
        }
      }
    }
  }
}

// ------------------------------------------------------- gated residual
// out = x + gate[req] * (z + bias), one wave per row; the row's x and z
// vectors (NVL per lane) are all loaded before any is combined.
template <typename T, int NVL>
__global__ __launch_bounds__(256) void gated_residual_kernel(
    const T* x, const T* z, const T* __restrict__ bias, const float* __restrict__ gate,
    int64_t gate_stride, T* out, int64_t n_rows, int hidden, ReqTable req) {
  typedef typename Vec16<T>::type V;
  constexpr int VN = Vec16<T>::n;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  const int r = find_req(req.cu, req.n_req, (int)row);
  const float* g = gate + (int64_t)r * gate_stride;
  const int nv = hidden / VN;
  V xv[NVL], zv[NVL];
#pragma unroll
  for (int i = 0; i < NVL; ++i) {
    const int c = lane + 64 * i;
    xv[i] = c < nv ? __builtin_nontemporal_load(reinterpret_cast<const V*>(x + row * hidden + c * VN)) : V{};
    zv[i] = c < nv ? __builtin_nontemporal_load(reinterpret_cast<const V*>(z + row * hidden + c * VN)) : V{};
  }
#pragma unroll
  for (int i = 0; i < NVL; ++i) {
    const int c = lane + 64 * i;
    if (c < nv) {
      V bv{};
      if (bias) bv = *reinterpret_cast<const V*>(bias + c * VN);
      V o;
#pragma unroll
      for (int e = 0; e < VN; e += 4) {
        f32x4 g4 = *reinterpret_cast<const f32x4*>(g + c * VN + e);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          o[e + u] = from_f<T>(to_f<T>(xv[i][e + u]) + g4[u] * (to_f<T>(zv[i][e + u]) + to_f<T>(bv[e + u])));
      }
      __builtin_nontemporal_store(o, reinterpret_cast<V*>(out + row * hidden + c * VN));
    }
  }
}

// ------------------------------------------------------- conditioning
// e[r] = [cos(t w_i), sin(t w_i)], w_i = 10000^(-i/half); computed in double.
__global__ void timestep_embed_kernel(const float* __restrict__ t, float* __restrict__ e, int n_req,
                                      int freq_dim) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  const int half = freq_dim / 2;
  if (idx >= n_req * half) return;
  const int r = idx / half, i = idx - r * half;
  const double w = exp(-log(10000.0) * (double)i / (double)half);
  double sn, cn;
  sincos((double)t[r] * w, &sn, &cn);
  e[(int64_t)r * freq_dim + i] = (float)cn;
  e[(int64_t)r * freq_dim + half + i] = (float)sn;
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

// y[r][o] = act(sum_i W[o][i] x[r][i] + b[o]) for up to 8 requests per pass;
// one wave per output row, W read once per pass with 16-byte vectors.
template <typename T, bool SILU_OUT>
__global__ __launch_bounds__(256) void gemv_kernel(const T* __restrict__ W, const T* __restrict__ b,
                                                   const float* __restrict__ x, float* __restrict__ y,
                                                   int n_out, int n_in, int n_req) {
  typedef typename Vec16<T>::type V;
  constexpr int VN = Vec16<T>::n;
  const int lane = threadIdx.x & 63;
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (o >= n_out) return;
  const T* wr = W + (int64_t)o * n_in;
  const int nv = n_in / VN;
  for (int r0 = 0; r0 < n_req; r0 += 8) {
    const int nr = min(8, n_req - r0);
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int c = lane; c < nv; c += 64) {
      V wv = *reinterpret_cast<const V*>(wr + c * VN);
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) {
        if (rr < nr) {
          const float* xr = x + (int64_t)(r0 + rr) * n_in + c * VN;
#pragma unroll
          for (int e = 0; e < VN; ++e) acc[rr] = fmaf(to_f<T>(wv[e]), xr[e], acc[rr]);
        }
      }
    }
#pragma unroll
    for (int rr = 0; rr < 8; ++rr) {
      if (rr < nr) {
        float s = wave_sum(acc[rr]);
        if (lane == 0) {
          s += b ? to_f<T>(b[o]) : 0.f;
          y[(int64_t)(r0 + rr) * n_out + o] = SILU_OUT ? silu(s) : s;
        }
      }
    }
  }
}

// The same product for rows of at most 64 NVL vectors: a lane loads all of
// its NVL weight vectors of the row first, so they are in flight together
// (the weights stream from memory once, and a wave with one load in flight
// at a time is latency-bound), then accumulates each request over them in
// the order of gemv_kernel (the results are the same bits).
template <typename T, bool SILU_OUT, int NVL>
__global__ __launch_bounds__(256) void gemv_row_kernel(const T* __restrict__ W, const T* __restrict__ b,
                                                       const float* __restrict__ x, float* __restrict__ y,
                                                       int n_out, int n_in, int n_req) {
  typedef typename Vec16<T>::type V;
  constexpr int VN = Vec16<T>::n;
  typedef float fxv __attribute__((ext_vector_type(VN)));
  const int lane = threadIdx.x & 63;
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (o >= n_out) return;
  const T* wr = W + (int64_t)o * n_in;
  const int nv = n_in / VN;
  const float bo = b ? to_f<T>(b[o]) : 0.f;
  // FULL: every lane has all NVL vectors (no per-lane tests, so the loads
  // are not split by branches)
  auto run = [&](auto full) __attribute__((always_inline)) {
    V wv[NVL];
#pragma unroll
    for (int u = 0; u < NVL; ++u) {
      const int c = lane + 64 * u;
      if (decltype(full)::value || c < nv) wv[u] = *reinterpret_cast<const V*>(wr + c * VN);
    }
    for (int r = 0; r < n_req; ++r) {
      const float* xr = x + (int64_t)r * n_in;
      fxv xv[NVL];   // the request's inputs under the lane's vectors, loaded together
#pragma unroll
      for (int u = 0; u < NVL; ++u) {
        const int c = lane + 64 * u;
        if (decltype(full)::value || c < nv) xv[u] = *reinterpret_cast<const fxv*>(xr + c * VN);
      }
      float acc = 0.f;
#pragma unroll
      for (int u = 0; u < NVL; ++u) {
        const int c = lane + 64 * u;
        if (decltype(full)::value || c < nv) {
#pragma unroll
          for (int e = 0; e < VN; ++e) acc = fmaf(to_f<T>(wv[u][e]), xv[u][e], acc);
        }
      }
      float sum = wave_sum(acc);
      if (lane == 0) {
        sum += bo;
        y[(int64_t)r * n_out + o] = SILU_OUT ? silu(sum) : sum;
      }
    }
  };
  if (nv == 64 * NVL) run(std::true_type{});
  else run(std::false_type{});
}

template <typename T, bool SILU_OUT>
void launch_gemv(const T* W, const T* b, const float* x, float* y, int n_out, int n_in, int n_req, hipStream_t s) {
  const unsigned grid = (unsigned)((n_out + 3) / 4);
  switch ((n_in / Vec16<T>::n + 63) / 64) {
#define DIT_GEMV_ROW(NVL) \
  case NVL: gemv_row_kernel<T, SILU_OUT, NVL><<<grid, 256, 0, s>>>(W, b, x, y, n_out, n_in, n_req); return;
    DIT_GEMV_ROW(1) DIT_GEMV_ROW(2) DIT_GEMV_ROW(3) DIT_GEMV_ROW(4) DIT_GEMV_ROW(5) DIT_GEMV_ROW(6)
    DIT_GEMV_ROW(7) DIT_GEMV_ROW(8) DIT_GEMV_ROW(9) DIT_GEMV_ROW(10) DIT_GEMV_ROW(11) DIT_GEMV_ROW(12)
    DIT_GEMV_ROW(13) DIT_GEMV_ROW(14) DIT_GEMV_ROW(15) DIT_GEMV_ROW(16)
#undef DIT_GEMV_ROW
    default: gemv_kernel<T, SILU_OUT><<<grid, 256, 0, s>>>(W, b, x, y, n_out, n_in, n_req);
  }
}

template <typename T, int NVL>
hipError_t gres_nvl(const GatedResArgs& p, hipStream_t s) {
  gated_residual_kernel<T, NVL><<<(unsigned)((p.n_rows + 3) / 4), 256, 0, s>>>(
      (const T*)p.x, (const T*)p.z, (const T*)p.bias, p.gate, p.gate_stride, (T*)p.out, p.n_rows, p.hidden,
      p.req);
  return hipGetLastError();
}

// Rows of up to 1024 16-byte vectors (8192 bf16, 4096 fp32 values).
template <typename T>
hipError_t gres_typed(const GatedResArgs& p, hipStream_t s) {
  switch ((p.hidden / Vec16<T>::n + 63) / 64) {
    case 1: return gres_nvl<T, 1>(p, s);
    case 2: return gres_nvl<T, 2>(p, s);
    case 3: case 4: return gres_nvl<T, 4>(p, s);
    case 5: case 6: return gres_nvl<T, 6>(p, s);
    case 7: case 8: return gres_nvl<T, 8>(p, s);
    case 9: case 10: return gres_nvl<T, 10>(p, s);
    case 11: case 12: return gres_nvl<T, 12>(p, s);
    case 13: case 14: case 15: case 16: return gres_nvl<T, 16>(p, s);
    default: return hipErrorInvalidValue;
  }
}

constexpr int kLnModWaves = 4;   // rows of the modulated LayerNorm per workgroup

template <typename T, int NVL>
hipError_t ln_nvl(const LnArgs& p, hipStream_t s) {
  if (p.affine) {
    layer_norm_affine_kernel<T, NVL><<<(unsigned)((p.n_rows + 3) / 4), 256, 0, s>>>(
        (const T*)p.x, (T*)p.out, p.n_rows, p.hidden, p.eps, (const T*)p.gamma, (const T*)p.beta);
  } else {
    layer_norm_mod_kernel<T, NVL, kLnModWaves>
        <<<(unsigned)((p.n_rows + kLnModWaves - 1) / kLnModWaves), kLnModWaves * 64, (size_t)p.hidden * 8, s>>>(
            (const T*)p.x, (T*)p.out, p.n_rows, p.hidden, p.eps, p.shift, p.scale, p.mod_stride, p.req);
  }
  return hipGetLastError();
}

// Rows of up to 1024 16-byte vectors (8192 bf16, 4096 fp32 values).
template <typename T>
hipError_t ln_typed(const LnArgs& p, hipStream_t s) {
  const int nvl = (p.hidden / Vec16<T>::n + 63) / 64;
  switch (nvl) {
    case 1: return ln_nvl<T, 1>(p, s);
    case 2: return ln_nvl<T, 2>(p, s);
    case 3: return ln_nvl<T, 3>(p, s);
    case 4: return ln_nvl<T, 4>(p, s);
    case 5: return ln_nvl<T, 5>(p, s);
    case 6: return ln_nvl<T, 6>(p, s);
    case 7: return ln_nvl<T, 7>(p, s);
    case 8: return ln_nvl<T, 8>(p, s);
    case 9: case 10: return ln_nvl<T, 10>(p, s);
    case 11: case 12: return ln_nvl<T, 12>(p, s);
    case 13: case 14: return ln_nvl<T, 14>(p, s);
    case 15: case 16: return ln_nvl<T, 16>(p, s);
    default: return hipErrorInvalidValue;
  }
}

template <typename T>
hipError_t cond_typed(const CondArgs& p, hipStream_t s) {
  if (p.w_t1) {
    const int half = p.freq_dim / 2;
    timestep_embed_kernel<<<(p.n_req * half + 255) / 256, 256, 0, s>>>(p.t, p.e, p.n_req, p.freq_dim);
    launch_gemv<T, true>((const T*)p.w_t1, (const T*)p.b_t1, p.e, p.a1, p.hidden, p.freq_dim, p.n_req, s);
    launch_gemv<T, true>((const T*)p.w_t2, (const T*)p.b_t2, p.a1, p.c, p.hidden, p.hidden, p.n_req, s);
  }
  if (p.w_ada) {
    const int n_out = p.n_mod * p.hidden;
    launch_gemv<T, false>((const T*)p.w_ada, (const T*)p.b_ada, p.c, p.mod, n_out, p.hidden, p.n_req, s);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_layer_norm(const LnArgs& p, hipStream_t s) {
  if (p.n_rows == 0) return hipSuccess;
  return p.dtype == DIT_BF16 ? ln_typed<bf16>(p, s) : ln_typed<float>(p, s);
}

namespace {

template <typename T, int NV>
void qk_nv(const NormRopeArgs& p, hipStream_t s) {
  qk_norm_rope_kernel<T, NV><<<(unsigned)((p.n_rows + 3) / 4), 256, 0, s>>>(
      (T*)p.q, (T*)p.k, p.row_stride, p.n_rows, p.n_heads, p.head_dim, (const T*)p.g_q, (const T*)p.g_k,
      p.eps, p.rope, p.sections[0], p.sections[1], p.sections[2], p.theta, p.tab);
}

template <typename T>
hipError_t qk_typed(const NormRopeArgs& p, hipStream_t s) {
  const int64_t nv = ((int64_t)p.n_heads * p.head_dim / Vec16<T>::n + 63) / 64;
  if (nv <= 1) qk_nv<T, 1>(p, s);
  else if (nv <= 2) qk_nv<T, 2>(p, s);
  else if (nv <= 3) qk_nv<T, 3>(p, s);
  else if (nv <= 4) qk_nv<T, 4>(p, s);
  else if (nv <= 6) qk_nv<T, 6>(p, s);
  else if (nv <= 8) qk_nv<T, 8>(p, s);
  else qk_nv<T, 10>(p, s);   // passes of 10 vectors per lane and tensor
  return hipGetLastError();
}

}  // namespace

hipError_t launch_qk_norm_rope(const NormRopeArgs& p, hipStream_t s) {
  if (p.n_rows == 0) return hipSuccess;
  return p.dtype == DIT_BF16 ? qk_typed<bf16>(p, s) : qk_typed<float>(p, s);
}

hipError_t launch_gated_residual(const GatedResArgs& p, hipStream_t s) {
  if (p.n_rows == 0) return hipSuccess;
  return p.dtype == DIT_BF16 ? gres_typed<bf16>(p, s) : gres_typed<float>(p, s);
}

hipError_t launch_conditioning(const CondArgs& p, hipStream_t s) {
  if (p.n_req == 0) return hipSuccess;
  return p.dtype == DIT_BF16 ? cond_typed<bf16>(p, s) : cond_typed<float>(p, s);
}

}  // namespace dit
