// Memory-bound kernels of the DiT block: LayerNorm with adaLN modulation or a
// shared affine, per-head RMSNorm with sectioned rotary embedding on q and k,
// the standalone gated residual, and the timestep-conditioning chain
// (sinusoid -> Linear-SiLU -> Linear-SiLU -> Linear to six modulation vectors).
//
// Every kernel moves 16-byte vectors per lane with consecutive lanes on
// consecutive addresses; a row is held in registers between its statistics
// pass and its output pass so it is read from HBM exactly once.
#include <math.h>

#include "common.hpp"
#include "kernels.hpp"

namespace dit {

namespace {

template <typename T> struct Vec16;
template <> struct Vec16<bf16> { typedef bf16x8 type; static constexpr int n = 8; };
template <> struct Vec16<float> { typedef f32x4 type; static constexpr int n = 4; };

constexpr int kLnMaxVec = 16;   // 16-byte vectors per lane: D <= 8192 (bf16), 4096 (fp32)

// ------------------------------------------------------------ LayerNorm
// out = (x - mean) / sqrt(var + eps) * mul + add, one wave per row.
//   modulate: mul = 1 + scale[req], add = shift[req] (fp32 vectors)
//   affine:   mul = gamma, add = beta (dtype vectors)
template <typename T, bool AFFINE>
__global__ __launch_bounds__(256) void layer_norm_kernel(
    const T* __restrict__ x, T* __restrict__ out, int64_t n_rows, int hidden, float eps,
    const float* __restrict__ shift, const float* __restrict__ scale, int64_t mod_stride,
    const T* __restrict__ gamma, const T* __restrict__ beta, ReqTable req) {
  typedef typename Vec16<T>::type V;
  constexpr int VN = Vec16<T>::n;
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_rows) return;
  const int nv = hidden / VN;
  const T* xr = x + row * hidden;
  V v[kLnMaxVec];
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < kLnMaxVec; ++i) {
    const int c = lane + 64 * i;
    if (c < nv) {
      v[i] = *reinterpret_cast<const V*>(xr + c * VN);
#pragma unroll
      for (int e = 0; e < VN; ++e) sum += to_f<T>(v[i][e]);
    }
  }
  const float mean = wave_sum(sum) / hidden;
  float sq = 0.f;
#pragma unroll
  for (int i = 0; i < kLnMaxVec; ++i) {
    const int c = lane + 64 * i;
    if (c < nv) {
#pragma unroll
      for (int e = 0; e < VN; ++e) {
        float d = to_f<T>(v[i][e]) - mean;
        sq += d * d;
      }
    }
  }
  const float rstd = rsqrtf(wave_sum(sq) / hidden + eps);
  const float* sh = nullptr;
  const float* sc = nullptr;
  if (!AFFINE) {
    const int r = find_req(req.cu, req.n_req, (int)row);
    sh = shift + (int64_t)r * mod_stride;
    sc = scale + (int64_t)r * mod_stride;
  }
  T* orow = out + row * hidden;
#pragma unroll
  for (int i = 0; i < kLnMaxVec; ++i) {
    const int c = lane + 64 * i;
    if (c < nv) {
      V o;
      if (AFFINE) {
        V g = *reinterpret_cast<const V*>(gamma + c * VN);
        V b = *reinterpret_cast<const V*>(beta + c * VN);
#pragma unroll
        for (int e = 0; e < VN; ++e)
          o[e] = from_f<T>((to_f<T>(v[i][e]) - mean) * rstd * to_f<T>(g[e]) + to_f<T>(b[e]));
      } else {
#pragma unroll
        for (int e = 0; e < VN; e += 4) {
          f32x4 s4 = *reinterpret_cast<const f32x4*>(sc + c * VN + e);
          f32x4 h4 = *reinterpret_cast<const f32x4*>(sh + c * VN + e);
#pragma unroll
          for (int u = 0; u < 4; ++u)
            o[e + u] = from_f<T>((to_f<T>(v[i][e + u]) - mean) * rstd * (1.0f + s4[u]) + h4[u]);
        }
      }
      *reinterpret_cast<V*>(orow + c * VN) = o;
    }
  }
}

// ---------------------------------------------------- QK RMSNorm + rotary
// One 256-thread block per row.  The rotary cos/sin of the row's head_dim/2
// pairs are computed once (in double) into LDS and shared by every head of q
// and k.  A group of head_dim/VN lanes holds one head; its RMS statistic is a
// shuffle reduction inside the group.
template <typename T>
__global__ __launch_bounds__(256) void qk_norm_rope_kernel(
    T* q, T* k, int64_t row_stride, int n_heads, int head_dim, const T* __restrict__ g_q,
    const T* __restrict__ g_k, float eps, int rope, int sec0, int sec1, int sec2, float theta,
    RopeTable tab) {
  typedef typename Vec16<T>::type V;
  constexpr int VN = Vec16<T>::n;
  __shared__ float cs[128][2];
  const int64_t row = blockIdx.x;
  const int half = head_dim / 2;
  if (rope) {
    if ((int)threadIdx.x < half) {
      const int j = threadIdx.x;
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
      cs[j][0] = (float)cn;
      cs[j][1] = (float)sn;
    }
    __syncthreads();
  }
  const int lanes_per_head = head_dim / VN;
  const int chunks_per_tensor = n_heads * lanes_per_head;
  const int n_tensors = k ? 2 : 1;
  const int total = n_tensors * chunks_per_tensor;
  // all threads of a wave run the same number of iterations (shuffles below)
  for (int base = 0; base < total; base += blockDim.x) {
    const int c = base + threadIdx.x;
    const bool active = c < total;
    const int tensor = active ? c / chunks_per_tensor : 0;
    const int cc = active ? c - tensor * chunks_per_tensor : 0;
    T* ptr = (tensor ? k : q) + row * row_stride + (int64_t)cc * VN;
    const T* gain = tensor ? g_k : g_q;
    const int dpos = (cc % lanes_per_head) * VN;   // offset inside the head
    V v{};
    if (active) v = *reinterpret_cast<const V*>(ptr);
    float f[VN];
#pragma unroll
    for (int e = 0; e < VN; ++e) f[e] = to_f<T>(v[e]);
    if (gain) {
      float sq = 0.f;
#pragma unroll
      for (int e = 0; e < VN; ++e) sq += f[e] * f[e];
      for (int o = lanes_per_head / 2; o > 0; o >>= 1) sq += __shfl_xor(sq, o, 64);
      const float rs = rsqrtf(sq / head_dim + eps);
      V g = active ? *reinterpret_cast<const V*>(gain + dpos) : V{};
#pragma unroll
      for (int e = 0; e < VN; ++e) f[e] = f[e] * rs * to_f<T>(g[e]);
    }
    if (rope) {
#pragma unroll
      for (int e = 0; e < VN; e += 2) {
        const int j = (dpos + e) >> 1;
        const float cn = cs[j][0], sn = cs[j][1];
        const float a = f[e], b = f[e + 1];
        f[e] = a * cn - b * sn;
        f[e + 1] = a * sn + b * cn;
      }
    }
    if (active) {
      V o;
#pragma unroll
      for (int e = 0; e < VN; ++e) o[e] = from_f<T>(f[e]);
      *reinterpret_cast<V*>(ptr) = o;
    }
  }
}

// ------------------------------------------------------- gated residual
// out = x + gate[req] * (z + bias), one wave per row.
template <typename T>
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
  for (int c = lane; c < nv; c += 64) {
    V xv = *reinterpret_cast<const V*>(x + row * hidden + c * VN);
    V zv = *reinterpret_cast<const V*>(z + row * hidden + c * VN);
    V bv{};
    if (bias) bv = *reinterpret_cast<const V*>(bias + c * VN);
    V o;
#pragma unroll
    for (int e = 0; e < VN; e += 4) {
      f32x4 g4 = *reinterpret_cast<const f32x4*>(g + c * VN + e);
#pragma unroll
      for (int u = 0; u < 4; ++u)
        o[e + u] = from_f<T>(to_f<T>(xv[e + u]) + g4[u] * (to_f<T>(zv[e + u]) + to_f<T>(bv[e + u])));
    }
    *reinterpret_cast<V*>(out + row * hidden + c * VN) = o;
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

template <typename T>
hipError_t ln_typed(const LnArgs& p, hipStream_t s) {
  const unsigned grid = (unsigned)((p.n_rows + 3) / 4);
  if (p.affine)
    layer_norm_kernel<T, true><<<grid, 256, 0, s>>>((const T*)p.x, (T*)p.out, p.n_rows, p.hidden, p.eps,
                                                    nullptr, nullptr, 0, (const T*)p.gamma,
                                                    (const T*)p.beta, p.req);
  else
    layer_norm_kernel<T, false><<<grid, 256, 0, s>>>((const T*)p.x, (T*)p.out, p.n_rows, p.hidden, p.eps,
                                                     p.shift, p.scale, p.mod_stride, nullptr, nullptr,
                                                     p.req);
  return hipGetLastError();
}

template <typename T>
hipError_t cond_typed(const CondArgs& p, hipStream_t s) {
  const int half = p.freq_dim / 2;
  timestep_embed_kernel<<<(p.n_req * half + 255) / 256, 256, 0, s>>>(p.t, p.e, p.n_req, p.freq_dim);
  gemv_kernel<T, true><<<(p.hidden + 3) / 4, 256, 0, s>>>((const T*)p.w_t1, (const T*)p.b_t1, p.e, p.a1,
                                                         p.hidden, p.freq_dim, p.n_req);
  gemv_kernel<T, true><<<(p.hidden + 3) / 4, 256, 0, s>>>((const T*)p.w_t2, (const T*)p.b_t2, p.a1, p.c,
                                                         p.hidden, p.hidden, p.n_req);
  gemv_kernel<T, false><<<(6 * p.hidden + 3) / 4, 256, 0, s>>>((const T*)p.w_ada, (const T*)p.b_ada, p.c,
                                                              p.mod, 6 * p.hidden, p.hidden, p.n_req);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_layer_norm(const LnArgs& p, hipStream_t s) {
  if (p.n_rows == 0) return hipSuccess;
  return p.dtype == DIT_BF16 ? ln_typed<bf16>(p, s) : ln_typed<float>(p, s);
}

hipError_t launch_qk_norm_rope(const NormRopeArgs& p, hipStream_t s) {
  if (p.n_rows == 0) return hipSuccess;
  const unsigned grid = (unsigned)p.n_rows;
  if (p.dtype == DIT_BF16)
    qk_norm_rope_kernel<bf16><<<grid, 256, 0, s>>>((bf16*)p.q, (bf16*)p.k, p.row_stride, p.n_heads,
                                                   p.head_dim, (const bf16*)p.g_q, (const bf16*)p.g_k,
                                                   p.eps, p.rope, p.sections[0], p.sections[1],
                                                   p.sections[2], p.theta, p.tab);
  else
    qk_norm_rope_kernel<float><<<grid, 256, 0, s>>>((float*)p.q, (float*)p.k, p.row_stride, p.n_heads,
                                                    p.head_dim, (const float*)p.g_q, (const float*)p.g_k,
                                                    p.eps, p.rope, p.sections[0], p.sections[1],
                                                    p.sections[2], p.theta, p.tab);
  return hipGetLastError();
}

hipError_t launch_gated_residual(const GatedResArgs& p, hipStream_t s) {
  if (p.n_rows == 0) return hipSuccess;
  const unsigned grid = (unsigned)((p.n_rows + 3) / 4);
  if (p.dtype == DIT_BF16)
    gated_residual_kernel<bf16><<<grid, 256, 0, s>>>((const bf16*)p.x, (const bf16*)p.z,
                                                     (const bf16*)p.bias, p.gate, p.gate_stride,
                                                     (bf16*)p.out, p.n_rows, p.hidden, p.req);
  else
    gated_residual_kernel<float><<<grid, 256, 0, s>>>((const float*)p.x, (const float*)p.z,
                                                      (const float*)p.bias, p.gate, p.gate_stride,
                                                      (float*)p.out, p.n_rows, p.hidden, p.req);
  return hipGetLastError();
}

hipError_t launch_conditioning(const CondArgs& p, hipStream_t s) {
  if (p.n_req == 0) return hipSuccess;
  return p.dtype == DIT_BF16 ? cond_typed<bf16>(p, s) : cond_typed<float>(p, s);
}

}  // namespace dit
