// Host-side launchers of the gfx950 kernels (arguments are validated by the
// C-ABI layer before any of these is called).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"
#include "dit_block.h"

namespace dit {

struct LinearArgs {
  const void* a; int64_t lda;
  const void* w; int64_t ldw;
  const void* bias;
  void* out; int64_t ldo;
  int64_t M; int N; int K;
  dit_epilogue epi;
  const void* res; int64_t ldr;
  const float* gate; int64_t gate_stride;
  ReqTable req;
  dit_dtype dtype;
  // plane_cols > 0: output column n goes to plane n / plane_cols, column
  // n % plane_cols, planes plane_stride elements apart (ldo = plane_cols);
  // plane_cols a multiple of 4
  int plane_cols = 0;
  int64_t plane_stride = 0;
};
hipError_t launch_linear(const LinearArgs& p, hipStream_t s);
// Compute units of the current device (cached per device).
int cu_count();
// Forces the bf16 GEMM's output tile width (192 or 256; 0: chosen per shape).
void set_gemm_tile_n(int bn);

struct AttnArgs {
  const void *q, *k, *v;
  void* o;
  int64_t q_stride, k_stride, v_stride, o_stride;  // elements
  ReqTable cq, ck;
  int n_heads, head_dim;
  float scale;
  dit_dtype dtype;
  // bf16 only: per-head RMSNorm of q with this gain [head_dim] as q is loaded
  // (NULL: q used as stored)
  const void* q_gain = nullptr;
  float q_eps = 0.f;
};
hipError_t launch_attention(const AttnArgs& p, hipStream_t s);
// bf16 self-attention's split of its last round (0 per shape, 1 never, 2 or 4 forced).
void set_attention_split(int mode);
// bf16 attention's shape (0 per launch, 4 or 8 waves forced).
void set_attention_shape(int waves);
// The shape a bf16 attention launch takes on `slots` compute units under the
// current settings, and the split of its last round (pieces per item and
// split items; 0 if none).  Host arithmetic only.
struct AttnPlan {
  int waves = 8;
  int split_pieces = 0;
  int split_items = 0;
};
AttnPlan attention_plan(const int* cu_q, const int* cu_k, int n_req, int n_heads, int slots);

// out = LN(x) * mul + add, mul/add per request (modulate: mul = 1 + scale) or
// shared (affine: gamma, beta).
struct LnArgs {
  const void* x;
  void* out;
  int64_t n_rows;
  int hidden;
  float eps;
  bool affine;
  const float* shift; const float* scale; int64_t mod_stride;  // modulate
  const void* gamma; const void* beta;                          // affine
  ReqTable req;
  dit_dtype dtype;
};
hipError_t launch_layer_norm(const LnArgs& p, hipStream_t s);

struct NormRopeArgs {
  void* q; void* k;
  int64_t row_stride, n_rows;
  int n_heads, head_dim;
  const void* g_q; const void* g_k;
  float eps;
  bool rope;
  int sections[3];
  float theta;
  RopeTable tab;
  dit_dtype dtype;
};
hipError_t launch_qk_norm_rope(const NormRopeArgs& p, hipStream_t s);

struct GatedResArgs {
  const void* x; const void* z; const void* bias;
  const float* gate; int64_t gate_stride;
  void* out;
  int64_t n_rows; int hidden;
  ReqTable req;
  dit_dtype dtype;
};
hipError_t launch_gated_residual(const GatedResArgs& p, hipStream_t s);

// Timestep conditioning: e (fp32 [R,F]) -> ... -> mod (fp32 [R,6D]).
// Timestep conditioning in two optional parts:
//  - w_t1 != NULL: e = sinusoid(t), a1 = SiLU(W_t1 e + b_t1), c = SiLU(W_t2 a1 + b_t2)
//    (c holds SiLU of the timestep MLP's output, the input of every modulation);
//  - w_ada != NULL: mod = W_ada c + b_ada with n_mod*hidden outputs per request.
struct CondArgs {
  const float* t; int n_req; int freq_dim; int hidden;
  const void *w_t1, *b_t1, *w_t2, *b_t2, *w_ada, *b_ada;
  int n_mod;
  float* e; float* a1; float* c;   // scratch [R,F], [R,D], [R,D]
  float* mod;
  dit_dtype dtype;
};
hipError_t launch_conditioning(const CondArgs& p, hipStream_t s);

struct LatentArgs {
  const float* latent;   // fp32 packed latent
  void* tokens;          // [rows, P] dtype (patchify: written; Euler: the velocity, read)
  const float* dt;       // device [n_req] (Euler only)
  float* latent_out;     // Euler only; may equal latent
  LatentTable tab;
  dit_dtype dtype;
};
hipError_t launch_patchify(const LatentArgs& p, hipStream_t s);
hipError_t launch_unpatchify_euler(const LatentArgs& p, hipStream_t s);

}  // namespace dit
