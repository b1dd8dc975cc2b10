/*
 * dit_block.h -- C ABI of the MI355X (gfx950) DiT block library.
 *
 * One DiT transformer block forward on one GPU's share of a request or of a
 * packed batch of requests: the denoising stage that the GF-DiT paper names as
 * dominating execution time (section 1, Introduction), where each step computes
 * bidirectionally over the entire latent sequence (section 2.1, Rescheduling
 * Boundaries), for the Wan2.2 video and Qwen-Image workloads of its evaluation
 * (section 6.1, Experimental Setup).  The paper does not define the block; it
 * is the adaLN-Zero DiT block with QK-RMSNorm, sectioned 3D rotary embeddings,
 * full self-attention, cross-attention to text and a GELU-tanh MLP.  A
 * denoising-step executor takes a task over its artifacts -- latent state,
 * conditioning and text embeddings (section 3.1, Reschedulable Trajectory
 * Tasks) -- which is the argument set of dit_block_forward.
 *
 * Conventions shared by every entry point:
 *  - Every pointer not marked "host" is device memory on the current HIP
 *    device.  The caller owns all memory; the library allocates and frees
 *    nothing and keeps no mutable global state, so calls are thread-safe
 *    (the one exception, dit_timestep_modulation_noalloc, says so).
 *  - Tensors are row-major.  Activations are token-major [rows, width];
 *    Linear weights are [out, in] (every GEMM is A . W^T); vectors are dense.
 *  - dtype DIT_BF16: activations, weights, norm gains and biases are bfloat16;
 *    accumulation, norm statistics, softmax and the modulation vectors are
 *    fp32.  dtype DIT_F32: everything is fp32.
 *  - Every call is asynchronous on `stream` and never synchronises.  Arguments
 *    are validated on the host before anything is launched; a failed check
 *    returns DIT_ERR_INVALID_ARG or DIT_ERR_UNSUPPORTED and launches nothing.
 *    A failed launch returns DIT_ERR_HIP.  Faults inside kernels surface at the
 *    caller's next synchronisation.  dit_last_error() gives a thread-local
 *    message for the last failure.  The library never aborts or exits.
 *  - Packed batches: request r owns rows cu_seqlens[r]..cu_seqlens[r+1] (host
 *    arrays, non-decreasing, starting at 0).  Rows never interact across
 *    requests.  At most DIT_MAX_REQ requests per call.
 *  - Device pointers must be 16-byte aligned, and row strides must keep every
 *    row 16-byte aligned.
 */
#ifndef DIT_BLOCK_H
#define DIT_BLOCK_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DIT_MAX_REQ 64
#define DIT_ABI_VERSION 4

typedef enum {
  DIT_OK = 0,
  DIT_ERR_INVALID_ARG = -1, /* a null pointer, a bad size, stride or table */
  DIT_ERR_UNSUPPORTED = -2, /* valid, but a shape this build has no kernel for */
  DIT_ERR_WORKSPACE = -3,   /* workspace smaller than dit_block_workspace_size */
  DIT_ERR_HIP = -4          /* a HIP launch or runtime call failed */
} dit_status;

typedef enum { DIT_F32 = 0, DIT_BF16 = 1 } dit_dtype;

/* Epilogues of dit_linear, applied to z = A . W^T + bias per element. */
typedef enum {
  DIT_EPI_NONE = 0,           /* out = z */
  DIT_EPI_GELU_TANH = 1,      /* out = 0.5 z (1 + tanh(sqrt(2/pi)(z + 0.044715 z^3))) */
  DIT_EPI_RESIDUAL = 2,       /* out = res + z */
  DIT_EPI_GATED_RESIDUAL = 3  /* out = res + gate[req(row)] * z (per-request fp32 gate) */
} dit_epilogue;

/* Hyper-parameters of one block.  hidden = n_heads * head_dim. */
typedef struct {
  int hidden;           /* D */
  int n_heads;          /* H */
  int head_dim;         /* d: 128 for bf16; 64 or 128 for fp32 */
  int mlp_hidden;       /* Dff */
  int freq_dim;         /* F: width of the sinusoidal timestep encoding (even) */
  int rope_sections[3]; /* (d_t, d_h, d_w): even, sum == head_dim; {0,0,0} = no rotary */
  float rope_theta;     /* rotary base, 10000 */
  int qk_norm;          /* 1: per-head RMSNorm on q, k (self) and cq, ck (cross) */
  float ln_eps;         /* LayerNorm epsilon (biased variance), 1e-6 */
  float rms_eps;        /* RMSNorm epsilon, 1e-6 */
  dit_dtype dtype;
} dit_block_config;

/* Device pointers to the block's parameters ([out, in] weights, dtype of the
 * config).  Shapes: w_t1 [D,F] b_t1 [D] w_t2 [D,D] b_t2 [D] w_ada [6D,D]
 * b_ada [6D] w_qkv [3D,D] b_qkv [3D] g_q,g_k [d] w_o [D,D] b_o [D] g_ca,b_ca [D]
 * w_cq [D,D] b_cq [D] w_ckv [2D,D] b_ckv [2D] g_cq,g_ck [d] w_co [D,D] b_co [D]
 * w_up [Dff,D] b_up [Dff] w_dn [D,Dff] b_dn [D].  The gains may be NULL when
 * qk_norm == 0. */
typedef struct {
  const void *w_t1, *b_t1, *w_t2, *b_t2, *w_ada, *b_ada;
  const void *w_qkv, *b_qkv, *g_q, *g_k, *w_o, *b_o;
  const void *g_ca, *b_ca, *w_cq, *b_cq, *w_ckv, *b_ckv, *g_cq, *g_ck, *w_co, *b_co;
  const void *w_up, *b_up, *w_dn, *b_dn;
} dit_block_weights;

/* A packed batch on this GPU.  All arrays are HOST memory and are read during
 * the call only (their values are baked into the launches). */
typedef struct {
  int n_req;                     /* 1..DIT_MAX_REQ */
  const int32_t *cu_seqlens;     /* host [n_req+1]: latent rows of each request here */
  const int32_t *cu_seqlens_txt; /* host [n_req+1]: text rows of each request */
  const int32_t *grid_fhw;       /* host [n_req*3]: full (F,H,W) token grid of each request */
  const int32_t *pos_offset;     /* host [n_req] or NULL (all 0): flattened grid index of
                                    the request's first row here (sequence-parallel shard) */
} dit_varlen;

/* ---------------------------------------------------------------- the block */

/* Bytes of device workspace dit_block_forward / _pre_attention /
 * _post_attention need for this config and batch (0 if the arguments are
 * invalid). */
size_t dit_block_workspace_size(const dit_block_config *cfg, const dit_varlen *vl);

/* One block: y = Block(x; t, txt).  x, y: [rows, D]; t: device fp32 [n_req]
 * timesteps; mod: device fp32 [n_req, 6, D] modulation vectors in the order
 * of dit_timestep_modulation, or NULL to compute them from t (with mod given,
 * t may be NULL and the block's w_t1..b_ada are not read: a model whose
 * blocks share one timestep MLP passes each block's modulation here);
 * txt: [txt_rows, D] text embeddings.  y may equal x.  The workspace (ws,
 * ws_bytes) must hold dit_block_workspace_size bytes, 256-byte aligned; its
 * contents are scratch. */
dit_status dit_block_forward(const dit_block_config *cfg, const dit_block_weights *w,
                             const dit_varlen *vl, const void *x, const float *t,
                             const float *mod, const void *txt, void *y, void *ws,
                             size_t ws_bytes, hipStream_t stream);

/* The block split at self-attention, the two points where a sequence-parallel
 * runtime exchanges rows for heads (an all-to-all each way) between GPUs.
 * Both halves take the conditioning the way dit_block_forward does: either
 * timesteps t (the block's own timestep MLP and adaLN projection run) or
 * precomputed modulation vectors (a model whose blocks share one timestep
 * MLP; w_t1..b_ada are then not read).
 *
 * Steps before self-attention, on this GPU's rows: modulated LayerNorm, QKV
 * projection, per-head RMSNorm and rotary on q and k.  With t != NULL (device
 * fp32 [n_req]) the modulation mod = adaLN(t) is computed and written to mod
 * (device fp32 [n_req, 6, D]); with t == NULL, mod is read as given.
 * qkv: three planes [3, rows, D] (written): q = qkv[0], k = qkv[1],
 * v = qkv[2], each row-major with row stride D, head j in columns
 * [j*d, (j+1)*d).  Separate planes keep each row kernel's and attention's
 * reads on whole contiguous rows. */
dit_status dit_block_pre_attention(const dit_block_config *cfg, const dit_block_weights *w,
                                   const dit_varlen *vl, const void *x, const float *t,
                                   float *mod, void *qkv, void *ws, size_t ws_bytes,
                                   hipStream_t stream);

/* Steps after self-attention, on this GPU's rows: o [rows, D] is the
 * attention output (heads concatenated).  Gated output projection,
 * cross-attention to each request's text, gated GELU-tanh MLP; writes y.
 * mod: device fp32 [n_req, 6, D] (from dit_block_pre_attention or
 * dit_timestep_modulation), or NULL to compute it from t (device fp32
 * [n_req]) in the workspace.  y may equal x. */
dit_status dit_block_post_attention(const dit_block_config *cfg, const dit_block_weights *w,
                                    const dit_varlen *vl, const void *x, const void *o,
                                    const void *txt, const float *t, const float *mod, void *y,
                                    void *ws, size_t ws_bytes, hipStream_t stream);

/* --------------------------------------------------------------- the stages */

/* Timestep conditioning (adaLN-Zero): e = [cos(t w), sin(t w)] with
 * w_i = 10000^(-i/(F/2)); c = W_t2 SiLU(W_t1 e + b_t1) + b_t2;
 * mod = W_ada SiLU(c) + b_ada, written as fp32 [n_req, 6, D] in the order
 * shift_sa, scale_sa, gate_sa, shift_ff, scale_ff, gate_ff.  ws must hold
 * (F + 2D) * n_req floats. */
dit_status dit_timestep_modulation(const dit_block_config *cfg, const dit_block_weights *w,
                                   int n_req, const float *t, float *mod, void *ws,
                                   size_t ws_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation:
 * dit_timestep_modulation with the same arguments and results but no
 * workspace.  Its scratch (the sinusoidal encoding and the timestep MLP's two
 * hidden vectors, (F + 2D) * n_req floats, each part 256-byte aligned) lives
 * in a static device array of DIT_NOALLOC_SCRATCH_BYTES bytes that every GPU
 * the library runs on holds until the process ends; the library looks up its
 * address once per device, on the first call there.  Nothing is allocated or
 * freed.  A size over the array gives DIT_ERR_UNSUPPORTED (nothing launched).
 * Every call on one GPU shares that GPU's array and leaves its contents
 * behind (each call writes all it reads, so nothing needs clearing); calls
 * that overlap on one GPU (other streams or threads) race on it. */
#define DIT_NOALLOC_SCRATCH_BYTES (8u << 20)
dit_status dit_timestep_modulation_noalloc(const dit_block_config *cfg, const dit_block_weights *w,
                                           int n_req, const float *t, float *mod,
                                           hipStream_t stream);

/* Scaled dot-product attention over a packed batch, non-causal, no mask:
 * for request r and head h, O = softmax(Q K^T * softmax_scale) V with queries
 * rows cu_q[r]..cu_q[r+1] and keys/values rows cu_k[r]..cu_k[r+1] (host
 * arrays; cu_q == cu_k for self-attention).  Head h of row i starts at
 * q + i*q_row_stride + h*head_dim (strides in elements; likewise k, v, o).
 * softmax_scale 0 selects the standard 1/sqrt(head_dim); any other finite
 * value is used as given (inf or NaN: DIT_ERR_INVALID_ARG).  o must not
 * overlap q, k or v: the byte range from o's first to its last row must not
 * meet that of q, k or v (checked, DIT_ERR_INVALID_ARG); q, k and v may share
 * one buffer.  bf16 needs head_dim 128, and k_row_stride and v_row_stride of
 * at most 2^24 elements (the kernel forms a key tile's offsets in 32 bits;
 * larger: DIT_ERR_INVALID_ARG); fp32 takes 64 or 128.  A request with
 * queries but no keys gets rows of zeros. */
dit_status dit_attention_varlen(const void *q, const void *k, const void *v, void *o,
                                int64_t q_row_stride, int64_t k_row_stride,
                                int64_t v_row_stride, int64_t o_row_stride,
                                const int32_t *cu_q, const int32_t *cu_k, int n_req,
                                int n_heads, int head_dim, float softmax_scale,
                                dit_dtype dtype, hipStream_t stream);

/* Modulated LayerNorm: out[i] = LN(x[i]) * (1 + scale[r]) + shift[r] for row i
 * of request r (LN over `hidden`, biased variance, eps inside the root).
 * shift, scale: device fp32, request r's vector at shift + r*mod_stride.
 * x, out: [n_rows, hidden] with n_rows = cu_seqlens[n_req]. */
dit_status dit_adaln_modulate(const void *x, const float *shift, const float *scale,
                              int64_t mod_stride, const int32_t *cu_seqlens, int n_req,
                              int hidden, float eps, void *out, dit_dtype dtype,
                              hipStream_t stream);

/* Affine LayerNorm: out = LN(x) * gamma + beta (gamma, beta: [hidden], dtype). */
dit_status dit_layer_norm_affine(const void *x, const void *gamma, const void *beta,
                                 int64_t n_rows, int hidden, float eps, void *out,
                                 dit_dtype dtype, hipStream_t stream);

/* out = epilogue(A . W^T + bias): A [M, K] (row stride lda), W [N, K] (ldw),
 * bias [N] or NULL, out [M, N] (ldo), res [M, N] (ldr; RESIDUAL epilogues,
 * may equal out), gate: device fp32, request r's [N] vector at
 * gate + r*gate_stride (GATED_RESIDUAL), rows grouped by cu_seqlens.
 * bf16 needs K % 64 == 0 and N % 8 == 0. */
dit_status dit_linear(const void *a, int64_t lda, const void *w, int64_t ldw,
                      const void *bias, void *out, int64_t ldo, int64_t M, int N, int K,
                      dit_epilogue epi, const void *res, int64_t ldr, const float *gate,
                      int64_t gate_stride, const int32_t *cu_seqlens, int n_req,
                      dit_dtype dtype, hipStream_t stream);

/* The bf16 GEMM computes 256 x 256 output tiles, or 256 x 192 where fewer
 * rounds of tiles over the compute units make that faster (shapes with few
 * tiles).  For tests and tuning: tile_n = 192 or 256 forces that width for
 * every later bf16 GEMM of this process (every entry point), 0 restores the
 * choice per shape; any other value gives DIT_ERR_INVALID_ARG.  Results do
 * not depend on the width.  Process-wide setting; not synchronised with work
 * in flight (set it between calls). */
dit_status dit_debug_gemm_tile_n(int tile_n);

/* The bf16 self-attention (key ranges over 1024) runs its work items in
 * rounds of one workgroup per compute unit.  When the last round would be at
 * most half full (one request), its items are split into 2 or 4 key pieces
 * that run as one short round and are merged by a second kernel; the pieces
 * live in a static device array of 34 MB that every GPU holds until the
 * process ends, and calls that split are serialised on it by an event (not
 * under graph capture, where no split happens).  For tests and tuning:
 * mode 2 or 4 forces a split of the last request's last items (as many as
 * one round of pieces holds) into that many pieces, 1 disables splitting,
 * 0 restores the choice per shape; other values give DIT_ERR_INVALID_ARG.
 * Process-wide; set it between calls. */
dit_status dit_debug_attention_split(int mode);

/* The bf16 attention runs one of two kernel shapes per call: 8 waves per
 * workgroup (256 query rows, one workgroup per compute unit) or 4 waves (128
 * query rows, two workgroups per compute unit).  Key ranges up to 1024 take
 * the 4-wave shape; so does a single request whose 8-wave items would end in
 * a split last round when the call holds at most 3 x 64 key tiles of
 * 256-query items per compute unit.  For tests and tuning: waves = 4 or 8
 * forces that shape (and the split setting above then applies to the 8-wave
 * shape only), 0 restores the choice per call; other values give
 * DIT_ERR_INVALID_ARG.  Without a split both shapes give the same bits.
 * Process-wide; set it between calls. */
dit_status dit_debug_attention_shape(int waves);

/* The shape (*waves: 4 or 8) and last-round split (*split_pieces: 0, 2 or 4
 * key pieces for each of the last request's last *split_items items) that a
 * bf16 attention call with these ranges takes on a GPU of `compute_units`
 * compute units, under the current debug settings.  Host arithmetic only: no
 * device is used.  cu_q, cu_k: host arrays of n_req + 1 offsets from 0, as
 * for dit_attention_varlen; the outputs are host ints.  A call under graph
 * capture runs the same shape without the split. */
dit_status dit_debug_attention_plan(const int32_t *cu_q, const int32_t *cu_k, int n_req, int n_heads,
                                    int compute_units, int *waves, int *split_pieces, int *split_items);

/* In place on q and (if not NULL) k, each [rows, n_heads*head_dim] with row
 * stride `row_stride`: per-head RMSNorm with gains g_q / g_k (skipped when the
 * gain is NULL), then, if vl != NULL and the sections are not all 0, the
 * sectioned rotary embedding at each row's grid position (vl->cu_seqlens,
 * grid_fhw and pos_offset give the position; n_rows = vl->cu_seqlens[n_req]).
 * Without vl, n_rows rows get the RMSNorm only. */
dit_status dit_qk_norm_rope(void *q, void *k, int64_t row_stride, int64_t n_rows, int n_heads,
                            int head_dim, const void *g_q, const void *g_k, float eps,
                            const int rope_sections[3], float rope_theta, const dit_varlen *vl,
                            dit_dtype dtype, hipStream_t stream);

/* Standalone gated residual: out[i] = x[i] + gate[r] * (z[i] + bias) for row i
 * of request r; x, z, out [n_rows, hidden]; bias [hidden] (dtype) or NULL;
 * gate device fp32 at gate + r*gate_stride.  hidden <= 8192 (bf16) or 4096
 * (fp32), else DIT_ERR_UNSUPPORTED.  out may alias x or z. */
dit_status dit_gated_residual(const void *x, const void *z, const void *bias, const float *gate,
                              int64_t gate_stride, const int32_t *cu_seqlens, int n_req,
                              int hidden, void *out, dit_dtype dtype, hipStream_t stream);

/* ------------------------------------------------------ one denoising step */

/* One denoising step is the unit the paper schedules as a trajectory task: it
 * advances a request's latent along its diffusion trajectory by one timestep
 * and leaves a complete latent state behind (section 2.1, Rescheduling
 * Boundaries; section 3.1, Reschedulable Trajectory Tasks).  The paper does
 * not define the model, so this is the standard DiT stack around the block:
 * patch embedding of the latent, a timestep MLP shared by all blocks, B blocks
 * with per-block adaLN-Zero modulation, an adaLN output layer and a
 * flow-matching Euler update.  The text keys and values of every block's
 * cross-attention do not depend on the latent or the timestep, so they are
 * computed once per request (dit_text_kv) and reused by every step.
 *
 * Latent of request r: fp32, channel-major [C, F*pt, H*ph, W*pw] where
 * (F, H, W) = vl->grid_fhw[r] is its token grid, stored contiguously; the
 * requests follow each other in order (request r starts after the
 * C*F*pt*H*ph*W*pw values of requests 0..r-1).  Token n = (f*H + h)*W + w of
 * the request covers the latent patch at (f*pt, h*ph, w*pw); its patch vector
 * has P = C*pt*ph*pw entries in the order (c, i, j, k) with i over time,
 * j over height and k over width, and the model's output uses the same order,
 * so unpatchify is the exact inverse of patchify.  The step needs whole
 * requests: cu_seqlens[r+1] - cu_seqlens[r] = F*H*W and pos_offset NULL or 0. */
typedef struct {
  dit_block_config block; /* shared by every block */
  int n_blocks;           /* B >= 1 */
  int in_channels;        /* C: latent channels (the velocity has the same) */
  int patch[3];           /* (pt, ph, pw) >= 1; bf16 needs P % 64 == 0, fp32 P % 4 == 0 */
} dit_model_config;

/* Device pointers (dtype of the config) except `blocks`, a HOST array of
 * n_blocks block weight sets.  Shapes with P = C*pt*ph*pw: w_t1 [D,F] b_t1 [D]
 * w_t2 [D,D] b_t2 [D] (the shared timestep MLP); w_pe [D,P] b_pe [D] (patch
 * embedding); w_hmod [2D,D] b_hmod [2D] (output adaLN: shift, scale);
 * w_out [P,D] b_out [P] (output projection).  The blocks' own w_t1..b_t2 are
 * not read: every block takes its modulation W_ada SiLU(c) + b_ada from the
 * shared c. */
typedef struct {
  const void *w_t1, *b_t1, *w_t2, *b_t2;
  const void *w_pe, *b_pe;
  const void *w_hmod, *b_hmod;
  const void *w_out, *b_out;
  const dit_block_weights *blocks;
} dit_model_weights;

/* Elements (not bytes) of the text key/value cache: n_blocks * txt_rows * 2D,
 * dtype of the config.  0 if the arguments are invalid. */
size_t dit_text_kv_elems(const dit_model_config *cfg, const dit_varlen *vl);

/* The cross-attention keys and values of every block: for block b,
 * kv[b] = [RMSNorm_heads(txt W_ck^T + b_ck) | txt W_cv^T + b_cv] (the norm only
 * with qk_norm), [txt_rows, 2D] at kv + b*txt_rows*2D.  txt: [txt_rows, D]. */
dit_status dit_text_kv(const dit_model_config *cfg, const dit_model_weights *w,
                       const dit_varlen *vl, const void *txt, void *kv,
                       hipStream_t stream);

/* Bytes of device workspace dit_denoise_step needs (0 if invalid). */
size_t dit_denoise_workspace_size(const dit_model_config *cfg, const dit_varlen *vl);

/* One flow-matching Euler step of every request in the batch:
 *   x   = patchify(latent) W_pe^T + b_pe                    [rows, D]
 *   c   = W_t2 SiLU(W_t1 emb(t) + b_t1) + b_t2              per request
 *   x   = Block_b(x; c, kv[b]) for b = 0..B-1
 *   v   = (LN(x)(1 + scale) + shift) W_out^T + b_out, (shift, scale) = W_hmod SiLU(c) + b_hmod
 *   latent_out = latent + dt[r] * unpatchify(v)
 * t, dt: device fp32 [n_req] (timestep given to the model, and the step of
 * the flow time, sigma_next - sigma; negative when denoising).  latent,
 * latent_out: fp32 as described above; latent_out may equal latent.  kv: the
 * cache from dit_text_kv.  Workspace as for dit_block_forward, sized by
 * dit_denoise_workspace_size. */
dit_status dit_denoise_step(const dit_model_config *cfg, const dit_model_weights *w,
                            const dit_varlen *vl, const float *latent, const float *t,
                            const float *dt, const void *kv, float *latent_out, void *ws,
                            size_t ws_bytes, hipStream_t stream);

/* The latent <-> token steps of dit_denoise_step on their own.
 * dit_patchify: tokens [rows, P] (dtype, rounded to nearest even for bf16)
 * from the fp32 latent.  dit_unpatchify_euler: latent_out = latent +
 * dt[r] * unpatchify(v), v [rows, P] (dtype); latent_out may equal latent. */
dit_status dit_patchify(const dit_model_config *cfg, const dit_varlen *vl, const float *latent,
                        void *tokens, hipStream_t stream);
dit_status dit_unpatchify_euler(const dit_model_config *cfg, const dit_varlen *vl,
                                const float *latent, const void *v, const float *dt,
                                float *latent_out, hipStream_t stream);

/* -------------------------------------------------------------- diagnostics */

const char *dit_status_string(dit_status s);
/* Thread-local description of the last failure in this thread ("" if none). */
const char *dit_last_error(void);
int dit_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DIT_BLOCK_H */
