// C ABI of the DiT block library: argument validation on the host (before
// any HIP call), workspace layout, and the order of launches of one block.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <string>

#include "dit_block.h"
#include "kernels.hpp"

using namespace dit;

namespace {

thread_local std::string g_last_error;

dit_status fail(dit_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

dit_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return DIT_OK;
  return fail(DIT_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define DIT_TRY(expr)                      \
  do {                                     \
    dit_status _s = (expr);                \
    if (_s != DIT_OK) return _s;           \
  } while (0)

#define DIT_HIP(expr, what) DIT_TRY(hip_status((expr), (what)))

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

size_t elem_size(dit_dtype dt) { return dt == DIT_BF16 ? 2 : 4; }

dit_status check_dtype(dit_dtype dt) {
  if (dt != DIT_F32 && dt != DIT_BF16) return fail(DIT_ERR_INVALID_ARG, "dtype %d is neither DIT_F32 nor DIT_BF16", (int)dt);
  return DIT_OK;
}

dit_status check_ptr(const void* p, const char* name, bool allow_null = false) {
  if (!p) {
    if (allow_null) return DIT_OK;
    return fail(DIT_ERR_INVALID_ARG, "%s is NULL", name);
  }
  if (!aligned16(p)) return fail(DIT_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return DIT_OK;
}

// A host cu_seqlens array of n_req+1 entries: starts at 0, non-decreasing.
dit_status check_cu(const int32_t* cu, int n_req, const char* name) {
  if (n_req < 1 || n_req > DIT_MAX_REQ)
    return fail(DIT_ERR_INVALID_ARG, "n_req = %d outside 1..%d", n_req, DIT_MAX_REQ);
  if (!cu) return fail(DIT_ERR_INVALID_ARG, "%s is NULL", name);
  if (cu[0] != 0) return fail(DIT_ERR_INVALID_ARG, "%s[0] = %d, must be 0", name, cu[0]);
  for (int r = 0; r < n_req; ++r)
    if (cu[r + 1] < cu[r]) return fail(DIT_ERR_INVALID_ARG, "%s decreases at %d", name, r);
  return DIT_OK;
}

// Byte range [lo, hi) of `rows` rows of `width` elements at a row stride.
struct Span { uintptr_t lo, hi; };

Span span(const void* p, int64_t rows, int64_t stride, int64_t width, int64_t es) {
  const uintptr_t lo = (uintptr_t)p;
  if (rows <= 0) return {lo, lo};
  return {lo, lo + (uintptr_t)(((rows - 1) * stride + width) * es)};
}

bool overlaps(const Span& a, const Span& b) { return a.lo < a.hi && b.lo < b.hi && a.lo < b.hi && b.lo < a.hi; }

ReqTable make_req(const int32_t* cu, int n_req) {
  ReqTable t;
  memset(&t, 0, sizeof(t));
  t.n_req = n_req;
  for (int r = 0; r <= n_req; ++r) t.cu[r] = cu[r];
  return t;
}

ReqTable single_req(int64_t n_rows) {
  ReqTable t;
  memset(&t, 0, sizeof(t));
  t.n_req = 1;
  t.cu[1] = (int)n_rows;
  return t;
}

bool rope_on(const int s[3]) { return s[0] != 0 || s[1] != 0 || s[2] != 0; }

dit_status check_sections(const int s[3], int head_dim) {
  if (!rope_on(s)) return DIT_OK;
  for (int i = 0; i < 3; ++i)
    if (s[i] < 0 || (s[i] & 1))
      return fail(DIT_ERR_INVALID_ARG, "rope section %d = %d must be even and >= 0", i, s[i]);
  if (s[0] + s[1] + s[2] != head_dim)
    return fail(DIT_ERR_INVALID_ARG, "rope sections sum to %d, head_dim is %d", s[0] + s[1] + s[2], head_dim);
  return DIT_OK;
}

dit_status check_varlen(const dit_varlen* vl, bool need_txt) {
  if (!vl) return fail(DIT_ERR_INVALID_ARG, "varlen is NULL");
  DIT_TRY(check_cu(vl->cu_seqlens, vl->n_req, "cu_seqlens"));
  if (need_txt) DIT_TRY(check_cu(vl->cu_seqlens_txt, vl->n_req, "cu_seqlens_txt"));
  return DIT_OK;
}

dit_status check_rope_table(const dit_varlen* vl, const int s[3], RopeTable* tab) {
  memset(tab, 0, sizeof(*tab));
  tab->n_req = vl->n_req;
  for (int r = 0; r <= vl->n_req; ++r) tab->cu[r] = vl->cu_seqlens[r];
  if (!rope_on(s)) return DIT_OK;
  if (!vl->grid_fhw) return fail(DIT_ERR_INVALID_ARG, "grid_fhw is NULL with rotary on");
  for (int r = 0; r < vl->n_req; ++r) {
    const int F = vl->grid_fhw[3 * r], H = vl->grid_fhw[3 * r + 1], W = vl->grid_fhw[3 * r + 2];
    if (F < 1 || H < 1 || W < 1)
      return fail(DIT_ERR_INVALID_ARG, "grid of request %d is (%d,%d,%d)", r, F, H, W);
    const int64_t cells = (int64_t)F * H * W;
    const int off = vl->pos_offset ? vl->pos_offset[r] : 0;
    const int rows = vl->cu_seqlens[r + 1] - vl->cu_seqlens[r];
    if (off < 0 || off + (int64_t)rows > cells)
      return fail(DIT_ERR_INVALID_ARG, "request %d: rows %d from offset %d exceed its grid of %lld cells", r,
                  rows, off, (long long)cells);
    tab->grid_hw[r] = H * W;
    tab->grid_w[r] = W;
    tab->grid_h[r] = H;
    tab->offset[r] = off;
  }
  return DIT_OK;
}

dit_status check_cfg(const dit_block_config* c) {
  if (!c) return fail(DIT_ERR_INVALID_ARG, "config is NULL");
  DIT_TRY(check_dtype(c->dtype));
  if (c->hidden <= 0 || c->n_heads <= 0 || c->head_dim <= 0 || c->mlp_hidden <= 0 || c->freq_dim <= 0)
    return fail(DIT_ERR_INVALID_ARG, "non-positive size in config");
  if (c->n_heads * c->head_dim != c->hidden)
    return fail(DIT_ERR_INVALID_ARG, "n_heads * head_dim = %d != hidden = %d", c->n_heads * c->head_dim, c->hidden);
  if (c->freq_dim & 1) return fail(DIT_ERR_INVALID_ARG, "freq_dim %d is odd", c->freq_dim);
  if (!(c->ln_eps > 0.f) || !(c->rms_eps > 0.f)) return fail(DIT_ERR_INVALID_ARG, "eps must be > 0");
  if (rope_on(c->rope_sections) && !(c->rope_theta > 0.f)) return fail(DIT_ERR_INVALID_ARG, "rope_theta must be > 0");
  DIT_TRY(check_sections(c->rope_sections, c->head_dim));
  if (c->dtype == DIT_BF16) {
    if (c->head_dim != 128) return fail(DIT_ERR_UNSUPPORTED, "bf16 head_dim %d (only 128)", c->head_dim);
    if (c->hidden % 64 || c->mlp_hidden % 64 || c->freq_dim % 64)
      return fail(DIT_ERR_UNSUPPORTED, "bf16 needs hidden, mlp_hidden and freq_dim multiples of 64");
    if (c->hidden > 8192) return fail(DIT_ERR_UNSUPPORTED, "bf16 hidden %d > 8192", c->hidden);
  } else {
    if (c->head_dim != 64 && c->head_dim != 128)
      return fail(DIT_ERR_UNSUPPORTED, "fp32 head_dim %d (64 or 128)", c->head_dim);
    if (c->hidden % 4 || c->mlp_hidden % 4 || c->freq_dim % 4)
      return fail(DIT_ERR_UNSUPPORTED, "fp32 needs hidden, mlp_hidden and freq_dim multiples of 4");
    if (c->hidden > 4096) return fail(DIT_ERR_UNSUPPORTED, "fp32 hidden %d > 4096", c->hidden);
  }
  return DIT_OK;
}

// The block's own conditioning chain: timestep MLP and adaLN projection.
dit_status check_cond_weights(const dit_block_weights* w) {
  if (!w) return fail(DIT_ERR_INVALID_ARG, "weights is NULL");
  DIT_TRY(check_ptr(w->w_t1, "w_t1")); DIT_TRY(check_ptr(w->b_t1, "b_t1"));
  DIT_TRY(check_ptr(w->w_t2, "w_t2")); DIT_TRY(check_ptr(w->b_t2, "b_t2"));
  DIT_TRY(check_ptr(w->w_ada, "w_ada")); DIT_TRY(check_ptr(w->b_ada, "b_ada"));
  return DIT_OK;
}

// tmlp: the block's own timestep MLP is read (not by the denoising step, whose
// blocks share the model's).
dit_status check_weights(const dit_block_config* c, const dit_block_weights* w, bool pre, bool post,
                         bool tmlp = true, bool ada = true) {
  if (!w) return fail(DIT_ERR_INVALID_ARG, "weights is NULL");
  const bool qn = c->qk_norm != 0;
  if (pre && tmlp) {
    DIT_TRY(check_ptr(w->w_t1, "w_t1")); DIT_TRY(check_ptr(w->b_t1, "b_t1"));
    DIT_TRY(check_ptr(w->w_t2, "w_t2")); DIT_TRY(check_ptr(w->b_t2, "b_t2"));
  }
  if (pre && ada) {
    DIT_TRY(check_ptr(w->w_ada, "w_ada")); DIT_TRY(check_ptr(w->b_ada, "b_ada"));
  }
  if (pre) {
    DIT_TRY(check_ptr(w->w_qkv, "w_qkv")); DIT_TRY(check_ptr(w->b_qkv, "b_qkv"));
    DIT_TRY(check_ptr(w->g_q, "g_q", !qn)); DIT_TRY(check_ptr(w->g_k, "g_k", !qn));
  }
  if (post) {
    DIT_TRY(check_ptr(w->w_o, "w_o")); DIT_TRY(check_ptr(w->b_o, "b_o"));
    DIT_TRY(check_ptr(w->g_ca, "g_ca")); DIT_TRY(check_ptr(w->b_ca, "b_ca"));
    DIT_TRY(check_ptr(w->w_cq, "w_cq")); DIT_TRY(check_ptr(w->b_cq, "b_cq"));
    DIT_TRY(check_ptr(w->w_ckv, "w_ckv")); DIT_TRY(check_ptr(w->b_ckv, "b_ckv"));
    DIT_TRY(check_ptr(w->g_cq, "g_cq", !qn)); DIT_TRY(check_ptr(w->g_ck, "g_ck", !qn));
    DIT_TRY(check_ptr(w->w_co, "w_co")); DIT_TRY(check_ptr(w->b_co, "b_co"));
    DIT_TRY(check_ptr(w->w_up, "w_up")); DIT_TRY(check_ptr(w->b_up, "b_up"));
    DIT_TRY(check_ptr(w->w_dn, "w_dn")); DIT_TRY(check_ptr(w->b_dn, "b_dn"));
  }
  return DIT_OK;
}

// ------------------------------------------------------------ workspace

struct Workspace {
  float* mod;
  float *e, *a1, *c;
  char *h, *qkv, *o, *x1, *cq, *ckv, *u;
};

inline size_t round256(size_t b) { return (b + 255) & ~(size_t)255; }

size_t layout(const dit_block_config* c, const dit_varlen* vl, char* base, Workspace* ws) {
  const size_t es = elem_size(c->dtype);
  const size_t R = vl->n_req, T = vl->cu_seqlens[vl->n_req];
  const size_t L = vl->cu_seqlens_txt ? vl->cu_seqlens_txt[vl->n_req] : 0;
  const size_t D = c->hidden, F = c->freq_dim, Dff = c->mlp_hidden;
  size_t off = 0;
  auto take = [&](size_t bytes) { char* p = base ? base + off : nullptr; off += round256(bytes); return p; };
  Workspace w;
  w.mod = (float*)take(R * 6 * D * 4);
  w.e = (float*)take(R * F * 4);
  w.a1 = (float*)take(R * D * 4);
  w.c = (float*)take(R * D * 4);
  w.h = take(T * D * es);
  w.qkv = take(T * 3 * D * es);
  w.o = take(T * D * es);
  w.x1 = take(T * D * es);
  w.cq = take(T * D * es);
  w.ckv = take(L * 2 * D * es);
  w.u = take(T * Dff * es);
  if (ws) *ws = w;
  return off;
}

dit_status check_ws(const dit_block_config* c, const dit_varlen* vl, void* ws, size_t ws_bytes, Workspace* out) {
  const size_t need = layout(c, vl, nullptr, nullptr);
  if (!ws) return fail(DIT_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (((uintptr_t)ws & 255u) != 0) return fail(DIT_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (ws_bytes < need) return fail(DIT_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, need);
  layout(c, vl, (char*)ws, out);
  return DIT_OK;
}

// ------------------------------------------------------------- stages

dit_status run_linear(const void* a, int64_t lda, const void* w, int64_t ldw, const void* bias, void* out,
                      int64_t ldo, int64_t M, int N, int K, dit_epilogue epi, const void* res, int64_t ldr,
                      const float* gate, int64_t gate_stride, const ReqTable& req, dit_dtype dt,
                      hipStream_t s, const char* what, int plane_cols = 0, int64_t plane_stride = 0) {
  LinearArgs p;
  p.a = a; p.lda = lda; p.w = w; p.ldw = ldw; p.bias = bias; p.out = out; p.ldo = ldo;
  p.M = M; p.N = N; p.K = K; p.epi = epi; p.res = res; p.ldr = ldr; p.gate = gate;
  p.gate_stride = gate_stride; p.req = req; p.dtype = dt;
  p.plane_cols = plane_cols; p.plane_stride = plane_stride;
  return hip_status(launch_linear(p, s), what);
}

dit_status run_ln_mod(const void* x, const float* shift, const float* scale, int64_t stride, const ReqTable& req,
                      int64_t n_rows, int hidden, float eps, void* out, dit_dtype dt, hipStream_t s) {
  LnArgs p;
  memset(&p, 0, sizeof(p));
  p.x = x; p.out = out; p.n_rows = n_rows; p.hidden = hidden; p.eps = eps; p.affine = false;
  p.shift = shift; p.scale = scale; p.mod_stride = stride; p.req = req; p.dtype = dt;
  return hip_status(launch_layer_norm(p, s), "layer_norm (modulate)");
}

dit_status run_ln_affine(const void* x, const void* g, const void* b, int64_t n_rows, int hidden, float eps,
                         void* out, dit_dtype dt, hipStream_t s) {
  LnArgs p;
  memset(&p, 0, sizeof(p));
  p.x = x; p.out = out; p.n_rows = n_rows; p.hidden = hidden; p.eps = eps; p.affine = true;
  p.gamma = g; p.beta = b; p.req = single_req(n_rows); p.dtype = dt;
  return hip_status(launch_layer_norm(p, s), "layer_norm (affine)");
}

dit_status run_norm_rope(void* q, void* k, int64_t stride, int64_t n_rows, int n_heads, int head_dim,
                         const void* gq, const void* gk, float eps, const int sec[3], float theta,
                         const RopeTable* tab, dit_dtype dt, hipStream_t s) {
  NormRopeArgs p;
  memset(&p, 0, sizeof(p));
  p.q = q; p.k = k; p.row_stride = stride; p.n_rows = n_rows; p.n_heads = n_heads; p.head_dim = head_dim;
  p.g_q = gq; p.g_k = gk; p.eps = eps; p.rope = tab != nullptr && rope_on(sec);
  for (int i = 0; i < 3; ++i) p.sections[i] = sec[i];
  p.theta = theta;
  if (tab) p.tab = *tab;
  p.dtype = dt;
  return hip_status(launch_qk_norm_rope(p, s), "qk_norm_rope");
}

dit_status run_attention(const void* q, const void* k, const void* v, void* o, int64_t qs, int64_t ks,
                         int64_t vs, int64_t os, const ReqTable& cq, const ReqTable& ck, int n_heads,
                         int head_dim, float scale, dit_dtype dt, hipStream_t s, const void* q_gain = nullptr,
                         float q_eps = 0.f) {
  AttnArgs p;
  p.q = q; p.k = k; p.v = v; p.o = o; p.q_stride = qs; p.k_stride = ks; p.v_stride = vs; p.o_stride = os;
  p.cq = cq; p.ck = ck; p.n_heads = n_heads; p.head_dim = head_dim; p.scale = scale; p.dtype = dt;
  p.q_gain = q_gain; p.q_eps = q_eps;
  return hip_status(launch_attention(p, s), "attention");
}

dit_status run_cond(const dit_block_config* c, const dit_block_weights* w, int n_req, const float* t, float* mod,
                    float* e, float* a1, float* cc, hipStream_t s) {
  CondArgs p;
  p.t = t; p.n_req = n_req; p.freq_dim = c->freq_dim; p.hidden = c->hidden;
  p.w_t1 = w->w_t1; p.b_t1 = w->b_t1; p.w_t2 = w->w_t2; p.b_t2 = w->b_t2; p.w_ada = w->w_ada; p.b_ada = w->b_ada;
  p.n_mod = 6; p.e = e; p.a1 = a1; p.c = cc; p.mod = mod; p.dtype = c->dtype;
  return hip_status(launch_conditioning(p, s), "timestep conditioning");
}

// S1..S3 on this GPU's rows: h = LN(x)(1+scale_sa)+shift_sa; [q|k|v] = h W^T + b; q,k RMSNorm + rotary.
// q, k and v are written as three planes [T, D] (row stride D), T * D elements apart: the row
// kernels and attention then read contiguous rows of one tensor.
dit_status pre_attention_impl(const dit_block_config* c, const dit_block_weights* w, const dit_varlen* vl,
                              const void* x, const float* mod, void* qkv, const Workspace& ws,
                              hipStream_t s) {
  const int D = c->hidden;
  const int64_t T = vl->cu_seqlens[vl->n_req];
  const ReqTable req = make_req(vl->cu_seqlens, vl->n_req);
  RopeTable tab;
  DIT_TRY(check_rope_table(vl, c->rope_sections, &tab));
  DIT_TRY(run_ln_mod(x, mod + 0 * D, mod + 1 * D, 6 * D, req, T, D, c->ln_eps, ws.h, c->dtype, s));
  DIT_TRY(run_linear(ws.h, D, w->w_qkv, D, w->b_qkv, qkv, D, T, 3 * D, D, DIT_EPI_NONE, nullptr, 0, nullptr,
                     0, req, c->dtype, s, "qkv projection", D, T * D));
  const size_t es = elem_size(c->dtype);
  DIT_TRY(run_norm_rope(qkv, (char*)qkv + T * D * es, D, T, c->n_heads, c->head_dim, c->qk_norm ? w->g_q : nullptr,
                        c->qk_norm ? w->g_k : nullptr, c->rms_eps, c->rope_sections, c->rope_theta, &tab,
                        c->dtype, s));
  return DIT_OK;
}

// Self-attention of one block over the q, k, v planes that pre_attention_impl wrote.
dit_status self_attention_impl(const dit_block_config* c, const dit_varlen* vl, const char* qkv, void* o,
                               hipStream_t s) {
  const int D = c->hidden;
  const int64_t T = vl->cu_seqlens[vl->n_req];
  const size_t plane = (size_t)T * D * elem_size(c->dtype);
  const ReqTable req = make_req(vl->cu_seqlens, vl->n_req);
  return run_attention(qkv, qkv + plane, qkv + 2 * plane, o, D, D, D, D, req, req, c->n_heads, c->head_dim,
                       1.0f / sqrtf((float)c->head_dim), c->dtype, s);
}

// Cross-attention keys and values of one block: kv = [RMS(txt W_ck^T + b_ck) | txt W_cv^T + b_cv].
dit_status text_kv_impl(const dit_block_config* c, const dit_block_weights* w, int64_t L, const ReqTable& req_txt,
                        const void* txt, void* kv, hipStream_t s) {
  const int D = c->hidden;
  DIT_TRY(run_linear(txt, D, w->w_ckv, D, w->b_ckv, kv, 2 * D, L, 2 * D, D, DIT_EPI_NONE, nullptr, 0, nullptr, 0,
                     req_txt, c->dtype, s, "text key/value projection"));
  if (c->qk_norm) {
    const int zero[3] = {0, 0, 0};
    DIT_TRY(run_norm_rope(kv, nullptr, 2 * D, L, c->n_heads, c->head_dim, w->g_ck, nullptr, c->rms_eps, zero, 0.f,
                          nullptr, c->dtype, s));
  }
  return DIT_OK;
}

// A second stream per device (default priority) with a fork and a join
// event, for the text key/value projection: it depends on the text and the
// weights only, so it runs beside the output projection, LayerNorm and
// cross-query projection instead of after them.  Where those leave compute
// units idle (a short sequence: 192 tiles of 256 x 256 on 256 CUs) its tiles
// fill them.  The mutex covers a call's enqueue from fork to join, so calls
// from several host threads never interleave their use of the two events.
struct SideStream {
  hipStream_t stream = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  std::mutex mu;
};
constexpr int kMaxSideDevices = 64;
std::mutex g_side_mu;
SideStream* g_side[kMaxSideDevices] = {};

// The current device's side stream, created on first use; NULL if it cannot
// be created (the caller then runs everything on its own stream).
SideStream* side_stream() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxSideDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_side_mu);
  if (!g_side[dev]) {
    SideStream* ss = new SideStream;
    const bool ok = hipStreamCreateWithFlags(&ss->stream, hipStreamNonBlocking) == hipSuccess &&
                    hipEventCreateWithFlags(&ss->fork, hipEventDisableTiming) == hipSuccess &&
                    hipEventCreateWithFlags(&ss->join, hipEventDisableTiming) == hipSuccess;
    if (!ok) {
      if (ss->join) (void)hipEventDestroy(ss->join);
      if (ss->fork) (void)hipEventDestroy(ss->fork);
      if (ss->stream) (void)hipStreamDestroy(ss->stream);
      delete ss;
      (void)hipGetLastError();
      return nullptr;
    }
    g_side[dev] = ss;
  }
  return g_side[dev];
}

// S5..S12 on this GPU's rows given the self-attention output o.
// With kv != NULL the text keys and values come from that cache ([txt_rows, 2D],
// normalised keys) and txt is not read; kv_side != NULL: kv is still being
// written on that side stream, whose join event s waits for before the
// cross-attention (the caller holds its mutex).
dit_status post_attention_impl(const dit_block_config* c, const dit_block_weights* w, const dit_varlen* vl,
                               const void* x, const void* o, const void* txt, const float* mod, void* y,
                               const Workspace& ws, hipStream_t s, const void* kv = nullptr,
                               SideStream* kv_side = nullptr) {
  const int D = c->hidden, Dff = c->mlp_hidden;
  const int64_t T = vl->cu_seqlens[vl->n_req];
  const int64_t L = vl->cu_seqlens_txt[vl->n_req];
  const size_t es = elem_size(c->dtype);
  const ReqTable req = make_req(vl->cu_seqlens, vl->n_req);
  const ReqTable req_txt = make_req(vl->cu_seqlens_txt, vl->n_req);
  const dit_dtype dt = c->dtype;
  // [ck | cv] = txt W_ckv^T + b_ckv ; ck = RMS(ck), on the side stream when there is one
  const char* ckv = (const char*)kv;
  SideStream* side = kv ? kv_side : nullptr;
  std::unique_lock<std::mutex> side_lock;
  if (!ckv) {
    side = side_stream();
    if (side) {
      side_lock = std::unique_lock<std::mutex>(side->mu);
      DIT_HIP(hipEventRecord(side->fork, s), "hipEventRecord");
      DIT_HIP(hipStreamWaitEvent(side->stream, side->fork, 0), "hipStreamWaitEvent");
      DIT_TRY(text_kv_impl(c, w, L, req_txt, txt, ws.ckv, side->stream));
      DIT_HIP(hipEventRecord(side->join, side->stream), "hipEventRecord");
    } else {
      DIT_TRY(text_kv_impl(c, w, L, req_txt, txt, ws.ckv, s));
    }
    ckv = ws.ckv;
  }
  // x1 = x + gate_sa (o W_o^T + b_o)
  DIT_TRY(run_linear(o, D, w->w_o, D, w->b_o, ws.x1, D, T, D, D, DIT_EPI_GATED_RESIDUAL, x, D, mod + 2 * D, 6 * D,
                     req, dt, s, "output projection"));
  // hc = LN(x1) g_ca + b_ca ; cq = RMS(hc W_cq^T + b_cq)
  DIT_TRY(run_ln_affine(ws.x1, w->g_ca, w->b_ca, T, D, c->ln_eps, ws.h, dt, s));
  DIT_TRY(run_linear(ws.h, D, w->w_cq, D, w->b_cq, ws.cq, D, T, D, D, DIT_EPI_NONE, nullptr, 0, nullptr, 0, req, dt,
                     s, "cross query projection"));
  // bf16: the RMSNorm of cq happens as the cross-attention loads it
  const bool cq_norm_in_attn = c->qk_norm && dt == DIT_BF16;
  if (c->qk_norm && !cq_norm_in_attn) {
    const int zero[3] = {0, 0, 0};
    DIT_TRY(run_norm_rope(ws.cq, nullptr, D, T, c->n_heads, c->head_dim, w->g_cq, nullptr, c->rms_eps, zero, 0.f,
                          nullptr, dt, s));
  }
  if (side) DIT_HIP(hipStreamWaitEvent(s, side->join, 0), "hipStreamWaitEvent");
  // oc = cross attention (queries: the request's latent rows, keys: its text rows)
  DIT_TRY(run_attention(ws.cq, ckv, ckv + D * es, ws.o, D, 2 * D, 2 * D, D, req, req_txt, c->n_heads,
                        c->head_dim, 1.0f / sqrtf((float)c->head_dim), dt, s,
                        cq_norm_in_attn ? w->g_cq : nullptr, c->rms_eps));
  // x2 = x1 + (oc W_co^T + b_co), in place in x1
  DIT_TRY(run_linear(ws.o, D, w->w_co, D, w->b_co, ws.x1, D, T, D, D, DIT_EPI_RESIDUAL, ws.x1, D, nullptr, 0, req,
                     dt, s, "cross output projection"));
  // h2 = LN(x2)(1+scale_ff)+shift_ff ; u = gelu(h2 W_up^T + b_up) ; y = x2 + gate_ff (u W_dn^T + b_dn)
  DIT_TRY(run_ln_mod(ws.x1, mod + 3 * D, mod + 4 * D, 6 * D, req, T, D, c->ln_eps, ws.h, dt, s));
  DIT_TRY(run_linear(ws.h, D, w->w_up, D, w->b_up, ws.u, Dff, T, Dff, D, DIT_EPI_GELU_TANH, nullptr, 0, nullptr, 0,
                     req, dt, s, "mlp up projection"));
  DIT_TRY(run_linear(ws.u, Dff, w->w_dn, Dff, w->b_dn, y, D, T, D, Dff, DIT_EPI_GATED_RESIDUAL, ws.x1, D,
                     mod + 5 * D, 6 * D, req, dt, s, "mlp down projection"));
  return DIT_OK;
}

// The bf16 attention numbers its work items (128- or 256-query tiles x
// heads) in int and splits them over the XCDs with products that must stay
// below 2^31: at most 2^26 256-query tiles (so 2^27 of 128 queries).
dit_status check_attn_items(const int32_t* cu, int n_req, int n_heads) {
  int64_t items = 0;
  for (int r = 0; r < n_req; ++r) items += (int64_t)(cu[r + 1] - cu[r] + 255) / 256 * n_heads;
  if (items > (1 << 26))
    return fail(DIT_ERR_UNSUPPORTED, "attention of %lld work items (at most 2^26 256-query tiles x heads)",
                (long long)items);
  return DIT_OK;
}

dit_status check_block_call(const dit_block_config* c, const dit_block_weights* w, const dit_varlen* vl, bool pre,
                            bool post, bool cond = true) {
  DIT_TRY(check_cfg(c));
  DIT_TRY(check_weights(c, w, pre, post, cond, cond));
  DIT_TRY(check_varlen(vl, post));
  DIT_TRY(check_attn_items(vl->cu_seqlens, vl->n_req, c->n_heads));
  if (pre) {
    RopeTable tab;
    DIT_TRY(check_rope_table(vl, c->rope_sections, &tab));
  }
  return DIT_OK;
}


// ------------------------------------------------------------ denoising step

int patch_len(const dit_model_config* m) { return m->in_channels * m->patch[0] * m->patch[1] * m->patch[2]; }

dit_status check_model_cfg(const dit_model_config* m) {
  if (!m) return fail(DIT_ERR_INVALID_ARG, "model config is NULL");
  DIT_TRY(check_cfg(&m->block));
  if (m->n_blocks < 1) return fail(DIT_ERR_INVALID_ARG, "n_blocks = %d", m->n_blocks);
  if (m->in_channels < 1 || m->patch[0] < 1 || m->patch[1] < 1 || m->patch[2] < 1)
    return fail(DIT_ERR_INVALID_ARG, "in_channels %d, patch (%d,%d,%d) must be >= 1", m->in_channels, m->patch[0],
                m->patch[1], m->patch[2]);
  const int64_t P = (int64_t)m->in_channels * m->patch[0] * m->patch[1] * m->patch[2];
  if (P > 8192) return fail(DIT_ERR_UNSUPPORTED, "patch vector of %lld values (at most 8192)", (long long)P);
  if (m->block.dtype == DIT_BF16 && P % 64)
    return fail(DIT_ERR_UNSUPPORTED, "bf16 needs C*pt*ph*pw %% 64 == 0 (it is %lld)", (long long)P);
  if (m->block.dtype == DIT_F32 && P % 4)
    return fail(DIT_ERR_UNSUPPORTED, "fp32 needs C*pt*ph*pw %% 4 == 0 (it is %lld)", (long long)P);
  return DIT_OK;
}

// Whole requests only; fills the latent geometry.
dit_status check_model_varlen(const dit_model_config* m, const dit_varlen* vl, LatentTable* tab) {
  DIT_TRY(check_varlen(vl, true));
  if (!vl->grid_fhw) return fail(DIT_ERR_INVALID_ARG, "grid_fhw is NULL");
  memset(tab, 0, sizeof(*tab));
  tab->n_req = vl->n_req;
  tab->C = m->in_channels;
  tab->pt = m->patch[0]; tab->ph = m->patch[1]; tab->pw = m->patch[2];
  const int64_t P = patch_len(m);
  // tiles of about 2048 patch values (the latent kernels' LDS transpose)
  int max_w = 1;
  for (int r = 0; r < vl->n_req; ++r) max_w = vl->grid_fhw[3 * r + 2] > max_w ? vl->grid_fhw[3 * r + 2] : max_w;
  tab->wt = (int)(2048 / P) < 1 ? 1 : (int)(2048 / P);
  if (tab->wt > max_w) tab->wt = max_w;
  for (int r = 0; r < vl->n_req; ++r) {
    const int F = vl->grid_fhw[3 * r], H = vl->grid_fhw[3 * r + 1], W = vl->grid_fhw[3 * r + 2];
    if (F < 1 || H < 1 || W < 1) return fail(DIT_ERR_INVALID_ARG, "grid of request %d is (%d,%d,%d)", r, F, H, W);
    const int64_t cells = (int64_t)F * H * W;
    const int rows = vl->cu_seqlens[r + 1] - vl->cu_seqlens[r];
    if (cells != rows)
      return fail(DIT_ERR_INVALID_ARG, "request %d has %d rows, its whole grid has %lld tokens", r, rows,
                  (long long)cells);
    if (vl->pos_offset && vl->pos_offset[r] != 0)
      return fail(DIT_ERR_INVALID_ARG, "request %d: pos_offset %d (the step needs whole requests)", r,
                  vl->pos_offset[r]);
    tab->lat_off[r + 1] = tab->lat_off[r] + cells * P;
    const int64_t tiles = tab->tile_off[r] + (int64_t)F * H * ((W + tab->wt - 1) / tab->wt);
    if (tiles > 0x7FFFFFFF) return fail(DIT_ERR_UNSUPPORTED, "latent of %lld tiles", (long long)tiles);
    tab->tile_off[r + 1] = (int)tiles;
    tab->row0[r] = vl->cu_seqlens[r];
    tab->grid_h[r] = H;
    tab->grid_w[r] = W;
  }
  return DIT_OK;
}

dit_status check_model_weights(const dit_model_config* m, const dit_model_weights* w) {
  if (!w) return fail(DIT_ERR_INVALID_ARG, "model weights is NULL");
  DIT_TRY(check_ptr(w->w_t1, "w_t1")); DIT_TRY(check_ptr(w->b_t1, "b_t1"));
  DIT_TRY(check_ptr(w->w_t2, "w_t2")); DIT_TRY(check_ptr(w->b_t2, "b_t2"));
  DIT_TRY(check_ptr(w->w_pe, "w_pe")); DIT_TRY(check_ptr(w->b_pe, "b_pe"));
  DIT_TRY(check_ptr(w->w_hmod, "w_hmod")); DIT_TRY(check_ptr(w->b_hmod, "b_hmod"));
  DIT_TRY(check_ptr(w->w_out, "w_out")); DIT_TRY(check_ptr(w->b_out, "b_out"));
  if (!w->blocks) return fail(DIT_ERR_INVALID_ARG, "blocks is NULL");
  for (int b = 0; b < m->n_blocks; ++b) {
    const dit_status st = check_weights(&m->block, &w->blocks[b], true, true, false);
    if (st != DIT_OK) return fail(st, "block %d: %s", b, g_last_error.c_str());
  }
  return DIT_OK;
}

struct ModelWorkspace {
  char *x, *tok;
  Workspace blk;
};

// x [rows, D] (the residual stream), tok [rows, P] (patch vectors, then the
// velocity), then a block workspace without text keys/values (they are cached).
size_t model_layout(const dit_model_config* m, const dit_varlen* vl, char* base, ModelWorkspace* ws) {
  const size_t es = elem_size(m->block.dtype);
  const size_t T = vl->cu_seqlens[vl->n_req];
  size_t off = 0;
  ModelWorkspace w;
  w.x = base ? base + off : nullptr;
  off += round256(T * m->block.hidden * es);
  w.tok = base ? base + off : nullptr;
  off += round256(T * patch_len(m) * es);
  dit_varlen no_txt = *vl;
  no_txt.cu_seqlens_txt = nullptr;
  off += layout(&m->block, &no_txt, base ? base + off : nullptr, &w.blk);
  if (ws) *ws = w;
  return off;
}

dit_status run_latent(bool euler, const dit_model_config* m, const LatentTable& tab, const float* latent,
                      void* tokens, const float* dt, float* out, hipStream_t s) {
  LatentArgs p;
  p.latent = latent; p.tokens = tokens; p.dt = dt; p.latent_out = out; p.tab = tab; p.dtype = m->block.dtype;
  return euler ? hip_status(launch_unpatchify_euler(p, s), "unpatchify + Euler update")
               : hip_status(launch_patchify(p, s), "patchify");
}

// The conditioning chain with explicit parts (see CondArgs).
dit_status run_cond_parts(const dit_block_config* c, int n_req, const float* t, const void* w_t1, const void* b_t1,
                          const void* w_t2, const void* b_t2, const void* w_mod, const void* b_mod, int n_mod,
                          float* mod, const Workspace& ws, hipStream_t s, const char* what) {
  CondArgs p;
  p.t = t; p.n_req = n_req; p.freq_dim = c->freq_dim; p.hidden = c->hidden;
  p.w_t1 = w_t1; p.b_t1 = b_t1; p.w_t2 = w_t2; p.b_t2 = b_t2; p.w_ada = w_mod; p.b_ada = b_mod; p.n_mod = n_mod;
  p.e = ws.e; p.a1 = ws.a1; p.c = ws.c; p.mod = mod; p.dtype = c->dtype;
  return hip_status(launch_conditioning(p, s), what);
}

}  // namespace

// Scratch of dit_timestep_modulation_noalloc: one array per GPU, held until
// the process ends.  Host code never uses the name `scratch` as an address
// (on the host it is a stand-in, not device memory); it uses the device
// address looked up with hipGetSymbolAddress, once per device.
static __device__ __align__(256) char scratch[DIT_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array (looked up on the
// first call on that device, with that device current).
dit_status scratch_address(void** out) {
  int dev = -1;
  DIT_HIP(hipGetDevice(&dev), "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(DIT_ERR_UNSUPPORTED, "device %d (at most %d devices)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    DIT_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (!p) return fail(DIT_ERR_HIP, "hipGetSymbolAddress(scratch) gave NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return DIT_OK;
}

// Checks shared by both conditioning entry points; the scratch layout is
// e [R,F], a1 [R,D], c [R,D], each 256-byte aligned.
dit_status check_modulation_call(const dit_block_config* cfg, const dit_block_weights* w, int n_req, const float* t,
                                 float* mod) {
  DIT_TRY(check_cfg(cfg));
  DIT_TRY(check_cond_weights(w));
  if (n_req < 1 || n_req > DIT_MAX_REQ) return fail(DIT_ERR_INVALID_ARG, "n_req = %d outside 1..%d", n_req, DIT_MAX_REQ);
  DIT_TRY(check_ptr(t, "t"));
  DIT_TRY(check_ptr(mod, "mod"));
  return DIT_OK;
}

size_t modulation_scratch_bytes(const dit_block_config* cfg, int n_req) {
  return round256((size_t)cfg->freq_dim * n_req * 4) + 2 * round256((size_t)cfg->hidden * n_req * 4);
}

dit_status run_modulation(const dit_block_config* cfg, const dit_block_weights* w, int n_req, const float* t,
                          float* mod, char* p, hipStream_t stream) {
  float* e = (float*)p;
  p += round256((size_t)cfg->freq_dim * n_req * 4);
  float* a1 = (float*)p;
  p += round256((size_t)cfg->hidden * n_req * 4);
  float* cc = (float*)p;
  return run_cond(cfg, w, n_req, t, mod, e, a1, cc, stream);
}

}  // namespace

namespace dit {
// Sets this thread's dit_last_error() message (used by the other C-ABI units).
void set_last_error(const std::string& msg) { g_last_error = msg; }
}  // namespace dit

extern "C" {

int dit_abi_version(void) { return DIT_ABI_VERSION; }

const char* dit_status_string(dit_status s) {
  switch (s) {
    case DIT_OK: return "ok";
    case DIT_ERR_INVALID_ARG: return "invalid argument";
    case DIT_ERR_UNSUPPORTED: return "unsupported shape or type";
    case DIT_ERR_WORKSPACE: return "workspace too small";
    case DIT_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* dit_last_error(void) { return g_last_error.c_str(); }

size_t dit_block_workspace_size(const dit_block_config* cfg, const dit_varlen* vl) {
  if (check_cfg(cfg) != DIT_OK || check_varlen(vl, true) != DIT_OK) return 0;
  return layout(cfg, vl, nullptr, nullptr);
}

dit_status dit_block_forward(const dit_block_config* cfg, const dit_block_weights* w, const dit_varlen* vl,
                             const void* x, const float* t, const float* mod, const void* txt, void* y, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_block_call(cfg, w, vl, true, true, mod == nullptr));
  DIT_TRY(check_ptr(x, "x"));
  if (mod) DIT_TRY(check_ptr(mod, "mod"));
  else DIT_TRY(check_ptr(t, "t"));
  DIT_TRY(check_ptr(txt, "txt"));
  DIT_TRY(check_ptr(y, "y"));
  Workspace W;
  DIT_TRY(check_ws(cfg, vl, ws, ws_bytes, &W));
  // The text keys and values depend on txt and the weights only: on the side
  // stream from the start, beside the conditioning, LayerNorm and QKV
  // projection, joined before the cross-attention.
  SideStream* side = side_stream();
  std::unique_lock<std::mutex> side_lock;
  if (side) {
    const int64_t L = vl->cu_seqlens_txt[vl->n_req];
    side_lock = std::unique_lock<std::mutex>(side->mu);
    DIT_HIP(hipEventRecord(side->fork, stream), "hipEventRecord");
    DIT_HIP(hipStreamWaitEvent(side->stream, side->fork, 0), "hipStreamWaitEvent");
    DIT_TRY(text_kv_impl(cfg, w, L, make_req(vl->cu_seqlens_txt, vl->n_req), txt, W.ckv, side->stream));
    DIT_HIP(hipEventRecord(side->join, side->stream), "hipEventRecord");
  }
  const float* m = mod;
  if (!m) {
    DIT_TRY(run_cond(cfg, w, vl->n_req, t, W.mod, W.e, W.a1, W.c, stream));
    m = W.mod;
  }
  DIT_TRY(pre_attention_impl(cfg, w, vl, x, m, W.qkv, W, stream));
  DIT_TRY(self_attention_impl(cfg, vl, W.qkv, W.o, stream));
  return post_attention_impl(cfg, w, vl, x, W.o, txt, m, y, W, stream, side ? W.ckv : nullptr, side);
}

dit_status dit_block_pre_attention(const dit_block_config* cfg, const dit_block_weights* w, const dit_varlen* vl,
                                   const void* x, const float* t, float* mod, void* qkv, void* ws, size_t ws_bytes,
                                   hipStream_t stream) {
  g_last_error.clear();
  // with t: mod is written from the block's timestep MLP; without: mod is read
  DIT_TRY(check_block_call(cfg, w, vl, true, false, t != nullptr));
  DIT_TRY(check_ptr(x, "x"));
  DIT_TRY(check_ptr(t, "t", true));
  DIT_TRY(check_ptr(mod, "mod"));
  DIT_TRY(check_ptr(qkv, "qkv"));
  Workspace W;
  DIT_TRY(check_ws(cfg, vl, ws, ws_bytes, &W));
  if (t) DIT_TRY(run_cond(cfg, w, vl->n_req, t, mod, W.e, W.a1, W.c, stream));
  return pre_attention_impl(cfg, w, vl, x, mod, qkv, W, stream);
}

dit_status dit_block_post_attention(const dit_block_config* cfg, const dit_block_weights* w, const dit_varlen* vl,
                                    const void* x, const void* o, const void* txt, const float* t, const float* mod,
                                    void* y, void* ws, size_t ws_bytes, hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_block_call(cfg, w, vl, false, true));
  // without mod the modulation comes from t through the block's timestep MLP
  if (!mod) DIT_TRY(check_cond_weights(w));
  DIT_TRY(check_ptr(x, "x"));
  DIT_TRY(check_ptr(o, "o"));
  DIT_TRY(check_ptr(txt, "txt"));
  if (mod) DIT_TRY(check_ptr(mod, "mod"));
  else DIT_TRY(check_ptr(t, "t"));
  DIT_TRY(check_ptr(y, "y"));
  Workspace W;
  DIT_TRY(check_ws(cfg, vl, ws, ws_bytes, &W));
  const float* m = mod;
  if (!m) {
    DIT_TRY(run_cond(cfg, w, vl->n_req, t, W.mod, W.e, W.a1, W.c, stream));
    m = W.mod;
  }
  return post_attention_impl(cfg, w, vl, x, o, txt, m, y, W, stream);
}

dit_status dit_timestep_modulation(const dit_block_config* cfg, const dit_block_weights* w, int n_req,
                                   const float* t, float* mod, void* ws, size_t ws_bytes, hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_modulation_call(cfg, w, n_req, t, mod));
  const size_t need = modulation_scratch_bytes(cfg, n_req);
  if (!ws || ((uintptr_t)ws & 255u)) return fail(DIT_ERR_WORKSPACE, "workspace NULL or not 256-byte aligned");
  if (ws_bytes < need) return fail(DIT_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, need);
  return run_modulation(cfg, w, n_req, t, mod, (char*)ws, stream);
}

dit_status dit_debug_gemm_tile_n(int tile_n) {
  g_last_error.clear();
  if (tile_n != 0 && tile_n != 192 && tile_n != 256)
    return fail(DIT_ERR_INVALID_ARG, "GEMM tile width %d (0, 192 or 256)", tile_n);
  set_gemm_tile_n(tile_n);
  return DIT_OK;
}

dit_status dit_debug_attention_split(int mode) {
  g_last_error.clear();
  if (mode != 0 && mode != 1 && mode != 2 && mode != 4)
    return fail(DIT_ERR_INVALID_ARG, "attention split mode %d (0, 1, 2 or 4)", mode);
  set_attention_split(mode);
  return DIT_OK;
}

dit_status dit_debug_attention_shape(int waves) {
  g_last_error.clear();
  if (waves != 0 && waves != 4 && waves != 8)
    return fail(DIT_ERR_INVALID_ARG, "attention shape of %d waves (0, 4 or 8)", waves);
  set_attention_shape(waves);
  return DIT_OK;
}

dit_status dit_debug_attention_plan(const int32_t* cu_q, const int32_t* cu_k, int n_req, int n_heads,
                                    int compute_units, int* waves, int* split_pieces, int* split_items) {
  g_last_error.clear();
  DIT_TRY(check_cu(cu_q, n_req, "cu_q"));
  DIT_TRY(check_cu(cu_k, n_req, "cu_k"));
  if (n_heads < 1) return fail(DIT_ERR_INVALID_ARG, "n_heads = %d", n_heads);
  if (compute_units < 1 || compute_units > 65536)
    return fail(DIT_ERR_INVALID_ARG, "compute_units = %d outside 1..65536", compute_units);
  if (!waves || !split_pieces || !split_items) return fail(DIT_ERR_INVALID_ARG, "an output pointer is NULL");
  DIT_TRY(check_attn_items(cu_q, n_req, n_heads));
  const AttnPlan pl = attention_plan(cu_q, cu_k, n_req, n_heads, compute_units);
  *waves = pl.waves;
  *split_pieces = pl.split_pieces;
  *split_items = pl.split_items;
  return DIT_OK;
}

dit_status dit_timestep_modulation_noalloc(const dit_block_config* cfg, const dit_block_weights* w, int n_req,
                                           const float* t, float* mod, hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_modulation_call(cfg, w, n_req, t, mod));
  const size_t need = modulation_scratch_bytes(cfg, n_req);
  if (need > DIT_NOALLOC_SCRATCH_BYTES)
    return fail(DIT_ERR_UNSUPPORTED, "scratch of %zu bytes needed, the static array holds %zu", need,
                (size_t)DIT_NOALLOC_SCRATCH_BYTES);
  void* p = nullptr;
  DIT_TRY(scratch_address(&p));
  return run_modulation(cfg, w, n_req, t, mod, (char*)p, stream);
}

dit_status dit_attention_varlen(const void* q, const void* k, const void* v, void* o, int64_t q_row_stride,
                                int64_t k_row_stride, int64_t v_row_stride, int64_t o_row_stride,
                                const int32_t* cu_q, const int32_t* cu_k, int n_req, int n_heads, int head_dim,
                                float softmax_scale, dit_dtype dtype, hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_dtype(dtype));
  DIT_TRY(check_ptr(q, "q")); DIT_TRY(check_ptr(k, "k")); DIT_TRY(check_ptr(v, "v")); DIT_TRY(check_ptr(o, "o"));
  DIT_TRY(check_cu(cu_q, n_req, "cu_q"));
  DIT_TRY(check_cu(cu_k, n_req, "cu_k"));
  if (n_heads < 1) return fail(DIT_ERR_INVALID_ARG, "n_heads = %d", n_heads);
  if (!isfinite(softmax_scale)) return fail(DIT_ERR_INVALID_ARG, "softmax_scale is not finite");
  if (dtype == DIT_BF16 && head_dim != 128) return fail(DIT_ERR_UNSUPPORTED, "bf16 attention head_dim %d (only 128)", head_dim);
  if (dtype == DIT_F32 && head_dim != 64 && head_dim != 128)
    return fail(DIT_ERR_UNSUPPORTED, "fp32 attention head_dim %d (64 or 128)", head_dim);
  // 0 selects the standard scale 1/sqrt(head_dim)
  const float scale = softmax_scale == 0.f ? 1.0f / sqrtf((float)head_dim) : softmax_scale;
  const int64_t width = (int64_t)n_heads * head_dim;
  const int64_t vec = dtype == DIT_BF16 ? 8 : 4;
  const int64_t strides[4] = {q_row_stride, k_row_stride, v_row_stride, o_row_stride};
  for (int i = 0; i < 4; ++i)
    if (strides[i] < width || strides[i] % vec)
      return fail(DIT_ERR_INVALID_ARG, "row stride %lld: must be >= n_heads*head_dim = %lld and a multiple of %lld",
                  (long long)strides[i], (long long)width, (long long)vec);
  // the bf16 kernel forms a key tile's offsets (64 rows of k or v) in 32 bits
  if (dtype == DIT_BF16 && (k_row_stride > (int64_t)1 << 24 || v_row_stride > (int64_t)1 << 24))
    return fail(DIT_ERR_INVALID_ARG, "k/v row stride %lld / %lld: at most %lld elements for bf16",
                (long long)k_row_stride, (long long)v_row_stride, (long long)1 << 24);
  // o is written while q, k and v are still being read: its byte range must
  // not meet theirs (ranges from the first to the last byte a row touches)
  const int64_t es = (int64_t)elem_size(dtype);
  const Span so = span(o, cu_q[n_req], o_row_stride, width, es);
  const Span in[3] = {span(q, cu_q[n_req], q_row_stride, width, es), span(k, cu_k[n_req], k_row_stride, width, es),
                      span(v, cu_k[n_req], v_row_stride, width, es)};
  const char* names[3] = {"q", "k", "v"};
  for (int i = 0; i < 3; ++i)
    if (overlaps(so, in[i])) return fail(DIT_ERR_INVALID_ARG, "o overlaps %s", names[i]);
  DIT_TRY(check_attn_items(cu_q, n_req, n_heads));
  return run_attention(q, k, v, o, q_row_stride, k_row_stride, v_row_stride, o_row_stride, make_req(cu_q, n_req),
                       make_req(cu_k, n_req), n_heads, head_dim, scale, dtype, stream);
}

dit_status dit_adaln_modulate(const void* x, const float* shift, const float* scale, int64_t mod_stride,
                              const int32_t* cu_seqlens, int n_req, int hidden, float eps, void* out,
                              dit_dtype dtype, hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_dtype(dtype));
  DIT_TRY(check_ptr(x, "x")); DIT_TRY(check_ptr(shift, "shift")); DIT_TRY(check_ptr(scale, "scale"));
  DIT_TRY(check_ptr(out, "out"));
  DIT_TRY(check_cu(cu_seqlens, n_req, "cu_seqlens"));
  const int vec = dtype == DIT_BF16 ? 8 : 4;
  if (hidden < vec || hidden % vec) return fail(DIT_ERR_INVALID_ARG, "hidden %d must be a positive multiple of %d", hidden, vec);
  if (hidden > (dtype == DIT_BF16 ? 8192 : 4096)) return fail(DIT_ERR_UNSUPPORTED, "hidden %d too large", hidden);
  if (mod_stride < 0 || mod_stride % 4) return fail(DIT_ERR_INVALID_ARG, "mod_stride %lld must be a multiple of 4 and >= 0", (long long)mod_stride);
  if (!(eps > 0.f)) return fail(DIT_ERR_INVALID_ARG, "eps must be > 0");
  return run_ln_mod(x, shift, scale, mod_stride, make_req(cu_seqlens, n_req), cu_seqlens[n_req], hidden, eps, out,
                    dtype, stream);
}

dit_status dit_layer_norm_affine(const void* x, const void* gamma, const void* beta, int64_t n_rows, int hidden,
                                 float eps, void* out, dit_dtype dtype, hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_dtype(dtype));
  DIT_TRY(check_ptr(x, "x")); DIT_TRY(check_ptr(gamma, "gamma")); DIT_TRY(check_ptr(beta, "beta"));
  DIT_TRY(check_ptr(out, "out"));
  if (n_rows < 0 || n_rows > 0x7FFFFFFF) return fail(DIT_ERR_INVALID_ARG, "n_rows %lld", (long long)n_rows);
  const int vec = dtype == DIT_BF16 ? 8 : 4;
  if (hidden < vec || hidden % vec) return fail(DIT_ERR_INVALID_ARG, "hidden %d must be a positive multiple of %d", hidden, vec);
  if (hidden > (dtype == DIT_BF16 ? 8192 : 4096)) return fail(DIT_ERR_UNSUPPORTED, "hidden %d too large", hidden);
  if (!(eps > 0.f)) return fail(DIT_ERR_INVALID_ARG, "eps must be > 0");
  return run_ln_affine(x, gamma, beta, n_rows, hidden, eps, out, dtype, stream);
}

dit_status dit_linear(const void* a, int64_t lda, const void* w, int64_t ldw, const void* bias, void* out, int64_t ldo,
                      int64_t M, int N, int K, dit_epilogue epi, const void* res, int64_t ldr, const float* gate,
                      int64_t gate_stride, const int32_t* cu_seqlens, int n_req, dit_dtype dtype,
                      hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_dtype(dtype));
  DIT_TRY(check_ptr(a, "a")); DIT_TRY(check_ptr(w, "w")); DIT_TRY(check_ptr(out, "out"));
  DIT_TRY(check_ptr(bias, "bias", true));
  if (M < 0 || M > 0x7FFFFFFF || N < 1 || K < 1) return fail(DIT_ERR_INVALID_ARG, "bad GEMM size M=%lld N=%d K=%d", (long long)M, N, K);
  if (epi < DIT_EPI_NONE || epi > DIT_EPI_GATED_RESIDUAL) return fail(DIT_ERR_INVALID_ARG, "epilogue %d", (int)epi);
  const int64_t vec = dtype == DIT_BF16 ? 8 : 4;
  if (lda < K || ldw < K || ldo < N || lda % vec || ldw % vec || ldo % vec)
    return fail(DIT_ERR_INVALID_ARG, "leading dimensions must cover the row and be multiples of %lld", (long long)vec);
  if (dtype == DIT_BF16 && (K % 64 || N % 8)) return fail(DIT_ERR_UNSUPPORTED, "bf16 GEMM needs K %% 64 == 0 and N %% 8 == 0 (K=%d N=%d)", K, N);
  if (dtype == DIT_F32 && N % 4) return fail(DIT_ERR_UNSUPPORTED, "fp32 GEMM needs N %% 4 == 0");
  ReqTable req = single_req(M);
  if (epi == DIT_EPI_RESIDUAL || epi == DIT_EPI_GATED_RESIDUAL) {
    DIT_TRY(check_ptr(res, "res"));
    if (ldr < N || ldr % vec) return fail(DIT_ERR_INVALID_ARG, "ldr %lld", (long long)ldr);
  }
  if (epi == DIT_EPI_GATED_RESIDUAL) {
    DIT_TRY(check_ptr(gate, "gate"));
    if (gate_stride < 0 || gate_stride % 4) return fail(DIT_ERR_INVALID_ARG, "gate_stride %lld", (long long)gate_stride);
    DIT_TRY(check_cu(cu_seqlens, n_req, "cu_seqlens"));
    if (cu_seqlens[n_req] != M) return fail(DIT_ERR_INVALID_ARG, "cu_seqlens ends at %d, M is %lld", cu_seqlens[n_req], (long long)M);
    req = make_req(cu_seqlens, n_req);
  }
  return run_linear(a, lda, w, ldw, bias, out, ldo, M, N, K, epi, res, ldr, gate, gate_stride, req, dtype, stream,
                    "linear");
}

dit_status dit_qk_norm_rope(void* q, void* k, int64_t row_stride, int64_t n_rows, int n_heads, int head_dim,
                            const void* g_q, const void* g_k, float eps, const int rope_sections[3], float rope_theta,
                            const dit_varlen* vl, dit_dtype dtype, hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_dtype(dtype));
  DIT_TRY(check_ptr(q, "q")); DIT_TRY(check_ptr(k, "k", true));
  DIT_TRY(check_ptr(g_q, "g_q", true)); DIT_TRY(check_ptr(g_k, "g_k", true));
  if (k && !g_k && g_q) return fail(DIT_ERR_INVALID_ARG, "g_k is NULL while g_q is set");
  if (head_dim != 64 && head_dim != 128) return fail(DIT_ERR_UNSUPPORTED, "head_dim %d (64 or 128)", head_dim);
  if (n_heads < 1) return fail(DIT_ERR_INVALID_ARG, "n_heads %d", n_heads);
  const int64_t vec = dtype == DIT_BF16 ? 8 : 4;
  if (row_stride < (int64_t)n_heads * head_dim || row_stride % vec) return fail(DIT_ERR_INVALID_ARG, "row_stride %lld", (long long)row_stride);
  if (!(eps > 0.f)) return fail(DIT_ERR_INVALID_ARG, "eps must be > 0");
  const int zero[3] = {0, 0, 0};
  const int* sec = rope_sections ? rope_sections : zero;
  DIT_TRY(check_sections(sec, head_dim));
  RopeTable tab;
  const RopeTable* tp = nullptr;
  if (vl && rope_on(sec)) {
    if (!(rope_theta > 0.f)) return fail(DIT_ERR_INVALID_ARG, "rope_theta must be > 0");
    DIT_TRY(check_varlen(vl, false));
    DIT_TRY(check_rope_table(vl, sec, &tab));
    if (n_rows != vl->cu_seqlens[vl->n_req]) return fail(DIT_ERR_INVALID_ARG, "n_rows %lld != cu_seqlens[n_req] %d", (long long)n_rows, vl->cu_seqlens[vl->n_req]);
    tp = &tab;
  }
  if (n_rows < 0 || n_rows > 0x7FFFFFFF) return fail(DIT_ERR_INVALID_ARG, "n_rows %lld", (long long)n_rows);
  return run_norm_rope(q, k, row_stride, n_rows, n_heads, head_dim, g_q, k ? g_k : nullptr, eps, sec, rope_theta, tp,
                       dtype, stream);
}

dit_status dit_gated_residual(const void* x, const void* z, const void* bias, const float* gate, int64_t gate_stride,
                              const int32_t* cu_seqlens, int n_req, int hidden, void* out, dit_dtype dtype,
                              hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_dtype(dtype));
  DIT_TRY(check_ptr(x, "x")); DIT_TRY(check_ptr(z, "z")); DIT_TRY(check_ptr(bias, "bias", true));
  DIT_TRY(check_ptr(gate, "gate")); DIT_TRY(check_ptr(out, "out"));
  DIT_TRY(check_cu(cu_seqlens, n_req, "cu_seqlens"));
  const int vec = dtype == DIT_BF16 ? 8 : 4;
  if (hidden < vec || hidden % vec) return fail(DIT_ERR_INVALID_ARG, "hidden %d must be a positive multiple of %d", hidden, vec);
  if (hidden > (dtype == DIT_BF16 ? 8192 : 4096)) return fail(DIT_ERR_UNSUPPORTED, "hidden %d too large", hidden);
  if (gate_stride < 0 || gate_stride % 4) return fail(DIT_ERR_INVALID_ARG, "gate_stride %lld", (long long)gate_stride);
  GatedResArgs p;
  p.x = x; p.z = z; p.bias = bias; p.gate = gate; p.gate_stride = gate_stride; p.out = out;
  p.n_rows = cu_seqlens[n_req]; p.hidden = hidden; p.req = make_req(cu_seqlens, n_req); p.dtype = dtype;
  return hip_status(launch_gated_residual(p, stream), "gated_residual");
}

size_t dit_text_kv_elems(const dit_model_config* cfg, const dit_varlen* vl) {
  if (check_model_cfg(cfg) != DIT_OK || check_varlen(vl, true) != DIT_OK) return 0;
  return (size_t)cfg->n_blocks * vl->cu_seqlens_txt[vl->n_req] * 2 * cfg->block.hidden;
}

dit_status dit_text_kv(const dit_model_config* cfg, const dit_model_weights* w, const dit_varlen* vl,
                       const void* txt, void* kv, hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_model_cfg(cfg));
  DIT_TRY(check_varlen(vl, true));
  if (!w || !w->blocks) return fail(DIT_ERR_INVALID_ARG, "model weights or their blocks are NULL");
  const dit_block_config* c = &cfg->block;
  for (int b = 0; b < cfg->n_blocks; ++b) {
    const dit_block_weights* bw = &w->blocks[b];
    if (check_ptr(bw->w_ckv, "w_ckv") != DIT_OK || check_ptr(bw->b_ckv, "b_ckv") != DIT_OK ||
        check_ptr(bw->g_ck, "g_ck", !c->qk_norm) != DIT_OK)
      return fail(DIT_ERR_INVALID_ARG, "block %d: %s", b, g_last_error.c_str());
  }
  DIT_TRY(check_ptr(txt, "txt"));
  DIT_TRY(check_ptr(kv, "kv"));
  const int64_t L = vl->cu_seqlens_txt[vl->n_req];
  const ReqTable req_txt = make_req(vl->cu_seqlens_txt, vl->n_req);
  const size_t per_block = (size_t)L * 2 * c->hidden * elem_size(c->dtype);
  for (int b = 0; b < cfg->n_blocks; ++b)
    DIT_TRY(text_kv_impl(c, &w->blocks[b], L, req_txt, txt, (char*)kv + b * per_block, stream));
  return DIT_OK;
}

size_t dit_denoise_workspace_size(const dit_model_config* cfg, const dit_varlen* vl) {
  LatentTable tab;
  if (check_model_cfg(cfg) != DIT_OK || check_model_varlen(cfg, vl, &tab) != DIT_OK) return 0;
  return model_layout(cfg, vl, nullptr, nullptr);
}

dit_status dit_denoise_step(const dit_model_config* cfg, const dit_model_weights* w, const dit_varlen* vl,
                            const float* latent, const float* t, const float* dt, const void* kv, float* latent_out,
                            void* ws, size_t ws_bytes, hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_model_cfg(cfg));
  LatentTable tab;
  DIT_TRY(check_model_varlen(cfg, vl, &tab));
  DIT_TRY(check_model_weights(cfg, w));
  const dit_block_config* c = &cfg->block;
  RopeTable rope;
  DIT_TRY(check_rope_table(vl, c->rope_sections, &rope));
  DIT_TRY(check_attn_items(vl->cu_seqlens, vl->n_req, c->n_heads));
  DIT_TRY(check_ptr(latent, "latent")); DIT_TRY(check_ptr(t, "t")); DIT_TRY(check_ptr(dt, "dt"));
  DIT_TRY(check_ptr(kv, "kv")); DIT_TRY(check_ptr(latent_out, "latent_out"));
  const size_t need = model_layout(cfg, vl, nullptr, nullptr);
  if (!ws) return fail(DIT_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if (((uintptr_t)ws & 255u) != 0) return fail(DIT_ERR_WORKSPACE, "workspace is not 256-byte aligned");
  if (ws_bytes < need) return fail(DIT_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, need);
  ModelWorkspace W;
  model_layout(cfg, vl, (char*)ws, &W);

  const int D = c->hidden, P = patch_len(cfg), R = vl->n_req;
  const int64_t T = vl->cu_seqlens[R], L = vl->cu_seqlens_txt[R];
  const size_t es = elem_size(c->dtype);
  const dit_dtype dty = c->dtype;
  const ReqTable req = make_req(vl->cu_seqlens, R);
  // x = patchify(latent) W_pe^T + b_pe
  DIT_TRY(run_latent(false, cfg, tab, latent, W.tok, nullptr, nullptr, stream));
  DIT_TRY(run_linear(W.tok, P, w->w_pe, P, w->b_pe, W.x, D, T, D, P, DIT_EPI_NONE, nullptr, 0, nullptr, 0, req, dty,
                     stream, "patch embedding"));
  // SiLU(c) of the shared timestep MLP, once for all blocks
  DIT_TRY(run_cond_parts(c, R, t, w->w_t1, w->b_t1, w->w_t2, w->b_t2, nullptr, nullptr, 0, nullptr, W.blk, stream,
                         "timestep MLP"));
  const Workspace& B = W.blk;
  for (int b = 0; b < cfg->n_blocks; ++b) {
    const dit_block_weights* bw = &w->blocks[b];
    DIT_TRY(run_cond_parts(c, R, t, nullptr, nullptr, nullptr, nullptr, bw->w_ada, bw->b_ada, 6, B.mod, B, stream,
                           "block modulation"));
    DIT_TRY(pre_attention_impl(c, bw, vl, W.x, B.mod, B.qkv, B, stream));
    DIT_TRY(self_attention_impl(c, vl, B.qkv, B.o, stream));
    DIT_TRY(post_attention_impl(c, bw, vl, W.x, B.o, nullptr, B.mod, W.x, B, stream,
                                (const char*)kv + (size_t)b * L * 2 * D * es));
  }
  // output layer: v = (LN(x)(1 + scale) + shift) W_out^T + b_out with (shift, scale) = W_hmod SiLU(c) + b_hmod
  DIT_TRY(run_cond_parts(c, R, t, nullptr, nullptr, nullptr, nullptr, w->w_hmod, w->b_hmod, 2, B.mod, B, stream,
                         "output modulation"));
  DIT_TRY(run_ln_mod(W.x, B.mod, B.mod + D, 2 * D, req, T, D, c->ln_eps, B.h, dty, stream));
  DIT_TRY(run_linear(B.h, D, w->w_out, D, w->b_out, W.tok, P, T, P, D, DIT_EPI_NONE, nullptr, 0, nullptr, 0, req, dty,
                     stream, "output projection"));
  // latent_out = latent + dt * unpatchify(v)
  return run_latent(true, cfg, tab, latent, W.tok, dt, latent_out, stream);
}

dit_status dit_patchify(const dit_model_config* cfg, const dit_varlen* vl, const float* latent, void* tokens,
                        hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_model_cfg(cfg));
  LatentTable tab;
  DIT_TRY(check_model_varlen(cfg, vl, &tab));
  DIT_TRY(check_ptr(latent, "latent")); DIT_TRY(check_ptr(tokens, "tokens"));
  return run_latent(false, cfg, tab, latent, tokens, nullptr, nullptr, stream);
}

dit_status dit_unpatchify_euler(const dit_model_config* cfg, const dit_varlen* vl, const float* latent, const void* v,
                                const float* dt, float* latent_out, hipStream_t stream) {
  g_last_error.clear();
  DIT_TRY(check_model_cfg(cfg));
  LatentTable tab;
  DIT_TRY(check_model_varlen(cfg, vl, &tab));
  DIT_TRY(check_ptr(latent, "latent")); DIT_TRY(check_ptr(v, "v")); DIT_TRY(check_ptr(dt, "dt"));
  DIT_TRY(check_ptr(latent_out, "latent_out"));
  return run_latent(true, cfg, tab, latent, const_cast<void*>(v), dt, latent_out, stream);
}

}  // extern "C"
