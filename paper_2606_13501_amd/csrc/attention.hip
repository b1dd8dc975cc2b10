// Scaled dot-product attention over a packed batch, non-causal (the denoising
// step attends bidirectionally over the whole latent sequence).
//
// bf16, head_dim 128: flash-style kernel for gfx950.  One 512-thread workgroup
// (8 waves, 2 per SIMD) owns 256 query rows of one (request, head); each wave
// owns 32 of them.  K and V tiles of 64 keys are staged through LDS (two
// stages; V is stored transposed, d-major).  Per tile a wave computes
// S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (K as the A operand), so that every
// lane holds 16 scores of ONE query row: the running max and sum of that row
// live in the lane, P^T feeds the next MFMA straight from the lane's registers,
// and O^T = V^T P^T leaves the output of the same query row in the same lane.
// The key order inside each 32-key block is permuted (bits 2 and 3 of the key
// index swapped) so that the 8 keys a lane contributes to a PV MFMA are
// contiguous in the transposed V tile (one 16-byte LDS read).  Softmax runs in
// fp32 with exp2 and the log2(e) folded into the scale; P is rounded to bf16
// for the PV product.
//
// fp32: one thread per (query row, head) with an exact online softmax.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace dit {

namespace {

constexpr int D = 128;           // head_dim of the bf16 kernel
constexpr int BQ = 256;          // query rows per workgroup
constexpr int BKV = 64;          // keys per LDS tile
constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
// K rows (one key, 256 B) are padded to a 272-byte pitch, so that fragment
// reads of 8 or 16 consecutive rows hit distinct banks and every K fragment
// address is a per-lane base plus an immediate.  V^T rows (one d, 64 keys =
// 128 B) are unpadded; their 16-byte chunks are XOR-swizzled with
// vt_swizzle(d), conflict-free both for the transposing writes and for the
// fragment reads.
constexpr int kKPitch = D * 2 + 16;
constexpr int kVPitch = BKV * 2;
constexpr int kKBytes = BKV * kKPitch;   // 17 KiB
constexpr int kVSlots = 3;               // V^T tiles live one step longer than K tiles
constexpr int kVBytes = D * kVPitch;     // 18 KiB
constexpr int kXcds = 8;

struct AttnWork {
  int n_req;                        // requests, in scheduling order (longest first)
  int q_start[DIT_MAX_REQ];
  int q_len[DIT_MAX_REQ];
  int k_start[DIT_MAX_REQ];
  int k_len[DIT_MAX_REQ];
  int tiles_q[DIT_MAX_REQ];         // query tiles of one head
  int prefix[DIT_MAX_REQ + 1];      // work items before request i (all heads)
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  uint32_t n = bytes > 0xFFFFFFFFll ? 0xFFFFFFFFu : (uint32_t)(bytes < 0 ? 0 : bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}

__device__ __forceinline__ int vt_swizzle(int d) { return (d & 7) ^ ((d >> 3) & 3); }

// swap bits 2 and 3 of a key index inside its 16-key group
__device__ __forceinline__ int perm23(int x) {
  return (x & ~12) | ((x & 4) << 1) | ((x & 8) >> 1);
}

__global__ __launch_bounds__(kThreads, 1) void attn_fwd_bf16(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    bf16* __restrict__ O, int64_t qs, int64_t ks, int64_t vs, int64_t os, int n_heads,
    float scale_log2, AttnWork work) {
  // K(j) in K slot j & 1, V(j) in V slot j % 3
  __shared__ __attribute__((aligned(16))) char smem[2 * kKBytes + kVSlots * kVBytes];
  char* const kslots = smem;
  char* const vslots = smem + 2 * kKBytes;

  // ---- work item: XCD-contiguous numbering, requests longest first
  const int nb = gridDim.x;
  const int b = blockIdx.x;
  const int w = (b % kXcds) * (nb / kXcds) + b / kXcds;
  if (w >= work.prefix[work.n_req]) return;
  int r = 0;
  while (w >= work.prefix[r + 1]) ++r;
  const int local = w - work.prefix[r];
  const int head = local / work.tiles_q[r];
  const int qt = local - head * work.tiles_q[r];
  const int q0 = work.q_start[r] + qt * BQ;
  const int q_end = work.q_start[r] + work.q_len[r];
  const int k0 = work.k_start[r];
  const int n_k = work.k_len[r];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar branches
  const int fr = lane & 31;
  const int fh = lane >> 5;

  // ---- Q fragments (MFMA B operand of S^T): row fr of this wave, d 16kk + 8fh .. +7
  const int my_q = q0 + wave * 32 + fr;
  bf16x8 qf[8];
  {
    const int qrow = min(my_q, q_end - 1);
    const bf16* qp = Q + (int64_t)qrow * qs + head * D + 8 * fh;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) qf[kk] = *reinterpret_cast<const bf16x8*>(qp + 16 * kk);
  }

  // ---- global -> LDS staging (all 512 threads share every tile)
  // buffer resources are rebased at every tile so offsets stay small; loads
  // past the request's last key return zeros
  const bf16* k_head = K + (int64_t)k0 * ks + head * D;
  const bf16* v_head = V + (int64_t)k0 * vs + head * D;
  // K: 2 chunks of 16 B per thread: key (tid >> 4) + 32 i, chunk tid & 15;
  // key k is stored in row slot perm23(k) so that MFMA row fr reads slot fr
  const int kl_key = tid >> 4;
  const int kl_c = tid & 15;
  const int kl_voff = kl_key * (int)ks * 2 + kl_c * 16;
  const int kl_st = perm23(kl_key) * kKPitch + kl_c * 16;   // + 32 kKPitch for i = 1
  // V: keys 4 kg .. 4 kg + 3, d 4 dc .. 4 dc + 3 (8-byte loads; a wave reads
  // two whole 256-byte key rows per load), written transposed as V^T
  const int vl_lo = tid & 1;
  const int vl_dc = (tid >> 1) & 31;
  const int vl_kg = 2 * (tid >> 6) + vl_lo;
  const int vl_voff = (4 * vl_kg) * (int)vs * 2 + vl_dc * 8;
  int vl_st[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int d = 4 * vl_dc + e;
    vl_st[e] = d * kVPitch + (((vl_kg >> 1) ^ vt_swizzle(d)) << 4) + (vl_kg & 1) * 8;
  }

  // two register staging sets: the loads of tile t go to set t & 1, two
  // steps before the tile is read from LDS
  u32x4 kreg[2][2];
  u32x2 vreg[2][4];
  auto gload = [&](int kt, auto set) {
    constexpr int S = decltype(set)::value;
    const int kb0 = kt * BKV;
    const __amdgpu_buffer_rsrc_t krs = make_rsrc(k_head + (int64_t)kb0 * ks, (int64_t)(n_k - kb0) * ks * 2);
#pragma unroll
    for (int i = 0; i < 2; ++i)
      kreg[S][i] = __builtin_amdgcn_raw_buffer_load_b128(krs, kl_voff, 32 * i * (int)ks * 2, 0);
    // keys past the request end lie past the end of the buffer range and load
    // as zeros, so P = 0 times V stays exact (no select on the loaded value,
    // which would wait for the load right here)
    const __amdgpu_buffer_rsrc_t vrs = make_rsrc(v_head + (int64_t)kb0 * vs, (int64_t)(n_k - kb0) * vs * 2);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      vreg[S][i] = __builtin_amdgcn_raw_buffer_load_b64(vrs, vl_voff, i * (int)vs * 2, 0);
  };
  auto sstore = [&](int kt, auto set) {
    constexpr int S = decltype(set)::value;
    char* kb = kslots + (kt & 1) * kKBytes;
#pragma unroll
    for (int i = 0; i < 2; ++i) *reinterpret_cast<u32x4*>(kb + kl_st + 32 * i * kKPitch) = kreg[S][i];
    char* vb = vslots + (kt % kVSlots) * kVBytes;
    // transpose 4 keys x 4 d: element (key i, d e) -> V^T[d e][key i]
    const uint16_t* vv = reinterpret_cast<const uint16_t*>(vreg[S]);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      u32x2 t;
      t[0] = (uint32_t)vv[0 * 4 + e] | ((uint32_t)vv[1 * 4 + e] << 16);
      t[1] = (uint32_t)vv[2 * 4 + e] | ((uint32_t)vv[3 * 4 + e] << 16);
      *reinterpret_cast<u32x2*>(vb + vl_st[e]) = t;
    }
  };

  // ---- fragment read offsets inside a slot
  // K (A operand of S^T): slot 32 blk + fr (= key 32 blk + perm23(fr)), d 16 kk + 8 fh
  const int koff = fr * kKPitch + fh * 16;             // + blk 32 kKPitch + kk 32
  // V^T (A operand of O^T): row d = 32 dblk + fr, 16-byte chunk 2 (2 blk + hs) + fh
  // (vt_swizzle(32 dblk + fr) == vt_swizzle(fr))
  int voff[4];                                         // [2 blk + hs], + dblk 32 kVPitch
#pragma unroll
  for (int c4 = 0; c4 < 4; ++c4) voff[c4] = fr * kVPitch + (((2 * c4 + fh) ^ vt_swizzle(fr)) << 4);

  const int n_tiles = (n_k + BKV - 1) / BKV;
  const int n_full = n_k / BKV;

  f32x16 oacc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) oacc[i] = f32x16{};
  f32x16 s[2];          // scores of the current tile: s[blk][4i + j] = S[q = fr][key 32 blk + perm23(8 i + 4 fh + j)]
  bf16x8 pf[2][2];      // probabilities of the current tile, PV operand
  float m_tile = 0.f;   // max of the current tile's scores of the lane's row (times scale_log2)
  // Running max of (score * scale_log2) of the lane's query row.  It is only
  // raised when a tile's max exceeds it by more than kLazy (log2 units), so
  // that the O rescale is skipped for most tiles; probabilities are then
  // bounded by 2^kLazy, harmless in fp32 and bf16.
  constexpr float kLazy = 8.0f;
  float m_run = -INFINITY;
  float l_run = 0.f;    // this lane's share of the running sum

  // S(j) = K(j) Q^T, as four independent MFMA chains (even and odd d-steps of
  // each 32-key block) summed at the end, so that no MFMA waits on the result
  // of the one issued just before it
  auto mma_s = [&](int j) {
    const char* kb = kslots + (j & 1) * kKBytes + koff;
    f32x16 s2[2][2];
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
#pragma unroll
      for (int blk = 0; blk < 2; ++blk) {
        bf16x8 kf = *reinterpret_cast<const bf16x8*>(kb + blk * 32 * kKPitch + kk * 32);
        s2[blk][kk & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kk], kk < 2 ? f32x16{} : s2[blk][kk & 1], 0, 0, 0);
      }
    }
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) s[blk] = s2[blk][0] + s2[blk][1];
    // keep four fragment reads in flight ahead of the MFMAs
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 1);
#pragma unroll
    for (int i = 0; i < 12; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 1);
  };
  // O^T += V^T(j) P^T(j)
  auto mma_pv = [&](int j) {
    const char* vb = vslots + (j % kVSlots) * kVBytes;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int hs = 0; hs < 2; ++hs)
#pragma unroll
        for (int dblk = 0; dblk < 4; ++dblk) {
          bf16x8 vf = *reinterpret_cast<const bf16x8*>(vb + voff[2 * blk + hs] + dblk * 32 * kVPitch);
          oacc[dblk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[blk][hs], oacc[dblk], 0, 0, 0);
        }
    // keep four fragment reads in flight ahead of the MFMAs
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 2);
#pragma unroll
    for (int i = 0; i < 12; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 2);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 2);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 2);
  };
  // mask of the ragged last tile (masked == true), then the row max of S(j)
  auto row_max = [&](int j, auto masked) {
    if (decltype(masked)::value) {
#pragma unroll
      for (int blk = 0; blk < 2; ++blk)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = j * BKV + 32 * blk + perm23(8 * (v >> 2) + 4 * fh + (v & 3));
          if (key >= n_k) s[blk][v] = -INFINITY;
        }
    }
    // the lane's 32 scores, then the other half-wave's 32 (same row)
    float mx = fmaxf(fmaxf(s[0][0], s[0][1]), s[0][2]);
#pragma unroll
    for (int v = 3; v < 15; v += 2) mx = fmaxf(fmaxf(mx, s[0][v]), s[0][v + 1]);
    mx = fmaxf(mx, s[0][15]);
#pragma unroll
    for (int v = 0; v < 16; v += 2) mx = fmaxf(fmaxf(mx, s[1][v]), s[1][v + 1]);
    auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
    m_tile = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * scale_log2;
  };
  // online softmax of S into P
  auto softmax = [&]() {
    if (__builtin_amdgcn_ballot_w64(m_tile > m_run + kLazy) != 0) {
      const float m_new = fmaxf(m_run, m_tile);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int i = 0; i < 4; ++i) oacc[i] *= alpha;
    }
    float psum = 0.f;
#pragma unroll
    for (int blk = 0; blk < 2; ++blk)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[blk][v], scale_log2, -m_run));
        psum += p;
        pf[blk][v >> 3][v & 7] = (bf16)p;
      }
    l_run += psum;
  };
  // ---- main loop.  Step j computes tile j from LDS, issues the loads of
  // tile j+2 (register set j & 1) at its start and stores tile j+1 (loaded
  // one step earlier, set (j+1) & 1) to LDS before its barrier, so every load
  // has two steps to arrive.  Full tiles inside the loop (unrolled by two for
  // the register sets), the ragged last tile (with its key mask) after it.
  // Waves 0-3 run S(j), softmax(j), PV(j) between two barriers.  Waves 4-7
  // run the same sequence but take the barrier before PV(j), which they
  // compute at the start of the next step: the two waves sharing a SIMD are
  // then half a step apart, one on the matrix core while the other runs its
  // softmax.  V(j) is read until the step after j, hence three V slots.
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  gload(0, S0{});
  sstore(0, S0{});
  if (n_tiles > 1) gload(1, S1{});
  // every load issued so far (Q fragments included) has completed: without
  // this the waits for the Q loads land inside the loop, where they would
  // also wait for each step's K and V prefetch
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
  __syncthreads();
  const bool lead = wave < kWaves / 2;
  auto step_full = [&](int j, auto set) {
    constexpr int S = decltype(set)::value;
    if (j + 2 < n_tiles) gload(j + 2, std::integral_constant<int, S>{});
    if (!lead && j > 0) mma_pv(j - 1);
    mma_s(j);
    row_max(j, std::false_type{});
    softmax();
    if (lead) mma_pv(j);
    if (j + 1 < n_tiles) sstore(j + 1, std::integral_constant<int, 1 - S>{});
    __syncthreads();
  };
  int j = 0;
  for (; j + 2 <= n_full; j += 2) {
    step_full(j, S0{});
    step_full(j + 1, S1{});
  }
  if (j < n_full) {
    step_full(j, S0{});
    ++j;
  }
  if (!lead && n_full > 0) mma_pv(n_full - 1);
  if (n_full < n_tiles) {
    mma_s(n_full);
    row_max(n_full, std::true_type{});
    softmax();
    mma_pv(n_full);
  }

  // ---- normalise and store: oacc[dblk][4i + j] = O[q = fr][d = 32 dblk + 8 i + 4 fh + j]
  // (the S^T rows of a lane are keys perm23(8 i + 4 fh + j); for the PV MFMA of
  // half hs the lane's 8 values are keys 16 hs + 8 fh + 0..7 of the block)
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;   // no keys: output 0
  if (my_q < q_end) {
    bf16* op = O + (int64_t)my_q * os + head * D + 4 * fh;
#pragma unroll
    for (int dblk = 0; dblk < 4; ++dblk)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        bf16x4 ov;
#pragma unroll
        for (int j = 0; j < 4; ++j) ov[j] = (bf16)(oacc[dblk][4 * i + j] * inv);
        *reinterpret_cast<bf16x4*>(op + 32 * dblk + 8 * i) = ov;
      }
  }
}

// ------------------------------------------------------------------- fp32

__global__ __launch_bounds__(64) void attn_fwd_f32(
    const float* __restrict__ Q, const float* __restrict__ K, const float* __restrict__ V,
    float* __restrict__ O, int64_t qs, int64_t ks, int64_t vs, int64_t os, int n_heads, int head_dim,
    float scale, ReqTable cq, ReqTable ck, int n_q) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n_q * n_heads) return;
  const int row = idx / n_heads;
  const int head = idx - row * n_heads;
  const int r = find_req(cq.cu, cq.n_req, row);
  const int kb = ck.cu[r], ke = ck.cu[r + 1];
  const float* q = Q + (int64_t)row * qs + head * head_dim;
  float m = -INFINITY, l = 0.f;
  float acc[128];
  for (int e = 0; e < head_dim; ++e) acc[e] = 0.f;
  for (int j = kb; j < ke; ++j) {
    const float* k = K + (int64_t)j * ks + head * head_dim;
    float s = 0.f;
    for (int e = 0; e < head_dim; ++e) s = fmaf(q[e], k[e], s);
    s *= scale;
    float m_new = fmaxf(m, s);
    float a = expf(m - m_new);
    float p = expf(s - m_new);
    l = l * a + p;
    const float* v = V + (int64_t)j * vs + head * head_dim;
    for (int e = 0; e < head_dim; ++e) acc[e] = acc[e] * a + p * v[e];
    m = m_new;
  }
  float* o = O + (int64_t)row * os + head * head_dim;
  const float inv = ke > kb ? 1.0f / l : 0.f;
  for (int e = 0; e < head_dim; ++e) o[e] = acc[e] * inv;
}

}  // namespace

hipError_t launch_attention(const AttnArgs& p, hipStream_t s) {
  const int n_req = p.cq.n_req;
  if (p.dtype == DIT_F32) {
    const int n_q = p.cq.cu[n_req];
    if (n_q == 0) return hipSuccess;
    const int total = n_q * p.n_heads;
    attn_fwd_f32<<<(total + 63) / 64, 64, 0, s>>>(
        (const float*)p.q, (const float*)p.k, (const float*)p.v, (float*)p.o, p.q_stride, p.k_stride,
        p.v_stride, p.o_stride, p.n_heads, p.head_dim, p.scale, p.cq, p.ck, n_q);
    return hipGetLastError();
  }
  // requests with queries, longest key range first (their tiles do the most work)
  AttnWork w{};
  int order[DIT_MAX_REQ];
  int n = 0;
  for (int r = 0; r < n_req; ++r)
    if (p.cq.cu[r + 1] > p.cq.cu[r]) order[n++] = r;
  for (int i = 1; i < n; ++i) {
    int x = order[i], j = i - 1;
    int lx = p.ck.cu[x + 1] - p.ck.cu[x];
    while (j >= 0 && (p.ck.cu[order[j] + 1] - p.ck.cu[order[j]]) < lx) { order[j + 1] = order[j]; --j; }
    order[j + 1] = x;
  }
  w.n_req = n;
  w.prefix[0] = 0;
  for (int i = 0; i < n; ++i) {
    int r = order[i];
    w.q_start[i] = p.cq.cu[r];
    w.q_len[i] = p.cq.cu[r + 1] - p.cq.cu[r];
    w.k_start[i] = p.ck.cu[r];
    w.k_len[i] = p.ck.cu[r + 1] - p.ck.cu[r];
    w.tiles_q[i] = (w.q_len[i] + BQ - 1) / BQ;
    w.prefix[i + 1] = w.prefix[i] + w.tiles_q[i] * p.n_heads;
  }
  const int items = w.prefix[n];
  if (items == 0) return hipSuccess;
  const int grid = (items + kXcds - 1) / kXcds * kXcds;
  const float scale_log2 = p.scale * 1.4426950408889634f;
  attn_fwd_bf16<<<grid, kThreads, 0, s>>>((const bf16*)p.q, (const bf16*)p.k, (const bf16*)p.v,
                                          (bf16*)p.o, p.q_stride, p.k_stride, p.v_stride, p.o_stride,
                                          p.n_heads, scale_log2, w);
  return hipGetLastError();
}

}  // namespace dit
