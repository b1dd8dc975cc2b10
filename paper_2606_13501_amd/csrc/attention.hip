// Scaled dot-product attention over a packed batch, non-causal (the denoising
// step attends bidirectionally over the whole latent sequence).
//
// bf16, head_dim 128: flash-style kernel for gfx950.  One 512-thread
// workgroup (8 waves, two per SIMD) owns 256 query rows of one (request,
// head); each wave owns 32 of them.  Two waves per SIMD let the matrix core
// run one wave's MFMAs while the other wave's softmax, LDS reads and waits
// are in progress, with no hand-made phase offset between them.  K and V
// tiles of 64 keys stream from global memory straight into an LDS ring of 4
// tiles (buffer loads with the lds modifier: no registers, no LDS store
// instructions), issued 3 tiles ahead of use.  Both are stored row-major with
// their 16-byte chunks XOR-swizzled per row.
//
// Per tile a wave computes S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (K as
// the A operand, Q fragments held in registers), two 32-key halves as two
// independent accumulation chains, so every lane holds the scores of its
// query row: P^T feeds the PV MFMA straight from the lane's registers, and
// O^T = V^T P^T leaves the output of the same row in the same lane.  The V^T
// operand is read from the row-major V tile with the transposing LDS read
// (ds_read_b64_tr_b16); its source rows are chosen so that the 8 keys a lane
// contributes match the order of the lane's scores (bits 2 and 3 of the key
// index swapped).
//
// Softmax is fp32 with exp2, against a per-row reference fixed for the whole
// pass (the first tile's row max): no rescale of O inside the loop.  Q is
// scaled by log2(e)/sqrt(d) once, in registers, and the first S MFMA of a
// tile accumulates onto the negated reference, so the matrix core delivers
// score - reference in log2 units and the softmax is an exp2, a conversion
// and an add per score.  If any row of the workgroup exceeded its reference
// by more than 2^64 (where the probabilities could overflow), the work item
// is recomputed with a safe reference, so the result is always the exact
// softmax up to rounding.
//
// fp32: one thread per (query row, head) with an exact online softmax.
#include <float.h>

#include <atomic>
#include <mutex>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace dit {

namespace {

constexpr int D = 128;                 // head_dim of the bf16 kernel
constexpr int BKV = 64;                // keys per tile
constexpr int kTileBytes = BKV * D * 2;          // one K or V tile (16 KiB)
constexpr int kSlotBytes = 2 * kTileBytes;       // K tile + V tile
constexpr int kXcds = 8;
// Two shapes of the bf16 kernel, both with 32 query rows per wave:
//  - long key ranges: 8 waves (256 query rows) per workgroup, one workgroup
//    per compute unit, an LDS ring of 4 K/V tiles issued 3 ahead;
//  - short key ranges (cross-attention to text, short requests): 4 waves
//    (128 query rows), two workgroups per compute unit, a ring of 2 tiles
//    issued 2 ahead.  A work item is then only a few tiles long, and the
//    second workgroup's tiles keep the matrix cores busy while one workgroup
//    loads its queries and first tiles or stores its output.
constexpr int kShortKeys = 1024;       // longest key range that takes the short shape
constexpr float kHeadroom = 64.0f;   // log2 units; probabilities stay below 2^64

struct AttnWork {
  int n_req;                        // requests, in scheduling order (longest first)
  int q_start[DIT_MAX_REQ];
  int q_len[DIT_MAX_REQ];
  int k_start[DIT_MAX_REQ];
  int k_len[DIT_MAX_REQ];
  int tiles_q[DIT_MAX_REQ];         // query tiles of one head
  int prefix[DIT_MAX_REQ + 1];      // work items before request i (all heads)
  // Split items (split_s > 0): workgroup split_base + b computes key piece
  // b % split_s of item split_first + b / split_s of request split_req (the
  // first split_first items of that request are whole items) and writes its
  // unnormalised output, row reference and row sum to part, for split_n
  // pieces in all (see the launcher)
  int split_s, split_req, split_first, split_base, split_n;
  float* part;
};

// 16 bytes per lane from global memory straight into LDS: lane i writes LDS
// bytes lds + OFF + 16 i .. +15 (one scalar add into m0 per load).  Inline
// assembly, so the compiler does not make every later LDS read wait for it;
// completion is tracked by hand (wait_vmcnt) and the workgroup barrier
// publishes the data.  Raw buffer descriptors (stride 0): loads past the
// record count return zeros.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
template <uint32_t OFF>
__device__ __forceinline__ void load_lds16(const u32x4& desc, uint32_t voff, uint32_t lds) {
  asm volatile("s_add_u32 m0, %0, %3\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :: "s"(lds), "v"(voff), "s"(desc), "n"(OFF) : "m0", "scc");
}
#pragma clang diagnostic pop
template <int N> __device__ __forceinline__ void wait_vmcnt() { asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N)); }

// S^T MFMAs as inline assembly with vector-register operands: the compiler
// would otherwise place the scores in accumulation registers and copy them to
// vector registers for the softmax.  It does not see these as MFMAs, so the
// distance from the last MFMA of a score block to its first vector read is
// kept by hand: the last MFMA pair of a tile and the wait states after it
// (13; the compiler puts 12 between this MFMA and a vector read of its
// result) are one asm statement, so nothing that reads the scores, not even
// a register copy the allocator adds, can come between them.
__device__ __forceinline__ void mfma_s_first(f32x16& d, const bf16x8& a, const bf16x8& b) {
  // d as an in-out operand (its old value unused) keeps the scores in the
  // same registers from tile to tile, without copies
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "+v"(d) : "v"(a), "v"(b));
}
// the first MFMA of a score block starting from the bias c (the negated row
// reference) instead of zero
__device__ __forceinline__ void mfma_s_bias(f32x16& d, const bf16x8& a, const bf16x8& b, const f32x16& c) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %3" : "+v"(d) : "v"(a), "v"(b), "v"(c));
}
__device__ __forceinline__ void mfma_s_acc(f32x16& d, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(d) : "v"(a), "v"(b));
}
// the last MFMA of both score blocks, then the wait states
__device__ __forceinline__ void mfma_s_last(f32x16& d0, f32x16& d1, const bf16x8& a0, const bf16x8& a1,
                                            const bf16x8& b) {
  asm volatile(
      "v_mfma_f32_32x32x16_bf16 %0, %2, %4, %0\n\tv_mfma_f32_32x32x16_bf16 %1, %3, %4, %1\n\ts_nop 7\n\ts_nop 4"
      : "+v"(d0), "+v"(d1)
      : "v"(a0), "v"(a1), "v"(b));
}

typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// QNORM: q is RMS-normalised per head (gain q_gain, epsilon q_eps) as it is
// loaded, before the softmax scale is applied.
template <int WAVES, int RING, bool QNORM>
__global__ __launch_bounds__(WAVES * 64, WAVES == 4 ? 2 : 1) void attn_fwd_bf16(
    const bf16* __restrict__ Q, const bf16* __restrict__ K, const bf16* __restrict__ V,
    bf16* __restrict__ O, int64_t qs, int64_t ks, int64_t vs, int64_t os, int n_heads,
    float scale_log2, const bf16* __restrict__ q_gain, float q_eps, AttnWork work) {
  static_assert((WAVES == 8 && RING == 4) || (WAVES == 4 && RING == 2), "two shapes");
  constexpr int BQ = 32 * WAVES;                          // query rows per workgroup
  constexpr int kPieces = kTileBytes / 1024 / WAVES;      // 1 KiB loads per wave and operand
  constexpr int kLoadsPerTile = 2 * kPieces;              // this wave's loads of one tile
  constexpr int kAhead = RING == 4 ? 3 : 2;               // tiles issued ahead of the one computed
  // slot t % RING holds K(t) (first 16 KiB) and V(t)
  __shared__ __attribute__((aligned(1024))) char smem[RING * kSlotBytes];
  __shared__ int redo_flag[2];   // one flag per pass that may ask for another

  // ---- work item.  Workgroups are dispatched to the XCDs round-robin, so
  // workgroup b runs on XCD b % 8 as that XCD's (b / 8)-th.  Each XCD takes
  // the same contiguous eighth of every request's items (head-major, requests
  // longest first): the long requests' work is spread over all XCDs, and the
  // query tiles of one head stay together on one XCD, sharing its K/V in L2.
  int r = 0, local = -1, piece = -1;
  if (work.split_s > 0 && (int)blockIdx.x >= work.split_base) {
    const int b = (int)blockIdx.x - work.split_base;
    r = work.split_req;
    local = work.split_first + b / work.split_s;
    piece = b % work.split_s;
  } else {
    const int xcd = blockIdx.x % kXcds;
    int j = blockIdx.x / kXcds;
    for (; r < work.n_req; ++r) {
      const int n_r = work.prefix[r + 1] - work.prefix[r];
      const int lo = xcd * n_r / kXcds, hi = (xcd + 1) * n_r / kXcds;
      if (j < hi - lo) {
        local = lo + j;
        break;
      }
      j -= hi - lo;
    }
    if (local < 0) return;
  }
  const int head = local / work.tiles_q[r];
  const int qt = local - head * work.tiles_q[r];
  const int q0 = work.q_start[r] + qt * BQ;
  const int q_end = work.q_start[r] + work.q_len[r];
  int k0 = work.k_start[r];
  int n_k = work.k_len[r];
  if (piece >= 0) {   // this piece's key tiles: a contiguous 1 / split_s of the request's
    const int kt_all = (n_k + BKV - 1) / BKV;
    const int per = (kt_all + work.split_s - 1) / work.split_s;
    const int kt0 = min(piece * per, kt_all);
    k0 += kt0 * BKV;
    n_k = max(0, min(n_k - kt0 * BKV, per * BKV));
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform: scalar branches
  const int fr = lane & 31;
  const int fh = lane >> 5;
  if (tid < 2) redo_flag[tid] = 0;

  // ---- Q fragments (B operand of S^T): query q0 + 32 wave + fr, d 16 kc +
  // 8 fh .. +7, scaled by log2(e)/sqrt(d) and rounded to bf16 once (a
  // relative error of at most 2^-9 per element, the size of q's own rounding)
  const int my_q = q0 + 32 * wave + fr;
  bf16x8 qf[8];
  bf16x8 gf[QNORM ? 8 : 1];
  {
    const bf16* qp = Q + (int64_t)min(my_q, q_end - 1) * qs + head * D + 8 * fh;
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) qf[kc] = *reinterpret_cast<const bf16x8*>(qp + 16 * kc);
    if constexpr (QNORM) {
#pragma unroll
      for (int kc = 0; kc < 8; ++kc) gf[kc] = *reinterpret_cast<const bf16x8*>(q_gain + 8 * fh + 16 * kc);
    }
  }
  // the Q loads complete here, before any tile load is issued (otherwise the
  // compiler's wait for them would also wait for the tile loads)
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
  typedef float f32x8 __attribute__((ext_vector_type(8)));
  float q_mul = scale_log2;
  if constexpr (QNORM) {
    // RMSNorm over the head: this lane holds 64 of its 128 values, the lane
    // 32 apart the other 64
    float ss = 0.f;
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) {
      const f32x8 f = __builtin_convertvector(qf[kc], f32x8);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = fmaf(f[e], f[e], ss);
    }
    auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(ss), __float_as_uint(ss), false, false);
    const float tot = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
    q_mul = scale_log2 * rsqrtf(tot * (1.0f / D) + q_eps);
  }
#pragma unroll
  for (int kc = 0; kc < 8; ++kc) {
    f32x8 f = __builtin_convertvector(qf[kc], f32x8) * q_mul;
    if constexpr (QNORM) f *= __builtin_convertvector(gf[QNORM ? kc : 0], f32x8);
    qf[kc] = __builtin_convertvector(f, bf16x8);
  }

  // ---- global -> LDS.  A tile (K or V) is 16 pieces of 1 KiB = 4 key rows
  // of 256 B; wave w loads pieces 2 w, 2 w + 1 of both.  Lane i of piece p
  // fills LDS chunk i of the piece: row 4 p + i / 16, physical chunk i % 16,
  // which holds logical chunk (i % 16) ^ swizzle(row):
  //   K: swizzle(row) = row % 16   (fragment reads of 16 rows at one chunk)
  //   V: swizzle(row) = 4 (row % 4) (transposing reads of 4 rows x 64 B)
  const bf16* k_head = K + (int64_t)k0 * ks + head * D;
  const bf16* v_head = V + (int64_t)k0 * vs + head * D;
  uint32_t k_voff[kPieces], v_voff[kPieces];
#pragma unroll
  for (int u = 0; u < kPieces; ++u) {
    const int row = 4 * (kPieces * wave + u) + (lane >> 4);
    const int pc = lane & 15;
    k_voff[u] = (uint32_t)(row * (int)ks * 2 + ((pc ^ (row & 15)) << 4));
    v_voff[u] = (uint32_t)(row * (int)vs * 2 + ((pc ^ (4 * (row & 3))) << 4));
  }
  const uint32_t lds_base = (uint32_t)(uintptr_t)(lds_char*)smem;
  // Rows past the request's last key read as zero (descriptor bound).  The
  // tiles are issued in order, so the next tile's base addresses and its
  // rows left advance by one tile per issue: a few scalar instructions
  // instead of 64-bit products and clamps per tile, which all eight waves
  // would otherwise run on the one scalar unit of the compute unit right
  // after each barrier.  The record count is capped at the 32-bit range.
  const uint32_t k_row_b = (uint32_t)ks * 2u, v_row_b = (uint32_t)vs * 2u;
  const int cap_rows = (int)min((uint32_t)INT_MAX, 0xFFFFFFFFu / max(max(k_row_b, v_row_b), 1u));
  uint64_t k_next = 0, v_next = 0;
  int rows_left = 0;
  auto rewind = [&]() __attribute__((always_inline)) {
    k_next = (uint64_t)(uintptr_t)k_head;
    v_next = (uint64_t)(uintptr_t)v_head;
    rows_left = n_k;
  };
  auto issue = [&](int t) __attribute__((always_inline)) {
    const uint32_t rows = (uint32_t)min(max(rows_left, 0), cap_rows);
    const u32x4 kd = u32x4{(uint32_t)k_next, (uint32_t)(k_next >> 32) & 0xFFFFu, rows * k_row_b, 0x00020000u};
    const u32x4 vd = u32x4{(uint32_t)v_next, (uint32_t)(v_next >> 32) & 0xFFFFu, rows * v_row_b, 0x00020000u};
    k_next += (uint64_t)(BKV * k_row_b);
    v_next += (uint64_t)(BKV * v_row_b);
    rows_left -= BKV;
    const uint32_t st = lds_base + (uint32_t)((t % RING) * kSlotBytes) + kPieces * wave * 1024;
#pragma unroll
    for (int u = 0; u < kPieces; ++u) {
      static_assert(kPieces <= 4, "LDS offsets below");
      if (u == 0) {
        load_lds16<0>(kd, k_voff[u], st);
        load_lds16<kTileBytes>(vd, v_voff[u], st);
      } else if (u == 1) {
        load_lds16<1024>(kd, k_voff[u], st);
        load_lds16<kTileBytes + 1024>(vd, v_voff[u], st);
      } else if (u == 2) {
        load_lds16<2048>(kd, k_voff[u], st);
        load_lds16<kTileBytes + 2048>(vd, v_voff[u], st);
      } else {
        load_lds16<3072>(kd, k_voff[u], st);
        load_lds16<kTileBytes + 3072>(vd, v_voff[u], st);
      }
    }
  };

  // ---- fragment addresses inside a slot
  // K (A operand of S^T): key row 32 hb + fr, logical chunk 2 kc + fh:
  //   fr * 256 + (((2 kc + fh) ^ (fr % 16)) << 4) = k_lane ^ (kc << 5)
  const int k_lane = fr * 256 + ((fh ^ (fr & 15)) << 4);
  // V^T (A operand of O^T) by transposing reads.  Lanes 16 g .. 16 g + 15
  // (h = g / 2, dh = g % 2) fetch d 32 db + 16 dh .. +15 of 4 key rows; source
  // lane s reads row 16 kc + 4 h + 8 half + s / 4, d 32 db + 16 dh + 4 (s % 4)
  // .. +3 (8 bytes), and lane s receives d 32 db + 16 dh + s of those 4 keys.
  // Logical chunk 4 db + 2 dh + (s / 2) % 2 lies at physical chunk
  // (that) ^ 4 (s / 4), i.e. v_lane ^ (db << 6) plus the row offset.
  int v_lane;
  {
    const int s16 = lane & 15, g = lane >> 4;
    const int h = g >> 1, dh = g & 1, m = s16 >> 2;
    v_lane = kTileBytes + (4 * h + m) * 256 + 64 * m + 16 * (2 * dh + ((s16 >> 1) & 1)) + 8 * (s16 & 1);
  }

  const int n_tiles = (n_k + BKV - 1) / BKV;
  // Scores of a tile: sq[hb][4 i + j] = S[key 32 hb + 8 i + 4 fh + j][query 32 wave + fr]
  f32x16 sq[2];
  bf16x8 pq[4];         // pq[kc]: P^T operand of keys 16 kc .. 16 kc + 15 (scores 8 (kc % 2) .. +7 of half kc / 2)
  f32x16 oacc[4];       // oacc[db][4 i + j] = O[query 32 wave + fr][d 32 db + 8 i + 4 fh + j]
  // Softmax reference of the lane's row (log2 units): P = 2^(score - m_ref).
  // It is fixed for the whole pass (no O rescale inside the loop).  The first
  // pass takes the first tile's row max and checks afterwards that every row
  // sum l stayed <= 2^kHeadroom (then every probability did, and O cannot
  // have overflowed).  A row over that bound is computed again: with m_ref
  // raised by log2(l) when l is finite, which caps its probabilities at 1;
  // that pass also tracks x_max = max(score - m_ref), so a row whose sum had
  // overflowed gets m_ref = its exact max in a last pass.
  float m_ref = 0.f, x_max = -INFINITY;
  float l_run[4];       // this lane's share of the row sum, four partial sums
  f32x16 nref;          // -m_ref in every element, the bias of S

  // S(t) for both 32-key halves (two independent chains); FIRST: from zero
  auto S = [&](int t, auto first) __attribute__((always_inline)) {
    const int so = (t % RING) * kSlotBytes + k_lane;
    bf16x8 ka[8], kb[8];
    ka[0] = *reinterpret_cast<const bf16x8*>(smem + so);
    kb[0] = *reinterpret_cast<const bf16x8*>(smem + so + 32 * 256);
#pragma unroll
    for (int kc = 0; kc < 8; ++kc) {
      if (kc + 1 < 8) {
        ka[kc + 1] = *reinterpret_cast<const bf16x8*>(smem + (so ^ ((kc + 1) << 5)));
        kb[kc + 1] = *reinterpret_cast<const bf16x8*>(smem + (so ^ ((kc + 1) << 5)) + 32 * 256);
      }
      if (kc == 7) {
        mfma_s_last(sq[0], sq[1], ka[7], kb[7], qf[7]);
      } else if (kc > 0) {
        mfma_s_acc(sq[0], ka[kc], qf[kc]);
        mfma_s_acc(sq[1], kb[kc], qf[kc]);
      } else if (decltype(first)::value) {
        mfma_s_first(sq[0], ka[0], qf[0]);
        mfma_s_first(sq[1], kb[0], qf[0]);
      } else {
        mfma_s_bias(sq[0], ka[0], qf[0], nref);
        mfma_s_bias(sq[1], kb[0], qf[0], nref);
      }
    }
  };
  // P(t) from S(t).  FIRST: S(t) came from zero (the reference is set, in the
  // first pass, and subtracted here); LAST: keys past the request end -> -inf
  auto softmax = [&](int t, auto first, auto last, auto track) __attribute__((always_inline)) {
    if (decltype(last)::value && n_k % BKV != 0) {
#pragma unroll
      for (int hb = 0; hb < 2; ++hb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = t * BKV + 32 * hb + 8 * (v >> 2) + 4 * fh + (v & 3);
          if (key >= n_k) sq[hb][v] = -INFINITY;
        }
    }
    if (decltype(first)::value) {
      if (!decltype(track)::value) {
        // first pass: the reference is the row max of the first tile
        float mx = fmaxf(sq[0][0], sq[1][0]);
#pragma unroll
        for (int v = 1; v < 16; ++v) mx = fmaxf(mx, fmaxf(sq[0][v], sq[1][v]));
        auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
        m_ref = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        sq[0][v] -= m_ref;
        sq[1][v] -= m_ref;
        nref[v] = -m_ref;
      }
    }
#pragma unroll
    for (int hb = 0; hb < 2; ++hb)
#pragma unroll
      for (int jp = 0; jp < 8; ++jp) {
        const float x0 = sq[hb][2 * jp], x1 = sq[hb][2 * jp + 1];   // score - m_ref, log2 units
        if (decltype(track)::value) x_max = fmaxf(fmaxf(x_max, x0), x1);
        const float p0 = __builtin_amdgcn_exp2f(x0), p1 = __builtin_amdgcn_exp2f(x1);
        const bf16x2 pr = __builtin_convertvector((f32x2){p0, p1}, bf16x2);
        pq[2 * hb + (jp >> 2)][2 * (jp & 3)] = pr[0];
        pq[2 * hb + (jp >> 2)][2 * (jp & 3) + 1] = pr[1];
        l_run[2 * (jp & 1)] += p0;
        l_run[2 * (jp & 1) + 1] += p1;
      }
  };
  auto PV = [&](int t) __attribute__((always_inline)) {
    const int so = (t % RING) * kSlotBytes;
#pragma unroll
    for (int kc = 0; kc < 4; ++kc)
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const int ad = so + (v_lane ^ (db << 6)) + kc * 16 * 256;
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)((lds_char*)smem + ad));
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)((lds_char*)smem + ad + 8 * 256));
        const bf16x8 vf = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pq[kc], oacc[db], 0, 0, 0);
      }
  };
  // One step: S(t), P(t), O += V(t) P(t); then tile t + 1 must be in LDS for
  // every wave.  Ring of 4: a wave's loads of tile t + 2 may stay in flight,
  // and tile t + 3 goes into the slot of tile t - 1, which every wave has
  // finished.  Ring of 2: tile t + 1 is the only one in flight, and tile
  // t + 2 goes into the slot of tile t, which every wave has just finished.
  // STEADY: a middle tile with at least kAhead tiles after it (the deeper
  // wait and the issue are unconditional: no per-tile scalar tests)
  auto step = [&](int t, auto first, auto last, auto track, auto steady) __attribute__((always_inline)) {
    S(t, first);
    softmax(t, first, last, track);
    PV(t);
    if (!decltype(last)::value) {
      if (decltype(steady)::value) {
        if (RING == 4) wait_vmcnt<kLoadsPerTile>();
        else wait_vmcnt<0>();
        __syncthreads();
        issue(t + kAhead);
      } else {
        if (RING == 4 && t + 2 < n_tiles) wait_vmcnt<kLoadsPerTile>();
        else wait_vmcnt<0>();
        __syncthreads();
        if (t + kAhead < n_tiles) issue(t + kAhead);
      }
    }
  };
  using kOn = std::true_type;
  using kOff = std::false_type;
  auto run_pass = [&](auto track) __attribute__((always_inline)) {
#pragma unroll
    for (int db = 0; db < 4; ++db) oacc[db] = f32x16{};
    l_run[0] = l_run[1] = l_run[2] = l_run[3] = 0.f;
    x_max = -INFINITY;
    rewind();
    const int n_pre = min(kAhead, n_tiles);
    for (int t = 0; t < n_pre; ++t) issue(t);
    // tile 0 in LDS
    if (n_pre == 3) wait_vmcnt<2 * kLoadsPerTile>();
    else if (n_pre == 2) wait_vmcnt<kLoadsPerTile>();
    else wait_vmcnt<0>();
    __syncthreads();
    if (n_tiles == 1) {
      step(0, kOn{}, kOn{}, track, kOff{});
    } else {
      step(0, kOn{}, kOff{}, track, kOff{});
      // no compiler-tracked load may still be pending when the loop starts:
      // its tracking would otherwise put a vmcnt wait (which also waits for
      // the tile loads in flight) at the top of every iteration.  (The short
      // shape's items are a few tiles long: there this wait would cost a
      // tile's load latency per item.)
      if constexpr (RING == 4) __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0), once per work item
      int t = 1;
      for (; t + kAhead < n_tiles; ++t) step(t, kOff{}, kOff{}, track, kOn{});
      for (; t + 1 < n_tiles; ++t) step(t, kOff{}, kOff{}, track, kOff{});
      step(n_tiles - 1, kOff{}, kOn{}, track, kOff{});
    }
  };

  // this lane's row: row sum (the lanes l and l + 32 hold halves) and x_max
  auto row_sum = [&]() __attribute__((always_inline)) {
    const float l_lane = (l_run[0] + l_run[1]) + (l_run[2] + l_run[3]);
    auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l_lane), __float_as_uint(l_lane), false, false);
    return __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
  };
  auto row_xmax = [&]() __attribute__((always_inline)) {
    auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x_max), __float_as_uint(x_max), false, false);
    return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
  };
  constexpr float kMaxSum = 18446744073709551616.0f;   // 2^kHeadroom
  if (n_tiles > 0) {
    run_pass(kOff{});
    const float l0 = row_sum();
    const bool over = !(l0 <= kMaxSum);   // also true for inf / NaN
    if (__builtin_amdgcn_ballot_w64(over) != 0 && lane == 0) redo_flag[0] = 1;
    __syncthreads();
    if (__builtin_amdgcn_readfirstlane(redo_flag[0]) != 0) {
      // finite sums: probabilities <= 1 after the shift (l >= 2^x_max)
      if (l0 > kMaxSum && l0 <= FLT_MAX) m_ref += __log2f(l0);
      for (int pass = 1;; ++pass) {
        run_pass(kOn{});
        if (pass == 2) break;
        const float xm = row_xmax();
        if (__builtin_amdgcn_ballot_w64(xm > kHeadroom) != 0 && lane == 0) redo_flag[1] = 1;
        __syncthreads();
        if (__builtin_amdgcn_readfirstlane(redo_flag[1]) == 0) break;
        m_ref += xm;   // the exact row max: every x <= 0
      }
    }
  } else {
#pragma unroll
    for (int db = 0; db < 4; ++db) oacc[db] = f32x16{};
    l_run[0] = l_run[1] = l_run[2] = l_run[3] = 0.f;
  }

  // ---- normalise and store
  const float l_tot = row_sum();
  if (piece >= 0) {
    // a piece: its unnormalised output (fp32), and the row's reference and
    // sum, for the merge kernel; rows past the request are written too (the
    // merge skips them)
    const int row = ((int)blockIdx.x - work.split_base) * BQ + 32 * wave + fr;
    float* po = work.part + (int64_t)row * D + 4 * fh;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        *reinterpret_cast<f32x4*>(po + 32 * db + 8 * i) =
            f32x4{oacc[db][4 * i], oacc[db][4 * i + 1], oacc[db][4 * i + 2], oacc[db][4 * i + 3]};
    if (fh == 0) {
      float* pm = work.part + (int64_t)work.split_n * BQ * D + 2 * (int64_t)row;
      pm[0] = m_ref;
      pm[1] = l_tot;
    }
    return;
  }
  const float inv = l_tot > 0.f ? 1.0f / l_tot : 0.f;   // no keys: output 0
  if (my_q < q_end) {
    bf16* op = O + (int64_t)my_q * os + head * D + 4 * fh;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        bf16x4 ov;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) ov[jj] = (bf16)(oacc[db][4 * i + jj] * inv);
        *reinterpret_cast<bf16x4*>(op + 32 * db + 8 * i) = ov;
      }
  }
}

// Merge of split items (256-query pieces of the 8-wave shape): row q of item
// it gets O = sum_p 2^(m_p - m) O_p / sum_p 2^(m_p - m) l_p over the pieces p
// that had keys (l_p > 0), with m their largest reference; O_p, m_p, l_p as
// the pieces wrote them (P = 2^(score - m_p), in log2 units).  One wave per
// row, two columns per lane.
__global__ __launch_bounds__(256) void attn_merge_kernel(bf16* __restrict__ O, int64_t os, const float* part,
                                                         int n_pieces, AttnWork work) {
  constexpr int BQ = 256;
  const int row = (int)blockIdx.x * 4 + (threadIdx.x >> 6);   // split item it, row rl
  const int lane = threadIdx.x & 63;
  const int S = work.split_s;
  const int it = row / BQ, rl = row - it * BQ;
  if (it >= n_pieces / S) return;
  const int r = work.split_req;
  const int local = work.split_first + it;
  const int head = local / work.tiles_q[r];
  const int qt = local - head * work.tiles_q[r];
  const int q = work.q_start[r] + qt * BQ + rl;
  if (q >= work.q_start[r] + work.q_len[r]) return;
  const float* ml = part + (int64_t)n_pieces * BQ * D;
  float m = -INFINITY;
  for (int p = 0; p < S; ++p) {
    const int64_t idx = (int64_t)(it * S + p) * BQ + rl;
    if (ml[2 * idx + 1] > 0.f) m = fmaxf(m, ml[2 * idx]);
  }
  float l = 0.f, o0 = 0.f, o1 = 0.f;
  for (int p = 0; p < S; ++p) {
    const int64_t idx = (int64_t)(it * S + p) * BQ + rl;
    const float lp = ml[2 * idx + 1];
    if (!(lp > 0.f)) continue;
    const float wp = exp2f(ml[2 * idx] - m);
    const float2 v = *reinterpret_cast<const float2*>(part + idx * D + 2 * lane);
    l = fmaf(wp, lp, l);
    o0 = fmaf(wp, v.x, o0);
    o1 = fmaf(wp, v.y, o1);
  }
  const float inv = l > 0.f ? 1.0f / l : 0.f;
  bf16x2 ov;
  ov[0] = (bf16)(o0 * inv);
  ov[1] = (bf16)(o1 * inv);
  *reinterpret_cast<bf16x2*>(O + (int64_t)q * os + head * D + 2 * lane) = ov;
}

// ------------------------------------------------------------------- fp32

// One thread per (query row, head); HD is a compile-time head size, so q and
// the output accumulator stay in registers and K, V rows are read as 16-byte
// vectors.  Online softmax in fp32.
template <int HD>
__global__ __launch_bounds__(64) void attn_fwd_f32(
    const float* __restrict__ Q, const float* __restrict__ K, const float* __restrict__ V,
    float* __restrict__ O, int64_t qs, int64_t ks, int64_t vs, int64_t os, int n_heads, float scale,
    ReqTable cq, ReqTable ck, int n_q) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n_q * n_heads) return;
  const int row = idx / n_heads;
  const int head = idx - row * n_heads;
  const int r = find_req(cq.cu, cq.n_req, row);
  const int kb = ck.cu[r], ke = ck.cu[r + 1];
  f32x4 q[HD / 4], acc[HD / 4];
  const f32x4* qp = reinterpret_cast<const f32x4*>(Q + (int64_t)row * qs + head * HD);
#pragma unroll
  for (int e = 0; e < HD / 4; ++e) {
    q[e] = qp[e];
    acc[e] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  float m = -INFINITY, l = 0.f;
  for (int j = kb; j < ke; ++j) {
    const f32x4* kp = reinterpret_cast<const f32x4*>(K + (int64_t)j * ks + head * HD);
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int e = 0; e < HD / 4; e += 2) {
      const f32x4 a = kp[e], b = kp[e + 1];
      s0 = fmaf(q[e][0], a[0], fmaf(q[e][1], a[1], fmaf(q[e][2], a[2], fmaf(q[e][3], a[3], s0))));
      s1 = fmaf(q[e + 1][0], b[0], fmaf(q[e + 1][1], b[1], fmaf(q[e + 1][2], b[2], fmaf(q[e + 1][3], b[3], s1))));
    }
    const float s = (s0 + s1) * scale;
    const float m_new = fmaxf(m, s);
    const float a = expf(m - m_new);
    const float p = expf(s - m_new);
    l = l * a + p;
    const f32x4* vp = reinterpret_cast<const f32x4*>(V + (int64_t)j * vs + head * HD);
#pragma unroll
    for (int e = 0; e < HD / 4; ++e) {
      const f32x4 v = vp[e];
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[e][c] = fmaf(p, v[c], acc[e][c] * a);
    }
    m = m_new;
  }
  f32x4* op = reinterpret_cast<f32x4*>(O + (int64_t)row * os + head * HD);
  const float inv = ke > kb ? 1.0f / l : 0.f;
#pragma unroll
  for (int e = 0; e < HD / 4; ++e) op[e] = acc[e] * inv;
}

}  // namespace

// Pieces of split work items (see launch_attention): at most kMaxPieces
// pieces of 256 rows, each its fp32 output [256][128], then the rows'
// reference and sum [256][2].  One array per GPU, held until the process
// ends; calls that split are serialised on it by an event (below).
constexpr int kMaxPieces = 256;
static __device__ __align__(256) float attn_part[kMaxPieces * (256 * D + 2 * 256)];

namespace {

std::atomic<int> g_split_mode{0};   // 0 per shape, 1 never, 2 or 4 forced
std::atomic<int> g_shape_mode{0};   // 0 per shape, 4 or 8 waves forced

struct SplitState {
  std::mutex mu;               // a call's enqueue from the event wait to the event record
  hipEvent_t done = nullptr;   // recorded after the last merge that read attn_part
  float* part = nullptr;       // device address of this GPU's attn_part
  bool used = false;
};

// This device's split state, created on first use (NULL if it cannot be).
SplitState* split_state() {
  static std::mutex mu;
  static SplitState* st[64] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!st[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(attn_part)) != hipSuccess || !ptr) {
      (void)hipGetLastError();
      return nullptr;
    }
    SplitState* x = new SplitState;
    x->part = (float*)ptr;
    if (hipEventCreateWithFlags(&x->done, hipEventDisableTiming) != hipSuccess) {
      (void)hipGetLastError();
      delete x;
      return nullptr;
    }
    st[dev] = x;
  }
  return st[dev];
}

struct Split {
  int s = 0;   // key pieces per split item (0: no split)
  int n = 0;   // split items: the last request's last n
};

// Work items of query tiles of bq rows: the requests with queries, longest
// key range first (their tiles do the most work).  Returns the largest key
// range.
int build_work(const int* cu_q, const int* cu_k, int n_req, int n_heads, int bq, AttnWork& w) {
  int order[DIT_MAX_REQ];
  int n = 0, max_k = 0;
  for (int r = 0; r < n_req; ++r)
    if (cu_q[r + 1] > cu_q[r]) {
      order[n++] = r;
      max_k = max(max_k, cu_k[r + 1] - cu_k[r]);
    }
  for (int i = 1; i < n; ++i) {
    int x = order[i], j = i - 1;
    int lx = cu_k[x + 1] - cu_k[x];
    while (j >= 0 && (cu_k[order[j] + 1] - cu_k[order[j]]) < lx) { order[j + 1] = order[j]; --j; }
    order[j + 1] = x;
  }
  w = AttnWork{};
  w.n_req = n;
  w.prefix[0] = 0;
  for (int i = 0; i < n; ++i) {
    int r = order[i];
    w.q_start[i] = cu_q[r];
    w.q_len[i] = cu_q[r + 1] - cu_q[r];
    w.k_start[i] = cu_k[r];
    w.k_len[i] = cu_k[r + 1] - cu_k[r];
    w.tiles_q[i] = (w.q_len[i] + bq - 1) / bq;
    w.prefix[i + 1] = w.prefix[i] + w.tiles_q[i] * n_heads;
  }
  return max_k;
}

// A launch of the 8-wave shape runs its items in rounds of one workgroup per
// compute unit.  When the last round is at most half full (a single request;
// at 720p 11,840 items on 256 CUs leave 64 for a 47th round), those items are
// split into 2 or 4 key pieces, so the last round is 1/2 or 1/4 as long.
// Counts only; the launcher drops the split under graph capture (the split
// serialises calls through an event recorded outside it).
Split plan_split(const AttnWork& w, int slots, int mode) {
  Split sp;
  if (mode == 1 || w.n_req < 1) return sp;
  const int n = w.n_req, last = n - 1;
  const int items = w.prefix[n], items_last = w.prefix[n] - w.prefix[last];
  const int kt_last = (w.k_len[last] + BKV - 1) / BKV;
  if (mode == 2 || mode == 4) {
    sp.s = mode;
    sp.n = min(items_last, slots / mode);
  } else if (n == 1) {
    const int rounds = (items + slots - 1) / slots;
    const int left = items - (rounds - 1) * slots;
    if (rounds >= 2 && left <= slots / 2) {
      sp.s = left <= slots / 4 ? 4 : 2;
      sp.n = left;
    }
  }
  if (sp.s == 0 || sp.n < 1 || sp.n > items_last || kt_last < 8 * sp.s || sp.n * sp.s > kMaxPieces)
    return Split{};
  return sp;
}

// Longest launch (in 64-key tiles of 256-query items, per compute unit) that
// takes the 4-wave shape instead of a split last round.
constexpr int kSmallLaunchTiles = 3 * 64;

// The shape and split of a bf16 attention launch on `slots` compute units.
// Key ranges up to kShortKeys take the 4-wave shape.  So does a single request
// whose 8-wave items would end in a split last round, when the launch is
// short (at most kSmallLaunchTiles key tiles per compute unit): there the
// pieces' fixed costs and their merge outweigh the 4-wave shape's 2-3% slower
// key tiles.  Measured (self-attention, 8-wave with its split against 4-wave):
// 4,096 tokens x 24 heads 198 against 177 us, 2,048 x 40 106 against 88 us,
// 4,096 x 40 309 against 289 us; but 6,144 x 24 (96-tile items) 397 against
// 405 us, and with a full last round the 8-wave shape is 2-3% faster.
AttnPlan plan_attention(const int* cu_q, const int* cu_k, int n_req, int n_heads, int slots, int split_mode,
                        int shape_mode, AttnWork& w) {
  AttnPlan pl;
  const int max_k = build_work(cu_q, cu_k, n_req, n_heads, 256, w);
  bool four = max_k <= kShortKeys;
  if (shape_mode == 4 || shape_mode == 8) {
    four = shape_mode == 4;
  } else if (!four && split_mode == 0 && slots > 0 && plan_split(w, slots, 0).s > 0) {
    int64_t tiles = 0;
    for (int i = 0; i < w.n_req; ++i)
      tiles += (int64_t)(w.prefix[i + 1] - w.prefix[i]) * ((w.k_len[i] + BKV - 1) / BKV);
    four = tiles <= (int64_t)kSmallLaunchTiles * slots;
  }
  if (four) {
    build_work(cu_q, cu_k, n_req, n_heads, 128, w);
    pl.waves = 4;
    return pl;
  }
  pl.waves = 8;
  if (slots > 0) {
    const Split sp = plan_split(w, slots, split_mode);
    pl.split_pieces = sp.s;
    pl.split_items = sp.n;
  }
  return pl;
}

}  // namespace

AttnPlan attention_plan(const int* cu_q, const int* cu_k, int n_req, int n_heads, int slots) {
  AttnWork w;
  return plan_attention(cu_q, cu_k, n_req, n_heads, slots, g_split_mode.load(std::memory_order_relaxed),
                        g_shape_mode.load(std::memory_order_relaxed), w);
}

void set_attention_split(int mode) { g_split_mode.store(mode, std::memory_order_relaxed); }
void set_attention_shape(int waves) { g_shape_mode.store(waves, std::memory_order_relaxed); }

hipError_t launch_attention(const AttnArgs& p, hipStream_t s) {
  const int n_req = p.cq.n_req;
  if (p.dtype == DIT_F32) {
    const int n_q = p.cq.cu[n_req];
    if (n_q == 0) return hipSuccess;
    const int total = n_q * p.n_heads;
    if (p.head_dim == 64)
      attn_fwd_f32<64><<<(total + 63) / 64, 64, 0, s>>>(
          (const float*)p.q, (const float*)p.k, (const float*)p.v, (float*)p.o, p.q_stride, p.k_stride,
          p.v_stride, p.o_stride, p.n_heads, p.scale, p.cq, p.ck, n_q);
    else
      attn_fwd_f32<128><<<(total + 63) / 64, 64, 0, s>>>(
          (const float*)p.q, (const float*)p.k, (const float*)p.v, (float*)p.o, p.q_stride, p.k_stride,
          p.v_stride, p.o_stride, p.n_heads, p.scale, p.cq, p.ck, n_q);
    return hipGetLastError();
  }
  AttnWork w;
  const AttnPlan pl = plan_attention(p.cq.cu, p.ck.cu, n_req, p.n_heads, cu_count(),
                                     g_split_mode.load(std::memory_order_relaxed),
                                     g_shape_mode.load(std::memory_order_relaxed), w);
  const bool short_keys = pl.waves == 4;
  const int n = w.n_req;
  const int items = w.prefix[n];
  if (items == 0) return hipSuccess;
  if (items > (1 << 27)) return hipErrorInvalidValue;   // keeps (xcd + 1) * n_r in range
  // each XCD's share of every request (see the kernel); the grid covers the largest
  auto grid_of = [](const AttnWork& wk) {
    int per_xcd = 0;
    for (int x = 0; x < kXcds; ++x) {
      int len = 0;
      for (int i = 0; i < wk.n_req; ++i) {
        const int n_r = wk.prefix[i + 1] - wk.prefix[i];
        len += (x + 1) * n_r / kXcds - x * n_r / kXcds;
      }
      per_xcd = len > per_xcd ? len : per_xcd;
    }
    return per_xcd * kXcds;
  };
  const float scale_log2 = p.scale * 1.4426950408889634f;
  const bf16* g = (const bf16*)p.q_gain;
  auto launch = [&](const AttnWork& wk, int grid) {
    if (grid <= 0) return;
#define DIT_ATTN_ARGS                                                                                          \
  (const bf16*)p.q, (const bf16*)p.k, (const bf16*)p.v, (bf16*)p.o, p.q_stride, p.k_stride, p.v_stride,        \
      p.o_stride, p.n_heads, scale_log2, g, p.q_eps, wk
    if (short_keys) {
      if (g) attn_fwd_bf16<4, 2, true><<<grid, 256, 0, s>>>(DIT_ATTN_ARGS);
      else attn_fwd_bf16<4, 2, false><<<grid, 256, 0, s>>>(DIT_ATTN_ARGS);
    } else {
      if (g) attn_fwd_bf16<8, 4, true><<<grid, 512, 0, s>>>(DIT_ATTN_ARGS);
      else attn_fwd_bf16<8, 4, false><<<grid, 512, 0, s>>>(DIT_ATTN_ARGS);
    }
  };
  Split sp;
  sp.s = pl.split_pieces;
  sp.n = pl.split_items;
  if (sp.s > 0) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone || !split_state()) {
      (void)hipGetLastError();
      sp = Split{};
    }
  }
  if (sp.s == 0) {
    launch(w, grid_of(w));
    return hipGetLastError();
  }
  // The last request's last n_split items as `split` key pieces each: their
  // workgroups follow all whole items in the same launch (so they fill the
  // compute units as the last whole items finish), then a merge kernel.
  const int split = sp.s, n_split = sp.n;
  const int last = n - 1;
  const int items_last = w.prefix[n] - w.prefix[last];
  AttnWork wp = w;
  wp.prefix[n] -= n_split;   // whole items: all but those
  if (n_split == items_last) wp.n_req = last;
  SplitState* st = split_state();   // exists: choose_split checked
  std::lock_guard<std::mutex> lock(st->mu);
  if (st->used) {
    const hipError_t e = hipStreamWaitEvent(s, st->done, 0);   // the previous call's merge has read the pieces
    if (e != hipSuccess) return e;
  }
  wp.split_s = split;
  wp.split_req = last;
  wp.split_first = items_last - n_split;
  wp.split_base = grid_of(wp);
  wp.split_n = n_split * split;
  wp.part = st->part;
  launch(wp, wp.split_base + wp.split_n);
  attn_merge_kernel<<<n_split * 256 / 4, 256, 0, s>>>((bf16*)p.o, p.o_stride, st->part, wp.split_n, wp);
  const hipError_t e = hipEventRecord(st->done, s);
  if (e != hipSuccess) return e;
  st->used = true;
#undef DIT_ATTN_ARGS
  return hipGetLastError();
}

}  // namespace dit
