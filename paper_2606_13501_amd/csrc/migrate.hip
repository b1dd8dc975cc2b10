// Layout-aware artifact migration: the transfer plan of one field (host) and
// a one-GPU executor that copies each entry's box from a source slice buffer
// into a destination slice buffer.
//
// A box's innermost dimension is contiguous in both dense slices, so the copy
// works in rows of the box: unit u is the widest power of two (<= 16 bytes)
// that divides the row length, both slices' row pitches and both base offsets,
// and consecutive lanes copy consecutive units of a row, rows following each
// other in the flattened (row, unit) index.
#include <stdarg.h>
#include <stdio.h>

#include <string>
#include <vector>

#include "common.hpp"
#include "dit_migrate.h"

namespace dit {
void set_last_error(const std::string& msg);
}

namespace {

dit_status mig_fail(dit_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  dit::set_last_error(buf);
  return st;
}

dit_status check_slices(const dit_mig_field* f, const dit_mig_slice* s, int n, const char* what) {
  if (n < 0) return mig_fail(DIT_ERR_INVALID_ARG, "n_%s = %d", what, n);
  if (n > 0 && !s) return mig_fail(DIT_ERR_INVALID_ARG, "%s slices are NULL", what);
  for (int i = 0; i < n; ++i)
    for (int d = 0; d < f->n_dims; ++d) {
      if (s[i].start[d] < 0 || s[i].start[d] > s[i].end[d] || s[i].end[d] > f->shape[d])
        return mig_fail(DIT_ERR_INVALID_ARG, "%s slice %d: [%lld, %lld) in dimension %d of extent %lld", what, i,
                        (long long)s[i].start[d], (long long)s[i].end[d], d, (long long)f->shape[d]);
      if (f->kind == DIT_MIG_REPLICATED && (s[i].start[d] != 0 || s[i].end[d] != f->shape[d]))
        return mig_fail(DIT_ERR_INVALID_ARG, "replicated field: %s slice %d does not cover the shape", what, i);
    }
  return DIT_OK;
}

dit_status check_field(const dit_mig_field* f) {
  if (!f) return mig_fail(DIT_ERR_INVALID_ARG, "field is NULL");
  if (f->kind != DIT_MIG_SHARDED && f->kind != DIT_MIG_REPLICATED && f->kind != DIT_MIG_METADATA)
    return mig_fail(DIT_ERR_INVALID_ARG, "kind %d", (int)f->kind);
  if (f->n_dims < 1 || f->n_dims > DIT_MIG_MAX_DIMS) return mig_fail(DIT_ERR_INVALID_ARG, "n_dims %d", f->n_dims);
  for (int d = 0; d < f->n_dims; ++d)
    if (f->shape[d] < 0) return mig_fail(DIT_ERR_INVALID_ARG, "shape[%d] = %lld", d, (long long)f->shape[d]);
  const int eb = f->elem_bytes;
  if (eb != 1 && eb != 2 && eb != 4 && eb != 8 && eb != 16)
    return mig_fail(DIT_ERR_INVALID_ARG, "elem_bytes %d", eb);
  if (f->kind != DIT_MIG_METADATA && f->n_src < 1 && f->n_dst > 0)
    return mig_fail(DIT_ERR_INVALID_ARG, "no source slices");
  const dit_status st = check_slices(f, f->src, f->n_src, "src");
  if (st != DIT_OK) return st;
  return check_slices(f, f->dst, f->n_dst, "dst");
}

void build_plan(const dit_mig_field* f, std::vector<dit_mig_entry>& out) {
  const int nd = f->n_dims;
  if (f->kind == DIT_MIG_METADATA) return;
  int64_t vol = 1;
  for (int d = 0; d < nd; ++d) vol *= f->shape[d];
  for (int j = 0; j < f->n_dst; ++j) {
    const dit_mig_slice& ds = f->dst[j];
    if (f->kind == DIT_MIG_REPLICATED) {
      int k = j % f->n_src;
      for (int i = 0; i < f->n_src; ++i)
        if (f->src[i].rank == ds.rank) { k = i; break; }
      dit_mig_entry e{};
      e.src_index = k; e.dst_index = j; e.src_rank = f->src[k].rank; e.dst_rank = ds.rank;
      for (int d = 0; d < nd; ++d) e.extent[d] = f->shape[d];
      e.bytes = vol * f->elem_bytes;
      out.push_back(e);
      continue;
    }
    for (int i = 0; i < f->n_src; ++i) {
      const dit_mig_slice& ss = f->src[i];
      dit_mig_entry e{};
      bool empty = false;
      int64_t n = 1;
      for (int d = 0; d < nd; ++d) {
        const int64_t lo = ss.start[d] > ds.start[d] ? ss.start[d] : ds.start[d];
        const int64_t hi = ss.end[d] < ds.end[d] ? ss.end[d] : ds.end[d];
        if (hi <= lo) { empty = true; break; }
        e.src_off[d] = lo - ss.start[d];
        e.dst_off[d] = lo - ds.start[d];
        e.extent[d] = hi - lo;
        n *= hi - lo;
      }
      if (empty) continue;
      e.src_index = i; e.dst_index = j; e.src_rank = ss.rank; e.dst_rank = ds.rank;
      e.bytes = n * f->elem_bytes;
      out.push_back(e);
    }
  }
}

// A box copy in units of U bytes: rows of `row_units` units; row r of the box
// (r over the product of the outer extents) starts at src_row(r), dst_row(r).
struct BoxCopy {
  int64_t rows, row_units;
  int64_t e1, e2;                      // extents of dimensions 1 and 2 (of the padded 4-D box)
  int64_t s_base, s_p0, s_p1, s_p2;    // source: base and pitches of dimensions 0..2, in units
  int64_t d_base, d_p0, d_p1, d_p2;
};

template <typename U>
__global__ __launch_bounds__(256) void box_copy_kernel(const U* __restrict__ src, U* __restrict__ dst, BoxCopy b) {
  const int64_t total = b.rows * b.row_units;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = idx / b.row_units, c = idx - r * b.row_units;
    const int64_t i2 = r % b.e2, i1 = (r / b.e2) % b.e1, i0 = r / (b.e2 * b.e1);
    dst[b.d_base + i0 * b.d_p0 + i1 * b.d_p1 + i2 * b.d_p2 + c] =
        src[b.s_base + i0 * b.s_p0 + i1 * b.s_p1 + i2 * b.s_p2 + c];
  }
}

template <typename U>
hipError_t launch_box(const void* src, void* dst, const BoxCopy& b, hipStream_t s) {
  const int64_t total = b.rows * b.row_units;
  if (total == 0) return hipSuccess;
  const int64_t blocks = (total + 255) / 256;
  box_copy_kernel<U><<<(unsigned)(blocks < 16384 ? blocks : 16384), 256, 0, s>>>((const U*)src, (U*)dst, b);
  return hipGetLastError();
}

}  // namespace

extern "C" dit_status dit_migration_plan(const dit_mig_field* f, dit_mig_entry* entries, int64_t capacity,
                                         int64_t* n_entries) {
  dit::set_last_error("");
  if (!n_entries) return mig_fail(DIT_ERR_INVALID_ARG, "n_entries is NULL");
  dit_status st = check_field(f);
  if (st != DIT_OK) return st;
  std::vector<dit_mig_entry> plan;
  build_plan(f, plan);
  *n_entries = (int64_t)plan.size();
  if ((int64_t)plan.size() > capacity || (!entries && !plan.empty()))
    return mig_fail(DIT_ERR_WORKSPACE, "plan has %lld entries, capacity %lld", (long long)plan.size(),
                    (long long)capacity);
  for (size_t k = 0; k < plan.size(); ++k) entries[k] = plan[k];
  return DIT_OK;
}

extern "C" dit_status dit_migration_execute(const dit_mig_field* f, const dit_mig_entry* entries, int64_t n,
                                            const void* const* src_bufs, void* const* dst_bufs,
                                            hipStream_t stream) {
  dit::set_last_error("");
  dit_status st = check_field(f);
  if (st != DIT_OK) return st;
  if (n < 0 || (n > 0 && (!entries || !src_bufs || !dst_bufs)))
    return mig_fail(DIT_ERR_INVALID_ARG, "entries or buffers are NULL");
  const int nd = f->n_dims, eb = f->elem_bytes;
  // validate every entry against its slices before launching anything
  for (int64_t k = 0; k < n; ++k) {
    const dit_mig_entry& e = entries[k];
    if (e.src_index < 0 || e.src_index >= f->n_src || e.dst_index < 0 || e.dst_index >= f->n_dst)
      return mig_fail(DIT_ERR_INVALID_ARG, "entry %lld: slice index out of range", (long long)k);
    const dit_mig_slice& ss = f->src[e.src_index];
    const dit_mig_slice& ds = f->dst[e.dst_index];
    for (int d = 0; d < nd; ++d)
      if (e.extent[d] < 0 || e.src_off[d] < 0 || e.dst_off[d] < 0 ||
          e.src_off[d] + e.extent[d] > ss.end[d] - ss.start[d] || e.dst_off[d] + e.extent[d] > ds.end[d] - ds.start[d])
        return mig_fail(DIT_ERR_INVALID_ARG, "entry %lld: box outside its slices in dimension %d", (long long)k, d);
    const void* sp = src_bufs[e.src_index];
    void* dp = dst_bufs[e.dst_index];
    if (!sp || !dp || ((uintptr_t)sp & 15u) || ((uintptr_t)dp & 15u))
      return mig_fail(DIT_ERR_INVALID_ARG, "entry %lld: buffer NULL or not 16-byte aligned", (long long)k);
  }
  for (int64_t k = 0; k < n; ++k) {
    const dit_mig_entry& e = entries[k];
    const dit_mig_slice& ss = f->src[e.src_index];
    const dit_mig_slice& ds = f->dst[e.dst_index];
    // pad to 4 dimensions (leading extents 1); slice extents and offsets in elements
    int64_t ext[4], so[4], dof[4], sx[4], dx[4];
    for (int d = 0; d < 4; ++d) {
      const int g = d - (4 - nd);
      ext[d] = g >= 0 ? e.extent[g] : 1;
      so[d] = g >= 0 ? e.src_off[g] : 0;
      dof[d] = g >= 0 ? e.dst_off[g] : 0;
      sx[d] = g >= 0 ? ss.end[g] - ss.start[g] : 1;
      dx[d] = g >= 0 ? ds.end[g] - ds.start[g] : 1;
    }
    // element pitches of dimensions 0..2 and base offsets
    const int64_t sp2 = sx[3], sp1 = sx[2] * sp2, sp0 = sx[1] * sp1;
    const int64_t dp2 = dx[3], dp1 = dx[2] * dp2, dp0 = dx[1] * dp1;
    const int64_t sbase = so[0] * sp0 + so[1] * sp1 + so[2] * sp2 + so[3];
    const int64_t dbase = dof[0] * dp0 + dof[1] * dp1 + dof[2] * dp2 + dof[3];
    // widest unit dividing every byte quantity of the copy
    int64_t g = ext[3] * eb;
    const int64_t q[6] = {sp2 * eb, sp1 * eb, dp2 * eb, dp1 * eb, sbase * eb, dbase * eb};
    int u = 16;
    auto divides = [&](int64_t v) { return v % u == 0; };
    while (u > 1) {
      bool ok = divides(g);
      for (int t = 0; t < 6; ++t) ok = ok && divides(q[t]);
      if (ok) break;
      u >>= 1;
    }
    BoxCopy b;
    b.rows = ext[0] * ext[1] * ext[2];
    b.row_units = ext[3] * eb / u;
    b.e1 = ext[1]; b.e2 = ext[2];
    b.s_base = sbase * eb / u; b.s_p0 = sp0 * eb / u; b.s_p1 = sp1 * eb / u; b.s_p2 = sp2 * eb / u;
    b.d_base = dbase * eb / u; b.d_p0 = dp0 * eb / u; b.d_p1 = dp1 * eb / u; b.d_p2 = dp2 * eb / u;
    if (b.rows == 0 || b.row_units == 0) continue;
    hipError_t err;
    const void* sp = src_bufs[e.src_index];
    void* dp = dst_bufs[e.dst_index];
    switch (u) {
      case 16: err = launch_box<uint4>(sp, dp, b, stream); break;
      case 8: err = launch_box<uint2>(sp, dp, b, stream); break;
      case 4: err = launch_box<uint32_t>(sp, dp, b, stream); break;
      case 2: err = launch_box<uint16_t>(sp, dp, b, stream); break;
      default: err = launch_box<uint8_t>(sp, dp, b, stream); break;
    }
    if (err != hipSuccess)
      return mig_fail(DIT_ERR_HIP, "box copy of entry %lld: %s", (long long)k, hipGetErrorString(err));
  }
  return DIT_OK;
}
