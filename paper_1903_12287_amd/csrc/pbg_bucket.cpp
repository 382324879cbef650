// pbg_bucket_edges: edge bucketing on the device (Sec. 4.1).
//
// Up to BUCKET_DIRECT_MAX buckets: a counting sort in two passes over the ids
// (count per bucket and unit of consecutive edges, with the range checks;
// after a scan, write each edge's local ids at its stable position), with
// 8 bytes per bucket and unit of work memory.  More buckets: range check of
// every id first, then bucket keys b = part(src) * P + part(dst), a stable
// radix sort of (b, position), bucket offsets by lower bound, and the local
// ids gathered in sorted order (16 bytes per edge of sort buffers).  Either
// way nothing is written on an error, and the work memory is allocated for
// the call and released before it returns.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>

#include "kernels.h"
#include "runtime_internal.h"

namespace {

struct DevBuf {
  std::vector<void*> ptrs;
  bool failed = false;
  void* get(size_t bytes) {
    void* p = nullptr;
    if (hipMalloc(&p, std::max<size_t>(bytes, 16)) != hipSuccess) {
      (void)hipGetLastError();
      failed = true;
      return nullptr;
    }
    ptrs.push_back(p);
    return p;
  }
  ~DevBuf() {
    for (void* p : ptrs) (void)hipFree(p);
  }
};

int key_bits(uint64_t max_key) {
  int b = 0;
  while (b < 32 && (max_key >> b) != 0) ++b;
  return b;
}

}  // namespace

extern "C" pbg_status pbg_bucket_edges(pbg_ctx* ctx, const int64_t* src, const int32_t* rel,
                                       const int64_t* dst, int64_t n, int64_t* offsets,
                                       int32_t* src_local, int32_t* rel_out, int32_t* dst_local) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  ctx->err.clear();
  if (n < 0 || n > 0x7FFFFFFFll) return set_err(ctx, PBG_ERR_INVALID_ARG, "n must be in [0, 2^31 - 1]");
  if (!offsets) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL offsets");
  if (n > 0 && (!src || !dst || !src_local || !dst_local))
    return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL edge array");
  const int P = ctx->P;
  const int nb = P * P;
  if (nb > (1 << 24)) return set_err(ctx, PBG_ERR_UNSUPPORTED, "too many buckets");
  if (ctx->T > 1) return bucket_edges_typed(ctx, src, rel, dst, n, offsets, src_local, rel_out, dst_local);
  hipStream_t s = ctx->cs;
  DevBuf buf;
  if (nb <= BUCKET_DIRECT_MAX) {
    // counting sort: count per (bucket, unit) with the id checks, scan, and
    // write the local ids at their positions (no key or position arrays)
    const int64_t units = bucket_direct_units(n);
    const int64_t nh = (int64_t)nb * units;
    uint32_t* flag = (uint32_t*)buf.get(16);
    uint32_t* hist = (uint32_t*)buf.get((size_t)nh * 4);
    uint32_t* start = (uint32_t*)buf.get((size_t)nh * 4);
    uint32_t* tmp = (uint32_t*)buf.get((size_t)exclusive_scan_tmp_entries(nh) * 4);
    if (buf.failed)
      return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "bucketing workspace (%lld edges) could not be allocated",
                     (long long)n);
    hipError_t e = hipMemsetAsync(flag, 0, 4, s);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipMemsetAsync");
    launch_bucket_count(src, dst, rel, n, ctx->n, ctx->R, ctx->ps, P, hist, flag, s);
    if (nh > 0) launch_exclusive_scan(hist, nh, start, tmp, nullptr, s);
    uint32_t hflag = 0;
    e = hipMemcpyAsync(&hflag, flag, 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(ctx, e, "bucket counts");
    if (hflag & 3u)
      return set_err(ctx, PBG_ERR_INVALID_ARG, "an entity id is outside [0, %lld)", (long long)ctx->n);
    if (hflag & 4u) return set_err(ctx, PBG_ERR_INVALID_ARG, "a relation id is outside [0, %d)", ctx->R);
    launch_bucket_scatter(src, dst, rel, n, ctx->ps, P, start, offsets, src_local, rel_out, dst_local, s);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(ctx, e, "bucketing");
    return PBG_OK;
  }
  uint32_t* flag = (uint32_t*)buf.get(16);
  uint32_t* keys = (uint32_t*)buf.get((size_t)n * 4);
  uint32_t* vals = (uint32_t*)buf.get((size_t)n * 4);
  SortWork w;
  memset(&w, 0, sizeof(w));
  w.keys_alt = (uint32_t*)buf.get((size_t)n * 4);
  w.vals_alt = (uint32_t*)buf.get((size_t)n * 4);
  w.hist = (uint32_t*)buf.get((size_t)radix_hist_entries(n) * 4);
  w.scan_tmp = (uint32_t*)buf.get((size_t)radix_scan_tmp_entries(n) * 4);
  w.max_n = (int)n;
  if (buf.failed)
    return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "bucketing workspace (%lld edges) could not be allocated",
                   (long long)n);
  hipError_t e = hipMemsetAsync(flag, 0, 4, s);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipMemsetAsync");
  launch_check_ids64(src, n, ctx->n, flag, 1u, s);
  launch_check_ids64(dst, n, ctx->n, flag, 2u, s);
  if (rel) launch_check_ids(rel, n, ctx->R, flag, 4u, s);
  uint32_t hflag = 0;
  e = hipMemcpyAsync(&hflag, flag, 4, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(ctx, e, "id range check");
  if (hflag & 3u) return set_err(ctx, PBG_ERR_INVALID_ARG, "an entity id is outside [0, %lld)", (long long)ctx->n);
  if (hflag & 4u) return set_err(ctx, PBG_ERR_INVALID_ARG, "a relation id is outside [0, %d)", ctx->R);

  launch_bucket_keys(src, dst, n, ctx->ps, P, keys, vals, s);
  launch_radix_sort(keys, vals, (int)n, key_bits((uint64_t)nb - 1), w, s);
  launch_bucket_offsets(keys, n, nb, offsets, s);
  launch_bucket_gather(vals, src, rel, dst, n, ctx->ps, src_local, rel_out, dst_local, s);
  e = hipGetLastError();
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(ctx, e, "bucketing");
  return PBG_OK;
}
