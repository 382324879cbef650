// Edge bucketing (Sec. 4.1): entities are split into P contiguous ranges of
// ps = ceil(n / P) ids, and edge (s, r, d) belongs to bucket
// b = part(s) * P + part(d).  The edges are grouped by b with a stable radix
// sort of (b, position) pairs, so the input order survives inside a bucket;
// bucket offsets are the lower bounds of each b in the sorted keys, and the
// local ids are gathered through the sorted positions.
#include "kernels.h"

namespace {

__global__ void bucket_keys_kernel(const int64_t* src, const int64_t* dst, int64_t n, int64_t ps,
                                   int P, uint32_t* keys, uint32_t* vals) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t pi = (uint32_t)(src[i] / ps);
    const uint32_t pj = (uint32_t)(dst[i] / ps);
    keys[i] = pi * (uint32_t)P + pj;
    vals[i] = (uint32_t)i;
  }
}

// offsets[b] = first position whose key is >= b, for b in [0, nb]
__global__ void bucket_offsets_kernel(const uint32_t* keys, int64_t n, int nb, int64_t* offsets) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b > nb) return;
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = lo + ((hi - lo) >> 1);
    if (keys[mid] < (uint32_t)b) lo = mid + 1;
    else hi = mid;
  }
  offsets[b] = lo;
}

__global__ void bucket_gather_kernel(const uint32_t* vals, const int64_t* src, const int32_t* rel,
                                     const int64_t* dst, int64_t n, int64_t ps, int32_t* src_local,
                                     int32_t* rel_out, int32_t* dst_local) {
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n;
       k += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = vals[k];
    const int64_t s = src[i], d = dst[i];
    src_local[k] = (int32_t)(s - (s / ps) * ps);
    dst_local[k] = (int32_t)(d - (d / ps) * ps);
    if (rel_out) rel_out[k] = rel ? rel[i] : 0;
  }
}

int grid_cap(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b < 1) b = 1;
  if (b > 16384) b = 16384;
  return (int)b;
}

}  // namespace

void launch_bucket_keys(const int64_t* src, const int64_t* dst, int64_t n, int64_t ps, int P,
                        uint32_t* keys, uint32_t* vals, hipStream_t s) {
  if (n <= 0) return;
  bucket_keys_kernel<<<grid_cap(n), 256, 0, s>>>(src, dst, n, ps, P, keys, vals);
}

void launch_bucket_offsets(const uint32_t* keys, int64_t n, int nb, int64_t* offsets, hipStream_t s) {
  bucket_offsets_kernel<<<(nb + 1 + 255) / 256, 256, 0, s>>>(keys, n, nb, offsets);
}

void launch_bucket_gather(const uint32_t* vals, const int64_t* src, const int32_t* rel,
                          const int64_t* dst, int64_t n, int64_t ps, int32_t* src_local,
                          int32_t* rel_out, int32_t* dst_local, hipStream_t s) {
  if (n <= 0) return;
  bucket_gather_kernel<<<grid_cap(n), 256, 0, s>>>(vals, src, rel, dst, n, ps, src_local, rel_out,
                                                   dst_local);
}
