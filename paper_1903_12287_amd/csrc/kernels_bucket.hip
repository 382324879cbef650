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

// ---- entity types: each relation's (partition size, entity count) of its
// source and destination type in geo[r * 4 .. r * 4 + 3].  Bit 4 of flag: a
// relation id out of range (its edge keyed with relation 0, never used), bits
// 1 / 2: a source / destination id out of its type's range.
__global__ void typed_bucket_keys_kernel(const int64_t* src, const int32_t* rel, const int64_t* dst, int64_t n,
                                         const int64_t* geo, int R, int P, uint32_t* keys, uint32_t* vals,
                                         uint32_t* flag) {
  uint32_t bad = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    int r = rel ? rel[i] : 0;
    if (r < 0 || r >= R) {
      bad |= 4u;
      r = 0;
    }
    const int64_t* gr = geo + (int64_t)r * 4;
    const int64_t s = src[i], d = dst[i];
    if (s < 0 || s >= gr[1]) bad |= 1u;
    if (d < 0 || d >= gr[3]) bad |= 2u;
    const int64_t ps = s < 0 || s >= gr[1] ? 0 : s / gr[0];
    const int64_t pd = d < 0 || d >= gr[3] ? 0 : d / gr[2];
    keys[i] = (uint32_t)(ps * P + pd);
    vals[i] = (uint32_t)i;
  }
  if (bad) atomicOr(flag, bad);
}

__global__ void typed_bucket_gather_kernel(const uint32_t* vals, const int64_t* src, const int32_t* rel,
                                           const int64_t* dst, int64_t n, const int64_t* geo, int32_t* src_local,
                                           int32_t* rel_out, int32_t* dst_local) {
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n;
       k += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = vals[k];
    const int r = rel ? rel[i] : 0;
    const int64_t* gr = geo + (int64_t)r * 4;
    const int64_t s = src[i], d = dst[i];
    src_local[k] = (int32_t)(s - (s / gr[0]) * gr[0]);
    dst_local[k] = (int32_t)(d - (d / gr[2]) * gr[2]);
    if (rel_out) rel_out[k] = r;
  }
}

// ---- direct counting sort (at most BUCKET_DIRECT_MAX buckets) -------------
// The edges are cut into tiles of BUCKET_TILE consecutive edges.  Pass 1 counts
// each tile's edges per bucket (and checks the ids); an exclusive scan over
// [bucket][tile] gives each tile its first output position per bucket.  Pass 2
// places the tile's edges in LDS in bucket order, keeping the input order
// inside a bucket (lanes of a wave are ranked by lane, waves and rounds in
// order), and then writes each bucket's run of the tile to consecutive
// positions, so the global writes are contiguous runs.
constexpr int BT_WAVES = BUCKET_TILE / 512;     // waves per tile, 512 edges (8 rounds) each

// part(v) = floor(v / ps) through a double reciprocal, corrected to exact
__device__ __forceinline__ int64_t part_of(int64_t v, int64_t ps, double inv_ps) {
  int64_t q = (int64_t)((double)v * inv_ps);
  if (q * ps > v) --q;
  else if ((q + 1) * ps <= v) ++q;
  return q;
}

// lanes of this wave whose key equals mine (keys < 2^bits, active lanes only)
__device__ __forceinline__ uint64_t match_key(uint32_t key, int bits, uint64_t active) {
  uint64_t m = active;
  for (int b = 0; b < bits; ++b) {
    const uint64_t on = __ballot((key >> b) & 1u);
    m &= ((key >> b) & 1u) ? on : ~on;
  }
  return m;
}

__global__ __launch_bounds__(BUCKET_TILE / 8) void bucket_count_kernel(const int64_t* src, const int64_t* dst,
                                                                       const int32_t* rel, int64_t n,
                                                                       int64_t n_ent, int32_t n_rel, int64_t ps,
                                                                       double inv_ps, int P, int bits,
                                                                       int64_t tiles, uint32_t* hist,
                                                                       uint32_t* flag) {
  __shared__ uint32_t cnt[BUCKET_DIRECT_MAX];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nb = P * P;
  const int64_t tile = blockIdx.x;
  for (int b = threadIdx.x; b < nb; b += blockDim.x) cnt[b] = 0u;
  __syncthreads();
  const int64_t e0 = tile * BUCKET_TILE + (int64_t)w * 512, e1 = min(n, e0 + 512);
  uint32_t bad = 0u;
  for (int64_t r = e0; r < e1; r += 64) {
    const int64_t i = r + lane;
    const bool act = i < e1;
    uint32_t key = 0u;
    if (act) {
      const int64_t s = src[i], d = dst[i];
      if (s < 0 || s >= n_ent) bad |= 1u;
      if (d < 0 || d >= n_ent) bad |= 2u;
      if (rel) {
        const int32_t q = rel[i];
        if (q < 0 || q >= n_rel) bad |= 4u;
      }
      const int64_t pi = part_of(min(max(s, (int64_t)0), n_ent - 1), ps, inv_ps);
      const int64_t pj = part_of(min(max(d, (int64_t)0), n_ent - 1), ps, inv_ps);
      key = (uint32_t)(pi * P + pj);
    }
    const uint64_t m = match_key(key, bits, __ballot(act));
    // the lowest lane of each key adds the key's count
    if (act && (m & ((1ull << lane) - 1ull)) == 0ull) atomicAdd(&cnt[key], (uint32_t)__popcll(m));
  }
  if (bad) atomicOr(flag, bad);
  __syncthreads();
  for (int b = threadIdx.x; b < nb; b += blockDim.x) hist[(int64_t)b * tiles + tile] = cnt[b];
}

__global__ __launch_bounds__(BUCKET_TILE / 8) void bucket_scatter_kernel(const int64_t* src, const int64_t* dst,
                                                                         const int32_t* rel, int64_t n,
                                                                         int64_t ps, double inv_ps, int P, int bits,
                                                                         int64_t tiles, const uint32_t* start,
                                                                         int32_t* src_local, int32_t* rel_out,
                                                                         int32_t* dst_local) {
  __shared__ int32_t t_sl[BUCKET_TILE], t_dl[BUCKET_TILE], t_rq[BUCKET_TILE];
  __shared__ uint8_t t_key[BUCKET_TILE];
  __shared__ uint32_t wcnt[BT_WAVES][BUCKET_DIRECT_MAX];   // per wave, then the wave's base in the tile
  __shared__ uint32_t koff[BUCKET_DIRECT_MAX];              // first tile slot of each bucket
  __shared__ uint32_t gpos[BUCKET_DIRECT_MAX];              // first output position of each bucket's run
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int nb = P * P;
  const int64_t tile = blockIdx.x;
  for (int b = threadIdx.x; b < nb; b += blockDim.x) {
#pragma unroll
    for (int q = 0; q < BT_WAVES; ++q) wcnt[q][b] = 0u;
    gpos[b] = start[(int64_t)b * tiles + tile];
  }
  __syncthreads();
  // rounds of this wave: keys, local ids and rank among the wave's earlier
  // edges of the same bucket
  const int64_t e0 = tile * BUCKET_TILE + (int64_t)w * 512;
  uint32_t key[8], rank[8];
  int32_t sl[8], dl[8], rq[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    const int64_t i = e0 + 64 * u + lane;
    const bool act = i < n;
    key[u] = 0u;
    sl[u] = dl[u] = rq[u] = 0;
    if (act) {
      const int64_t s = src[i], d = dst[i];
      const int64_t pi = part_of(s, ps, inv_ps), pj = part_of(d, ps, inv_ps);
      key[u] = (uint32_t)(pi * P + pj);
      sl[u] = (int32_t)(s - pi * ps);
      dl[u] = (int32_t)(d - pj * ps);
      rq[u] = rel ? rel[i] : 0;
    }
    const uint64_t m = match_key(key[u], bits, __ballot(act));
    const uint64_t below = m & ((1ull << lane) - 1ull);
    rank[u] = act ? wcnt[w][key[u]] + (uint32_t)__popcll(below) : 0xFFFFFFFFu;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    if (act && below == 0ull) wcnt[w][key[u]] += (uint32_t)__popcll(m);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  }
  __syncthreads();
  // per bucket: the waves' bases inside the bucket, then the buckets' bases in
  // the tile (exclusive scan over the buckets)
  for (int b = threadIdx.x; b < nb; b += blockDim.x) {
    uint32_t run = 0u;
#pragma unroll
    for (int q = 0; q < BT_WAVES; ++q) {
      const uint32_t c = wcnt[q][b];
      wcnt[q][b] = run;
      run += c;
    }
    koff[b] = run;   // bucket total for now
  }
  __syncthreads();
  if (w == 0) {
    // exclusive scan of the bucket totals by one wave, four buckets per lane
    uint32_t c[BUCKET_DIRECT_MAX / 64];
    uint32_t sum = 0u;
#pragma unroll
    for (int q = 0; q < BUCKET_DIRECT_MAX / 64; ++q) {
      const int b = (BUCKET_DIRECT_MAX / 64) * lane + q;
      c[q] = b < nb ? koff[b] : 0u;
      sum += c[q];
    }
    uint32_t inc = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(inc, o, 64);
      if (lane >= o) inc += y;
    }
    uint32_t run = inc - sum;
#pragma unroll
    for (int q = 0; q < BUCKET_DIRECT_MAX / 64; ++q) {
      const int b = (BUCKET_DIRECT_MAX / 64) * lane + q;
      if (b < nb) koff[b] = run;
      run += c[q];
    }
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < 8; ++u) {
    if (rank[u] == 0xFFFFFFFFu) continue;
    const uint32_t slot = koff[key[u]] + wcnt[w][key[u]] + rank[u];
    t_sl[slot] = sl[u];
    t_dl[slot] = dl[u];
    t_rq[slot] = rq[u];
    t_key[slot] = (uint8_t)key[u];
  }
  __syncthreads();
  const int tn = (int)min((int64_t)BUCKET_TILE, n - tile * BUCKET_TILE);
  for (int p = threadIdx.x; p < tn; p += blockDim.x) {
    const uint32_t b = t_key[p];
    const uint32_t o = gpos[b] + ((uint32_t)p - koff[b]);
    src_local[o] = t_sl[p];
    dst_local[o] = t_dl[p];
    if (rel_out) rel_out[o] = t_rq[p];
  }
}

// offsets[b] = first output position of bucket b (the scanned count of its
// first tile), offsets[nb] = n
__global__ void bucket_direct_offsets_kernel(const uint32_t* start, int64_t tiles, int nb, int64_t n,
                                             int64_t* offsets) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b > nb) return;
  offsets[b] = b == nb ? n : (tiles == 0 ? 0 : (int64_t)start[(int64_t)b * tiles]);
}

int grid_cap(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b < 1) b = 1;
  if (b > 16384) b = 16384;
  return (int)b;
}

}  // namespace

int64_t bucket_direct_units(int64_t n) { return (n + BUCKET_TILE - 1) / BUCKET_TILE; }

static int key_bits_of(int nb) {
  int b = 0;
  while ((1 << b) < nb) ++b;
  return b;
}

void launch_bucket_count(const int64_t* src, const int64_t* dst, const int32_t* rel, int64_t n, int64_t n_ent,
                         int32_t n_rel, int64_t ps, int P, uint32_t* hist, uint32_t* flag, hipStream_t s) {
  const int64_t tiles = bucket_direct_units(n);
  if (tiles == 0) return;
  bucket_count_kernel<<<(unsigned)tiles, BUCKET_TILE / 8, 0, s>>>(src, dst, rel, n, n_ent, n_rel, ps,
                                                                  1.0 / (double)ps, P, key_bits_of(P * P), tiles,
                                                                  hist, flag);
}

void launch_bucket_scatter(const int64_t* src, const int64_t* dst, const int32_t* rel, int64_t n, int64_t ps,
                           int P, const uint32_t* start, int64_t* offsets, int32_t* src_local,
                           int32_t* rel_out, int32_t* dst_local, hipStream_t s) {
  const int64_t tiles = bucket_direct_units(n);
  const int nb = P * P;
  bucket_direct_offsets_kernel<<<(nb + 1 + 255) / 256, 256, 0, s>>>(start, tiles, nb, n, offsets);
  if (tiles == 0) return;
  bucket_scatter_kernel<<<(unsigned)tiles, BUCKET_TILE / 8, 0, s>>>(src, dst, rel, n, ps, 1.0 / (double)ps, P,
                                                                    key_bits_of(nb), tiles, start, src_local,
                                                                    rel_out, dst_local);
}

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

void launch_typed_bucket_keys(const int64_t* src, const int32_t* rel, const int64_t* dst, int64_t n,
                              const int64_t* geo, int R, int P, uint32_t* keys, uint32_t* vals, uint32_t* flag,
                              hipStream_t s) {
  if (n <= 0) return;
  typed_bucket_keys_kernel<<<grid_cap(n), 256, 0, s>>>(src, rel, dst, n, geo, R, P, keys, vals, flag);
}

void launch_typed_bucket_gather(const uint32_t* vals, const int64_t* src, const int32_t* rel, const int64_t* dst,
                                int64_t n, const int64_t* geo, int32_t* src_local, int32_t* rel_out,
                                int32_t* dst_local, hipStream_t s) {
  if (n <= 0) return;
  typed_bucket_gather_kernel<<<grid_cap(n), 256, 0, s>>>(vals, src, rel, dst, n, geo, src_local, rel_out,
                                                          dst_local);
}
