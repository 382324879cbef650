// Deterministic sparse update (replaces the paper's lock-free HOGWILD
// updates, Sec. 4): the contribution rows of a step are sorted by
// (table, row) with a stable radix sort, each run of equal keys is summed in
// position order, and row-wise Adagrad (Sec. 3.1: one accumulator per
// embedding row, summed over the row) is applied once per touched row.
// Long runs (hub rows of heavy-tailed graphs) are cut into pieces of PIECE
// positions that are summed in parallel, then combined in order: the result
// does not depend on scheduling.
#include "kernels.h"
#include "row_ops.h"

#define PIECE 32
#define SORT_IPT 16
#define SORT_TILE (256 * SORT_IPT)

namespace {

// ---------------------------------------------------------------- scan
// exclusive prefix sum of uint32 over tiles of SORT_TILE elements
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* tot, uint32_t* smem) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) smem[w] = x;
  __syncthreads();
  uint32_t base = 0, all = 0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) {
    if (i < w) base += smem[i];
    all += smem[i];
  }
  __syncthreads();
  *tot = all;
  return base + x - v;
}

__global__ __launch_bounds__(256) void scan_tile_sums(const uint32_t* in, int64_t n, uint32_t* sums) {
  __shared__ uint32_t smem[4];
  const int64_t base = (int64_t)blockIdx.x * SORT_TILE + (int64_t)threadIdx.x * SORT_IPT;
  uint32_t s = 0;
  for (int i = 0; i < SORT_IPT; ++i)
    if (base + i < n) s += in[base + i];
  uint32_t tot;
  block_exclusive_scan(s, &tot, smem);
  if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

// single workgroup: exclusive scan of up to any number of tile sums
__global__ __launch_bounds__(256) void scan_sums_inplace(uint32_t* sums, int nb) {
  __shared__ uint32_t smem[4];
  __shared__ uint32_t carry;
  if (threadIdx.x == 0) carry = 0;
  __syncthreads();
  for (int base = 0; base < nb; base += 256) {
    const int i = base + threadIdx.x;
    const uint32_t v = i < nb ? sums[i] : 0;
    uint32_t tot;
    const uint32_t ex = block_exclusive_scan(v, &tot, smem);
    if (i < nb) sums[i] = carry + ex;
    __syncthreads();
    if (threadIdx.x == 0) carry += tot;
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void scan_tiles(const uint32_t* in, int64_t n, const uint32_t* sums,
                                                  uint32_t* out, uint32_t* total) {
  __shared__ uint32_t smem[4];
  const int64_t base = (int64_t)blockIdx.x * SORT_TILE + (int64_t)threadIdx.x * SORT_IPT;
  uint32_t v[SORT_IPT];
  uint32_t s = 0;
  for (int i = 0; i < SORT_IPT; ++i) {
    v[i] = (base + i < n) ? in[base + i] : 0;
    s += v[i];
  }
  uint32_t tot;
  uint32_t run = sums[blockIdx.x] + block_exclusive_scan(s, &tot, smem);
  for (int i = 0; i < SORT_IPT; ++i) {
    if (base + i < n) out[base + i] = run;
    run += v[i];
  }
  if (total && blockIdx.x == gridDim.x - 1 && threadIdx.x == blockDim.x - 1) *total = run;
}

// ---------------------------------------------------------------- radix sort
__global__ __launch_bounds__(256) void radix_hist(const uint32_t* keys, int n, int shift, int nblocks,
                                                  uint32_t* hist) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int base = blockIdx.x * SORT_TILE;
  for (int r = 0; r < SORT_IPT; ++r) {
    const int idx = base + r * 256 + threadIdx.x;
    if (idx < n) atomicAdd(&h[(keys[idx] >> shift) & 255u], 1u);   // integer: order-free
  }
  __syncthreads();
  hist[(int64_t)threadIdx.x * nblocks + blockIdx.x] = h[threadIdx.x];
}

__global__ __launch_bounds__(256) void radix_scatter(const uint32_t* keys, const uint32_t* vals, int n,
                                                     int shift, int nblocks, const uint32_t* offs,
                                                     uint32_t* okeys, uint32_t* ovals) {
  __shared__ uint32_t run[256];
  __shared__ uint32_t wc[4][256];
  __shared__ uint32_t gofs[256];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  run[tid] = 0;
  for (int q = 0; q < 4; ++q) wc[q][tid] = 0;
  gofs[tid] = offs[(int64_t)tid * nblocks + blockIdx.x];
  __syncthreads();
  const unsigned long long lt = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
  const int base = blockIdx.x * SORT_TILE;
  for (int r = 0; r < SORT_IPT; ++r) {
    const int idx = base + r * 256 + tid;
    const bool valid = idx < n;
    const uint32_t key = valid ? keys[idx] : 0u;
    const uint32_t val = valid ? vals[idx] : 0u;
    const uint32_t dig = (key >> shift) & 255u;
    unsigned long long peers = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool on = (dig >> bit) & 1u;
      const unsigned long long bal = __ballot(on);
      peers &= on ? bal : ~bal;
    }
    const uint32_t rank = (uint32_t)__popcll(peers & lt);
    if (valid && rank == 0) wc[w][dig] = (uint32_t)__popcll(peers);
    __syncthreads();
    if (valid) {
      uint32_t off = run[dig] + rank;
      for (int q = 0; q < w; ++q) off += wc[q][dig];
      const uint32_t pos = gofs[dig] + off;
      okeys[pos] = key;
      ovals[pos] = val;
    }
    __syncthreads();
    run[tid] += wc[0][tid] + wc[1][tid] + wc[2][tid] + wc[3][tid];
    for (int q = 0; q < 4; ++q) wc[q][tid] = 0;
    __syncthreads();
  }
}

// ---------------------------------------------------------------- segments
__global__ void seg_flags(const uint32_t* keys, int n, uint32_t* flags) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    flags[i] = (i == 0 || keys[i] != keys[i - 1]) ? 1u : 0u;
}

// segment starts; piece flags (a piece starts at a segment start and every
// PIECE positions inside a segment)
__global__ void seg_starts(const uint32_t* flags, const uint32_t* segex, int n, uint32_t* seg_start) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    if (flags[i]) seg_start[segex[i]] = (uint32_t)i;
}

__global__ void piece_flags(const uint32_t* flags, const uint32_t* segex, const uint32_t* seg_start,
                            int n, uint32_t* pflags) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    const uint32_t sid = segex[i] + flags[i] - 1u;
    pflags[i] = ((uint32_t)i - seg_start[sid]) % PIECE == 0 ? 1u : 0u;
  }
}

__global__ void piece_starts(const uint32_t* pflags, const uint32_t* pex, const uint32_t* flags,
                             const uint32_t* segex, int n, uint32_t* piece_start,
                             uint32_t* seg_first_piece, const uint32_t* counts) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    if (pflags[i]) piece_start[pex[i]] = (uint32_t)i;
    if (flags[i]) seg_first_piece[segex[i]] = pex[i];
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    piece_start[counts[1]] = (uint32_t)n;
    seg_first_piece[counts[0]] = counts[1];
  }
}

// one wave per piece: in-order sum of its contribution rows
__global__ __launch_bounds__(256) void piece_sum(const uint32_t* vals, const float* rows, int64_t ld,
                                                 int width, const uint32_t* piece_start,
                                                 const uint32_t* counts, float* partial) {
  const int lane = threadIdx.x & 63;
  const uint32_t npieces = counts[1];
  for (uint32_t p = blockIdx.x * 4 + (threadIdx.x >> 6); p < npieces; p += gridDim.x * 4) {
    const uint32_t lo = piece_start[p], hi = piece_start[p + 1];
    for (int f0 = 0; f0 < width; f0 += 64 * ROWQ) {
      float acc[ROWQ];
#pragma unroll
      for (int q = 0; q < ROWQ; ++q) acc[q] = 0.0f;
      for (uint32_t i = lo; i < hi; ++i) {
        const float* row = rows + (int64_t)vals[i] * ld;
#pragma unroll
        for (int q = 0; q < ROWQ; ++q) {
          const int f = f0 + lane + 64 * q;
          if (f < width) acc[q] += row[f];
        }
      }
#pragma unroll
      for (int q = 0; q < ROWQ; ++q) {
        const int f = f0 + lane + 64 * q;
        if (f < width) partial[(int64_t)p * width + f] = acc[q];
      }
    }
  }
}

// one wave per touched entity row: g = sum of its pieces, then
//   G += |g|^2,  theta -= lr g / (sqrt(G) + eps)
__global__ __launch_bounds__(256) void entity_adagrad(StepGeom g, StepBufs b, const uint32_t* keys,
                                                      const uint32_t* seg_start,
                                                      const uint32_t* seg_first_piece,
                                                      const uint32_t* counts, const float* partial,
                                                      float lr) {
  const int lane = threadIdx.x & 63;
  const uint32_t nseg = counts[0];
  const int d = g.d;
  const uint32_t mask = (1u << g.rb) - 1u;
  for (uint32_t sgi = blockIdx.x * 4 + (threadIdx.x >> 6); sgi < nseg; sgi += gridDim.x * 4) {
    const uint32_t key = keys[seg_start[sgi]];
    const uint32_t tbl = key >> g.rb;
    const uint32_t row = key & mask;
    float* emb = (tbl ? b.emb_j : b.emb_i) + (int64_t)row * d;
    float* G = (tbl ? b.G_j : b.G_i) + row;
    Row acc;
    row_zero(acc);
    for (uint32_t p = seg_first_piece[sgi]; p < seg_first_piece[sgi + 1]; ++p) {
      Row part;
      row_load(part, partial + (int64_t)p * d, d, false, lane);
      row_add(acc, part);
    }
    const float gg = row_dot(acc, acc);
    const float Gn = *G + gg;
    const float scale = lr / (sqrtf(Gn) + PBG_EPS_ADAGRAD);
    Row th;
    row_load(th, emb, d, false, lane);
    row_axpy(th, -scale, acc);
#pragma unroll
    for (int q = 0; q < ROWQ; ++q)
      if (lane + 64 * q < d) emb[lane + 64 * q] = th.v[q];
    if (lane == 0) *G = Gn;
  }
}

// relations with several ids: element-wise Adagrad per relation segment
__global__ __launch_bounds__(256) void relation_adagrad_sorted(float* relp, float* relG, int dr,
                                                               const uint32_t* keys,
                                                               const uint32_t* seg_start,
                                                               const uint32_t* seg_first_piece,
                                                               const uint32_t* counts,
                                                               const float* partial, float lr) {
  const int lane = threadIdx.x & 63;
  const uint32_t nseg = counts[0];
  for (uint32_t sgi = blockIdx.x * 4 + (threadIdx.x >> 6); sgi < nseg; sgi += gridDim.x * 4) {
    const uint32_t r = keys[seg_start[sgi]];
    for (int f = lane; f < dr; f += 64) {
      float gsum = 0.0f;
      for (uint32_t p = seg_first_piece[sgi]; p < seg_first_piece[sgi + 1]; ++p)
        gsum += partial[(int64_t)p * dr + f];
      const int64_t o = (int64_t)r * dr + f;
      const float Gn = relG[o] + gsum * gsum;
      relG[o] = Gn;
      relp[o] -= lr * gsum / (sqrtf(Gn) + PBG_EPS_ADAGRAD);
    }
  }
}

// First level of the single-relation gradient sum: block (c, piece) adds, in
// a fixed order, the contribution rows of chunk c that fall in its piece of
// the chunk's row list (the Cc edge rows, then the U uniform rows when they
// carry relation gradient).  Spreading a chunk over RELSUM_PIECES blocks keeps
// enough waves in flight to stream the rows at HBM speed.
__global__ __launch_bounds__(256) void relation_chunk_sums(StepGeom g, const float* rows, int64_t ld,
                                                           int include_uniform, float* partial) {
  __shared__ float red[4][512];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = blockIdx.x;
  const int piece = blockIdx.y;
  const int Cc = chunk_edges(g, c);
  const int nrows = Cc + (include_uniform ? g.U : 0);
  const int per = (nrows + RELSUM_PIECES - 1) / RELSUM_PIECES;
  const int k0 = piece * per;
  const int k1 = min(nrows, k0 + per);
  const float* base = rows + (int64_t)c * g.N * ld;
  float acc[ROWQ];
#pragma unroll
  for (int q = 0; q < ROWQ; ++q) acc[q] = 0.0f;
#pragma unroll 4
  for (int k = k0 + w; k < k1; k += 4) {
    const int row = k < Cc ? k : g.C + (k - Cc);
    const float* r = base + (int64_t)row * ld;
#pragma unroll
    for (int q = 0; q < ROWQ; ++q) {
      const int f = lane + 64 * q;
      if (f < g.dr) acc[q] += r[f];
    }
  }
#pragma unroll
  for (int q = 0; q < ROWQ; ++q) {
    const int f = lane + 64 * q;
    if (f < g.dr) red[w][f] = acc[q];
  }
  __syncthreads();
  float* out = partial + ((int64_t)c * RELSUM_PIECES + piece) * g.dr;
  for (int f = threadIdx.x; f < g.dr; f += 256) out[f] = (red[0][f] + red[1][f]) + (red[2][f] + red[3][f]);
}

// Second level and element-wise Adagrad: 64 elements per block; wave w adds a
// contiguous quarter of the partial rows in order, then the four quarter sums
// are combined in a fixed order.
__global__ __launch_bounds__(256) void relation_single_adagrad(float* relp, float* relG, int width,
                                                               const float* partial, int nparts,
                                                               float lr) {
  __shared__ float red[4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int f = blockIdx.x * 64 + lane;
  const int per = (nparts + 3) / 4;
  const int p0 = w * per, p1 = min(nparts, p0 + per);
  float gsum = 0.0f;
  if (f < width) {
#pragma unroll 8
    for (int c = p0; c < p1; ++c) gsum += partial[(int64_t)c * width + f];
  }
  red[w][lane] = gsum;
  __syncthreads();
  if (w != 0 || f >= width) return;
  const float gt = (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
  const float Gn = relG[f] + gt * gt;
  relG[f] = Gn;
  relp[f] -= lr * gt / (sqrtf(Gn) + PBG_EPS_ADAGRAD);
}

int grid_for(int64_t n, int per_block, int cap) {
  int64_t b = (n + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (int)b;
}

}  // namespace

void launch_exclusive_scan(const uint32_t* in, int64_t n, uint32_t* out, uint32_t* tmp,
                           uint32_t* total, hipStream_t s) {
  const int nb = (int)((n + SORT_TILE - 1) / SORT_TILE);
  scan_tile_sums<<<nb, 256, 0, s>>>(in, n, tmp);
  scan_sums_inplace<<<1, 256, 0, s>>>(tmp, nb);
  scan_tiles<<<nb, 256, 0, s>>>(in, n, tmp, out, total);
}

void launch_radix_sort(uint32_t* keys, uint32_t* vals, int n, int bits, SortWork& w, hipStream_t s) {
  if (n <= 1 || bits <= 0) return;
  const int nblocks = (n + SORT_TILE - 1) / SORT_TILE;
  uint32_t* k_in = keys;
  uint32_t* v_in = vals;
  uint32_t* k_out = w.keys_alt;
  uint32_t* v_out = w.vals_alt;
  const int passes = (bits + 7) / 8;
  for (int p = 0; p < passes; ++p) {
    const int shift = 8 * p;
    radix_hist<<<nblocks, 256, 0, s>>>(k_in, n, shift, nblocks, w.hist);
    launch_exclusive_scan(w.hist, (int64_t)256 * nblocks, w.hist, w.scan_tmp, nullptr, s);
    radix_scatter<<<nblocks, 256, 0, s>>>(k_in, v_in, n, shift, nblocks, w.hist, k_out, v_out);
    uint32_t* t = k_in; k_in = k_out; k_out = t;
    t = v_in; v_in = v_out; v_out = t;
  }
  if (k_in != keys) {
    (void)hipMemcpyAsync(keys, k_in, (size_t)n * 4, hipMemcpyDeviceToDevice, s);
    (void)hipMemcpyAsync(vals, v_in, (size_t)n * 4, hipMemcpyDeviceToDevice, s);
  }
}

// builds segments (runs of equal sorted keys) and PIECE-long pieces, then
// sums every piece; leaves counts[0] = segments, counts[1] = pieces
static void build_and_sum_pieces(const uint32_t* keys, const uint32_t* vals, int n, const float* rows,
                                 int64_t ld, int width, SortWork& w, hipStream_t s) {
  const int gb = grid_for(n, 256, 4096);
  uint32_t* flags = w.flags;
  uint32_t* segex = w.keys_alt;     // the sort's ping-pong buffers are free here
  uint32_t* pflags = w.vals_alt;
  uint32_t* pex = w.piece_seg;
  seg_flags<<<gb, 256, 0, s>>>(keys, n, flags);
  launch_exclusive_scan(flags, n, segex, w.scan_tmp, w.counts + 0, s);
  seg_starts<<<gb, 256, 0, s>>>(flags, segex, n, w.seg_start);
  piece_flags<<<gb, 256, 0, s>>>(flags, segex, w.seg_start, n, pflags);
  launch_exclusive_scan(pflags, n, pex, w.scan_tmp, w.counts + 1, s);
  piece_starts<<<gb, 256, 0, s>>>(pflags, pex, flags, segex, n, w.piece_start, w.seg_first_piece,
                                  w.counts);
  piece_sum<<<grid_for(n, 4, 8192), 256, 0, s>>>(vals, rows, ld, width, w.piece_start, w.counts,
                                                  w.partial);
}

void launch_entity_update(const StepGeom& g, const StepBufs& b, int n, SortWork& w, float lr,
                          hipStream_t s) {
  if (n <= 0) return;
  build_and_sum_pieces(b.keys, b.vals, n, b.dn, g.dp, g.d, w, s);
  entity_adagrad<<<grid_for(n, 4, 8192), 256, 0, s>>>(g, b, b.keys, w.seg_start, w.seg_first_piece,
                                                       w.counts, w.partial, lr);
}

void launch_relation_update_sorted(const StepGeom& g, const StepBufs& b, int n, SortWork& w, float lr,
                                   hipStream_t s) {
  if (n <= 0) return;
  build_and_sum_pieces(b.rkeys, b.rvals, n, b.relc, g.dr, g.dr, w, s);
  relation_adagrad_sorted<<<grid_for(n, 4, 8192), 256, 0, s>>>(b.relp, b.relG, g.dr, b.rkeys,
                                                               w.seg_start, w.seg_first_piece,
                                                               w.counts, w.partial, lr);
}

void launch_relation_chunk_sums(const StepGeom& g, const float* rows, int64_t ld, int include_uniform,
                                float* partial, hipStream_t s) {
  relation_chunk_sums<<<dim3(g.nchunks, RELSUM_PIECES), 256, 0, s>>>(g, rows, ld, include_uniform, partial);
}

void launch_relation_single_adagrad(float* relp, float* relG, int width, const float* partial,
                                    int nparts, float lr, hipStream_t s) {
  relation_single_adagrad<<<(width + 63) / 64, 256, 0, s>>>(relp, relG, width, partial, nparts, lr);
}
