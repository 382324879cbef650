// Deterministic sparse update (replaces the paper's lock-free HOGWILD
// updates, Sec. 4): the contribution rows of a step are sorted by
// (table, row) with a stable radix sort, each run of equal keys (a segment)
// is summed in position order, and row-wise Adagrad (Sec. 3.1: one
// accumulator per embedding row, summed over the row) is applied once per
// touched row.
//
// The sorted positions are cut into fixed blocks of SEG_BLOCK.  A wave per block sums
// every piece of the block (a piece = the positions of one segment inside the
// block) in position order; a segment that lies inside one block is updated
// there and then.  A segment that crosses block boundaries (a hub row of a
// heavy-tailed graph) leaves one partial sum per block it touches, and the
// wave of the block where it starts adds them in block order and updates it.
// No scan or compaction is needed, and the summation order is fixed, so the
// result does not depend on scheduling.
#include "kernels.h"
#include "row_ops.h"

// scan tiles and radix-sort tiles: SORT_IPT * 256 values per workgroup
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
// Sorts of several independent segments run as one launch: segment
// blockIdx.y holds n_full keys at keys + y * stride (the last n_last), with
// its own digit counts at hist + y * 256 * nblocks.
struct SortSeg {
  int64_t stride;
  int n_full, n_last, nseg;
  __device__ __forceinline__ int n(int y) const { return y == nseg - 1 ? n_last : n_full; }
};

// Per-block digit counts; each thread loads its IPT keys up front.
template <int IPT>
__global__ __launch_bounds__(256) void radix_hist(const uint32_t* keys, SortSeg sg, int shift, int nblocks,
                                                  uint32_t* hist) {
  __shared__ uint32_t h[256];
  const int n = sg.n(blockIdx.y);
  keys += blockIdx.y * sg.stride;
  hist += (int64_t)blockIdx.y * 256 * nblocks;
  h[threadIdx.x] = 0;
  const int base = blockIdx.x * (256 * IPT);
  uint32_t k[IPT];
#pragma unroll
  for (int r = 0; r < IPT; ++r) {
    const int idx = base + r * 256 + threadIdx.x;
    k[r] = idx < n ? keys[idx] : 0u;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < IPT; ++r) {
    const int idx = base + r * 256 + threadIdx.x;
    if (idx < n) atomicAdd(&h[(k[r] >> shift) & 255u], 1u);   // integer: order-free
  }
  __syncthreads();
  hist[(int64_t)threadIdx.x * nblocks + blockIdx.x] = h[threadIdx.x];
}

// Stable scatter.  Wave w of a block owns the 64 * IPT consecutive keys
// base + w * 64 IPT ..., walked 64 at a time in order: wave ballots over
// the digit bits rank each key among the equal digits of its round, a per-wave
// count per digit carries the rank across rounds, and after one barrier the
// waves' counts give each wave its base per digit (earlier waves first).
// Keys and values are loaded up front.  RAW: `offs` holds the raw digit
// counts [256][nblocks] (nblocks <= 64) and every block derives its own first
// position per digit from them (its digit's earlier blocks, plus a block scan
// of the digit totals), so no separate scan launch is needed.
template <int IPT, bool RAW>
__global__ __launch_bounds__(256) void radix_scatter(const uint32_t* keys, const uint32_t* vals, SortSeg sg,
                                                     int shift, int nblocks, const uint32_t* offs,
                                                     uint32_t* okeys, uint32_t* ovals) {
  __shared__ uint32_t smem[4];
  const int n = sg.n(blockIdx.y);
  {
    const int64_t o = blockIdx.y * sg.stride;
    keys += o;
    vals += o;
    okeys += o;
    ovals += o;
    offs += (int64_t)blockIdx.y * 256 * nblocks;
  }
  constexpr int R = IPT;                     // rounds of 64 keys per wave (a quarter of the tile)
  __shared__ uint32_t cnt[4][256];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int base = blockIdx.x * (256 * IPT) + w * (64 * R);
  uint32_t kr[R], vr[R], rk[R];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int idx = base + r * 64 + lane;
    kr[r] = idx < n ? keys[idx] : 0u;
    vr[r] = idx < n ? vals[idx] : 0u;
  }
  uint32_t first;   // first output position of digit tid in this block
  if (RAW) {
    const uint32_t* hrow = offs + (int64_t)tid * nblocks;
    uint32_t v[64];
#pragma unroll
    for (int i = 0; i < 64; ++i) v[i] = i < nblocks ? hrow[i] : 0u;
    uint32_t tot = 0u, pre = 0u;
#pragma unroll
    for (int i = 0; i < 64; ++i) {
      tot += v[i];
      if (i < (int)blockIdx.x) pre += v[i];
    }
    uint32_t all;
    first = block_exclusive_scan(tot, &all, smem) + pre;
  } else {
    first = offs[(int64_t)tid * nblocks + blockIdx.x];
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) cnt[q][tid] = 0u;
  __syncthreads();
  const unsigned long long lt = (lane == 0) ? 0ull : ((~0ull) >> (64 - lane));
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const bool valid = base + r * 64 + lane < n;
    const uint32_t dig = (kr[r] >> shift) & 255u;
    unsigned long long peers = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool on = (dig >> bit) & 1u;
      const unsigned long long bal = __ballot(on);
      peers &= on ? bal : ~bal;
    }
    const uint32_t below = (uint32_t)__popcll(peers & lt);
    rk[r] = valid ? cnt[w][dig] + below : 0u;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    if (valid && below == 0u) cnt[w][dig] += (uint32_t)__popcll(peers);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  }
  __syncthreads();
  {
    // digit tid: each wave's first output position
    uint32_t run = first;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t c = cnt[q][tid];
      cnt[q][tid] = run;
      run += c;
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < R; ++r) {
    if (base + r * 64 + lane >= n) continue;
    const uint32_t pos = cnt[w][(kr[r] >> shift) & 255u] + rk[r];
    okeys[pos] = kr[r];
    ovals[pos] = vr[r];
  }
}


// ---------------------------------------------------------------- segments
enum { SEG_ENTITY = 0, SEG_RELATION = 1 };

// applies the summed gradient g of the segment with key `key`
template <int MODE, int RQ>
__device__ __forceinline__ void seg_apply(const StepGeom& g, const StepBufs& b, uint32_t key,
                                          const RowT<RQ>& acc, int width, float lr, int lane) {
  if (MODE == SEG_ENTITY) {
    const uint32_t tbl = key >> g.rb;
    const uint32_t row = key & ((1u << g.rb) - 1u);
    float* emb = (tbl ? b.emb_j : b.emb_i) + (int64_t)row * g.d;
    float* G = (tbl ? b.G_j : b.G_i) + row;
    const float gg = row_dot(acc, acc);
    const float Gn = *G + gg;
    const float scale = lr * adagrad_rcp(Gn);
#pragma unroll
    for (int q = 0; q < RQ; ++q) {
      const int f = lane + 64 * q;
      if (f < g.d) emb[f] -= scale * acc.v[q];
    }
    if (lane == 0) *G = Gn;
  } else {
    float* p = b.relp + (int64_t)key * width;
    float* G = b.relG + (int64_t)key * width;
#pragma unroll
    for (int q = 0; q < RQ; ++q) {
      const int f = lane + 64 * q;
      if (f < width) {
        const float gf = acc.v[q];
        const float Gn = G[f] + gf * gf;
        G[f] = Gn;
        p[f] -= lr * gf * adagrad_rcp(Gn);
      }
    }
  }
}

// Rows as RQ contiguous floats per lane (lane L holds elements RQ L .. RQ L +
// RQ - 1): one 8- or 16-byte access per lane instead of RQ strided ones.  vec:
// the row pitch and the width are multiples of RQ (the row starts are then
// aligned for the vector access); the lane holding the width's end, and every
// lane when vec is false, moves element by element.
template <int RQ>
__device__ __forceinline__ void crow_load(float (&v)[RQ], const float* r, int lane, int width, bool vec) {
  const int f0 = RQ * lane;
  if (vec && f0 + RQ <= width) {
    if (RQ == 2) {
      const float2 x = *(const float2*)(r + f0);
      v[0] = x.x;
      v[1] = x.y;
    } else {
#pragma unroll
      for (int c = 0; c < RQ / 4; ++c) {
        const float4 x = *(const float4*)(r + f0 + 4 * c);
        v[4 * c] = x.x;
        v[4 * c + 1] = x.y;
        v[4 * c + 2] = x.z;
        v[4 * c + 3] = x.w;
      }
    }
  } else {
#pragma unroll
    for (int q = 0; q < RQ; ++q) v[q] = f0 + q < width ? r[f0 + q] : 0.0f;
  }
}

template <int RQ>
__device__ __forceinline__ void crow_store(float* r, const float (&v)[RQ], int lane, int width, bool vec) {
  const int f0 = RQ * lane;
  if (vec && f0 + RQ <= width) {
    if (RQ == 2) {
      *(float2*)(r + f0) = make_float2(v[0], v[1]);
    } else {
#pragma unroll
      for (int c = 0; c < RQ / 4; ++c)
        *(float4*)(r + f0 + 4 * c) = make_float4(v[4 * c], v[4 * c + 1], v[4 * c + 2], v[4 * c + 3]);
    }
  } else {
#pragma unroll
    for (int q = 0; q < RQ; ++q)
      if (f0 + q < width) r[f0 + q] = v[q];
  }
}

// Second level of the single-relation gradient sum: the operator backward
// left nblk rows per chunk (one per block of its grid); block (c, piece) adds,
// in row order, the rows of chunk c that fall in its piece (wave w the rows
// k0 + w, k0 + w + 4, ..., 32 / RQ of them loaded at a time).
template <int RQ>
__device__ __forceinline__ void relation_block_sums_body(const float* rows, int nblk, int dr, float* partial, int c,
                                                         int piece) {
  __shared__ float red[4][RQ * 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int per = (nblk + RELSUM_PIECES - 1) / RELSUM_PIECES;
  const int k0 = piece * per;
  const int k1 = min(nblk, k0 + per);
  const float* base = rows + (int64_t)c * nblk * dr;
  float acc[RQ];
#pragma unroll
  for (int q = 0; q < RQ; ++q) acc[q] = 0.0f;
  constexpr int B = 32 / RQ;
  for (int k = k0 + w; k < k1; k += 4 * B) {
    float v[B][RQ];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int kk = k + 4 * u;
      const float* r = base + (int64_t)kk * dr;
#pragma unroll
      for (int q = 0; q < RQ; ++q) {
        const int f = lane + 64 * q;
        v[u][q] = (kk < k1 && f < dr) ? r[f] : 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < B; ++u)
#pragma unroll
      for (int q = 0; q < RQ; ++q) acc[q] += v[u][q];
  }
#pragma unroll
  for (int q = 0; q < RQ; ++q) red[w][lane + 64 * q] = acc[q];
  __syncthreads();
  float* out = partial + ((int64_t)c * RELSUM_PIECES + piece) * dr;
  for (int f = threadIdx.x; f < dr; f += 256) out[f] = (red[0][f] + red[1][f]) + (red[2][f] + red[3][f]);
}

// The same element-wise Adagrad in 256-thread workgroups (64 elements each,
// wave w of 4 adding a contiguous quarter of the partial rows in order), for
// the workgroups that ride along with the entity update's second launch.
__device__ __forceinline__ void relation_adagrad4_body(float* relp, float* relG, int width, const float* partial,
                                                       int nparts, float lr, int blk) {
  __shared__ float red4[4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int f = blk * 64 + lane;
  const int per = (nparts + 3) / 4;
  const int p0 = w * per, p1 = min(nparts, p0 + per);
  float gsum = 0.0f;
  if (f < width) {
#pragma unroll 16
    for (int c = p0; c < p1; ++c) gsum += partial[(int64_t)c * width + f];
  }
  red4[w][lane] = gsum;
  __syncthreads();
  if (w != 0 || f >= width) return;
  const float gt = (red4[0][lane] + red4[1][lane]) + (red4[2][lane] + red4[3][lane]);
  const float Gn = relG[f] + gt * gt;
  relG[f] = Gn;
  relp[f] -= lr * gt * adagrad_rcp(Gn);
}

// The single relation's gradient sums and Adagrad step ride along with the
// entity update: workgroups past the update's own run them, the block sums
// with its first launch and the Adagrad step over their partial rows with
// the second (rows NULL: no riders).
struct RelRider {
  const float* rows;   // the operator backward's block rows, nblk per chunk
  int nblk, nchunks, dr, nparts;
  float* partial;      // RELSUM_PIECES rows per chunk
  float* relp;
  float* relG;
};

// Block of SEG_BLOCK sorted positions, one wave.  RQ floats of a row per lane
// (lane L holds elements RQ L .. RQ L + RQ - 1; width <= 64 RQ).  The rows are
// loaded SB positions at a time, together with the embedding rows of the
// whole segments ending among them, all loads in flight together, and a
// running sum restarted at every piece start leaves each piece's in-order
// total at its last position.  Whole segments are updated in place; the (at
// most two) pieces that continue into a neighbouring block are written to
// `partial` at their first position.
template <int MODE, int RQ>
__global__ __launch_bounds__(256) void seg_update_local(StepGeom g, StepBufs b, const uint32_t* keys,
                                                        const uint32_t* vals, int n, const float* rows,
                                                        int64_t ld, int width, float* partial, uint32_t* segflag,
                                                        float lr, RelRider rr, int own_blocks) {
  if ((int)blockIdx.x >= own_blocks) {
    const int k = blockIdx.x - own_blocks;
    relation_block_sums_body<RQ>(rr.rows, rr.nblk, rr.dr, rr.partial, k / RELSUM_PIECES, k % RELSUM_PIECES);
    return;
  }
  constexpr int SB = 16 / RQ;                      // positions per batch of loads
  const int lane = threadIdx.x & 63;
  const int blk = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int p0 = blk * SEG_BLOCK;
  if (p0 >= n) return;
  const int np = min(SEG_BLOCK, n - p0);
  const int pos = p0 + (lane & (SEG_BLOCK - 1));
  const bool valid = lane < SEG_BLOCK && pos < p0 + np;
  const uint32_t k = valid ? keys[pos] : 0u;
  const uint32_t vidx = valid ? vals[pos] : 0u;
  const bool diff_prev = valid && (pos == 0 || keys[pos - 1] != k);
  const bool diff_next = valid && (pos == n - 1 || keys[pos + 1] != k);
  const uint32_t pstart = (uint32_t)__ballot(valid && (pos == p0 || diff_prev));
  const uint32_t segs = (uint32_t)__ballot(diff_prev);
  const uint32_t sege = (uint32_t)__ballot(diff_next);
  const uint32_t live = np == 32 ? 0xFFFFFFFFu : ((1u << np) - 1u);
  const uint32_t pend = ((pstart >> 1) | (1u << (np - 1))) & live;   // last position of each piece
  const bool cont_prev = !(segs & 1u);                  // first piece continues an earlier block
  const bool cont_next = !((sege >> (np - 1)) & 1u);    // last piece continues into the next block
  const int last_start = 31 - __builtin_clz(pstart);
  // piece flags of this block for the spanning-segment pass: bit 1 the first
  // piece continues an earlier block, bit 2 the last piece continues into the
  // next, bit 4 the block is one piece continuing an earlier block; bits
  // 8..12 the position of the last piece's start; bits 16..21 the number of
  // segments starting in the block (the touched rows, summed by that pass)
  if (lane == 0)
    segflag[blk] = (cont_prev ? 1u : 0u) | (cont_next ? 2u : 0u) | ((pstart == 1u && cont_prev) ? 4u : 0u) |
                   ((uint32_t)last_start << 8) | ((uint32_t)__builtin_popcount(segs) << 16);
  // pieces that are whole segments (updated here), as a position mask: the
  // first piece unless it continues an earlier block, the last unless it
  // continues into the next
  const uint32_t first_end = pend & (~pend + 1u);
  const uint32_t last_end = 1u << (np - 1);
  const uint32_t whole = pend & ~(cont_prev ? first_end : 0u) & ~(cont_next ? last_end : 0u);
  // this lane's position: the row's table, row id and Adagrad state, read
  // with the contributions so that one round of loads serves both
  const uint32_t tbl = k >> g.rb;
  const uint32_t rowid = k & ((1u << g.rb) - 1u);
  float gold = 0.0f;
  if (MODE == SEG_ENTITY && valid && ((whole >> (pos - p0)) & 1u)) gold = (tbl ? b.G_j : b.G_i)[rowid];

  // row pointers are wave-uniform (the position's value and key are read
  // from their lane into scalar registers), so the addresses cost no vector
  // instructions
  // the keys, values and Adagrad state of the block have landed before the
  // loop: their lanes are read into scalar registers inside it, and without
  // this wait every such read would wait for all loads in flight
  __builtin_amdgcn_s_waitcnt(0x0F70);
  const bool vec_c = (ld % RQ) == 0 && (width % RQ) == 0;
  const bool vec_e = (g.d % RQ) == 0 && (width % RQ) == 0;
  float run[RQ];
#pragma unroll
  for (int q = 0; q < RQ; ++q) run[q] = 0.0f;
#pragma unroll 1
  for (int b0 = 0; b0 < np; b0 += SB) {
    // the batch's contribution rows and, for whole segments ending in it, the
    // embedding rows they update: all loads in flight together
    float t[SB][RQ], th[SB][RQ];
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      const int uu = b0 + u;
#pragma unroll
      for (int q = 0; q < RQ; ++q) t[u][q] = th[u][q] = 0.0f;
      if (uu < np) {
        const uint32_t vu = (uint32_t)__builtin_amdgcn_readlane((int)vidx, uu);
        crow_load<RQ>(t[u], rows + (int64_t)vu * ld, lane, width, vec_c);
        if (MODE == SEG_ENTITY && ((whole >> uu) & 1u)) {
          const uint32_t key = (uint32_t)__builtin_amdgcn_readlane((int)k, uu);
          const float* emb = ((key >> g.rb) ? b.emb_j : b.emb_i) + (int64_t)(key & ((1u << g.rb) - 1u)) * g.d;
          crow_load<RQ>(th[u], emb, lane, width, vec_e);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      const int uu = b0 + u;
      const bool restart = (pstart >> (uu & 31)) & 1u;
#pragma unroll
      for (int q = 0; q < RQ; ++q) {
        run[q] = restart ? t[u][q] : run[q] + t[u][q];
        t[u][q] = run[q];
      }
    }
    // pieces ending in this batch: whole segments are updated, the rest saved
#pragma unroll
    for (int u = 0; u < SB; ++u) {
      const int uu = b0 + u;
      if (uu >= np || !((pend >> uu) & 1u)) continue;
      const uint32_t key = (uint32_t)__builtin_amdgcn_readlane((int)k, uu);
      if (!((whole >> uu) & 1u)) {
        const bool first = !(pstart & ((2u << uu) - 2u));   // no piece start in (0, uu]
        const int s0 = first ? 0 : last_start;
        crow_store<RQ>(partial + (int64_t)(p0 + s0) * width, t[u], lane, width, vec_c);
      } else if (MODE == SEG_ENTITY) {
        const uint32_t tb = key >> g.rb;
        const uint32_t row = key & ((1u << g.rb) - 1u);
        float* emb = (tb ? b.emb_j : b.emb_i) + (int64_t)row * g.d;
        float gs = 0.0f;
#pragma unroll
        for (int q = 0; q < RQ; ++q) gs += t[u][q] * t[u][q];
        const float Gn = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gold), uu)) + wave_sum(gs);
        const float scale = lr * adagrad_rcp(Gn);
        float nv[RQ];
#pragma unroll
        for (int q = 0; q < RQ; ++q) nv[q] = th[u][q] - scale * t[u][q];
        crow_store<RQ>(emb, nv, lane, width, vec_e);
        if (lane == 0) (tb ? b.G_j : b.G_i)[row] = Gn;
      } else {
        float* p = b.relp + (int64_t)key * width;
        float* G = b.relG + (int64_t)key * width;
        float pv[RQ], Gv[RQ];
        crow_load<RQ>(pv, p, lane, width, vec_c);
        crow_load<RQ>(Gv, G, lane, width, vec_c);
#pragma unroll
        for (int q = 0; q < RQ; ++q) {
          const float gf = t[u][q];
          Gv[q] += gf * gf;
          pv[q] -= lr * gf * adagrad_rcp(Gv[q]);
        }
        crow_store<RQ>(G, Gv, lane, width, vec_c);
        crow_store<RQ>(p, pv, lane, width, vec_c);
      }
    }
  }
}

// segments that cross block boundaries, updated by the wave of the block
// where they start: its last piece plus the leading piece of every following
// block the segment covers, added in block order, 16 loads in flight; the
// extent comes from the piece flags the local pass left per block
template <int MODE, int RQ>
__global__ __launch_bounds__(256) void seg_update_span(StepGeom g, StepBufs b, const uint32_t* keys, int n,
                                                       int width, const float* partial, const uint32_t* segflag,
                                                       float lr, RelRider rr, int own_blocks) {
  if ((int)blockIdx.x >= own_blocks) {
    relation_adagrad4_body(rr.relp, rr.relG, rr.dr, rr.partial, rr.nparts, lr, blockIdx.x - own_blocks);
    return;
  }
  const int lane = threadIdx.x & 63;
  const int blk = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int p0 = blk * SEG_BLOCK;
  const int p1 = p0 + SEG_BLOCK;
  const int nblk = (n + SEG_BLOCK - 1) / SEG_BLOCK;
  if (MODE == SEG_ENTITY && blk == 0 && b.nuniq) {
    // the step's touched rows: the blocks' segment counts (integer sum)
    uint32_t cnt = 0;
    for (int j = lane; j < nblk; j += 64) cnt += (segflag[j] >> 16) & 63u;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) cnt += (uint32_t)__shfl_xor((int)cnt, o, 64);
    if (lane == 0) atomicAdd(b.nuniq, (unsigned long long)cnt);
  }
  if (p1 >= n) return;
  const uint32_t f = segflag[blk];
  if (!(f & 2u) || (f & 4u)) return;     // nothing crosses the end, or the segment started earlier
  const int s = p0 + (int)((f >> 8) & 31u);   // start of the crossing segment
  const uint32_t key = keys[s];
  // blocks the segment covers entirely (flags 2 | 4), 64 flags per probe; it
  // ends inside the first following block that is not one of them
  int nfull = 0;
  for (int j0 = blk + 1;; j0 += 64) {
    const int j = j0 + lane;
    const uint32_t fj = j < nblk ? segflag[j] : 0u;
    const uint64_t stop = __ballot((fj & 6u) != 6u);
    if (stop) {
      nfull += __ffsll((unsigned long long)stop) - 1;
      break;
    }
    nfull += 64;
  }
  const int nparts = 1 + nfull + 1;   // block of s, the covered blocks, the block where it ends
  RowT<RQ> acc;
  row_zero(acc);
  for (int i0 = 0; i0 < nparts; i0 += 16) {
    float t[16][RQ];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int i = i0 + u;
      const int at = i == 0 ? s : p1 + (i - 1) * SEG_BLOCK;
      const float* part = partial + (int64_t)at * width;
#pragma unroll
      for (int q = 0; q < RQ; ++q) {
        const int f = lane + 64 * q;
        t[u][q] = (i < nparts && f < width) ? part[f] : 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < 16; ++u)
#pragma unroll
      for (int q = 0; q < RQ; ++q) acc.v[q] += t[u][q];
  }
  seg_apply<MODE, RQ>(g, b, key, acc, width, lr, lane);
}

template <int RQ>
__global__ __launch_bounds__(256) void relation_block_sums(const float* rows, int nblk, int dr, float* partial) {
  relation_block_sums_body<RQ>(rows, nblk, dr, partial, blockIdx.x, blockIdx.y);
}

// Second level and element-wise Adagrad: 64 elements per block; wave w of 16
// adds a contiguous sixteenth of the partial rows in order (all its loads in
// flight at once), then the sixteen sums are combined in a fixed order.
__global__ __launch_bounds__(1024) void relation_single_adagrad(float* relp, float* relG, int width,
                                                                const float* partial, int nparts,
                                                                float lr) {
  __shared__ float red[16][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int f = blockIdx.x * 64 + lane;
  const int per = (nparts + 15) / 16;
  const int p0 = w * per, p1 = min(nparts, p0 + per);
  float gsum = 0.0f;
  if (f < width) {
#pragma unroll 16
    for (int c = p0; c < p1; ++c) gsum += partial[(int64_t)c * width + f];
  }
  red[w][lane] = gsum;
  __syncthreads();
  if (w != 0 || f >= width) return;
  float gt = 0.0f;
#pragma unroll
  for (int q = 0; q < 16; ++q) gt += red[q][lane];
  const float Gn = relG[f] + gt * gt;
  relG[f] = Gn;
  relp[f] -= lr * gt * adagrad_rcp(Gn);
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

int64_t exclusive_scan_tmp_entries(int64_t n) { return (n + SORT_TILE - 1) / SORT_TILE + 1; }

int radix_tile(int64_t) { return SORT_TILE; }

int64_t radix_hist_entries(int64_t n) { return 256 * ((n + radix_tile(n) - 1) / radix_tile(n)); }

int64_t radix_scan_tmp_entries(int64_t n) { return (radix_hist_entries(n) + SORT_TILE - 1) / SORT_TILE + 1; }

int64_t radix_segments_hist_entries(int64_t n, int nseg) {
  return std::max<int64_t>(nseg, 1) * radix_hist_entries(n) + radix_scan_tmp_entries(n);
}

// LSD passes of 8 bits over nseg segments at once (each segment on its own;
// nblocks <= 64 per segment for the single-launch digit offsets, else one
// segment through the multi-launch scan).  Ping-pong with the alternate
// buffers; the result ends in either.
static void radix_passes(uint32_t* keys, uint32_t* vals, uint32_t* keys_alt, uint32_t* vals_alt, SortSeg sg,
                         int bits, uint32_t* hist, uint32_t* scan_tmp, uint32_t** out_keys, uint32_t** out_vals,
                         hipStream_t s) {
  uint32_t* k_in = keys;
  uint32_t* v_in = vals;
  const int nmax = std::max(sg.n_full, sg.n_last);
  if (nmax > 1 && bits > 0) {
    const int tile = radix_tile(nmax);
    const int nblocks = (nmax + tile - 1) / tile;
    const int64_t nh = (int64_t)256 * nblocks;
    uint32_t* k_out = keys_alt;
    uint32_t* v_out = vals_alt;
    const int passes = (bits + 7) / 8;
    const dim3 grid(nblocks, sg.nseg);
    for (int p = 0; p < passes; ++p) {
      const int shift = 8 * p;
      radix_hist<SORT_IPT><<<grid, 256, 0, s>>>(k_in, sg, shift, nblocks, hist);
      if (nblocks <= 64) {
        radix_scatter<SORT_IPT, true><<<grid, 256, 0, s>>>(k_in, v_in, sg, shift, nblocks, hist, k_out, v_out);
      } else {
        launch_exclusive_scan(hist, nh, hist, scan_tmp, nullptr, s);
        radix_scatter<SORT_IPT, false><<<grid, 256, 0, s>>>(k_in, v_in, sg, shift, nblocks, hist, k_out, v_out);
      }
      uint32_t* t = k_in; k_in = k_out; k_out = t;
      t = v_in; v_in = v_out; v_out = t;
    }
  }
  *out_keys = k_in;
  *out_vals = v_in;
}

void launch_radix_sort_to(uint32_t* keys, uint32_t* vals, int n, int bits, SortWork& w, uint32_t** out_keys,
                          uint32_t** out_vals, hipStream_t s) {
  const SortSeg sg{0, n, n, 1};
  radix_passes(keys, vals, w.keys_alt, w.vals_alt, sg, bits, w.hist, w.scan_tmp, out_keys, out_vals, s);
}

void launch_radix_sort_segments(uint32_t* keys, uint32_t* vals, uint32_t* keys_alt, uint32_t* vals_alt,
                                int64_t stride, int n_full, int n_last, int nseg, int bits, uint32_t* hist,
                                uint32_t** out_keys, uint32_t** out_vals, hipStream_t s) {
  if (nseg <= 0) {
    *out_keys = keys;
    *out_vals = vals;
    return;
  }
  const int nmax = std::max(n_full, n_last);
  if ((nmax + radix_tile(nmax) - 1) / radix_tile(nmax) <= 64) {
    const SortSeg sg{stride, n_full, n_last, nseg};
    radix_passes(keys, vals, keys_alt, vals_alt, sg, bits, hist, nullptr, out_keys, out_vals, s);
    return;
  }
  // segments too long for single-launch offsets: one at a time (the same
  // number of passes, so every result lands in the same buffer)
  for (int y = 0; y < nseg; ++y) {
    const int64_t o = y * stride;
    const int n = y == nseg - 1 ? n_last : n_full;
    const SortSeg sg{0, n, n, 1};
    uint32_t *ok = nullptr, *ov = nullptr;
    radix_passes(keys + o, vals + o, keys_alt + o, vals_alt + o, sg, bits, hist, hist + radix_hist_entries(nmax),
                 &ok, &ov, s);
    if (y == 0) {
      *out_keys = ok - o;
      *out_vals = ov - o;
    }
  }
}

void launch_radix_sort(uint32_t* keys, uint32_t* vals, int n, int bits, SortWork& w, hipStream_t s) {
  uint32_t *k = nullptr, *v = nullptr;
  launch_radix_sort_to(keys, vals, n, bits, w, &k, &v, s);
  if (k != keys) {
    (void)hipMemcpyAsync(keys, k, (size_t)n * 4, hipMemcpyDeviceToDevice, s);
    (void)hipMemcpyAsync(vals, v, (size_t)n * 4, hipMemcpyDeviceToDevice, s);
  }
}

template <int MODE>
static void seg_update(const StepGeom& g, const StepBufs& b, const uint32_t* keys, const uint32_t* vals, int n,
                       const float* rows, int64_t ld, int width, SortWork& w, float lr, hipStream_t s,
                       const RelRider* rider = nullptr) {
  if (n < 0) n = 0;
  if (n == 0 && !rider) return;
  const int blocks = (n + 4 * SEG_BLOCK - 1) / (4 * SEG_BLOCK);
  RelRider rr{};
  int extra1 = 0, extra2 = 0;
  if (rider) {
    rr = *rider;
    extra1 = rr.nchunks * RELSUM_PIECES;
    extra2 = (rr.dr + 63) / 64;
  }
  if (width <= 128) {
    seg_update_local<MODE, 2><<<blocks + extra1, 256, 0, s>>>(g, b, keys, vals, n, rows, ld, width, w.partial,
                                                               w.segflag, lr, rr, blocks);
    seg_update_span<MODE, 2><<<blocks + extra2, 256, 0, s>>>(g, b, keys, n, width, w.partial, w.segflag, lr, rr,
                                                              blocks);
  } else if (width <= 256) {
    seg_update_local<MODE, 4><<<blocks + extra1, 256, 0, s>>>(g, b, keys, vals, n, rows, ld, width, w.partial,
                                                               w.segflag, lr, rr, blocks);
    seg_update_span<MODE, 4><<<blocks + extra2, 256, 0, s>>>(g, b, keys, n, width, w.partial, w.segflag, lr, rr,
                                                              blocks);
  } else {
    seg_update_local<MODE, 8><<<blocks + extra1, 256, 0, s>>>(g, b, keys, vals, n, rows, ld, width, w.partial,
                                                               w.segflag, lr, rr, blocks);
    seg_update_span<MODE, 8><<<blocks + extra2, 256, 0, s>>>(g, b, keys, n, width, w.partial, w.segflag, lr, rr,
                                                              blocks);
  }
}

void launch_entity_update(const StepGeom& g, const StepBufs& b, const uint32_t* keys, const uint32_t* vals,
                          int n, SortWork& w, float lr, hipStream_t s) {
  seg_update<SEG_ENTITY>(g, b, keys, vals, n, b.dn, g.dp, g.d, w, lr, s);
}

bool launch_entity_update_with_relation(const StepGeom& g, const StepBufs& b, const uint32_t* keys,
                                        const uint32_t* vals, int n, SortWork& w, float lr, int nblk, float* partial,
                                        float* relp, float* relG, hipStream_t s) {
  // the riders use the entity kernels' row width
  if (row_width_for(g.dr) != row_width_for(g.d)) return false;
  const RelRider rr{b.relc, nblk, g.nchunks, g.dr, g.nchunks * RELSUM_PIECES, partial, relp, relG};
  seg_update<SEG_ENTITY>(g, b, keys, vals, n, b.dn, g.dp, g.d, w, lr, s, &rr);
  return true;
}

void launch_relation_update_sorted(const StepGeom& g, const StepBufs& b, const uint32_t* keys,
                                   const uint32_t* vals, int n, SortWork& w, float lr, hipStream_t s) {
  seg_update<SEG_RELATION>(g, b, keys, vals, n, b.relc, g.dr, g.dr, w, lr, s);
}

void launch_relation_block_sums(const StepGeom& g, const float* rows, int nblk, float* partial, hipStream_t s) {
  const dim3 grid(g.nchunks, RELSUM_PIECES);
  switch (row_width_for(g.dr)) {
    case 2: relation_block_sums<2><<<grid, 256, 0, s>>>(rows, nblk, g.dr, partial); break;
    case 4: relation_block_sums<4><<<grid, 256, 0, s>>>(rows, nblk, g.dr, partial); break;
    default: relation_block_sums<8><<<grid, 256, 0, s>>>(rows, nblk, g.dr, partial); break;
  }
}

void launch_relation_single_adagrad(float* relp, float* relG, int width, const float* partial,
                                    int nparts, float lr, hipStream_t s) {
  relation_single_adagrad<<<(width + 63) / 64, 1024, 0, s>>>(relp, relG, width, partial, nparts, lr);
}
