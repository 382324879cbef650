// Argument range checks and per-edge scoring.
#include "kernels.h"
#include "row_ops.h"

namespace {

__global__ void check_ids_kernel(const int32_t* ids, int64_t n, int32_t limit, uint32_t* flag,
                                 uint32_t bit) {
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t v = ids[i];
    bad |= (v < 0) | (v >= limit);
  }
  if (__ballot(bad) && (threadIdx.x & 63) == 0) atomicOr(flag, bit);
}

__global__ void check_ids64_kernel(const int64_t* ids, int64_t n, int64_t limit, uint32_t* flag,
                                   uint32_t bit) {
  bool bad = false;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t v = ids[i];
    bad |= (v < 0) | (v >= limit);
  }
  if (__ballot(bad) && (threadIdx.x & 63) == 0) atomicOr(flag, bit);
}

// f(s, r, d) = sim(g(x_s, theta_r), x_d), one wave per edge
__global__ __launch_bounds__(256) void score_edges_kernel(StepGeom g, const float* emb_i,
                                                          const float* emb_j, const float* relp,
                                                          const float* relT, const int32_t* src,
                                                          const int32_t* rel, const int32_t* dst,
                                                          int64_t n, float* out) {
  __shared__ float stage[4][512];
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int64_t e = (int64_t)blockIdx.x * 4 + w;
  if (e >= n) return;
  const bool cplx = g.op == OP_COMPLEX;
  const int d = g.d;
  const int r = rel ? rel[e] : 0;
  Row x, y, th;
  row_load(x, emb_i + (int64_t)src[e] * d, d, cplx, lane);
  row_load(y, emb_j + (int64_t)dst[e] * d, d, cplx, lane);
  Row gq;
  if (g.op == OP_LINEAR) {
    mat_apply(gq, relT + (int64_t)r * d * d, x, stage[w], d, lane);
  } else {
    if (g.op != OP_IDENTITY) row_load(th, relp + (int64_t)r * g.dr, d, cplx, lane);
    else row_zero(th);
    gq = op_forward(g.op, x, th);
  }
  if (g.cmp == CMP_COS) {
    row_normalize(gq);
    row_normalize(y);
  }
  const float s = row_dot(gq, y);
  if (lane == 0) out[e] = s;
}

// uniform draws of chunks [chunk0, chunk0 + n_chunks): out[c][side][k]
__global__ void sample_negatives_kernel(uint64_t seed, uint32_t bucket, int64_t chunk0, int64_t n_chunks,
                                        int U, uint32_t rows_j, uint32_t rows_i, int32_t* out) {
  const int64_t total = n_chunks * 2 * U;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t c = idx / (2 * U);
    const int rem = (int)(idx - c * 2 * U);
    const int side = rem / U, k = rem % U;
    out[idx] = uniform_negative(seed, bucket, (uint64_t)(chunk0 + c), (uint32_t)side, (uint32_t)k,
                                side == 0 ? rows_j : rows_i);
  }
}

__global__ void fill_u32_kernel(uint32_t* p, int64_t n, uint32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

int blocks_for(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b < 1) b = 1;
  if (b > 8192) b = 8192;
  return (int)b;
}

}  // namespace

void launch_check_ids(const int32_t* ids, int64_t n, int32_t limit, uint32_t* flag, uint32_t bit,
                      hipStream_t s) {
  if (n <= 0) return;
  check_ids_kernel<<<blocks_for(n), 256, 0, s>>>(ids, n, limit, flag, bit);
}

void launch_check_ids64(const int64_t* ids, int64_t n, int64_t limit, uint32_t* flag, uint32_t bit,
                        hipStream_t s) {
  if (n <= 0) return;
  check_ids64_kernel<<<blocks_for(n), 256, 0, s>>>(ids, n, limit, flag, bit);
}

void launch_score_edges(const StepGeom& g, const float* emb_i, const float* emb_j, const float* relp,
                        const float* relT, const int32_t* src, const int32_t* rel,
                        const int32_t* dst, int64_t n, float* out, hipStream_t s) {
  if (n <= 0) return;
  const int64_t blocks = (n + 3) / 4;
  score_edges_kernel<<<(unsigned)blocks, 256, 0, s>>>(g, emb_i, emb_j, relp, relT, src, rel, dst, n,
                                                      out);
}

void launch_sample_negatives(uint64_t seed, uint32_t bucket, int64_t chunk0, int64_t n_chunks, int U,
                             uint32_t rows_j, uint32_t rows_i, int32_t* out, hipStream_t s) {
  const int64_t total = n_chunks * 2 * U;
  if (total <= 0) return;
  sample_negatives_kernel<<<blocks_for(total), 256, 0, s>>>(seed, bucket, chunk0, n_chunks, U, rows_j,
                                                           rows_i, out);
}

void launch_fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s) {
  if (n <= 0) return;
  fill_u32_kernel<<<blocks_for(n), 256, 0, s>>>(p, n, v);
}
