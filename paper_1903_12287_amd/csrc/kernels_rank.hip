// Filtered link-prediction ranks (Sec. 5.4, filtered protocol): every held-out
// triple (s, r, d) is ranked against all entities on both sides,
//   destination side  1 + #{d' != d : (s, r, d') not known, f(s, r, d') >= f(s, r, d)}
//   source side       1 + #{s' != s : (s', r, d) not known, f(s', r, d) >= f(s, r, d)}
// with f(s, r, d) = sim(g(x_s, theta_r), x_d) (Sec. 3.1).
//
// The candidate scores of a block of queries form one matrix product
// S = Q . T^T against a candidate table T (MFMA, kernels_gemm.hip):
//   destination side  Q = g(x_s) (dot) or its unit vector (cos); T = the
//                     entity table (unit rows for cos);
//   source side       Q = g*(x_d) (dot, the adjoint: <g(x), y> = <x, g*(y)>;
//                     translation adds the per-query constant <theta_r, x_d>)
//                     or the unit x_d (cos); T = the entity table (dot) or the
//                     unit rows of g(x) under the single relation (cos).
//   reciprocal predicates: the source side's Q = g(x_d, theta_{r+R}) (a unit
//                     vector for cos) against the entity table, and its own
//                     positive score sim(Q, x_s), which replaces the
//                     destination side's in pos once that side is counted.
// The count kernel then reads each query's row of S once, counts the
// candidates at or above the positive score, and takes back the known
// triples' candidates by reading the same stored scores, so that the count
// and the filter correction agree element by element.
#include <algorithm>

#include "kernels.h"
#include "row_ops.h"

namespace {

// candidate tables: one wave per entity row
__global__ __launch_bounds__(256) void rank_tables_kernel(StepGeom g, const float* emb, const float* relp,
                                                          const float* relT, int64_t n_ent, float* T0, float* T1) {
  __shared__ float stage[4][512];
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n_ent) return;
  const bool cplx = g.op == OP_COMPLEX;
  Row x;
  row_load(x, emb + row * g.d, g.d, cplx, lane);
  if (g.cmp == CMP_DOT) {
    row_store(x, T0 + row * g.dp, g.d, g.dp, cplx, lane);
    return;
  }
  Row xh = x;
  row_normalize(xh);
  row_store(xh, T0 + row * g.dp, g.d, g.dp, cplx, lane);
  if (T1) {
    // cos with a non-identity operator: one relation, applied to every source candidate
    Row gx;
    if (g.op == OP_LINEAR) {
      mat_apply(gx, relT, x, stage[threadIdx.x >> 6], g.d, lane);   // A x
    } else {
      Row th;
      row_load(th, relp, g.d, cplx, lane);
      gx = op_forward(g.op, x, th);
    }
    row_normalize(gx);
    row_store(gx, T1 + row * g.dp, g.d, g.dp, cplx, lane);
  }
}

// queries of rows [e0, e0 + rows) for one side; side 0 also writes the
// positive score p_e = f(s, r, d), computed as pbg_score_edges does, and the
// source side with reciprocal predicates its own
__global__ __launch_bounds__(256) void rank_queries_kernel(StepGeom g, const float* emb, const float* relp,
                                                           const float* relT, const int32_t* src,
                                                           const int32_t* rel, const int32_t* dst,
                                                           int64_t e0, int rows, int side, float* Q,
                                                           float* pos, float* bias) {
  __shared__ float stage[4][512];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int q = blockIdx.x * 4 + w;
  if (q >= rows) return;
  const int64_t e = e0 + q;
  const bool cplx = g.op == OP_COMPLEX;
  const int d = g.d;
  const int r = rel ? rel[e] : 0;
  Row x, y, th;
  row_load(x, emb + (int64_t)src[e] * d, d, cplx, lane);
  row_load(y, emb + (int64_t)dst[e] * d, d, cplx, lane);
  if (g.op != OP_IDENTITY && g.op != OP_LINEAR) row_load(th, relp + (int64_t)r * g.dr, d, cplx, lane);
  else row_zero(th);
  float* qrow = Q + (int64_t)q * g.dp;
  if (side == 0) {
    Row gq;
    if (g.op == OP_LINEAR) mat_apply(gq, relT + (int64_t)r * d * d, x, stage[w], d, lane);   // A x
    else gq = op_forward(g.op, x, th);
    if (g.cmp == CMP_COS) {
      row_normalize(gq);
      row_normalize(y);
    }
    const float p = row_dot(gq, y);
    row_store(gq, qrow, d, g.dp, cplx, lane);
    if (lane == 0) pos[e] = p;
  } else if (g.recip) {
    Row k;
    if (g.op == OP_LINEAR) {
      mat_apply(k, relT + (int64_t)(r + g.R) * d * d, y, stage[w], d, lane);   // A_{r+R} y
    } else {
      Row tr;
      if (g.op != OP_IDENTITY) row_load(tr, relp + (int64_t)(r + g.R) * g.dr, d, cplx, lane);
      else row_zero(tr);
      k = op_forward(g.op, y, tr);
    }
    if (g.cmp == CMP_COS) {
      row_normalize(k);
      row_normalize(x);
    }
    const float p1 = row_dot(k, x);
    row_store(k, qrow, d, g.dp, cplx, lane);
    if (lane == 0) {
      pos[e] = p1;
      bias[q] = 0.0f;
    }
  } else {
    Row k;
    float bs = 0.0f;
    if (g.cmp == CMP_COS) {
      k = y;
      row_normalize(k);
    } else if (g.op == OP_LINEAR) {
      mat_apply(k, relp + (int64_t)r * d * d, y, stage[w], d, lane);                       // A^T y
    } else if (g.op == OP_TRANSLATION) {
      k = y;
      bs = row_dot(th, y);
    } else {
      k = op_adjoint(g.op, y, th);
    }
    row_store(k, qrow, d, g.dp, cplx, lane);
    if (lane == 0) bias[q] = bs;
  }
}

// first index in [lo, hi) whose (a, b) key is not below (ka, kb)
__device__ int64_t lower_bound2(const int32_t* a, const int32_t* b, int64_t lo, int64_t hi, int32_t ka,
                                int32_t kb) {
  while (lo < hi) {
    const int64_t mid = lo + ((hi - lo) >> 1);
    const bool less = a[mid] < ka || (a[mid] == ka && b[mid] < kb);
    if (less) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// one wave per query row of the stored score block; column t is entity t,
// or entity cand[t] when a candidate list is given (no filter then)
__global__ __launch_bounds__(256) void rank_count_kernel(const float* S, int64_t ldS, int64_t n_ent,
                                                         const int32_t* cand,
                                                         int64_t e0, int rows, int side, int64_t n_eval,
                                                         const int32_t* src, const int32_t* rel,
                                                         const int32_t* dst, const float* pos,
                                                         const float* bias, const int32_t* ka,
                                                         const int32_t* kb, const int32_t* kc,
                                                         int64_t n_known, int32_t* ranks) {
  const int lane = threadIdx.x & 63;
  const int q = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (q >= rows) return;
  const int64_t e = e0 + q;
  const int32_t s = src[e], d = dst[e];
  const int32_t r = rel ? rel[e] : 0;
  const int32_t true_id = side == 0 ? d : s;
  const float p = pos[e];
  const float bq = side == 1 ? bias[q] : 0.0f;
  const float* row = S + (int64_t)q * ldS;
  uint32_t cnt = 0;
  for (int64_t t = lane; t < n_ent; t += 64) {
    const float v = row[t] + bq;
    const int64_t id = cand ? (int64_t)cand[t] : t;
    cnt += (v >= p && id != true_id) ? 1u : 0u;
  }
  // filter: candidates of known triples sharing (s, r) (side 0) or (d, r) (side 1);
  // the known triples are sorted by (s, r, d) for side 0 and (d, r, s) for side 1
  const int32_t k1 = side == 0 ? s : d;
  int64_t lo = 0, hi = 0;
  if (lane == 0 && n_known > 0) {
    lo = lower_bound2(ka, kb, 0, n_known, k1, r);
    hi = lower_bound2(ka, kb, lo, n_known, k1, r + 1);   // end of the (k1, r) group
  }
  lo = __shfl(lo, 0, 64);
  hi = __shfl(hi, 0, 64);
  for (int64_t i = lo + lane; i < hi; i += 64) {
    const int32_t c = kc[i];
    if (c == true_id || (i > lo && kc[i - 1] == c)) continue;   // the triple itself, duplicates
    const float v = row[c] + bq;
    if (v >= p) cnt -= 1u;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
  if (lane == 0) ranks[(side == 0 ? 0 : n_eval) + e] = (int32_t)(1u + cnt);
}

// MRR and Hits@10 over the ranks, in a fixed order (fp64)
__global__ __launch_bounds__(256) void rank_metrics_kernel(const int32_t* ranks, int64_t n, double* out) {
  __shared__ double s_rr[256];
  __shared__ double s_h[256];
  double rr = 0.0, h = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 256) {
    const int32_t k = ranks[i];
    rr += 1.0 / (double)k;
    h += k <= 10 ? 1.0 : 0.0;
  }
  s_rr[threadIdx.x] = rr;
  s_h[threadIdx.x] = h;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      s_rr[threadIdx.x] += s_rr[threadIdx.x + o];
      s_h[threadIdx.x] += s_h[threadIdx.x + o];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    out[0] = n > 0 ? s_rr[0] / (double)n : 0.0;
    out[1] = n > 0 ? s_h[0] / (double)n : 0.0;
  }
}

// known-triple sort: keys of one field through the current permutation
__global__ void perm_keys_kernel(const int32_t* field, const uint32_t* perm, int64_t n, uint32_t* keys,
                                 uint32_t* vals_init) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t j = vals_init ? i : (int64_t)perm[i];
    keys[i] = field ? (uint32_t)field[j] : 0u;
    if (vals_init) vals_init[i] = (uint32_t)i;
  }
}

__global__ void gather3_kernel(const uint32_t* perm, const int32_t* a, const int32_t* b, const int32_t* c,
                               int64_t n, int32_t* oa, int32_t* ob, int32_t* oc) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t j = perm[i];
    oa[i] = a[j];
    ob[i] = b ? b[j] : 0;
    oc[i] = c[j];
  }
}

int grid_of(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b < 1) b = 1;
  if (b > 16384) b = 16384;
  return (int)b;
}

}  // namespace

void launch_rank_tables(const StepGeom& g, const float* emb, const float* relp, const float* relT, int64_t n_ent,
                        float* T0, float* T1, hipStream_t s) {
  if (n_ent <= 0) return;
  rank_tables_kernel<<<(unsigned)((n_ent + 3) / 4), 256, 0, s>>>(g, emb, relp, relT, n_ent, T0, T1);
}

void launch_rank_queries(const StepGeom& g, const float* emb, const float* relp, const float* relT,
                         const int32_t* src, const int32_t* rel, const int32_t* dst, int64_t e0, int rows,
                         int side, float* Q, float* pos, float* bias, hipStream_t s) {
  if (rows <= 0) return;
  rank_queries_kernel<<<(rows + 3) / 4, 256, 0, s>>>(g, emb, relp, relT, src, rel, dst, e0, rows, side, Q,
                                                     pos, bias);
}

void launch_rank_count(const float* S, int64_t ldS, int64_t n_ent, const int32_t* cand, int64_t e0, int rows,
                       int side, int64_t n_eval, const int32_t* src, const int32_t* rel, const int32_t* dst,
                       const float* pos, const float* bias, const int32_t* ka, const int32_t* kb,
                       const int32_t* kc, int64_t n_known, int32_t* ranks, hipStream_t s) {
  if (rows <= 0) return;
  rank_count_kernel<<<(rows + 3) / 4, 256, 0, s>>>(S, ldS, n_ent, cand, e0, rows, side, n_eval, src, rel, dst,
                                                   pos, bias, ka, kb, kc, n_known, ranks);
}

// rows out[i] = T[idx[i]] of ld floats
__global__ void gather_rows_kernel(const float* T, const int32_t* idx, int64_t n, int ld, float* out) {
  const int64_t total = n * ld;
  for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < total; k += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = k / ld;
    out[k] = T[(int64_t)idx[i] * ld + (k - i * ld)];
  }
}

void launch_gather_rows(const float* T, const int32_t* idx, int64_t n, int ld, float* out, hipStream_t s) {
  if (n <= 0) return;
  const int64_t total = n * ld;
  const unsigned blocks = (unsigned)std::min<int64_t>((total + 255) / 256, 4096);
  gather_rows_kernel<<<blocks, 256, 0, s>>>(T, idx, n, ld, out);
}

void launch_rank_metrics(const int32_t* ranks, int64_t n, double* out, hipStream_t s) {
  rank_metrics_kernel<<<1, 256, 0, s>>>(ranks, n, out);
}

void launch_perm_keys(const int32_t* field, const uint32_t* perm, int64_t n, uint32_t* keys,
                      uint32_t* vals_init, hipStream_t s) {
  if (n <= 0) return;
  perm_keys_kernel<<<grid_of(n), 256, 0, s>>>(field, perm, n, keys, vals_init);
}

void launch_gather3(const uint32_t* perm, const int32_t* a, const int32_t* b, const int32_t* c, int64_t n,
                    int32_t* oa, int32_t* ob, int32_t* oc, hipStream_t s) {
  if (n <= 0) return;
  gather3_kernel<<<grid_of(n), 256, 0, s>>>(perm, a, b, c, n, oa, ob, oc);
}
