// The linear operator g(x) = A_r x (Sec. 3.1 operator table, RESCAL) where it
// is not one matrix product over the step: several relations (a matrix per
// edge), and the cos comparator (whose source candidates need A x_t before
// they are normalised).
//
// Several relations, dot comparator (the source corruptions use the adjoint,
// <A x_t, y> = <x_t, A^T y>):
//   forward   Q_e = A_r x_e,  K_e = A_r^T y_e,  p_e = <Q_e, y_e>, one wave per edge
//   backward  source row += A_r^T dQ_e, destination row += A_r dK_e
//   relation  dA_r = sum over the edges of r of dQ_e x_e^T + y_e dK_e^T, in the
//             edges' order, then element-wise Adagrad, one workgroup per
//             relation segment of the sorted relation keys
// One relation with cos: the source candidate rows A x_t (a contraction over
// the step) are normalised here, and the positive scores follow.
// Reciprocal predicates (any relation count, dot or cos): Q_e = A_r x_e and
// K_e = A_{r+R} y_e per edge (normalised for cos), each side's positive score;
// backward source row += A_r^T dQ_e, destination row += A_{r+R}^T dK_e;
// dA_r = sum of dQ_e x_e^T and dA_{r+R} = sum of dK_e y_e^T over the sorted
// relation keys.
#include "kernels.h"
#include "row_ops.h"

namespace {

constexpr int kWaves = 4;

template <int RQ>
__global__ __launch_bounds__(256) void linear_rows_kernel(StepGeom g, StepBufs b) {
  using RowQ = RowT<RQ>;
  __shared__ float stage[kWaves][512];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = blockIdx.y;
  const int e = blockIdx.x * kWaves + w;
  if (e >= chunk_edges(g, c)) return;   // no block-level barriers below
  const int d = g.d, dp = g.dp;
  const int64_t ce = (int64_t)c * g.C + e;
  const int r = edge_relation(g, b.rel, chunk_first(g, c) + e);
  const float* A = b.relp + (int64_t)r * d * d;
  RowQ x, y, q, k;
  if (g.recip) {
    const bool cos = g.cmp == CMP_COS;
    const float* Bm = b.relp + (int64_t)(r + g.R) * d * d;
    const float* xs = cos ? b.lin_x + ((int64_t)(c * 2 + 0) * g.C + e) * dp : b.nn + ((int64_t)(c * 2 + 1) * g.N + e) * dp;
    const float* yd = cos ? b.lin_x + ((int64_t)(c * 2 + 1) * g.C + e) * dp : b.nn + ((int64_t)(c * 2 + 0) * g.N + e) * dp;
    row_load(x, xs, d, false, lane);   // raw x_s
    row_load(y, yd, d, false, lane);   // raw x_d
    mat_rows_apply(q, A, x, stage[w], d, lane);    // A_r x
    mat_rows_apply(k, Bm, y, stage[w], d, lane);   // A_{r+R} y
    if (cos) {
      const float nq = row_normalize(q);
      const float nk = row_normalize(k);
      // the unit entity rows the gather stored
      row_load(y, b.nn + ((int64_t)(c * 2 + 0) * g.N + e) * dp, d, false, lane);
      row_load(x, b.nn + ((int64_t)(c * 2 + 1) * g.N + e) * dp, d, false, lane);
      if (lane == 0) {
        b.qnrm[(int64_t)(c * 2 + 0) * g.C + e] = nq;
        b.qnrm[(int64_t)(c * 2 + 1) * g.C + e] = nk;
      }
    }
    row_store(q, b.qk + ((int64_t)(c * 2 + 0) * g.C + e) * dp, d, dp, false, lane);
    row_store(k, b.qk + ((int64_t)(c * 2 + 1) * g.C + e) * dp, d, dp, false, lane);
    const float p0 = row_dot(q, y);
    const float p1 = row_dot(k, x);
    if (lane == 0) {
      b.pos[(int64_t)(c * 2 + 0) * g.C + e] = p0;
      b.pos[(int64_t)(c * 2 + 1) * g.C + e] = p1;
    }
    return;
  }
  row_load(x, b.nn + ((int64_t)(c * 2 + 1) * g.N + e) * dp, d, false, lane);   // raw x_s
  row_load(y, b.nn + ((int64_t)(c * 2 + 0) * g.N + e) * dp, d, false, lane);   // raw x_d
  mat_rows_apply(q, A, x, stage[w], d, lane);   // A x
  mat_apply(k, A, y, stage[w], d, lane);        // A^T y
  row_store(q, b.qk + ((int64_t)(c * 2 + 0) * g.C + e) * dp, d, dp, false, lane);
  row_store(k, b.qk + ((int64_t)(c * 2 + 1) * g.C + e) * dp, d, dp, false, lane);
  const float p = row_dot(q, y);
  if (lane == 0) b.pos[ce] = p;
}

template <int RQ>
__global__ __launch_bounds__(256) void linear_rows_backward_kernel(StepGeom g, StepBufs b) {
  using RowQ = RowT<RQ>;
  __shared__ float stage[kWaves][512];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = blockIdx.y;
  const int e = blockIdx.x * kWaves + w;
  if (e >= chunk_edges(g, c)) return;
  const int d = g.d, dp = g.dp;
  const int r = edge_relation(g, b.rel, chunk_first(g, c) + e);
  const float* A = b.relp + (int64_t)r * d * d;
  // the operator backward left dQ (with the positive score's term) in dq
  // side 0 and dK in dq side 1 (reciprocal predicates: the gradients of
  // A_r x_s and A_{r+R} x_d)
  RowQ dQ, dK, ts, td;
  row_load(dQ, b.dq + ((int64_t)(c * 2 + 0) * g.C + e) * dp, d, false, lane);
  row_load(dK, b.dq + ((int64_t)(c * 2 + 1) * g.C + e) * dp, d, false, lane);
  mat_apply(ts, A, dQ, stage[w], d, lane);         // A^T dQ
  if (g.recip) mat_apply(td, b.relp + (int64_t)(r + g.R) * d * d, dK, stage[w], d, lane);   // A_{r+R}^T dK
  else mat_rows_apply(td, A, dK, stage[w], d, lane);                                        // A dK
  float* srow = b.dn + ((int64_t)(c * 2 + 1) * g.N + e) * dp;
  float* drow = b.dn + ((int64_t)(c * 2 + 0) * g.N + e) * dp;
  RowQ s0, d0;
  row_load(s0, srow, d, false, lane);
  row_load(d0, drow, d, false, lane);
  row_add(s0, ts);
  row_add(d0, td);
  row_store(s0, srow, d, dp, false, lane);
  row_store(d0, drow, d, dp, false, lane);
}

// Sorted relation keys (stable: edges of one relation in step order); vals
// hold chunk * relN + edge (reciprocal predicates: + C for the source-side
// row r + R, whose gradient is dK y^T).  The workgroup at the first position
// of a relation's run sums that relation's matrix gradient over the run and applies
// element-wise Adagrad; the others leave at once.  Every element belongs to
// one thread, and the edges are added in order: the result is reproducible.
constexpr int kLinBatch = 4;     // edges staged in LDS at a time
constexpr int kLinElems = 8;     // matrix elements per thread per pass

__global__ __launch_bounds__(256) void linear_relation_update_kernel(StepGeom g, StepBufs b, const uint32_t* keys,
                                                                     const uint32_t* vals, int n, float lr) {
  __shared__ float rows[kLinBatch][4][512];   // dQ, x, y, dK of each staged edge
  __shared__ int seg_end;
  const int p0 = blockIdx.x;
  const uint32_t r = keys[p0];
  if (p0 > 0 && keys[p0 - 1] == r) return;   // uniform per workgroup
  const int tid = threadIdx.x;
  if (tid == 0) seg_end = n;
  __syncthreads();
  // end of the run: the first position past p0 with another key
  for (int base = p0 + 1; base < n; base += 256) {
    const int q = base + tid;
    if (q < n && keys[q] != r) atomicMin(&seg_end, q);
    __syncthreads();
    const bool found = seg_end < n;
    __syncthreads();   // every thread has read seg_end before the next round writes it
    if (found) break;
  }
  const int end = seg_end;
  const int d = g.d, dp = g.dp;
  const int64_t nel = (int64_t)d * d;
  float* A = b.relp + (int64_t)r * nel;
  float* GA = b.relG + (int64_t)r * nel;
  for (int64_t el0 = 0; el0 < nel; el0 += 256 * kLinElems) {
    float acc[kLinElems];
    int kk[kLinElems], ll[kLinElems];
#pragma unroll
    for (int u = 0; u < kLinElems; ++u) {
      acc[u] = 0.0f;
      const int64_t el = el0 + tid + 256 * u;
      kk[u] = (int)(el / d);
      ll[u] = (int)(el - (int64_t)kk[u] * d);
    }
    for (int q0 = p0; q0 < end; q0 += kLinBatch) {
      const int nb = min(kLinBatch, end - q0);
      __syncthreads();
      for (int idx = tid; idx < nb * 4 * d; idx += 256) {
        const int eb = idx / (4 * d), rem = idx - eb * 4 * d;
        const int which = rem / d, f = rem - which * d;
        const uint32_t v = vals[q0 + eb];
        const int c = (int)(v / (uint32_t)g.relN);
        int e = (int)(v - (uint32_t)c * g.relN);
        float val;
        if (g.recip) {
          // dQ x^T (row r) or dK y^T (row r + R); the raw rows: the candidate
          // tiles (dot) or lin_x (cos)
          const int rev = e >= g.C ? 1 : 0;
          e -= rev * g.C;
          const bool cos = g.cmp == CMP_COS;
          const float* raw = cos ? b.lin_x + ((int64_t)(c * 2 + rev) * g.C + e) * dp
                                 : b.nn + ((int64_t)(c * 2 + 1 - rev) * g.N + e) * dp;
          if (which == 0) val = b.dq[((int64_t)(c * 2 + rev) * g.C + e) * dp + f];
          else if (which == 1) val = raw[f];
          else val = 0.0f;
        } else {
          const float* src;
          if (which == 0) src = b.dq + ((int64_t)(c * 2 + 0) * g.C + e) * dp;        // dQ_e
          else if (which == 1) src = b.nn + ((int64_t)(c * 2 + 1) * g.N + e) * dp;   // x_e
          else if (which == 2) src = b.nn + ((int64_t)(c * 2 + 0) * g.N + e) * dp;   // y_e
          else src = b.dq + ((int64_t)(c * 2 + 1) * g.C + e) * dp;                   // dK_e
          val = src[f];
        }
        rows[eb][which][f] = val;
      }
      __syncthreads();
      for (int eb = 0; eb < nb; ++eb) {
#pragma unroll
        for (int u = 0; u < kLinElems; ++u) {
          if (el0 + tid + 256 * u < nel)
            acc[u] += rows[eb][0][kk[u]] * rows[eb][1][ll[u]] + rows[eb][2][kk[u]] * rows[eb][3][ll[u]];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kLinElems; ++u) {
      const int64_t el = el0 + tid + 256 * u;
      if (el < nel) {
        const float gv = acc[u];
        const float Gn = GA[el] + gv * gv;
        GA[el] = Gn;
        A[el] -= lr * gv / (sqrtf(Gn) + PBG_EPS_ADAGRAD);
      }
    }
  }
}

// linear + cos: the source candidate rows A x_t of every chunk (a contraction
// left them in the candidate tile of side 1) are normalised in place, with
// their norms kept for the backward; for the chunk's edges the positive
// score <A x_s / |A x_s|, x_d / |x_d|> follows
template <int RQ>
__global__ __launch_bounds__(256) void normalize_candidates_kernel(StepGeom g, StepBufs b) {
  using RowQ = RowT<RQ>;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int c = blockIdx.y;
  const int Cc = chunk_edges(g, c);
  const int t = blockIdx.x * kWaves + w;
  if (t >= Cc + g.U) return;
  const int d = g.d, dp = g.dp;
  float* row = b.nn + ((int64_t)(c * 2 + 1) * g.N + t) * dp;
  RowQ v;
  row_load(v, row, d, false, lane);
  const float nv = row_normalize(v);
  row_store(v, row, d, dp, false, lane);
  if (lane == 0) b.nrm[(int64_t)(c * 2 + 1) * g.N + t] = nv;
  if (t < Cc) {
    RowQ y;
    row_load(y, b.nn + ((int64_t)(c * 2 + 0) * g.N + t) * dp, d, false, lane);
    const float p = row_dot(v, y);
    if (lane == 0) b.pos[(int64_t)c * g.C + t] = p;
  }
}

}  // namespace

void launch_linear_rows(const StepGeom& g, const StepBufs& b, hipStream_t s) {
  dim3 grid((g.C + kWaves - 1) / kWaves, g.nchunks);
  switch (row_width_for(g.d)) {
    case 2: linear_rows_kernel<2><<<grid, 256, 0, s>>>(g, b); break;
    case 4: linear_rows_kernel<4><<<grid, 256, 0, s>>>(g, b); break;
    default: linear_rows_kernel<8><<<grid, 256, 0, s>>>(g, b); break;
  }
}

void launch_linear_rows_backward(const StepGeom& g, const StepBufs& b, hipStream_t s) {
  dim3 grid((g.C + kWaves - 1) / kWaves, g.nchunks);
  switch (row_width_for(g.d)) {
    case 2: linear_rows_backward_kernel<2><<<grid, 256, 0, s>>>(g, b); break;
    case 4: linear_rows_backward_kernel<4><<<grid, 256, 0, s>>>(g, b); break;
    default: linear_rows_backward_kernel<8><<<grid, 256, 0, s>>>(g, b); break;
  }
}

void launch_linear_relation_update(const StepGeom& g, const StepBufs& b, const uint32_t* keys,
                                   const uint32_t* vals, int n, float lr, hipStream_t s) {
  if (n <= 0) return;
  linear_relation_update_kernel<<<n, 256, 0, s>>>(g, b, keys, vals, n, lr);
}

void launch_normalize_candidates(const StepGeom& g, const StepBufs& b, hipStream_t s) {
  dim3 grid((g.N + kWaves - 1) / kWaves, g.nchunks);
  switch (row_width_for(g.d)) {
    case 2: normalize_candidates_kernel<2><<<grid, 256, 0, s>>>(g, b); break;
    case 4: normalize_candidates_kernel<4><<<grid, 256, 0, s>>>(g, b); break;
    default: normalize_candidates_kernel<8><<<grid, 256, 0, s>>>(g, b); break;
  }
}
