// Gather + relation operator + uniform negatives (Sec. 3.1 score function,
// Sec. 4.3 batched negatives, Fig. 3).
//
// One wave per work item; the items of chunk c are
//   e in [0, Cc)              an edge: its source and destination rows,
//   Cc + q, q in [0, U4)      uniform destination candidates 4q .. 4q+3 (partition j),
//   Cc + U4 + q               uniform source candidates 4q .. 4q+3 (partition i),
// with U4 = ceil(U / 4): the four draws of one Philox block go to one wave.
// For the dot comparator the source corruptions use the adjoint of g
// (<g(x), y> = <x, g*(y)>, plus <theta, y> for translation), so every
// candidate row is copied raw.  For cos every packed row is a unit vector and
// the source candidates carry g (one relation, or the identity operator).
// With reciprocal predicates both queries carry an operator, Q = g(x_s,
// theta_r) and K = g(x_d, theta_{r+R}), each side has its own positive score,
// and every candidate row is the entity itself (a unit vector for cos).
#include <algorithm>
#include "kernels.h"
#include "row_ops.h"

namespace {

// EP edges per edge item: 2 for the cos comparator without reciprocal
// predicates or the linear operator (both edges' four rows load together),
// else 1.
template <int RQ, bool RECIP, int EP>
__global__ __launch_bounds__(256) void gather_op_kernel(StepGeom g, StepBufs b) {
  using Row = RowT<RQ>;
  const int lane = threadIdx.x & 63;
  const int c = blockIdx.y;
  const int Cc = chunk_edges(g, c);
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
  const bool cplx = g.op == OP_COMPLEX;
  const int ne = (Cc + EP - 1) / EP;   // edge items
  const bool active = item < ne + 2 * ((g.U + 3) >> 2);
  const int d = g.d, dp = g.dp;

  if (!active) return;   // no block-level barriers below: idle waves may leave
  if (EP == 2 && item < ne) {
    // ---- edges 2 item and 2 item + 1 (the second may not exist)
    const int e0 = 2 * item;
    const bool two = e0 + 1 < Cc;
    const int64_t eg0 = chunk_first(g, c) + e0;
    const int64_t eg1 = two ? eg0 + 1 : eg0;
    const int s0 = b.src[eg0], t0 = b.dst[eg0], s1 = b.src[eg1], t1 = b.dst[eg1];
    const int r0 = edge_relation(g, b.rel, eg0), r1 = edge_relation(g, b.rel, eg1);
    Row x0, y0, x1, y1, th0, th1;
    row_load(x0, b.emb_i + (int64_t)s0 * d, d, cplx, lane);
    row_load(y0, b.emb_j + (int64_t)t0 * d, d, cplx, lane);
    row_load(x1, b.emb_i + (int64_t)s1 * d, d, cplx, lane);
    row_load(y1, b.emb_j + (int64_t)t1 * d, d, cplx, lane);
    if (g.op != OP_IDENTITY) {
      row_load(th0, b.relp + (int64_t)r0 * g.dr, d, cplx, lane);
      row_load(th1, b.relp + (int64_t)r1 * g.dr, d, cplx, lane);
    } else {
      row_zero(th0);
      row_zero(th1);
    }
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      if (k == 1 && !two) break;
      const int e = e0 + k;
      Row gq = op_forward(g.op, k ? x1 : x0, k ? th1 : th0);
      Row y = k ? y1 : y0;
      const float nq = row_normalize(gq);
      const float ny = row_normalize(y);
      const float p = row_dot(gq, y);
      // Q and K are these candidate rows (QK_IN_NN)
      row_store(gq, b.nn + ((int64_t)(c * 2 + 1) * g.N + e) * dp, d, dp, cplx, lane);
      row_store(y, b.nn + ((int64_t)(c * 2 + 0) * g.N + e) * dp, d, dp, cplx, lane);
      if (lane == 0) {
        b.pos[(int64_t)c * g.C + e] = p;
        b.bias[(int64_t)c * g.C + e] = 0.0f;
        b.nrm[(int64_t)(c * 2 + 0) * g.N + e] = ny;
        b.nrm[(int64_t)(c * 2 + 1) * g.N + e] = nq;
      }
    }
    return;
  }
  if (EP == 1 && item < Cc) {
    // ---- edge item
    const int e = item;
    const int64_t eg = chunk_first(g, c) + e;   // in the step's edge arrays
    const int s = b.src[eg];
    const int t = b.dst[eg];
    const int r = edge_relation(g, b.rel, eg);
    Row x, y, th;
    row_load(x, b.emb_i + (int64_t)s * d, d, cplx, lane);
    row_load(y, b.emb_j + (int64_t)t * d, d, cplx, lane);
    if (g.op != OP_IDENTITY && g.op != OP_LINEAR) row_load(th, b.relp + (int64_t)r * g.dr, d, cplx, lane);
    else row_zero(th);
    float* qrow = b.qk + ((int64_t)(c * 2 + 0) * g.C + e) * dp;
    float* krow = b.qk + ((int64_t)(c * 2 + 1) * g.C + e) * dp;
    float* n0row = b.nn + ((int64_t)(c * 2 + 0) * g.N + e) * dp;
    float* n1row = b.nn + ((int64_t)(c * 2 + 1) * g.N + e) * dp;
    if (RECIP) {
      if (g.op == OP_LINEAR) {
        // Q = A_r x and K = A_{r+R} y follow per edge from the raw rows (cos:
        // kept in lin_x, the candidate rows here are unit vectors)
        if (g.cmp == CMP_COS) {
          row_store(x, b.lin_x + ((int64_t)(c * 2 + 0) * g.C + e) * dp, d, dp, cplx, lane);
          row_store(y, b.lin_x + ((int64_t)(c * 2 + 1) * g.C + e) * dp, d, dp, cplx, lane);
          const float nx = row_normalize(x);
          const float ny = row_normalize(y);
          if (lane == 0) {
            b.nrm[(int64_t)(c * 2 + 0) * g.N + e] = ny;
            b.nrm[(int64_t)(c * 2 + 1) * g.N + e] = nx;
          }
        }
        row_store(y, n0row, d, dp, cplx, lane);
        row_store(x, n1row, d, dp, cplx, lane);
        return;
      }
      Row tr;
      if (g.op != OP_IDENTITY) row_load(tr, b.relp + (int64_t)(r + g.R) * g.dr, d, cplx, lane);
      else row_zero(tr);
      Row gq = op_forward(g.op, x, th);
      Row gk = op_forward(g.op, y, tr);
      float nq = 0.f, nk = 0.f, nx = 0.f, ny = 0.f;
      if (g.cmp == CMP_COS) {
        nq = row_normalize(gq);
        nk = row_normalize(gk);
        nx = row_normalize(x);
        ny = row_normalize(y);
      }
      const float p0 = row_dot(gq, y);
      const float p1 = row_dot(gk, x);
      row_store(gq, qrow, d, dp, cplx, lane);
      row_store(gk, krow, d, dp, cplx, lane);
      row_store(y, n0row, d, dp, cplx, lane);
      row_store(x, n1row, d, dp, cplx, lane);
      if (lane == 0) {
        b.pos[(int64_t)(c * 2 + 0) * g.C + e] = p0;
        b.pos[(int64_t)(c * 2 + 1) * g.C + e] = p1;
        if (g.cmp == CMP_COS) {
          b.nrm[(int64_t)(c * 2 + 0) * g.N + e] = ny;
          b.nrm[(int64_t)(c * 2 + 1) * g.N + e] = nx;
          b.qnrm[(int64_t)(c * 2 + 0) * g.C + e] = nq;
          b.qnrm[(int64_t)(c * 2 + 1) * g.C + e] = nk;
        }
      }
      return;
    }
    if (g.op == OP_LINEAR) {
      if (g.cmp == CMP_COS) {
        // one relation: the source candidates A x_t are formed afterwards by
        // a contraction over the step's raw source rows, then normalised;
        // the destination row is normalised here
        const float ny = row_normalize(y);
        row_store(y, n0row, d, dp, cplx, lane);
        row_store(x, b.lin_x + ((int64_t)c * g.N + e) * dp, d, dp, cplx, lane);
        if (lane == 0) {
          b.bias[(int64_t)c * g.C + e] = 0.0f;
          b.nrm[(int64_t)(c * 2 + 0) * g.N + e] = ny;
        }
        return;
      }
      // dot: Q = A x and K = A^T y are formed afterwards from these raw rows
      // (one relation: as contractions over the whole step; several: per edge)
      row_store(y, n0row, d, dp, cplx, lane);
      row_store(x, n1row, d, dp, cplx, lane);
      if (lane == 0) b.bias[(int64_t)c * g.C + e] = 0.0f;
      return;
    }
    Row gq = op_forward(g.op, x, th);
    if (g.cmp == CMP_DOT) {
      Row k;
      if (g.op == OP_TRANSLATION) k = y;
      else k = op_adjoint(g.op, y, th);
      const float p = row_dot(gq, y);
      const float bs = g.op == OP_TRANSLATION ? row_dot(th, y) : 0.0f;
      row_store(gq, qrow, d, dp, cplx, lane);
      row_store(k, krow, d, dp, cplx, lane);
      row_store(y, n0row, d, dp, cplx, lane);
      row_store(x, n1row, d, dp, cplx, lane);
      if (lane == 0) {
        b.pos[(int64_t)c * g.C + e] = p;
        b.bias[(int64_t)c * g.C + e] = bs;
      }
    } else {
      const float nq = row_normalize(gq);
      const float ny = row_normalize(y);
      const float p = row_dot(gq, y);
      // Q and K are these candidate rows (QK_IN_NN)
      row_store(gq, n1row, d, dp, cplx, lane);
      row_store(y, n0row, d, dp, cplx, lane);
      if (lane == 0) {
        b.pos[(int64_t)c * g.C + e] = p;
        b.bias[(int64_t)c * g.C + e] = 0.0f;
        b.nrm[(int64_t)(c * 2 + 0) * g.N + e] = ny;
        b.nrm[(int64_t)(c * 2 + 1) * g.N + e] = nq;
      }
    }
    return;
  }

  // ---- uniform candidates: four consecutive draws k0 .. k0 + 3 of one side
  // per wave (one Philox block gives all four words, the four rows load
  // together)
  const int ng = (g.U + 3) >> 2;
  const int grp = item - ne;
  const int side = grp < ng ? 0 : 1;
  const int k0 = 4 * (grp - side * ng);
  const uint32_t rows = side == 0 ? (uint32_t)g.rows_j : (uint32_t)g.rows_i;
  int32_t u[4];
  uniform_negatives4(g.seed, g.bucket, (uint64_t)(g.chunk0 + c), (uint32_t)side, (uint32_t)k0, rows, u);
  const float* tbl = side == 0 ? b.emb_j : b.emb_i;
  Row v[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (k0 + q < g.U) row_load(v[q], tbl + (int64_t)u[q] * d, d, cplx, lane);
    else row_zero(v[q]);
  }
  float nv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  // linear + cos: the raw source candidates go to lin_x (A x and its norm follow)
  const bool raw_linear = g.op == OP_LINEAR && g.cmp == CMP_COS && side == 1 && !RECIP;
  const bool unit = g.cmp == CMP_COS && !raw_linear;
  if (unit) {
    if (side == 1 && g.op != OP_IDENTITY && !RECIP) {
      // the chunk's relation (one relation, or relation-grouped chunks): its
      // operator is applied to every source candidate
      const int rc = Cc > 0 ? wave_uniform(edge_relation(g, b.rel, chunk_first(g, c))) : 0;
      Row th;
      row_load(th, b.relp + (int64_t)rc * g.dr, d, cplx, lane);
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = op_forward(g.op, v[q], th);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) nv[q] = row_normalize(v[q]);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int k = k0 + q;
    if (k >= g.U) break;
    const int t = Cc + k;
    float* dstrow = raw_linear ? b.lin_x + ((int64_t)c * g.N + t) * dp
                               : b.nn + ((int64_t)(c * 2 + side) * g.N + t) * dp;
    row_store(v[q], dstrow, d, dp, cplx, lane);
    if (lane == 0) {
      b.neg[(int64_t)(c * 2 + side) * g.U + k] = u[q];
      if (unit) b.nrm[(int64_t)(c * 2 + side) * g.N + t] = nv[q];
    }
  }
}

// Sort keys of a window of steps, from the edges and the negative draws
// alone (so that the sorts of a whole window run as one batch before its
// steps).  The key block of chunk c of step w starts at w * stride +
// 2 (c U + f_c), f_c the offset of the chunk's first edge in its step, and
// holds [side 0: Nc][side 1: Nc]: (table, row) of the row each contribution
// row reaches and, as value, that contribution row's position in the step;
// edge e: destination t (side 0) and source s (side 1), then the uniform
// draws of each side.  With several relation rows the relation of every edge
// is keyed too (at w * rstride + f_c + e, value c relN + e, its row of the
// relation contributions), and either, with uniform_rel, the chunk's relation
// for each uniform source candidate (the cos comparator with an operator
// applies it there; at w * rstride + m_w + c U + k, m_w the step's edge count,
// value c relN + C + k) or, with reciprocal predicates, every edge's source-
// side row r + R (at w * rstride + m_w + f_c + e, value c relN + C + e).  One
// thread per edge or per four draws; src / dst / rel start at the window's
// first edge.
// Chunks: consecutive (cstart NULL: n_edges edges) or relation-grouped
// (bounds cstart[0 .. nchunks], offsets in the call's edge arrays).
__global__ __launch_bounds__(256) void window_keys_kernel(StepGeom g, const int32_t* src, const int32_t* dst,
                                                          const int32_t* rel, int64_t n_edges,
                                                          const int32_t* cstart, int nchunks, int64_t chunk0,
                                                          int S, int64_t stride, uint32_t* keys, uint32_t* vals,
                                                          uint32_t* rkeys, uint32_t* rvals, int64_t rstride,
                                                          int uniform_rel) {
  const int c = blockIdx.y, w = blockIdx.z;
  const int64_t cw = (int64_t)w * S + c;   // chunk within the window
  int Cc, first;
  int64_t e0;                              // first edge of the chunk in the window's arrays
  if (cstart) {
    if (cw >= nchunks) return;
    Cc = cstart[cw + 1] - cstart[cw];
    e0 = cstart[cw] - cstart[0];
    first = cstart[cw] - cstart[(int64_t)w * S];
  } else {
    const int64_t left = n_edges - cw * g.C;
    if (left <= 0) return;
    Cc = (int)std::min<int64_t>(g.C, left);
    e0 = cw * g.C;
    first = c * g.C;
  }
  const int Nc = Cc + g.U;
  const int ng = (g.U + 3) >> 2;
  const int item = blockIdx.x * 256 + threadIdx.x;
  const uint32_t tbl_j = g.same_table ? 0u : 1u;
  const int64_t kbase = w * stride + 2 * ((int64_t)c * g.U + first);
  int64_t m_w = 0;   // edges of the step
  if (rkeys && (uniform_rel || g.recip)) {
    const int64_t w0 = (int64_t)w * S;
    if (cstart) m_w = cstart[std::min<int64_t>(w0 + S, nchunks)] - cstart[w0];
    else m_w = std::min<int64_t>((int64_t)S * g.C, n_edges - w0 * g.C);
  }
  if (item < Cc) {
    const int e = item;
    const int64_t eg = e0 + e;
    keys[kbase + e] = (tbl_j << g.rb) | (uint32_t)dst[eg];
    vals[kbase + e] = (uint32_t)((c * 2 + 0) * g.N + e);
    keys[kbase + Nc + e] = (uint32_t)src[eg];
    vals[kbase + Nc + e] = (uint32_t)((c * 2 + 1) * g.N + e);
    if (rkeys) {
      const uint32_t r = (uint32_t)(rel ? rel[eg] : 0);
      const int64_t rw = (int64_t)w * rstride + first + e;
      rkeys[rw] = r;
      rvals[rw] = (uint32_t)((int64_t)c * g.relN + e);
      if (g.recip) {
        rkeys[rw + m_w] = r + (uint32_t)g.R;
        rvals[rw + m_w] = (uint32_t)((int64_t)c * g.relN + g.C + e);
      }
    }
    return;
  }
  const int grp = item - Cc;
  if (grp >= 2 * ng) return;
  const int side = grp < ng ? 0 : 1;
  const int k0 = 4 * (grp - side * ng);
  const uint32_t rows = side == 0 ? (uint32_t)g.rows_j : (uint32_t)g.rows_i;
  int32_t u[4];
  uniform_negatives4(g.seed, g.bucket, (uint64_t)(chunk0 + cw), (uint32_t)side, (uint32_t)k0, rows, u);
  const uint32_t r_c = (uniform_rel && side == 1) ? (uint32_t)rel[e0] : 0u;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int k = k0 + q;
    if (k >= g.U) break;
    const int t = Cc + k;
    keys[kbase + side * Nc + t] = side == 0 ? ((tbl_j << g.rb) | (uint32_t)u[q]) : (uint32_t)u[q];
    vals[kbase + side * Nc + t] = (uint32_t)((c * 2 + side) * g.N + t);
    if (uniform_rel && side == 1) {
      const int64_t rw = (int64_t)w * rstride + m_w + (int64_t)c * g.U + k;
      rkeys[rw] = r_c;
      rvals[rw] = (uint32_t)((int64_t)c * g.relN + g.C + k);
    }
  }
}

// the single relation's matrix A as row-padded copies A [d][dp] and A^T [d][dp]
// (pad columns zero), the B operands of the linear operator's contractions
__global__ void pad_linear_kernel(const float* A, int d, int dp, float* Ap, float* ATp) {
  const int n = d * dp;
  for (int idx = blockIdx.x * blockDim.x + threadIdx.x; idx < n; idx += gridDim.x * blockDim.x) {
    const int r = idx / dp, k = idx - r * dp;
    Ap[idx] = k < d ? A[r * d + k] : 0.0f;
    ATp[idx] = k < d ? A[k * d + r] : 0.0f;
  }
}

// p_e = <Q_e, x_d,e> once Q has been formed by contraction (linear operator)
__global__ __launch_bounds__(256) void positive_scores_kernel(StepGeom g, StepBufs b) {
  const int lane = threadIdx.x & 63;
  const int c = blockIdx.y;
  const int e = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (e >= chunk_edges(g, c)) return;
  Row q, y;
  row_load(q, b.qk + ((int64_t)(c * 2 + 0) * g.C + e) * g.dp, g.d, false, lane);
  row_load(y, b.nn + ((int64_t)(c * 2 + 0) * g.N + e) * g.dp, g.d, false, lane);
  const float p = row_dot(q, y);
  if (lane == 0) b.pos[(int64_t)c * g.C + e] = p;
}

// row-major d x d matrices -> transposed copies (linear operator)
__global__ void transpose_rel_kernel(const float* A, float* AT, int R, int d) {
  const int64_t n = (int64_t)R * d * d;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < n;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = idx / ((int64_t)d * d);
    const int rem = (int)(idx - r * d * d);
    const int k = rem / d, l = rem % d;
    AT[r * d * d + (int64_t)l * d + k] = A[idx];
  }
}

}  // namespace

void launch_window_keys(const StepGeom& g, const int32_t* src, const int32_t* dst, const int32_t* rel,
                        int64_t n_edges, const int32_t* cstart, int nchunks, int64_t chunk0, int S, int nsteps,
                        int64_t stride, uint32_t* keys, uint32_t* vals, uint32_t* rkeys, uint32_t* rvals,
                        int64_t rstride, int uniform_rel, hipStream_t s) {
  if (nsteps <= 0 || n_edges <= 0) return;
  dim3 grid((g.C + 2 * ((g.U + 3) / 4) + 255) / 256, S, nsteps);
  window_keys_kernel<<<grid, 256, 0, s>>>(g, src, dst, rel, n_edges, cstart, nchunks, chunk0, S, stride, keys, vals,
                                          rkeys, rvals, rstride, uniform_rel);
}

void launch_gather(const StepGeom& g, const StepBufs& b, hipStream_t s) {
  dim3 grid((g.C + 2 * ((g.U + 3) / 4) + 3) / 4, g.nchunks);
  // reciprocal predicates take their own instantiation, which keeps the
  // common kernel as small as it is without them
  const int rq = row_width_for(g.d);
  if (g.recip) {
    if (rq == 2) gather_op_kernel<2, true, 1><<<grid, 256, 0, s>>>(g, b);
    else if (rq == 4) gather_op_kernel<4, true, 1><<<grid, 256, 0, s>>>(g, b);
    else gather_op_kernel<8, true, 1><<<grid, 256, 0, s>>>(g, b);
  } else {
    if (QK_IN_NN(g) && g.op != OP_LINEAR) {
      const dim3 grid2(((g.C + 1) / 2 + 2 * ((g.U + 3) / 4) + 3) / 4, g.nchunks);
      if (rq == 2) gather_op_kernel<2, false, 2><<<grid2, 256, 0, s>>>(g, b);
      else if (rq == 4) gather_op_kernel<4, false, 2><<<grid2, 256, 0, s>>>(g, b);
      else gather_op_kernel<8, false, 2><<<grid2, 256, 0, s>>>(g, b);
    } else if (rq == 2) {
      gather_op_kernel<2, false, 1><<<grid, 256, 0, s>>>(g, b);
    } else if (rq == 4) {
      gather_op_kernel<4, false, 1><<<grid, 256, 0, s>>>(g, b);
    } else {
      gather_op_kernel<8, false, 1><<<grid, 256, 0, s>>>(g, b);
    }
  }
}

void launch_transpose_rel(const float* A, float* AT, int R, int d, hipStream_t s) {
  const int64_t n = (int64_t)R * d * d;
  int blocks = (int)((n + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  transpose_rel_kernel<<<blocks, 256, 0, s>>>(A, AT, R, d);
}

void launch_pad_linear(const float* A, int d, int dp, float* Ap, float* ATp, hipStream_t s) {
  const int n = d * dp;
  int blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  pad_linear_kernel<<<blocks, 256, 0, s>>>(A, d, dp, Ap, ATp);
}

void launch_positive_scores(const StepGeom& g, const StepBufs& b, hipStream_t s) {
  dim3 grid((g.C + 3) / 4, g.nchunks);
  positive_scores_kernel<<<grid, 256, 0, s>>>(g, b);
}
