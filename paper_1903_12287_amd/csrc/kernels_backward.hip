// Loss values and gradients of a step (Sec. 3.1 losses) and the backward pass
// through the comparator and the relation operator.
//
// After the contractions, for chunk c and side s:
//   dq[c][s][e] = sum_t dS_s[e][t] N_s[t]      (gradient of side s's query row)
//   dn[c][s][t] = sum_e dS_s[e][t] Q_s[e]      (gradient of candidate row t)
// The positive score p_e = sim(g(x_s), x_d) is computed once and shared by
// both sides; dL/dp_e collects both sides.  With reciprocal predicates each
// side has its own positive score and its own dL/dp.  op_backward folds everything that
// reaches one embedding row of the chunk into that row's contribution,
// in place in dn: side 0 rows are destinations (in-chunk, then uniform
// draws from partition j), side 1 rows are sources (partition i).
#include "kernels.h"
#include "finalize_body.h"
#include "row_ops.h"

namespace {

// ---- per-edge dL/dp, translation bias gradient, losses ------------------------
__global__ __launch_bounds__(FIN_THREADS) void finalize_kernel(StepGeom g, StepBufs b, int softmax_scales,
                                                                double* parts) {
  finalize_block(g, b, softmax_scales, parts, blockIdx.y, blockIdx.x, gridDim.x);
}

// Step losses from the finalisation's partials: wave t adds the n partials of
// step t in a fixed order (lane l sums partials l, l + 64, ..., then a fixed
// butterfly over the wave).
__global__ __launch_bounds__(64) void step_loss_kernel(const double* parts, int64_t stride, int n_full, int n_last,
                                                       int64_t nsteps, double* out) {
  const int64_t t = blockIdx.x;
  if (t >= nsteps) return;
  const int n = t == nsteps - 1 ? n_last : n_full;
  const double* p = parts + t * stride;
  double sum = 0.0;
#pragma unroll 8
  for (int i = threadIdx.x; i < n; i += 64) sum += p[i];
  sum = wave_sum_d(sum);
  if (threadIdx.x == 0) out[t] = sum;
}

// ---- operator / comparator backward: contributions and sort keys -----------
// Reciprocal predicates, edge e of chunk c: Q = g(x_s, theta_r) and
// K = g(x_d, theta_{r+R}) against the entity rows (unit vectors for cos), the
// positive scores p0 = sim(Q, x_d) and p1 = sim(K, x_s).  The source row
// collects its candidate gradient, p1's term and J_g(theta_r)^T dQ, the
// destination row likewise with p0 and theta_{r+R}; the two parameter rows'
// contributions go to relc rows c relN + e and c relN + C + e.  The linear
// operator leaves dL/dQ and dL/dK in dq for its per-edge products.
template <int RQ>
__device__ __forceinline__ void op_backward_reciprocal(const StepGeom& g, const StepBufs& b, int c, int e, int s,
                                                       int t, int r, const RowT<RQ>& th, int lane) {
  using RowR = RowT<RQ>;
  const bool cplx = g.op == OP_COMPLEX;
  const bool cos = g.cmp == CMP_COS;
  const int d = g.d, dp = g.dp;
  const float dp0 = b.dpos[pos_index(g, c, 0, e)];
  const float dp1 = b.dpos[pos_index(g, c, 1, e)];
  RowR tr;
  if (g.op != OP_IDENTITY && g.op != OP_LINEAR) row_load(tr, b.relp + (int64_t)(r + g.R) * g.dr, d, cplx, lane);
  else row_zero(tr);
  float* dq0 = b.dq + ((int64_t)(c * 2 + 0) * g.C + e) * dp;
  float* dq1 = b.dq + ((int64_t)(c * 2 + 1) * g.C + e) * dp;
  float* dn0 = b.dn + ((int64_t)(c * 2 + 0) * g.N + e) * dp;
  float* dn1 = b.dn + ((int64_t)(c * 2 + 1) * g.N + e) * dp;
  RowR Q, K, xh, yh, dQ, dK, dX, dY;
  row_load(Q, b.qk + ((int64_t)(c * 2 + 0) * g.C + e) * dp, d, cplx, lane);
  row_load(K, b.qk + ((int64_t)(c * 2 + 1) * g.C + e) * dp, d, cplx, lane);
  row_load(yh, b.nn + ((int64_t)(c * 2 + 0) * g.N + e) * dp, d, cplx, lane);
  row_load(xh, b.nn + ((int64_t)(c * 2 + 1) * g.N + e) * dp, d, cplx, lane);
  row_load(dQ, dq0, d, cplx, lane);
  row_load(dK, dq1, d, cplx, lane);
  row_load(dY, dn0, d, cplx, lane);
  row_load(dX, dn1, d, cplx, lane);
  row_axpy(dQ, dp0, yh);   // p0 = <Q, y>
  row_axpy(dK, dp1, xh);   // p1 = <K, x>
  row_axpy(dY, dp0, Q);
  row_axpy(dX, dp1, K);
  RowR x = xh, y = yh;     // the operators' inputs
  if (cos) {
    dQ = normalize_backward(Q, b.qnrm[(int64_t)(c * 2 + 0) * g.C + e], dQ);
    dK = normalize_backward(K, b.qnrm[(int64_t)(c * 2 + 1) * g.C + e], dK);
    dY = normalize_backward(yh, b.nrm[(int64_t)(c * 2 + 0) * g.N + e], dY);
    dX = normalize_backward(xh, b.nrm[(int64_t)(c * 2 + 1) * g.N + e], dX);
    if (g.op == OP_DIAGONAL || g.op == OP_COMPLEX) {
      row_load(x, b.emb_i + (int64_t)s * d, d, cplx, lane);
      row_load(y, b.emb_j + (int64_t)t * d, d, cplx, lane);
    }
  }
  if (g.op == OP_LINEAR) {
    row_store(dQ, dq0, d, dp, cplx, lane);
    row_store(dK, dq1, d, dp, cplx, lane);
  } else {
    row_add(dX, op_adjoint(g.op, dQ, th));   // identity: dQ itself
    row_add(dY, op_adjoint(g.op, dK, tr));
  }
  if (g.op != OP_LINEAR && g.op != OP_IDENTITY) {
    const RowR gf = op_param_grad(g.op, x, dQ);
    const RowR gr = op_param_grad(g.op, y, dK);
    row_store(gf, b.relc + ((int64_t)c * g.relN + e) * g.dr, d, g.dr, cplx, lane);
    row_store(gr, b.relc + ((int64_t)c * g.relN + g.C + e) * g.dr, d, g.dr, cplx, lane);
  }
  row_store(dY, dn0, d, dp, cplx, lane);
  row_store(dX, dn1, d, dp, cplx, lane);
}

// One item of the operator / normalisation backward: edge `item` of chunk c,
// or four uniform candidates of one side.  Relation-parameter gradient rows
// go to relc, or with RELSUM (one relation shared by every edge) are added to
// rsum.
template <int RQ, bool RELSUM>
__device__ __forceinline__ void op_backward_item(const StepGeom& g, const StepBufs& b, int c, int Cc, int item,
                                                 int lane, RowT<RQ>& rsum) {
  using Row = RowT<RQ>;
  const bool cplx = g.op == OP_COMPLEX;
  const int d = g.d, dp = g.dp;
  const bool cos = g.cmp == CMP_COS;
  const bool has_rel = g.op != OP_IDENTITY;

  if (item < Cc) {
    const int e = item;
    const int64_t ce = (int64_t)c * g.C + e;
    const int64_t eg = chunk_first(g, c) + e;   // in the step's edge arrays
    const int s = b.src[eg];
    const int t = b.dst[eg];
    const int r = edge_relation(g, b.rel, eg);
    Row th;
    if (has_rel && g.op != OP_LINEAR) row_load(th, b.relp + (int64_t)r * g.dr, d, cplx, lane);
    else row_zero(th);
    if (!RELSUM && g.recip) {   // reciprocal predicates make 2R relation operators: never RELSUM
      op_backward_reciprocal(g, b, c, e, s, t, r, th, lane);
      return;
    }
    const float dpe = b.dpos[ce];
    float* dq0 = b.dq + ((int64_t)(c * 2 + 0) * g.C + e) * dp;
    const float* dq1 = b.dq + ((int64_t)(c * 2 + 1) * g.C + e) * dp;
    float* dn0 = b.dn + ((int64_t)(c * 2 + 0) * g.N + e) * dp;
    float* dn1 = b.dn + ((int64_t)(c * 2 + 1) * g.N + e) * dp;
    const float* q = QK_IN_NN(g) ? b.nn + ((int64_t)(c * 2 + 1) * g.N + e) * dp
                                 : b.qk + ((int64_t)(c * 2 + 0) * g.C + e) * dp;
    const float* kr = QK_IN_NN(g) ? b.nn + ((int64_t)(c * 2 + 0) * g.N + e) * dp
                                  : b.qk + ((int64_t)(c * 2 + 1) * g.C + e) * dp;
    Row Q, Kv, gq0, gq1, gn0, gn1;
    row_load(Q, q, d, cplx, lane);
    row_load(Kv, kr, d, cplx, lane);
    row_load(gq0, dq0, d, cplx, lane);
    row_load(gq1, dq1, d, cplx, lane);
    if (g.dq_has_dn) {
      // the ranking backward added dn of side 1 - s into dq of side s
      row_zero(gn0);
      row_zero(gn1);
    } else {
      row_load(gn0, dn0, d, cplx, lane);
      row_load(gn1, dn1, d, cplx, lane);
    }
    Row gs, gd, grel;
    row_zero(grel);
    if (!cos) {
      // raw rows: x_s is N1[e], x_d is N0[e]
      Row x, y;
      row_load(x, b.nn + ((int64_t)(c * 2 + 1) * g.N + e) * dp, d, cplx, lane);
      row_load(y, b.nn + ((int64_t)(c * 2 + 0) * g.N + e) * dp, d, cplx, lane);
      Row dQ = gq0;
      row_axpy(dQ, dpe, y);                         // positive: dp * x_d
      const float dsum = b.dsum1[ce];               // gradient of the translation bias
      // source row: J_g^T dQ + its in-chunk candidate gradient
      // (linear: A^T dQ and A dK are added afterwards by contractions over the
      // whole step, see the launch sequence)
      if (g.op == OP_LINEAR) row_zero(gs);
      else gs = op_adjoint(g.op, dQ, th);
      row_add(gs, gn1);
      // destination row: candidate gradient + positive + J_{g*}^T dK (+ bias)
      gd = gn0;
      row_axpy(gd, dpe, Q);
      Row jk;
      if (g.op == OP_LINEAR) row_zero(jk);
      else if (g.op == OP_DIAGONAL || g.op == OP_COMPLEX) jk = op_forward(g.op, gq1, th);
      else jk = gq1;
      row_add(gd, jk);
      if (g.op == OP_TRANSLATION) row_axpy(gd, dsum, th);
      if (g.op == OP_TRANSLATION) {
        grel = dQ;
        row_axpy(grel, dsum, y);
      } else if (g.op == OP_DIAGONAL || g.op == OP_COMPLEX) {
        grel = op_param_grad(g.op, x, dQ);
        row_add(grel, op_adjoint_param_grad(g.op, y, gq1));
      } else if (g.op == OP_LINEAR) {
        row_store(dQ, dq0, d, dp, false, lane);     // dA = dQ^T X + Y^T dK, by contraction
      }
    } else {
      const float nq = b.nrm[(int64_t)(c * 2 + 1) * g.N + e];
      const float ny = b.nrm[(int64_t)(c * 2 + 0) * g.N + e];
      Row dQh = gq0;                                 // Q^ is also source candidate e
      row_axpy(dQh, dpe, Kv);
      row_add(dQh, gn1);
      Row dYh = gn0;                                 // x^_d is destination candidate e and K^_e
      row_add(dYh, gq1);
      row_axpy(dYh, dpe, Q);
      const Row dv = normalize_backward(Q, nq, dQh); // dL/dg(x_s)
      gs = op_adjoint(g.op, dv, th);                 // linear: dv itself (A^T dv follows)
      gd = normalize_backward(Kv, ny, dYh);
      if (g.op == OP_TRANSLATION) {
        grel = dv;
      } else if (g.op == OP_DIAGONAL || g.op == OP_COMPLEX) {
        Row x;
        row_load(x, b.emb_i + (int64_t)s * d, d, cplx, lane);
        grel = op_param_grad(g.op, x, dv);
      }
    }
    row_store(gd, dn0, d, dp, cplx, lane);
    // linear + cos: dL/d(A x_s) goes to lin_v, and the source row gradient
    // A^T dv is formed by a contraction over the step's source candidates
    float* srow = (cos && g.op == OP_LINEAR) ? b.lin_v + ((int64_t)c * g.N + e) * dp : dn1;
    row_store(gs, srow, d, dp, cplx, lane);
    if (RELSUM) row_add(rsum, grel);
    else if (has_rel && g.op != OP_LINEAR)
      row_store(grel, b.relc + ((int64_t)c * g.relN + e) * g.dr, d, g.dr, cplx, lane);
    return;
  }

  // uniform candidate rows, four consecutive candidates of one side per wave
  // (all their rows load together); with the dot comparator their gradients
  // are dS^T Q as the contraction left them
  if (!cos) return;
  const int ng = (g.U + 3) >> 2;
  const int grp = item - Cc;
  const int side = grp < ng ? 0 : 1;
  const int k0 = 4 * (grp - side * ng);
  const int nq = min(4, g.U - k0);
  const int64_t rbase = (int64_t)(c * 2 + side) * g.N + Cc + k0;   // row of candidate k0
  int32_t u[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) u[q] = q < nq ? b.neg[(int64_t)(c * 2 + side) * g.U + k0 + q] : 0;
  {
    Row vh[4], gv[4];
    float nv[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (q < nq) {
        row_load(vh[q], b.nn + (rbase + q) * dp, d, cplx, lane);
        row_load(gv[q], b.dn + (rbase + q) * dp, d, cplx, lane);
        nv[q] = b.nrm[rbase + q];
      } else {
        row_zero(vh[q]);
        row_zero(gv[q]);
        nv[q] = 1.0f;
      }
    }
    Row th;
    // the single relation's operator was applied here (linear: A^T dv follows
    // as a contraction, the gradient of A too)
    const bool lin_side = side == 1 && g.op == OP_LINEAR && !g.recip;
    const bool op_side = side == 1 && has_rel && !lin_side && !g.recip;
    // the chunk's relation (one relation, or relation-grouped chunks)
    const int rc = (op_side && Cc > 0) ? wave_uniform(edge_relation(g, b.rel, chunk_first(g, c))) : 0;
    if (op_side) row_load(th, b.relp + (int64_t)rc * g.dr, d, cplx, lane);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (q >= nq) break;
      Row dv = normalize_backward(vh[q], nv[q], gv[q]);
      if (op_side) {
        Row grel = dv;   // translation: the parameter gradient is dv itself
        if (g.op != OP_TRANSLATION) {
          Row x;
          row_load(x, b.emb_i + (int64_t)u[q] * d, d, cplx, lane);
          grel = op_param_grad(g.op, x, dv);
        }
        if (RELSUM) row_add(rsum, grel);
        else row_store(grel, b.relc + ((int64_t)c * g.relN + g.C + k0 + q) * g.dr, d, g.dr, cplx, lane);
        dv = op_adjoint(g.op, dv, th);
      }
      float* drow = lin_side ? b.lin_v + ((int64_t)c * g.N + Cc + k0 + q) * dp : b.dn + (rbase + q) * dp;
      row_store(dv, drow, d, dp, cplx, lane);
    }
  }
}

template <int RQ, bool RELSUM>
__global__ __launch_bounds__(256) void op_backward_kernel(StepGeom g, StepBufs b) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int c = blockIdx.y;
  const int Cc = chunk_edges(g, c);
  const int item = blockIdx.x * 4 + w;
  RowT<RQ> rsum;
  row_zero(rsum);
  if (item < Cc + 2 * ((g.U + 3) >> 2)) op_backward_item<RQ, RELSUM>(g, b, c, Cc, item, lane, rsum);
  if (!RELSUM) return;
  // one relation: the four waves' sums are added in wave order and the block
  // writes one row, relc row blockIdx.x of chunk c (every block writes its
  // row, zero where no wave had an item)
  __shared__ float red[4][RQ * 64];
#pragma unroll
  for (int q = 0; q < RQ; ++q) red[w][q * 64 + lane] = rsum.v[q];
  __syncthreads();
  if (w != 0) return;
  RowT<RQ> tot;
#pragma unroll
  for (int q = 0; q < RQ; ++q) {
    const int f = q * 64 + lane;
    tot.v[q] = (red[0][f] + red[1][f]) + (red[2][f] + red[3][f]);
  }
  row_store(tot, b.relc + ((int64_t)c * gridDim.x + blockIdx.x) * g.dr, g.d, g.dr, g.op == OP_COMPLEX, lane);
}

}  // namespace


void launch_finalize(const StepGeom& g, const StepBufs& b, double* parts, bool softmax_scales, hipStream_t s) {
  const int fb = fin_blocks(g.C);
  finalize_kernel<<<dim3(fb, g.nchunks), FIN_THREADS, 0, s>>>(g, b, softmax_scales ? 1 : 0, parts);
}

void launch_step_losses(const double* parts, int64_t stride, int n_full, int n_last, int64_t nsteps, double* out,
                        hipStream_t s) {
  if (nsteps <= 0) return;
  step_loss_kernel<<<(unsigned)nsteps, 64, 0, s>>>(parts, stride, n_full, n_last, nsteps, out);
}

void launch_op_backward(const StepGeom& g, const StepBufs& b, hipStream_t s) {
  // waves for the uniform candidates only where the cos normalisation has a
  // backward to run
  dim3 grid(op_backward_blocks(g.C, g.U, g.cmp), g.nchunks);
  const int rq = row_width_for(g.d);
  if (g.relsum) {
    if (rq == 2) op_backward_kernel<2, true><<<grid, 256, 0, s>>>(g, b);
    else if (rq == 4) op_backward_kernel<4, true><<<grid, 256, 0, s>>>(g, b);
    else op_backward_kernel<8, true><<<grid, 256, 0, s>>>(g, b);
  } else {
    if (rq == 2) op_backward_kernel<2, false><<<grid, 256, 0, s>>>(g, b);
    else if (rq == 4) op_backward_kernel<4, false><<<grid, 256, 0, s>>>(g, b);
    else op_backward_kernel<8, false><<<grid, 256, 0, s>>>(g, b);
  }
}
