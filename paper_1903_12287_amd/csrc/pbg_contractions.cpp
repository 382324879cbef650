// Launch sequences of the three chunk contractions of a step (score with its
// loss epilogue, dQ = dS.N, dN = dS^T.Q), in float32 or with bfloat16 inputs.
#include <hip/hip_runtime.h>

#include <cstring>

#include "kernels.h"
#include "runtime_internal.h"

static int rup(int v, int m) { return (v + m - 1) / m * m; }

// dQ = dS . N and dN = dS^T . Q on the bf16 matrix instructions.  A is dS:
// the ranking bit matrix (rows for dQ, columns for dN), else bf16 rows dsh.
// B is N^T [f][t] / Q^T [f][e] in bf16, as `planes` pieces (1: bf16 operands;
// 3: the exact pieces of the float32 operands, ranking only) n_ps / q_ps
// elements apart.
static void run_backward_h(const StepGeom& g, const StepBufs& b, const uint16_t* dsh, const uint16_t* nT,
                           int64_t n_ps, const uint16_t* qT, int64_t q_ps, int64_t q_cs, int64_t q_ss, int q_ld,
                           int planes, hipStream_t cs, bool merge = false) {
  const int C = g.C, N = g.N, dp = g.dp, Np = g.Np, nch = g.nchunks;
  const int dpb = rup(g.d, 32), Cpb = rup(C, 32), Npb = rup(N, 32);
  const bool bits = g.loss == LOSS_RANKING;
  const int nw = (Np + 15) / 16, ldw = rup(C, 8);
  // dQ = dS . N:  A = dS (rows), B = N^T [f][t]
  GemmArgsH qa;
  memset(&qa, 0, sizeof(qa));
  if (bits) {
    qa.A = b.dsb;
    qa.amode = GA_BITS_ROW;
    qa.a_cs = 2ll * nw * ldw;
    qa.a_ss = (int64_t)nw * ldw;
    qa.lda = ldw;
  } else {
    qa.A = dsh;
    qa.amode = GA_KC;
    qa.a_cs = 2ll * C * Npb;
    qa.a_ss = (int64_t)C * Npb;
    qa.lda = Npb;
  }
  qa.B = nT;
  qa.planes = planes;
  qa.b_ps = n_ps;
  qa.Cm = b.dq;
  qa.b_cs = 2ll * dpb * Npb;
  qa.b_ss = (int64_t)dpb * Npb;
  qa.c_cs = 2ll * C * dp;
  qa.c_ss = (int64_t)C * dp;
  qa.ldb = Npb;
  qa.ldc = dp;
  qa.mdim = DIM_CC;
  qa.ndim = DIM_FIXED;
  qa.Nfix = dp;
  qa.kdim = DIM_NC;
  qa.C = C;
  qa.U = g.U;
  qa.m_step = g.m_step;
  qa.cstart = g.cstart;
  qa.nsides = 2;
  // dN = dS^T . Q:  A = dS read by columns, B = Q^T [f][e]
  GemmArgsH na = qa;
  na.amode = bits ? GA_BITS_COL : GA_MC;
  na.B = qT;
  na.b_ps = q_ps;
  na.Cm = b.dn;
  na.b_cs = q_cs;
  na.b_ss = q_ss;
  na.c_cs = 2ll * N * dp;
  na.c_ss = (int64_t)N * dp;
  na.ldb = q_ld;
  na.mdim = DIM_NC;
  na.kdim = DIM_CC;
  // the relation weight of each chunk scales its gradients (NULL: weight 1)
  qa.cscale = na.cscale = g.cweight;
  // dN rows e < Cc of side 1 - s into dQ of side s (the same vectors)
  qa.merge_cc = na.merge_cc = merge ? 1 : 0;
  launch_gemm_bf16_pair(qa, na, nch * 2, cs);
}

// Arguments of the float32 score contraction of a step with its loss
// epilogue (operands, dS and row-partial outputs); *epi receives the epilogue
// the loss takes
static GemmArgsH score_args_f32(const StepGeom& g, const StepBufs& b, int* epi_out) {
  const int C = g.C, U = g.U, N = g.N, dp = g.dp, Np = g.Np;
  // ranking: dS is 0 or 1 and travels as bits, 16 columns per word
  const bool bits = g.loss == LOSS_RANKING;
  GemmArgsH fa;
  memset(&fa, 0, sizeof(fa));
  fa.Bf = b.nn;
  fa.Cm = b.ds;
  if (QK_IN_NN(g)) {
    // side s reads the candidate rows of side 1 - s, so the scores of side 1
    // against the chunk's own candidates are the transposed ones of side 0
    fa.Af = b.nn + (int64_t)N * dp;
    fa.a_cs = 2ll * N * dp;
    fa.a_ss = -(int64_t)N * dp;
    fa.share_cc = 1;
  } else {
    fa.Af = b.qk;
    fa.a_cs = 2ll * C * dp;
    fa.a_ss = (int64_t)C * dp;
  }
  fa.b_cs = 2ll * N * dp;
  fa.b_ss = (int64_t)N * dp;
  fa.c_cs = 2ll * C * Np;
  fa.c_ss = (int64_t)C * Np;
  fa.lda = dp;
  fa.ldb = dp;
  fa.ldc = Np;
  fa.mdim = DIM_CC;
  fa.ndim = DIM_NC;
  fa.kdim = DIM_FIXED;
  fa.Kfix = g.d;
  fa.C = C;
  fa.U = U;
  fa.m_step = g.m_step;
  fa.cstart = g.cstart;
  fa.nsides = 2;
  fa.pos = b.pos;
  fa.pos_sides = g.recip ? 2 : 1;
  fa.bias = (g.op == OP_TRANSLATION && g.cmp == CMP_DOT && !g.recip) ? b.bias : nullptr;
  fa.rowpart = b.rowpart;
  fa.nct = g.nct;
  fa.loss = g.loss;
  fa.margin = g.margin;
  const int nw = (Np + 15) / 16, ldw = rup(C, 8);   // bit-matrix words per row, row pitch
  int epi = g.loss == LOSS_SOFTMAX ? EPI_SOFTMAX_EXP : EPI_LOSS;
  if (bits) {
    epi = EPI_LOSS_BITS;
    fa.dsb = b.dsb;
    fa.cb_cs = 2ll * nw * ldw;
    fa.cb_ss = (int64_t)nw * ldw;
    fa.ldcb = ldw;
    fa.nwcb = nw;
  }
  *epi_out = epi;
  return fa;
}

void run_contractions_f32(pbg_ctx* ctx, const StepGeom& g, const StepBufs& b, int64_t t, hipStream_t cs,
                          const std::function<void(int)>& mark, bool forward_only) {
  const int C = g.C, U = g.U, N = g.N, dp = g.dp, Np = g.Np, nch = g.nchunks;
  const bool bits = g.loss == LOSS_RANKING;
  int epi = EPI_LOSS;
  const GemmArgsH fa = score_args_f32(g, b, &epi);
  launch_score_split(fa, epi, nch * 2, cs);
  mark(2);
  // softmax: the score pass leaves exp(s - tile max), the finalisation each
  // row's log-sum-exp and per-tile scales, and the backward forms dS as it
  // stages the exponentials
  double* const parts = ctx->lossparts + t * ctx->lossparts_pps;
  if (forward_only) {
    launch_finalize(g, b, parts, g.loss == LOSS_SOFTMAX, cs);
    mark(3);
    return;
  }
  // Q and N in three exact bf16 pieces each, transposed (the B operands of
  // both backward products), in the same launch as the finalisation.  On the
  // second stream beside the score contraction it delays the score kernel by
  // as much as it saves here.
  const int dpb = rup(g.d, 32), Cpb = rup(C, 32), Npb = rup(N, 32);
  const BufsH& h = ctx->h;
  // with QK_IN_NN, Q^T of side s is the first C columns of N^T of side 1 - s
  const bool qn = QK_IN_NN(g);
  launch_finalize_split3_t(g, b, parts, g.loss == LOSS_SOFTMAX, qn ? nullptr : b.qk, (int64_t)C * dp, C, h.qkT3,
                           (int64_t)dpb * Cpb, h.q3_ps, Cpb, b.nn, (int64_t)N * dp, N, h.nnT3, (int64_t)dpb * Npb,
                           h.n3_ps, Npb, dp, dpb, nch * 2, cs);
  mark(3);
  if (bits) {
    // dS is 0 or 1: its products with the pieces are exact (float32 sums)
    if (qn)
      run_backward_h(g, b, nullptr, h.nnT3, h.n3_ps, h.nnT3 + (int64_t)dpb * Npb, h.n3_ps, 2ll * dpb * Npb,
                     -(int64_t)dpb * Npb, Npb, 3, cs, g.dq_has_dn != 0);
    else
      run_backward_h(g, b, nullptr, h.nnT3, h.n3_ps, h.qkT3, h.q3_ps, 2ll * dpb * Cpb, (int64_t)dpb * Cpb, Cpb, 3,
                     cs);
    return;
  }
  // general float32 dS (logistic, softmax): split into pieces as it is staged,
  // six piece products
  GemmArgsH qa;
  memset(&qa, 0, sizeof(qa));
  qa.Af = b.ds;
  qa.smscale = g.loss == LOSS_SOFTMAX ? b.rowscale : nullptr;
  qa.nct = g.nct;
  qa.a_cs = 2ll * C * Np;
  qa.a_ss = (int64_t)C * Np;
  qa.lda = Np;
  qa.B = h.nnT3;
  qa.planes = 3;
  qa.b_ps = h.n3_ps;
  qa.b_cs = 2ll * dpb * Npb;
  qa.b_ss = (int64_t)dpb * Npb;
  qa.ldb = Npb;
  qa.Cm = b.dq;
  qa.c_cs = 2ll * C * dp;
  qa.c_ss = (int64_t)C * dp;
  qa.ldc = dp;
  qa.mdim = DIM_CC;
  qa.ndim = DIM_FIXED;
  qa.Nfix = dp;
  qa.kdim = DIM_NC;
  qa.C = C;
  qa.U = U;
  qa.m_step = g.m_step;
  qa.cstart = g.cstart;
  qa.nsides = 2;
  GemmArgsH na = qa;
  if (qn) {
    na.B = h.nnT3 + (int64_t)dpb * Npb;   // Q^T of side s: N^T of side 1 - s
    na.b_ps = h.n3_ps;
    na.b_cs = 2ll * dpb * Npb;
    na.b_ss = -(int64_t)dpb * Npb;
    na.ldb = Npb;
  } else {
    na.B = h.qkT3;
    na.b_ps = h.q3_ps;
    na.b_cs = 2ll * dpb * Cpb;
    na.b_ss = (int64_t)dpb * Cpb;
    na.ldb = Cpb;
  }
  na.Cm = b.dn;
  na.c_cs = 2ll * N * dp;
  na.c_ss = (int64_t)N * dp;
  na.mdim = DIM_NC;
  na.kdim = DIM_CC;
  qa.cscale = na.cscale = g.cweight;   // the chunks' relation weights
  launch_gemm_split_pair(qa, na, nch * 2, cs);
}

// Operands of the bf16-input score contraction of a step (the rounded copies
// of Q and N) and its epilogue's per-row inputs
static GemmArgsH score_args_bf16(pbg_ctx* ctx, const StepGeom& g, const StepBufs& b) {
  const int C = g.C, U = g.U, N = g.N, d = g.d;
  const int dpb = rup(d, 32);
  const BufsH& h = ctx->h;
  const bool qn = QK_IN_NN(g);
  GemmArgsH fa;
  memset(&fa, 0, sizeof(fa));
  fa.B = h.nn;
  fa.amode = GA_KC;
  if (qn) {
    fa.A = h.nn + (int64_t)N * dpb;
    fa.a_cs = 2ll * N * dpb;
    fa.a_ss = -(int64_t)N * dpb;
  } else {
    fa.A = h.qk;
    fa.a_cs = 2ll * C * dpb;
    fa.a_ss = (int64_t)C * dpb;
  }
  fa.b_cs = 2ll * N * dpb;
  fa.b_ss = (int64_t)N * dpb;
  fa.lda = dpb;
  fa.ldb = dpb;
  fa.mdim = DIM_CC;
  fa.ndim = DIM_NC;
  fa.kdim = DIM_FIXED;
  fa.Kfix = d;
  fa.C = C;
  fa.U = U;
  fa.m_step = g.m_step;
  fa.cstart = g.cstart;
  fa.nsides = 2;
  fa.pos = b.pos;
  fa.pos_sides = g.recip ? 2 : 1;
  fa.bias = (g.op == OP_TRANSLATION && g.cmp == CMP_DOT && !g.recip) ? b.bias : nullptr;
  fa.rowpart = b.rowpart;
  fa.nct = g.nct;
  fa.loss = g.loss;
  fa.margin = g.margin;
  return fa;
}

void run_contractions_bf16(pbg_ctx* ctx, const StepGeom& g, const StepBufs& b, int64_t t,
                           hipStream_t cs, const std::function<void(int)>& mark, bool forward_only) {
  const int C = g.C, U = g.U, N = g.N, d = g.d, dp = g.dp, Np = g.Np, nch = g.nchunks;
  const int dpb = rup(d, 32), Cpb = rup(C, 32), Npb = rup(N, 32);
  const BufsH& h = ctx->h;
  // bf16 operands: rows [e][f], [t][f] and the transposed copies [f][e], [f][t]
  // with QK_IN_NN, the Q rows of side s are the first C rows of N of side
  // 1 - s (and Q^T the first C columns of N^T): only N is converted
  const bool qn = QK_IN_NN(g);
  launch_to_bf16_t(qn ? nullptr : b.qk, (int64_t)C * dp, C, h.qk, (int64_t)C * dpb, h.qkT, (int64_t)dpb * Cpb, Cpb, b.nn,
                   (int64_t)N * dp, N, h.nn, (int64_t)N * dpb, h.nnT, (int64_t)dpb * Npb, Npb, dp, dpb, nch * 2, cs);
  mark(1);   // recorded again: the score bracket starts after the operand rounding

  const bool bits = g.loss == LOSS_RANKING;
  const int nw = (Np + 15) / 16, ldw = rup(C, 8);
  GemmArgsH fa = score_args_bf16(ctx, g, b);
  if (bits) {
    fa.dsb = b.dsb;
    fa.cb_cs = 2ll * nw * ldw;
    fa.cb_ss = (int64_t)nw * ldw;
    fa.ldcb = ldw;
    fa.nwcb = nw;
    launch_gemm_bf16(fa, EPI_LOSS_BITS, nch * 2, cs);
    mark(2);
  } else if (g.loss == LOSS_SOFTMAX) {
    fa.Cm = b.ds;
    fa.c_cs = 2ll * C * Np;
    fa.c_ss = (int64_t)C * Np;
    fa.ldc = Np;
    launch_gemm_bf16(fa, EPI_SOFTMAX_STATS, nch * 2, cs);
    mark(2);
    launch_softmax_rows_bf16(g, b, h.ds, Npb, cs);
  } else {
    fa.dsh = h.ds;
    fa.c_cs = 2ll * C * Npb;
    fa.c_ss = (int64_t)C * Npb;
    fa.ldc = Npb;
    launch_gemm_bf16(fa, EPI_LOSS, nch * 2, cs);
    mark(2);
  }
  launch_finalize(g, b, ctx->lossparts + t * ctx->lossparts_pps, false, cs);
  mark(3);
  if (forward_only) return;

  if (qn)
    run_backward_h(g, b, h.ds, h.nnT, 0, h.nnT + (int64_t)dpb * Npb, 0, 2ll * dpb * Npb, -(int64_t)dpb * Npb, Npb,
                   1, cs);
  else
    run_backward_h(g, b, h.ds, h.nnT, 0, h.qkT, 0, 2ll * dpb * Cpb, (int64_t)dpb * Cpb, Cpb, 1, cs);
}

// Linear operator with one relation (Sec. 4.3: with a single relation the
// operator of a batch is one matrix product): Q = X A^T and K = Y A over all
// chunks of the step, from the raw rows the gather left in the candidate
// buffers (x_s is source candidate e, x_d destination candidate e), then the
// positive scores.  Ap / ATp are A and A^T with rows padded to dp.
static GemmArgs linear_args(const StepGeom& g, const float* A, int64_t a_cs, const float* B, float* Cm,
                            int64_t c_cs) {
  GemmArgs la;
  memset(&la, 0, sizeof(la));
  la.A = A;
  la.B = B;
  la.Cm = Cm;
  la.a_cs = a_cs;
  la.c_cs = c_cs;
  la.lda = g.dp;
  la.ldb = g.dp;
  la.ldc = g.dp;
  la.mdim = DIM_CC;
  la.ndim = DIM_FIXED;
  la.Nfix = g.d;
  la.kdim = DIM_FIXED;
  la.Kfix = g.d;
  la.C = g.C;
  la.U = g.U;
  la.m_step = g.m_step;
  la.cstart = g.cstart;
  la.nsides = 1;
  return la;
}

void run_linear_forward(const StepGeom& g, const StepBufs& b, const float* Ap, const float* ATp, hipStream_t cs) {
  const int64_t n_cs = 2ll * g.N * g.dp, q_cs = 2ll * g.C * g.dp;
  if (g.cmp == CMP_COS) {
    // A x_t for every source candidate (raw rows in lin_x) into the candidate
    // tile of side 1, then normalised, with the positive scores
    GemmArgs q = linear_args(g, b.lin_x, (int64_t)g.N * g.dp, Ap, b.nn + (int64_t)g.N * g.dp, n_cs);
    q.mdim = DIM_NC;
    launch_gemm_f32(q, GEMM_NT, g.nchunks, cs);
    launch_normalize_candidates(g, b, cs);
    return;
  }
  GemmArgs q = linear_args(g, b.nn + (int64_t)g.N * g.dp, n_cs, Ap, b.qk, q_cs);     // Q = X A^T
  launch_gemm_f32(q, GEMM_NT, g.nchunks, cs);
  GemmArgs k = linear_args(g, b.nn, n_cs, ATp, b.qk + (int64_t)g.C * g.dp, q_cs);    // K = Y A
  launch_gemm_f32(k, GEMM_NT, g.nchunks, cs);
  launch_positive_scores(g, b, cs);
}

// the operator's part of the row gradients.  dot: source rows += dQ A (i.e.
// A^T dQ), destination rows += dK A^T (i.e. A dK), added to the
// contributions that the operator backward left in the candidate-gradient
// buffer.  cos: every source candidate row's gradient is A^T dv, dv the
// gradient of its A x_t that the operator backward left in lin_v
void run_linear_backward(const StepGeom& g, const StepBufs& b, const float* Ap, const float* ATp,
                         hipStream_t cs) {
  const int64_t n_cs = 2ll * g.N * g.dp, q_cs = 2ll * g.C * g.dp;
  if (g.cmp == CMP_COS) {
    GemmArgs s = linear_args(g, b.lin_v, (int64_t)g.N * g.dp, ATp, b.dn + (int64_t)g.N * g.dp, n_cs);
    s.mdim = DIM_NC;
    launch_gemm_f32(s, GEMM_NT, g.nchunks, cs);
    return;
  }
  GemmArgs s = linear_args(g, b.dq, q_cs, ATp, b.dn + (int64_t)g.N * g.dp, n_cs);
  s.accumulate = 1;
  launch_gemm_f32(s, GEMM_NT, g.nchunks, cs);
  GemmArgs d = linear_args(g, b.dq + (int64_t)g.C * g.dp, q_cs, Ap, b.dn, n_cs);
  d.accumulate = 1;
  launch_gemm_f32(d, GEMM_NT, g.nchunks, cs);
}

// Gradient of the single relation matrix, one d x d partial per product and
// chunk into `partial`; returns the number of partials.  dot: dA = dQ^T X +
// Y^T dK over the chunk's edges; cos: dA = V^T X over its source candidates.
int run_linear_relation_grad(const StepGeom& g, const StepBufs& b, float* partial, hipStream_t cs) {
  const int d = g.d, dp = g.dp, C = g.C, N = g.N;
  GemmArgs la;
  memset(&la, 0, sizeof(la));
  la.lda = dp;
  la.ldb = dp;
  la.ldc = d;
  la.mdim = DIM_FIXED;
  la.Mfix = d;
  la.ndim = DIM_FIXED;
  la.Nfix = d;
  la.C = C;
  la.U = g.U;
  la.m_step = g.m_step;
  la.cstart = g.cstart;
  la.nsides = 1;
  la.Cm = partial;
  if (g.cmp == CMP_COS) {
    la.A = b.lin_v;                    // V^T: (m = row of A, k = candidate)
    la.B = b.lin_x;                    // raw source candidates x_t
    la.a_cs = (int64_t)N * dp;
    la.b_cs = (int64_t)N * dp;
    la.c_cs = (int64_t)d * d;
    la.kdim = DIM_NC;
    launch_gemm_f32(la, GEMM_TN, g.nchunks, cs);
    return g.nchunks;
  }
  la.A = b.dq;                         // dQ^T: (m = row of A, k = edge)
  la.B = b.nn + (int64_t)N * dp;       // source rows x_s (N1[e])
  la.a_cs = 2ll * C * dp;
  la.b_cs = 2ll * N * dp;
  la.c_cs = 2ll * d * d;
  la.kdim = DIM_CC;
  launch_gemm_f32(la, GEMM_TN, g.nchunks, cs);
  GemmArgs lb = la;
  lb.A = b.nn;                         // destination rows x_d (N0[e])
  lb.B = b.dq + (int64_t)C * dp;       // dK
  lb.Cm = partial + (int64_t)d * d;
  lb.a_cs = 2ll * N * dp;
  lb.b_cs = 2ll * C * dp;
  launch_gemm_f32(lb, GEMM_TN, g.nchunks, cs);
  return 2 * g.nchunks;
}

// The score contraction of a step again, with the plain store epilogue, into
// out [nchunks][2][C][C+U] (row pitch C+U): the same operands and main loop as
// the loss epilogue's launch, so the same float32 values.  The translation
// bias of the source side (translation with dot) is added afterwards, as the
// epilogues add it.
void run_score_store(pbg_ctx* ctx, const StepGeom& g, const StepBufs& b, float* out, hipStream_t cs) {
  GemmArgsH fa;
  if (ctx->flags & PBG_F_BF16_SCORE) {
    fa = score_args_bf16(ctx, g, b);
  } else {
    int epi = EPI_LOSS;
    fa = score_args_f32(g, b, &epi);
  }
  fa.Cm = out;
  fa.dsh = nullptr;
  fa.dsb = nullptr;
  fa.c_cs = 2ll * g.C * g.N;
  fa.c_ss = (int64_t)g.C * g.N;
  fa.ldc = g.N;
  if (ctx->flags & PBG_F_BF16_SCORE) launch_gemm_bf16(fa, EPI_STORE, g.nchunks * 2, cs);
  else launch_score_split(fa, EPI_STORE, g.nchunks * 2, cs);
  if (g.op == OP_TRANSLATION && g.cmp == CMP_DOT && !g.recip) launch_add_side_bias(g, b.bias, out, cs);
}
