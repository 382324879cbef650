// pbg_rank_eval: filtered link-prediction ranks, MRR and Hits@10 (Sec. 5.4);
// pbg_rank_sampled: raw ranks against a caller-drawn candidate list (Sec. 5,
// Freebase evaluation: candidates sampled by prevalence).
//
// Sequence on the compute stream: range checks of every id (nothing is
// written on an error); the candidate tables (for a candidate list, its rows
// gathered in list order); the known triples sorted twice
// (by (s, r, d) for destination-side filtering, by (d, r, s) for source-side
// filtering) with three stable radix passes each; then, per side and block of
// queries, the queries, the score block S = Q . T^T on the matrix cores and
// the count kernel; finally the fp64 metric reduction.  Workspace is
// allocated for the call and released before it returns.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <vector>

#include "kernels.h"
#include "runtime_internal.h"

namespace {

struct CallBuf {
  std::vector<void*> ptrs;
  bool failed = false;
  void* get(size_t bytes) {
    void* p = nullptr;
    if (hipMalloc(&p, std::max<size_t>(bytes, 16)) != hipSuccess) {
      (void)hipGetLastError();
      failed = true;
      return nullptr;
    }
    ptrs.push_back(p);
    return p;
  }
  ~CallBuf() {
    for (void* p : ptrs) (void)hipFree(p);
  }
};

int bits_of(uint64_t max_value) {
  int b = 0;
  while (b < 32 && (max_value >> b) != 0) ++b;
  return b;
}

// stable lexicographic sort of the known triples by (first, second, third):
// least significant field first, carrying the permutation in vals
void sort_known(const int32_t* first, int first_bits, const int32_t* second, int second_bits,
                const int32_t* third, int third_bits, int64_t n, uint32_t* keys, uint32_t* vals,
                SortWork& w, int32_t* oa, int32_t* ob, int32_t* oc, hipStream_t s) {
  launch_perm_keys(third, nullptr, n, keys, vals, s);
  launch_radix_sort(keys, vals, (int)n, third_bits, w, s);
  if (second && second_bits > 0) {
    launch_perm_keys(second, vals, n, keys, nullptr, s);
    launch_radix_sort(keys, vals, (int)n, second_bits, w, s);
  }
  launch_perm_keys(first, vals, n, keys, nullptr, s);
  launch_radix_sort(keys, vals, (int)n, first_bits, w, s);
  launch_gather3(vals, first, second, third, n, oa, ob, oc, s);
}

// Ranks against all entities with the known triples filtered out (cand ==
// nullptr), or raw ranks against the n_cand entities cand[] (no filter).
pbg_status rank_impl(pbg_ctx* ctx, const char* name, const int32_t* src, const int32_t* rel, const int32_t* dst,
                     int64_t n, const int32_t* known_src, const int32_t* known_rel, const int32_t* known_dst,
                     int64_t n_known, const int32_t* cand, int64_t n_cand, int32_t* ranks, double* mrr_host,
                     double* hits10_host) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  ctx->err.clear();
  if (ctx->T > 1) return set_err(ctx, PBG_ERR_UNSUPPORTED, "%s takes one entity type", name);
  if (ctx->P != 1) return set_err(ctx, PBG_ERR_UNSUPPORTED, "%s needs a single partition", name);
  const bool recip = reciprocal(ctx);
  if (ctx->cmp == CMP_COS && ctx->op != OP_IDENTITY && ctx->R > 1 && !recip)
    return set_err(ctx, PBG_ERR_UNSUPPORTED,
                   "%s: cos with an operator needs a single relation (or reciprocal predicates)", name);
  if (n < 0 || n > 0x3FFFFFFFll || n_known < 0 || n_known > 0x7FFFFFFFll)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "n or n_known out of range");
  if (cand && (n_cand <= 0 || n_cand > 0x7FFFFFFFll))
    return set_err(ctx, PBG_ERR_INVALID_ARG, "n_cand out of range");
  const Partition& pt = ctx->parts[0];
  if (!pt.emb || pt.where != PBG_MEM_DEVICE)
    return set_err(ctx, PBG_ERR_STATE, "partition 0 must be bound in device memory");
  if (ctx->op != OP_IDENTITY && !ctx->relp) return set_err(ctx, PBG_ERR_STATE, "relation parameters are not bound");
  if (n > 0 && (!src || !dst || !ranks)) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL array");
  if (n_known > 0 && (!known_src || !known_dst)) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL known array");
  if (ctx->R > 1 && ((n > 0 && !rel) || (n_known > 0 && !known_rel)))
    return set_err(ctx, PBG_ERR_INVALID_ARG, "relation ids may be NULL only with one relation");
  if (n == 0) {
    if (mrr_host) *mrr_host = 0.0;
    if (hits10_host) *hits10_host = 0.0;
    return PBG_OK;
  }
  hipStream_t s = ctx->cs;
  const int64_t n_ent = ctx->n;
  const int64_t n_col = cand ? n_cand : n_ent;   // score columns
  const int d = ctx->d, dp = (d + 3) / 4 * 4;
  const bool linear = ctx->op == OP_LINEAR;
  // cos with an operator applies it to every source candidate, except with
  // reciprocal predicates (the source side's query carries theta_{r+R})
  const bool sep_src_table = ctx->cmp == CMP_COS && ctx->op != OP_IDENTITY && !recip;

  // query block: the score block stays near 1 GiB
  int64_t qb = ((int64_t)1 << 28) / std::max<int64_t>(n_col, 1);
  qb = std::max<int64_t>(128, qb / 128 * 128);
  qb = std::min<int64_t>(qb, (n + 127) / 128 * 128);

  CallBuf buf;
  uint32_t* flag = (uint32_t*)buf.get(16);
  float* T0 = (float*)buf.get((size_t)n_ent * dp * 4);
  float* T1 = sep_src_table ? (float*)buf.get((size_t)n_ent * dp * 4) : nullptr;
  float* relT = linear ? (float*)buf.get((size_t)relation_rows(ctx) * d * d * 4) : nullptr;
  float* pos = (float*)buf.get((size_t)n * 4);
  float* bias = (float*)buf.get((size_t)qb * 4);
  float* Q = (float*)buf.get((size_t)qb * dp * 4);
  float* S = (float*)buf.get((size_t)qb * n_col * 4);
  float* C0 = cand ? (float*)buf.get((size_t)n_cand * dp * 4) : nullptr;
  float* C1 = cand && sep_src_table ? (float*)buf.get((size_t)n_cand * dp * 4) : nullptr;
  double* metrics = (double*)buf.get(16);
  int32_t* kx[6] = {nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  uint32_t *keys = nullptr, *vals = nullptr;
  SortWork w;
  memset(&w, 0, sizeof(w));
  if (n_known > 0) {
    for (auto& p : kx) p = (int32_t*)buf.get((size_t)n_known * 4);
    keys = (uint32_t*)buf.get((size_t)n_known * 4);
    vals = (uint32_t*)buf.get((size_t)n_known * 4);
    w.keys_alt = (uint32_t*)buf.get((size_t)n_known * 4);
    w.vals_alt = (uint32_t*)buf.get((size_t)n_known * 4);
    w.hist = (uint32_t*)buf.get((size_t)radix_hist_entries(n_known) * 4);
    w.scan_tmp = (uint32_t*)buf.get((size_t)radix_scan_tmp_entries(n_known) * 4);
    w.max_n = (int)n_known;
  }
  if (buf.failed) return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "rank-eval workspace could not be allocated");

  hipError_t e = hipMemsetAsync(flag, 0, 4, s);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipMemsetAsync");
  launch_check_ids(src, n, (int32_t)n_ent, flag, 1u, s);
  launch_check_ids(dst, n, (int32_t)n_ent, flag, 1u, s);
  if (rel) launch_check_ids(rel, n, ctx->R, flag, 2u, s);
  launch_check_ids(known_src, n_known, (int32_t)n_ent, flag, 4u, s);
  launch_check_ids(known_dst, n_known, (int32_t)n_ent, flag, 4u, s);
  if (known_rel) launch_check_ids(known_rel, n_known, ctx->R, flag, 8u, s);
  if (cand) launch_check_ids(cand, n_cand, (int32_t)n_ent, flag, 16u, s);
  uint32_t hflag = 0;
  e = hipMemcpyAsync(&hflag, flag, 4, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(ctx, e, "id range check");
  if (hflag) return set_err(ctx, PBG_ERR_INVALID_ARG, "an id is out of range (flags %u: 1 eval entity, 2 eval "
                            "relation, 4 known entity, 8 known relation, 16 candidate)", hflag);

  StepGeom g;
  memset(&g, 0, sizeof(g));
  g.d = d;
  g.dp = dp;
  g.dr = ctx->dr;
  g.op = ctx->op;
  g.cmp = ctx->cmp;
  g.recip = recip ? 1 : 0;
  g.R = ctx->R;
  if (linear) launch_transpose_rel(ctx->relp, relT, relation_rows(ctx), d, s);
  launch_rank_tables(g, pt.emb, ctx->relp, relT, n_ent, T0, T1, s);
  if (cand) {
    // the candidates' rows of the tables, in candidate order
    launch_gather_rows(T0, cand, n_cand, dp, C0, s);
    if (T1) launch_gather_rows(T1, cand, n_cand, dp, C1, s);
  }

  const int ebits = bits_of((uint64_t)n_ent - 1), rbits = bits_of((uint64_t)ctx->R - 1);
  if (n_known > 0) {
    // destination side: groups (s, r), candidates d; source side: groups (d, r), candidates s
    sort_known(known_src, ebits, known_rel, rbits, known_dst, ebits, n_known, keys, vals, w, kx[0], kx[1],
               kx[2], s);
    sort_known(known_dst, ebits, known_rel, rbits, known_src, ebits, n_known, keys, vals, w, kx[3], kx[4],
               kx[5], s);
  }

  for (int side = 0; side < 2; ++side) {
    const float* T = cand ? (side == 1 && C1 ? C1 : C0) : (side == 1 && T1 ? T1 : T0);
    for (int64_t e0 = 0; e0 < n; e0 += qb) {
      const int rows = (int)std::min<int64_t>(qb, n - e0);
      launch_rank_queries(g, pt.emb, ctx->relp, relT, src, rel, dst, e0, rows, side, Q, pos, bias, s);
      // candidate scores S = Q . T^T, float32 operands as exact bf16 pieces
      GemmArgsH a;
      memset(&a, 0, sizeof(a));
      a.Af = Q;
      a.Bf = T;
      a.Cm = S;
      a.lda = dp;
      a.ldb = dp;
      a.ldc = (int)n_col;
      a.mdim = DIM_FIXED;
      a.Mfix = rows;
      a.ndim = DIM_FIXED;
      a.Nfix = (int)n_col;
      a.kdim = DIM_FIXED;
      a.Kfix = dp;
      a.C = 1;
      a.nsides = 1;
      launch_score_split(a, EPI_STORE, 1, s);
      launch_rank_count(S, n_col, n_col, cand, e0, rows, side, n, src, rel, dst, pos, bias,
                        side == 0 ? kx[0] : kx[3], side == 0 ? kx[1] : kx[4], side == 0 ? kx[2] : kx[5],
                        n_known, ranks, s);
    }
  }
  launch_rank_metrics(ranks, 2 * n, metrics, s);
  double hm[2] = {0.0, 0.0};
  e = hipGetLastError();
  if (e == hipSuccess) e = hipMemcpyAsync(hm, metrics, 16, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(ctx, e, name);
  if (mrr_host) *mrr_host = hm[0];
  if (hits10_host) *hits10_host = hm[1];
  return PBG_OK;
}

}  // namespace

extern "C" pbg_status pbg_rank_eval(pbg_ctx* ctx, const int32_t* src, const int32_t* rel, const int32_t* dst,
                                    int64_t n, const int32_t* known_src, const int32_t* known_rel,
                                    const int32_t* known_dst, int64_t n_known, int32_t* ranks,
                                    double* mrr_host, double* hits10_host) {
  return rank_impl(ctx, "pbg_rank_eval", src, rel, dst, n, known_src, known_rel, known_dst, n_known, nullptr, 0,
                   ranks, mrr_host, hits10_host);
}

extern "C" pbg_status pbg_rank_sampled(pbg_ctx* ctx, const int32_t* src, const int32_t* rel, const int32_t* dst,
                                       int64_t n, const int32_t* cand, int64_t n_cand, int32_t* ranks,
                                       double* mrr_host, double* hits10_host) {
  if (ctx && !cand && n > 0) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL candidate array");
  return rank_impl(ctx, "pbg_rank_sampled", src, rel, dst, n, nullptr, nullptr, nullptr, 0, cand, n_cand, ranks,
                   mrr_host, hits10_host);
}
