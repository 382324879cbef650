// pbg_inspect_step: the forward half of one training step (Sec. 3.1 scores and
// losses, Sec. 4.3 batched negatives), run by the same launch sequence as
// pbg_train_bucket, with what it computed copied out and nothing updated.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>

#include "kernels.h"
#include "pbg.h"
#include "runtime_internal.h"

static int rup(int v, int m) { return (v + m - 1) / m * m; }

extern "C" pbg_status pbg_inspect_step(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src_local,
                                       const int32_t* rel, const int32_t* dst_local, int64_t n_edges,
                                       const pbg_neg_config* neg, uint64_t seed, float* scores, float* dscores,
                                       float* row_loss, float* pos, double* loss_host) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  ctx->err.clear();
  BucketTables tb;
  pbg_status st = PBG_OK;
  if (ctx->T > 1) {
    // entity types: the edges must form one run (one pair of tables)
    st = typed_single_run(ctx, i, j, src_local, rel, dst_local, n_edges, neg, &tb);
  } else {
    st = check_bucket_call(ctx, i, j, src_local, rel, dst_local, n_edges, neg);
    tb = partition_tables(ctx, i, j);
  }
  if (st != PBG_OK) return st;
  const int C = neg->chunk_size, U = neg->num_uniform, S = neg->chunks_per_step;
  if (loss_host) *loss_host = 0.0;
  if (n_edges == 0) return PBG_OK;
  const bool grouped = grouped_chunks(ctx, neg);
  if (grouped) {
    st = relation_chunk_bounds(ctx, rel, n_edges, C);
    if (st != PBG_OK) return st;
  }
  const int64_t nchunks = grouped ? (int64_t)ctx->cstart_host.size() - 1 : (n_edges + C - 1) / C;
  if (nchunks > S)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "pbg_inspect_step takes at most one step (%d chunks)", S);
  st = ensure_steploss(ctx, 1);
  if (st != PBG_OK) return st;
  st = ensure_lossparts(ctx, 1, nchunks * fin_blocks(C));
  if (st != PBG_OK) return st;

  hipStream_t cs = ctx->cs;
  StepGeom g;
  bucket_geom(ctx, i, j, tb, C, U, seed, g);
  StepBufs b = bucket_bufs(ctx, tb);
  const int nch = (int)nchunks;
  g.nchunks = nch;
  g.m_step = (int)n_edges;
  g.chunk0 = neg->first_chunk;
  g.cstart = grouped ? ctx->cstart_dev : nullptr;
  b.src = src_local;
  b.dst = dst_local;
  b.rel = rel;
  const int N = C + U;
  const size_t block = (size_t)nch * 2 * C * N;   // floats of a [nch][2][C][N] output
  hipError_t e = hipSuccess;
  if (row_loss) {
    e = hipMemsetAsync(row_loss, 0, (size_t)nch * 2 * C * 4, cs);
    b.rowloss = row_loss;
  }
  if (e == hipSuccess && scores) e = hipMemsetAsync(scores, 0, block * 4, cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipMemsetAsync");

  run_gather_forward(ctx, g, b, cs);
  const bool bf16 = (ctx->flags & PBG_F_BF16_SCORE) != 0;
  auto no_mark = [](int) {};
  if (bf16) run_contractions_bf16(ctx, g, b, 0, cs, no_mark, true);
  else run_contractions_f32(ctx, g, b, 0, cs, no_mark, true);

  if (scores) run_score_store(ctx, g, b, scores, cs);
  if (dscores) {
    const int Np = g.Np, Npb = rup(N, 32);
    const int nw = (Np + 15) / 16, ldw = rup(C, 8);
    if (ctx->loss == PBG_LOSS_RANKING)
      launch_expand_ds(g, DS_BITS, b.dsb, nw, ldw, nullptr, nullptr, nullptr, 0, dscores, cs);
    else if (bf16)
      launch_expand_ds(g, DS_BF16, nullptr, 0, 0, nullptr, nullptr, ctx->h.ds, Npb, dscores, cs);
    else if (ctx->loss == PBG_LOSS_SOFTMAX)
      launch_expand_ds(g, DS_F32_SCALED, nullptr, 0, 0, b.ds, b.rowscale, nullptr, Np, dscores, cs);
    else
      launch_expand_ds(g, DS_F32, nullptr, 0, 0, b.ds, nullptr, nullptr, Np, dscores, cs);
  }
  if (pos) launch_copy_pos(g, b.pos, pos, cs);
  launch_step_losses(ctx->lossparts, ctx->lossparts_pps, nch * fin_blocks(C), nch * fin_blocks(C), 1,
                     ctx->steploss_dev, cs);
  double loss = 0.0;
  e = hipGetLastError();
  if (e == hipSuccess) e = hipMemcpyAsync(&loss, ctx->steploss_dev, 8, hipMemcpyDeviceToHost, cs);
  if (e == hipSuccess) e = hipStreamSynchronize(cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "inspect_step");
  if (loss_host) *loss_host = loss;
  return PBG_OK;
}
