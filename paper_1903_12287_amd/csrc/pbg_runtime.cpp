// Host runtime behind the C ABI of include/pbg.h: context, argument checks,
// workspace, and the launch sequence of one training step.
//
// A step (chunks_per_step chunks of a bucket) is, on the compute stream:
//   gather + operator + uniform draws  ->  score contraction with the loss
//   epilogue (softmax: + row pass)  ->  per-edge finalisation (dL/dp, loss)
//   ->  dQ = dS.N and dN = dS^T.Q  ->  operator backward into per-row
//   contributions  ->  stable sort of the contributions by row  ->  segment
//   sums + row-wise Adagrad  ->  relation sums + element-wise Adagrad.
// No host synchronisation happens inside the step loop.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "kernels.h"
#include "pbg.h"
#include "runtime_internal.h"

static const char* kNullCtxError = "pbg: NULL context";

pbg_status set_err(pbg_ctx* ctx, pbg_status st, const char* fmt, ...) {
  if (!ctx) return st;
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  ctx->err = buf;
  return st;
}

pbg_status hip_fail(pbg_ctx* ctx, hipError_t e, const char* what) {
  return set_err(ctx, PBG_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

void* Arena::get(size_t bytes) {
  if (bytes == 0) bytes = 16;
  bytes = (bytes + 255) & ~(size_t)255;
  void* p = nullptr;
  if (hipMalloc(&p, bytes) != hipSuccess) {
    (void)hipGetLastError();
    failed = true;
    return nullptr;
  }
  ptrs.push_back(p);
  return p;
}

void Arena::release() {
  for (void* p : ptrs) (void)hipFree(p);
  ptrs.clear();
  failed = false;
}

static int bits_for(uint64_t v) {  // bits needed for values in [0, v]
  int b = 0;
  while (b < 64 && (v >> b) != 0) ++b;
  return b;
}

static int round_up(int v, int m) { return (v + m - 1) / m * m; }

bool alloc_sortwork(Arena& a, SortWork& w, int64_t max_n, int width) {
  w.max_n = (int)max_n;
  w.keys_alt = (uint32_t*)a.get(max_n * 4);
  w.vals_alt = (uint32_t*)a.get(max_n * 4);
  w.hist = (uint32_t*)a.get(radix_hist_entries(max_n) * 4);
  w.scan_tmp = (uint32_t*)a.get(radix_scan_tmp_entries(max_n) * 4);
  w.partial = width > 0 ? (float*)a.get(max_n * (int64_t)width * 4) : nullptr;
  w.segflag = (uint32_t*)a.get((max_n / SEG_BLOCK + 2) * 4);
  return !a.failed;
}

pbg_status ensure_workspace(pbg_ctx* ctx, int C, int U, int S) {
  if (ctx->ws_ready && ctx->wC == C && ctx->wU == U && ctx->wS == S) return PBG_OK;
  (void)hipStreamSynchronize(ctx->cs);
  ctx->ws.release();
  ctx->ws_ready = false;
  Arena& a = ctx->ws;
  const int N = C + U;
  const int d = ctx->d, dp = round_up(d, 4), Np = round_up(N, 4);
  const int nct = (Np + PBG_SCORE_BN - 1) / PBG_SCORE_BN;
  const int64_t s = S;
  StepBufs& b = ctx->bufs;
  memset(&b, 0, sizeof(b));
  b.qk = (float*)a.get(s * 2 * C * dp * 4);
  b.nn = (float*)a.get(s * 2 * N * dp * 4);
  b.nrm = (float*)a.get(s * 2 * N * 4);
  const int64_t psides = reciprocal(ctx) ? 2 : 1;   // positive scores per edge
  b.pos = (float*)a.get(s * psides * C * 4);
  b.bias = (float*)a.get(s * C * 4);
  b.neg = (int32_t*)a.get(s * 2 * std::max(U, 1) * 4);
  // the ranking loss keeps dS as bits (word-column major, row pitch C rounded
  // up to 8); dS as floats serves the other losses (raw scores for softmax)
  const bool ranking = ctx->loss == PBG_LOSS_RANKING;
  b.ds = ranking ? nullptr : (float*)a.get(s * 2 * C * (int64_t)Np * 4);
  b.dsb = ranking ? (uint16_t*)a.get(s * 2 * (int64_t)round_up(C, 8) * ((Np + 15) / 16) * 2) : nullptr;
  b.rowpart = (float*)a.get(s * 2 * C * nct * 2 * 4);
  if (ctx->loss == PBG_LOSS_SOFTMAX) b.rowscale = (float*)a.get(s * 2 * nct * (int64_t)C * 4);
  b.dpos = (float*)a.get(s * psides * C * 4);
  b.dsum1 = (float*)a.get(s * C * 4);
  b.dq = (float*)a.get(s * 2 * C * dp * 4);
  b.dn = (float*)a.get(s * 2 * N * dp * 4);
  const bool has_rel = ctx->op != OP_IDENTITY;
  const bool linear = ctx->op == OP_LINEAR;
  // rows per chunk: contributions, or with one relation the operator
  // backward's per-block sums
  const int relN = reciprocal(ctx) ? 2 * C : (single_relation_sums(ctx) ? op_backward_blocks(C, U, ctx->cmp) : N);
  if (has_rel && !linear) b.relc = (float*)a.get(s * relN * ctx->dr * 4);
  if (reciprocal(ctx) && ctx->cmp == PBG_CMP_COS) b.qnrm = (float*)a.get(s * 2 * C * 4);
  const int64_t nkeys = s * 2 * N;
  // a window of steps: keys, values, the sort's alternate buffers and counts
  b.keys = (uint32_t*)a.get(kSortWindow * nkeys * 4);
  b.vals = (uint32_t*)a.get(kSortWindow * nkeys * 4);
  ctx->wkeys_alt = (uint32_t*)a.get(kSortWindow * nkeys * 4);
  ctx->wvals_alt = (uint32_t*)a.get(kSortWindow * nkeys * 4);
  ctx->whist = (uint32_t*)a.get(radix_segments_hist_entries(nkeys, kSortWindow) * 4);
  if (sorted_relation_keys(ctx)) {
    // the edges' relations, then (cos with an operator) the chunk relation of
    // every uniform source candidate or (reciprocal predicates) every edge's
    // source-side row
    const int64_t per = s * (reciprocal(ctx) ? 2 * C : C + (chunk_relation_operator(ctx) ? U : 0));
    b.rkeys = (uint32_t*)a.get(kSortWindow * per * 4);
    b.rvals = (uint32_t*)a.get(kSortWindow * per * 4);
  }
  const int width = std::max(d, has_rel && !linear ? ctx->dr : 0);
  if (!alloc_sortwork(a, ctx->sw, std::max<int64_t>(nkeys, s * C), width)) {
    ctx->ws.release();
    return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "workspace allocation failed (C=%d U=%d S=%d)", C, U, S);
  }
  if (has_rel) {
    const int64_t w = linear ? 2 * s * (int64_t)d * d : s * RELSUM_PIECES * (int64_t)ctx->dr;
    ctx->relpartial = (float*)a.get(w * 4);
  }
  if (linear) {
    ctx->relA = (float*)a.get((int64_t)d * dp * 4);
    ctx->relAT = (float*)a.get((int64_t)d * dp * 4);
    if (ctx->cmp == PBG_CMP_COS) {
      b.lin_x = (float*)a.get(s * std::max(N, 2 * C) * dp * 4);
      b.lin_v = (float*)a.get(s * N * dp * 4);
    }
  }
  ctx->flag_dev = (uint32_t*)a.get(16);
  ctx->h = BufsH();
  if (ctx->flags & PBG_F_BF16_SCORE) {
    const int dpb = round_up(d, 32), Cpb = round_up(C, 32), Npb = round_up(N, 32);
    ctx->h.qk = (uint16_t*)a.get(s * 2 * C * dpb * 2);
    ctx->h.nn = (uint16_t*)a.get(s * 2 * N * dpb * 2);
    ctx->h.qkT = (uint16_t*)a.get(s * 2 * dpb * Cpb * 2);
    ctx->h.nnT = (uint16_t*)a.get(s * 2 * dpb * Npb * 2);
    if (!ranking) ctx->h.ds = (uint16_t*)a.get(s * 2 * C * (int64_t)Npb * 2);
  } else {
    // float32 backward on the bf16 instructions: transposed pieces of Q and N
    const int dpb = round_up(d, 32), Cpb = round_up(C, 32), Npb = round_up(N, 32);
    ctx->h.q3_ps = s * 2 * dpb * (int64_t)Cpb;
    ctx->h.n3_ps = s * 2 * dpb * (int64_t)Npb;
    ctx->h.qkT3 = (uint16_t*)a.get(3 * ctx->h.q3_ps * 2);
    ctx->h.nnT3 = (uint16_t*)a.get(3 * ctx->h.n3_ps * 2);
  }
  if (a.failed) {
    ctx->ws.release();
    return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "workspace allocation failed (C=%d U=%d S=%d)", C, U, S);
  }
  // rows of a short last chunk beyond its edges are never scored, but the
  // bf16 transposes copy them: start from zeros so they always hold finite values
  hipError_t ez = hipMemsetAsync(b.qk, 0, (size_t)s * 2 * C * dp * 4, ctx->cs);
  if (ez == hipSuccess) ez = hipMemsetAsync(b.nn, 0, (size_t)s * 2 * N * dp * 4, ctx->cs);
  if (ez == hipSuccess) ez = hipStreamSynchronize(ctx->cs);
  if (ez != hipSuccess) {
    ctx->ws.release();
    return hip_fail(ctx, ez, "workspace initialisation");
  }
  ctx->wC = C;
  ctx->wU = U;
  ctx->wS = S;
  ctx->ws_ready = true;
  return PBG_OK;
}

static bool ensure_events(pbg_ctx* ctx, size_t n) {
  while (ctx->events.size() < n) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) {
      (void)hipGetLastError();
      return false;
    }
    ctx->events.push_back(e);
  }
  return true;
}

pbg_status ensure_lossparts(pbg_ctx* ctx, int64_t nsteps, int64_t pps) {
  const int64_t n = std::max<int64_t>(nsteps, 1) * std::max<int64_t>(pps, 1);
  ctx->lossparts_pps = pps;
  if (ctx->lossparts_cap >= n && ctx->lossparts) return PBG_OK;
  if (ctx->lossparts) (void)hipFree(ctx->lossparts);
  ctx->lossparts = nullptr;
  ctx->lossparts_cap = 0;
  if (hipMalloc(&ctx->lossparts, (size_t)n * 8) != hipSuccess) {
    (void)hipGetLastError();
    ctx->lossparts = nullptr;
    return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "loss-partial buffer allocation failed");
  }
  ctx->lossparts_cap = n;
  return PBG_OK;
}

pbg_status ensure_steploss(pbg_ctx* ctx, int64_t nsteps) {
  if (ctx->steploss_cap >= nsteps && ctx->steploss_dev) return PBG_OK;
  if (ctx->steploss_dev) (void)hipFree(ctx->steploss_dev);
  ctx->steploss_dev = nullptr;
  ctx->steploss_cap = 0;
  // one double per step, then the 64-bit count of touched rows
  if (hipMalloc(&ctx->steploss_dev, (size_t)(std::max<int64_t>(nsteps, 1) + 1) * 8) != hipSuccess) {
    (void)hipGetLastError();
    ctx->steploss_dev = nullptr;
    return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "step-loss buffer allocation failed");
  }
  ctx->steploss_cap = nsteps;
  return PBG_OK;
}

pbg_status relation_chunk_bounds(pbg_ctx* ctx, const int32_t* rel, int64_t n, int C) {
  std::vector<int32_t> r((size_t)n);
  hipError_t e = hipMemcpyAsync(r.data(), rel, (size_t)n * 4, hipMemcpyDeviceToHost, ctx->cs);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "relation copy");
  std::vector<int32_t>& cs = ctx->cstart_host;
  cs.clear();
  ctx->crel_host.clear();
  int64_t run0 = 0;
  for (int64_t k = 0; k <= n; ++k) {
    if (k < n && k > 0 && r[k] < r[k - 1])
      return set_err(ctx, PBG_ERR_INVALID_ARG,
                     "relation-grouped chunks need the edges sorted by relation (edge %lld)", (long long)k);
    if (k == n || (k > 0 && r[k] != r[k - 1])) {
      for (int64_t c = run0; c < k; c += C) {
        cs.push_back((int32_t)c);
        ctx->crel_host.push_back(r[run0]);
      }
      run0 = k;
    }
  }
  cs.push_back((int32_t)n);
  const int64_t need = (int64_t)cs.size();
  if (ctx->cstart_cap < need) {
    if (ctx->cstart_dev) (void)hipFree(ctx->cstart_dev);
    ctx->cstart_dev = nullptr;
    ctx->cstart_cap = 0;
    if (hipMalloc(&ctx->cstart_dev, (size_t)need * 4) != hipSuccess) {
      (void)hipGetLastError();
      ctx->cstart_dev = nullptr;
      return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "chunk bound allocation failed");
    }
    ctx->cstart_cap = need;
  }
  e = hipMemcpyAsync(ctx->cstart_dev, cs.data(), (size_t)need * 4, hipMemcpyHostToDevice, ctx->cs);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "chunk bound copy");
  return PBG_OK;
}

// --------------------------------------------------------------------------
// C ABI
// --------------------------------------------------------------------------
extern "C" {

pbg_status pbg_bucket_init(pbg_ctx** out, int64_t num_entities, int32_t num_partitions,
                           int32_t num_relations, int32_t dim, int32_t op, int32_t cmp, int32_t loss,
                           float margin, uint32_t flags) {
  if (!out) return PBG_ERR_INVALID_ARG;
  *out = nullptr;
  pbg_ctx* ctx = new (std::nothrow) pbg_ctx();
  if (!ctx) return PBG_ERR_OUT_OF_MEMORY;
  auto fail = [&](pbg_status st, const char* msg) {
    // keep the context so the caller can read the message, then report
    ctx->err = msg;
    ctx->invalid = true;
    *out = ctx;
    return st;
  };
  if (num_entities < 1 || num_partitions < 1 || num_relations < 1)
    return fail(PBG_ERR_INVALID_ARG, "num_entities, num_partitions and num_relations must be >= 1");
  if (dim < 1 || dim > 512) return fail(PBG_ERR_INVALID_ARG, "dim must be in [1, 512]");
  if (op < PBG_OP_IDENTITY || op > PBG_OP_COMPLEX_DIAGONAL) return fail(PBG_ERR_INVALID_ARG, "unknown operator");
  if (cmp < PBG_CMP_DOT || cmp > PBG_CMP_COS) return fail(PBG_ERR_INVALID_ARG, "unknown comparator");
  if (loss < PBG_LOSS_RANKING || loss > PBG_LOSS_SOFTMAX) return fail(PBG_ERR_INVALID_ARG, "unknown loss");
  if (op == PBG_OP_COMPLEX_DIAGONAL && (dim % 2)) return fail(PBG_ERR_INVALID_ARG, "complex_diagonal needs an even dim");
  if (!std::isfinite(margin)) return fail(PBG_ERR_INVALID_ARG, "margin must be finite");
  if (flags & ~(uint32_t)(PBG_F_BF16_SCORE | PBG_F_PHASE_TIMING | PBG_F_SCORE_TIMING | PBG_F_RECIPROCAL))
    return fail(PBG_ERR_INVALID_ARG, "unknown flags");
  const int64_t ps = (num_entities + num_partitions - 1) / num_partitions;
  if ((int64_t)(num_partitions - 1) * ps >= num_entities)
    return fail(PBG_ERR_INVALID_ARG, "a partition would be empty (num_partitions too large for num_entities)");
  if (ps > (1ll << 30)) return fail(PBG_ERR_INVALID_ARG, "partitions above 2^30 rows are not supported");
  if (cmp == PBG_CMP_COS && op == PBG_OP_LINEAR && num_relations > 1 && !(flags & PBG_F_RECIPROCAL))
    return fail(PBG_ERR_UNSUPPORTED,
                "cos with the linear operator needs a single relation (or reciprocal predicates)");
  ctx->n = num_entities;
  ctx->P = num_partitions;
  ctx->R = num_relations;
  ctx->d = dim;
  ctx->op = op;
  ctx->cmp = cmp;
  ctx->loss = loss;
  ctx->margin = margin;
  ctx->flags = flags;
  ctx->ps = ps;
  ctx->dr = op == PBG_OP_IDENTITY ? 0 : (op == PBG_OP_LINEAR ? dim * dim : dim);
  ctx->parts.assign(num_partitions, Partition());
  ctx->T = 1;
  ctx->type_n.assign(1, num_entities);
  ctx->type_part.assign(1, 1);
  ctx->rel_st.assign(num_relations, 0);
  ctx->rel_dt.assign(num_relations, 0);
  if (hipGetDevice(&ctx->device) != hipSuccess) {
    (void)hipGetLastError();
    return fail(PBG_ERR_DEVICE, "no HIP device");
  }
  if (noalloc_scratch_init(ctx) != PBG_OK) {
    ctx->invalid = true;
    *out = ctx;
    return PBG_ERR_DEVICE;
  }
  *out = ctx;
  return PBG_OK;
}

void pbg_free(pbg_ctx* ctx) {
  if (!ctx) return;
  (void)hipDeviceSynchronize();
  ctx->ws.release();
  if (ctx->steploss_dev) (void)hipFree(ctx->steploss_dev);
  if (ctx->lossparts) (void)hipFree(ctx->lossparts);
  if (ctx->cstart_dev) (void)hipFree(ctx->cstart_dev);
  if (ctx->cweight_dev) (void)hipFree(ctx->cweight_dev);
  for (auto& s : ctx->slots) {
    if (s.emb) (void)hipFree(s.emb);
    if (s.ready) (void)hipEventDestroy(s.ready);
    if (s.released) (void)hipEventDestroy(s.released);
  }
  if (ctx->own_xs) (void)hipStreamDestroy(ctx->own_xs);
  if (ctx->hflag) (void)hipHostFree(ctx->hflag);
  if (ctx->check_ev) (void)hipEventDestroy(ctx->check_ev);
  for (hipEvent_t e : ctx->events) (void)hipEventDestroy(e);
  delete ctx;
}

const char* pbg_last_error(const pbg_ctx* ctx) {
  if (!ctx) return kNullCtxError;
  return ctx->err.c_str();
}

int64_t pbg_partition_rows(const pbg_ctx* ctx, int32_t p) { return table_rows(ctx, 0, p); }

int64_t pbg_relation_param_floats(const pbg_ctx* ctx) {
  if (!ctx || ctx->invalid) return -1;
  return (int64_t)relation_rows(ctx) * ctx->dr;
}

pbg_status pbg_bind_partition(pbg_ctx* ctx, int32_t p, float* emb, float* adagrad, int32_t where) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  if (p < 0 || p >= ctx->P) return set_err(ctx, PBG_ERR_INVALID_ARG, "partition %d out of range", p);
  if (!emb || !adagrad) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL embedding or accumulator");
  if (where != PBG_MEM_DEVICE && where != PBG_MEM_PINNED_HOST)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "unknown memory kind %d", where);
  ctx->parts[p].emb = emb;
  ctx->parts[p].G = adagrad;
  ctx->parts[p].where = where;
  ctx->err.clear();
  return PBG_OK;
}

pbg_status pbg_bind_relations(pbg_ctx* ctx, float* params, float* adagrad) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  if (ctx->op == PBG_OP_IDENTITY) return PBG_OK;
  if (!params || !adagrad) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL relation parameters or accumulator");
  ctx->relp = params;
  ctx->relG = adagrad;
  ctx->err.clear();
  return PBG_OK;
}

pbg_status pbg_set_streams(pbg_ctx* ctx, void* compute_stream, void* copy_stream) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  ctx->cs = (hipStream_t)compute_stream;
  ctx->xs = (hipStream_t)copy_stream;
  return PBG_OK;
}

pbg_status pbg_get_stats(const pbg_ctx* ctx, pbg_stats* out_host) {
  if (!ctx || !out_host) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return PBG_ERR_STATE;
  *out_host = ctx->stats;
  return PBG_OK;
}

pbg_status pbg_get_step_losses(const pbg_ctx* ctx, double* out_host, int64_t capacity,
                               int64_t* n_steps_host) {
  if (!ctx || (capacity > 0 && !out_host)) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return PBG_ERR_STATE;
  const int64_t n = (int64_t)ctx->step_losses.size();
  for (int64_t k = 0; k < std::min(capacity, n); ++k) out_host[k] = ctx->step_losses[k];
  if (n_steps_host) *n_steps_host = n;
  return PBG_OK;
}

}  // extern "C"

// --------------------------------------------------------------------------
// training
// --------------------------------------------------------------------------
pbg_status check_neg_config(pbg_ctx* ctx, const pbg_neg_config* neg) {
  if (!neg) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL negative config");
  if (neg->chunk_size < 1 || neg->chunk_size > (1 << 16))
    return set_err(ctx, PBG_ERR_INVALID_ARG, "chunk_size must be in [1, 65536]");
  if (neg->num_uniform < 0 || neg->num_uniform > (1 << 16))
    return set_err(ctx, PBG_ERR_INVALID_ARG, "num_uniform must be in [0, 65536]");
  if (neg->chunk_size + neg->num_uniform < 2)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "chunk_size + num_uniform must be >= 2");
  if (neg->chunks_per_step < 1 || neg->chunks_per_step > 4096)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "chunks_per_step must be in [1, 4096]");
  if (neg->chunking != PBG_CHUNK_CONSECUTIVE && neg->chunking != PBG_CHUNK_BY_RELATION)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "unknown chunking %d", neg->chunking);
  if (neg->first_chunk < 0 || neg->first_chunk > 0xFFFFFFFFll)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "first_chunk out of range");
  const int64_t keys = (int64_t)neg->chunks_per_step * 2 * (neg->chunk_size + neg->num_uniform);
  if (keys > (1ll << 28)) return set_err(ctx, PBG_ERR_INVALID_ARG, "step too large");
  return PBG_OK;
}

int64_t table_rows(const pbg_ctx* ctx, int t, int p) {
  if (!ctx || ctx->invalid || t < 0 || t >= ctx->T) return -1;
  const int parts = ctx->type_part[(size_t)t] ? ctx->P : 1;
  if (p < 0 || p >= parts) return -1;
  const int64_t n = ctx->type_n[(size_t)t];
  const int64_t ps = (n + parts - 1) / parts;
  return std::min<int64_t>(ps, n - (int64_t)p * ps);
}

BucketTables partition_tables(pbg_ctx* ctx, int32_t i, int32_t j) {
  BucketTables tb;
  tb.emb_i = ctx->parts[i].emb;
  tb.G_i = ctx->parts[i].G;
  tb.emb_j = ctx->parts[j].emb;
  tb.G_j = ctx->parts[j].G;
  tb.rows_i = pbg_partition_rows(ctx, i);
  tb.rows_j = pbg_partition_rows(ctx, j);
  tb.same = i == j;
  return tb;
}

void bucket_geom(const pbg_ctx* ctx, int32_t i, int32_t j, const BucketTables& tb, int C, int U, uint64_t seed,
                 StepGeom& g) {
  const int N = C + U;
  const int d = ctx->d, dp = round_up(d, 4), Np = round_up(N, 4);
  const int64_t rows_i = tb.rows_i, rows_j = tb.rows_j;
  memset(&g, 0, sizeof(g));
  g.C = C;
  g.U = U;
  g.N = N;
  g.d = d;
  g.dp = dp;
  g.Np = Np;
  g.dr = ctx->dr;
  g.nct = (Np + PBG_SCORE_BN - 1) / PBG_SCORE_BN;
  g.op = ctx->op;
  g.cmp = ctx->cmp;
  g.loss = ctx->loss;
  g.margin = ctx->margin;
  g.same_table = tb.same ? 1 : 0;
  g.rows_i = (int)rows_i;
  g.rows_j = (int)rows_j;
  g.rb = bits_for((uint64_t)std::max(rows_i, rows_j) - 1);
  if (g.rb < 1) g.rb = 1;
  g.bucket = (uint32_t)(i * ctx->P + j);
  g.seed = seed;
  g.recip = reciprocal(ctx) ? 1 : 0;
  g.R = ctx->R;
  g.relN = g.recip ? 2 * C : N;
  g.relsum = single_relation_sums(ctx) ? 1 : 0;
  g.dq_has_dn = merged_ranking_backward(ctx, g) ? 1 : 0;
}

StepBufs bucket_bufs(pbg_ctx* ctx, const BucketTables& tb) {
  StepBufs b = ctx->bufs;
  b.nuniq = (unsigned long long*)(ctx->steploss_dev + std::max<int64_t>(ctx->steploss_cap, 1));
  b.emb_i = tb.emb_i;
  b.emb_j = tb.emb_j;
  b.G_i = tb.G_i;
  b.G_j = tb.G_j;
  b.relp = ctx->relp;
  b.relG = ctx->relG;
  if (!sorted_relation_keys(ctx)) {
    b.rkeys = nullptr;
    b.rvals = nullptr;
  }
  return b;
}

void run_gather_forward(pbg_ctx* ctx, const StepGeom& g, const StepBufs& b, hipStream_t cs) {
  const bool linear1 = linear_step_contractions(ctx);
  if (linear1) launch_pad_linear(ctx->relp, g.d, g.dp, ctx->relA, ctx->relAT, cs);
  launch_gather(g, b, cs);
  if (linear1) run_linear_forward(g, b, ctx->relA, ctx->relAT, cs);
  else if (ctx->op == OP_LINEAR) launch_linear_rows(g, b, cs);
}

// Runs the step loop on already-validated, device-resident partitions.
pbg_status chunk_weights(pbg_ctx* ctx, bool grouped, int64_t nchunks, const float** out) {
  *out = nullptr;
  if (ctx->relw.empty() || nchunks <= 0) return PBG_OK;
  std::vector<float> w((size_t)nchunks);
  if (grouped) {
    for (int64_t c = 0; c < nchunks; ++c) w[(size_t)c] = ctx->relw[(size_t)ctx->crel_host[(size_t)c]];
  } else {
    // consecutive chunks may mix relations: one weight for all of them
    for (float v : ctx->relw)
      if (v != ctx->relw[0])
        return set_err(ctx, PBG_ERR_UNSUPPORTED,
                       "relation weights that differ need relation-grouped chunks (PBG_CHUNK_BY_RELATION)");
    std::fill(w.begin(), w.end(), ctx->relw[0]);
  }
  if (ctx->cweight_cap < nchunks) {
    if (ctx->cweight_dev) (void)hipFree(ctx->cweight_dev);
    ctx->cweight_dev = nullptr;
    ctx->cweight_cap = 0;
    if (hipMalloc(&ctx->cweight_dev, (size_t)nchunks * 4) != hipSuccess) {
      (void)hipGetLastError();
      ctx->cweight_dev = nullptr;
      return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "chunk weight allocation failed");
    }
    ctx->cweight_cap = nchunks;
  }
  hipError_t e = hipMemcpyAsync(ctx->cweight_dev, w.data(), (size_t)nchunks * 4, hipMemcpyHostToDevice, ctx->cs);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "chunk weight copy");
  *out = ctx->cweight_dev;
  return PBG_OK;
}

pbg_status train_bucket_device(pbg_ctx* ctx, int32_t i, int32_t j, const BucketTables& tb, const int32_t* src,
                               const int32_t* rel, const int32_t* dst, int64_t n_edges, const pbg_neg_config* neg,
                               float lr, uint64_t seed, double* loss_out, std::vector<double>* step_losses) {
  const int C = neg->chunk_size, U = neg->num_uniform, S = neg->chunks_per_step;
  pbg_status st = ensure_workspace(ctx, C, U, S);
  if (st != PBG_OK) return st;
  // relation-grouped chunks: bounds in the call's edge arrays (checked before
  // anything is updated)
  const bool grouped = grouped_chunks(ctx, neg);
  if (ctx->check_pending && (grouped || !ctx->relw.empty())) {
    // the host reads relation ids below: their range is checked first
    st = finish_id_check(ctx, i, j);
    if (st != PBG_OK) return st;
  }
  if (grouped) {
    st = relation_chunk_bounds(ctx, rel, n_edges, C);
    if (st != PBG_OK) return st;
  }
  const std::vector<int32_t>& cbound = ctx->cstart_host;
  const int64_t nchunks = grouped ? (int64_t)cbound.size() - 1 : (n_edges + C - 1) / C;
  const float* cweight = nullptr;
  st = chunk_weights(ctx, grouped, nchunks, &cweight);
  if (st != PBG_OK) return st;
  // first edge of chunk c (c <= nchunks)
  auto chunk_at = [&](int64_t c) -> int64_t {
    return grouped ? (int64_t)cbound[(size_t)c] : std::min<int64_t>(n_edges, c * C);
  };
  const int64_t nsteps = (nchunks + S - 1) / S;
  const bool uniform_rel = chunk_relation_operator(ctx);
  const bool recip = reciprocal(ctx);
  // relation keys per step
  const int64_t rstride = (int64_t)S * (recip ? 2 * C : C + (uniform_rel ? U : 0));
  st = ensure_steploss(ctx, nsteps);
  if (st != PBG_OK) return st;
  const int64_t fb = fin_blocks(C);
  st = ensure_lossparts(ctx, nsteps, (int64_t)S * fb);
  if (st != PBG_OK) return st;
  hipStream_t cs = ctx->cs;
  const int N = C + U;
  const int d = ctx->d, dp = round_up(d, 4);
  StepGeom g;
  bucket_geom(ctx, i, j, tb, C, U, seed, g);
  const int key_bits = g.rb + (g.same_table ? 0 : 1);
  const int rel_bits = bits_for((uint64_t)relation_rows(ctx) - 1);
  const bool has_rel = ctx->op != OP_IDENTITY;
  const bool linear = ctx->op == OP_LINEAR;

  StepBufs b = bucket_bufs(ctx, tb);
  if (hipMemsetAsync(b.nuniq, 0, 8, cs) != hipSuccess) return hip_fail(ctx, hipGetLastError(), "counter reset");

  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  (void)hipEventCreate(&ev0);
  (void)hipEventCreate(&ev1);
  const bool timing = (ctx->flags & PBG_F_PHASE_TIMING) != 0;
  const bool score_timing = timing || (ctx->flags & PBG_F_SCORE_TIMING) != 0;
  if (score_timing && !ensure_events(ctx, (size_t)nsteps * kPhaseEvents))
    return set_err(ctx, PBG_ERR_DEVICE, "hipEventCreate failed");
  // events 1 and 2 of a step bracket the score contraction
  auto sampled = [&](int64_t step) { return timing || step % kScoreSample == 0; };
  auto mark = [&](int64_t step, int k) {
    if (timing || (score_timing && (k == 1 || k == 2) && sampled(step)))
      (void)hipEventRecord(ctx->events[(size_t)step * kPhaseEvents + k], cs);
  };
  (void)hipEventRecord(ev0, cs);

  const int64_t kstride = (int64_t)S * 2 * N;   // sort keys per step (a full step)
  uint32_t* const win_keys = ctx->bufs.keys;
  uint32_t* const win_vals = ctx->bufs.vals;
  uint32_t* const win_rkeys = b.rkeys;
  uint32_t* const win_rvals = b.rvals;
  uint32_t *wsk = nullptr, *wsv = nullptr;   // the window's sorted keys and values
  for (int64_t t = 0; t < nsteps; ++t) {
    const int64_t c0 = t * S;
    const int nch = (int)std::min<int64_t>(S, nchunks - c0);
    const int64_t e_lo = chunk_at(c0);
    const int m_step = (int)(chunk_at(c0 + nch) - e_lo);
    g.nchunks = nch;
    g.m_step = m_step;
    g.chunk0 = neg->first_chunk + c0;
    g.cstart = grouped ? ctx->cstart_dev + c0 : nullptr;
    g.cweight = cweight ? cweight + c0 : nullptr;
    b.src = src + e_lo;
    b.dst = dst + e_lo;
    b.rel = rel ? rel + e_lo : nullptr;

    // the sort keys (table, row) of every contribution row follow from the
    // edges and the negative draws alone: at the start of each window of
    // steps, its keys are built and its sorts run as one batch
    const int64_t wi = t % kSortWindow;
    if (wi == 0) {
      const int wn = (int)std::min<int64_t>(kSortWindow, nsteps - t);
      const int64_t cw1 = std::min<int64_t>(nchunks, (t + wn) * (int64_t)S);   // chunks of the window end here
      if (grouped) {
        // steps of relation-grouped chunks hold fewer keys than a full step:
        // the rest of each step's key block sorts last, past every real key
        launch_fill_u32(win_keys, wn * kstride, 1u << key_bits, cs);
      }
      launch_window_keys(g, src + e_lo, dst + e_lo, rel ? rel + e_lo : nullptr, chunk_at(cw1) - e_lo,
                         grouped ? ctx->cstart_dev + c0 : nullptr, (int)(cw1 - c0), neg->first_chunk + c0, S, wn,
                         kstride, win_keys, win_vals, win_rkeys, win_rvals, rstride, uniform_rel ? 1 : 0, cs);
      const int64_t tl = t + wn - 1;   // the window's last step
      const int nch_l = (int)std::min<int64_t>(S, nchunks - tl * S);
      const int m_l = (int)(chunk_at(tl * S + nch_l) - chunk_at(tl * S));
      if (grouped)
        launch_radix_sort_segments(win_keys, win_vals, ctx->wkeys_alt, ctx->wvals_alt, kstride, (int)kstride,
                                   (int)kstride, wn, key_bits + 1, ctx->whist, &wsk, &wsv, cs);
      else
        launch_radix_sort_segments(win_keys, win_vals, ctx->wkeys_alt, ctx->wvals_alt, kstride, (int)kstride,
                                   2 * (nch_l * U + m_l), wn, key_bits, ctx->whist, &wsk, &wsv, cs);
    }
    if (ctx->check_pending) {
      const pbg_status cst = finish_id_check(ctx, i, j);
      if (cst != PBG_OK) {
        (void)hipStreamSynchronize(cs);   // the queued sort touches scratch only
        (void)hipEventDestroy(ev0);
        (void)hipEventDestroy(ev1);
        return cst;
      }
    }
    const int nkeys = 2 * (nch * U + m_step);
    uint32_t* skeys = wsk + wi * kstride;
    uint32_t* svals = wsv + wi * kstride;
    if (win_rkeys) {
      b.rkeys = win_rkeys + wi * rstride;
      b.rvals = win_rvals + wi * rstride;
    }
    // relation keys of the step: the edges', then the uniform source
    // candidates' or the edges' source-side rows
    const int n_relkeys = recip ? 2 * m_step : m_step + (uniform_rel ? nch * U : 0);

    mark(t, 0);

    run_gather_forward(ctx, g, b, cs);
    mark(t, 1);

    if (ctx->flags & PBG_F_BF16_SCORE) {
      run_contractions_bf16(ctx, g, b, t, cs, [&](int k) { mark(t, k); }, false);
    } else {
      run_contractions_f32(ctx, g, b, t, cs, [&](int k) { mark(t, k); }, false);
    }

    mark(t, 4);
    launch_op_backward(g, b, cs);
    if (linear_step_contractions(ctx)) run_linear_backward(g, b, ctx->relA, ctx->relAT, cs);
    else if (linear) launch_linear_rows_backward(g, b, cs);
    mark(t, 5);

    // entities: contribution rows in (table, row) order, segment sums, Adagrad;
    // one relation: its gradient sums and update ride along as extra
    // workgroups of the same two launches
    const bool rel_riders = single_relation_sums(ctx) &&
                            launch_entity_update_with_relation(g, b, skeys, svals, nkeys, ctx->sw, lr,
                                                               op_backward_blocks(g.C, g.U, g.cmp), ctx->relpartial,
                                                               ctx->relp, ctx->relG, cs);
    if (!rel_riders) launch_entity_update(g, b, skeys, svals, nkeys, ctx->sw, lr, cs);

    // relations
    if (has_rel) {
      if (linear_step_contractions(ctx)) {
        // dA per chunk by contraction, then the fixed-order sum of the
        // partials and element-wise Adagrad
        const int nparts = run_linear_relation_grad(g, b, ctx->relpartial, cs);
        launch_relation_single_adagrad(ctx->relp, ctx->relG, d * d, ctx->relpartial, nparts, lr, cs);
      } else if (linear) {
        uint32_t *rk = nullptr, *rv = nullptr;
        launch_radix_sort_to(b.rkeys, b.rvals, n_relkeys, rel_bits, ctx->sw, &rk, &rv, cs);
        launch_linear_relation_update(g, b, rk, rv, n_relkeys, lr, cs);
      } else if (sorted_relation_keys(ctx)) {
        uint32_t *rk = nullptr, *rv = nullptr;
        launch_radix_sort_to(b.rkeys, b.rvals, n_relkeys, rel_bits, ctx->sw, &rk, &rv, cs);
        launch_relation_update_sorted(g, b, rk, rv, n_relkeys, ctx->sw, lr, cs);
      } else {
        // one relation: the operator backward left one gradient row per
        // block of its grid; their fixed-order sums, then element-wise
        // Adagrad (unless they rode along with the entity update)
        if (!rel_riders) {
          launch_relation_block_sums(g, b.relc, op_backward_blocks(g.C, g.U, g.cmp), ctx->relpartial, cs);
          launch_relation_single_adagrad(ctx->relp, ctx->relG, ctx->dr, ctx->relpartial, nch * RELSUM_PIECES,
                                         lr, cs);
        }
      }
    }
    mark(t, 6);
  }
  {
    const int nch_last = (int)(nchunks - (nsteps - 1) * S);
    launch_step_losses(ctx->lossparts, ctx->lossparts_pps, (int)(S * fb), (int)(nch_last * fb), nsteps,
                       ctx->steploss_dev, cs);
  }
  (void)hipEventRecord(ev1, cs);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    (void)hipEventDestroy(ev0);
    (void)hipEventDestroy(ev1);
    return hip_fail(ctx, e, "kernel launch");
  }
  std::vector<double> losses((size_t)nsteps);
  unsigned long long nuniq = 0;
  e = hipMemcpyAsync(losses.data(), ctx->steploss_dev, (size_t)nsteps * 8, hipMemcpyDeviceToHost, cs);
  if (e == hipSuccess) e = hipMemcpyAsync(&nuniq, b.nuniq, 8, hipMemcpyDeviceToHost, cs);
  if (e == hipSuccess) e = hipStreamSynchronize(cs);
  float ms = 0.f;
  if (e == hipSuccess) (void)hipEventElapsedTime(&ms, ev0, ev1);
  (void)hipEventDestroy(ev0);
  (void)hipEventDestroy(ev1);
  if (e != hipSuccess) return hip_fail(ctx, e, "training step");
  double total = 0.0;
  for (double v : losses) total += v;
  if (loss_out) *loss_out = total;
  if (step_losses) step_losses->insert(step_losses->end(), losses.begin(), losses.end());
  ctx->stats.total_ms += ms;
  if (score_timing) {
    double* acc[6] = {&ctx->stats.gather_ms, &ctx->stats.score_ms, &ctx->stats.epilogue_ms,
                      &ctx->stats.backward_ms, &ctx->stats.opbwd_ms, &ctx->stats.update_ms};
    for (int64_t t = 0; t < nsteps; ++t) {
      if (!sampled(t)) continue;
      ++ctx->stats.score_timed_steps;
      for (int k = timing ? 0 : 1; k < (timing ? 6 : 2); ++k) {
        float pm = 0.f;
        (void)hipEventElapsedTime(&pm, ctx->events[(size_t)t * kPhaseEvents + k],
                                  ctx->events[(size_t)t * kPhaseEvents + k + 1]);
        *acc[k] += pm;
      }
    }
  }
  ctx->stats.edges += n_edges;
  ctx->stats.chunks += nchunks;
  ctx->stats.steps += nsteps;
  // algorithmic work (full chunks approximated by the actual chunk sizes)
  const double U_d = U;
  for (int64_t c = 0; c < nchunks; ++c) {
    const double Cc = (double)(chunk_at(c + 1) - chunk_at(c));
    const double Nc = Cc + U_d;
    ctx->stats.gather_bytes += (2 * Cc + 2 * U_d) * d * 4.0;
    ctx->stats.score_flops += 12.0 * Cc * Nc * d;
    ctx->stats.update_bytes += (2 * Cc + 2 * U_d) * d * 4.0;   // contribution rows read
  }
  // each touched row: its embedding read and written, its Adagrad scalar read
  // and written
  ctx->stats.update_bytes += (double)nuniq * (2.0 * d * 4 + 8);
  return PBG_OK;
}

pbg_status check_bucket_call(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src_local,
                             const int32_t* rel, const int32_t* dst_local, int64_t n_edges,
                             const pbg_neg_config* neg, bool defer) {
  ctx->check_pending = false;
  if (i < 0 || i >= ctx->P || j < 0 || j >= ctx->P)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "bucket (%d, %d) out of range", i, j);
  pbg_status st = check_neg_config(ctx, neg);
  if (st != PBG_OK) return st;
  if (n_edges < 0 || n_edges > 0x7FFFFFFFll) return set_err(ctx, PBG_ERR_INVALID_ARG, "n_edges out of range");
  const Partition& pi = ctx->parts[i];
  const Partition& pj = ctx->parts[j];
  if (!pi.emb || !pj.emb) return set_err(ctx, PBG_ERR_STATE, "partition %d or %d is not bound", i, j);
  if (pi.where != PBG_MEM_DEVICE || pj.where != PBG_MEM_DEVICE)
    return set_err(ctx, PBG_ERR_STATE, "training needs device-resident partitions");
  if (ctx->op != OP_IDENTITY && !ctx->relp) return set_err(ctx, PBG_ERR_STATE, "relation parameters are not bound");
  if (n_edges == 0) return PBG_OK;
  if (ctx->R > 1 && !rel) return set_err(ctx, PBG_ERR_INVALID_ARG, "rel may be NULL only with one relation");
  if (!src_local || !dst_local) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL edge arrays");
  if (chunk_relation_operator(ctx) && !grouped_chunks(ctx, neg))
    return set_err(ctx, PBG_ERR_UNSUPPORTED,
                   "cos with an operator and several relations needs relation-grouped chunks (PBG_CHUNK_BY_RELATION)");
  st = ensure_workspace(ctx, neg->chunk_size, neg->num_uniform, neg->chunks_per_step);
  if (st != PBG_OK) return st;
  // device-side range check before any update
  hipStream_t cs = ctx->cs;
  hipError_t e = hipMemsetAsync(ctx->flag_dev, 0, 4, cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipMemsetAsync");
  launch_check_ids(src_local, n_edges, (int32_t)pbg_partition_rows(ctx, i), ctx->flag_dev, 1u, cs);
  launch_check_ids(dst_local, n_edges, (int32_t)pbg_partition_rows(ctx, j), ctx->flag_dev, 2u, cs);
  if (rel) launch_check_ids(rel, n_edges, ctx->R, ctx->flag_dev, 4u, cs);
  if (!ctx->hflag && hipHostMalloc((void**)&ctx->hflag, 16) != hipSuccess) {
    (void)hipGetLastError();
    ctx->hflag = nullptr;
    return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "page-locked flag allocation failed");
  }
  if (!ctx->check_ev && hipEventCreateWithFlags(&ctx->check_ev, hipEventDisableTiming) != hipSuccess) {
    (void)hipGetLastError();
    ctx->check_ev = nullptr;
    return set_err(ctx, PBG_ERR_DEVICE, "hipEventCreate failed");
  }
  e = hipMemcpyAsync(ctx->hflag, ctx->flag_dev, 4, hipMemcpyDeviceToHost, cs);
  if (e == hipSuccess) e = hipEventRecord(ctx->check_ev, cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "id range check");
  if (defer) {
    ctx->check_pending = true;
    return PBG_OK;
  }
  return finish_id_check(ctx, i, j);
}

pbg_status finish_id_check(pbg_ctx* ctx, int32_t i, int32_t j) {
  ctx->check_pending = false;
  const hipError_t e = hipEventSynchronize(ctx->check_ev);
  if (e != hipSuccess) return hip_fail(ctx, e, "id range check");
  const uint32_t flag = *(volatile uint32_t*)ctx->hflag;
  if (flag & 1u) return set_err(ctx, PBG_ERR_INVALID_ARG, "a source id is outside partition %d", i);
  if (flag & 2u) return set_err(ctx, PBG_ERR_INVALID_ARG, "a destination id is outside partition %d", j);
  if (flag & 4u) return set_err(ctx, PBG_ERR_INVALID_ARG, "a relation id is outside [0, %d)", ctx->R);
  return PBG_OK;
}

extern "C" pbg_status pbg_train_bucket(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src_local,
                                       const int32_t* rel, const int32_t* dst_local, int64_t n_edges,
                                       const pbg_neg_config* neg, float lr, uint64_t seed,
                                       double* loss_host) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  ctx->err.clear();
  if (!std::isfinite(lr) || lr < 0.f) return set_err(ctx, PBG_ERR_INVALID_ARG, "lr must be finite and >= 0");
  if (ctx->T > 1) {
    // entity types: the call's runs are checked and trained one by one
    ctx->stats = pbg_stats();
    ctx->step_losses.clear();
    return train_bucket_typed(ctx, i, j, src_local, rel, dst_local, n_edges, neg, lr, seed, loss_host,
                              &ctx->step_losses);
  }
  // the id check's verdict is awaited after the first window's sort keys are
  // queued (they need no valid ids), so the device does not idle meanwhile
  pbg_status st = check_bucket_call(ctx, i, j, src_local, rel, dst_local, n_edges, neg, true);
  if (st != PBG_OK) return st;
  ctx->stats = pbg_stats();
  ctx->step_losses.clear();
  if (n_edges == 0) {
    if (loss_host) *loss_host = 0.0;
    return PBG_OK;
  }
  return train_bucket_device(ctx, i, j, partition_tables(ctx, i, j), src_local, rel, dst_local, n_edges, neg, lr,
                             seed, loss_host, &ctx->step_losses);
}

extern "C" pbg_status pbg_score_edges(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src_local,
                                      const int32_t* rel, const int32_t* dst_local, int64_t n,
                                      float* scores) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  ctx->err.clear();
  if (ctx->T > 1) return set_err(ctx, PBG_ERR_UNSUPPORTED, "pbg_score_edges takes one entity type");
  if (i < 0 || i >= ctx->P || j < 0 || j >= ctx->P)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "bucket (%d, %d) out of range", i, j);
  if (n < 0 || n > 0x7FFFFFFFll) return set_err(ctx, PBG_ERR_INVALID_ARG, "n out of range");
  const Partition& pi = ctx->parts[i];
  const Partition& pj = ctx->parts[j];
  if (!pi.emb || !pj.emb || pi.where != PBG_MEM_DEVICE || pj.where != PBG_MEM_DEVICE)
    return set_err(ctx, PBG_ERR_STATE, "partitions %d and %d must be bound in device memory", i, j);
  if (ctx->op != OP_IDENTITY && !ctx->relp) return set_err(ctx, PBG_ERR_STATE, "relation parameters are not bound");
  if (n == 0) return PBG_OK;
  if (ctx->R > 1 && !rel) return set_err(ctx, PBG_ERR_INVALID_ARG, "rel may be NULL only with one relation");
  if (!src_local || !dst_local || !scores) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL array");
  hipStream_t cs = ctx->cs;
  uint32_t* flag_dev = nullptr;
  float* relT = nullptr;
  hipError_t e = hipMalloc(&flag_dev, 16);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipMalloc");
  if (ctx->op == OP_LINEAR) {
    e = hipMalloc(&relT, (size_t)ctx->R * ctx->d * ctx->d * 4);
    if (e != hipSuccess) {
      (void)hipFree(flag_dev);
      return hip_fail(ctx, e, "hipMalloc");
    }
  }
  (void)hipMemsetAsync(flag_dev, 0, 4, cs);
  launch_check_ids(src_local, n, (int32_t)pbg_partition_rows(ctx, i), flag_dev, 1u, cs);
  launch_check_ids(dst_local, n, (int32_t)pbg_partition_rows(ctx, j), flag_dev, 2u, cs);
  if (rel) launch_check_ids(rel, n, ctx->R, flag_dev, 4u, cs);
  uint32_t flag = 0;
  e = hipMemcpyAsync(&flag, flag_dev, 4, hipMemcpyDeviceToHost, cs);
  if (e == hipSuccess) e = hipStreamSynchronize(cs);
  pbg_status st = PBG_OK;
  if (e != hipSuccess) st = hip_fail(ctx, e, "id range check");
  else if (flag) st = set_err(ctx, PBG_ERR_INVALID_ARG, "an id is out of range (flags %u)", flag);
  if (st == PBG_OK) {
    StepGeom g;
    memset(&g, 0, sizeof(g));
    g.d = ctx->d;
    g.dp = round_up(ctx->d, 4);
    g.dr = ctx->dr;
    g.op = ctx->op;
    g.cmp = ctx->cmp;
    if (relT) launch_transpose_rel(ctx->relp, relT, ctx->R, ctx->d, cs);
    launch_score_edges(g, pi.emb, pj.emb, ctx->relp, relT, src_local, rel, dst_local, n, scores, cs);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipStreamSynchronize(cs);
    if (e != hipSuccess) st = hip_fail(ctx, e, "score_edges");
  }
  (void)hipFree(flag_dev);
  if (relT) (void)hipFree(relT);
  return st;
}

extern "C" pbg_status pbg_sample_negatives(pbg_ctx* ctx, int32_t i, int32_t j, int64_t first_chunk,
                                           int64_t n_chunks, int32_t num_uniform, uint64_t seed,
                                           int32_t* out) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  ctx->err.clear();
  if (i < 0 || i >= ctx->P || j < 0 || j >= ctx->P)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "bucket (%d, %d) out of range", i, j);
  if (first_chunk < 0 || n_chunks < 0 || first_chunk + n_chunks > 0x100000000ll || num_uniform < 0)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "chunk range or num_uniform out of range");
  if (n_chunks == 0 || num_uniform == 0) return PBG_OK;
  if (!out) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL output");
  launch_sample_negatives(seed, (uint32_t)(i * ctx->P + j), first_chunk, n_chunks, num_uniform,
                          (uint32_t)pbg_partition_rows(ctx, j), (uint32_t)pbg_partition_rows(ctx, i),
                          out, ctx->cs);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "sample_negatives");
  return PBG_OK;
}

extern "C" pbg_status pbg_group_by_relation(pbg_ctx* ctx, const int32_t* src, const int32_t* rel,
                                            const int32_t* dst, int64_t n, int32_t* src_out, int32_t* rel_out,
                                            int32_t* dst_out) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  ctx->err.clear();
  if (n < 0 || n > 0x7FFFFFFFll) return set_err(ctx, PBG_ERR_INVALID_ARG, "n out of range");
  if (n == 0) return PBG_OK;
  if (!src || !rel || !dst || !src_out || !rel_out || !dst_out)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL array");
  hipStream_t cs = ctx->cs;
  // a stable radix sort of (relation, position) pairs, then one gather
  Arena a;
  uint32_t* flag = (uint32_t*)a.get(16);
  uint32_t* keys = (uint32_t*)a.get((size_t)n * 4);
  uint32_t* vals = (uint32_t*)a.get((size_t)n * 4);
  SortWork w{};
  if (a.failed || !alloc_sortwork(a, w, n, 0)) {
    a.release();
    return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "work buffer allocation failed");
  }
  hipError_t e = hipMemsetAsync(flag, 0, 4, cs);
  if (e == hipSuccess) {
    launch_check_ids(rel, n, ctx->R, flag, 4u, cs);
    uint32_t hflag = 0;
    e = hipMemcpyAsync(&hflag, flag, 4, hipMemcpyDeviceToHost, cs);
    if (e == hipSuccess) e = hipStreamSynchronize(cs);
    if (e == hipSuccess && hflag) {
      a.release();
      return set_err(ctx, PBG_ERR_INVALID_ARG, "a relation id is outside [0, %d)", ctx->R);
    }
  }
  if (e == hipSuccess) {
    launch_perm_keys(rel, nullptr, n, keys, vals, cs);
    launch_radix_sort(keys, vals, (int)n, std::max(1, bits_for((uint64_t)ctx->R - 1)), w, cs);
    launch_gather3(vals, src, rel, dst, n, src_out, rel_out, dst_out, cs);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipStreamSynchronize(cs);
  }
  a.release();
  if (e != hipSuccess) return hip_fail(ctx, e, "group_by_relation");
  return PBG_OK;
}
