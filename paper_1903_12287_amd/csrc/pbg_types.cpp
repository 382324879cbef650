// Entity types (Sec. 3.1: negatives only from the entity type of the edge's
// relation; Sec. 4.1 and Fig. 1 centre: small types need not be partitioned)
// and per-relation edge weights (Sec. 1 and 6: per-relation configuration).
//
// A typed context keeps one table per (type, partition); a type kept whole has
// its single table at partition 0, so its edges fall into buckets (0, *) or
// (*, 0).  A bucket's edges, sorted by relation, train in runs: maximal blocks
// of consecutive relations with the same (source type, destination type).
// Each run is one call of the step loop on its two tables, so its chunks
// draw their negatives from those tables and no step mixes two runs; the
// chunk numbers (and so the Philox counters) continue across runs.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "kernels.h"
#include "runtime_internal.h"

namespace {

struct TypedRun {
  int64_t lo = 0, hi = 0;   // edges of the call
  int64_t chunk0 = 0;       // chunks of the call before the run
  int st = 0, dt = 0;
  BucketTables tb;
};

struct DevPtrs {
  std::vector<void*> ptrs;
  void* get(size_t bytes) {
    void* p = nullptr;
    if (hipMalloc(&p, std::max<size_t>(bytes, 16)) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    ptrs.push_back(p);
    return p;
  }
  ~DevPtrs() {
    for (void* p : ptrs) (void)hipFree(p);
  }
};

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// the relation ids of a call (device) on the host, range-checked
pbg_status relations_on_host(pbg_ctx* ctx, const int32_t* rel, int64_t n, std::vector<int32_t>& r) {
  r.assign((size_t)n, 0);
  if (!rel || n == 0) return PBG_OK;
  hipError_t e = hipMemcpyAsync(r.data(), rel, (size_t)n * 4, hipMemcpyDeviceToHost, ctx->cs);
  if (e == hipSuccess) e = hipStreamSynchronize(ctx->cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "relation copy");
  for (int64_t k = 0; k < n; ++k)
    if (r[(size_t)k] < 0 || r[(size_t)k] >= ctx->R)
      return set_err(ctx, PBG_ERR_INVALID_ARG, "a relation id is outside [0, %d)", ctx->R);
  return PBG_OK;
}

// The runs of a typed call on bucket (i, j), with every check made before
// anything trains: arguments, relation order, the partition of whole types,
// bound device-resident tables, and every id against its table's rows.
pbg_status typed_runs(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src, const int32_t* rel, const int32_t* dst,
                      int64_t n, const pbg_neg_config* neg, std::vector<TypedRun>& runs) {
  runs.clear();
  if (i < 0 || i >= ctx->P || j < 0 || j >= ctx->P)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "bucket (%d, %d) out of range", i, j);
  pbg_status st = check_neg_config(ctx, neg);
  if (st != PBG_OK) return st;
  if (n < 0 || n > 0x7FFFFFFFll) return set_err(ctx, PBG_ERR_INVALID_ARG, "n_edges out of range");
  if (ctx->op != OP_IDENTITY && !ctx->relp) return set_err(ctx, PBG_ERR_STATE, "relation parameters are not bound");
  if (n == 0) return PBG_OK;
  if (ctx->R > 1 && !rel) return set_err(ctx, PBG_ERR_INVALID_ARG, "rel may be NULL only with one relation");
  if (!src || !dst) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL edge arrays");
  if (ctx->R > 1 && neg->chunking != PBG_CHUNK_BY_RELATION)
    return set_err(ctx, PBG_ERR_UNSUPPORTED,
                   "entity types need relation-grouped chunks (PBG_CHUNK_BY_RELATION) with several relations");
  if (chunk_relation_operator(ctx) && !grouped_chunks(ctx, neg))
    return set_err(ctx, PBG_ERR_UNSUPPORTED,
                   "cos with an operator and several relations needs relation-grouped chunks (PBG_CHUNK_BY_RELATION)");
  std::vector<int32_t> r;
  st = relations_on_host(ctx, rel, n, r);
  if (st != PBG_OK) return st;
  const int C = neg->chunk_size;
  int64_t chunks = 0, rel_lo = 0;
  for (int64_t k = 0; k <= n; ++k) {
    if (k > 0 && k < n && r[(size_t)k] < r[(size_t)k - 1])
      return set_err(ctx, PBG_ERR_INVALID_ARG, "entity types need the edges sorted by relation (edge %lld)",
                     (long long)k);
    const bool rel_end = k == n || (k > 0 && r[(size_t)k] != r[(size_t)k - 1]);
    if (k > 0 && rel_end) {
      // relation run [rel_lo, k): join the current type run or start one
      const int rr = r[(size_t)rel_lo];
      const int s_t = ctx->rel_st[(size_t)rr], d_t = ctx->rel_dt[(size_t)rr];
      if (runs.empty() || runs.back().st != s_t || runs.back().dt != d_t) {
        TypedRun tr;
        tr.lo = rel_lo;
        tr.chunk0 = chunks;
        tr.st = s_t;
        tr.dt = d_t;
        runs.push_back(tr);
      }
      runs.back().hi = k;
      // relation-grouped chunks of C edges (with one relation: consecutive)
      chunks += ceil_div(k - rel_lo, C);
      rel_lo = k;
    }
  }
  for (TypedRun& tr : runs) {
    if ((!ctx->type_part[(size_t)tr.st] && i != 0) || (!ctx->type_part[(size_t)tr.dt] && j != 0))
      return set_err(ctx, PBG_ERR_INVALID_ARG,
                     "bucket (%d, %d) holds edges of relation %d, whose %s type is kept whole (partition 0 only)", i,
                     j, r[(size_t)tr.lo], !ctx->type_part[(size_t)tr.st] && i != 0 ? "source" : "destination");
    const Partition ps = resolve_table(ctx, tr.st, i);
    const Partition pd = resolve_table(ctx, tr.dt, j);
    if (!ps.emb || !pd.emb)
      return set_err(ctx, PBG_ERR_STATE, "table (type %d, partition %d) or (type %d, partition %d) is not bound",
                     tr.st, i, tr.dt, j);
    if (ps.where != PBG_MEM_DEVICE || pd.where != PBG_MEM_DEVICE)
      return set_err(ctx, PBG_ERR_STATE, "training needs device-resident tables");
    tr.tb.emb_i = ps.emb;
    tr.tb.G_i = ps.G;
    tr.tb.emb_j = pd.emb;
    tr.tb.G_j = pd.G;
    tr.tb.rows_i = table_rows(ctx, tr.st, i);
    tr.tb.rows_j = table_rows(ctx, tr.dt, j);
    tr.tb.same = tr.st == tr.dt && i == j;
  }
  st = ensure_workspace(ctx, neg->chunk_size, neg->num_uniform, neg->chunks_per_step);
  if (st != PBG_OK) return st;
  hipStream_t cs = ctx->cs;
  hipError_t e = hipMemsetAsync(ctx->flag_dev, 0, 4, cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "hipMemsetAsync");
  for (const TypedRun& tr : runs) {
    launch_check_ids(src + tr.lo, tr.hi - tr.lo, (int32_t)tr.tb.rows_i, ctx->flag_dev, 1u, cs);
    launch_check_ids(dst + tr.lo, tr.hi - tr.lo, (int32_t)tr.tb.rows_j, ctx->flag_dev, 2u, cs);
  }
  uint32_t flag = 0;
  e = hipMemcpyAsync(&flag, ctx->flag_dev, 4, hipMemcpyDeviceToHost, cs);
  if (e == hipSuccess) e = hipStreamSynchronize(cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "id range check");
  if (flag & 1u) return set_err(ctx, PBG_ERR_INVALID_ARG, "a source id is outside its type's table");
  if (flag & 2u) return set_err(ctx, PBG_ERR_INVALID_ARG, "a destination id is outside its type's table");
  return PBG_OK;
}

}  // namespace

pbg_status train_bucket_typed(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src, const int32_t* rel,
                              const int32_t* dst, int64_t n_edges, const pbg_neg_config* neg, float lr, uint64_t seed,
                              double* loss_out, std::vector<double>* step_losses) {
  std::vector<TypedRun> runs;
  pbg_status st = typed_runs(ctx, i, j, src, rel, dst, n_edges, neg, runs);
  if (st != PBG_OK) return st;
  double total = 0.0;
  for (const TypedRun& tr : runs) {
    pbg_neg_config nr = *neg;
    nr.first_chunk = neg->first_chunk + tr.chunk0;
    double loss = 0.0;
    st = train_bucket_device(ctx, i, j, tr.tb, src + tr.lo, rel ? rel + tr.lo : nullptr, dst + tr.lo, tr.hi - tr.lo,
                             &nr, lr, seed, &loss, step_losses);
    if (st != PBG_OK) return st;
    total += loss;
  }
  if (loss_out) *loss_out = total;
  return PBG_OK;
}

pbg_status typed_single_run(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src, const int32_t* rel,
                            const int32_t* dst, int64_t n_edges, const pbg_neg_config* neg, BucketTables* tb) {
  std::vector<TypedRun> runs;
  pbg_status st = typed_runs(ctx, i, j, src, rel, dst, n_edges, neg, runs);
  if (st != PBG_OK) return st;
  if (runs.size() > 1)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "the edges span several (source type, destination type) pairs");
  if (runs.empty()) {
    *tb = BucketTables();
    return PBG_OK;
  }
  *tb = runs[0].tb;
  return PBG_OK;
}

// Host checks of a typed epoch, before anything trains: every table bound,
// every relation id in range and sorted within its bucket, every relation's
// types able to have edges in the bucket, every id inside its table.
pbg_status validate_typed_epoch(pbg_ctx* ctx, const int64_t* off, const int32_t* hs, const int32_t* hr,
                                const int32_t* hd) {
  const int P = ctx->P;
  const int nb = P * P;
  for (int t = 0; t < ctx->T; ++t)
    for (int p = 0; p < (ctx->type_part[(size_t)t] ? P : 1); ++p)
      if (!table_of(ctx, t, p).emb)
        return set_err(ctx, PBG_ERR_STATE, "table (type %d, partition %d) is not bound", t, p);
  for (int b = 0; b < nb; ++b) {
    const int i = b / P, j = b % P;
    const int64_t lo = off[b], hi = off[b + 1];
    for (int64_t k = lo; k < hi; ++k) {
      const int32_t r = hr ? hr[k] : 0;
      if (r < 0 || r >= ctx->R) return set_err(ctx, PBG_ERR_INVALID_ARG, "a relation id is outside [0, %d)", ctx->R);
      if (k > lo && hr && r < hr[k - 1])
        return set_err(ctx, PBG_ERR_INVALID_ARG, "entity types need each bucket's edges sorted by relation (bucket %d)",
                       b);
      const int st = ctx->rel_st[(size_t)r], dt = ctx->rel_dt[(size_t)r];
      const int64_t ri = table_rows(ctx, st, i), rj = table_rows(ctx, dt, j);
      if (ri < 0 || rj < 0)
        return set_err(ctx, PBG_ERR_INVALID_ARG, "bucket %d holds an edge of relation %d, whose types have no "
                                                 "partition there", b, r);
      if (hs[k] < 0 || hs[k] >= ri || hd[k] < 0 || hd[k] >= rj)
        return set_err(ctx, PBG_ERR_INVALID_ARG, "an id of bucket %d is outside its type's table", b);
    }
  }
  return PBG_OK;
}

// One epoch over a typed graph whose tables are all device-resident (checked
// by validate_typed_epoch): the buckets with edges in inside-out order
// (Sec. 4.1, Fig. 1 right), each trained as pbg_train_bucket trains it.
pbg_status train_epoch_typed(pbg_ctx* ctx, const int64_t* off, const int32_t* hs, const int32_t* hr,
                             const int32_t* hd, const pbg_neg_config* neg, float lr, uint64_t seed,
                             double* loss_host) {
  const int P = ctx->P;
  int64_t max_bucket = 0;
  for (int b = 0; b < P * P; ++b) max_bucket = std::max(max_bucket, off[b + 1] - off[b]);
  ctx->stats = pbg_stats();
  ctx->step_losses.clear();
  DevPtrs buf;
  int32_t* ds = (int32_t*)buf.get((size_t)max_bucket * 4);
  int32_t* dd = (int32_t*)buf.get((size_t)max_bucket * 4);
  int32_t* dr = hr ? (int32_t*)buf.get((size_t)max_bucket * 4) : nullptr;
  if (!ds || !dd || (hr && !dr)) return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "edge staging buffers could not be allocated");
  double total = 0.0;
  std::vector<std::pair<int, int>> order;
  order.push_back({0, 0});
  for (int k = 1; k < P; ++k) {
    for (int m = 0; m < k; ++m) {
      order.push_back({k, m});
      order.push_back({m, k});
    }
    order.push_back({k, k});
  }
  for (const auto& bk : order) {
    const int b = bk.first * P + bk.second;
    const int64_t lo = off[b], n = off[b + 1] - off[b];
    if (n == 0) continue;
    hipError_t e = hipMemcpyAsync(ds, hs + lo, (size_t)n * 4, hipMemcpyHostToDevice, ctx->cs);
    if (e == hipSuccess) e = hipMemcpyAsync(dd, hd + lo, (size_t)n * 4, hipMemcpyHostToDevice, ctx->cs);
    if (e == hipSuccess && dr) e = hipMemcpyAsync(dr, hr + lo, (size_t)n * 4, hipMemcpyHostToDevice, ctx->cs);
    if (e != hipSuccess) return hip_fail(ctx, e, "edge staging");
    double loss = 0.0;
    pbg_status st = train_bucket_typed(ctx, bk.first, bk.second, ds, dr, dd, n, neg, lr, seed, &loss,
                                       &ctx->step_losses);
    if (st != PBG_OK) return st;
    total += loss;
  }
  if (loss_host) *loss_host = total;
  return PBG_OK;
}

// Typed bucketing: every relation's (partition size, entity count) of its
// source and destination type on the device, then the bucket keys, a stable
// radix sort, the offsets and the local ids (nothing is written on an error).
pbg_status bucket_edges_typed(pbg_ctx* ctx, const int64_t* src, const int32_t* rel, const int64_t* dst, int64_t n,
                              int64_t* offsets, int32_t* src_local, int32_t* rel_out, int32_t* dst_local) {
  const int P = ctx->P, R = ctx->R;
  const int nb = P * P;
  std::vector<int64_t> geo((size_t)R * 4);
  for (int r = 0; r < R; ++r) {
    const int st = ctx->rel_st[(size_t)r], dt = ctx->rel_dt[(size_t)r];
    geo[(size_t)r * 4 + 0] = ceil_div(ctx->type_n[(size_t)st], ctx->type_part[(size_t)st] ? P : 1);
    geo[(size_t)r * 4 + 1] = ctx->type_n[(size_t)st];
    geo[(size_t)r * 4 + 2] = ceil_div(ctx->type_n[(size_t)dt], ctx->type_part[(size_t)dt] ? P : 1);
    geo[(size_t)r * 4 + 3] = ctx->type_n[(size_t)dt];
  }
  hipStream_t s = ctx->cs;
  DevPtrs buf;
  int64_t* geo_d = (int64_t*)buf.get(geo.size() * 8);
  uint32_t* flag = (uint32_t*)buf.get(16);
  uint32_t* keys = (uint32_t*)buf.get((size_t)n * 4);
  uint32_t* vals = (uint32_t*)buf.get((size_t)n * 4);
  SortWork w;
  memset(&w, 0, sizeof(w));
  w.keys_alt = (uint32_t*)buf.get((size_t)n * 4);
  w.vals_alt = (uint32_t*)buf.get((size_t)n * 4);
  w.hist = (uint32_t*)buf.get((size_t)radix_hist_entries(n) * 4);
  w.scan_tmp = (uint32_t*)buf.get((size_t)radix_scan_tmp_entries(n) * 4);
  w.max_n = (int)n;
  if (!geo_d || !flag || !keys || !vals || !w.keys_alt || !w.vals_alt || !w.hist || !w.scan_tmp)
    return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "bucketing workspace (%lld edges) could not be allocated", (long long)n);
  hipError_t e = hipMemcpyAsync(geo_d, geo.data(), geo.size() * 8, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipMemsetAsync(flag, 0, 4, s);
  if (e != hipSuccess) return hip_fail(ctx, e, "bucketing set-up");
  launch_typed_bucket_keys(src, rel, dst, n, geo_d, R, P, keys, vals, flag, s);
  uint32_t hflag = 0;
  e = hipMemcpyAsync(&hflag, flag, 4, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(ctx, e, "bucket keys");
  if (hflag & 4u) return set_err(ctx, PBG_ERR_INVALID_ARG, "a relation id is outside [0, %d)", R);
  if (hflag & 3u) return set_err(ctx, PBG_ERR_INVALID_ARG, "an entity id is outside its type's range");
  int bits = 0;
  while (bits < 32 && ((uint64_t)(nb - 1) >> bits) != 0) ++bits;
  launch_radix_sort(keys, vals, (int)n, bits, w, s);
  launch_bucket_offsets(keys, n, nb, offsets, s);
  launch_typed_bucket_gather(vals, src, rel, dst, n, geo_d, src_local, rel_out, dst_local, s);
  e = hipGetLastError();
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(ctx, e, "bucketing");
  return PBG_OK;
}

// --------------------------------------------------------------------------
// C ABI
// --------------------------------------------------------------------------
extern "C" pbg_status pbg_set_entity_types(pbg_ctx* ctx, int32_t num_types, const int64_t* type_entities,
                                           const int32_t* type_partitioned, const int32_t* rel_src_type,
                                           const int32_t* rel_dst_type) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  ctx->err.clear();
  if (num_types < 1 || num_types > 4096) return set_err(ctx, PBG_ERR_INVALID_ARG, "num_types must be in [1, 4096]");
  if (!type_entities || !type_partitioned || !rel_src_type || !rel_dst_type)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL type array");
  const int P = ctx->P;
  for (int t = 0; t < num_types; ++t) {
    const int64_t n = type_entities[t];
    if (n < 1) return set_err(ctx, PBG_ERR_INVALID_ARG, "type %d has no entities", t);
    const int parts = type_partitioned[t] ? P : 1;
    const int64_t ps = ceil_div(n, parts);
    if ((int64_t)(parts - 1) * ps >= n)
      return set_err(ctx, PBG_ERR_INVALID_ARG, "type %d would leave a partition empty", t);
    if (ps > (1ll << 30)) return set_err(ctx, PBG_ERR_INVALID_ARG, "tables above 2^30 rows are not supported");
  }
  for (int r = 0; r < ctx->R; ++r)
    if (rel_src_type[r] < 0 || rel_src_type[r] >= num_types || rel_dst_type[r] < 0 || rel_dst_type[r] >= num_types)
      return set_err(ctx, PBG_ERR_INVALID_ARG, "relation %d names a type outside [0, %d)", r, num_types);
  (void)hipStreamSynchronize(ctx->cs);
  ctx->T = num_types;
  ctx->type_n.assign(type_entities, type_entities + num_types);
  ctx->type_part.assign(num_types, 0);
  for (int t = 0; t < num_types; ++t) ctx->type_part[(size_t)t] = type_partitioned[t] ? 1 : 0;
  ctx->rel_st.assign(rel_src_type, rel_src_type + ctx->R);
  ctx->rel_dt.assign(rel_dst_type, rel_dst_type + ctx->R);
  ctx->parts.assign((size_t)num_types * P, Partition());   // every table is bound again
  ctx->n = ctx->type_n[0];
  ctx->ps = ceil_div(ctx->n, ctx->type_part[0] ? P : 1);
  return PBG_OK;
}

extern "C" pbg_status pbg_bind_type_partition(pbg_ctx* ctx, int32_t t, int32_t p, float* emb, float* adagrad,
                                              int32_t where) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  if (table_rows(ctx, t, p) < 0)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "table (type %d, partition %d) does not exist", t, p);
  if (!emb || !adagrad) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL embedding or accumulator");
  if (where != PBG_MEM_DEVICE && where != PBG_MEM_PINNED_HOST)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "unknown memory kind %d", where);
  Partition& tp = table_of(ctx, t, p);
  tp.emb = emb;
  tp.G = adagrad;
  tp.where = where;
  ctx->err.clear();
  return PBG_OK;
}

extern "C" int64_t pbg_type_partition_rows(const pbg_ctx* ctx, int32_t t, int32_t p) { return table_rows(ctx, t, p); }

extern "C" pbg_status pbg_set_relation_weights(pbg_ctx* ctx, const float* weights_host) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  ctx->err.clear();
  if (!weights_host) {
    ctx->relw.clear();
    return PBG_OK;
  }
  for (int r = 0; r < ctx->R; ++r)
    if (!std::isfinite(weights_host[r]) || weights_host[r] < 0.f)
      return set_err(ctx, PBG_ERR_INVALID_ARG, "relation weight %d must be finite and >= 0", r);
  ctx->relw.assign(weights_host, weights_host + ctx->R);
  return PBG_OK;
}
