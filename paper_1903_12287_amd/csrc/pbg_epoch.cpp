// pbg_train_epoch: one epoch over all buckets of a partitioned graph with the
// partitions swapped between page-locked host memory and HBM slots
// (Sec. 4.1: buckets are trained one at a time in inside-out order, Fig. 1
// right; only the two partitions of the current bucket need to be resident).
//
// Buckets with edges are visited in inside-out order.  Partitions live in at
// most max_resident HBM slots.  Transfers run on the copy stream and are
// ordered against the compute stream with events only:
//   load p into slot v:  copy stream waits for v's last compute use, writes the
//                        evicted partition back (D2H), then reads p (H2D) and
//                        records `ready`;
//   train bucket (i, j): compute stream waits for the two slots' `ready` and
//                        the bucket's edges, trains, records `released`.
// While bucket t trains, the copy stream already moves bucket t+1's edges and
// any of its partitions that fit in a slot not used by buckets t and t+1.
// The victim of a load is an empty slot, else the slot whose partition is
// needed again furthest in the future.  The schedule is fixed by P, the
// offsets and max_resident, and every bucket is trained exactly as
// pbg_train_bucket trains it, so the result is bitwise that of training the
// buckets one after another on device-resident partitions.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstring>
#include <vector>

#include "kernels.h"
#include "runtime_internal.h"

namespace {

std::vector<std::pair<int, int>> inside_out(int P) {
  std::vector<std::pair<int, int>> o;
  o.push_back({0, 0});
  for (int k = 1; k < P; ++k) {
    for (int m = 0; m < k; ++m) {
      o.push_back({k, m});
      o.push_back({m, k});
    }
    o.push_back({k, k});
  }
  return o;
}

struct EdgeBuf {
  int32_t* src = nullptr;
  int32_t* rel = nullptr;
  int32_t* dst = nullptr;
  hipEvent_t ready = nullptr;
  hipEvent_t consumed = nullptr;
  bool used = false;
  int bucket = -1;
};

struct EpochRun {
  pbg_ctx* ctx;
  hipStream_t cs, xs;
  const int64_t* off;
  const int32_t *hsrc, *hrel, *hdst;
  std::vector<std::pair<int, int>> order;   // non-empty buckets
  // tables each of those buckets needs in a slot: table t * P + p, type 0's
  // partitions i and j without entity types, the swapped tables of the
  // bucket's relations with them
  std::vector<std::vector<int>> need;
  std::vector<void*> allocs;
  std::vector<hipEvent_t> evs;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> copy_spans;
  EdgeBuf eb[2];
  int64_t loads = 0;

  ~EpochRun() {
    for (auto& e : evs) (void)hipEventDestroy(e);
    for (void* p : allocs) (void)hipFree(p);
  }
  hipEvent_t new_event() {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    evs.push_back(e);
    return e;
  }
  int64_t rows(int tid) const { return table_rows(ctx, tid / ctx->P, tid % ctx->P); }

  int64_t next_use(int tid, size_t from) const {
    for (size_t t = from; t < order.size(); ++t)
      if (std::find(need[t].begin(), need[t].end(), tid) != need[t].end()) return (int64_t)t;
    return INT64_MAX;
  }
  int slot_of(int p) const {
    for (size_t v = 0; v < ctx->slots.size(); ++v)
      if (ctx->slots[v].part == p) return (int)v;
    return -1;
  }
  void span_begin(hipEvent_t& a) {
    a = new_event();
    if (a) (void)hipEventRecord(a, xs);
  }
  void span_end(hipEvent_t a) {
    hipEvent_t b = new_event();
    if (a && b) {
      (void)hipEventRecord(b, xs);
      copy_spans.push_back({a, b});
    }
  }

  // write the partition held by slot v back to its host arrays (copy stream)
  void write_back(int v) {
    Slot& s = ctx->slots[v];
    if (s.part < 0) return;
    if (s.used) (void)hipStreamWaitEvent(xs, s.released, 0);
    const Partition& hp = ctx->parts[s.part];
    const int64_t r = rows(s.part);
    (void)hipMemcpyAsync(hp.emb, s.emb, (size_t)r * ctx->d * 4, hipMemcpyDeviceToHost, xs);
    (void)hipMemcpyAsync(hp.G, s.G, (size_t)r * 4, hipMemcpyDeviceToHost, xs);
  }

  // brings partition p into a slot that holds none of `keep`; false when no
  // slot qualifies
  bool load(int p, size_t t_now, const std::vector<int>& keep) {
    int best = -1;
    int64_t best_next = -1;
    for (size_t v = 0; v < ctx->slots.size(); ++v) {
      const int q = ctx->slots[v].part;
      if (std::find(keep.begin(), keep.end(), q) != keep.end() && q >= 0) continue;
      const int64_t nu = q < 0 ? INT64_MAX : next_use(q, t_now);
      if (best < 0 || (q < 0 && ctx->slots[best].part >= 0) ||
          ((q < 0) == (ctx->slots[best].part < 0) && nu > best_next)) {
        best = (int)v;
        best_next = nu;
      }
    }
    if (best < 0) return false;
    Slot& s = ctx->slots[best];
    hipEvent_t a;
    span_begin(a);
    write_back(best);
    const Partition& hp = ctx->parts[p];
    const int64_t r = rows(p);
    (void)hipMemcpyAsync(s.emb, hp.emb, (size_t)r * ctx->d * 4, hipMemcpyHostToDevice, xs);
    (void)hipMemcpyAsync(s.G, hp.G, (size_t)r * 4, hipMemcpyHostToDevice, xs);
    (void)hipEventRecord(s.ready, xs);
    span_end(a);
    s.part = p;
    ++loads;
    return true;
  }

  // edges of bucket b into staging buffer k (copy stream)
  void stage_edges(int k, int b) {
    EdgeBuf& e = eb[k];
    if (e.used) (void)hipStreamWaitEvent(xs, e.consumed, 0);
    const int64_t lo = off[b], n = off[b + 1] - off[b];
    hipEvent_t a;
    span_begin(a);
    (void)hipMemcpyAsync(e.src, hsrc + lo, (size_t)n * 4, hipMemcpyHostToDevice, xs);
    (void)hipMemcpyAsync(e.dst, hdst + lo, (size_t)n * 4, hipMemcpyHostToDevice, xs);
    if (hrel) (void)hipMemcpyAsync(e.rel, hrel + lo, (size_t)n * 4, hipMemcpyHostToDevice, xs);
    (void)hipEventRecord(e.ready, xs);
    span_end(a);
    e.bucket = b;
  }
};

pbg_status ensure_slots(pbg_ctx* ctx, int count, int64_t cap) {
  bool ok = (int)ctx->slots.size() == count;
  for (auto& s : ctx->slots) ok = ok && s.rows_cap >= cap;
  if (ok) {
    for (auto& s : ctx->slots) {
      s.part = -1;
      s.used = false;
    }
    return PBG_OK;
  }
  (void)hipDeviceSynchronize();
  for (auto& s : ctx->slots) {
    if (s.emb) (void)hipFree(s.emb);
    if (s.ready) (void)hipEventDestroy(s.ready);
    if (s.released) (void)hipEventDestroy(s.released);
  }
  ctx->slots.assign(count, Slot());
  const size_t emb_bytes = ((size_t)cap * ctx->d * 4 + 255) & ~(size_t)255;
  for (auto& s : ctx->slots) {
    void* p = nullptr;
    if (hipMalloc(&p, emb_bytes + (size_t)cap * 4) != hipSuccess) {
      (void)hipGetLastError();
      return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "could not allocate %d HBM partition slots", count);
    }
    s.emb = (float*)p;
    s.G = (float*)((char*)p + emb_bytes);
    s.rows_cap = cap;
    if (hipEventCreateWithFlags(&s.ready, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&s.released, hipEventDisableTiming) != hipSuccess) {
      (void)hipGetLastError();
      return set_err(ctx, PBG_ERR_DEVICE, "hipEventCreate failed");
    }
  }
  return PBG_OK;
}

}  // namespace

extern "C" pbg_status pbg_train_epoch(pbg_ctx* ctx, const int64_t* offsets_host, const int32_t* src_local_host,
                                      const int32_t* rel_host, const int32_t* dst_local_host,
                                      const pbg_neg_config* neg, float lr, uint64_t seed, int32_t max_resident,
                                      double* loss_host) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  ctx->err.clear();
  const int P = ctx->P;
  if (!offsets_host) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL offsets");
  pbg_status st = check_neg_config(ctx, neg);
  if (st != PBG_OK) return st;
  if (neg->first_chunk != 0) return set_err(ctx, PBG_ERR_INVALID_ARG, "first_chunk must be 0 for an epoch");
  if (!std::isfinite(lr) || lr < 0.f) return set_err(ctx, PBG_ERR_INVALID_ARG, "lr must be finite and >= 0");
  if (max_resident < 2) return set_err(ctx, PBG_ERR_INVALID_ARG, "max_resident must be >= 2");
  const int32_t asked_slots = max_resident;
  max_resident = std::min(max_resident, P);
  if (max_resident < 2) max_resident = 2;
  const int nb = P * P;
  if (offsets_host[0] != 0) return set_err(ctx, PBG_ERR_INVALID_ARG, "offsets[0] must be 0");
  int64_t max_bucket = 0;
  for (int b = 0; b < nb; ++b) {
    const int64_t n = offsets_host[b + 1] - offsets_host[b];
    if (n < 0) return set_err(ctx, PBG_ERR_INVALID_ARG, "offsets must be non-decreasing");
    if (n > 0x7FFFFFFFll) return set_err(ctx, PBG_ERR_INVALID_ARG, "bucket %d has more than 2^31 - 1 edges", b);
    max_bucket = std::max(max_bucket, n);
  }
  const int64_t total = offsets_host[nb];
  if (total > 0 && (!src_local_host || !dst_local_host))
    return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL edge arrays");
  if (ctx->R > 1 && total > 0 && !rel_host)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "rel may be NULL only with one relation");
  const bool typed = ctx->T > 1;
  const int32_t* rel_used = ctx->R > 1 ? rel_host : nullptr;
  bool any_pinned = false;
  if (typed) {
    // entity types: every id, relation and bucket membership checked on the
    // host; tables bound in page-locked host memory are swapped through HBM
    // slots, tables in device memory are used in place
    st = validate_typed_epoch(ctx, offsets_host, src_local_host, rel_used, dst_local_host);
    if (st != PBG_OK) return st;
    for (int t = 0; t < ctx->T; ++t)
      for (int p = 0; p < (ctx->type_part[(size_t)t] ? P : 1); ++p)
        any_pinned = any_pinned || table_of(ctx, t, p).where == PBG_MEM_PINNED_HOST;
    if (!any_pinned) return train_epoch_typed(ctx, offsets_host, src_local_host, rel_used, dst_local_host, neg, lr,
                                              seed, loss_host);
  } else {
    for (int p = 0; p < P; ++p)
      if (!ctx->parts[p].emb || ctx->parts[p].where != PBG_MEM_PINNED_HOST)
        return set_err(ctx, PBG_ERR_STATE, "partition %d must be bound in page-locked host memory", p);
  }
  if (ctx->op != OP_IDENTITY && !ctx->relp) return set_err(ctx, PBG_ERR_STATE, "relation parameters are not bound");
  if (chunk_relation_operator(ctx) && !grouped_chunks(ctx, neg))
    return set_err(ctx, PBG_ERR_UNSUPPORTED,
                   "cos with an operator and several relations needs relation-grouped chunks (PBG_CHUNK_BY_RELATION)");
  if (grouped_chunks(ctx, neg) && rel_host) {
    // every bucket's edges sorted by relation, checked before anything trains
    for (int b = 0; b < nb; ++b)
      for (int64_t k = offsets_host[b] + 1; k < offsets_host[b + 1]; ++k)
        if (rel_host[k] < rel_host[k - 1])
          return set_err(ctx, PBG_ERR_INVALID_ARG,
                         "relation-grouped chunks need each bucket's edges sorted by relation (bucket %d)", b);
  }

  ctx->stats = pbg_stats();
  ctx->step_losses.clear();
  const auto t0 = std::chrono::steady_clock::now();
  if (!ctx->xs && !ctx->own_xs) {
    if (hipStreamCreateWithFlags(&ctx->own_xs, hipStreamNonBlocking) != hipSuccess) {
      (void)hipGetLastError();
      return set_err(ctx, PBG_ERR_DEVICE, "could not create a copy stream");
    }
  }
  EpochRun run;
  run.ctx = ctx;
  run.cs = ctx->cs;
  run.xs = ctx->xs ? ctx->xs : ctx->own_xs;
  run.off = offsets_host;
  run.hsrc = src_local_host;
  run.hrel = ctx->R > 1 ? rel_host : nullptr;
  run.hdst = dst_local_host;
  int64_t slot_rows = ctx->ps;   // rows a slot holds
  for (auto& bk : inside_out(P)) {
    const int b = bk.first * P + bk.second;
    if (offsets_host[b + 1] <= offsets_host[b]) continue;
    run.order.push_back(bk);
    std::vector<int> nd;
    if (!typed) {
      nd.push_back(bk.first);
      if (bk.second != bk.first) nd.push_back(bk.second);
    } else {
      // the swapped tables of the bucket's relations
      std::vector<char> seen((size_t)ctx->R, 0);
      for (int64_t k = offsets_host[b]; k < offsets_host[b + 1]; ++k) seen[(size_t)(rel_used ? rel_used[k] : 0)] = 1;
      for (int r = 0; r < ctx->R; ++r) {
        if (!seen[(size_t)r]) continue;
        for (int tid : {ctx->rel_st[(size_t)r] * P + bk.first, ctx->rel_dt[(size_t)r] * P + bk.second})
          if (ctx->parts[(size_t)tid].where == PBG_MEM_PINNED_HOST &&
              std::find(nd.begin(), nd.end(), tid) == nd.end())
            nd.push_back(tid);
      }
    }
    run.need.push_back(nd);
  }
  if (run.order.empty()) {
    if (loss_host) *loss_host = 0.0;
    return PBG_OK;
  }
  if (typed) {
    // slots: as many as asked for, at most one per swapped table, at least
    // the most tables one bucket needs; each as large as the largest one
    int swapped = 0;
    size_t most = 0;
    slot_rows = 0;
    for (int tid = 0; tid < ctx->T * P; ++tid)
      if (ctx->parts[(size_t)tid].where == PBG_MEM_PINNED_HOST) {
        ++swapped;
        slot_rows = std::max(slot_rows, run.rows(tid));
      }
    for (const auto& nd : run.need) most = std::max(most, nd.size());
    if ((size_t)asked_slots < most)
      return set_err(ctx, PBG_ERR_INVALID_ARG, "a bucket needs %d swapped tables at once; max_resident is %d",
                     (int)most, asked_slots);
    max_resident = std::max(1, std::min(asked_slots, swapped));
  }

  // staging buffers for two buckets' edges, and the id-check flag
  for (auto& e : run.eb) {
    for (int32_t** a : {&e.src, &e.dst, &e.rel}) {
      if (a == &e.rel && !run.hrel) continue;
      void* p = nullptr;
      if (hipMalloc(&p, std::max<size_t>((size_t)max_bucket * 4, 16)) != hipSuccess) {
        (void)hipGetLastError();
        return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "edge staging buffers could not be allocated");
      }
      run.allocs.push_back(p);
      *a = (int32_t*)p;
    }
    e.ready = run.new_event();
    e.consumed = run.new_event();
    if (!e.ready || !e.consumed) return set_err(ctx, PBG_ERR_DEVICE, "hipEventCreate failed");
  }
  void* flag_p = nullptr;
  if (hipMalloc(&flag_p, 16) != hipSuccess) {
    (void)hipGetLastError();
    return set_err(ctx, PBG_ERR_OUT_OF_MEMORY, "flag allocation failed");
  }
  run.allocs.push_back(flag_p);
  uint32_t* flag = (uint32_t*)flag_p;

  // every id is checked before any parameter changes (with entity types on
  // the host, above)
  hipError_t e = hipMemsetAsync(flag, 0, 4, run.xs);
  for (size_t t = 0; t < run.order.size() && e == hipSuccess && !typed; ++t) {
    const int i = run.order[t].first, j = run.order[t].second;
    const int b = i * P + j;
    const int k = (int)(t & 1);
    run.stage_edges(k, b);
    const int64_t n = offsets_host[b + 1] - offsets_host[b];
    launch_check_ids(run.eb[k].src, n, (int32_t)run.rows(i), flag, 1u, run.xs);
    launch_check_ids(run.eb[k].dst, n, (int32_t)run.rows(j), flag, 2u, run.xs);
    if (run.hrel) launch_check_ids(run.eb[k].rel, n, ctx->R, flag, 4u, run.xs);
    (void)hipEventRecord(run.eb[k].consumed, run.xs);
    run.eb[k].used = true;
    e = hipGetLastError();
  }
  uint32_t hflag = 0;
  if (e == hipSuccess) e = hipMemcpyAsync(&hflag, flag, 4, hipMemcpyDeviceToHost, run.xs);
  if (e == hipSuccess) e = hipStreamSynchronize(run.xs);
  if (e != hipSuccess) return hip_fail(ctx, e, "edge id check");
  if (hflag & 1u) return set_err(ctx, PBG_ERR_INVALID_ARG, "a source id is outside its partition");
  if (hflag & 2u) return set_err(ctx, PBG_ERR_INVALID_ARG, "a destination id is outside its partition");
  if (hflag & 4u) return set_err(ctx, PBG_ERR_INVALID_ARG, "a relation id is outside [0, %d)", ctx->R);
  run.copy_spans.clear();
  for (auto& eb : run.eb) {
    eb.used = false;
    eb.bucket = -1;
  }

  st = ensure_slots(ctx, max_resident, slot_rows);
  if (st != PBG_OK) return st;
  if (typed) ctx->table_override.assign((size_t)ctx->T * P, Partition());
  if (st != PBG_OK) return st;

  double total_loss = 0.0;
  const size_t T = run.order.size();
  for (size_t t = 0; t < T; ++t) {
    const int i = run.order[t].first, j = run.order[t].second;
    const int b = i * P + j;
    const int k = (int)(t & 1);
    const std::vector<int>& need = run.need[t];
    for (int p : need)
      if (run.slot_of(p) < 0 && !run.load(p, t, need))
        return set_err(ctx, PBG_ERR_STATE, "no free partition slot (max_resident %d)", max_resident);
    if (run.eb[k].bucket != b) run.stage_edges(k, b);
    // prefetch the next bucket while this one trains
    if (t + 1 < T) {
      const int i2 = run.order[t + 1].first, j2 = run.order[t + 1].second;
      run.stage_edges((int)((t + 1) & 1), i2 * P + j2);
      std::vector<int> keep = need;
      keep.insert(keep.end(), run.need[t + 1].begin(), run.need[t + 1].end());
      for (int p : run.need[t + 1])
        if (run.slot_of(p) < 0) run.load(p, t + 1, keep);
    }
    for (int p : need) (void)hipStreamWaitEvent(run.cs, ctx->slots[run.slot_of(p)].ready, 0);
    (void)hipStreamWaitEvent(run.cs, run.eb[k].ready, 0);
    const int64_t n = offsets_host[b + 1] - offsets_host[b];
    double loss = 0.0;
    if (typed) {
      // the bucket's swapped tables are read from their slots
      for (int p : need) {
        const Slot& sl = ctx->slots[run.slot_of(p)];
        Partition& ov = ctx->table_override[(size_t)p];
        ov.emb = sl.emb;
        ov.G = sl.G;
        ov.where = PBG_MEM_DEVICE;
      }
      st = train_bucket_typed(ctx, i, j, run.eb[k].src, run.hrel ? run.eb[k].rel : nullptr, run.eb[k].dst, n, neg, lr,
                              seed, &loss, &ctx->step_losses);
      for (int p : need) ctx->table_override[(size_t)p] = Partition();
    } else {
      const Slot& si = ctx->slots[run.slot_of(i)];
      const Slot& sj = ctx->slots[run.slot_of(j)];
      BucketTables tb;
      tb.emb_i = si.emb;
      tb.G_i = si.G;
      tb.emb_j = sj.emb;
      tb.G_j = sj.G;
      tb.rows_i = run.rows(i);
      tb.rows_j = run.rows(j);
      tb.same = i == j;
      st = train_bucket_device(ctx, i, j, tb, run.eb[k].src, run.hrel ? run.eb[k].rel : nullptr, run.eb[k].dst, n,
                               neg, lr, seed, &loss, &ctx->step_losses);
    }
    if (st != PBG_OK) {
      ctx->table_override.clear();
      return st;
    }
    total_loss += loss;
    for (int p : need) {
      Slot& sl = ctx->slots[run.slot_of(p)];
      (void)hipEventRecord(sl.released, run.cs);
      sl.used = true;
    }
    (void)hipEventRecord(run.eb[k].consumed, run.cs);
    run.eb[k].used = true;
  }
  for (size_t v = 0; v < ctx->slots.size(); ++v) {
    run.write_back((int)v);
    ctx->slots[v].part = -1;
    ctx->slots[v].used = false;
  }
  ctx->table_override.clear();
  e = hipGetLastError();
  if (e == hipSuccess) e = hipStreamSynchronize(run.xs);
  if (e == hipSuccess) e = hipStreamSynchronize(run.cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "partition transfers");
  double copy_ms = 0.0;
  for (auto& sp : run.copy_spans) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, sp.first, sp.second) == hipSuccess) copy_ms += ms;
  }
  (void)hipGetLastError();
  ctx->stats.copy_ms = copy_ms;
  ctx->stats.partition_loads = run.loads;
  ctx->stats.total_ms =
      std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
  if (loss_host) *loss_host = total_loss;
  return PBG_OK;
}
