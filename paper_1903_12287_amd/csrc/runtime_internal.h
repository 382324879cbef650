// Internal state of a context (host side).
#pragma once

#include <hip/hip_runtime.h>

#include <functional>
#include <string>
#include <vector>

#include "kernels.h"
#include "pbg.h"

struct Partition {
  float* emb = nullptr;  // [rows x dim]
  float* G = nullptr;    // [rows]
  int where = -1;        // PBG_MEM_DEVICE / PBG_MEM_PINNED_HOST
};

// device allocations owned by the library, released together
struct Arena {
  std::vector<void*> ptrs;
  bool failed = false;
  void* get(size_t bytes);
  void release();
};

// an HBM slot holding one partition during pbg_train_epoch: the embedding rows
// followed by the row-wise Adagrad accumulator, in one allocation
struct Slot {
  float* emb = nullptr;
  float* G = nullptr;
  int64_t rows_cap = 0;
  int part = -1;
  hipEvent_t ready = nullptr;     // load finished (copy stream)
  hipEvent_t released = nullptr;  // last use finished (compute stream)
  bool used = false;              // `released` has been recorded
};

// bf16 operand copies of a step (PBG_F_BF16_SCORE)
struct BufsH {
  uint16_t* qk = nullptr;   // [S][2][C][dpb]
  uint16_t* nn = nullptr;   // [S][2][N][dpb]
  uint16_t* qkT = nullptr;  // [S][2][dpb][Cpb]
  uint16_t* nnT = nullptr;  // [S][2][dpb][Npb]
  uint16_t* ds = nullptr;   // [S][2][C][Npb] dS rows (logistic, softmax)
  // float32 ranking backward: the exact three-piece split of Q^T and N^T,
  // [3][S][2][dpb][Cpb] and [3][S][2][dpb][Npb], planes q3_ps / n3_ps apart
  uint16_t* qkT3 = nullptr;
  uint16_t* nnT3 = nullptr;
  int64_t q3_ps = 0, n3_ps = 0;
};

struct pbg_ctx {
  int64_t n = 0;                   // entities of type 0 (the only type without pbg_set_entity_types)
  int P = 1, R = 1, d = 1, op = 0, cmp = 0, loss = 0;
  float margin = 0.f;
  uint32_t flags = 0;
  int64_t ps = 0;
  int dr = 0;
  int device = 0;
  bool invalid = false;
  hipStream_t cs = nullptr;  // compute stream
  hipStream_t xs = nullptr;  // copy stream
  std::vector<Partition> parts;    // table (type t, partition p) at t * P + p
  // during a typed epoch: the HBM slot standing in for a swapped table (emb
  // NULL: none), same indexing
  std::vector<Partition> table_override;
  // entity types (Sec. 3.1, Sec. 4.1): entities per type, whether a type is
  // split into P partitions (else one table at partition 0), and the source
  // and destination type of every relation
  int T = 1;
  std::vector<int64_t> type_n;
  std::vector<int> type_part;
  std::vector<int> rel_st, rel_dt;
  // per-relation edge weights (empty: every weight 1), and the weights of the
  // current call's chunks on the device
  std::vector<float> relw;
  float* cweight_dev = nullptr;
  int64_t cweight_cap = 0;
  float* relp = nullptr;
  float* relG = nullptr;
  std::string err;

  // training workspace
  Arena ws;
  bool ws_ready = false;
  int wC = 0, wU = 0, wS = 0;
  StepBufs bufs{};
  BufsH h{};
  SortWork sw{};
  // sort keys / values of a window of steps ([kSortWindow][2 S N]) and the
  // alternate buffers and digit counts of their batched sort
  uint32_t* wkeys_alt = nullptr;
  uint32_t* wvals_alt = nullptr;
  uint32_t* whist = nullptr;
  float* relpartial = nullptr;
  float* relA = nullptr;    // linear operator: A and A^T, rows padded to dp
  float* relAT = nullptr;
  uint32_t* flag_dev = nullptr;
  uint32_t* hflag = nullptr;          // page-locked copy of the id check's flags
  hipEvent_t check_ev = nullptr;      // the copy has landed
  bool check_pending = false;
  double* steploss_dev = nullptr;
  int64_t steploss_cap = 0;
  // the finalisation's loss partials of every step of a call, lossparts_pps
  // apart (added up per step after the call's last step)
  double* lossparts = nullptr;
  int64_t lossparts_cap = 0, lossparts_pps = 0;
  // relation-grouped chunks of the current call: bounds in the call's edge
  // arrays (host copy and device copy)
  std::vector<int32_t> cstart_host;
  std::vector<int32_t> crel_host;  // the relation of each of those chunks
  int32_t* cstart_dev = nullptr;
  int64_t cstart_cap = 0;

  std::vector<double> step_losses;
  pbg_stats stats{};
  std::vector<Slot> slots;
  hipStream_t own_xs = nullptr;    // copy stream created for pbg_train_epoch when none was given
  std::vector<hipEvent_t> events;  // phase-timing events, kPhaseEvents per step
};

constexpr int kPhaseEvents = 7;
// score-only timing brackets every kScoreSample-th step (each event record
// costs the compute stream a few microseconds)
constexpr int kScoreSample = 4;
// steps whose entity sort keys are built and sorted together, as one batch
constexpr int kSortWindow = 32;

pbg_status set_err(pbg_ctx* ctx, pbg_status st, const char* fmt, ...);
// device address of the static scratch of pbg_score_edges_noalloc on the
// context's device (taken once per device; called by pbg_bucket_init)
pbg_status noalloc_scratch_init(pbg_ctx* ctx);

// the three contractions of step t (forward_only: the score contraction with
// its loss epilogue and the per-edge finalisation only)
void run_contractions_f32(pbg_ctx* ctx, const StepGeom& g, const StepBufs& b, int64_t t, hipStream_t cs,
                          const std::function<void(int)>& mark, bool forward_only);
void run_contractions_bf16(pbg_ctx* ctx, const StepGeom& g, const StepBufs& b, int64_t t,
                           hipStream_t cs, const std::function<void(int)>& mark, bool forward_only);
void run_score_store(pbg_ctx* ctx, const StepGeom& g, const StepBufs& b, float* out, hipStream_t cs);
// the linear operator with one relation, as contractions over the step (A
// and A^T row-padded in Ap / ATp)
void run_linear_forward(const StepGeom& g, const StepBufs& b, const float* Ap, const float* ATp, hipStream_t cs);
void run_linear_backward(const StepGeom& g, const StepBufs& b, const float* Ap, const float* ATp,
                         hipStream_t cs);
int run_linear_relation_grad(const StepGeom& g, const StepBufs& b, float* partial, hipStream_t cs);
// gather + relation operator + uniform draws of a step (with the linear
// operator's products)
void run_gather_forward(pbg_ctx* ctx, const StepGeom& g, const StepBufs& b, hipStream_t cs);
pbg_status hip_fail(pbg_ctx* ctx, hipError_t e, const char* what);
bool alloc_sortwork(Arena& a, SortWork& w, int64_t max_n, int width);
pbg_status check_neg_config(pbg_ctx* ctx, const pbg_neg_config* neg);
// the argument and state checks of a training call on bucket (i, j), then the
// device-side range check of every id (nothing is modified on failure)
pbg_status check_bucket_call(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src_local,
                             const int32_t* rel, const int32_t* dst_local, int64_t n_edges,
                             const pbg_neg_config* neg,
                             bool defer = false);
// the id range check's verdict (waits for it); with defer the check above only
// launches it, and the caller finishes it once it has queued work that needs
// no valid ids (check_pending)
pbg_status finish_id_check(pbg_ctx* ctx, int32_t i, int32_t j);
pbg_status ensure_workspace(pbg_ctx* ctx, int C, int U, int S);
// chunk bounds of a call's edges for PBG_CHUNK_BY_RELATION (rel: device, n
// edges sorted by relation): ctx->cstart_host / cstart_dev; INVALID_ARG when
// the relations are not in nondecreasing order
pbg_status relation_chunk_bounds(pbg_ctx* ctx, const int32_t* rel, int64_t n, int C);
// the call's chunks are relation-grouped (PBG_CHUNK_BY_RELATION with several
// relations; with one relation both chunkings are the same)
inline bool grouped_chunks(const pbg_ctx* ctx, const pbg_neg_config* neg) {
  return neg->chunking == PBG_CHUNK_BY_RELATION && ctx->R > 1;
}
inline bool reciprocal(const pbg_ctx* ctx) { return (ctx->flags & PBG_F_RECIPROCAL) != 0; }
// relation parameter rows (R, or 2R with reciprocal predicates)
inline int relation_rows(const pbg_ctx* ctx) { return reciprocal(ctx) ? 2 * ctx->R : ctx->R; }
// the cos comparator with an operator and several relations applies each
// chunk's relation to its source candidates: relation-grouped chunks only
// (not with reciprocal predicates, where no candidate carries the operator)
inline bool chunk_relation_operator(const pbg_ctx* ctx) {
  return ctx->cmp == PBG_CMP_COS && ctx->op != PBG_OP_IDENTITY && ctx->R > 1 && !reciprocal(ctx);
}
// relation gradients summed through sorted relation keys (more than one
// parameter row), not by the single-relation sums
inline bool sorted_relation_keys(const pbg_ctx* ctx) {
  return ctx->op != PBG_OP_IDENTITY && relation_rows(ctx) > 1;
}
// one relation operator with a parameter row (translation, diagonal, complex
// diagonal; no reciprocal predicates): the operator backward adds each
// block's parameter-gradient rows, and the fixed-order sum of those rows and
// the element-wise Adagrad step follow it
inline bool single_relation_sums(const pbg_ctx* ctx) {
  return ctx->op != PBG_OP_IDENTITY && ctx->op != PBG_OP_LINEAR && !sorted_relation_keys(ctx);
}
// The float32 ranking backward with the queries as candidate rows (QK_IN_NN)
// merges dN rows e < Cc of one side into dQ of the other (kernels.h, merge_cc).
inline bool merged_ranking_backward(const pbg_ctx* ctx, const StepGeom& g) {
  return QK_IN_NN(g) && g.loss == LOSS_RANKING && !(ctx->flags & PBG_F_BF16_SCORE);
}
// the linear operator as contractions over the whole step (one relation
// matrix); otherwise one matrix-vector product per edge
inline bool linear_step_contractions(const pbg_ctx* ctx) {
  return ctx->op == PBG_OP_LINEAR && relation_rows(ctx) == 1;
}
pbg_status ensure_steploss(pbg_ctx* ctx, int64_t nsteps);
// room for nsteps steps of pps loss partials each (sets lossparts_pps)
pbg_status ensure_lossparts(pbg_ctx* ctx, int64_t nsteps, int64_t pps);

// rows of table (type t, partition p), or -1
int64_t table_rows(const pbg_ctx* ctx, int t, int p);
inline Partition& table_of(pbg_ctx* ctx, int t, int p) { return ctx->parts[(size_t)t * ctx->P + p]; }
// the table training reads: its HBM slot during a typed epoch, else as bound
inline Partition resolve_table(const pbg_ctx* ctx, int t, int p) {
  const size_t k = (size_t)t * ctx->P + p;
  if (k < ctx->table_override.size() && ctx->table_override[k].emb) return ctx->table_override[k];
  return ctx->parts[k];
}
// the source and destination tables of a bucket's edges (one run of the
// call: a single (source type, destination type) pair)
struct BucketTables {
  float* emb_i = nullptr;
  float* G_i = nullptr;
  float* emb_j = nullptr;
  float* G_j = nullptr;
  int64_t rows_i = 0, rows_j = 0;
  bool same = false;   // one table serves both sides
};
// partitions i and j of type 0
BucketTables partition_tables(pbg_ctx* ctx, int32_t i, int32_t j);
// geometry of the steps of bucket (i, j) (chunk and candidate counts, padded
// strides, table rows, key widths) and the step buffers bound to the given
// tables and the context's workspace
void bucket_geom(const pbg_ctx* ctx, int32_t i, int32_t j, const BucketTables& tb, int C, int U, uint64_t seed,
                 StepGeom& g);
StepBufs bucket_bufs(pbg_ctx* ctx, const BucketTables& tb);
pbg_status train_bucket_device(pbg_ctx* ctx, int32_t i, int32_t j, const BucketTables& tb, const int32_t* src,
                               const int32_t* rel, const int32_t* dst, int64_t n_edges, const pbg_neg_config* neg,
                               float lr, uint64_t seed, double* loss_out, std::vector<double>* step_losses);
// relation weights of the call's chunks into ctx->cweight_dev (NULL when no
// weights are set); UNSUPPORTED when consecutive chunks would mix relations of
// different weights.  Needs ctx->crel_host for relation-grouped chunks.
pbg_status chunk_weights(pbg_ctx* ctx, bool grouped, int64_t nchunks, const float** out);
// typed contexts: the runs of a call and their training (pbg_types.cpp)
pbg_status train_bucket_typed(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src, const int32_t* rel,
                              const int32_t* dst, int64_t n_edges, const pbg_neg_config* neg, float lr, uint64_t seed,
                              double* loss_out, std::vector<double>* step_losses);
// the tables of a typed call whose edges form one run (pbg_inspect_step)
pbg_status typed_single_run(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src, const int32_t* rel,
                            const int32_t* dst, int64_t n_edges, const pbg_neg_config* neg, BucketTables* tb);
// host checks of a typed epoch's edges (ids, relations, order, bucket
// membership); then the epoch with every table in device memory
pbg_status validate_typed_epoch(pbg_ctx* ctx, const int64_t* offsets_host, const int32_t* src_host,
                                const int32_t* rel_host, const int32_t* dst_host);
pbg_status train_epoch_typed(pbg_ctx* ctx, const int64_t* offsets_host, const int32_t* src_host,
                             const int32_t* rel_host, const int32_t* dst_host, const pbg_neg_config* neg, float lr,
                             uint64_t seed, double* loss_host);
pbg_status bucket_edges_typed(pbg_ctx* ctx, const int64_t* src, const int32_t* rel, const int64_t* dst, int64_t n,
                              int64_t* offsets, int32_t* src_local, int32_t* rel_out, int32_t* dst_local);
