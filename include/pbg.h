/*
 * pbg.h -- C ABI of the MI355X (gfx950) bucket-training library for
 * PyTorch-BigGraph-style multi-relation graph embeddings (Lerer et al.,
 * "PyTorch-BigGraph: A Large-scale Graph Embedding System", SysML 2019).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every function that can fail returns a pbg_status; PBG_OK is 0.  A failed
 *    call leaves a message behind for pbg_last_error(ctx).  Nothing aborts and
 *    no C++ exception crosses this boundary.
 *  - On any error no caller-owned parameter (embeddings, accumulators,
 *    relation parameters, outputs) has been modified: argument checks, and a
 *    device-side range check of every id, run before the first update.
 *  - All arrays are owned by the caller.  Unless its name ends in _host, an
 *    array is a device pointer on the device that was current when the context
 *    was created.  The library allocates only its own workspace (device memory
 *    for packed tiles, scores, sort buffers and partition slots), grows it on
 *    demand and frees it in pbg_free.
 *  - Work is enqueued on the caller's streams (pbg_set_streams; the null
 *    stream by default).  Every call is synchronous on return.  A context is
 *    not thread-safe; distinct contexts are independent.
 *  - Same inputs and the same chunks_per_step give bitwise-identical results:
 *    there are no floating-point atomics and every reduction has a fixed order.
 *  - Embedding tables are float32, row-major [rows x dim].  Ids are int32 local
 *    rows of a partition unless stated otherwise.
 */
#ifndef PBG_H
#define PBG_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PBG_OK = 0,
  PBG_ERR_INVALID_ARG = 1,   /* bad value, size, pointer or out-of-range id */
  PBG_ERR_UNSUPPORTED = 2,   /* a combination this version does not implement */
  PBG_ERR_OUT_OF_MEMORY = 3, /* workspace could not be allocated */
  PBG_ERR_DEVICE = 4,        /* a HIP runtime call failed */
  PBG_ERR_STATE = 5          /* wrong call order (e.g. an unbound partition) */
} pbg_status;

/* Relation operators g(x, theta_r) (Sec. 3.1, operator table):
 *  IDENTITY          g(x) = x                       (no relation parameters)
 *  TRANSLATION       g(x) = x + theta_r             (TransE; dim floats per relation)
 *  DIAGONAL          g(x) = x (.) theta_r           (DistMult; dim floats)
 *  LINEAR            g(x) = A_r x, A_r row-major    (RESCAL; dim*dim floats)
 *  COMPLEX_DIAGONAL  g(x) = x * theta_r over C^(dim/2), both stored as
 *                    [re(0..h-1) | im(0..h-1)]      (ComplEx; dim floats)
 * The operator acts on the source side; the destination is used as is. */
enum { PBG_OP_IDENTITY = 0, PBG_OP_TRANSLATION = 1, PBG_OP_DIAGONAL = 2,
       PBG_OP_LINEAR = 3, PBG_OP_COMPLEX_DIAGONAL = 4 };

/* Comparators sim(a, b) (Sec. 3.1): DOT <a, b> (for complex embeddings in the
 * split layout this is Re<a, conj(b)>); COS <a, b> / (max(|a|,1e-12) max(|b|,1e-12)). */
enum { PBG_CMP_DOT = 0, PBG_CMP_COS = 1 };

/* Losses per edge e and corruption side, over that side's valid negatives n_t
 * (Sec. 3.1; all summed over edges, sides and chunks):
 *  RANKING   sum_t max(0, margin - p_e + n_t)
 *  LOGISTIC  softplus(-p_e) + (1/K_e) sum_t softplus(n_t),  K_e = #valid negatives
 *  SOFTMAX   logsumexp({p_e} U {n_t}) - p_e */
enum { PBG_LOSS_RANKING = 0, PBG_LOSS_LOGISTIC = 1, PBG_LOSS_SOFTMAX = 2 };

/* Flags for pbg_bucket_init. */
enum {
  /* Round the inputs of the score and score-gradient contractions to bfloat16
   * (round to nearest even) and accumulate in float32; embeddings, Adagrad
   * state, losses and the loss epilogue stay float32. */
  PBG_F_BF16_SCORE = 1u,
  /* Record HIP events around every kernel group of every step on the compute
   * stream and report the summed times in pbg_stats (each event adds a few
   * microseconds to a step). */
  PBG_F_PHASE_TIMING = 2u,
  /* Record HIP events around the score contraction of every fourth step only
   * (score_ms and score_timed_steps in pbg_stats); PBG_F_PHASE_TIMING times
   * it on every step.  With bf16 score inputs the bracket holds the score
   * contraction alone, not the rounding of its operands. */
  PBG_F_SCORE_TIMING = 4u,
  /* Reciprocal predicates (Sec. 5.4: separate relation parameters for source
   * and destination negatives).  Relation r keeps a second parameter row
   * r + R.  The destination side scores sim(g(x_s, theta_r), x_t) as without
   * the flag; the source side scores sim(g(x_d, theta_{r+R}), x_t), with its
   * own positive sim(g(x_d, theta_{r+R}), x_s), so the operator never touches
   * a candidate.  The edge score f (pbg_score_edges) uses theta_r; the source
   * side of pbg_rank_eval / pbg_rank_sampled uses theta_{r+R}.  Every operator
   * and comparator works with any number of relations and either chunking. */
  PBG_F_RECIPROCAL = 8u
};

/* Where a bound partition lives. */
enum { PBG_MEM_DEVICE = 0, PBG_MEM_PINNED_HOST = 1 };

typedef struct pbg_ctx pbg_ctx;

/* Chunking of a call's edges (Sec. 4.3).
 *  CONSECUTIVE  chunk c holds edges [c*chunk_size, min((c+1)*chunk_size, n_edges))
 *               in the given order (relations may mix within a chunk);
 *  BY_RELATION  the edges must be sorted by relation (nondecreasing; e.g. by
 *               pbg_group_by_relation), and each relation's run of edges is
 *               cut into chunks of chunk_size, its last chunk holding the rest,
 *               so that every chunk holds one relation (Sec. 4.3: batches of
 *               edges that share their relation type).  With one relation the
 *               two are the same.  The cos comparator with an operator and
 *               several relations needs it (every source candidate of a chunk
 *               takes the operator of the chunk's relation). */
enum { PBG_CHUNK_CONSECUTIVE = 0, PBG_CHUNK_BY_RELATION = 1 };

/* Batched negatives (Sec. 4.3, Fig. 3).  The call's edges are cut into chunks
 * (see chunking); every edge of a chunk is scored against the chunk's other
 * edges' entities plus num_uniform entities drawn uniformly (separately per
 * side) from the partition of the corrupted side; the induced positive is
 * excluded.  A step of chunks_per_step consecutive chunks takes its gradient
 * at the step-start parameters and applies one Adagrad update.  first_chunk
 * numbers the first chunk of the call, so that a bucket may be trained in
 * several calls with the same negatives as one call (the uniform draws are
 * keyed by chunk number). */
typedef struct {
  int32_t chunk_size;       /* >= 1 */
  int32_t num_uniform;      /* >= 0; chunk_size + num_uniform >= 2 */
  int32_t chunks_per_step;  /* >= 1 (40 matches the paper's 40 training threads) */
  int32_t chunking;         /* PBG_CHUNK_CONSECUTIVE or PBG_CHUNK_BY_RELATION */
  int64_t first_chunk;      /* >= 0 */
} pbg_neg_config;

/* Timings and work of the last pbg_train_bucket / pbg_train_epoch call. */
typedef struct {
  int64_t edges;            /* edges trained */
  int64_t chunks;
  int64_t steps;
  double total_ms;          /* wall time of the call on the compute stream */
  /* per kernel group, summed over steps (only with PBG_F_PHASE_TIMING) */
  double gather_ms;         /* gather + operator + uniform draws */
  double score_ms;          /* score contraction with its fused loss epilogue */
  double epilogue_ms;       /* softmax row pass + per-edge finalisation */
  double backward_ms;       /* the two score-gradient contractions */
  double opbwd_ms;          /* operator / comparator backward */
  double update_ms;         /* sort + segment sums + Adagrad (entities and relations) */
  double gather_bytes;      /* algorithmic bytes of the gathers: (2C+2U)*dim*4 per chunk */
  double score_flops;       /* algorithmic flops of the three contractions: 12*C*N*dim per chunk */
  double update_bytes;      /* algorithmic bytes of the entity Adagrad updates: contribution rows
                               read ((2C+2U)*dim*4 per chunk), then per touched row its embedding
                               read and written and its Adagrad scalar read and written */
  double copy_ms;           /* partition / edge transfers (pbg_train_epoch) */
  int64_t partition_loads;  /* host-to-device partition loads (pbg_train_epoch) */
  int64_t score_timed_steps; /* steps whose score contraction score_ms sums */
} pbg_stats;

/* Creates a context for a graph of num_entities entities of one type split
 * into num_partitions contiguous ranges of ceil(n/P) ids, the last holding the
 * remainder (Sec. 4.1), num_relations relations, embedding dimension dim.
 * Returns INVALID_ARG for unknown enums, dim < 1 or dim > 512, odd dim with
 * COMPLEX_DIAGONAL, P < 1, a partition left empty, num_relations < 1 or a
 * non-finite margin.  Without PBG_F_RECIPROCAL: UNSUPPORTED for COS with the
 * LINEAR operator and more than one relation; COS with another operator and
 * several relations is trained with relation-grouped chunks only
 * (PBG_CHUNK_BY_RELATION; with consecutive chunks the training calls return
 * UNSUPPORTED: the source corruptions of an edge need its own relation's
 * operator applied to every candidate before the normalisation), and
 * pbg_rank_eval / pbg_rank_sampled return UNSUPPORTED for it.  With
 * PBG_F_RECIPROCAL none of these limits applies.  out NULL: INVALID_ARG and
 * nothing else.  On any other failure *out may still hold a context that only
 * carries the message: read it with pbg_last_error and release it with
 * pbg_free; every other call on it returns PBG_ERR_STATE (the row and size
 * queries return -1). */
pbg_status pbg_bucket_init(pbg_ctx** out, int64_t num_entities, int32_t num_partitions,
                           int32_t num_relations, int32_t dim, int32_t op, int32_t cmp,
                           int32_t loss, float margin, uint32_t flags);

/* Releases the context and its workspace (NULL is allowed).  Buffers bound
 * with pbg_bind_partition / pbg_bind_relations belong to the caller and may
 * be freed after this call (not before). */
void pbg_free(pbg_ctx* ctx);

/* Message of the last failed call on ctx ("" if none; a static message when
 * ctx is NULL).  Valid until the next call on ctx. */
const char* pbg_last_error(const pbg_ctx* ctx);

/* Rows of partition p (Sec. 4.1), or -1 for a bad p. */
int64_t pbg_partition_rows(const pbg_ctx* ctx, int32_t p);

/* Floats of all relation parameters: R*dim (translation, diagonal, complex),
 * R*dim*dim (linear) or 0 (identity); twice that with PBG_F_RECIPROCAL (rows
 * 0..R-1 for theta_r, rows R..2R-1 for the source side's theta_{r+R}). */
int64_t pbg_relation_param_floats(const pbg_ctx* ctx);

/* Edge bucketing (Sec. 4.1): edge (s, r, d) with global ids goes to bucket
 * b = part(s) * P + part(d).  Writes offsets[P*P+1] (device, int64; bucket b
 * holds positions [offsets[b], offsets[b+1])) and, in that order and stably
 * (input order inside each bucket), the local ids and relations.  rel may be
 * NULL (all relation 0; then rel_out may be NULL too).  Ids outside
 * [0, num_entities) or relations outside [0, R) give INVALID_ARG with no
 * output written.  n <= 2^31 - 1. */
pbg_status pbg_bucket_edges(pbg_ctx* ctx, const int64_t* src, const int32_t* rel,
                            const int64_t* dst, int64_t n, int64_t* offsets,
                            int32_t* src_local, int32_t* rel_out, int32_t* dst_local);

/* Binds partition p: emb [rows(p) x dim] float32 and its row-wise Adagrad
 * accumulator adagrad [rows(p)] float32 (one value per row, Sec. 3.1).  where
 * is PBG_MEM_DEVICE (device memory) or PBG_MEM_PINNED_HOST (page-locked host
 * memory, for pbg_train_epoch, which swaps partitions through HBM slots).
 * Initial values are the caller's; the library updates them in place.
 * Lifetime: the library keeps the two pointers, not copies of the data.  Both
 * buffers must stay allocated until the partition is bound again or the
 * context is released with pbg_free; freeing one earlier and then calling
 * any training, scoring or ranking entry point is undefined (the kernels
 * would read and write freed device memory).  Rebinding is allowed between
 * calls (every call is synchronous on return). */
pbg_status pbg_bind_partition(pbg_ctx* ctx, int32_t p, float* emb, float* adagrad, int32_t where);

/* Binds the relation parameters (device, [R x width] float32, or [2R x width]
 * with PBG_F_RECIPROCAL; width = dim, dim*dim for LINEAR) and their element-wise Adagrad accumulators
 * (same shape).  Not needed (and ignored) for IDENTITY.  Lifetime as for
 * pbg_bind_partition: both buffers must stay allocated until they are bound
 * again or pbg_free. */
pbg_status pbg_bind_relations(pbg_ctx* ctx, float* params, float* adagrad);

/* Streams (hipStream_t) for compute and for partition transfers.  NULL means
 * the null stream.  Streams must have the default priority. */
pbg_status pbg_set_streams(pbg_ctx* ctx, void* compute_stream, void* copy_stream);

/* One training pass over the edges of bucket (i, j) (Sec. 3.1 model and loss,
 * Sec. 4.1 bucket, Sec. 4.3 batched negatives; Adagrad with the accumulator
 * summed over each embedding row).  src_local / dst_local are int32 rows of
 * partitions i / j (device), rel is int32 in [0, R) or NULL when R == 1.
 * Uniform negative k of chunk c and side sigma (0: destinations, drawn from
 * partition j; 1: sources, drawn from partition i) is
 * floor(w * rows / 2^32) with w = word (k mod 4) of
 * Philox4x32-10(counter = (k / 4, c, i*P + j, sigma), key = (seed low 32 bits,
 * seed high 32 bits)).  Each step applies
 *   G_row += |g_row|^2 ;  theta_row -= lr * g_row / (sqrt(G_row) + 1e-10)
 * to every entity row it touches (g summed over the step) and the element-wise
 * form to relation parameters.  Partitions i and j must be bound in device
 * memory.  loss_host (nullable) receives the summed loss of the call. */
pbg_status pbg_train_bucket(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src_local,
                            const int32_t* rel, const int32_t* dst_local, int64_t n_edges,
                            const pbg_neg_config* neg, float lr, uint64_t seed,
                            double* loss_host);

/* Entity types (Sec. 3.1: negatives only from the entity type of the edge's
 * relation; Sec. 4.1 and Fig. 1 centre: a small type may stay unpartitioned).
 * Replaces the single type of pbg_bucket_init with num_types types: type t
 * has type_entities[t] entities (host int64) and is split into the context's
 * P contiguous partitions when type_partitioned[t] != 0, else kept whole in
 * one table at partition 0.  Relation r goes from type rel_src_type[r] to
 * type rel_dst_type[r] (host int32, R entries).  Ids of entities are per type.
 * Every table is unbound afterwards (bind them with pbg_bind_type_partition);
 * call it before any training.  INVALID_ARG for num_types outside [1, 4096],
 * a type without entities or with an empty partition, or a relation naming a
 * type outside [0, num_types).
 * With several types:
 *  - pbg_bucket_edges takes per-type ids; edge (s, r, d) goes to bucket
 *    (partition of s in its type, partition of d in its type), 0 for a whole
 *    type (so with every destination type whole only the P buckets (i, 0)
 *    have edges);
 *  - pbg_train_bucket on bucket (i, j) takes the bucket's edges sorted by
 *    relation (PBG_CHUNK_BY_RELATION when R > 1) and trains them in runs of
 *    consecutive relations that share a (source type, destination type):
 *    each run's chunks score against, and draw their uniform negatives from,
 *    table (source type, i) and table (destination type, j); steps never span
 *    two runs; chunk numbers continue across runs.  Each run's ids are
 *    checked against its tables before anything trains;
 *  - pbg_train_epoch takes each table where it is bound: tables in device
 *    memory are used in place, tables in page-locked host memory are swapped
 *    through at most max_resident HBM slots (at least as many as the swapped
 *    tables one bucket needs at once, else INVALID_ARG); all ids are checked
 *    on the host first;
 *  - pbg_inspect_step takes edges of one run;
 *  - pbg_score_edges, pbg_score_edges_noalloc, pbg_rank_eval and
 *    pbg_rank_sampled return UNSUPPORTED;
 *  - pbg_bind_partition, pbg_partition_rows and pbg_sample_negatives refer to
 *    type 0. */
pbg_status pbg_set_entity_types(pbg_ctx* ctx, int32_t num_types, const int64_t* type_entities,
                                const int32_t* type_partitioned, const int32_t* rel_src_type,
                                const int32_t* rel_dst_type);

/* Binds table (type t, partition p) as pbg_bind_partition binds a partition
 * (rows: pbg_type_partition_rows).  INVALID_ARG for a table that does not
 * exist (p > 0 of a whole type). */
pbg_status pbg_bind_type_partition(pbg_ctx* ctx, int32_t t, int32_t p, float* emb, float* adagrad, int32_t where);

/* Rows of table (type t, partition p), or -1 when it does not exist. */
int64_t pbg_type_partition_rows(const pbg_ctx* ctx, int32_t t, int32_t p);

/* Per-relation edge weights (Sec. 1 and 6: per-relation configuration):
 * weights_host[r] (host float32, R entries, finite and >= 0) multiplies the
 * loss of every edge of relation r on both sides, and so its gradients.
 * NULL restores weight 1 for every relation.  The weight is applied per
 * chunk, so a training call whose chunks may mix relations of different
 * weights (consecutive chunks with R > 1) returns UNSUPPORTED unless all
 * weights are equal.  The training calls' losses include the weights;
 * pbg_inspect_step reports the unweighted loss (loss_host, row_loss, dscores). */
pbg_status pbg_set_relation_weights(pbg_ctx* ctx, const float* weights_host);

/* Relation-grouped order of a bucket's edges (Sec. 4.3): writes the n edges
 * (src, rel, dst: device int32) stably sorted by relation to src_out,
 * rel_out, dst_out (device int32, not overlapping the inputs), the order that
 * PBG_CHUNK_BY_RELATION takes.  Relations outside [0, R) give INVALID_ARG with
 * nothing written. */
pbg_status pbg_group_by_relation(pbg_ctx* ctx, const int32_t* src, const int32_t* rel, const int32_t* dst,
                                 int64_t n, int32_t* src_out, int32_t* rel_out, int32_t* dst_out);

/* Per-step losses of the last pbg_train_bucket call: copies
 * min(capacity, steps) values to out_host and the step count to n_steps_host. */
pbg_status pbg_get_step_losses(const pbg_ctx* ctx, double* out_host, int64_t capacity,
                               int64_t* n_steps_host);

/* One epoch over all buckets in inside-out order (Sec. 4.1, Fig. 1 right):
 * (0,0), then for k = 1..P-1: (k,0),(0,k),(k,1),(1,k),...,(k,k-1),(k-1,k),(k,k);
 * empty buckets are skipped.  Edges are bucketed (pbg_bucket_edges layout) in
 * page-locked host memory; offsets_host [P*P+1] is host memory.  Every
 * partition must be bound as PBG_MEM_PINNED_HOST: at most max_resident (>= 2)
 * partitions are held in HBM slots at a time, loaded and written back on the
 * copy stream, ordered with events against the compute stream.  On return the
 * host partitions hold the trained values.  Each bucket is trained as by
 * pbg_train_bucket with first_chunk 0 and the given seed. */
pbg_status pbg_train_epoch(pbg_ctx* ctx, const int64_t* offsets_host,
                           const int32_t* src_local_host, const int32_t* rel_host,
                           const int32_t* dst_local_host, const pbg_neg_config* neg,
                           float lr, uint64_t seed, int32_t max_resident, double* loss_host);

/* Scores f(s, r, d) = sim(g(theta_s, theta_r), theta_d) of n edges of bucket
 * (i, j) (Sec. 3.1), computed as in training; scores is float32 [n] (device). */
pbg_status pbg_score_edges(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src_local,
                           const int32_t* rel, const int32_t* dst_local, int64_t n,
                           float* scores);

/* Filtered link-prediction ranks (Sec. 5, filtered protocol of the FB15k
 * experiments): for each triple (s, r, d), its destination rank
 * 1 + #{d' != d : (s, r, d') not known, f(s, r, d') >= f(s, r, d)} among all
 * entities, then its source rank symmetrically.  ranks is int32 [2n] (device):
 * destination ranks first, then source ranks.  The known triples (device,
 * duplicates allowed) are the filter.  mrr_host / hits10_host (nullable)
 * receive the mean of 1/rank and of [rank <= 10] over the 2n ranks.  Only for
 * P == 1 (else UNSUPPORTED). */
pbg_status pbg_rank_eval(pbg_ctx* ctx, const int32_t* src, const int32_t* rel, const int32_t* dst,
                         int64_t n, const int32_t* known_src, const int32_t* known_rel,
                         const int32_t* known_dst, int64_t n_known, int32_t* ranks,
                         double* mrr_host, double* hits10_host);

/* Raw link-prediction ranks against a given candidate set (Sec. 5, Freebase
 * evaluation: for graphs too large to rank against every entity, each eval
 * edge is ranked against candidate nodes sampled by their prevalence in the
 * training data; the caller draws the candidates and passes their ids).
 * For each triple (s, r, d): destination rank
 * 1 + #{j : cand[j] != d, f(s, r, cand[j]) >= f(s, r, d)}, then source rank
 * 1 + #{j : cand[j] != s, f(cand[j], r, d) >= f(s, r, d)}; no filter, and a
 * candidate listed k times counts k times.  The same n_cand candidates
 * (device int32, entity ids of partition 0) serve every triple and both
 * sides.  ranks is int32 [2n] (device): destination ranks first.  mrr_host /
 * hits10_host (nullable) as for pbg_rank_eval.  Only for P == 1 (else
 * UNSUPPORTED); an id out of range is INVALID_ARG and nothing is written. */
pbg_status pbg_rank_sampled(pbg_ctx* ctx, const int32_t* src, const int32_t* rel, const int32_t* dst,
                            int64_t n, const int32_t* cand, int64_t n_cand, int32_t* ranks,
                            double* mrr_host, double* hits10_host);

/* The uniform negatives pbg_train_bucket draws (Sec. 4.3; Philox map as
 * described there) for chunks first_chunk .. first_chunk + n_chunks - 1 of
 * bucket (i, j): out (device, int32) is [n_chunks][2][num_uniform], side 0
 * (destinations, rows of partition j) then side 1 (sources, partition i).
 * Produced by the same device code as training; for inspection and tests. */
pbg_status pbg_sample_negatives(pbg_ctx* ctx, int32_t i, int32_t j, int64_t first_chunk,
                                int64_t n_chunks, int32_t num_uniform, uint64_t seed, int32_t* out);

/* Inspection of one step (for tests and diagnostics): runs the forward half
 * of a training step on the n_edges <= chunk_size * chunks_per_step edges of
 * bucket (i, j) -- gather, relation operator, uniform draws of chunks
 * neg->first_chunk onwards, the chunk score contraction with its loss
 * epilogue and the per-edge finalisation (Sec. 3.1 score f and losses,
 * Sec. 4.3 batched negatives) -- with the same kernels and launch sequence as
 * pbg_train_bucket, then copies out what they computed.  No parameter or
 * accumulator is modified; arguments and ids are checked as for
 * pbg_train_bucket.  With nch the number of chunks of the call (at most
 * chunks_per_step; ceil(n_edges / chunk_size) for consecutive chunks), N = chunk_size +
 * num_uniform, Cc the edges of chunk c and candidates t = the chunk's Cc
 * in-chunk entities followed by its num_uniform draws, every output is a
 * nullable device float32 array whose entries outside [Cc] x [Cc + U] are 0:
 *   scores    [nch][2][chunk_size][N]: side 0 f(s_e, r_e, candidate t of the
 *             destination side), side 1 f(candidate t of the source side,
 *             r_e, d_e), from the score contraction's main loop over the same
 *             operands with a plain store epilogue (so the values the loss
 *             epilogue saw, up to the bias it adds the same way);
 *   dscores   [nch][2][chunk_size][N]: dL/dS as the epilogue left it (0 on the
 *             excluded induced positive);
 *   row_loss  [nch][2][chunk_size]: each edge's loss on each side;
 *   pos       [nch][chunk_size]: the positive scores p_e; with
 *             PBG_F_RECIPROCAL [nch][2][chunk_size], each side's own positive.
 * loss_host (nullable) receives the summed loss of the step. */
pbg_status pbg_inspect_step(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src_local,
                            const int32_t* rel, const int32_t* dst_local, int64_t n_edges,
                            const pbg_neg_config* neg, uint64_t seed, float* scores, float* dscores,
                            float* row_loss, float* pos, double* loss_host);

/* Largest relation parameter count (R * dim * dim floats, the linear
 * operator only) that pbg_score_edges_noalloc accepts. */
#define PBG_NOALLOC_MAX_REL_FLOATS (2 * 1024 * 1024)

/* pbg_score_edges for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * Same arguments, results and errors as pbg_score_edges, computed by the same
 * kernels; the scratch that pbg_score_edges allocates per call (the id-check
 * flag and, for LINEAR, a transposed copy of the relation matrices) is a
 * static device array of the library instead, 8 MiB + 256 bytes, held on
 * each device the library runs on until the process ends.  INVALID_ARG when
 * the operator is LINEAR and R * dim * dim exceeds
 * PBG_NOALLOC_MAX_REL_FLOATS.  The context's device must be current.  All
 * calls on one device share that device's array: calls that overlap on one
 * device (several host threads, or several streams in flight) race. */
pbg_status pbg_score_edges_noalloc(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src_local,
                                   const int32_t* rel, const int32_t* dst_local, int64_t n, float* scores);

/* Timings and algorithmic work of the last training call. */
pbg_status pbg_get_stats(const pbg_ctx* ctx, pbg_stats* out_host);

#ifdef __cplusplus
}
#endif

#endif /* PBG_H */
