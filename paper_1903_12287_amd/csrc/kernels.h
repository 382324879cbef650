// Launch entry points of the gfx950 kernels (host side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "geometry.h"

// ---- matrix-core contractions -------------------------------------------------
// EPI_LOSS_BITS: ranking loss with dS (0 or 1) written as bits, 16 columns per
// uint16 word, word (w, row) at dsb[w * ldcb + row] (nwcb words per row; batch
// strides cb_cs / cb_ss in words)
enum { EPI_STORE = 0, EPI_LOSS = 1, EPI_SOFTMAX_STATS = 2, EPI_LOSS_BITS = 3, EPI_SOFTMAX_EXP = 4 };
enum { DIM_CC = 0, DIM_NC = 1, DIM_FIXED = 2 };
// float32 operand layouts: NT  A[m][k], B[n][k];  TN  A[k][m], B[k][n]
enum { GEMM_NT = 0, GEMM_TN = 2 };

struct GemmArgs {
  const float* A;
  const float* B;
  float* Cm;
  int64_t a_cs, a_ss, b_cs, b_ss, c_cs, c_ss;  // strides (floats) per chunk and per side
  int lda, ldb, ldc;
  int mdim, ndim, kdim;  // DIM_* selectors
  int Mfix, Nfix, Kfix;
  int C, U, m_step;      // chunk geometry (m_step = 0: not chunked)
  const int32_t* cstart; // relation-grouped chunks: chunk c holds cstart[c + 1] - cstart[c] edges
  int nsides;            // batches per chunk
  int accumulate;        // add to C instead of overwriting it
};

// float32 contraction C = A . B (or C += A . B) of `batches` (chunk, side)
// pairs; the tiling and grid follow from the largest M and N of the batches
void launch_gemm_f32(const GemmArgs& a, int layout, int batches, hipStream_t s);

// bf16 contractions, fp32 accumulation.  B is bf16 [n][k] (k contiguous,
// zero-padded to 8); A is one of
enum {
  GA_KC = 0,        // bf16 [m][k], k contiguous
  GA_MC = 1,        // bf16 [k][m], m contiguous
  GA_BITS_ROW = 2,  // the ranking dS bit matrix (dsb layout), A[m][k] = bit (row m, column k)
  GA_BITS_COL = 3   // the same matrix transposed: A[m][k] = bit (row k, column m)
};
struct GemmArgsH {
  const uint16_t* A;
  const uint16_t* B;     // planes pieces of B, b_ps elements apart
  int planes;            // 1, or 3: the exact bf16 pieces of a float32 operand (A = bit matrix only)
  int64_t b_ps;
  const float* Af;       // launch_score_split: float32 operands [m][k] and [n][k]
  const float* Bf;
  const float* smscale;  // launch_gemm_split_pair: Af holds exp(s - tile max) of the softmax loss and
                         // smscale[(z * nct + tile) * C + row] = exp(tile max - lse) (z = chunk*2 + side)
  float* Cm;             // fp32 output (STORE, SOFTMAX_STATS)
  uint16_t* dsh;         // EPI_LOSS: dS rows in bf16 (strides c_*, ldc)
  uint16_t* dsb;         // EPI_LOSS_BITS output (as in GemmArgs)
  int64_t cb_cs, cb_ss;
  int ldcb, nwcb;
  int64_t a_cs, a_ss, b_cs, b_ss, c_cs, c_ss;
  int lda, ldb, ldc;     // in elements (bf16 or float), or words for a bit matrix
  int amode;             // GA_*
  int mdim, ndim, kdim;
  int Mfix, Nfix, Kfix;
  int C, U, m_step;
  const int32_t* cstart;
  int nsides;
  const float* pos;      // positive scores [c][C], or [c][2][C] with pos_sides = 2
  int pos_sides;         // 2: one positive score per side (reciprocal predicates)
  const float* bias;
  float* rowpart;
  int nct;
  int loss;
  float margin;
  const float* cscale;   // EPI_STORE: output of chunk c times cscale[c] (NULL: as is)
  int share_cc;          // launch_score_split with Q of each side the first C candidate rows of the
                         // other: the in-chunk block of side 1 is the transpose of side 0's, and side 0's
                         // full tiles inside it produce side 1's too
  int merge_cc;          // ranking backward with the same Q / candidate rows (launch_gemm_bf16_pair, three
                         // planes): a0's dQ rows e < Cc of side s also take dN of candidate e of side 1 - s
                         // (the same vector; a0.A's other side read by columns over k < Cc), and a1's dN rows
                         // start at Cc rounded down to 16 (the rows below are left unwritten)
};

// bf16-input score contraction with a loss epilogue (EPI_LOSS, EPI_LOSS_BITS or
// EPI_SOFTMAX_STATS) or the plain store (EPI_STORE: float32 scores to Cm)
void launch_gemm_bf16(const GemmArgsH& a, int epi, int batches, hipStream_t s);
// float32 score contraction with its loss epilogue (EPI_LOSS: float32 dS in
// Cm; EPI_LOSS_BITS; EPI_SOFTMAX_STATS) on the bf16 instructions, operands
// Af / Bf split into exact bf16 pieces on the way into LDS
void launch_score_split(const GemmArgsH& a, int epi, int batches, hipStream_t s);
// dQ = dS . N (a0: Af = dS rows [e][t]) and dN = dS^T . Q (a1: Af = the same
// dS rows, read by columns) in one launch, dS a general float32 matrix split
// into exact bf16 pieces on the way into LDS, B the three transposed planes
// of N / Q (planes = 3, b_ps apart); six piece products.  With smscale set,
// Af holds the per-tile exponentials of the softmax loss and dS is formed on
// the way
void launch_gemm_split_pair(const GemmArgsH& a0, const GemmArgsH& a1, int batches, hipStream_t s);
// two EPI_STORE products in one launch: a0 with A as dS rows (GA_BITS_ROW or
// GA_KC), a1 with A as dS columns (GA_BITS_COL or GA_MC), same planes
void launch_gemm_bf16_pair(const GemmArgsH& a0, const GemmArgsH& a1, int batches, hipStream_t s);
// bf16 path: Q and N rows (fp32, [rows][ld_src]) rounded once to bf16 rows
// [rows][kp] and transposed copies [kp][ldT], both operands in one launch.
// q = nullptr: N only
void launch_to_bf16_t(const float* q, int64_t q_bs, int q_rows, uint16_t* qh, int64_t qh_bs, uint16_t* qT,
                      int64_t qT_bs, int q_ldT, const float* n, int64_t n_bs, int n_rows, uint16_t* nh,
                      int64_t nh_bs, uint16_t* nT, int64_t nT_bs, int n_ldT, int ld_src, int kp, int batches,
                      hipStream_t s);
// fp32 rows [rows][ld_src] of Q and of N -> the exact bf16 pieces
// x = h + m + l as three transposed planes [kp][ld_T] each (ps elements
// apart, rows past `rows` up to ld_T zero), both operands in one launch.
// ld_src is a multiple of 4, ld_T of 8.  q = nullptr: N only.
// launch_finalize and launch_split3_t (same arguments) as one launch
void launch_finalize_split3_t(const StepGeom& g, const StepBufs& b, double* parts, bool softmax_scales,
                              const float* q, int64_t q_bs, int q_rows, uint16_t* qT, int64_t qT_bs, int64_t q_ps,
                              int q_ldT, const float* n, int64_t n_bs, int n_rows, uint16_t* nT, int64_t nT_bs,
                              int64_t n_ps, int n_ldT, int ld_src, int kp, int batches, hipStream_t s);
void launch_split3_t(const float* q, int64_t q_bs, int q_rows, uint16_t* qT, int64_t qT_bs, int64_t q_ps,
                     int q_ldT, const float* n, int64_t n_bs, int n_rows, uint16_t* nT, int64_t nT_bs,
                     int64_t n_ps, int n_ldT, int ld_src, int kp, int batches, hipStream_t s);

// ---- gather / operator / negatives --------------------------------------------
void launch_gather(const StepGeom& g, const StepBufs& b, hipStream_t s);
// sort keys and values of the contribution rows of a window of nsteps steps
// of S chunks ([step][stride], compact per step), and relation keys
// ([step][rstride], compact per step) when rkeys is set: the edges' relations,
// then with uniform_rel the chunk's relation of every uniform source
// candidate.  Chunks consecutive (cstart NULL) or relation-grouped (bounds
// cstart[0 .. nchunks] of the window's chunks, offsets in the call's arrays)
void launch_window_keys(const StepGeom& g, const int32_t* src, const int32_t* dst, const int32_t* rel,
                        int64_t n_edges, const int32_t* cstart, int nchunks, int64_t chunk0, int S, int nsteps,
                        int64_t stride, uint32_t* keys, uint32_t* vals, uint32_t* rkeys, uint32_t* rvals,
                        int64_t rstride, int uniform_rel, hipStream_t s);
void launch_transpose_rel(const float* A, float* AT, int R, int d, hipStream_t s);
// linear operator (one relation): padded copies of A and A^T, and the positive
// scores once Q has been formed by contraction
void launch_pad_linear(const float* A, int d, int dp, float* Ap, float* ATp, hipStream_t s);
void launch_positive_scores(const StepGeom& g, const StepBufs& b, hipStream_t s);
// linear operator with several relations (dot): Q = A_r x, K = A_r^T y and p
// per edge; the rows' operator backward; the sorted per-relation gradient
// sums with element-wise Adagrad (keys / vals: sorted relation ids and
// chunk * N + edge)
void launch_linear_rows(const StepGeom& g, const StepBufs& b, hipStream_t s);
void launch_linear_rows_backward(const StepGeom& g, const StepBufs& b, hipStream_t s);
void launch_linear_relation_update(const StepGeom& g, const StepBufs& b, const uint32_t* keys,
                                   const uint32_t* vals, int n, float lr, hipStream_t s);
// linear operator with cos: normalise the source candidates A x_t in place
// (norms to nrm) and form the positive scores
void launch_normalize_candidates(const StepGeom& g, const StepBufs& b, hipStream_t s);

// ---- loss finalisation and backward -----------------------------------------
void launch_softmax_rows_bf16(const StepGeom& g, const StepBufs& b, uint16_t* dsh, int ldh, hipStream_t s);
// The finalisation runs fin_blocks(C) workgroups of FIN_THREADS rows per
// chunk; softmax_scales: it also writes rowscale = exp(tile max - lse) for the
// backward on split pieces (score epilogue EPI_SOFTMAX_EXP)
#define FIN_THREADS 256
inline int fin_blocks(int C) { return (C + FIN_THREADS - 1) / FIN_THREADS; }
// parts: the step's fin_blocks(C) loss partials per chunk, [chunk][block]
void launch_finalize(const StepGeom& g, const StepBufs& b, double* parts, bool softmax_scales, hipStream_t s);
// out[t] = the fixed-order sum of the n partials of step t (stride apart;
// n_full per step, n_last in the last)
void launch_step_losses(const double* parts, int64_t stride, int n_full, int n_last, int64_t nsteps, double* out,
                        hipStream_t s);
void launch_op_backward(const StepGeom& g, const StepBufs& b, hipStream_t s);
// blocks per chunk of the operator backward's grid (relc rows per chunk with
// relsum): one wave per edge, and with cos one per four uniform candidates of
// a side
inline int op_backward_blocks(int C, int U, int cmp) {
  const int items = C + (cmp == CMP_COS ? 2 * ((U + 3) / 4) : 0);
  return (items + 3) / 4;
}

// ---- sort, segments, updates ----------------------------------------------------
// sorted positions per wave of the segment update (a power of two <= 32)
#define SEG_BLOCK 32

struct SortWork {
  uint32_t* keys_alt;   // [max_n] ping-pong buffers of the sort
  uint32_t* vals_alt;
  uint32_t* hist;       // [256][max blocks]
  uint32_t* scan_tmp;   // block sums of the multi-launch scan
  float* partial;       // [max_n][width] per-block partial sums of segments
  uint32_t* segflag;    // [max_n / SEG_BLOCK + 2] piece flags per block of sorted positions
  int max_n;
};

// work-buffer sizes (entries) of a radix sort of n keys: digit histograms and
// the multi-launch scan's block sums
int64_t radix_hist_entries(int64_t n);
int64_t radix_scan_tmp_entries(int64_t n);
// stable LSD radix sort of (key, value) pairs on the low `bits` bits of the
// keys; the result is left in keys / vals
void launch_radix_sort(uint32_t* keys, uint32_t* vals, int n, int bits, SortWork& w, hipStream_t s);
// the same sort without the final copy: *out_keys / *out_vals receive the
// buffers that hold the result (keys / vals or the work buffers)
// nseg independent sorts in one set of launches: segment y holds n_full
// pairs at keys / vals + y * stride (the last segment n_last), sorted stably
// on the low `bits` bits, results at *out_keys / *out_vals + y * stride (the
// inputs or the alternate buffers, of the same layout).  hist holds
// radix_segments_hist_entries(max n, nseg) entries.
void launch_radix_sort_segments(uint32_t* keys, uint32_t* vals, uint32_t* keys_alt, uint32_t* vals_alt,
                                int64_t stride, int n_full, int n_last, int nseg, int bits, uint32_t* hist,
                                uint32_t** out_keys, uint32_t** out_vals, hipStream_t s);
int64_t radix_segments_hist_entries(int64_t n, int nseg);
void launch_radix_sort_to(uint32_t* keys, uint32_t* vals, int n, int bits, SortWork& w, uint32_t** out_keys,
                          uint32_t** out_vals, hipStream_t s);

// Adagrad over sorted contribution rows (keys / vals as left by the sort):
// entity tables (row-wise accumulator) and relations with several ids
// (element-wise accumulators)
void launch_entity_update(const StepGeom& g, const StepBufs& b, const uint32_t* keys, const uint32_t* vals,
                          int n, SortWork& w, float lr, hipStream_t s);
void launch_relation_update_sorted(const StepGeom& g, const StepBufs& b, const uint32_t* keys,
                                   const uint32_t* vals, int n, SortWork& w, float lr, hipStream_t s);
// pieces per chunk of the single-relation gradient sum (partial rows per chunk)
#define RELSUM_PIECES 8
// sums of the nblk rows per chunk that the operator backward leaves with
// StepGeom::relsum, RELSUM_PIECES partial rows per chunk
void launch_relation_block_sums(const StepGeom& g, const float* rows, int nblk, float* partial, hipStream_t s);
// the entity update with the single relation's block sums (b.relc, nblk rows
// per chunk, into partial) and its Adagrad step riding along as extra
// workgroups of its two launches; false (nothing launched) when the
// relation rows need another row width than the entity rows
bool launch_entity_update_with_relation(const StepGeom& g, const StepBufs& b, const uint32_t* keys,
                                        const uint32_t* vals, int n, SortWork& w, float lr, int nblk, float* partial,
                                        float* relp, float* relG, hipStream_t s);
void launch_relation_single_adagrad(float* relp, float* relG, int width, const float* partial,
                                    int nparts, float lr, hipStream_t s);
void launch_exclusive_scan(const uint32_t* in, int64_t n, uint32_t* out, uint32_t* tmp,
                           uint32_t* total, hipStream_t s);
// entries of `tmp` that launch_exclusive_scan needs for n values (n > 0)
int64_t exclusive_scan_tmp_entries(int64_t n);

// ---- bucketing (Sec. 4.1) ----------------------------------------------------
// direct counting sort for up to BUCKET_DIRECT_MAX buckets: pass 1 counts each
// tile's edges per bucket into hist[bucket][tile] and ORs id-range failures
// into *flag (1 src, 2 dst, 4 rel); after an exclusive scan of hist, pass 2
// writes the offsets and every edge's local ids at its stable position
#define BUCKET_DIRECT_MAX 256
#define BUCKET_TILE 4096
int64_t bucket_direct_units(int64_t n);
void launch_bucket_count(const int64_t* src, const int64_t* dst, const int32_t* rel, int64_t n, int64_t n_ent,
                         int32_t n_rel, int64_t ps, int P, uint32_t* hist, uint32_t* flag, hipStream_t s);
void launch_bucket_scatter(const int64_t* src, const int64_t* dst, const int32_t* rel, int64_t n, int64_t ps,
                           int P, const uint32_t* start, int64_t* offsets, int32_t* src_local,
                           int32_t* rel_out, int32_t* dst_local, hipStream_t s);
void launch_bucket_keys(const int64_t* src, const int64_t* dst, int64_t n, int64_t ps, int P,
                        uint32_t* keys, uint32_t* vals, hipStream_t s);
void launch_bucket_offsets(const uint32_t* keys, int64_t n, int nb, int64_t* offsets, hipStream_t s);
// entity types: bucket keys from each relation's type geometry geo [R][4] =
// (source partition size, source entities, destination partition size,
// destination entities), range checks into flag (1 source, 2 destination,
// 4 relation); then local ids through the sorted positions
void launch_typed_bucket_keys(const int64_t* src, const int32_t* rel, const int64_t* dst, int64_t n,
                              const int64_t* geo, int R, int P, uint32_t* keys, uint32_t* vals, uint32_t* flag,
                              hipStream_t s);
void launch_typed_bucket_gather(const uint32_t* vals, const int64_t* src, const int32_t* rel, const int64_t* dst,
                                int64_t n, const int64_t* geo, int32_t* src_local, int32_t* rel_out,
                                int32_t* dst_local, hipStream_t s);
void launch_bucket_gather(const uint32_t* vals, const int64_t* src, const int32_t* rel,
                          const int64_t* dst, int64_t n, int64_t ps, int32_t* src_local,
                          int32_t* rel_out, int32_t* dst_local, hipStream_t s);

// ---- filtered ranks (Sec. 5.4) -------------------------------------------------
// T0: every entity row (unit rows for cos); T1 (cos with an operator, one
// relation): the unit rows of g(x) (relT: the linear operator's A^T rows)
void launch_rank_tables(const StepGeom& g, const float* emb, const float* relp, const float* relT, int64_t n_ent,
                        float* T0, float* T1, hipStream_t s);
void launch_rank_queries(const StepGeom& g, const float* emb, const float* relp, const float* relT,
                         const int32_t* src, const int32_t* rel, const int32_t* dst, int64_t e0, int rows,
                         int side, float* Q, float* pos, float* bias, hipStream_t s);
// cand: entity id of each score column (nullptr: column t is entity t)
void launch_rank_count(const float* S, int64_t ldS, int64_t n_ent, const int32_t* cand, int64_t e0, int rows,
                       int side, int64_t n_eval, const int32_t* src, const int32_t* rel, const int32_t* dst,
                       const float* pos, const float* bias, const int32_t* ka, const int32_t* kb,
                       const int32_t* kc, int64_t n_known, int32_t* ranks, hipStream_t s);
// out[i] = T[idx[i]], rows of ld floats (ids checked by the caller)
void launch_gather_rows(const float* T, const int32_t* idx, int64_t n, int ld, float* out, hipStream_t s);
void launch_rank_metrics(const int32_t* ranks, int64_t n, double* out, hipStream_t s);
void launch_perm_keys(const int32_t* field, const uint32_t* perm, int64_t n, uint32_t* keys,
                      uint32_t* vals_init, hipStream_t s);
void launch_gather3(const uint32_t* perm, const int32_t* a, const int32_t* b, const int32_t* c, int64_t n,
                    int32_t* oa, int32_t* ob, int32_t* oc, hipStream_t s);

// ---- checks, scoring, ranking --------------------------------------------------
void launch_check_ids(const int32_t* ids, int64_t n, int32_t limit, uint32_t* flag, uint32_t bit,
                      hipStream_t s);
// p[0 .. n) = v (a kernel, so that it may sit in a captured graph)
void launch_fill_u32(uint32_t* p, int64_t n, uint32_t v, hipStream_t s);
void launch_check_ids64(const int64_t* ids, int64_t n, int64_t limit, uint32_t* flag, uint32_t bit,
                        hipStream_t s);
void launch_score_edges(const StepGeom& g, const float* emb_i, const float* emb_j, const float* relp,
                        const float* relT, const int32_t* src, const int32_t* rel,
                        const int32_t* dst, int64_t n, float* out, hipStream_t s);
void launch_sample_negatives(uint64_t seed, uint32_t bucket, int64_t chunk0, int64_t n_chunks, int U,
                             uint32_t rows_j, uint32_t rows_i, int32_t* out, hipStream_t s);

// ---- inspection of a step's forward half ----------------------------------------
enum { DS_BITS = 0, DS_F32 = 1, DS_F32_SCALED = 2, DS_BF16 = 3 };
// out [c][2][C][N] of the source side (side 1) += the per-edge translation bias
void launch_add_side_bias(const StepGeom& g, const float* bias, float* out, hipStream_t s);
// dL/dS as float32 [c][2][C][N] from the layout `mode` (DS_*) the loss left it in
void launch_expand_ds(const StepGeom& g, int mode, const uint16_t* bits, int nw, int ldw, const float* f32,
                      const float* scale, const uint16_t* h, int ld, float* out, hipStream_t s);
void launch_copy_pos(const StepGeom& g, const float* pos, float* out, hipStream_t s);
