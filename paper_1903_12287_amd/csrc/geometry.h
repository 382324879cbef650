// Layout of one training step's workspace, shared by host code and kernels.
//
// A step holds `nchunks` chunks of a bucket (i, j).  Chunk c has
// Cc = min(C, m_step - c*C) edges and Nc = Cc + U candidates per side: the
// chunk's own destinations (or sources) followed by U uniform draws.
//
// Packed float32 buffers (row stride dp = dim rounded up to 4, pad columns 0):
//   qk  [S][2][C][dp]   side 0: Q = g(x_s) (dot) or its unit vector (cos)
//                       side 1: K = g*(x_d) (dot) or the unit x_d (cos);
//                       reciprocal predicates: K = g(x_d, theta_{r+R}) (or its
//                       unit vector), and nn holds the raw (or unit) entities
//   nn  [S][2][N][dp]   side 0: destination candidates, side 1: source candidates
//   ds  [S][2][C][Np]   score gradient dL/dS (raw scores between softmax passes);
//                       for the ranking loss dL/dS is 0 or 1 and is kept as bits,
//                       dsb [S][2][ceil(Np/16)][C] 16-bit words (16 columns of a
//                       row per word, stored word-column major)
//   dq  [S][2][C][dp]   dS . N per side
//   dn  [S][2][N][dp]   dS^T . Q per side, turned in place into the per-row
//                       gradient contributions of the step
// Row index of candidate t of side s in chunk c: (c*2 + s)*N + t.
#pragma once

#include <stdint.h>

enum { OP_IDENTITY = 0, OP_TRANSLATION = 1, OP_DIAGONAL = 2, OP_LINEAR = 3, OP_COMPLEX = 4 };
enum { CMP_DOT = 0, CMP_COS = 1 };

// With the cos comparator the packed Q and K rows of a chunk equal its first
// C source and destination candidate rows (g(x_s) and x_d, both normalised),
// so Q / K row e of side s is read from row e of the candidate tile of side
// 1 - s and never written separately.  Not with reciprocal predicates: there
// the candidates never carry the operator and both queries do.
#define QK_IN_NN(g) ((g).cmp == CMP_COS && !(g).recip)
enum { LOSS_RANKING = 0, LOSS_LOGISTIC = 1, LOSS_SOFTMAX = 2 };

#define PBG_EPS_NORM 1e-12f
#define PBG_EPS_ADAGRAD 1e-10f
#define PBG_SCORE_BN 128  // column tile of the score contraction

struct StepGeom {
  int C, U, N;      // chunk capacity, uniform draws per side, N = C + U
  int d, dp, Np;    // dim, padded row stride, padded score-row stride
  int dr;           // floats per relation parameter row
  int nct;          // column tiles of the score contraction per chunk-side
  int nchunks;      // chunks in this step
  int m_step;       // edges in this step
  int op, cmp, loss;
  float margin;
  int same_table;   // partitions i and j are the same table
  int rows_i, rows_j;
  int rb;           // bits of a row id in a sort key
  uint32_t bucket;  // i*P + j
  uint64_t seed;
  int64_t chunk0;   // chunk number (within the bucket) of the step's first chunk
  const int32_t* cstart;  // relation-grouped chunks: bounds of the step's chunks (device), else NULL
  int recip;        // reciprocal predicates: the source side uses relation row r + R
  int R;            // relations (the offset of the source side's rows)
  int relN;         // rows of relc per chunk (N; 2C with reciprocal predicates)
  int relsum;       // one relation operator for every edge (not linear): the operator backward adds the
                    // parameter-gradient rows of each block and relc holds one row per block
  const float* cweight;   // relation weight of each chunk of the step (device), NULL: all 1
  int dq_has_dn;    // with QK_IN_NN: dq of side s, row e < Cc, already holds dn of side 1 - s, row e (the
                    // ranking backward merged them), and those dn rows are not written
};

// index of edge e's positive score of side s in pos / dpos: one shared
// score per edge, or one per side with reciprocal predicates
__host__ __device__ inline int64_t pos_index(const StepGeom& g, int c, int side, int e) {
  return g.recip ? ((int64_t)(c * 2 + side) * g.C + e) : ((int64_t)c * g.C + e);
}

// A value that every lane of the wave reads from the same address, kept in a
// scalar register.  The loads that bring it are vector loads, so without this
// everything derived from it (tile bounds, row limits, scales) would live in
// vector registers, and a conditional use would wait for all of the wave's
// outstanding memory operations, stores included.
__device__ __forceinline__ int wave_uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ float wave_uniform(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, v)));
}

// Chunk c of a step: its edge count and the offset of its first edge in the
// step's edge arrays.  Consecutive chunks hold C edges each (the step's last
// one may be short); relation-grouped chunks have their bounds in cstart
// (offsets in the call's edge arrays, cstart[c + 1] the end of chunk c).
// c must be the same in every lane of the wave.
__device__ inline int chunk_edges(const StepGeom& g, int c) {
  if (g.cstart) return wave_uniform(g.cstart[c + 1] - g.cstart[c]);
  const int r = g.m_step - c * g.C;
  return r < g.C ? r : g.C;
}

__device__ inline int chunk_first(const StepGeom& g, int c) {
  return g.cstart ? wave_uniform(g.cstart[c] - g.cstart[0]) : c * g.C;
}

// Relation of edge eg of the step.  With one relation every (validated) id is
// 0, so the id array is not read and the relation row's load does not wait
// for it.
__device__ inline int edge_relation(const StepGeom& g, const int32_t* rel, int64_t eg) {
  return (rel && g.R > 1) ? rel[eg] : 0;
}

struct StepBufs {
  // edges of the step (device, int32)
  const int32_t* src;
  const int32_t* dst;
  const int32_t* rel;   // NULL: relation 0
  // parameters
  float* emb_i;
  float* emb_j;
  float* G_i;
  float* G_j;
  float* relp;          // [R][dr]
  float* relG;
  // packed tiles and intermediates
  float* qk;
  float* nn;
  float* nrm;           // [S][2][N] norms of the raw vectors behind nn (cos)
  float* pos;           // [S][C] positive scores ([S][2][C] with reciprocal predicates)
  float* bias;          // [S][C] <theta_r, x_d> (translation + dot)
  int32_t* neg;         // [S][2][U] uniform draws (side 0 from partition j, side 1 from i)
  float* ds;            // [S][2][C][Np] dL/dS (logistic, softmax)
  uint16_t* dsb;        // [S][2][ceil(Np/16)][C] dL/dS bits (ranking, float32 path)
  float* rowpart;       // [S][2][C][nct][2]  per score tile: (loss, dS sum) or, for
                        // softmax, (tile max, sum exp(s - tile max))
  float* rowscale;      // [S][2][nct][C]  softmax on split pieces: exp(tile max - lse)
  float* rowloss;       // [S][2][C] each edge's loss per side (inspection only; NULL in training)
  float* dpos;          // [S][C] dL/dp ([S][2][C] with reciprocal predicates)
  float* dsum1;         // [S][C] sum_t dS1[e][t]
  unsigned long long* nuniq;   // rows touched by the entity updates of the call (segment count)
  float* dq;
  float* dn;
  float* relc;          // [S][relN][dr] relation gradient contributions: edge rows, then the
                        // uniform source candidates' (cos with an operator) or, with
                        // reciprocal predicates, the edges' source-side rows r + R; with
                        // relsum [S][blocks of the operator backward][dr], one summed row
                        // per block
  float* qnrm;          // reciprocal + cos: [S][2][C] norms of the raw queries
  float* lin_x;         // linear + cos: [S][N][dp] raw source candidate rows x_t (reciprocal
                        // predicates: [S][2][C][dp], the edges' raw x_s, then x_d)
  float* lin_v;         // linear + cos, one relation: [S][N][dp] dL/d(A x_t) of the source candidates
  uint32_t* keys;       // [S*2N] sort keys of the contribution rows
  uint32_t* vals;       // [S*2N] contribution row index
  uint32_t* rkeys;      // relation ids of the contribution rows (R > 1 or reciprocal predicates)
  uint32_t* rvals;      // their relc row index
};
