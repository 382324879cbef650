// bfloat16 inputs / float32 accumulation for the three chunk contractions
// (Sec. 4.3 batched negatives; the score block of a chunk is one product).
//
//   forward  S  = Q  . N^T  :  A = Q    [e][f],  B = N   [t][f]
//   dQ       dQ = dS . N    :  A = dS   [e][t],  B = N^T [f][t]
//   dN       dN = dS^T . Q  :  A = dS^T [t][e],  B = Q^T [f][e]
// The B operands are contiguous along k: the bf16 copies of Q and N and their
// transposes are produced once per step (LDS-tiled transpose).  The A operand
// of the backward products is dS itself, read in place: for the ranking loss
// from its bit matrix (rows for dQ, columns for dN), otherwise from bf16 dS
// rows (transposed on the way into LDS for dN), so no copy of dS^T exists.
//
// Float32 backward of the ranking loss on the same instruction: there dS is
// 0 or 1, and a float32 operand x splits exactly into three bf16 pieces,
// x = h + m + l (h = bf16(x), m = bf16(x - h), l = x - h - m, which needs at
// most 8 significant bits).  Every product dS * piece is then exact and the
// sums run in float32, so dS . N equals a float32 contraction up to the order
// of the float32 additions.  The kernel takes B as PL = 3 planes (pieces) and
// adds the three products into one accumulator.
//
// Layout and schedule follow the float32 kernel: 256-thread workgroups of
// 2 x 2 waves on 128 x BN tiles, buffer loads with hardware zero-fill,
// register prefetch one k-slice ahead, double-buffered LDS tiles and all
// tiles of one batch on one XCD.  A slice is 32 deep, one
// v_mfma_f32_16x16x32_bf16 step: lane L feeds A[L % 16][8 (L / 16) + i] and
// B[8 (L / 16) + i][L % 16], i = 0..7, one 16-byte LDS read each; the
// accumulator holds D[4 (L / 16) + r][L % 16] in register r.
// LDS tiles are [row][k], 32 bf16 (64 bytes) per row with no padding: the
// 16-byte group q of row x is kept at group q ^ (((x >> 1) ^ ((x >> 3) & 1)) & 3),
// which repeats every 16 rows.
// A fragment read (16 consecutive rows, one group each) then touches every
// 16-byte bank group once, whether the LDS serves 16 lanes over 64 banks or
// 8 lanes over 32 banks per cycle, and so do the tile stores (four groups of
// consecutive rows).
#include <algorithm>

#include "kernels.h"
#include "device_common.h"
#include "finalize_body.h"

namespace {

constexpr int BM = 128;
constexpr int BK = 32;          // k per slice = bf16 elements per LDS tile row
constexpr uint32_t OOB = 0x80000000u;

typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// A buffer descriptor must be wave-uniform.  Tile base addresses are, but
// their 64-bit products are formed on the vector unit, and a descriptor left
// in vector registers would make the compiler wrap every load that uses it in
// a loop over lanes; reading the address back from the first lane keeps it
// scalar.
__device__ __forceinline__ rsrc_t make_rsrc(const void* p) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), (short)0, 0x7FFFFFF0, 0x00020000);
}
__device__ __forceinline__ u32x4 bload16(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

__device__ __forceinline__ float bf16_to_f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint16_t f_to_bf16(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

// two floats -> one packed bf16 pair (a in the low half), round to nearest even
__device__ __forceinline__ uint32_t f2_to_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, (bf16x2_t){(__bf16)a, (__bf16)b});
}

// x = h + m + l exactly, each piece a bf16: h = bf16(x) leaves a remainder of
// at most 16 significant bits, m = bf16 of that remainder leaves at most 8,
// which l holds exactly (for |x| >= 2^-110, where every piece is a normal
// number).  Two floats at a time: pc[0..2] = packed h, m, l.
// The empty asm statements hide h and m from the optimiser, which would
// otherwise form h << 16 from a second conversion of a alone (one extra
// instruction per level and pair).
__device__ __forceinline__ void split3_pair(float a, float b, uint32_t* pc) {
  uint32_t h = f2_to_bf16x2(a, b);
  __asm__("" : "+v"(h));
  const float ra = a - __uint_as_float(h << 16), rb = b - __uint_as_float(h & 0xFFFF0000u);
  uint32_t m = f2_to_bf16x2(ra, rb);
  __asm__("" : "+v"(m));
  pc[0] = h;
  pc[1] = m;
  pc[2] = f2_to_bf16x2(ra - __uint_as_float(m << 16), rb - __uint_as_float(m & 0xFFFF0000u));
}

__device__ __forceinline__ int pick_dim(int sel, int fixed, int Cc, int Nc) {
  return sel == DIM_CC ? Cc : (sel == DIM_NC ? Nc : fixed);
}

// element offset of the 16-byte group q of row x in a swizzled LDS tile
__device__ __forceinline__ int swz(int x, int q) {
  return x * BK + ((q ^ (((x >> 1) ^ ((x >> 3) & 1)) & 3)) << 3);
}

// two bits t (0..3) -> the packed bf16 pair (bit 0 low, bit 1 high) of 0.0 / 1.0:
// t * 0x8001 puts bit 0 at bit 0 and bit 1 at bit 16, and 0x3F80 is 1.0
__device__ __forceinline__ uint32_t bit_pair(uint32_t t) { return ((t * 0x8001u) & 0x10001u) * 0x3F80u; }

// One operand tile of TX rows x BK k as LDS [row][k] bf16 (swizzled); each
// thread moves TX * BK / 8 / 256 groups of eight elements per slice.  Loaded
// words stay raw in registers until the store, after the slice's matrix work.
//   GA_KC        global [x][k] bf16, ld elements, k contiguous (zero-padded to 8)
//   GA_MC        global [k][x] bf16, x contiguous: eight x of one k go to eight
//                tile rows
//   GA_BITS_ROW  bit matrix (dsb layout), tile row x = matrix row, k = column
//   GA_BITS_COL  bit matrix, tile row x = matrix column, k = matrix row; the
//                words of eight consecutive rows of one word column are 16
//                contiguous bytes (row pitch a multiple of 8)
template <int TX, int MODE>
struct TileH {
  static constexpr int LOADS = TX * BK / 8 / 256;
  static constexpr int SIZE = TX * BK;

  __device__ __forceinline__ static void load(u32x4* r, rsrc_t rs, int ld, int x0, int xdim, int k0, int kdim, int tid) {
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int f = tid + 256 * q;
      uint32_t off = OOB;
      if (MODE == GA_MC) {
        const int k = f / (TX / 8), xq = f % (TX / 8);
        const int gk = k0 + k, gx = x0 + 8 * xq;
        if (gk < kdim && gx < ((xdim + 7) & ~7)) off = (uint32_t)(((int64_t)gk * ld + gx) * 2);
        r[q] = bload16(rs, off);
      } else {
        const int x = f >> 2, kq = f & 3;
        const int gx = x0 + x, gk = k0 + 8 * kq;
        if (MODE == GA_KC) {
          if (gx < xdim && gk < ((kdim + 7) & ~7)) off = (uint32_t)(((int64_t)gx * ld + gk) * 2);
          r[q] = bload16(rs, off);
        } else if (MODE == GA_BITS_ROW) {
          if (gx < xdim && gk < ((kdim + 7) & ~7)) off = (uint32_t)(((int64_t)(gk >> 4) * ld + gx) * 2);
          const uint32_t w = __builtin_amdgcn_raw_buffer_load_b16(rs, off, 0, 0);
          r[q] = (u32x4){w, 0u, 0u, 0u};
        } else {
          if (gx < ((xdim + 7) & ~7) && gk < kdim) off = (uint32_t)(((int64_t)(gx >> 4) * ld + gk) * 2);
          r[q] = bload16(rs, off);
        }
      }
    }
  }

  __device__ __forceinline__ static void store(uint16_t* s, const u32x4* r, int tid, int x0, int k0, int kdim) {
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int f = tid + 256 * q;
      if (MODE == GA_MC) {
        const int k = f / (TX / 8), xq = f % (TX / 8);
        const u32x4 v = r[q];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int x = 8 * xq + i;
          s[swz(x, k >> 3) + (k & 7)] = (uint16_t)((i & 1) ? (v[i >> 1] >> 16) : (v[i >> 1] & 0xFFFFu));
        }
      } else {
        const int x = f >> 2, kq = f & 3;
        u32x4 v = r[q];
        if (MODE == GA_BITS_ROW) {
          // bits of columns k0 + 8 kq + 0..7 -> four packed bf16 pairs
          const uint32_t bits = v.x >> ((8 * kq) & 15);
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = bit_pair(__builtin_amdgcn_ubfe(bits, 2 * i, 2));
        } else if (MODE == GA_BITS_COL) {
          // bit b of the words of rows gk .. gk + 7 (two rows per dword)
          const int b = (x0 + x) & 15;
#pragma unroll
          for (int i = 0; i < 4; ++i) v[i] = ((v[i] >> b) & 0x00010001u) * 0x3F80u;
          const int nv = kdim - (k0 + 8 * kq);   // rows from nv on lie outside the chunk
          if (nv < 8) {
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] &= (2 * i + 1 < nv) ? 0xFFFFFFFFu : (2 * i < nv ? 0xFFFFu : 0u);
          }
        }
        *(u32x4*)(s + swz(x, kq)) = v;
      }
    }
  }
};

// LDS of one workgroup: the A tile and PL B tiles (NB buffers), row partials
template <int BN, int PL>
struct SmemH {
  // three B planes: one buffer (three workgroups per CU); otherwise two
  static constexpr int NB = PL == 3 ? 1 : 2;
  uint16_t As[NB][BM * BK];
  uint16_t Bs[NB][PL][BN * BK];
  float red[2][BM][2];
  float rowv[2][BM];
};

// Position of a workgroup's TM x BN tile (TM = 128 rows unless stated): `id` numbers the workgroup among
// the nwg of its product (hardware order) and is remapped so that all tiles of
// one batch (chunk, side) run on one XCD.
struct TileGeo {
  int c, side, Nc, M, N, K, m0, n0, tn;
};

// false: nothing to compute (the tile lies beyond this batch's rows, or beyond
// its columns, where a loss epilogue still leaves neutral row partials)
template <int BN, int EPI, int TM = BM>
__device__ __forceinline__ bool tile_geo(const GemmArgsH& a, int tiles_n, int tiles_m, int nwg, int id,
                                         TileGeo& t) {
  const int q8 = nwg >> 3, r8 = nwg & 7, xcd = id & 7;
  const int lid = xcd * q8 + min(xcd, r8) + (id >> 3);
  t.tn = lid % tiles_n;
  const int rest = lid / tiles_n;
  const int tm = rest % tiles_m;
  const int z = rest / tiles_m;
  t.c = z / a.nsides;
  t.side = z - t.c * a.nsides;
  int Cc = a.C;
  t.Nc = a.C + a.U;
  if (a.cstart) {
    Cc = wave_uniform(a.cstart[t.c + 1] - a.cstart[t.c]);
    t.Nc = Cc + a.U;
  } else if (a.m_step > 0) {
    Cc = min(a.C, a.m_step - t.c * a.C);
    t.Nc = Cc + a.U;
  }
  t.M = pick_dim(a.mdim, a.Mfix, Cc, t.Nc);
  t.N = pick_dim(a.ndim, a.Nfix, Cc, t.Nc);
  t.K = pick_dim(a.kdim, a.Kfix, Cc, t.Nc);
  t.m0 = tm * TM;
  t.n0 = t.tn * BN;
  // shared in-chunk blocks: side 1's full tiles of [0, Cc) x [0, Cc) come
  // from side 0's tiles (tn, tm), transposed
  if (a.share_cc && t.side == 1 && tm < Cc / TM && t.tn < Cc / BN) return false;
  // merged ranking backward: the dN rows below Cc (rounded down to a 16-row
  // bit word) are taken by the other side's dQ
  if (a.merge_cc && a.mdim == DIM_NC) t.m0 += Cc & ~15;
  if (t.m0 >= t.M) return false;
  if (t.n0 >= t.N) {
    const int tid = threadIdx.x;
    if (EPI != EPI_STORE && tid < TM && t.m0 + tid < t.M) {
      float* rp = a.rowpart + (((int64_t)(t.c * 2 + t.side) * a.C + t.m0 + tid) * a.nct + t.tn) * 2;
      rp[0] = (EPI == EPI_SOFTMAX_STATS || EPI == EPI_SOFTMAX_EXP) ? -INFINITY : 0.0f;
      rp[1] = 0.0f;
    }
    return false;
  }
  return true;
}

// per-row values of the tile for the loss epilogues, read once at the start
// of the tile while its first operands load: the hinge threshold
// margin - p + bias (-inf for rows past the batch) for the ranking bits, else
// the positive score p and the bias
template <int EPI, int TM = BM>
__device__ __forceinline__ void load_rowv(const GemmArgsH& a, const TileGeo& t, float (&rowv)[2][TM]) {
  const int tid = threadIdx.x;
  if (tid < TM) {
    const int m = t.m0 + tid;
    const bool mrow = m < t.M;
    const int64_t o = (int64_t)t.c * a.C + m;
    // row of pos: chunk c (pos_sides = 1), or chunk c and side (pos_sides = 2);
    // arithmetic rather than a select keeps the tile loop free of spills
    const int64_t op = (int64_t)(t.c * a.pos_sides + (a.pos_sides - 1) * t.side) * a.C + m;
    const float p = mrow ? a.pos[op] : 0.0f;
    const float bm = (mrow && a.bias && t.side == 1) ? a.bias[o] : 0.0f;
    if (EPI == EPI_LOSS_BITS) {
      rowv[0][tid] = mrow ? a.margin - p + bm : -INFINITY;
    } else {
      rowv[0][tid] = p;
      rowv[1][tid] = bm;
    }
  }
}

// Ranking loss rows of a tile (MASKED: the tile holds columns past the batch
// or the masked diagonal).  Hinge z = s + margin - p, dS = [z > 0]; each lane
// group's ballot word is the bit-matrix word of its row for these 16 columns
// and its population count that row's share of the dS row sum.
template <int BN, bool MASKED, int TM = BM>
__device__ __forceinline__ void bits_rows(const GemmArgsH& a, const TileGeo& t, v4f (&acc)[TM / 32][BN / 32],
                                          float (&red)[2][TM][2], const float (&rowv)[2][TM]) {
  constexpr int WN = BN / 2, WMR = TM / 2;
  constexpr int JN = WN / 16, IM = TM / 32;
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int l16 = lane & 15, g = lane >> 4;
  const int colb = t.n0 + WN * wn + l16;
  const int wcol0 = (t.n0 + WN * wn) >> 4;
  // the words of four consecutive rows are adjacent (word-column major)
  uint16_t* dbase = a.dsb + t.c * a.cb_cs + t.side * a.cb_ss + (int64_t)wcol0 * a.ldcb + t.m0 + WMR * wm + 4 * g;
#pragma unroll
  for (int i = 0; i < IM; ++i) {
    const int mb = WMR * wm + 16 * i + 4 * g;   // first of this lane group's four rows
    const v4f thr = *(const v4f*)&rowv[0][mb];
    float ls[4] = {-0.0f, -0.0f, -0.0f, -0.0f};   // -0 + x is x: the first add folds away
    uint32_t cnt[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < JN; ++j) {
      uint32_t wd[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        // s + thr > 0 exactly when s > -thr (an IEEE sum is positive exactly
        // when the exact sum is), so the compare needs no add; the hinge sum
        // of the row is the sum of its selected scores plus thr per bit
        const float s = acc[i][j][r];
        bool hit = s > -thr[r];
        if (MASKED) {
          const int n = colb + 16 * j;
          if (n >= t.N || n == t.m0 + mb + r) hit = false;
        }
        const uint64_t mk = __ballot(hit);
        ls[r] += hit ? s : 0.0f;   // one select on the compare already made
        wd[r] = (uint32_t)(mk >> (16 * g)) & 0xFFFFu;
        cnt[r] += __builtin_popcount(wd[r]);
      }
      if (l16 == 0 && t.m0 + mb < t.M && wcol0 + j < a.nwcb)
        *(uint2*)(dbase + (int64_t)j * a.ldcb + 16 * i) = make_uint2(wd[0] | (wd[1] << 16), wd[2] | (wd[3] << 16));
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float v0 = group16_sum(ls[r]);
      if (l16 == 0) {
        red[wn][mb + r][0] = fmaf(thr[r], (float)cnt[r], v0);   // rows past the batch: unused
        red[wn][mb + r][1] = (float)cnt[r];
      }
    }
  }
}

// logistic loss (dS rows in bf16 or float32) and softmax statistics (raw
// scores + per-tile max and sum of exp) rows of a tile
template <int BN, int EPI, bool MASKED, int TM = BM>
__device__ __forceinline__ void value_rows(const GemmArgsH& a, const TileGeo& t, v4f (&acc)[TM / 32][BN / 32],
                                           float (&red)[2][TM][2], const float (&rowv)[2][TM]) {
  constexpr int WN = BN / 2, WMR = TM / 2;
  constexpr int JN = WN / 16, IM = TM / 32;
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int l16 = lane & 15, g = lane >> 4;
  const int c = t.c, side = t.side, M = t.M, N = t.N, m0 = t.m0;
  const int colb = t.n0 + WN * wn + l16;
  const float kinv = (t.Nc - 1 > 0) ? 1.0f / (float)(t.Nc - 1) : 0.0f;
#pragma unroll
  for (int i = 0; i < IM; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ml = WMR * wm + 16 * i + 4 * g + r;
      const int m = m0 + ml;
      const bool mrow = m < M;
      const float p = rowv[0][ml];
      const float bm = rowv[1][ml];
      const int64_t orow = c * a.c_cs + side * a.c_ss + (int64_t)m * a.ldc;
      float v0, v1;
      if (EPI == EPI_LOSS) {
        float lsum = 0.0f, dsum = 0.0f;
#pragma unroll
        for (int j = 0; j < JN; ++j) {
          const int n = colb + 16 * j;
          const float s = acc[i][j][r] + bm;
          const bool valid = mrow && !(MASKED && (n >= N || n == m));
          float dsv = 0.0f;
          if (valid) {
            if (a.loss == LOSS_RANKING) {
              const float zz = a.margin - p + s;
              if (zz > 0.0f) {
                dsv = 1.0f;
                lsum += zz;
              }
            } else {
              float sg, sp;
              logistic_pair(s, sg, sp);
              dsv = sg * kinv;
              lsum += sp * kinv;
            }
          }
          dsum += dsv;
          if (mrow && n < a.ldc) {
            if (a.dsh) a.dsh[orow + n] = f_to_bf16(dsv);
            else a.Cm[orow + n] = dsv;
          }
        }
        v0 = group16_sum(lsum);
        v1 = group16_sum(dsum);
      } else {  // EPI_SOFTMAX_STATS
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < JN; ++j) {
          const int n = colb + 16 * j;
          const float s = acc[i][j][r] + bm;
          if (mrow && !(MASKED && (n >= N || n == m))) mx = fmaxf(mx, s);
          if (mrow && n < a.ldc) a.Cm[orow + n] = s;
        }
        mx = group16_max(mx);
        float se = 0.0f;
#pragma unroll
        for (int j = 0; j < JN; ++j) {
          const int n = colb + 16 * j;
          if (mrow && !(MASKED && (n >= N || n == m))) se += expf(acc[i][j][r] + bm - mx);
        }
        v0 = mx;
        v1 = group16_sum(se);
      }
      if (l16 == 0) {
        red[wn][ml][0] = v0;
        red[wn][ml][1] = v1;
      }
    }
}

// Softmax rows of a tile for the backward on split pieces: the tile's row
// maximum M over the valid columns (both column halves), then exp(s - M) on
// the valid columns and 0 elsewhere (columns past the batch, the diagonal)
// goes to Cm and its row sum to the partials.  dS = exp(s - M) exp(M - lse)
// is completed in the backward once lse is known.
template <int BN, bool MASKED, int TM = BM>
__device__ __forceinline__ void softmax_exp_rows(const GemmArgsH& a, const TileGeo& t,
                                                 v4f (&acc)[TM / 32][BN / 32], float (&red)[2][TM][2],
                                                 const float (&rowv)[2][TM]) {
  constexpr int WN = BN / 2, WMR = TM / 2;
  constexpr int JN = WN / 16, IM = TM / 32;
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int l16 = lane & 15, g = lane >> 4;
  const int M = t.M, N = t.N, m0 = t.m0;
  const int colb = t.n0 + WN * wn + l16;
#pragma unroll
  for (int i = 0; i < IM; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ml = WMR * wm + 16 * i + 4 * g + r;
      const int m = m0 + ml;
      const float bm = rowv[1][ml];
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < JN; ++j) {
        const int n = colb + 16 * j;
        acc[i][j][r] += bm;
        if (m < M && !(MASKED && (n >= N || n == m))) mx = fmaxf(mx, acc[i][j][r]);
      }
      mx = group16_max(mx);
      if (l16 == 0) red[wn][ml][0] = mx;
    }
  __syncthreads();
  float* Cm = a.Cm + t.c * a.c_cs + t.side * a.c_ss;
#pragma unroll
  for (int i = 0; i < IM; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ml = WMR * wm + 16 * i + 4 * g + r;
      const int m = m0 + ml;
      const float mt = fmaxf(red[0][ml][0], red[1][ml][0]);
      float se = 0.0f;
#pragma unroll
      for (int j = 0; j < JN; ++j) {
        const int n = colb + 16 * j;
        const bool valid = m < M && !(MASKED && (n >= N || n == m));
        const float ev = valid ? expf(acc[i][j][r] - mt) : 0.0f;
        se += ev;
        if (m < M && n < a.ldc) Cm[(int64_t)m * a.ldc + n] = ev;
      }
      se = group16_sum(se);
      if (l16 == 0) red[wn][ml][1] = se;
    }
}

// Stores the tile (EPI_STORE) or runs the loss epilogue on it: dS leaves as
// bits (ranking), as bf16 rows (logistic, when dsh is set) or float32 rows in
// Cm, or the raw float32 scores go to Cm for the softmax row pass; row
// partials (loss, dS sum / max, sum exp) are combined over the tile's two
// column halves and written per column tile.
template <int BN, int EPI, int TM = BM>
__device__ __forceinline__ void tile_epilogue(const GemmArgsH& a, const TileGeo& t, v4f (&acc)[TM / 32][BN / 32],
                                              float (&red)[2][TM][2], const float (&rowv)[2][TM]) {
  constexpr int WN = BN / 2, WMR = TM / 2;
  constexpr int JN = WN / 16, IM = TM / 32;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int l16 = lane & 15, g = lane >> 4;
  const int c = t.c, side = t.side, M = t.M, N = t.N, Nc = t.Nc, m0 = t.m0, n0 = t.n0;
  const int colb = n0 + WN * wn + l16;
  if (EPI == EPI_STORE) {
    float* Cm = a.Cm + c * a.c_cs + side * a.c_ss;
    // the chunk's weight (1 without weights: the product is exact), read once
    // into a scalar register
    const float sc = a.cscale ? wave_uniform(a.cscale[c]) : 1.0f;
#pragma unroll
    for (int i = 0; i < IM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + WMR * wm + 16 * i + 4 * g + r;
        if (m < M) {
#pragma unroll
          for (int j = 0; j < JN; ++j) {
            const int n = colb + 16 * j;
            if (n < N) Cm[(int64_t)m * a.ldc + n] = acc[i][j][r] * sc;
          }
        }
      }
    return;
  }

  // column tiles past the batch's last column and tiles that meet the masked
  // diagonal need per-element checks
  const bool masked = (n0 + BN > N) || (m0 < n0 + BN && n0 < m0 + TM);
  if (EPI == EPI_LOSS_BITS) {
    if (masked) bits_rows<BN, true, TM>(a, t, acc, red, rowv);
    else bits_rows<BN, false, TM>(a, t, acc, red, rowv);
  } else if (EPI == EPI_SOFTMAX_EXP) {
    if (masked) softmax_exp_rows<BN, true, TM>(a, t, acc, red, rowv);
    else softmax_exp_rows<BN, false, TM>(a, t, acc, red, rowv);
  } else {
    if (masked) value_rows<BN, EPI, true, TM>(a, t, acc, red, rowv);
    else value_rows<BN, EPI, false, TM>(a, t, acc, red, rowv);
  }
  __syncthreads();
  if (tid < TM && m0 + tid < M) {
    const int ml = tid;
    float v0, v1;
    if (EPI == EPI_LOSS || EPI == EPI_LOSS_BITS) {
      v0 = red[0][ml][0] + red[1][ml][0];
      v1 = red[0][ml][1] + red[1][ml][1];
    } else if (EPI == EPI_SOFTMAX_EXP) {
      v0 = fmaxf(red[0][ml][0], red[1][ml][0]);
      v1 = red[0][ml][1] + red[1][ml][1];
    } else {
      const float ma = red[0][ml][0], mb = red[1][ml][0];
      const float mx = fmaxf(ma, mb);
      v0 = mx;
      v1 = (mx == -INFINITY) ? 0.0f
                             : (ma == -INFINITY ? 0.0f : red[0][ml][1] * expf(ma - mx)) +
                                   (mb == -INFINITY ? 0.0f : red[1][ml][1] * expf(mb - mx));
    }
    float* rp = a.rowpart + (((int64_t)(c * 2 + side) * a.C + m0 + ml) * a.nct + t.tn) * 2;
    rp[0] = v0;
    rp[1] = v1;
  }
}


// The 128 x 128 tile held as four 64 x 64 wave blocks in the matrix-instruction
// layout (acc[i][j][r] is row 16 i + 4 g + r, column 16 j + l16 of the block of
// wave (wm, wn)) becomes its transpose: wave (wm, wn) ends with block (wn, wm)
// transposed.  The two off-diagonal waves swap through LDS first, then the two
// diagonal ones transpose in place; a block passes through a [64][68] float32
// slot (rows padded so that the 4-byte writes and 16-byte reads meet distinct
// banks).  L: kTransposeFloats floats.  Every wave of the workgroup calls it.
constexpr int kTransposeLd = 68;
constexpr int kTransposeFloats = 2 * 64 * kTransposeLd;
__device__ __forceinline__ void transpose_tile(v4f (&acc)[4][4], float* L, int wm, int wn, int l16, int g) {
  constexpr int LD = kTransposeLd;
  const bool off = wm != wn;
#pragma unroll
  for (int phase = 0; phase < 2; ++phase) {
    const bool mine = (phase == 0) == off;
    if (mine) {
      float* s = L + wm * 64 * LD;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) s[(16 * i + 4 * g + r) * LD + 16 * j + l16] = acc[i][j][r];
    }
    __syncthreads();
    if (mine) {
      const float* s = L + wn * 64 * LD;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = *(const v4f*)(s + (16 * j + l16) * LD + 16 * i + 4 * g);
    }
    __syncthreads();
  }
}

// One 128 x BN output tile of A . B with bf16 operands (B in PL planes).
template <int BN, int AMODE, int EPI, int PL>
__device__ __forceinline__ void gemm_bf16_tile(const GemmArgsH& a, int tiles_n, int tiles_m, int nwg, int id,
                                               SmemH<BN, PL>& sm) {
  constexpr int WN = BN / 2;
  constexpr int JN = WN / 16;
  using TA = TileH<BM, AMODE>;
  using TB = TileH<BN, GA_KC>;
  auto& As = sm.As;
  auto& Bs = sm.Bs;
  TileGeo t;
  if (!tile_geo<BN, EPI>(a, tiles_n, tiles_m, nwg, id, t)) return;
  if (EPI != EPI_STORE) load_rowv<EPI>(a, t, sm.rowv);
  const int c = t.c, side = t.side, M = t.M, N = t.N, K = t.K, m0 = t.m0, n0 = t.n0;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int l16 = lane & 15, g = lane >> 4;

  const rsrc_t ra_s = make_rsrc(a.A + c * a.a_cs + side * a.a_ss);
  const rsrc_t rb_s = make_rsrc(a.B + c * a.b_cs + side * a.b_ss);

  v4f acc[4][JN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < JN; ++j) acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};

  // one plane resource per B piece (planes b_ps elements apart)
  rsrc_t rb[PL];
  rb[0] = rb_s;
#pragma unroll
  for (int p = 1; p < PL; ++p) rb[p] = make_rsrc(a.B + p * a.b_ps + c * a.b_cs + side * a.b_ss);

  u32x4 pa[TA::LOADS], pb[PL][TB::LOADS];
  const int nk = (K + BK - 1) / BK;
  TA::load(pa, ra_s, a.lda, m0, M, 0, K, tid);
#pragma unroll
  for (int p = 0; p < PL; ++p) TB::load(pb[p], rb[p], a.ldb, n0, N, 0, K, tid);
  TA::store(As[0], pa, tid, m0, 0, K);
#pragma unroll
  for (int p = 0; p < PL; ++p) TB::store(Bs[0][p], pb[p], tid, n0, 0, K);
  __syncthreads();

  // fragment offsets: row 16 i + l16 of the wave's block, group g (the
  // swizzle repeats every 16 rows)
  const int fa0 = swz(64 * wm + l16, g), fb0 = swz(WN * wn + l16, g);
  constexpr int NB = SmemH<BN, PL>::NB;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = NB == 2 ? (kt & 1) : 0;
    if (kt + 1 < nk) {
      TA::load(pa, ra_s, a.lda, m0, M, (kt + 1) * BK, K, tid);
#pragma unroll
      for (int p = 0; p < PL; ++p) TB::load(pb[p], rb[p], a.ldb, n0, N, (kt + 1) * BK, K, tid);
    }
    const uint16_t* as = As[buf];
    v8bf af[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) af[i] = *(const v8bf*)(as + fa0 + 16 * i * BK);
#pragma unroll
    for (int p = 0; p < PL; ++p) {
      const uint16_t* bs = Bs[buf][p];
      v8bf bf[JN];
#pragma unroll
      for (int j = 0; j < JN; ++j) bf[j] = *(const v8bf*)(bs + fb0 + 16 * j * BK);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < JN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) {
      // one buffer: every wave is done reading it before it is overwritten
      if (NB == 1) __syncthreads();
      const int nbuf = NB == 2 ? (buf ^ 1) : 0;
      TA::store(As[nbuf], pa, tid, m0, (kt + 1) * BK, K);
#pragma unroll
      for (int p = 0; p < PL; ++p) TB::store(Bs[nbuf][p], pb[p], tid, n0, (kt + 1) * BK, K);
    }
    __syncthreads();
  }

  tile_epilogue<BN, EPI>(a, t, acc, sm.red, sm.rowv);
}

// ---- float32 score contraction on the bf16 instructions --------------------
// S = Q . N^T with both operands float32: each element is split exactly into
// three bf16 pieces (x = h + m + l, as in split3_pair) when its tile is stored to
// LDS, and the tile is the sum of the piece products.  NPROD = 9 takes all
// nine, so every product is exact and only the float32 sums round; NPROD = 6
// leaves out m.l, l.m and l.l, whose sum is at most about 2^-23 |a| |b| per
// term (|m| <= 2^-8 |x|, |l| <= 2^-16 |x|), below the rounding bound of a
// float32 dot product of the same length.

// TX rows x 32 k of a float32 [x][k] matrix (k contiguous, ld floats): each
// thread moves groups of eight floats (two 16-byte loads) and stores their
// three pieces to three LDS planes (swizzled [row][k] bf16 tiles).
template <int TX>
struct TileS {
  static constexpr int LOADS = TX * BK / 8 / 256;   // groups of eight per thread

  __device__ __forceinline__ static void load(v4f* r, rsrc_t rs, int ld, int x0, int xdim, int k0, int kdim, int tid) {
    const int k4 = (kdim + 3) & ~3;
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int f = tid + 256 * q;
      const int x = f >> 2, kq = f & 3;
      const int gx = x0 + x, gk = k0 + 8 * kq;
      uint32_t o0 = OOB, o1 = OOB;
      if (gx < xdim) {
        const uint32_t base = (uint32_t)(((int64_t)gx * ld + gk) * 4);
        if (gk < k4) o0 = base;
        if (gk + 4 < k4) o1 = base + 16;
      }
      r[2 * q] = __builtin_amdgcn_raw_buffer_load_b128(rs, o0, 0, 0);
      r[2 * q + 1] = __builtin_amdgcn_raw_buffer_load_b128(rs, o1, 0, 0);
    }
  }

  // this thread's byte offsets at k = 0 (OOB for rows past xdim): a slice
  // that lies wholly inside k then loads at base + 4 k0, the k0 part as the
  // scalar offset, with no per-slice address arithmetic
  __device__ __forceinline__ static void bases(uint32_t* base, int ld, int x0, int xdim, int tid) {
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int f = tid + 256 * q;
      const int gx = x0 + (f >> 2);
      base[q] = gx < xdim ? (uint32_t)(((int64_t)gx * ld + 8 * (f & 3)) * 4) : OOB;
    }
  }

  __device__ __forceinline__ static void load_full(v4f* r, rsrc_t rs, const uint32_t* base, int k0) {
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      r[2 * q] = __builtin_amdgcn_raw_buffer_load_b128(rs, base[q], 4 * k0, 0);
      r[2 * q + 1] = __builtin_amdgcn_raw_buffer_load_b128(rs, base[q] + 16, 4 * k0, 0);
    }
  }

  __device__ __forceinline__ static void store(uint16_t (*s)[TX * BK], const v4f* r, int tid) {
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int f = tid + 256 * q;
      const int x = f >> 2, kq = f & 3;
      const float v[8] = {r[2 * q].x, r[2 * q].y, r[2 * q].z, r[2 * q].w,
                          r[2 * q + 1].x, r[2 * q + 1].y, r[2 * q + 1].z, r[2 * q + 1].w};
      uint32_t pc[3][4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint32_t pp[3];
        split3_pair(v[2 * i], v[2 * i + 1], pp);
#pragma unroll
        for (int p = 0; p < 3; ++p) pc[p][i] = pp[p];
      }
      const int o = swz(x, kq);
#pragma unroll
      for (int p = 0; p < 3; ++p) *(u32x4*)(s[p] + o) = (u32x4){pc[p][0], pc[p][1], pc[p][2], pc[p][3]};
    }
  }
};

// one LDS buffer of three A and three B planes (single-buffered, so that
// three workgroups fit a CU), and the row partials; rowv1: the per-row values
// of side 1's rows of a shared tile
template <int TM>
struct SmemST {
  uint16_t As[3][TM * BK];
  uint16_t Bs[3][128 * BK];
  float red[2][TM][2];
  float rowv[2][TM];
  float rowv1[2][TM];
};
using SmemS = SmemST<BM>;


// Score tile body: four waves of 64 x 64.  One A plane and one B plane in
// registers at a time (B planes are read again for each A plane).
template <int EPI, int NPROD>
__device__ __forceinline__ void score_split_body(const GemmArgsH& a, int tiles_n, int tiles_m) {
  constexpr int BN = 128, WN = 64, JN = 4, WMR = BM / 2, IM = BM / 32;
  __shared__ __align__(16) SmemS sm;
  static_assert(sizeof(sm.As) + sizeof(sm.Bs) >= kTransposeFloats * sizeof(float), "transpose slots");
  TileGeo t;
  if (!tile_geo<BN, EPI>(a, tiles_n, tiles_m, gridDim.x, blockIdx.x, t)) return;
  if (EPI != EPI_STORE) load_rowv<EPI>(a, t, sm.rowv);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int l16 = lane & 15, g = lane >> 4;

  const rsrc_t ra = make_rsrc(a.Af + t.c * a.a_cs + t.side * a.a_ss);
  const rsrc_t rb = make_rsrc(a.Bf + t.c * a.b_cs + t.side * a.b_ss);
  v4f acc[IM][JN];
#pragma unroll
  for (int i = 0; i < IM; ++i)
#pragma unroll
    for (int j = 0; j < JN; ++j) acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};

  v4f pa[2 * TileS<BM>::LOADS], pb[2 * TileS<BN>::LOADS];
  const int nk = (t.K + BK - 1) / BK;
  TileS<BM>::load(pa, ra, a.lda, t.m0, t.M, 0, t.K, tid);
  TileS<BN>::load(pb, rb, a.ldb, t.n0, t.N, 0, t.K, tid);
  TileS<BM>::store(sm.As, pa, tid);
  TileS<BN>::store(sm.Bs, pb, tid);
  __syncthreads();

  const int fa0 = swz(WMR * wm + l16, g), fb0 = swz(WN * wn + l16, g);
  uint32_t abase[TileS<BM>::LOADS], bbase[TileS<BN>::LOADS];
  TileS<BM>::bases(abase, a.lda, t.m0, t.M, tid);
  TileS<BN>::bases(bbase, a.ldb, t.n0, t.N, tid);
  // slices wholly inside k (rounded up to 4, the zero-padded row length)
  const int kfull = ((t.K + 3) & ~3) / BK;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < kfull) {
      TileS<BM>::load_full(pa, ra, abase, (kt + 1) * BK);
      TileS<BN>::load_full(pb, rb, bbase, (kt + 1) * BK);
    } else if (kt + 1 < nk) {
      TileS<BM>::load(pa, ra, a.lda, t.m0, t.M, (kt + 1) * BK, t.K, tid);
      TileS<BN>::load(pb, rb, a.ldb, t.n0, t.N, (kt + 1) * BK, t.K, tid);
    }
#pragma unroll
    for (int pa_ = 0; pa_ < 3; ++pa_) {
      v8bf af[IM];
#pragma unroll
      for (int i = 0; i < IM; ++i) af[i] = *(const v8bf*)(sm.As[pa_] + fa0 + 16 * i * BK);
#pragma unroll
      for (int pb_ = 0; pb_ < 3; ++pb_) {
        if (NPROD == 6 && pa_ + pb_ > 2) continue;
        v8bf bf[JN];
#pragma unroll
        for (int j = 0; j < JN; ++j) bf[j] = *(const v8bf*)(sm.Bs[pb_] + fb0 + 16 * j * BK);
#pragma unroll
        for (int i = 0; i < IM; ++i)
#pragma unroll
          for (int j = 0; j < JN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
      }
    }
    if (kt + 1 < nk) {
      __syncthreads();
      TileS<BM>::store(sm.As, pa, tid);
      TileS<BN>::store(sm.Bs, pb, tid);
      __syncthreads();
    }
  }
  // a full side-0 tile inside the in-chunk block also gives side 1's tile
  // (tm, tn) -> (tn, tm), its transpose (M = the chunk's edges here): a second
  // pass of the same epilogue on the transposed accumulators
  const bool shared = a.share_cc && t.side == 0 && t.m0 / BM < t.M / BM && t.tn < t.M / BN;
  for (int pass = 0; pass < (shared ? 2 : 1); ++pass) {
    if (pass == 1) {
      t.side = 1;
      const int m0 = t.m0;
      t.m0 = t.n0;
      t.n0 = m0;
      t.tn = m0 / BN;
      if (EPI != EPI_STORE) load_rowv<EPI>(a, t, sm.rowv1);   // visible after the transpose's barriers
      // every wave is past the first pass's barrier, so past its last reads of the planes
      transpose_tile(acc, reinterpret_cast<float*>(&sm.As[0][0]), wm, wn, l16, g);
    }
    tile_epilogue<BN, EPI>(a, t, acc, sm.red, pass ? sm.rowv1 : sm.rowv);
  }
}

// The ranking-bits epilogue keeps register use low enough for three waves per
// SIMD (a few spill slots, one 16-byte slot in the k loop), which pays for the
// short k loop of d = 128; the value epilogues spill more and run at two.
template <int EPI, int NPROD>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 3))) void score_split_kernel3(
    GemmArgsH a, int tiles_n, int tiles_m) {
  score_split_body<EPI, NPROD>(a, tiles_n, tiles_m);
}

template <int EPI, int NPROD>
__global__ __launch_bounds__(256) void score_split_kernel(GemmArgsH a, int tiles_n, int tiles_m) {
  score_split_body<EPI, NPROD>(a, tiles_n, tiles_m);
}

// ---- float32 backward products of a general dS on the bf16 instructions ----
// dQ = dS . N and dN = dS^T . Q for the logistic and softmax losses: dS is
// float32, so it is split into its three pieces on the way into LDS like the
// score operands, B comes as the three transposed planes of N or Q, and the
// six products hh, hm, mh, hl, mm, lh are summed (as in the score).

// TX rows (m) x 32 k of a float32 [k][m] matrix (m contiguous, ld floats):
// each thread loads two consecutive k rows of four consecutive m, splits the
// pairs (k, k + 1) of each m and stores them as one 32-bit word per plane
// into the [m][k] tile.
template <int TX>
struct TileSM {
  static constexpr int LOADS = TX * BK / 8 / 256;   // (k pair, m quad) per thread

  __device__ __forceinline__ static void load(v4f* r, rsrc_t rs, int ld, int x0, int xdim, int k0, int kdim,
                                              int tid) {
    const int x4 = (xdim + 3) & ~3;
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int f = tid + 256 * q;
      const int kp = f / (TX / 4), xq = f % (TX / 4);
      const int gk = k0 + 2 * kp, gx = x0 + 4 * xq;
      uint32_t o0 = OOB, o1 = OOB;
      if (gx < x4) {
        if (gk < kdim) o0 = (uint32_t)(((int64_t)gk * ld + gx) * 4);
        if (gk + 1 < kdim) o1 = (uint32_t)(((int64_t)(gk + 1) * ld + gx) * 4);
      }
      r[2 * q] = __builtin_amdgcn_raw_buffer_load_b128(rs, o0, 0, 0);
      r[2 * q + 1] = __builtin_amdgcn_raw_buffer_load_b128(rs, o1, 0, 0);
    }
  }

  __device__ __forceinline__ static void store(uint16_t (*s)[TX * BK], const v4f* r, int tid) {
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int f = tid + 256 * q;
      const int kp = f / (TX / 4), xq = f % (TX / 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint32_t pc[3];
        split3_pair(r[2 * q][i], r[2 * q + 1][i], pc);
        const int o = swz(4 * xq + i, kp >> 2) + ((2 * kp) & 7);
#pragma unroll
        for (int p = 0; p < 3; ++p) *(uint32_t*)(s[p] + o) = pc[p];
      }
    }
  }
};

// One 128 x 128 output tile of dS . B (AF = 0: dS rows, A = dS [m][k]) or
// dS^T . B (AF = 1: A[m][k] = dS[k][m]); one LDS buffer.  SM: softmax, dS is
// formed as A is staged, dS[e][t] = exp(s[e][t] - lse[e]) on the valid
// candidates t (t < Nc, t != e) of the valid rows e (e < Cc), else 0: the A
// source holds exp(s - M) per score tile (0 off the valid set) and each row
// is scaled by exp(M - lse) of its tile.
template <int AF, bool SM>
__device__ __forceinline__ void gemm_split_tile(const GemmArgsH& a, int tiles_n, int tiles_m, int nwg, int id,
                                                SmemS& sm) {
  constexpr int BN = 128, WN = 64, JN = 4;
  using TB = TileH<BN, GA_KC>;
  TileGeo t;
  if (!tile_geo<BN, EPI_STORE>(a, tiles_n, tiles_m, nwg, id, t)) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int l16 = lane & 15, g = lane >> 4;
  const rsrc_t ra = make_rsrc(a.Af + t.c * a.a_cs + t.side * a.a_ss);
  rsrc_t rb[3];
#pragma unroll
  for (int p = 0; p < 3; ++p) rb[p] = make_rsrc(a.B + p * a.b_ps + t.c * a.b_cs + t.side * a.b_ss);
  v4f acc[4][JN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < JN; ++j) acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};

  constexpr int AQ = AF == 0 ? TileS<BM>::LOADS : TileSM<BM>::LOADS;   // A groups per thread
  v4f pa[2 * AQ];
  u32x4 pb[3][TB::LOADS];
  // softmax: the scale exp(M - lse) of this thread's rows in the score tile
  // of the staged slice (AF = 0: one row per group, the tile of the slice's
  // columns, reloaded when the slice enters a new tile; AF = 1: two rows per
  // group, the tile of this output tile's rows)
  static_assert(BM == PBG_SCORE_BN && BK <= PBG_SCORE_BN, "slices and tiles within one score tile");
  const int Cc = AF == 0 ? t.M : t.K;
  const float* rsc = SM ? a.smscale + (int64_t)(t.c * 2 + t.side) * a.nct * a.C : nullptr;
  float lr[2 * AQ];
  const int nk = (t.K + BK - 1) / BK;
  auto load_a = [&](int k0) {
    if (AF == 0) {
      TileS<BM>::load(pa, ra, a.lda, t.m0, t.M, k0, t.K, tid);
      if (SM && (k0 & 127) == 0) {
        const float* rc = rsc + (int64_t)(k0 >> 7) * a.C;
#pragma unroll
        for (int q = 0; q < AQ; ++q) {
          const int e = t.m0 + ((tid + 256 * q) >> 2);
          lr[q] = e < Cc ? rc[e] : 0.0f;
        }
      }
    } else {
      TileSM<BM>::load(pa, ra, a.lda, t.m0, t.M, k0, t.K, tid);
      if (SM) {
        const float* rc = rsc + (int64_t)(t.m0 >> 7) * a.C;
#pragma unroll
        for (int q = 0; q < AQ; ++q) {
          const int e = k0 + 2 * ((tid + 256 * q) / (BM / 4));
          lr[2 * q] = e < Cc ? rc[e] : 0.0f;
          lr[2 * q + 1] = e + 1 < Cc ? rc[e + 1] : 0.0f;
        }
      }
    }
  };
  auto softmax_a = [&]() {
#pragma unroll
    for (int q = 0; q < AQ; ++q) {
      if (AF == 0) {
        pa[2 * q] *= lr[q];
        pa[2 * q + 1] *= lr[q];
      } else {
        pa[2 * q] *= lr[2 * q];
        pa[2 * q + 1] *= lr[2 * q + 1];
      }
    }
  };
  auto store_a = [&]() {
    if (SM) softmax_a();
    if (AF == 0) TileS<BM>::store(sm.As, pa, tid);
    else TileSM<BM>::store(sm.As, pa, tid);
  };
  load_a(0);
#pragma unroll
  for (int p = 0; p < 3; ++p) TB::load(pb[p], rb[p], a.ldb, t.n0, t.N, 0, t.K, tid);
  store_a();
#pragma unroll
  for (int p = 0; p < 3; ++p) TB::store(sm.Bs[p], pb[p], tid, 0, 0, 0);
  __syncthreads();

  const int fa0 = swz(64 * wm + l16, g), fb0 = swz(WN * wn + l16, g);
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) {
      load_a((kt + 1) * BK);
#pragma unroll
      for (int p = 0; p < 3; ++p) TB::load(pb[p], rb[p], a.ldb, t.n0, t.N, (kt + 1) * BK, t.K, tid);
    }
#pragma unroll
    for (int pa_ = 0; pa_ < 3; ++pa_) {
      v8bf af[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *(const v8bf*)(sm.As[pa_] + fa0 + 16 * i * BK);
#pragma unroll
      for (int pb_ = 0; pb_ < 3 - pa_; ++pb_) {
        v8bf bf[JN];
#pragma unroll
        for (int j = 0; j < JN; ++j) bf[j] = *(const v8bf*)(sm.Bs[pb_] + fb0 + 16 * j * BK);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < JN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
      }
    }
    if (kt + 1 < nk) {
      __syncthreads();
      store_a();
#pragma unroll
      for (int p = 0; p < 3; ++p) TB::store(sm.Bs[p], pb[p], tid, 0, 0, 0);
      __syncthreads();
    }
  }
  tile_epilogue<BN, EPI_STORE>(a, t, acc, sm.red, sm.rowv);
}

// dQ (workgroups [0, nwg0)) and dN (the rest) of a step in one launch
template <bool SM>
__global__ __launch_bounds__(256) void gemm_split_pair_kernel(GemmArgsH a0, int tn0, int tm0, int nwg0,
                                                              GemmArgsH a1, int tn1, int tm1) {
  __shared__ __align__(16) SmemS sm;
  const int id = blockIdx.x;
  if (id < nwg0) gemm_split_tile<0, SM>(a0, tn0, tm0, nwg0, id, sm);
  else gemm_split_tile<1, SM>(a1, tn1, tm1, (int)gridDim.x - nwg0, id - nwg0, sm);
}

template <int BN, int AMODE, int EPI, int PL>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgsH a, int tiles_n, int tiles_m) {
  __shared__ __align__(16) SmemH<BN, PL> sm;
  gemm_bf16_tile<BN, AMODE, EPI, PL>(a, tiles_n, tiles_m, gridDim.x, blockIdx.x, sm);
}

// two independent products in one launch (dQ and dN of a step): workgroups
// [0, nwg0) take the first, the rest the second, so that the long-k tiles of
// the first start first and the short ones of the second fill in behind them
template <int BN, int AM0, int AM1, int PL>
__global__ __launch_bounds__(256) void gemm_bf16_pair_kernel(GemmArgsH a0, int tn0, int tm0, int nwg0,
                                                             GemmArgsH a1, int tn1, int tm1) {
  __shared__ __align__(16) SmemH<BN, PL> sm;
  const int id = blockIdx.x;
  if (id < nwg0) gemm_bf16_tile<BN, AM0, EPI_STORE, PL>(a0, tn0, tm0, nwg0, id, sm);
  else gemm_bf16_tile<BN, AM1, EPI_STORE, PL>(a1, tn1, tm1, (int)gridDim.x - nwg0, id - nwg0, sm);
}

// ---- ranking backward with dS as bits: 256-row tiles, B through LDS DMA ---
// dQ = dS . N (AF = 0: A = dS rows from the bit matrix) and dN = dS^T . Q
// (AF = 1: A = dS columns) with B as PL bf16 planes [n][k].  A workgroup
// computes a 256 x BN tile as four waves of 128 x BN/2, so every B fragment
// read from LDS feeds eight matrix instructions.  dS takes no LDS: each lane
// loads the bits of its own eight A fragments (16 rows x 8 k each) straight
// into registers one slice ahead and expands them to 0 / 1 bf16.  B moves
// global -> LDS without registers (buffer loads with the LDS flag, 16 bytes a
// lane) into a two-stage ring, so the next slice streams in while this one's
// matrix instructions run, one barrier per slice.  The products and their
// order per output element are those of gemm_bf16_tile (k slices in order,
// planes in order), so the results are identical.
constexpr int BT = 256;   // rows of a bits-backward tile

template <int BN, int PL>
struct SmemD {
  uint16_t Bs[2][PL][BN * BK];
  uint16_t Ab[2][2 * BT];   // the slice's bit-matrix words (see dma_bits)
  uint16_t Ab1[2][2 * BT];  // merged dQ rows: the other side's words read by columns
  float red[2][BT][2];
  float rowv[2][BT];
};

// One plane's BN x BK tile of B into LDS at dst: wave w moves rows
// [16 w + 64 j, +16) for j < BN / 64, lane L the 16-byte group L % 4 of row
// L / 4 as the swizzle places it (the lane loads logical group
// (L % 4) ^ f(row)); rows past xdim and k past kdim (rounded to 8) read zeros.
template <int BN>
__device__ __forceinline__ void dma_b_tile(uint16_t* dst, rsrc_t rs, int ld, int x0, int xdim, int k0, int kdim,
                                           int w, int lane) {
  const int k8 = (kdim + 7) & ~7;
#pragma unroll
  for (int j = 0; j < BN / 64; ++j) {
    const int xr = 16 * w + 64 * j;
    const int x = xr + (lane >> 2);
    const int q = (lane & 3) ^ (((x >> 1) ^ ((x >> 3) & 1)) & 3);
    const int gx = x0 + x, gk = k0 + 8 * q;
    const uint32_t off = (gx < xdim && gk < k8) ? (uint32_t)(((int64_t)gx * ld + gk) * 2) : OOB;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(dst + xr * BK), 16, off,
                                             0, 0, 0);
  }
}

// The bit-matrix words of one slice (k0 .. k0 + 31) of a 256-row tile, 1 KB,
// into LDS: each wave moves 256 bytes, four bytes a lane.
//   AF = 0 (rows of dS): the two word columns k0 / 16, + 1 for rows
//          m0 .. m0 + 255; wave w: column k0 / 16 + w / 2, rows
//          m0 + 128 (w % 2) + 2 lane, + 1; LDS word (w / 2) 256 + row
//   AF = 1 (columns of dS): word columns m0 / 16 .. + 15, rows k0 .. k0 + 31;
//          wave w: columns 4 w + lane / 16, rows k0 + 2 (lane % 16), + 1;
//          LDS word 32 column + row
// The lane's byte offset at k0 = 0 is fixed for the tile (OOB past the
// matrix); soff moves it to the slice.
__device__ __forceinline__ void dma_bits(uint16_t* dst, rsrc_t rs, uint32_t off, int soff, int w) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(dst + 128 * w), 4, off,
                                           soff, 0, 0);
}

template <int AF>
__device__ __forceinline__ uint32_t bits_offset(int ld, int m0, int mdim, int kdim, int k0, int w, int lane) {
  if (AF == 0) {
    const int r = m0 + 128 * (w & 1) + 2 * lane;
    return r < mdim ? (uint32_t)(((int64_t)(w >> 1) * ld + r) * 2) : OOB;
  }
  const int wc = (m0 >> 4) + 4 * w + (lane >> 4);
  const int k = k0 + 2 * (lane & 15);
  return (16 * wc < mdim && k < kdim) ? (uint32_t)(((int64_t)wc * ld + 2 * (lane & 15)) * 2) : OOB;
}

// this lane's fragment i of the slice in LDS -> eight bf16 0 / 1 (AF = 0:
// row 16 i + l16 of the wave's 128, k = 8 g .. + 7; AF = 1: candidate
// 16 i + l16 of the wave's 128, rows 8 g .. + 7 of the slice, nv of them
// inside the chunk)
// AF = 0 looks the fragment's byte up in lut (entry b: the eight bf16 0 / 1
// of the bits of b, bit 0 first; see fill_bits_lut).
template <int AF, bool TAIL>
__device__ __forceinline__ v8bf expand_bits_frag(const uint16_t* ab, const u32x4* lut, int wm, int i, int l16, int g,
                                                 int nv) {
  u32x4 v;
  if (AF == 0) {
    const uint32_t word = ab[(g >> 1) * 256 + 128 * wm + 16 * i + l16];
    v = lut[__builtin_amdgcn_ubfe(word, 8 * (g & 1), 8)];
  } else {
    v = *(const u32x4*)(ab + (8 * wm + i) * 32 + 8 * g);
    const int b = l16;
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = ((v[q] >> b) & 0x00010001u) * 0x3F80u;
    if (TAIL && nv < 8) {
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] &= (2 * q + 1 < nv) ? 0xFFFFFFFFu : (2 * q < nv ? 0xFFFFu : 0u);
    }
  }
  return __builtin_bit_cast(v8bf, v);
}

// the 256 expansions of a byte of dS bits, one per thread of the workgroup
__device__ __forceinline__ void fill_bits_lut(u32x4* lut) {
  const uint32_t b = threadIdx.x;
  lut[b] = (u32x4){bit_pair(b & 3), bit_pair((b >> 2) & 3), bit_pair((b >> 4) & 3), bit_pair(b >> 6)};
}

// Merged dQ rows: each element of A is a count c in {0, 1, 2} (the bit of this
// side's dS row plus the bit of the other side's dS column), whose bf16 value
// 0, 1.0 (0x3F80) or 2.0 (0x4000) comes out of one byte permute: the selector
// of an element pair is 0x03000300 + c0 * 0x0101 + c1 * 0x01010000 (low byte
// c, high byte 3 + c) over the table bytes {00 80 00 | 00 3F 40}.
constexpr uint32_t kCountLo = 0x00008000u, kCountHi = 0x0000403Fu;
__device__ __forceinline__ void fill_count_lut(u32x4* lut) {
  const uint32_t b = threadIdx.x;
  u32x4 v;
#pragma unroll
  for (int q = 0; q < 4; ++q) v[q] = 0x03000300u + (((((b >> (2 * q)) & 3u) * 0x8001u) & 0x10001u) * 0x0101u);
  lut[b] = v;
}

// fragment i of a merged slice: this side's row bits (by byte, from lutc) plus
// the other side's column bits (AF = 1 layout in ab1, TAIL: only nv of the
// eight k inside the chunk)
template <bool TAIL>
__device__ __forceinline__ v8bf expand_count_frag(const uint16_t* ab, const uint16_t* ab1, const u32x4* lutc, int wm,
                                                  int i, int l16, int g, int nv) {
  const uint32_t word = ab[(g >> 1) * 256 + 128 * wm + 16 * i + l16];
  u32x4 sel = lutc[__builtin_amdgcn_ubfe(word, 8 * (g & 1), 8)];
  const u32x4 v = *(const u32x4*)(ab1 + (8 * wm + i) * 32 + 8 * g);
  u32x4 out;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    uint32_t e = ((v[q] >> l16) & 0x00010001u) * 0x0101u;
    if (TAIL) e &= (2 * q + 1 < nv) ? 0xFFFFFFFFu : (2 * q < nv ? 0xFFFFu : 0u);
    out[q] = __builtin_amdgcn_perm(kCountHi, kCountLo, sel[q] + e);
  }
  return __builtin_bit_cast(v8bf, out);
}

// MERGE (AF = 0, a.merge_cc): the merged dQ rows described at GemmArgsH; the
// slices k < Cc take the other side's column bits too (counts, lutc).
template <int BN, int AF, int PL, bool MERGE>
__device__ __forceinline__ void gemm_bits_tile(const GemmArgsH& a, int tiles_n, int tiles_m, int nwg, int id,
                                               SmemD<BN, PL>& sm, u32x4* lut, u32x4* lutc) {
  constexpr int WN = BN / 2, WMR = BT / 2;
  constexpr int JN = WN / 16, IM = WMR / 16;
  TileGeo t;
  if (!tile_geo<BN, EPI_STORE, BT>(a, tiles_n, tiles_m, nwg, id, t)) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int l16 = lane & 15, g = lane >> 4;
  const rsrc_t ra = make_rsrc(a.A + t.c * a.a_cs + t.side * a.a_ss);
  rsrc_t rb[PL];
#pragma unroll
  for (int p = 0; p < PL; ++p) rb[p] = make_rsrc(a.B + p * a.b_ps + t.c * a.b_cs + t.side * a.b_ss);

  v4f acc[IM][JN];
#pragma unroll
  for (int i = 0; i < IM; ++i)
#pragma unroll
    for (int j = 0; j < JN; ++j) acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};

  const int nk = (t.K + BK - 1) / BK;
  // bytes per slice of the bit-matrix DMA; the lane's offset is fixed except
  // in a ragged last slice of the AF = 1 rows
  const int a_step = AF == 0 ? 4 * a.lda : 2 * BK;
  uint32_t aoff = bits_offset<AF>(a.lda, t.m0, t.M, t.K, 0, w, lane);
  if (AF == 0) fill_bits_lut(lut);   // visible after the barrier below
  if (MERGE) fill_count_lut(lutc);
  dma_bits(sm.Ab[0], ra, aoff, 0, w);
  // merged rows: the other side's matrix by columns, rows k < kc = Cc (the dQ
  // tile's M)
  const rsrc_t ra1 = MERGE ? make_rsrc(a.A + t.c * a.a_cs + (1 - t.side) * a.a_ss) : ra;
  const int kc = MERGE ? t.M : 0;
  const int nk1 = (kc + BK - 1) / BK;
  uint32_t aoff1 = MERGE ? bits_offset<1>(a.lda, t.m0, t.M, kc, 0, w, lane) : 0;
  if (MERGE && nk1 > 0) dma_bits(sm.Ab1[0], ra1, aoff1, 0, w);
#pragma unroll
  for (int p = 0; p < PL; ++p) dma_b_tile<BN>(sm.Bs[0][p], rb[p], a.ldb, t.n0, t.N, 0, t.K, w, lane);
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this wave's loads have landed
  __syncthreads();

  const int fb0 = swz(WN * wn + l16, g);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    v8bf af[IM];
    const int nv = t.K - (kt * BK + 8 * g);
    // rows of dS past the chunk's edges (AF = 1) are masked in a slice that
    // reaches them only: the check is uniform, the masks are per lane
    if (MERGE && kt < nk1) {
      const int nv1 = kc - (kt * BK + 8 * g);
      if ((kt + 1) * BK > kc) {
#pragma unroll
        for (int i = 0; i < IM; ++i) af[i] = expand_count_frag<true>(sm.Ab[buf], sm.Ab1[buf], lutc, wm, i, l16, g, nv1);
      } else {
#pragma unroll
        for (int i = 0; i < IM; ++i) af[i] = expand_count_frag<false>(sm.Ab[buf], sm.Ab1[buf], lutc, wm, i, l16, g, nv1);
      }
    } else if (AF == 1 && (kt + 1) * BK > t.K) {
#pragma unroll
      for (int i = 0; i < IM; ++i) af[i] = expand_bits_frag<AF, true>(sm.Ab[buf], lut, wm, i, l16, g, nv);
    } else {
#pragma unroll
      for (int i = 0; i < IM; ++i) af[i] = expand_bits_frag<AF, false>(sm.Ab[buf], lut, wm, i, l16, g, nv);
    }
    if (kt + 1 < nk) {
      if (AF == 1 && kt + 2 == nk) aoff = bits_offset<AF>(a.lda, t.m0, t.M, t.K, (kt + 1) * BK, w, lane);
      dma_bits(sm.Ab[buf ^ 1], ra, aoff, (kt + 1) * a_step, w);
      if (MERGE && kt + 1 < nk1) {
        if (kt + 2 == nk1) aoff1 = bits_offset<1>(a.lda, t.m0, t.M, kc, (kt + 1) * BK, w, lane);
        dma_bits(sm.Ab1[buf ^ 1], ra1, aoff1, (kt + 1) * 2 * BK, w);
      }
#pragma unroll
      for (int p = 0; p < PL; ++p)
        dma_b_tile<BN>(sm.Bs[buf ^ 1][p], rb[p], a.ldb, t.n0, t.N, (kt + 1) * BK, t.K, w, lane);
    }
#pragma unroll
    for (int p = 0; p < PL; ++p) {
      const uint16_t* bs = sm.Bs[buf][p];
      v8bf bf[JN];
#pragma unroll
      for (int j = 0; j < JN; ++j) bf[j] = *(const v8bf*)(bs + fb0 + 16 * j * BK);
#pragma unroll
      for (int i = 0; i < IM; ++i)
#pragma unroll
        for (int j = 0; j < JN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    // the matrix instructions issue before the wait, so the loads of the next
    // slice overlap them; then every wave's loads have landed and every wave
    // is done with this buffer before it is refilled
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();
  }
  tile_epilogue<BN, EPI_STORE, BT>(a, t, acc, sm.red, sm.rowv);
}

template <int BN, int PL>
__global__ __launch_bounds__(256) void gemm_bits_pair_kernel(GemmArgsH a0, int tn0, int tm0, int nwg0,
                                                             GemmArgsH a1, int tn1, int tm1) {
  __shared__ __align__(16) SmemD<BN, PL> sm;
  __shared__ __align__(16) u32x4 lut[256];
  __shared__ __align__(16) u32x4 lutc[256];
  static_assert(sizeof(lut) / sizeof(lut[0]) == 256, "one entry per thread");
  const int id = blockIdx.x;
  if (id < nwg0) {
    if (a0.merge_cc) gemm_bits_tile<BN, 0, PL, true>(a0, tn0, tm0, nwg0, id, sm, lut, lutc);
    else gemm_bits_tile<BN, 0, PL, false>(a0, tn0, tm0, nwg0, id, sm, lut, lutc);
  } else {
    gemm_bits_tile<BN, 1, PL, false>(a1, tn1, tm1, (int)gridDim.x - nwg0, id - nwg0, sm, lut, lutc);
  }
}

// fp32 rows [rows][ld_src] (columns [d, ld_src) zero) of Q and of N -> bf16
// rows [rows][ld_dst] (columns up to kp) and the transposed copy [kp][ld_T]
// (rows [rows, ld_T) zero), both operands in one launch (blockIdx.z < nz0:
// the first).  64 x 64 tiles: 16-byte loads, rounded once, eight bytes per
// thread to the row-major copy and into an LDS tile, then eight consecutive
// rows of one column per 16-byte store of the transposed copy.  ld_src is a
// multiple of 4, ld_dst of 4, ld_T of 8.
struct Bf16T {
  const float* src;
  int64_t src_bs;
  int rows, ld_src;
  uint16_t* dst;
  int64_t dst_bs;
  int ld_dst;
  uint16_t* dstT;
  int64_t dstT_bs;
  int ld_T;
};

__global__ __launch_bounds__(256) void to_bf16_t_kernel(Bf16T o0, Bf16T o1, int nz0, int kp) {
  __shared__ uint16_t tile[64][72];
  const bool first = (int)blockIdx.z < nz0;
  const Bf16T& o = first ? o0 : o1;
  const int b = first ? blockIdx.z : blockIdx.z - nz0;
  const int r0 = blockIdx.y * 64, k0 = blockIdx.x * 64;
  if (r0 >= o.ld_T) return;
  const float* s = o.src + (int64_t)b * o.src_bs;
  uint16_t* dr = o.dst + (int64_t)b * o.dst_bs;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int it = threadIdx.x + 256 * j;
    const int rr = it >> 4, k4 = 4 * (it & 15);
    const int r = r0 + rr, k = k0 + k4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < o.rows && k < o.ld_src) v = *(const float4*)(s + (int64_t)r * o.ld_src + k);
    const uint32_t lo = f2_to_bf16x2(v.x, v.y), hi = f2_to_bf16x2(v.z, v.w);
    *(uint2*)&tile[rr][k4] = make_uint2(lo, hi);
    if (r < o.rows && k < kp) *(uint2*)(dr + (int64_t)r * o.ld_dst + k) = make_uint2(lo, hi);
  }
  __syncthreads();
  uint16_t* dT = o.dstT + (int64_t)b * o.dstT_bs;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int it = threadIdx.x + 256 * j;
    const int kk = it >> 3, r8 = 8 * (it & 7);
    const int k = k0 + kk, r = r0 + r8;
    if (k >= kp || r >= o.ld_T) continue;
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = (uint32_t)tile[r8 + 2 * i][kk] | ((uint32_t)tile[r8 + 2 * i + 1][kk] << 16);
    *(u32x4*)(dT + (int64_t)k * o.ld_T + r) = (u32x4){w[0], w[1], w[2], w[3]};
  }
}

// fp32 rows [rows][ld_src] (columns [d, ld_src) zero) -> the three exact
// bf16 pieces (split3_pair) of every element, transposed: planes [kp][ld_T],
// ps elements apart, rows [rows, rows_p) and columns past ld_src zero.  Two
// operands in one launch (blockIdx.z < nz0: the first).  64 x 64 tiles: each
// thread loads 16-byte groups into an LDS tile, then gathers eight
// consecutive rows of one column and writes 16 bytes per plane (eight lanes
// cover 64 rows of a plane row).  ld_src is a multiple of 4, rows_p and ld_T
// of 8.
struct Split3T {
  const float* src;
  int64_t src_bs;
  int rows, ld_src;
  uint16_t* dst;
  int64_t dst_bs, ps;
  int ld_T, rows_p;
};

// workgroup (bx, by, bz) of the split's grid
__device__ __forceinline__ void split3_t_block(const Split3T& o0, const Split3T& o1, int nz0, int kp, int bx, int by,
                                               int bz) {
  __shared__ float tile[64][65];
  const bool first = bz < nz0;
  const Split3T& o = first ? o0 : o1;
  const int b = first ? bz : bz - nz0;
  const int r0 = by * 64, k0 = bx * 64;
  if (r0 >= o.rows_p) return;
  const float* s = o.src + (int64_t)b * o.src_bs;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int it = threadIdx.x + 256 * j;
    const int rr = it >> 4, k4 = 4 * (it & 15);
    const int r = r0 + rr, k = k0 + k4;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (r < o.rows && k < o.ld_src) v = *(const float4*)(s + (int64_t)r * o.ld_src + k);
    tile[rr][k4] = v.x;
    tile[rr][k4 + 1] = v.y;
    tile[rr][k4 + 2] = v.z;
    tile[rr][k4 + 3] = v.w;
  }
  __syncthreads();
  uint16_t* dst = o.dst + (int64_t)b * o.dst_bs;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int it = threadIdx.x + 256 * j;
    const int kk = it >> 3, r8 = 8 * (it & 7);
    const int k = k0 + kk, r = r0 + r8;
    if (k >= kp || r >= o.rows_p) continue;
    uint32_t pc[4][3];
#pragma unroll
    for (int i = 0; i < 4; ++i) split3_pair(tile[r8 + 2 * i][kk], tile[r8 + 2 * i + 1][kk], pc[i]);
#pragma unroll
    for (int p = 0; p < 3; ++p)
      *(u32x4*)(dst + p * o.ps + (int64_t)k * o.ld_T + r) = (u32x4){pc[0][p], pc[1][p], pc[2][p], pc[3][p]};
  }
}

__global__ __launch_bounds__(256) void split3_t_kernel(Split3T o0, Split3T o1, int nz0, int kp) {
  split3_t_block(o0, o1, nz0, kp, blockIdx.x, blockIdx.y, blockIdx.z);
}

// The finalisation (nfin = fb x nchunks workgroups first) and the transposed
// piece split (gx x gy x gz workgroups after them) in one launch: the split
// reads only the candidate rows, so it need not wait for the finalisation,
// whose short, latency-bound workgroups run beside its streaming ones.
__global__ __launch_bounds__(256) void finalize_split3_t_kernel(StepGeom g, StepBufs b, int softmax_scales,
                                                                double* parts, int fb, int nfin, Split3T o0,
                                                                Split3T o1, int nz0, int kp, int gx, int gy) {
  const int id = blockIdx.x;
  if (id < nfin) {
    finalize_block(g, b, softmax_scales, parts, id / fb, id % fb, fb);
    return;
  }
  const int k = id - nfin;
  split3_t_block(o0, o1, nz0, kp, k % gx, (k / gx) % gy, k / (gx * gy));
}

// softmax row pass in bf16 mode: raw fp32 scores -> dS = softmax (masked),
// written as bf16 rows
__global__ __launch_bounds__(256) void softmax_rows_bf16_kernel(StepGeom g, const float* S, const float* rowpart,
                                                                const float* pos, uint16_t* dsh, int ldh) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int z = blockIdx.y;
  const int c = z >> 1;
  const int Cc = chunk_edges(g, c);
  if (row >= Cc) return;
  const int Nc = Cc + g.U;
  const float p = pos[pos_index(g, c, z & 1, row)];
  const float* rp = rowpart + ((int64_t)z * g.C + row) * g.nct * 2;
  float Mx = p;
  for (int ct = 0; ct < g.nct; ++ct) Mx = fmaxf(Mx, rp[2 * ct]);
  float Z = expf(p - Mx);
  for (int ct = 0; ct < g.nct; ++ct) {
    const float mx = rp[2 * ct];
    if (mx > -INFINITY) Z += rp[2 * ct + 1] * expf(mx - Mx);
  }
  const float lse = Mx + logf(Z);
  const float* srow = S + ((int64_t)z * g.C + row) * g.Np;
  uint16_t* hrow = dsh + ((int64_t)z * g.C) * ldh + (int64_t)row * ldh;
  const int Nh = (Nc + 31) & ~31;
  for (int t = lane; t < Nh; t += 64) {
    float v = 0.0f;
    if (t < Nc && t != row) v = expf(srow[t] - lse);
    hrow[t] = f_to_bf16(v);
  }
}


template <int BN, int AMODE, int EPI, int PL = 1>
void launch_t(const GemmArgsH& a, int tiles_n, int tiles_m, int batches, hipStream_t s) {
  const int64_t nwg = (int64_t)tiles_n * tiles_m * batches;
  gemm_bf16_kernel<BN, AMODE, EPI, PL><<<(unsigned)nwg, 256, 0, s>>>(a, tiles_n, tiles_m);
}

int dim_max(int sel, int fixed, int C, int U) { return sel == DIM_CC ? C : (sel == DIM_NC ? C + U : fixed); }

}  // namespace

void launch_gemm_bf16(const GemmArgsH& a, int epi, int batches, hipStream_t s) {
  const int maxM = dim_max(a.mdim, a.Mfix, a.C, a.U);
  const int maxN = dim_max(a.ndim, a.Nfix, a.C, a.U);
  if (maxM <= 0 || maxN <= 0 || batches <= 0) return;
  const int tiles_m = (maxM + BM - 1) / BM;
  const int tiles_n = (maxN + 127) / 128;   // = nct (PBG_SCORE_BN columns per tile)
  if (epi == EPI_LOSS) launch_t<128, GA_KC, EPI_LOSS>(a, tiles_n, tiles_m, batches, s);
  else if (epi == EPI_LOSS_BITS) launch_t<128, GA_KC, EPI_LOSS_BITS>(a, tiles_n, tiles_m, batches, s);
  else if (epi == EPI_SOFTMAX_STATS) launch_t<128, GA_KC, EPI_SOFTMAX_STATS>(a, tiles_n, tiles_m, batches, s);
  else launch_t<128, GA_KC, EPI_STORE>(a, tiles_n, tiles_m, batches, s);
}

namespace {
template <int BN, int AM0, int AM1, int PL>
void launch_pair_t(const GemmArgsH& a0, const GemmArgsH& a1, int batches, hipStream_t s) {
  const int tn0 = (dim_max(a0.ndim, a0.Nfix, a0.C, a0.U) + BN - 1) / BN;
  const int tm0 = (dim_max(a0.mdim, a0.Mfix, a0.C, a0.U) + BM - 1) / BM;
  const int tn1 = (dim_max(a1.ndim, a1.Nfix, a1.C, a1.U) + BN - 1) / BN;
  const int tm1 = (dim_max(a1.mdim, a1.Mfix, a1.C, a1.U) + BM - 1) / BM;
  const int64_t nwg0 = (int64_t)tn0 * tm0 * batches, nwg1 = (int64_t)tn1 * tm1 * batches;
  gemm_bf16_pair_kernel<BN, AM0, AM1, PL><<<(unsigned)(nwg0 + nwg1), 256, 0, s>>>(a0, tn0, tm0, (int)nwg0, a1,
                                                                                 tn1, tm1);
}

template <int BN, int PL>
void launch_bits_pair_t(const GemmArgsH& a0, const GemmArgsH& a1, int batches, hipStream_t s) {
  const int tn0 = (dim_max(a0.ndim, a0.Nfix, a0.C, a0.U) + BN - 1) / BN;
  const int tm0 = (dim_max(a0.mdim, a0.Mfix, a0.C, a0.U) + BT - 1) / BT;
  const int tn1 = (dim_max(a1.ndim, a1.Nfix, a1.C, a1.U) + BN - 1) / BN;
  // merged: dN rows from Cc rounded down to 16, at most U + 15 of them
  const int rows1 = a1.merge_cc ? a1.U + 15 : dim_max(a1.mdim, a1.Mfix, a1.C, a1.U);
  const int tm1 = (rows1 + BT - 1) / BT;
  const int64_t nwg0 = (int64_t)tn0 * tm0 * batches, nwg1 = (int64_t)tn1 * tm1 * batches;
  gemm_bits_pair_kernel<BN, PL><<<(unsigned)(nwg0 + nwg1), 256, 0, s>>>(a0, tn0, tm0, (int)nwg0, a1, tn1, tm1);
}

template <int BN>
void launch_pair_bn(const GemmArgsH& a0, const GemmArgsH& a1, int batches, hipStream_t s) {
  // three planes (float32 ranking backward): 256-row tiles with B streamed by
  // LDS DMA (0.226 -> 0.185 ms per social-network step); one plane (bf16
  // inputs): the 128-row tiles measured faster
  if (a0.planes == 3) launch_bits_pair_t<BN, 3>(a0, a1, batches, s);
  else if (a0.amode == GA_BITS_ROW) launch_pair_t<BN, GA_BITS_ROW, GA_BITS_COL, 1>(a0, a1, batches, s);
  else launch_pair_t<BN, GA_KC, GA_MC, 1>(a0, a1, batches, s);
}
}  // namespace

void launch_gemm_split_pair(const GemmArgsH& a0, const GemmArgsH& a1, int batches, hipStream_t s) {
  if (batches <= 0) return;
  const int tn0 = (dim_max(a0.ndim, a0.Nfix, a0.C, a0.U) + 127) / 128;
  const int tm0 = (dim_max(a0.mdim, a0.Mfix, a0.C, a0.U) + BM - 1) / BM;
  const int tn1 = (dim_max(a1.ndim, a1.Nfix, a1.C, a1.U) + 127) / 128;
  const int tm1 = (dim_max(a1.mdim, a1.Mfix, a1.C, a1.U) + BM - 1) / BM;
  const int64_t nwg0 = (int64_t)tn0 * tm0 * batches, nwg1 = (int64_t)tn1 * tm1 * batches;
  if (nwg0 + nwg1 <= 0) return;
  if (a0.smscale) gemm_split_pair_kernel<true><<<(unsigned)(nwg0 + nwg1), 256, 0, s>>>(a0, tn0, tm0, (int)nwg0, a1, tn1, tm1);
  else gemm_split_pair_kernel<false><<<(unsigned)(nwg0 + nwg1), 256, 0, s>>>(a0, tn0, tm0, (int)nwg0, a1, tn1, tm1);
}

void launch_gemm_bf16_pair(const GemmArgsH& a0, const GemmArgsH& a1, int batches, hipStream_t s) {
  const int maxN = std::max(dim_max(a0.ndim, a0.Nfix, a0.C, a0.U), dim_max(a1.ndim, a1.Nfix, a1.C, a1.U));
  if (maxN <= 0 || batches <= 0) return;
  if (maxN <= 64) launch_pair_bn<64>(a0, a1, batches, s);
  else launch_pair_bn<128>(a0, a1, batches, s);
}

void launch_score_split(const GemmArgsH& a, int epi, int batches, hipStream_t s) {
  constexpr int NPROD = 6;
  const int maxM = dim_max(a.mdim, a.Mfix, a.C, a.U);
  const int maxN = dim_max(a.ndim, a.Nfix, a.C, a.U);
  if (maxM <= 0 || maxN <= 0 || batches <= 0) return;
  const int tiles_m = (maxM + BM - 1) / BM;
  const int tiles_n = (maxN + 127) / 128;   // = nct (PBG_SCORE_BN columns per tile)
  const unsigned nwg = (unsigned)((int64_t)tiles_n * tiles_m * batches);
  if (epi == EPI_LOSS) score_split_kernel<EPI_LOSS, NPROD><<<nwg, 256, 0, s>>>(a, tiles_n, tiles_m);
  else if (epi == EPI_LOSS_BITS) score_split_kernel3<EPI_LOSS_BITS, NPROD><<<nwg, 256, 0, s>>>(a, tiles_n, tiles_m);
  else if (epi == EPI_SOFTMAX_EXP) score_split_kernel<EPI_SOFTMAX_EXP, NPROD><<<nwg, 256, 0, s>>>(a, tiles_n, tiles_m);
  else score_split_kernel<EPI_STORE, NPROD><<<nwg, 256, 0, s>>>(a, tiles_n, tiles_m);
}

void launch_to_bf16_t(const float* q, int64_t q_bs, int q_rows, uint16_t* qh, int64_t qh_bs, uint16_t* qT,
                      int64_t qT_bs, int q_ldT, const float* n, int64_t n_bs, int n_rows, uint16_t* nh,
                      int64_t nh_bs, uint16_t* nT, int64_t nT_bs, int n_ldT, int ld_src, int kp, int batches,
                      hipStream_t s) {
  if (batches <= 0 || kp <= 0) return;
  const Bf16T o0{q, q_bs, q_rows, ld_src, qh, qh_bs, kp, qT, qT_bs, q_ldT};
  const Bf16T o1{n, n_bs, n_rows, ld_src, nh, nh_bs, kp, nT, nT_bs, n_ldT};
  const int nq = q ? batches : 0;   // no Q: only N
  dim3 grid((kp + 63) / 64, (std::max(q ? q_ldT : 0, n_ldT) + 63) / 64, nq + batches);
  to_bf16_t_kernel<<<grid, 256, 0, s>>>(o0, o1, nq, kp);
}

void launch_finalize_split3_t(const StepGeom& g, const StepBufs& b, double* parts, bool softmax_scales,
                              const float* q, int64_t q_bs, int q_rows, uint16_t* qT, int64_t qT_bs, int64_t q_ps,
                              int q_ldT, const float* n, int64_t n_bs, int n_rows, uint16_t* nT, int64_t nT_bs,
                              int64_t n_ps, int n_ldT, int ld_src, int kp, int batches, hipStream_t s) {
  const int fb = fin_blocks(g.C);
  const int nfin = fb * g.nchunks;
  const Split3T o0{q, q_bs, q_rows, ld_src, qT, qT_bs, q_ps, q_ldT, q_ldT};
  const Split3T o1{n, n_bs, n_rows, ld_src, nT, nT_bs, n_ps, n_ldT, n_ldT};
  const int nq = q ? batches : 0;
  const int gx = (kp + 63) / 64, gy = (std::max(q ? q_ldT : 0, n_ldT) + 63) / 64;
  const int nsplit = (batches > 0 && kp > 0) ? gx * gy * (nq + batches) : 0;
  if (nfin + nsplit <= 0) return;
  finalize_split3_t_kernel<<<nfin + nsplit, 256, 0, s>>>(g, b, softmax_scales ? 1 : 0, parts, fb, nfin, o0, o1, nq,
                                                         kp, gx, gy);
}

void launch_split3_t(const float* q, int64_t q_bs, int q_rows, uint16_t* qT, int64_t qT_bs, int64_t q_ps,
                     int q_ldT, const float* n, int64_t n_bs, int n_rows, uint16_t* nT, int64_t nT_bs,
                     int64_t n_ps, int n_ldT, int ld_src, int kp, int batches, hipStream_t s) {
  if (batches <= 0 || kp <= 0) return;
  const Split3T o0{q, q_bs, q_rows, ld_src, qT, qT_bs, q_ps, q_ldT, q_ldT};
  const Split3T o1{n, n_bs, n_rows, ld_src, nT, nT_bs, n_ps, n_ldT, n_ldT};
  const int nq = q ? batches : 0;   // no Q: only N
  dim3 grid((kp + 63) / 64, (std::max(q ? q_ldT : 0, n_ldT) + 63) / 64, nq + batches);
  split3_t_kernel<<<grid, 256, 0, s>>>(o0, o1, nq, kp);
}

void launch_softmax_rows_bf16(const StepGeom& g, const StepBufs& b, uint16_t* dsh, int ldh, hipStream_t s) {
  dim3 grid((g.C + 3) / 4, g.nchunks * 2);
  softmax_rows_bf16_kernel<<<grid, 256, 0, s>>>(g, b.ds, b.rowpart, b.pos, dsh, ldh);
}
