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
// 16-byte group q of row x is kept at group q ^ ((x >> 2) & 3), so that the
// fragment reads of 16 consecutive rows and the tile stores of 16 rows x 4
// groups each touch all 64 banks once.
#include <algorithm>

#include "kernels.h"
#include "device_common.h"

namespace {

constexpr int BM = 128;
constexpr int BK = 32;          // k per slice = bf16 elements per LDS tile row
constexpr uint32_t OOB = 0x80000000u;

typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ rsrc_t make_rsrc(const void* p) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)p, (short)0, 0x7FFFFFF0, 0x00020000);
}
__device__ __forceinline__ u32x4 bload16(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

__device__ __forceinline__ float bf16_to_f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__device__ __forceinline__ uint16_t f_to_bf16(float x) {
  // round to nearest even (finite inputs)
  const uint32_t u = __float_as_uint(x);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// x = h + m + l exactly, each piece a bf16 (returned in the low 16 bits):
// h = bf16(x) leaves a remainder of at most 16 significant bits, m = bf16 of
// that remainder leaves at most 8, which l holds exactly
__device__ __forceinline__ void split3(float x, uint32_t* pc) {
  const uint16_t h = f_to_bf16(x);
  const float r1 = x - bf16_to_f(h);
  const uint16_t m = f_to_bf16(r1);
  pc[0] = h;
  pc[1] = m;
  pc[2] = f_to_bf16(r1 - bf16_to_f(m));
}

__device__ __forceinline__ int pick_dim(int sel, int fixed, int Cc, int Nc) {
  return sel == DIM_CC ? Cc : (sel == DIM_NC ? Nc : fixed);
}

// element offset of the 16-byte group q of row x in a swizzled LDS tile
__device__ __forceinline__ int swz(int x, int q) { return x * BK + ((q ^ ((x >> 2) & 3)) << 3); }

// 0.0 / 1.0 in bf16 for bits b and b+1 of v, packed low / high
__device__ __forceinline__ uint32_t bits2(uint32_t v, int b) {
  return (((v >> b) & 1u) * 0x3F80u) | ((((v >> (b + 1)) & 1u) * 0x3F80u) << 16);
}

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

  __device__ static void load(u32x4* r, rsrc_t rs, int ld, int x0, int xdim, int k0, int kdim, int tid) {
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

  __device__ static void store(uint16_t* s, const u32x4* r, int tid, int x0, int k0, int kdim) {
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
          const int b = (8 * kq) & 15;        // bit of column k0 + 8 kq in its word
          const uint32_t w = v.x;
          v = (u32x4){bits2(w, b), bits2(w, b + 2), bits2(w, b + 4), bits2(w, b + 6)};
        } else if (MODE == GA_BITS_COL) {
          const int b = (x0 + x) & 15;        // bit of this column in each row's word
          const int gk = k0 + 8 * kq;         // rows gk + i >= kdim lie outside the chunk
          uint32_t h[8];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            h[2 * i] = v[i] & 0xFFFFu;
            h[2 * i + 1] = v[i] >> 16;
          }
#pragma unroll
          for (int i = 0; i < 8; ++i) h[i] = (gk + i < kdim) ? ((h[i] >> b) & 1u) * 0x3F80u : 0u;
          v = (u32x4){h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
        }
        *(u32x4*)(s + swz(x, kq)) = v;
      }
    }
  }
};

// LDS of one workgroup: double-buffered A tile and PL B tiles, row partials
template <int BN, int PL>
struct SmemH {
  uint16_t As[2][BM * BK];
  uint16_t Bs[2][PL][BN * BK];
  float red[2][BM][2];
};

// One 128 x BN output tile; `id` numbers the workgroup among the nwg of this
// product (hardware order), remapped so that each batch stays on one XCD.
template <int BN, int AMODE, int EPI, int PL>
__device__ __forceinline__ void gemm_bf16_tile(const GemmArgsH& a, int tiles_n, int tiles_m, int nwg, int id,
                                               SmemH<BN, PL>& sm) {
  constexpr int WN = BN / 2;
  constexpr int JN = WN / 16;
  using TA = TileH<BM, AMODE>;
  using TB = TileH<BN, GA_KC>;
  auto& As = sm.As;
  auto& Bs = sm.Bs;
  auto& red = sm.red;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int l16 = lane & 15, g = lane >> 4;

  const int q8 = nwg >> 3, r8 = nwg & 7, xcd = id & 7;
  const int lid = xcd * q8 + min(xcd, r8) + (id >> 3);
  const int tn = lid % tiles_n;
  const int rest = lid / tiles_n;
  const int tm = rest % tiles_m;
  const int z = rest / tiles_m;

  const int c = z / a.nsides;
  const int side = z - c * a.nsides;
  int Cc = a.C, Nc = a.C + a.U;
  if (a.m_step > 0) {
    Cc = min(a.C, a.m_step - c * a.C);
    Nc = Cc + a.U;
  }
  const int M = pick_dim(a.mdim, a.Mfix, Cc, Nc);
  const int N = pick_dim(a.ndim, a.Nfix, Cc, Nc);
  const int K = pick_dim(a.kdim, a.Kfix, Cc, Nc);
  const int m0 = tm * BM;
  const int n0 = tn * BN;
  if (m0 >= M) return;

  float* rowpart = nullptr;
  if (EPI != EPI_STORE) rowpart = a.rowpart + ((int64_t)(c * 2 + side) * a.C) * a.nct * 2;
  if (n0 >= N) {
    // neutral row partials: no valid column in this tile
    if (EPI != EPI_STORE && tid < BM && m0 + tid < M) {
      float* rp = rowpart + ((int64_t)(m0 + tid) * a.nct + tn) * 2;
      rp[0] = (EPI == EPI_SOFTMAX_STATS) ? -INFINITY : 0.0f;
      rp[1] = 0.0f;
    }
    return;
  }

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

  // fragment offsets: row 16 i + l16 of the wave's block, group g (swizzled)
  const int fa0 = swz(64 * wm + l16, g), fb0 = swz(WN * wn + l16, g);
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
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
      TA::store(As[buf ^ 1], pa, tid, m0, (kt + 1) * BK, K);
#pragma unroll
      for (int p = 0; p < PL; ++p) TB::store(Bs[buf ^ 1][p], pb[p], tid, n0, (kt + 1) * BK, K);
    }
    __syncthreads();
  }

  const int colb = n0 + WN * wn + l16;
  if (EPI == EPI_STORE) {
    float* Cm = a.Cm + c * a.c_cs + side * a.c_ss;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + 64 * wm + 16 * i + 4 * g + r;
        if (m < M) {
#pragma unroll
          for (int j = 0; j < JN; ++j) {
            const int n = colb + 16 * j;
            if (n < N) Cm[(int64_t)m * a.ldc + n] = acc[i][j][r];
          }
        }
      }
    return;
  }

  // loss epilogues, as in the float32 kernel; dS leaves as bits (ranking),
  // bf16 (logistic) or raw fp32 scores for the softmax row pass
  const float* pos = a.pos + (int64_t)c * a.C;
  const float* bias = (a.bias && side == 1) ? a.bias + (int64_t)c * a.C : nullptr;
  const float kinv = (Nc - 1 > 0) ? 1.0f / (float)(Nc - 1) : 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int ml = 64 * wm + 16 * i + 4 * g + r;
      const int m = m0 + ml;
      const bool mrow = m < M;
      const float p = mrow ? pos[m] : 0.0f;
      const float bm = (bias && mrow) ? bias[m] : 0.0f;
      float v0, v1;
      if (EPI == EPI_LOSS || EPI == EPI_LOSS_BITS) {
        float lsum = 0.0f, dsum = 0.0f;
#pragma unroll
        for (int j = 0; j < JN; ++j) {
          const int n = colb + 16 * j;
          const float s = acc[i][j][r] + bm;
          const bool valid = mrow && n < N && n != m;
          float dsv = 0.0f;
          if (EPI == EPI_LOSS_BITS) {
            const float zz = a.margin - p + s;
            if (valid && zz > 0.0f) {
              dsv = 1.0f;
              lsum += zz;
            }
          } else if (valid) {
            float sg, sp;
            logistic_pair(s, sg, sp);
            dsv = sg * kinv;
            lsum += sp * kinv;
          }
          dsum += dsv;
          if (EPI == EPI_LOSS_BITS) {
            const uint64_t mask = __ballot(dsv != 0.0f);
            const int wcol = (n0 + WN * wn + 16 * j) >> 4;
            if (l16 == 0 && mrow && wcol < a.nwcb)
              a.dsb[c * a.cb_cs + side * a.cb_ss + (int64_t)wcol * a.ldcb + m] = (uint16_t)(mask >> (16 * g));
          } else if (mrow && n < a.ldc) {
            a.dsh[c * a.c_cs + side * a.c_ss + (int64_t)m * a.ldc + n] = f_to_bf16(dsv);
          }
        }
        v0 = group16_sum(lsum);
        v1 = group16_sum(dsum);
      } else {  // EPI_SOFTMAX_STATS
        float* Cm = a.Cm + c * a.c_cs + side * a.c_ss;
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < JN; ++j) {
          const int n = colb + 16 * j;
          const float s = acc[i][j][r] + bm;
          if (mrow && n < N && n != m) mx = fmaxf(mx, s);
          if (mrow && n < a.ldc) Cm[(int64_t)m * a.ldc + n] = s;
        }
        mx = group16_max(mx);
        float se = 0.0f;
#pragma unroll
        for (int j = 0; j < JN; ++j) {
          const int n = colb + 16 * j;
          if (mrow && n < N && n != m) se += expf(acc[i][j][r] + bm - mx);
        }
        v0 = mx;
        v1 = group16_sum(se);
      }
      if (l16 == 0) {
        red[wn][ml][0] = v0;
        red[wn][ml][1] = v1;
      }
    }
  __syncthreads();
  if (tid < BM && m0 + tid < M) {
    const int ml = tid;
    float v0, v1;
    if (EPI == EPI_LOSS || EPI == EPI_LOSS_BITS) {
      v0 = red[0][ml][0] + red[1][ml][0];
      v1 = red[0][ml][1] + red[1][ml][1];
    } else {
      const float ma = red[0][ml][0], mb = red[1][ml][0];
      const float mx = fmaxf(ma, mb);
      v0 = mx;
      v1 = (mx == -INFINITY) ? 0.0f
                             : (ma == -INFINITY ? 0.0f : red[0][ml][1] * expf(ma - mx)) +
                                   (mb == -INFINITY ? 0.0f : red[1][ml][1] * expf(mb - mx));
    }
    float* rp = rowpart + ((int64_t)(m0 + ml) * a.nct + tn) * 2;
    rp[0] = v0;
    rp[1] = v1;
  }
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

// fp32 packed rows -> bf16 rows (zero-padded to kp) and the transposed copy
// [kp][rows_p]: 64 x 64 tiles through LDS, coalesced on both sides.
__global__ __launch_bounds__(256) void to_bf16_transpose_kernel(const float* src, int64_t src_bs,
                                                                int rows, int ld_src, int d,
                                                                uint16_t* dst, int64_t dst_bs, int ld_dst,
                                                                uint16_t* dstT, int64_t dstT_bs,
                                                                int ld_T, int rows_p, int kp) {
  __shared__ uint16_t tile[64][66];
  const int b = blockIdx.z;
  const int r0 = blockIdx.y * 64, k0 = blockIdx.x * 64;
  const float* s = src + (int64_t)b * src_bs;
  uint16_t* o = dst + (int64_t)b * dst_bs;
  uint16_t* oT = dstT + (int64_t)b * dstT_bs;
  for (int q = threadIdx.x; q < 64 * 64; q += 256) {
    const int rr = q >> 6, kk = q & 63;
    const int r = r0 + rr, k = k0 + kk;
    float v = 0.0f;
    if (r < rows && k < d) v = s[(int64_t)r * ld_src + k];
    const uint16_t h = f_to_bf16(v);
    tile[rr][kk] = h;
    if (r < rows && k < kp) o[(int64_t)r * ld_dst + k] = h;
  }
  __syncthreads();
  for (int q = threadIdx.x; q < 64 * 64; q += 256) {
    const int kk = q >> 6, rr = q & 63;
    const int r = r0 + rr, k = k0 + kk;
    if (k < kp && r < rows_p) oT[(int64_t)k * ld_T + r] = (r < rows) ? tile[rr][kk] : (uint16_t)0;
  }
}

// fp32 rows -> the three exact bf16 pieces (h, m, l) of every element, each
// transposed: plane p is [kp][ld_T] (source column, then source row), planes
// ps elements apart; rows [rows, rows_p) and columns [d, kp) are zeros.
// rows_p and ld_T are multiples of 4 (each thread writes four rows).
__global__ __launch_bounds__(256) void split3_transpose_kernel(const float* src, int64_t src_bs, int rows,
                                                               int ld_src, int d, uint16_t* dstT,
                                                               int64_t dstT_bs, int64_t ps, int ld_T,
                                                               int rows_p, int kp) {
  __shared__ float tile[64][65];
  const int b = blockIdx.z;
  const int r0 = blockIdx.y * 64, k0 = blockIdx.x * 64;
  const float* s = src + (int64_t)b * src_bs;
  for (int q = threadIdx.x; q < 64 * 64; q += 256) {
    const int rr = q >> 6, kk = q & 63;
    const int r = r0 + rr, k = k0 + kk;
    tile[rr][kk] = (r < rows && k < d) ? s[(int64_t)r * ld_src + k] : 0.0f;
  }
  __syncthreads();
  uint16_t* o = dstT + (int64_t)b * dstT_bs;
  for (int q = threadIdx.x; q < 64 * 16; q += 256) {
    const int kk = q >> 4, r4 = 4 * (q & 15);
    const int k = k0 + kk, r = r0 + r4;
    if (k >= kp || r >= rows_p) continue;
    uint32_t pc[3][2];
#pragma unroll
    for (int i = 0; i < 4; i += 2) {
      uint32_t lo[3], hi[3];
      split3(tile[r4 + i][kk], lo);
      split3(tile[r4 + i + 1][kk], hi);
#pragma unroll
      for (int p = 0; p < 3; ++p) pc[p][i >> 1] = lo[p] | (hi[p] << 16);
    }
#pragma unroll
    for (int p = 0; p < 3; ++p)
      *(uint2*)(o + p * ps + (int64_t)k * ld_T + r) = make_uint2(pc[p][0], pc[p][1]);
  }
}

// softmax row pass in bf16 mode: raw fp32 scores -> dS = softmax (masked),
// written as bf16 rows and into the transposed copy
__global__ __launch_bounds__(256) void softmax_rows_bf16_kernel(StepGeom g, const float* S, const float* rowpart,
                                                                const float* pos, float* rowstat,
                                                                uint16_t* dsh, uint16_t* dsT, int ldh,
                                                                int ldt) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int z = blockIdx.y;
  const int c = z >> 1;
  const int Cc = chunk_edges(g, c);
  if (row >= Cc) return;
  const int Nc = Cc + g.U;
  const float p = pos[(int64_t)c * g.C + row];
  const float* rp = rowpart + ((int64_t)z * g.C + row) * g.nct * 2;
  float Mx = p;
  for (int ct = 0; ct < g.nct; ++ct) Mx = fmaxf(Mx, rp[2 * ct]);
  float Z = expf(p - Mx);
  for (int ct = 0; ct < g.nct; ++ct) {
    const float mx = rp[2 * ct];
    if (mx > -INFINITY) Z += rp[2 * ct + 1] * expf(mx - Mx);
  }
  const float lse = Mx + logf(Z);
  if (lane == 0) rowstat[(int64_t)z * g.C + row] = lse;
  const float* srow = S + ((int64_t)z * g.C + row) * g.Np;
  uint16_t* hrow = dsh + ((int64_t)z * g.C) * ldh + (int64_t)row * ldh;
  uint16_t* tcol = dsT ? dsT + ((int64_t)z * g.N) * ldt + row : nullptr;
  const int Nh = (Nc + 31) & ~31;
  for (int t = lane; t < Nh; t += 64) {
    float v = 0.0f;
    if (t < Nc && t != row) v = expf(srow[t] - lse);
    const uint16_t h = f_to_bf16(v);
    hrow[t] = h;
    if (dsT) tcol[(int64_t)t * ldt] = h;
  }
}


template <int BN, int AMODE, int EPI, int PL = 1>
void launch_t(const GemmArgsH& a, int tiles_n, int tiles_m, int batches, hipStream_t s) {
  const int64_t nwg = (int64_t)tiles_n * tiles_m * batches;
  gemm_bf16_kernel<BN, AMODE, EPI, PL><<<(unsigned)nwg, 256, 0, s>>>(a, tiles_n, tiles_m);
}

template <int BN>
void launch_store(const GemmArgsH& a, int tiles_n, int tiles_m, int batches, hipStream_t s) {
  if (a.planes == 3) {
    // float32 operand as three exact pieces: only the 0/1 ranking dS as A
    if (a.amode == GA_BITS_ROW) launch_t<BN, GA_BITS_ROW, EPI_STORE, 3>(a, tiles_n, tiles_m, batches, s);
    else launch_t<BN, GA_BITS_COL, EPI_STORE, 3>(a, tiles_n, tiles_m, batches, s);
    return;
  }
  switch (a.amode) {
    case GA_KC: launch_t<BN, GA_KC, EPI_STORE>(a, tiles_n, tiles_m, batches, s); break;
    case GA_MC: launch_t<BN, GA_MC, EPI_STORE>(a, tiles_n, tiles_m, batches, s); break;
    case GA_BITS_ROW: launch_t<BN, GA_BITS_ROW, EPI_STORE>(a, tiles_n, tiles_m, batches, s); break;
    default: launch_t<BN, GA_BITS_COL, EPI_STORE>(a, tiles_n, tiles_m, batches, s); break;
  }
}

int dim_max(int sel, int fixed, int C, int U) { return sel == DIM_CC ? C : (sel == DIM_NC ? C + U : fixed); }

}  // namespace

void launch_gemm_bf16(const GemmArgsH& a, int epi, int batches, hipStream_t s) {
  const int maxM = dim_max(a.mdim, a.Mfix, a.C, a.U);
  const int maxN = dim_max(a.ndim, a.Nfix, a.C, a.U);
  if (maxM <= 0 || maxN <= 0 || batches <= 0) return;
  const int tiles_m = (maxM + BM - 1) / BM;
  if (epi != EPI_STORE) {
    const int tiles_n = (maxN + 127) / 128;   // = nct (PBG_SCORE_BN columns per tile)
    if (epi == EPI_LOSS) launch_t<128, GA_KC, EPI_LOSS>(a, tiles_n, tiles_m, batches, s);
    else if (epi == EPI_LOSS_BITS) launch_t<128, GA_KC, EPI_LOSS_BITS>(a, tiles_n, tiles_m, batches, s);
    else launch_t<128, GA_KC, EPI_SOFTMAX_STATS>(a, tiles_n, tiles_m, batches, s);
    return;
  }
  if (maxN <= 64) launch_store<64>(a, (maxN + 63) / 64, tiles_m, batches, s);
  else launch_store<128>(a, (maxN + 127) / 128, tiles_m, batches, s);
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

template <int BN>
void launch_pair_bn(const GemmArgsH& a0, const GemmArgsH& a1, int batches, hipStream_t s) {
  if (a0.planes == 3) launch_pair_t<BN, GA_BITS_ROW, GA_BITS_COL, 3>(a0, a1, batches, s);
  else if (a0.amode == GA_BITS_ROW) launch_pair_t<BN, GA_BITS_ROW, GA_BITS_COL, 1>(a0, a1, batches, s);
  else launch_pair_t<BN, GA_KC, GA_MC, 1>(a0, a1, batches, s);
}
}  // namespace

void launch_gemm_bf16_pair(const GemmArgsH& a0, const GemmArgsH& a1, int batches, hipStream_t s) {
  const int maxN = std::max(dim_max(a0.ndim, a0.Nfix, a0.C, a0.U), dim_max(a1.ndim, a1.Nfix, a1.C, a1.U));
  if (maxN <= 0 || batches <= 0) return;
  if (maxN <= 64) launch_pair_bn<64>(a0, a1, batches, s);
  else launch_pair_bn<128>(a0, a1, batches, s);
}

void launch_to_bf16_transpose(const float* src, int64_t src_bs, int rows, int ld_src, int d,
                              uint16_t* dst, int64_t dst_bs, int ld_dst, uint16_t* dstT,
                              int64_t dstT_bs, int ld_T, int rows_p, int kp, int batches,
                              hipStream_t s) {
  dim3 grid((kp + 63) / 64, (rows_p + 63) / 64, batches);
  to_bf16_transpose_kernel<<<grid, 256, 0, s>>>(src, src_bs, rows, ld_src, d, dst, dst_bs, ld_dst, dstT,
                                                dstT_bs, ld_T, rows_p, kp);
}

void launch_split3_transpose(const float* src, int64_t src_bs, int rows, int ld_src, int d, uint16_t* dstT,
                             int64_t dstT_bs, int64_t ps, int ld_T, int rows_p, int kp, int batches,
                             hipStream_t s) {
  dim3 grid((kp + 63) / 64, (rows_p + 63) / 64, batches);
  split3_transpose_kernel<<<grid, 256, 0, s>>>(src, src_bs, rows, ld_src, d, dstT, dstT_bs, ps, ld_T, rows_p,
                                               kp);
}

void launch_softmax_rows_bf16(const StepGeom& g, const StepBufs& b, uint16_t* dsh, int ldh, hipStream_t s) {
  dim3 grid((g.C + 3) / 4, g.nchunks * 2);
  softmax_rows_bf16_kernel<<<grid, 256, 0, s>>>(g, b.ds, b.rowpart, b.pos, b.rowstat, dsh, nullptr, ldh, 0);
}
