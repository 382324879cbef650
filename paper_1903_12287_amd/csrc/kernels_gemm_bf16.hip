// bfloat16 inputs / float32 accumulation for the three chunk contractions
// (Sec. 4.3 batched negatives; the score block of a chunk is one product).
//
// Every product is written as C[m][n] = sum_k A[m][k] B[n][k] with both
// operands contiguous along k, in bf16 with rows zero-padded to a multiple
// of 32 elements:
//   forward  S  = Q  . N^T  :  A = Q   [e][f],   B = N   [t][f]
//   dQ       dQ = dS . N    :  A = dS  [e][t],   B = N^T [f][t]
//   dN       dN = dS^T . Q  :  A = dS^T[t][e],   B = Q^T [f][e]
// so the transposed operands are produced once (an LDS-tiled transpose for
// Q^T and N^T; the forward epilogue writes dS^T next to dS).
//
// A workgroup of 4 waves computes a 128 x (16*NB) tile; wave w owns rows
// [32w, 32w+32).  Tiles of 64 k are staged in LDS as [row][k] with a pitch of
// 72 elements (144 bytes: rows fall on distinct bank groups) and read as one
// 16-byte fragment per lane per v_mfma_f32_16x16x32_bf16.  Fragment layout
// (checked on the device): A lane L holds A[L % 16][8 (L / 16) + i],
// B lane L holds B[8 (L / 16) + i][L % 16] (i = 0..7), D as in the fp32 case.
#include "kernels.h"
#include "device_common.h"

namespace {

constexpr int BM = 128;
constexpr int BK = 64;
constexpr int PK = 72;  // LDS pitch in bf16 elements

struct alignas(16) bf8 {
  uint4 v;
};

__device__ __forceinline__ float bf16_to_f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

__device__ __forceinline__ uint16_t f_to_bf16(float x) {
  // round to nearest even (finite inputs)
  const uint32_t u = __float_as_uint(x);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ int pick_dim(int sel, int fixed, int Cc, int Nc) {
  return sel == DIM_CC ? Cc : (sel == DIM_NC ? Nc : fixed);
}

template <int NB, int EPI>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgsH a) {
  constexpr int BN = 16 * NB;
  constexpr int A_LOADS = BM * BK / 8 / 256;           // 16-byte loads of A per thread (4)
  constexpr int B_VEC = BN * BK / 8;                    // 16-byte vectors in a B tile
  constexpr int B_LOADS = (B_VEC + 255) / 256;
  __shared__ __align__(16) uint16_t As[2][BM * PK];
  __shared__ __align__(16) uint16_t Bs[2][BN * PK];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int z = blockIdx.z;
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
  const int Kp = (K + 31) & ~31;   // operands are zero beyond K up to a multiple of 32
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  if (m0 >= M) return;
  float* rowpart = nullptr;
  if (EPI != EPI_STORE) rowpart = a.rowpart + ((int64_t)(c * 2 + side) * a.C) * a.nct * 2;
  if (n0 >= N) {
    if (EPI != EPI_STORE && tid < BM && m0 + tid < M) {
      float* rp = rowpart + ((int64_t)(m0 + tid) * a.nct + blockIdx.x) * 2;
      rp[0] = (EPI == EPI_SOFTMAX_STATS) ? -INFINITY : 0.0f;
      rp[1] = 0.0f;
    }
    return;
  }
  const uint16_t* A = a.A + c * a.a_cs + side * a.a_ss;
  const uint16_t* B = a.B + c * a.b_cs + side * a.b_ss;

  v4f acc[2][NB];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};

  uint4 ra[A_LOADS], rb[B_LOADS];
  const uint4 z4 = make_uint4(0, 0, 0, 0);
  auto load_tiles = [&](int k0) {
#pragma unroll
    for (int q = 0; q < A_LOADS; ++q) {
      const int idx = tid + 256 * q;
      const int m = idx >> 3, kv = idx & 7;
      const int gm = m0 + m, gk = k0 + 8 * kv;
      ra[q] = (gm < M && gk < Kp) ? *(const uint4*)(A + (int64_t)gm * a.lda + gk) : z4;
    }
#pragma unroll
    for (int q = 0; q < B_LOADS; ++q) {
      const int idx = tid + 256 * q;
      const int n = idx >> 3, kv = idx & 7;
      const int gn = n0 + n, gk = k0 + 8 * kv;
      rb[q] = (idx < B_VEC && gn < N && gk < Kp) ? *(const uint4*)(B + (int64_t)gn * a.ldb + gk) : z4;
    }
  };
  auto store_tiles = [&](int buf) {
#pragma unroll
    for (int q = 0; q < A_LOADS; ++q) {
      const int idx = tid + 256 * q;
      *(uint4*)(&As[buf][(idx >> 3) * PK + 8 * (idx & 7)]) = ra[q];
    }
#pragma unroll
    for (int q = 0; q < B_LOADS; ++q) {
      const int idx = tid + 256 * q;
      if (idx < B_VEC) *(uint4*)(&Bs[buf][(idx >> 3) * PK + 8 * (idx & 7)]) = rb[q];
    }
  };

  const int nk = (Kp + BK - 1) / BK;
  load_tiles(0);
  store_tiles(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_tiles((kt + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK / 32; ++kk) {
      const int ko = 32 * kk + 8 * (lane >> 4);
      v8bf af[2], bfr[NB];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *(const v8bf*)(&As[buf][(32 * w + 16 * i + (lane & 15)) * PK + ko]);
#pragma unroll
      for (int j = 0; j < NB; ++j) bfr[j] = *(const v8bf*)(&Bs[buf][(16 * j + (lane & 15)) * PK + ko]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) store_tiles(buf ^ 1);
    __syncthreads();
  }

  const int col = lane & 15;
  const int rq = 4 * (lane >> 4);
  if (EPI == EPI_STORE) {
    float* Cm = a.Cm + c * a.c_cs + side * a.c_ss;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + 32 * w + 16 * i + rq + r;
        if (m < M) {
#pragma unroll
          for (int j = 0; j < NB; ++j) {
            const int n = n0 + 16 * j + col;
            if (n < N) Cm[(int64_t)m * a.ldc + n] = acc[i][j][r];
          }
        }
      }
    return;
  }

  if (EPI == EPI_SOFTMAX_STATS) {
    // raw fp32 scores + per-tile (max, sum exp) of the valid negatives
    float* Cm = a.Cm + c * a.c_cs + side * a.c_ss;
    const float* sbias = (a.bias && side == 1) ? a.bias + (int64_t)c * a.C : nullptr;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + 32 * w + 16 * i + rq + r;
        const bool mrow = m < M;
        const float bm = (sbias && mrow) ? sbias[m] : 0.0f;
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int n = n0 + 16 * j + col;
          const float s = acc[i][j][r] + bm;
          if (mrow && n < N && n != m) mx = fmaxf(mx, s);
          if (mrow && n < a.ldc) Cm[(int64_t)m * a.ldc + n] = s;
        }
        mx = group16_max(mx);
        float se = 0.0f;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int n = n0 + 16 * j + col;
          if (mrow && n < N && n != m) se += expf(acc[i][j][r] + bm - mx);
        }
        se = group16_sum(se);
        if (col == 0 && mrow) {
          float* rp = rowpart + ((int64_t)m * a.nct + blockIdx.x) * 2;
          rp[0] = mx;
          rp[1] = se;
        }
      }
    return;
  }

  // loss epilogue (ranking / logistic): dS in bf16, row-major and transposed
  uint16_t* dsh = a.dsh + c * a.c_cs + side * a.c_ss;      // [C][ldc]
  uint16_t* dsT = a.dsT + c * a.t_cs + side * a.t_ss;      // [N][ldt]
  const float* pos = a.pos + (int64_t)c * a.C;
  const float* bias = (a.bias && side == 1) ? a.bias + (int64_t)c * a.C : nullptr;
  const float kinv = (Nc - 1 > 0) ? 1.0f / (float)(Nc - 1) : 0.0f;
  const int Mp = (M + 31) & ~31;   // dS^T columns that the backward product reads
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    float dsv[NB][4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + 32 * w + 16 * i + rq + r;
      const bool mrow = m < M;
      const float p = mrow ? pos[m] : 0.0f;
      const float bm = (bias && mrow) ? bias[m] : 0.0f;
      float lsum = 0.0f, dsum = 0.0f;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int n = n0 + 16 * j + col;
        const float s = acc[i][j][r] + bm;
        const bool valid = mrow && n < N && n != m;
        float v = 0.0f;
        if (a.loss == LOSS_RANKING) {
          const float zz = a.margin - p + s;
          if (valid && zz > 0.0f) {
            v = 1.0f;
            lsum += zz;
          }
        } else if (valid) {
          v = sigmoidf(s) * kinv;
          lsum += softplusf(s) * kinv;
        }
        const uint16_t hv = f_to_bf16(v);
        dsv[j][r] = bf16_to_f(hv);
        dsum += v;
        if (mrow && n < a.ldc) dsh[(int64_t)m * a.ldc + n] = hv;
      }
      lsum = group16_sum(lsum);
      dsum = group16_sum(dsum);
      if (col == 0 && mrow) {
        float* rp = rowpart + ((int64_t)m * a.nct + blockIdx.x) * 2;
        rp[0] = lsum;
        rp[1] = dsum;
      }
    }
    // transposed copy: lane writes rows n, 4 consecutive columns m
    const int mb = m0 + 32 * w + 16 * i + rq;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int n = n0 + 16 * j + col;
      if (n < N && mb < Mp) {
        uint16_t* dst = dsT + (int64_t)n * a.ldt + mb;
        const uint32_t lo = (uint32_t)f_to_bf16(dsv[j][0]) | ((uint32_t)f_to_bf16(dsv[j][1]) << 16);
        const uint32_t hi = (uint32_t)f_to_bf16(dsv[j][2]) | ((uint32_t)f_to_bf16(dsv[j][3]) << 16);
        *(uint2*)dst = make_uint2(lo, hi);
      }
    }
  }
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
  uint16_t* tcol = dsT + ((int64_t)z * g.N) * ldt + row;
  const int Nh = (Nc + 31) & ~31;
  for (int t = lane; t < Nh; t += 64) {
    float v = 0.0f;
    if (t < Nc && t != row) v = expf(srow[t] - lse);
    const uint16_t h = f_to_bf16(v);
    hrow[t] = h;
    tcol[(int64_t)t * ldt] = h;
  }
}

// zero the dS^T columns [Cc, Cc rounded up to 32) of a short chunk
__global__ void zero_dsT_tail_kernel(StepGeom g, uint16_t* dsT, int ldt) {
  const int z = blockIdx.y;
  const int c = z >> 1;
  const int Cc = chunk_edges(g, c);
  const int Cp = (Cc + 31) & ~31;
  const int Nc = Cc + g.U;
  const int width = Cp - Cc;
  if (width == 0) return;
  for (int idx = blockIdx.x * blockDim.x + threadIdx.x; idx < Nc * width; idx += gridDim.x * blockDim.x) {
    const int t = idx / width, e = Cc + idx % width;
    dsT[((int64_t)z * g.N + t) * ldt + e] = 0;
  }
}

template <int EPI>
void launch_nb(int nb, const GemmArgsH& a, dim3 grid, hipStream_t s) {
  switch (nb) {
    case 1: gemm_bf16_kernel<1, EPI><<<grid, 256, 0, s>>>(a); break;
    case 2: gemm_bf16_kernel<2, EPI><<<grid, 256, 0, s>>>(a); break;
    case 3: gemm_bf16_kernel<3, EPI><<<grid, 256, 0, s>>>(a); break;
    case 4: gemm_bf16_kernel<4, EPI><<<grid, 256, 0, s>>>(a); break;
    case 5: gemm_bf16_kernel<5, EPI><<<grid, 256, 0, s>>>(a); break;
    case 6: gemm_bf16_kernel<6, EPI><<<grid, 256, 0, s>>>(a); break;
    case 7: gemm_bf16_kernel<7, EPI><<<grid, 256, 0, s>>>(a); break;
    default: gemm_bf16_kernel<8, EPI><<<grid, 256, 0, s>>>(a); break;
  }
}

}  // namespace

void launch_gemm_bf16(const GemmArgsH& a, int epi, int nb, int grid_n, int grid_m, int batches,
                      hipStream_t s) {
  dim3 grid(grid_n, grid_m, batches);
  if (epi == EPI_LOSS) gemm_bf16_kernel<8, EPI_LOSS><<<grid, 256, 0, s>>>(a);
  else if (epi == EPI_SOFTMAX_STATS) gemm_bf16_kernel<8, EPI_SOFTMAX_STATS><<<grid, 256, 0, s>>>(a);
  else launch_nb<EPI_STORE>(nb, a, grid, s);
}

void launch_to_bf16_transpose(const float* src, int64_t src_bs, int rows, int ld_src, int d,
                              uint16_t* dst, int64_t dst_bs, int ld_dst, uint16_t* dstT,
                              int64_t dstT_bs, int ld_T, int rows_p, int kp, int batches,
                              hipStream_t s) {
  dim3 grid((kp + 63) / 64, (rows_p + 63) / 64, batches);
  to_bf16_transpose_kernel<<<grid, 256, 0, s>>>(src, src_bs, rows, ld_src, d, dst, dst_bs, ld_dst,
                                                dstT, dstT_bs, ld_T, rows_p, kp);
}

void launch_softmax_rows_bf16(const StepGeom& g, const StepBufs& b, uint16_t* dsh, uint16_t* dsT,
                              int ldh, int ldt, hipStream_t s) {
  dim3 grid((g.C + 3) / 4, g.nchunks * 2);
  softmax_rows_bf16_kernel<<<grid, 256, 0, s>>>(g, b.ds, b.rowpart, b.pos, b.rowstat, dsh, dsT, ldh, ldt);
}

void launch_zero_dsT_tail(const StepGeom& g, uint16_t* dsT, int ldt, hipStream_t s) {
  dim3 grid(4, g.nchunks * 2);
  zero_dsT_tail_kernel<<<grid, 256, 0, s>>>(g, dsT, ldt);
}
