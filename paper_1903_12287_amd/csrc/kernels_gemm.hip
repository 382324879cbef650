// Chunk x candidates contractions on the gfx950 matrix cores (Sec. 4.3: the
// scores of a chunk against its negatives form one matrix product, Fig. 3).
//
//   forward   S  = Q . N^T   (C x N, K = dim)  + fused loss epilogue
//   backward  dQ = dS . N    (C x dim, K = N)
//             dN = dS^T . Q  (N x dim, K = C)
//
// One kernel template covers all three: a 256-thread workgroup (4 waves)
// computes a 128 x (16*NB) tile; wave w owns rows [32w, 32w+32) and all
// columns, i.e. 2 x NB blocks of v_mfma_f32_16x16x4_f32.  Operands are staged
// through LDS in [k][m] layout (pitch = 16 mod 64 floats: conflict-free
// fragment reads) with a register-prefetched double buffer, so the global
// read of tile k+1 overlaps the matrix work on tile k.  Either operand may be
// contiguous along k (rows of Q, N, dS) or along m/n (dS^T, N and Q in the
// backward products); the loader transposes on the way into LDS.
//
// Fragment layout of v_mfma_f32_16x16x4_f32 (checked on the device):
//   A: lane L holds A[L % 16][L / 16]; B: lane L holds B[L / 16][L % 16];
//   D: lane L, register r holds D[4 (L / 16) + r][L % 16].
#include "kernels.h"
#include "device_common.h"

namespace {

constexpr int BM = 128;
constexpr int BKT = 16;
constexpr int PA = 144;

__host__ __device__ constexpr int lds_pitch(int bn) { return ((bn - 16 + 63) / 64) * 64 + 16; }

__device__ __forceinline__ int pick_dim(int sel, int fixed, int Cc, int Nc) {
  return sel == DIM_CC ? Cc : (sel == DIM_NC ? Nc : fixed);
}

template <int NB, bool AK, bool BKC, int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  constexpr int BN = 16 * NB;
  constexpr int PB = lds_pitch(BN);
  constexpr int NBV = (64 * NB + 255) / 256;  // float4 loads of B per thread
  __shared__ __align__(16) float As[2][BKT * PA];
  __shared__ __align__(16) float Bs[2][BKT * PB];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
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
  const int m0 = blockIdx.y * BM;
  const int n0 = blockIdx.x * BN;
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

  const float* A = a.A + c * a.a_cs + side * a.a_ss;
  const float* B = a.B + c * a.b_cs + side * a.b_ss;
  const int Kp4 = (K + 3) & ~3;
  const int Mp4 = (M + 3) & ~3;
  const int Np4 = (N + 3) & ~3;

  v4f acc[2][NB];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};

  float4 ra[2], rb[NBV];
  const float4 zero4 = make_float4(0.f, 0.f, 0.f, 0.f);

  auto load_tiles = [&](int k0) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int idx = tid + 256 * q;
      if (AK) {
        const int m = idx >> 2, kq = idx & 3;
        const int gm = m0 + m, gk = k0 + 4 * kq;
        ra[q] = (gm < M && gk < Kp4) ? *(const float4*)(A + (int64_t)gm * a.lda + gk) : zero4;
      } else {
        const int k = idx >> 5, mq = idx & 31;
        const int gk = k0 + k, gm = m0 + 4 * mq;
        ra[q] = (gk < K && gm < Mp4) ? *(const float4*)(A + (int64_t)gk * a.lda + gm) : zero4;
      }
    }
#pragma unroll
    for (int q = 0; q < NBV; ++q) {
      const int idx = tid + 256 * q;
      rb[q] = zero4;
      if (idx < 64 * NB) {
        if (BKC) {
          const int n = idx >> 2, kq = idx & 3;
          const int gn = n0 + n, gk = k0 + 4 * kq;
          if (gn < N && gk < Kp4) rb[q] = *(const float4*)(B + (int64_t)gn * a.ldb + gk);
        } else {
          const int k = idx / (4 * NB), nq = idx % (4 * NB);
          const int gk = k0 + k, gn = n0 + 4 * nq;
          if (gk < K && gn < Np4) rb[q] = *(const float4*)(B + (int64_t)gk * a.ldb + gn);
        }
      }
    }
  };
  auto store_tiles = [&](int buf) {
    float* as = As[buf];
    float* bs = Bs[buf];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int idx = tid + 256 * q;
      if (AK) {
        const int m = idx >> 2, kq = idx & 3;
        as[(4 * kq + 0) * PA + m] = ra[q].x;
        as[(4 * kq + 1) * PA + m] = ra[q].y;
        as[(4 * kq + 2) * PA + m] = ra[q].z;
        as[(4 * kq + 3) * PA + m] = ra[q].w;
      } else {
        const int k = idx >> 5, mq = idx & 31;
        *(float4*)(as + k * PA + 4 * mq) = ra[q];
      }
    }
#pragma unroll
    for (int q = 0; q < NBV; ++q) {
      const int idx = tid + 256 * q;
      if (idx < 64 * NB) {
        if (BKC) {
          const int n = idx >> 2, kq = idx & 3;
          bs[(4 * kq + 0) * PB + n] = rb[q].x;
          bs[(4 * kq + 1) * PB + n] = rb[q].y;
          bs[(4 * kq + 2) * PB + n] = rb[q].z;
          bs[(4 * kq + 3) * PB + n] = rb[q].w;
        } else {
          const int k = idx / (4 * NB), nq = idx % (4 * NB);
          *(float4*)(bs + k * PB + 4 * nq) = rb[q];
        }
      }
    }
  };

  const int nk = (K + BKT - 1) / BKT;
  load_tiles(0);
  store_tiles(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_tiles((kt + 1) * BKT);
    const float* as = As[buf];
    const float* bs = Bs[buf];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int kr = 4 * kk + (lane >> 4);
      float af[2], bf[NB];
#pragma unroll
      for (int i = 0; i < 2; ++i) af[i] = as[kr * PA + 32 * w + 16 * i + (lane & 15)];
#pragma unroll
      for (int j = 0; j < NB; ++j) bf[j] = bs[kr * PB + 16 * j + (lane & 15)];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) store_tiles(buf ^ 1);
    __syncthreads();
  }

  float* Cm = a.Cm + c * a.c_cs + side * a.c_ss;
  const int col = lane & 15;
  const int rq = 4 * (lane >> 4);

  if (EPI == EPI_STORE) {
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

  // loss epilogues: M = Cc rows, valid columns [0, Nc) minus the diagonal,
  // stored columns [0, ldc)
  const float* pos = a.pos + (int64_t)c * a.C;
  // translation + dot: source corruptions score <x_t, x_d> + <theta_r, x_d>
  const float* bias = (a.bias && side == 1) ? a.bias + (int64_t)c * a.C : nullptr;
  const float kinv = (Nc - 1 > 0) ? 1.0f / (float)(Nc - 1) : 0.0f;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + 32 * w + 16 * i + rq + r;
      const bool mrow = m < M;
      const float p = mrow ? pos[m] : 0.0f;
      const float bm = (bias && mrow) ? bias[m] : 0.0f;
      if (EPI == EPI_LOSS) {
        float lsum = 0.0f, dsum = 0.0f;
#pragma unroll
        for (int j = 0; j < NB; ++j) {
          const int n = n0 + 16 * j + col;
          const float s = acc[i][j][r] + bm;
          const bool valid = mrow && n < N && n != m;
          float dsv = 0.0f;
          if (a.loss == LOSS_RANKING) {
            const float zz = a.margin - p + s;
            if (valid && zz > 0.0f) {
              dsv = 1.0f;
              lsum += zz;
            }
          } else {
            if (valid) {
              dsv = sigmoidf(s) * kinv;
              lsum += softplusf(s) * kinv;
            }
          }
          dsum += dsv;
          if (mrow && n < a.ldc) Cm[(int64_t)m * a.ldc + n] = dsv;
        }
        lsum = group16_sum(lsum);
        dsum = group16_sum(dsum);
        if (col == 0 && mrow) {
          float* rp = rowpart + ((int64_t)m * a.nct + blockIdx.x) * 2;
          rp[0] = lsum;
          rp[1] = dsum;
        }
      } else {  // EPI_SOFTMAX_STATS: raw scores + per-tile (max, sum exp)
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
    }
}

template <int NB, bool AK, bool BKC, int EPI>
void launch_nb(const GemmArgs& a, dim3 grid, hipStream_t s) {
  gemm_f32_kernel<NB, AK, BKC, EPI><<<grid, 256, 0, s>>>(a);
}

template <bool AK, bool BKC, int EPI>
void launch_any_nb(int nb, const GemmArgs& a, dim3 grid, hipStream_t s) {
  switch (nb) {
    case 1: launch_nb<1, AK, BKC, EPI>(a, grid, s); break;
    case 2: launch_nb<2, AK, BKC, EPI>(a, grid, s); break;
    case 3: launch_nb<3, AK, BKC, EPI>(a, grid, s); break;
    case 4: launch_nb<4, AK, BKC, EPI>(a, grid, s); break;
    case 5: launch_nb<5, AK, BKC, EPI>(a, grid, s); break;
    case 6: launch_nb<6, AK, BKC, EPI>(a, grid, s); break;
    case 7: launch_nb<7, AK, BKC, EPI>(a, grid, s); break;
    default: launch_nb<8, AK, BKC, EPI>(a, grid, s); break;
  }
}

}  // namespace

// column blocks of 16 per tile for an output of width n: as few tiles as
// possible, each at most 128 wide
int gemm_pick_nb(int n) {
  const int blocks = (n + 15) / 16;
  const int tiles = (blocks + 7) / 8;
  return (blocks + tiles - 1) / tiles;
}

void launch_gemm_f32(const GemmArgs& a, int layout, int epi, int nb, int grid_n, int grid_m,
                     int batches, hipStream_t s) {
  dim3 grid(grid_n, grid_m, batches);
  if (epi == EPI_LOSS) {
    launch_nb<8, true, true, EPI_LOSS>(a, grid, s);
  } else if (epi == EPI_SOFTMAX_STATS) {
    launch_nb<8, true, true, EPI_SOFTMAX_STATS>(a, grid, s);
  } else if (layout == GEMM_NT) {
    launch_any_nb<true, true, EPI_STORE>(nb, a, grid, s);
  } else if (layout == GEMM_NN) {
    launch_any_nb<true, false, EPI_STORE>(nb, a, grid, s);
  } else {
    launch_any_nb<false, false, EPI_STORE>(nb, a, grid, s);
  }
}
