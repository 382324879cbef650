// Float32 contractions on the gfx950 matrix cores (v_mfma_f32_16x16x4_f32),
// for the small products of the linear operator (Sec. 3.1: g(x) = A x with one
// relation, formed for a whole step: Q = X A^T, K = Y A, and in the backward
// X and Y gradients and dA).  The chunk x candidates contractions of the score
// and its backward run on the bf16 instructions (kernels_gemm_bf16.hip).
//
// A 256-thread workgroup (4 waves in a 2 x 2 arrangement) computes a 128 x BN
// tile (BN = 128, or 64 for narrow outputs); each wave owns 64 x BN/2 outputs,
// i.e. 4 x BN/32 blocks of 16 x 16.  Layouts: NT  A[m][k], B[n][k];
// TN  A[k][m], B[k][n].
//
// Operands reach LDS through buffer loads (a load whose offset is out of the
// buffer's range returns zeros, which pads ragged tiles without branches) and
// a register-held prefetch of the next 16-deep k-slice, double-buffered in
// LDS.  An operand that is contiguous along k is kept as [row][k] (pitch 20
// floats) and read back as one 128-bit fragment per 16 x 16 block and
// k-slice; an operand contiguous along its row index is kept as [k][row]
// (pitch BM + 4) and read one float per step.  Both layouts are free of LDS
// bank conflicts for the fragment reads.
//
// The 16x16x4 instruction sums A[m][k] B[k][n] over the four k held by the
// four 16-lane groups (lane L: A row L % 16, B column L % 16, k index L / 16).
// Lane group g supplies k = 4g + kk at step kk of a slice, so a 128-bit read
// of four consecutive k feeds four steps; every k of the slice is used once.
// Accumulator: lane L, register r holds D[4 (L / 16) + r][L % 16].
//
// Workgroups are numbered so that the tiles of one batch run on the same XCD,
// whose L2 then holds that batch's operands.
#include "kernels.h"
#include "device_common.h"

namespace {

constexpr int BM = 128;
constexpr int BK = 16;
constexpr int KP = BK + 4;     // pitch of a [row][k] tile
constexpr uint32_t OOB = 0x80000000u;

typedef __amdgpu_buffer_rsrc_t rsrc_t;

// A buffer descriptor must be wave-uniform.  Tile base addresses are, but
// their 64-bit products are formed on the vector unit, and a descriptor left
// in vector registers would make the compiler wrap every load that uses it in
// a loop over lanes; reading the address back from the first lane keeps it
// scalar.
__device__ __forceinline__ rsrc_t make_rsrc(const float* p) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), (short)0, 0x7FFFFFF0, 0x00020000);
}

__device__ __forceinline__ v4f bload(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

__device__ __forceinline__ int pick_dim(int sel, int fixed, int Cc, int Nc) {
  return sel == DIM_CC ? Cc : (sel == DIM_NC ? Nc : fixed);
}

// One operand tile of TX rows (M or N) x BK k.  KC: global [x][k] with leading
// dimension ld (k contiguous); otherwise global [k][x] (x contiguous).
template <int TX, bool KC>
struct Tile {
  static constexpr int LOADS = TX * BK / 4 / 256;   // float4 per thread
  static constexpr int PITCH = KC ? KP : TX + 4;
  static constexpr int SIZE = KC ? TX * KP : BK * (TX + 4);

  __device__ __forceinline__ static void load(v4f* r, rsrc_t rs, int ld, int x0, int xdim, int k0, int kdim, int tid) {
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int f = tid + 256 * q;
      uint32_t off = OOB;
      if (KC) {
        const int x = f >> 2, kq = f & 3;
        const int gx = x0 + x, gk = k0 + 4 * kq;
        if (gx < xdim && gk < ((kdim + 3) & ~3)) off = (uint32_t)(((int64_t)gx * ld + gk) * 4);
      } else {
        const int k = f / (TX / 4), xq = f % (TX / 4);
        const int gk = k0 + k, gx = x0 + 4 * xq;
        if (gk < kdim && gx < ((xdim + 3) & ~3)) off = (uint32_t)(((int64_t)gk * ld + gx) * 4);
      }
      r[q] = bload(rs, off);
    }
  }

  __device__ __forceinline__ static void store(float* s, const v4f* r, int tid) {
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int f = tid + 256 * q;
      if (KC) {
        const int x = f >> 2, kq = f & 3;
        *(v4f*)(s + x * KP + 4 * kq) = r[q];
      } else {
        const int k = f / (TX / 4), xq = f % (TX / 4);
        *(v4f*)(s + k * (TX + 4) + 4 * xq) = r[q];
      }
    }
  }
};

template <int BN, bool AK, bool BKC>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a, int tiles_n, int tiles_m) {
  constexpr int WN = BN / 2;       // columns per wave
  constexpr int JN = WN / 16;      // 16-wide column blocks per wave
  using TA = Tile<BM, AK>;
  using TB = Tile<BN, BKC>;
  __shared__ __align__(16) float As[2][TA::SIZE];
  __shared__ __align__(16) float Bs[2][TB::SIZE];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int w = tid >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int l16 = lane & 15, g = lane >> 4;

  // XCD-aware numbering: consecutive hardware ids go round-robin over 8 XCDs
  const int nwg = gridDim.x, id = blockIdx.x;
  const int q8 = nwg >> 3, r8 = nwg & 7, xcd = id & 7;
  const int lid = xcd * q8 + min(xcd, r8) + (id >> 3);
  const int tn = lid % tiles_n;
  const int rest = lid / tiles_n;
  const int tm = rest % tiles_m;
  const int z = rest / tiles_m;

  const int c = z / a.nsides;
  const int side = z - c * a.nsides;
  int Cc = a.C, Nc = a.C + a.U;
  if (a.cstart) {
    Cc = wave_uniform(a.cstart[c + 1] - a.cstart[c]);
    Nc = Cc + a.U;
  } else if (a.m_step > 0) {
    Cc = min(a.C, a.m_step - c * a.C);
    Nc = Cc + a.U;
  }
  const int M = pick_dim(a.mdim, a.Mfix, Cc, Nc);
  const int N = pick_dim(a.ndim, a.Nfix, Cc, Nc);
  const int K = pick_dim(a.kdim, a.Kfix, Cc, Nc);
  const int m0 = tm * BM;
  const int n0 = tn * BN;
  if (m0 >= M) return;

  if (n0 >= N) return;

  const rsrc_t ra_s = make_rsrc(a.A + c * a.a_cs + side * a.a_ss);
  const rsrc_t rb_s = make_rsrc(a.B + c * a.b_cs + side * a.b_ss);

  v4f acc[4][JN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < JN; ++j) acc[i][j] = (v4f){0.f, 0.f, 0.f, 0.f};

  v4f pa[TA::LOADS], pb[TB::LOADS];
  const int nk = (K + BK - 1) / BK;
  TA::load(pa, ra_s, a.lda, m0, M, 0, K, tid);
  TB::load(pb, rb_s, a.ldb, n0, N, 0, K, tid);
  TA::store(As[0], pa, tid);
  TB::store(Bs[0], pb, tid);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) {
      TA::load(pa, ra_s, a.lda, m0, M, (kt + 1) * BK, K, tid);
      TB::load(pb, rb_s, a.ldb, n0, N, (kt + 1) * BK, K, tid);
    }
    const float* as = As[buf];
    const float* bs = Bs[buf];
    if (AK && BKC) {
      v4f af[4], bf[JN];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *(const v4f*)(as + (64 * wm + 16 * i + l16) * KP + 4 * g);
#pragma unroll
      for (int j = 0; j < JN; ++j) bf[j] = *(const v4f*)(bs + (WN * wn + 16 * j + l16) * KP + 4 * g);
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < JN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i][kk], bf[j][kk], acc[i][j], 0, 0, 0);
    } else {
      v4f af4[4];
      if (AK) {
#pragma unroll
        for (int i = 0; i < 4; ++i) af4[i] = *(const v4f*)(as + (64 * wm + 16 * i + l16) * KP + 4 * g);
      }
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        float af[4], bf[JN];
        const int kr = 4 * g + kk;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          af[i] = AK ? af4[i][kk] : as[kr * (BM + 4) + 64 * wm + 16 * i + l16];
#pragma unroll
        for (int j = 0; j < JN; ++j) bf[j] = bs[kr * (BN + 4) + WN * wn + 16 * j + l16];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < JN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i], bf[j], acc[i][j], 0, 0, 0);
      }
    }
    if (kt + 1 < nk) {
      TA::store(As[buf ^ 1], pa, tid);
      TB::store(Bs[buf ^ 1], pb, tid);
    }
    __syncthreads();
  }

  float* Cm = a.Cm + c * a.c_cs + side * a.c_ss;
  const int colb = n0 + WN * wn + l16;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = m0 + 64 * wm + 16 * i + 4 * g + r;
      if (m < M) {
#pragma unroll
        for (int j = 0; j < JN; ++j) {
          const int n = colb + 16 * j;
          if (n < N) {
            float* o = Cm + (int64_t)m * a.ldc + n;
            *o = a.accumulate ? *o + acc[i][j][r] : acc[i][j][r];
          }
        }
      }
    }
}

template <int BN, bool AK, bool BKC>
void launch_t(const GemmArgs& a, int tiles_n, int tiles_m, int batches, hipStream_t s) {
  const int64_t nwg = (int64_t)tiles_n * tiles_m * batches;
  gemm_f32_kernel<BN, AK, BKC><<<(unsigned)nwg, 256, 0, s>>>(a, tiles_n, tiles_m);
}

int dim_max(int sel, int fixed, int C, int U) { return sel == DIM_CC ? C : (sel == DIM_NC ? C + U : fixed); }

}  // namespace

void launch_gemm_f32(const GemmArgs& a, int layout, int batches, hipStream_t s) {
  const int maxM = dim_max(a.mdim, a.Mfix, a.C, a.U);
  const int maxN = dim_max(a.ndim, a.Nfix, a.C, a.U);
  if (maxM <= 0 || maxN <= 0 || batches <= 0) return;
  const int tiles_m = (maxM + BM - 1) / BM;
  const bool narrow = maxN <= 64;
  const int tiles_n = (maxN + (narrow ? 63 : 127)) / (narrow ? 64 : 128);
  if (layout == GEMM_NT) {
    if (narrow) launch_t<64, true, true>(a, tiles_n, tiles_m, batches, s);
    else launch_t<128, true, true>(a, tiles_n, tiles_m, batches, s);
  } else {
    if (narrow) launch_t<64, false, false>(a, tiles_n, tiles_m, batches, s);
    else launch_t<128, false, false>(a, tiles_n, tiles_m, batches, s);
  }
}
