// Device-side helpers shared by the gfx950 kernels of the bucket-training path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "geometry.h"

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

#define PBG_WAVE 64

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two 32x32
// multiplies whose high and low halves are mixed with the other counter words
// and the key; the key is advanced by the Weyl constants between rounds.
// ---------------------------------------------------------------------------
struct Philox4 {
  uint32_t v[4];
};

__device__ __forceinline__ Philox4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2,
                                                 uint32_t c3, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    const uint32_t n0 = hi1 ^ c1 ^ k0;
    const uint32_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  Philox4 o;
  o.v[0] = c0;
  o.v[1] = c1;
  o.v[2] = c2;
  o.v[3] = c3;
  return o;
}

// Uniform negative k of (chunk, bucket, side) in [0, rows): floor(w * rows / 2^32).
__device__ __forceinline__ int32_t uniform_negative(uint64_t seed, uint32_t bucket, uint64_t chunk,
                                                    uint32_t side, uint32_t k, uint32_t rows) {
  const Philox4 w = philox4x32_10(k >> 2, (uint32_t)chunk, bucket, side, (uint32_t)seed,
                                  (uint32_t)(seed >> 32));
  const uint32_t word = w.v[k & 3u];
  return (int32_t)(((uint64_t)word * (uint64_t)rows) >> 32);
}

// the four candidates k4 .. k4 + 3 (k4 a multiple of 4) of one Philox block
__device__ __forceinline__ void uniform_negatives4(uint64_t seed, uint32_t bucket, uint64_t chunk, uint32_t side,
                                                   uint32_t k4, uint32_t rows, int32_t* out) {
  const Philox4 w = philox4x32_10(k4 >> 2, (uint32_t)chunk, bucket, side, (uint32_t)seed, (uint32_t)(seed >> 32));
#pragma unroll
  for (int q = 0; q < 4; ++q) out[q] = (int32_t)(((uint64_t)w.v[q] * (uint64_t)rows) >> 32);
}

// ---------------------------------------------------------------------------
// wave reductions (64 lanes)
// ---------------------------------------------------------------------------
// Lane exchanges inside a 16-lane row through DPP (no LDS round trip):
// quad_perm [1,0,3,2] and [2,3,0,1] swap lanes 1 and 2 apart, half-mirror
// swaps the two quads of each half-row, mirror the two halves of the row.
// Each step pairs lanes symmetrically, so all lanes of a row end with the
// same value (a + b and b + a are equal).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
#define PBG_DPP_QUAD_XOR1 0xB1
#define PBG_DPP_QUAD_XOR2 0x4E
#define PBG_DPP_ROW_HALF_MIRROR 0x141
#define PBG_DPP_ROW_MIRROR 0x140

// sum over the 16 consecutive lanes of a group (lanes 16g .. 16g+15)
__device__ __forceinline__ float group16_sum(float x) {
  x += dpp_f<PBG_DPP_QUAD_XOR1>(x);
  x += dpp_f<PBG_DPP_QUAD_XOR2>(x);
  x += dpp_f<PBG_DPP_ROW_HALF_MIRROR>(x);
  x += dpp_f<PBG_DPP_ROW_MIRROR>(x);
  return x;
}

__device__ __forceinline__ float group16_max(float x) {
  x = fmaxf(x, dpp_f<PBG_DPP_QUAD_XOR1>(x));
  x = fmaxf(x, dpp_f<PBG_DPP_QUAD_XOR2>(x));
  x = fmaxf(x, dpp_f<PBG_DPP_ROW_HALF_MIRROR>(x));
  x = fmaxf(x, dpp_f<PBG_DPP_ROW_MIRROR>(x));
  return x;
}

// sum over the wave: the four rows by DPP, then the rows pairwise
// Row-wise Adagrad step size 1 / (sqrt(G) + eps) (Sec. 3.1: the accumulated
// squared gradient of a row scales its update), from the hardware square
// root and reciprocal, each within one unit in the last place: every update
// of the library takes it from here, so all paths round alike.
__device__ __forceinline__ float adagrad_rcp(float G) {
  return __builtin_amdgcn_rcpf(__builtin_amdgcn_sqrtf(G) + PBG_EPS_ADAGRAD);
}

__device__ __forceinline__ float wave_sum(float x) {
  x = group16_sum(x);
  x += __shfl_xor(x, 16, PBG_WAVE);
  x += __shfl_xor(x, 32, PBG_WAVE);
  return x;
}

__device__ __forceinline__ double wave_sum_d(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, PBG_WAVE);
  return x;
}

// numerically stable softplus(x) = log(1 + e^x) and logistic sigmoid
__device__ __forceinline__ float softplusf(float x) {
  return fmaxf(x, 0.0f) + log1pf(expf(-fabsf(x)));
}
__device__ __forceinline__ float sigmoidf(float x) {
  if (x >= 0.0f) return 1.0f / (1.0f + expf(-x));
  const float e = expf(x);
  return e / (1.0f + e);
}

// sigmoid(s) and softplus(s) = log(1 + e^s) from one exponential
// e = exp(-|s|) in (0, 1]: sigmoid = 1/(1+e) or e/(1+e), softplus =
// max(s, 0) + log1p(e), with log1p(e) = log(u) * e / (u - 1), u = 1 + e,
// which stays accurate when e is tiny (u - 1 is then exact)
__device__ __forceinline__ void logistic_pair(float s, float& sig, float& sp) {
  const float e = __expf(-fabsf(s));
  const float u = 1.0f + e;
  const float r = 1.0f / u;
  sig = s >= 0.0f ? r : e * r;
  const float um1 = u - 1.0f;
  const float l1p = um1 == 0.0f ? e : __logf(u) * (e / um1);
  sp = fmaxf(s, 0.0f) + l1p;
}

// round-to-nearest-even fp32 -> bf16 (finite inputs)
__device__ __forceinline__ __bf16 to_bf16(float x) { return (__bf16)x; }
