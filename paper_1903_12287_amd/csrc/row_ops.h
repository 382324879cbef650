// One embedding row held by one wave in registers, and the relation operators
// of the model (operator table of Sec. 3.1) applied to it.
//
// Real layout:    lane L holds elements f = L + 64q, q = 0..7 (dim <= 512).
// Complex layout: lane L holds real parts f = L + 64q (q = 0..3, f < h) in
//                 v[q] and the matching imaginary parts f + h in v[4 + q],
//                 h = dim / 2, so that a complex product stays inside a lane.
// Dots of two rows in the same layout are the plain real dot of the rows.
#pragma once

#include "device_common.h"

#define ROWQ 8

struct Row {
  float v[ROWQ];
};

__device__ __forceinline__ void row_zero(Row& r) {
#pragma unroll
  for (int q = 0; q < ROWQ; ++q) r.v[q] = 0.0f;
}

// element index held in slot q by this lane
__device__ __forceinline__ int row_index(int q, int lane, int d, bool cplx) {
  if (!cplx) return lane + 64 * q;
  const int h = d >> 1;
  return q < 4 ? lane + 64 * q : h + lane + 64 * (q - 4);
}

__device__ __forceinline__ bool row_valid(int q, int lane, int d, bool cplx) {
  if (!cplx) return lane + 64 * q < d;
  const int h = d >> 1;
  return lane + 64 * (q & 3) < h;
}

__device__ __forceinline__ void row_load(Row& r, const float* p, int d, bool cplx, int lane) {
#pragma unroll
  for (int q = 0; q < ROWQ; ++q)
    r.v[q] = row_valid(q, lane, d, cplx) ? p[row_index(q, lane, d, cplx)] : 0.0f;
}

// stores the row and zeroes the pad columns [d, dp)
__device__ __forceinline__ void row_store(const Row& r, float* p, int d, int dp, bool cplx, int lane) {
#pragma unroll
  for (int q = 0; q < ROWQ; ++q)
    if (row_valid(q, lane, d, cplx)) p[row_index(q, lane, d, cplx)] = r.v[q];
  if (d + lane < dp) p[d + lane] = 0.0f;
}

__device__ __forceinline__ float row_dot(const Row& a, const Row& b) {
  float s = 0.0f;
#pragma unroll
  for (int q = 0; q < ROWQ; ++q) s += a.v[q] * b.v[q];
  return wave_sum(s);
}

__device__ __forceinline__ void row_scale(Row& r, float s) {
#pragma unroll
  for (int q = 0; q < ROWQ; ++q) r.v[q] *= s;
}

__device__ __forceinline__ void row_axpy(Row& y, float a, const Row& x) {
#pragma unroll
  for (int q = 0; q < ROWQ; ++q) y.v[q] += a * x.v[q];
}

__device__ __forceinline__ void row_add(Row& y, const Row& x) {
#pragma unroll
  for (int q = 0; q < ROWQ; ++q) y.v[q] += x.v[q];
}

// unit vector with the norm clamped at 1e-12; returns the (unclamped) norm
__device__ __forceinline__ float row_normalize(Row& r) {
  const float n = sqrtf(row_dot(r, r));
  row_scale(r, 1.0f / fmaxf(n, PBG_EPS_NORM));
  return n;
}

// gradient through v_hat = v / max(|v|, eps): given v_hat, |v| and dL/dv_hat
__device__ __forceinline__ Row normalize_backward(const Row& vh, float nrm, const Row& dvh) {
  Row g;
  if (nrm > PBG_EPS_NORM) {
    const float c = row_dot(vh, dvh);
    const float inv = 1.0f / nrm;
#pragma unroll
    for (int q = 0; q < ROWQ; ++q) g.v[q] = (dvh.v[q] - vh.v[q] * c) * inv;
  } else {
#pragma unroll
    for (int q = 0; q < ROWQ; ++q) g.v[q] = dvh.v[q] * (1.0f / PBG_EPS_NORM);
  }
  return g;
}

// Products with a d x d relation matrix.  `stage` is this wave's LDS scratch
// of >= d floats; `mat` is the row-major matrix (for A x) or its transpose.
//   mat_apply(out, mat, x):  out[k] = sum_l mat[l*d + k] * x[l]
// With mat = A^T this is A x; with mat = A it is A^T x.  Lanes read
// consecutive k, so the matrix reads are coalesced.
__device__ __forceinline__ void mat_apply(Row& out, const float* mat, const Row& x, float* stage,
                                          int d, int lane) {
#pragma unroll
  for (int q = 0; q < ROWQ; ++q)
    if (lane + 64 * q < d) stage[lane + 64 * q] = x.v[q];
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  Row o;
  row_zero(o);
  for (int l = 0; l < d; ++l) {
    const float xl = stage[l];
    const float* mrow = mat + (size_t)l * d;
#pragma unroll
    for (int q = 0; q < ROWQ; ++q)
      if (lane + 64 * q < d) o.v[q] += mrow[lane + 64 * q] * xl;
  }
  __builtin_amdgcn_wave_barrier();
  out = o;
}

// g(x, theta) for the non-matrix operators (real or complex layout)
__device__ __forceinline__ Row op_forward(int op, const Row& x, const Row& th) {
  Row o;
  if (op == OP_TRANSLATION) {
#pragma unroll
    for (int q = 0; q < ROWQ; ++q) o.v[q] = x.v[q] + th.v[q];
  } else if (op == OP_DIAGONAL) {
#pragma unroll
    for (int q = 0; q < ROWQ; ++q) o.v[q] = x.v[q] * th.v[q];
  } else if (op == OP_COMPLEX) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float xr = x.v[q], xi = x.v[4 + q], tr = th.v[q], ti = th.v[4 + q];
      o.v[q] = xr * tr - xi * ti;
      o.v[4 + q] = xr * ti + xi * tr;
    }
  } else {
    o = x;
  }
  return o;
}

// adjoint g*(y, theta) with <g(x), y> = <x, g*(y)> for the operators that are
// linear in x (identity, diagonal, complex); translation returns y itself.
// The same map is the transposed Jacobian of g with respect to x.
__device__ __forceinline__ Row op_adjoint(int op, const Row& y, const Row& th) {
  Row o;
  if (op == OP_DIAGONAL) {
#pragma unroll
    for (int q = 0; q < ROWQ; ++q) o.v[q] = y.v[q] * th.v[q];
  } else if (op == OP_COMPLEX) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float yr = y.v[q], yi = y.v[4 + q], tr = th.v[q], ti = th.v[4 + q];
      o.v[q] = tr * yr + ti * yi;       // conj(theta) * y
      o.v[4 + q] = tr * yi - ti * yr;
    }
  } else {
    o = y;
  }
  return o;
}

// dL/dtheta of g(x, theta) given dL/dg (translation, diagonal, complex)
__device__ __forceinline__ Row op_param_grad(int op, const Row& x, const Row& dg) {
  Row o;
  if (op == OP_DIAGONAL) {
#pragma unroll
    for (int q = 0; q < ROWQ; ++q) o.v[q] = x.v[q] * dg.v[q];
  } else if (op == OP_COMPLEX) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float xr = x.v[q], xi = x.v[4 + q], gr = dg.v[q], gi = dg.v[4 + q];
      o.v[q] = xr * gr + xi * gi;       // conj(x) * dg
      o.v[4 + q] = xr * gi - xi * gr;
    }
  } else {
    o = dg;
  }
  return o;
}

// dL/dtheta of the adjoint g*(y, theta) given dL/dg* (diagonal, complex)
__device__ __forceinline__ Row op_adjoint_param_grad(int op, const Row& y, const Row& dk) {
  Row o;
  if (op == OP_DIAGONAL) {
#pragma unroll
    for (int q = 0; q < ROWQ; ++q) o.v[q] = y.v[q] * dk.v[q];
  } else if (op == OP_COMPLEX) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float yr = y.v[q], yi = y.v[4 + q], kr = dk.v[q], ki = dk.v[4 + q];
      o.v[q] = yr * kr + yi * ki;       // y * conj(dk)
      o.v[4 + q] = yi * kr - yr * ki;
    }
  } else {
    row_zero(o);
  }
  return o;
}
