// One embedding row held by one wave in registers, and the relation operators
// of the model (operator table of Sec. 3.1) applied to it.
//
// RowT<RQ>: each lane holds RQ floats of the row (dim <= 64 RQ).
// Real layout:    lane L holds elements f = L + 64q, q = 0..RQ-1.
// Complex layout: lane L holds real parts f = L + 64q (q < RQ/2, f < h) in
//                 v[q] and the matching imaginary parts f + h in v[RQ/2 + q],
//                 h = dim / 2, so that a complex product stays inside a lane.
// Dots of two rows in the same layout are the plain real dot of the rows.
// Kernels pick the narrowest RQ that holds their dim (2 for dim <= 128, 4 for
// <= 256, 8 for <= 512); Row is the widest.
#pragma once

#include "device_common.h"

#define ROWQ 8

template <int RQ>
struct RowT {
  float v[RQ];
};
typedef RowT<ROWQ> Row;

// floats per lane a kernel instantiation needs for a row of `dim` elements
__host__ __device__ inline int row_width_for(int dim) { return dim <= 128 ? 2 : (dim <= 256 ? 4 : 8); }

template <int RQ>
__device__ __forceinline__ void row_zero(RowT<RQ>& r) {
#pragma unroll
  for (int q = 0; q < RQ; ++q) r.v[q] = 0.0f;
}

// element index held in slot q by this lane
template <int RQ>
__device__ __forceinline__ int row_index(int q, int lane, int d, bool cplx) {
  if (!cplx) return lane + 64 * q;
  const int h = d >> 1;
  return q < RQ / 2 ? lane + 64 * q : h + lane + 64 * (q - RQ / 2);
}

template <int RQ>
__device__ __forceinline__ bool row_valid(int q, int lane, int d, bool cplx) {
  if (!cplx) return lane + 64 * q < d;
  const int h = d >> 1;
  return lane + 64 * (q % (RQ / 2)) < h;
}

template <int RQ>
__device__ __forceinline__ void row_load(RowT<RQ>& r, const float* p, int d, bool cplx, int lane) {
#pragma unroll
  for (int q = 0; q < RQ; ++q)
    r.v[q] = row_valid<RQ>(q, lane, d, cplx) ? p[row_index<RQ>(q, lane, d, cplx)] : 0.0f;
}

// stores the row and zeroes the pad columns [d, dp) (dp - d <= 64)
template <int RQ>
__device__ __forceinline__ void row_store(const RowT<RQ>& r, float* p, int d, int dp, bool cplx, int lane) {
#pragma unroll
  for (int q = 0; q < RQ; ++q)
    if (row_valid<RQ>(q, lane, d, cplx)) p[row_index<RQ>(q, lane, d, cplx)] = r.v[q];
  if (d + lane < dp) p[d + lane] = 0.0f;
}

template <int RQ>
__device__ __forceinline__ float row_dot(const RowT<RQ>& a, const RowT<RQ>& b) {
  float s = 0.0f;
#pragma unroll
  for (int q = 0; q < RQ; ++q) s += a.v[q] * b.v[q];
  return wave_sum(s);
}

template <int RQ>
__device__ __forceinline__ void row_scale(RowT<RQ>& r, float s) {
#pragma unroll
  for (int q = 0; q < RQ; ++q) r.v[q] *= s;
}

template <int RQ>
__device__ __forceinline__ void row_axpy(RowT<RQ>& y, float a, const RowT<RQ>& x) {
#pragma unroll
  for (int q = 0; q < RQ; ++q) y.v[q] += a * x.v[q];
}

template <int RQ>
__device__ __forceinline__ void row_add(RowT<RQ>& y, const RowT<RQ>& x) {
#pragma unroll
  for (int q = 0; q < RQ; ++q) y.v[q] += x.v[q];
}

// unit vector with the norm clamped at 1e-12; returns the (unclamped) norm
template <int RQ>
__device__ __forceinline__ float row_normalize(RowT<RQ>& r) {
  const float n = sqrtf(row_dot(r, r));
  row_scale(r, 1.0f / fmaxf(n, PBG_EPS_NORM));
  return n;
}

// gradient through v_hat = v / max(|v|, eps): given v_hat, |v| and dL/dv_hat
template <int RQ>
__device__ __forceinline__ RowT<RQ> normalize_backward(const RowT<RQ>& vh, float nrm, const RowT<RQ>& dvh) {
  RowT<RQ> g;
  if (nrm > PBG_EPS_NORM) {
    const float c = row_dot(vh, dvh);
    const float inv = 1.0f / nrm;
#pragma unroll
    for (int q = 0; q < RQ; ++q) g.v[q] = (dvh.v[q] - vh.v[q] * c) * inv;
  } else {
#pragma unroll
    for (int q = 0; q < RQ; ++q) g.v[q] = dvh.v[q] * (1.0f / PBG_EPS_NORM);
  }
  return g;
}

// Products with a d x d relation matrix.  `stage` is this wave's LDS scratch
// of >= d floats; `mat` is the row-major matrix (for A x) or its transpose.
//   mat_apply(out, mat, x):  out[k] = sum_l mat[l*d + k] * x[l]
// With mat = A^T this is A x; with mat = A it is A^T x.  Lanes read
// consecutive k, so the matrix reads are coalesced.
template <int RQ>
__device__ __forceinline__ void mat_apply(RowT<RQ>& out, const float* mat, const RowT<RQ>& x, float* stage,
                                          int d, int lane) {
#pragma unroll
  for (int q = 0; q < RQ; ++q)
    if (lane + 64 * q < d) stage[lane + 64 * q] = x.v[q];
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  RowT<RQ> o;
  row_zero(o);
  for (int l = 0; l < d; ++l) {
    const float xl = stage[l];
    const float* mrow = mat + (size_t)l * d;
#pragma unroll
    for (int q = 0; q < RQ; ++q)
      if (lane + 64 * q < d) o.v[q] += mrow[lane + 64 * q] * xl;
  }
  __builtin_amdgcn_wave_barrier();
  out = o;
}

// out = M x for a row-major d x d matrix M (out[k] = sum_l M[k*d + l] x[l]):
// each lane walks its own output rows, so consecutive iterations read
// consecutive floats of each row (the lines stay in the vector cache).
template <int RQ>
__device__ __forceinline__ void mat_rows_apply(RowT<RQ>& out, const float* M, const RowT<RQ>& x, float* stage,
                                               int d, int lane) {
#pragma unroll
  for (int q = 0; q < RQ; ++q)
    if (lane + 64 * q < d) stage[lane + 64 * q] = x.v[q];
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  RowT<RQ> o;
  row_zero(o);
  for (int l = 0; l < d; ++l) {
    const float xl = stage[l];
#pragma unroll
    for (int q = 0; q < RQ; ++q)
      if (lane + 64 * q < d) o.v[q] += M[(size_t)(lane + 64 * q) * d + l] * xl;
  }
  __builtin_amdgcn_wave_barrier();
  out = o;
}

// g(x, theta) for the non-matrix operators (real or complex layout)
template <int RQ>
__device__ __forceinline__ RowT<RQ> op_forward(int op, const RowT<RQ>& x, const RowT<RQ>& th) {
  constexpr int H = RQ / 2;
  RowT<RQ> o;
  if (op == OP_TRANSLATION) {
#pragma unroll
    for (int q = 0; q < RQ; ++q) o.v[q] = x.v[q] + th.v[q];
  } else if (op == OP_DIAGONAL) {
#pragma unroll
    for (int q = 0; q < RQ; ++q) o.v[q] = x.v[q] * th.v[q];
  } else if (op == OP_COMPLEX) {
#pragma unroll
    for (int q = 0; q < H; ++q) {
      const float xr = x.v[q], xi = x.v[H + q], tr = th.v[q], ti = th.v[H + q];
      o.v[q] = xr * tr - xi * ti;
      o.v[H + q] = xr * ti + xi * tr;
    }
  } else {
    o = x;
  }
  return o;
}

// adjoint g*(y, theta) with <g(x), y> = <x, g*(y)> for the operators that are
// linear in x (identity, diagonal, complex); translation returns y itself.
// The same map is the transposed Jacobian of g with respect to x.
template <int RQ>
__device__ __forceinline__ RowT<RQ> op_adjoint(int op, const RowT<RQ>& y, const RowT<RQ>& th) {
  constexpr int H = RQ / 2;
  RowT<RQ> o;
  if (op == OP_DIAGONAL) {
#pragma unroll
    for (int q = 0; q < RQ; ++q) o.v[q] = y.v[q] * th.v[q];
  } else if (op == OP_COMPLEX) {
#pragma unroll
    for (int q = 0; q < H; ++q) {
      const float yr = y.v[q], yi = y.v[H + q], tr = th.v[q], ti = th.v[H + q];
      o.v[q] = tr * yr + ti * yi;       // conj(theta) * y
      o.v[H + q] = tr * yi - ti * yr;
    }
  } else {
    o = y;
  }
  return o;
}

// dL/dtheta of g(x, theta) given dL/dg (translation, diagonal, complex)
template <int RQ>
__device__ __forceinline__ RowT<RQ> op_param_grad(int op, const RowT<RQ>& x, const RowT<RQ>& dg) {
  constexpr int H = RQ / 2;
  RowT<RQ> o;
  if (op == OP_DIAGONAL) {
#pragma unroll
    for (int q = 0; q < RQ; ++q) o.v[q] = x.v[q] * dg.v[q];
  } else if (op == OP_COMPLEX) {
#pragma unroll
    for (int q = 0; q < H; ++q) {
      const float xr = x.v[q], xi = x.v[H + q], gr = dg.v[q], gi = dg.v[H + q];
      o.v[q] = xr * gr + xi * gi;       // conj(x) * dg
      o.v[H + q] = xr * gi - xi * gr;
    }
  } else {
    o = dg;
  }
  return o;
}

// dL/dtheta of the adjoint g*(y, theta) given dL/dg* (diagonal, complex)
template <int RQ>
__device__ __forceinline__ RowT<RQ> op_adjoint_param_grad(int op, const RowT<RQ>& y, const RowT<RQ>& dk) {
  constexpr int H = RQ / 2;
  RowT<RQ> o;
  if (op == OP_DIAGONAL) {
#pragma unroll
    for (int q = 0; q < RQ; ++q) o.v[q] = y.v[q] * dk.v[q];
  } else if (op == OP_COMPLEX) {
#pragma unroll
    for (int q = 0; q < H; ++q) {
      const float yr = y.v[q], yi = y.v[H + q], kr = dk.v[q], ki = dk.v[H + q];
      o.v[q] = yr * kr + yi * ki;       // y * conj(dk)
      o.v[H + q] = yi * kr - yr * ki;
    }
  } else {
    row_zero(o);
  }
  return o;
}
