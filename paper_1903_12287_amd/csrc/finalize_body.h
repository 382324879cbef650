// Loss values and per-edge gradients of a step (Sec. 3.1 losses): the
// finalisation's workgroup body, shared by its own kernel and by the kernel
// that runs it beside the transposed piece split.
#pragma once

#include "kernels.h"
#include "device_common.h"

// ---- per-edge dL/dp, translation bias gradient, losses ------------------------
// Workgroup blk of chunk c (FIN_THREADS rows): writes its share of the chunk
// loss to parts[c * nblk + blk].
__device__ __forceinline__ void finalize_block(const StepGeom& g, const StepBufs& b, int softmax_scales,
                                               double* parts, int c, int blk, int nblk) {
  const int Cc = chunk_edges(g, c);
  double acc = 0.0;
  const int e = blk * FIN_THREADS + threadIdx.x;
  if (e < Cc) {
    const int64_t ce = (int64_t)c * g.C + e;
    const float p = b.pos[pos_index(g, c, 0, e)];
    const float p1 = b.pos[pos_index(g, c, 1, e)];   // p itself without reciprocal predicates
    float l0 = 0.f, l1 = 0.f, d0 = 0.f, d1 = 0.f;
    if (g.loss != LOSS_SOFTMAX) {
      const float* r0 = b.rowpart + ((int64_t)(c * 2 + 0) * g.C + e) * g.nct * 2;
      const float* r1 = b.rowpart + ((int64_t)(c * 2 + 1) * g.C + e) * g.nct * 2;
#pragma unroll 8
      for (int ct = 0; ct < g.nct; ++ct) {
        const float2 a0 = *(const float2*)(r0 + 2 * ct), a1 = *(const float2*)(r1 + 2 * ct);
        l0 += a0.x;
        d0 += a0.y;
        l1 += a1.x;
        d1 += a1.y;
      }
    }
    double loss;
    float dp, dp1 = 0.f, dsum1;
    float side_loss[2];
    if (g.recip) {
      // each side with its own positive score
      const float ps[2] = {p, p1};
      const float ls[2] = {l0, l1}, dsn[2] = {d0, d1};
      float dps[2];
      loss = 0.0;
#pragma unroll
      for (int side = 0; side < 2; ++side) {
        const float pp = ps[side];
        if (g.loss == LOSS_RANKING) {
          side_loss[side] = ls[side];
          dps[side] = -dsn[side];
        } else if (g.loss == LOSS_LOGISTIC) {
          side_loss[side] = ls[side] + softplusf(-pp);
          dps[side] = sigmoidf(pp) - 1.0f;
        } else {
          const float* rp = b.rowpart + ((int64_t)(c * 2 + side) * g.C + e) * g.nct * 2;
          float M = pp;
          for (int ct = 0; ct < g.nct; ++ct) M = fmaxf(M, rp[2 * ct]);
          float Z = expf(pp - M);
          for (int ct = 0; ct < g.nct; ++ct) {
            const float mx = rp[2 * ct];
            if (mx > -INFINITY) Z += rp[2 * ct + 1] * expf(mx - M);
          }
          const float lse = M + logf(Z);
          if (softmax_scales) {
            float* rs = b.rowscale + (int64_t)(c * 2 + side) * g.nct * g.C + e;
            for (int ct = 0; ct < g.nct; ++ct) {
              const float mx = rp[2 * ct];
              rs[(int64_t)ct * g.C] = mx > -INFINITY ? expf(mx - lse) : 0.0f;
            }
          }
          side_loss[side] = lse - pp;
          dps[side] = expf(pp - lse) - 1.0f;
        }
        loss += (double)side_loss[side];
      }
      dp = dps[0];
      dp1 = dps[1];
      dsum1 = 0.0f;   // no translation bias: both queries carry the operator
    } else if (g.loss == LOSS_RANKING) {
      loss = (double)l0 + (double)l1;
      dp = -(d0 + d1);
      dsum1 = d1;
      side_loss[0] = l0;
      side_loss[1] = l1;
    } else if (g.loss == LOSS_LOGISTIC) {
      const float sp = softplusf(-p);
      loss = (double)l0 + (double)l1 + 2.0 * (double)sp;
      dp = 2.0f * (sigmoidf(p) - 1.0f);
      dsum1 = d1;
      side_loss[0] = l0 + sp;
      side_loss[1] = l1 + sp;
    } else {
      // log-sum-exp of each side's row over {p} and its valid candidates, from
      // the per-tile (max M, sum exp(s - M)) partials; each tile's sum is then
      // replaced by exp(M - lse), which turns the stored exp(s - M) into dS
      float lse[2];
#pragma unroll
      for (int side = 0; side < 2; ++side) {
        const float* rp = b.rowpart + ((int64_t)(c * 2 + side) * g.C + e) * g.nct * 2;
        float M = p;
        for (int ct = 0; ct < g.nct; ++ct) M = fmaxf(M, rp[2 * ct]);
        float Z = expf(p - M);
        for (int ct = 0; ct < g.nct; ++ct) {
          const float mx = rp[2 * ct];
          if (mx > -INFINITY) Z += rp[2 * ct + 1] * expf(mx - M);
        }
        lse[side] = M + logf(Z);
        if (softmax_scales) {
          float* rs = b.rowscale + (int64_t)(c * 2 + side) * g.nct * g.C + e;
          for (int ct = 0; ct < g.nct; ++ct) {
            const float mx = rp[2 * ct];
            rs[(int64_t)ct * g.C] = mx > -INFINITY ? expf(mx - lse[side]) : 0.0f;
          }
        }
      }
      const float lse0 = lse[0], lse1 = lse[1];
      loss = ((double)lse0 - p) + ((double)lse1 - p);
      const float s0 = expf(p - lse0), s1 = expf(p - lse1);
      dp = (s0 - 1.0f) + (s1 - 1.0f);
      dsum1 = 1.0f - s1;
      side_loss[0] = lse0 - p;
      side_loss[1] = lse1 - p;
    }
    if (b.rowloss) {
      b.rowloss[(int64_t)(c * 2 + 0) * g.C + e] = side_loss[0];
      b.rowloss[(int64_t)(c * 2 + 1) * g.C + e] = side_loss[1];
    }
    if (g.cweight) {
      // the chunk's relation weight multiplies the edge's loss and every
      // gradient (the contractions' share is scaled as they store it)
      const float w = wave_uniform(g.cweight[c]);
      loss *= (double)w;
      dp *= w;
      dp1 *= w;
      dsum1 *= w;
    }
    b.dpos[pos_index(g, c, 0, e)] = dp;
    if (g.recip) b.dpos[pos_index(g, c, 1, e)] = dp1;
    b.dsum1[ce] = dsum1;
    acc += loss;
  }
  // fixed-order block reduction of this workgroup's share of the chunk loss
  __shared__ double red[FIN_THREADS];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int o = FIN_THREADS / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) parts[(int64_t)c * nblk + blk] = red[0];
}

