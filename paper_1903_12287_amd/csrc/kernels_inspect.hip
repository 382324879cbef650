// Inspection of one step's forward half (Sec. 3.1 scores and losses, Sec. 4.3
// chunk score blocks): copies of what the score contraction, its loss epilogue
// and the per-edge finalisation left in the workspace, in a plain layout.
// Nothing here takes part in training.
#include "kernels.h"

namespace {

// S[c][1][e][t] += bias[c][e]: the translation bias <theta_r, x_d> of the
// source side (translation with dot), added as the loss epilogues add it
__global__ __launch_bounds__(256) void add_side_bias_kernel(StepGeom g, const float* bias, float* out) {
  const int c = blockIdx.z;
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int Cc = chunk_edges(g, c);
  if (t >= Cc + g.U) return;
  for (int e = blockIdx.y; e < Cc; e += gridDim.y)
    out[((int64_t)(c * 2 + 1) * g.C + e) * g.N + t] += bias[(int64_t)c * g.C + e];
}

// dL/dS of every (chunk, side, edge, candidate) as the loss epilogue and the
// finalisation left it, as float32 [c][2][C][N]; entries outside the chunk's
// Cc rows and Cc + U columns are 0.
//   DS_BITS       the ranking bit matrix (word (w, row) at w * ldw + row)
//   DS_F32        float32 rows [C][ld]
//   DS_F32_SCALED float32 exp(s - tile max) rows times the row's tile scale
//                 exp(tile max - lse) ([2 c + side][nct][C])
//   DS_BF16       bf16 rows [C][ld]
__global__ __launch_bounds__(256) void expand_ds_kernel(StepGeom g, int mode, const uint16_t* bits, int nw,
                                                        int ldw, const float* f32, const float* scale,
                                                        const uint16_t* h, int ld, float* out) {
  const int z = blockIdx.z;
  const int c = z >> 1;
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= g.N) return;
  const int Cc = chunk_edges(g, c);
  for (int e = blockIdx.y; e < g.C; e += gridDim.y) {
    float v = 0.0f;
    if (e < Cc && t < Cc + g.U) {
      if (mode == DS_BITS) {
        const uint16_t w = bits[(int64_t)z * nw * ldw + (int64_t)(t >> 4) * ldw + e];
        v = ((w >> (t & 15)) & 1u) ? 1.0f : 0.0f;
      } else if (mode == DS_BF16) {
        v = __uint_as_float((uint32_t)h[((int64_t)z * g.C + e) * ld + t] << 16);
      } else {
        v = f32[((int64_t)z * g.C + e) * ld + t];
        if (mode == DS_F32_SCALED) v *= scale[((int64_t)z * g.nct + t / PBG_SCORE_BN) * g.C + e];
      }
    }
    out[((int64_t)z * g.C + e) * g.N + t] = v;
  }
}

// positive scores [c][C], or [c][2][C] with reciprocal predicates (0 past a
// short chunk's edges)
__global__ __launch_bounds__(256) void copy_pos_kernel(StepGeom g, const float* pos, float* out) {
  const int z = blockIdx.y;   // chunk, or chunk * 2 + side
  const int c = g.recip ? z >> 1 : z;
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= g.C) return;
  out[(int64_t)z * g.C + e] = e < chunk_edges(g, c) ? pos[(int64_t)z * g.C + e] : 0.0f;
}

}  // namespace

void launch_add_side_bias(const StepGeom& g, const float* bias, float* out, hipStream_t s) {
  if (g.nchunks <= 0) return;
  dim3 grid((g.N + 255) / 256, g.C < 4096 ? g.C : 4096, g.nchunks);
  add_side_bias_kernel<<<grid, 256, 0, s>>>(g, bias, out);
}

void launch_expand_ds(const StepGeom& g, int mode, const uint16_t* bits, int nw, int ldw, const float* f32,
                      const float* scale, const uint16_t* h, int ld, float* out, hipStream_t s) {
  if (g.nchunks <= 0) return;
  dim3 grid((g.N + 255) / 256, g.C < 4096 ? g.C : 4096, g.nchunks * 2);
  expand_ds_kernel<<<grid, 256, 0, s>>>(g, mode, bits, nw, ldw, f32, scale, h, ld, out);
}

void launch_copy_pos(const StepGeom& g, const float* pos, float* out, hipStream_t s) {
  if (g.nchunks <= 0) return;
  dim3 grid((g.C + 255) / 256, g.nchunks * (g.recip ? 2 : 1));
  copy_pos_kernel<<<grid, 256, 0, s>>>(g, pos, out);
}
