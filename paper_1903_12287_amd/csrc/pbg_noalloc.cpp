// pbg_score_edges_noalloc: edge scores (Sec. 3.1 score f) for callers that
// cannot allocate device memory.  The scratch that pbg_score_edges allocates
// per call (the id-check flag and, for the linear operator, the transposed
// relation matrices) lives here in one file-scope device array instead.
//
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is taken once per device with hipGetSymbolAddress (at
// context creation, with that device current) and only that address is
// passed to kernels and copies.  Every call on a device shares the device's
// array, so calls that overlap on one device race.
#include <hip/hip_runtime.h>

#include <cstring>
#include <mutex>

#include "kernels.h"
#include "pbg.h"
#include "runtime_internal.h"

namespace {

// 256 bytes of flags, then the transposed relation matrices
constexpr int64_t kFlagFloats = 64;
constexpr int64_t kScratchFloats = kFlagFloats + PBG_NOALLOC_MAX_REL_FLOATS;

__device__ __align__(256) float scratch[kScratchFloats];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

pbg_status noalloc_scratch_init(pbg_ctx* ctx) {
  if (ctx->device < 0 || ctx->device >= kMaxDevices)
    return set_err(ctx, PBG_ERR_DEVICE, "device %d out of the supported range", ctx->device);
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_ptr[ctx->device]) return PBG_OK;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !p) {
    (void)hipGetLastError();
    return set_err(ctx, PBG_ERR_DEVICE, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
  }
  g_ptr[ctx->device] = p;
  return PBG_OK;
}

extern "C" pbg_status pbg_score_edges_noalloc(pbg_ctx* ctx, int32_t i, int32_t j, const int32_t* src_local,
                                              const int32_t* rel, const int32_t* dst_local, int64_t n,
                                              float* scores) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  if (ctx->invalid) return set_err(ctx, PBG_ERR_STATE, "context failed to initialise");
  ctx->err.clear();
  if (ctx->T > 1) return set_err(ctx, PBG_ERR_UNSUPPORTED, "pbg_score_edges_noalloc takes one entity type");
  if (i < 0 || i >= ctx->P || j < 0 || j >= ctx->P)
    return set_err(ctx, PBG_ERR_INVALID_ARG, "bucket (%d, %d) out of range", i, j);
  if (n < 0 || n > 0x7FFFFFFFll) return set_err(ctx, PBG_ERR_INVALID_ARG, "n out of range");
  const int64_t rel_floats = ctx->op == OP_LINEAR ? (int64_t)ctx->R * ctx->d * ctx->d : 0;
  if (rel_floats > PBG_NOALLOC_MAX_REL_FLOATS)
    return set_err(ctx, PBG_ERR_INVALID_ARG,
                   "the linear operator's %lld relation floats exceed the static scratch of %lld floats",
                   (long long)rel_floats, (long long)PBG_NOALLOC_MAX_REL_FLOATS);
  const Partition& pi = ctx->parts[i];
  const Partition& pj = ctx->parts[j];
  if (!pi.emb || !pj.emb || pi.where != PBG_MEM_DEVICE || pj.where != PBG_MEM_DEVICE)
    return set_err(ctx, PBG_ERR_STATE, "partitions %d and %d must be bound in device memory", i, j);
  if (ctx->op != OP_IDENTITY && !ctx->relp) return set_err(ctx, PBG_ERR_STATE, "relation parameters are not bound");
  if (n == 0) return PBG_OK;
  if (ctx->R > 1 && !rel) return set_err(ctx, PBG_ERR_INVALID_ARG, "rel may be NULL only with one relation");
  if (!src_local || !dst_local || !scores) return set_err(ctx, PBG_ERR_INVALID_ARG, "NULL array");
  float* base = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    if (ctx->device >= 0 && ctx->device < kMaxDevices) base = (float*)g_ptr[ctx->device];
  }
  if (!base) return set_err(ctx, PBG_ERR_STATE, "static scratch of device %d is not set up", ctx->device);
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess || cur != ctx->device)
    return set_err(ctx, PBG_ERR_STATE, "the context's device %d must be current (current: %d)", ctx->device, cur);
  uint32_t* flag_dev = (uint32_t*)base;
  float* relT = ctx->op == OP_LINEAR ? base + kFlagFloats : nullptr;

  hipStream_t cs = ctx->cs;
  // the flag keeps the last call's value: cleared by a kernel, not a memset
  launch_fill_u32(flag_dev, 1, 0u, cs);
  launch_check_ids(src_local, n, (int32_t)pbg_partition_rows(ctx, i), flag_dev, 1u, cs);
  launch_check_ids(dst_local, n, (int32_t)pbg_partition_rows(ctx, j), flag_dev, 2u, cs);
  if (rel) launch_check_ids(rel, n, ctx->R, flag_dev, 4u, cs);
  uint32_t flag = 0;
  hipError_t e = hipMemcpyAsync(&flag, flag_dev, 4, hipMemcpyDeviceToHost, cs);
  if (e == hipSuccess) e = hipStreamSynchronize(cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "id range check");
  if (flag) return set_err(ctx, PBG_ERR_INVALID_ARG, "an id is out of range (flags %u)", flag);
  StepGeom g;
  memset(&g, 0, sizeof(g));
  g.d = ctx->d;
  g.dp = (ctx->d + 3) / 4 * 4;
  g.dr = ctx->dr;
  g.op = ctx->op;
  g.cmp = ctx->cmp;
  if (relT) launch_transpose_rel(ctx->relp, relT, ctx->R, ctx->d, cs);
  launch_score_edges(g, pi.emb, pj.emb, ctx->relp, relT, src_local, rel, dst_local, n, scores, cs);
  e = hipGetLastError();
  if (e == hipSuccess) e = hipStreamSynchronize(cs);
  if (e != hipSuccess) return hip_fail(ctx, e, "score_edges_noalloc");
  return PBG_OK;
}
