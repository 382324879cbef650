// Entry points completed in later steps of the build-up (bucketing, epoch, ranking).
#include "runtime_internal.h"

extern "C" pbg_status pbg_train_epoch(pbg_ctx* ctx, const int64_t*, const int32_t*, const int32_t*,
                                      const int32_t*, const pbg_neg_config*, float, uint64_t, int32_t,
                                      double*) {
  if (!ctx) return PBG_ERR_INVALID_ARG;
  return set_err(ctx, PBG_ERR_UNSUPPORTED, "pbg_train_epoch is not built yet");
}
