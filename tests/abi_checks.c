/*
 * Error paths of the C ABI (include/pbg.h), driven from C so that the host
 * runtime can run under AddressSanitizer: NULL contexts, argument errors at
 * initialisation, a context whose initialisation failed, and the row and size
 * queries.  None of these may touch a device, so the program runs on a host
 * without a GPU.  Exit status 0 and "abi checks passed" on success.
 */
#include <stdio.h>
#include <string.h>

#include "pbg.h"

static int failures = 0;

#define CHECK(cond)                                                   \
  do {                                                                \
    if (!(cond)) {                                                    \
      fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                     \
    }                                                                 \
  } while (0)

/* every entry point that takes a context, with empty arguments; each must
 * return `want` on ctx */
static void every_call(pbg_ctx* ctx, pbg_status want) {
  pbg_neg_config neg;
  memset(&neg, 0, sizeof(neg));
  neg.chunk_size = 1;
  neg.num_uniform = 1;
  neg.chunks_per_step = 1;
  double d = 0.0;
  int64_t n = 0;
  pbg_stats st;
  CHECK(pbg_bucket_edges(ctx, NULL, NULL, NULL, 0, NULL, NULL, NULL, NULL) == want);
  CHECK(pbg_bind_partition(ctx, 0, NULL, NULL, 0) == want);
  CHECK(pbg_bind_relations(ctx, NULL, NULL) == want);
  CHECK(pbg_set_streams(ctx, NULL, NULL) == want);
  CHECK(pbg_train_bucket(ctx, 0, 0, NULL, NULL, NULL, 0, &neg, 0.1f, 1, &d) == want);
  CHECK(pbg_set_entity_types(ctx, 1, NULL, NULL, NULL, NULL) == want);
  CHECK(pbg_bind_type_partition(ctx, 0, 0, NULL, NULL, 0) == want);
  CHECK(pbg_set_relation_weights(ctx, NULL) == want);
  CHECK(pbg_group_by_relation(ctx, NULL, NULL, NULL, 0, NULL, NULL, NULL) == want);
  CHECK(pbg_get_step_losses(ctx, NULL, 0, &n) == want);
  CHECK(pbg_train_epoch(ctx, NULL, NULL, NULL, NULL, &neg, 0.1f, 1, 1, &d) == want);
  CHECK(pbg_score_edges(ctx, 0, 0, NULL, NULL, NULL, 0, NULL) == want);
  CHECK(pbg_score_edges_noalloc(ctx, 0, 0, NULL, NULL, NULL, 0, NULL) == want);
  CHECK(pbg_rank_eval(ctx, NULL, NULL, NULL, 0, NULL, NULL, NULL, 0, NULL, &d, &d) == want);
  CHECK(pbg_rank_sampled(ctx, NULL, NULL, NULL, 0, NULL, 0, NULL, &d, &d) == want);
  CHECK(pbg_sample_negatives(ctx, 0, 0, 0, 0, 1, 1, NULL) == want);
  CHECK(pbg_inspect_step(ctx, 0, 0, NULL, NULL, NULL, 0, &neg, 1, NULL, NULL, NULL, NULL, &d) == want);
  CHECK(pbg_get_stats(ctx, &st) == want);
  CHECK(pbg_partition_rows(ctx, 0) == -1);
  CHECK(pbg_type_partition_rows(ctx, 0, 0) == -1);
  CHECK(pbg_relation_param_floats(ctx) == -1);
  CHECK(pbg_last_error(ctx) != NULL);
}

/* initialisation that must fail with `want`; the context it may leave
 * behind carries a message and rejects every other call */
static void failed_init(int64_t n, int32_t P, int32_t R, int32_t dim, int32_t op, int32_t cmp, int32_t loss,
                        float margin, uint32_t flags, pbg_status want) {
  pbg_ctx* ctx = (pbg_ctx*)1;
  CHECK(pbg_bucket_init(&ctx, n, P, R, dim, op, cmp, loss, margin, flags) == want);
  if (ctx) {
    CHECK(strlen(pbg_last_error(ctx)) > 0);
    every_call(ctx, PBG_ERR_STATE);
    pbg_free(ctx);
  }
}

int main(void) {
  every_call(NULL, PBG_ERR_INVALID_ARG);
  pbg_free(NULL);
  CHECK(pbg_bucket_init(NULL, 10, 1, 1, 8, PBG_OP_TRANSLATION, PBG_CMP_COS, PBG_LOSS_RANKING, 0.1f, 0) ==
        PBG_ERR_INVALID_ARG);
  const float inf = 1.0f / 0.0f;
  failed_init(0, 1, 1, 8, PBG_OP_TRANSLATION, PBG_CMP_COS, PBG_LOSS_RANKING, 0.1f, 0, PBG_ERR_INVALID_ARG);
  failed_init(10, 0, 1, 8, PBG_OP_TRANSLATION, PBG_CMP_COS, PBG_LOSS_RANKING, 0.1f, 0, PBG_ERR_INVALID_ARG);
  failed_init(10, 1, 0, 8, PBG_OP_TRANSLATION, PBG_CMP_COS, PBG_LOSS_RANKING, 0.1f, 0, PBG_ERR_INVALID_ARG);
  failed_init(10, 1, 1, 0, PBG_OP_TRANSLATION, PBG_CMP_COS, PBG_LOSS_RANKING, 0.1f, 0, PBG_ERR_INVALID_ARG);
  failed_init(10, 1, 1, 513, PBG_OP_TRANSLATION, PBG_CMP_COS, PBG_LOSS_RANKING, 0.1f, 0, PBG_ERR_INVALID_ARG);
  failed_init(10, 1, 1, 7, PBG_OP_COMPLEX_DIAGONAL, PBG_CMP_DOT, PBG_LOSS_RANKING, 0.1f, 0, PBG_ERR_INVALID_ARG);
  failed_init(10, 1, 1, 8, 99, PBG_CMP_DOT, PBG_LOSS_RANKING, 0.1f, 0, PBG_ERR_INVALID_ARG);
  failed_init(10, 1, 1, 8, -1, PBG_CMP_DOT, PBG_LOSS_RANKING, 0.1f, 0, PBG_ERR_INVALID_ARG);
  failed_init(10, 1, 1, 8, PBG_OP_DIAGONAL, 7, PBG_LOSS_RANKING, 0.1f, 0, PBG_ERR_INVALID_ARG);
  failed_init(10, 1, 1, 8, PBG_OP_DIAGONAL, PBG_CMP_DOT, 9, 0.1f, 0, PBG_ERR_INVALID_ARG);
  failed_init(10, 1, 1, 8, PBG_OP_DIAGONAL, PBG_CMP_DOT, PBG_LOSS_RANKING, inf, 0, PBG_ERR_INVALID_ARG);
  failed_init(10, 1, 1, 8, PBG_OP_DIAGONAL, PBG_CMP_DOT, PBG_LOSS_RANKING, 0.1f, 1u << 20, PBG_ERR_INVALID_ARG);
  failed_init(9, 4, 1, 8, PBG_OP_DIAGONAL, PBG_CMP_DOT, PBG_LOSS_RANKING, 0.1f, 0, PBG_ERR_INVALID_ARG);
  failed_init(10, 1, 3, 8, PBG_OP_LINEAR, PBG_CMP_COS, PBG_LOSS_RANKING, 0.1f, 0, PBG_ERR_UNSUPPORTED);
  if (failures) {
    fprintf(stderr, "%d abi checks failed\n", failures);
    return 1;
  }
  printf("abi checks passed\n");
  return 0;
}
