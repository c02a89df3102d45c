/* A plain C99 consumer of the library's public header: it must compile with
 * a C compiler (no HIP or C++ types), link against the shared library, and
 * report the layout of every public struct so the Python binding can be
 * checked against it.  It makes only calls that fail argument validation
 * before touching a device, so it runs without a GPU. */
#include <stddef.h>
#include <stdio.h>

#include "esopt.h"

int main(void) {
    printf("es_tensor_t %zu data %zu numel %zu tensor_id %zu offset8 %zu\n", sizeof(es_tensor_t),
           offsetof(es_tensor_t, data), offsetof(es_tensor_t, numel),
           offsetof(es_tensor_t, tensor_id), offsetof(es_tensor_t, offset8));
    printf("es_qtensor_t %zu data %zu scales %zu numel %zu row %zu tensor_id %zu\n",
           sizeof(es_qtensor_t), offsetof(es_qtensor_t, data), offsetof(es_qtensor_t, scales),
           offsetof(es_qtensor_t, numel), offsetof(es_qtensor_t, row),
           offsetof(es_qtensor_t, tensor_id));
    printf("es_block_t %zu data %zu rows %zu cols %zu row_len %zu row0 %zu col0 %zu "
           "tensor_id %zu reserved %zu\n",
           sizeof(es_block_t), offsetof(es_block_t, data), offsetof(es_block_t, rows),
           offsetof(es_block_t, cols), offsetof(es_block_t, row_len), offsetof(es_block_t, row0),
           offsetof(es_block_t, col0), offsetof(es_block_t, tensor_id),
           offsetof(es_block_t, reserved));
    printf("es_update_opts_t %zu alpha %zu sigma %zu zscore_eps %zu flags %zu round_seed %zu\n",
           sizeof(es_update_opts_t), offsetof(es_update_opts_t, alpha),
           offsetof(es_update_opts_t, sigma), offsetof(es_update_opts_t, zscore_eps),
           offsetof(es_update_opts_t, flags), offsetof(es_update_opts_t, round_seed));
    printf("flags %u %u %u %u max_members %u\n", ES_UPDATE_DIV_SIGMA, ES_REWARDS_ARE_WEIGHTS,
           ES_UPDATE_STOCHASTIC_ROUND, ES_UPDATE_MASTER, ES_MAX_MEMBERS);
    printf("es_qblock_t %zu data %zu scales %zu rows %zu cols %zu row_len %zu row0 %zu "
           "col0 %zu row %zu tensor_id %zu\n",
           sizeof(es_qblock_t), offsetof(es_qblock_t, data), offsetof(es_qblock_t, scales),
           offsetof(es_qblock_t, rows), offsetof(es_qblock_t, cols),
           offsetof(es_qblock_t, row_len), offsetof(es_qblock_t, row0),
           offsetof(es_qblock_t, col0), offsetof(es_qblock_t, row),
           offsetof(es_qblock_t, tensor_id));
    es_plan_t* plan = NULL;
    printf("plan_create_null %d\n", es_plan_create(NULL, 1, &plan));
    printf("plan_create_blocks_null %d\n", es_plan_create_blocks(NULL, 1, &plan));
    printf("perturb_null %d\n", es_perturb(NULL, 1, 1, 1e-3f, NULL));
    printf("set_master_null %d\n", es_plan_set_master(NULL, NULL, 0));
    es_qplan_t* qplan = NULL;
    printf("qplan_create_null %d\n", es_qplan_create(NULL, 1, &qplan));
    printf("qplan_create_shards_null %d\n",
           es_qplan_create_shards(NULL, NULL, 1, ES_QFORMAT_E4M3, &qplan));
    printf("qplan_create_blocks_null %d\n",
           es_qplan_create_blocks(NULL, 1, ES_QFORMAT_INT8, &qplan));
    printf("strerror %s\n", es_strerror(ES_ERR_INVALID_ARG));
    printf("sigma_cosine %.17g\n", es_sigma_cosine(1e-3, 1e-4, 50, 100));
    return 0;
}
