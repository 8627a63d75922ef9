/* A C99 client of libwb's host calls (no GPU needed): describes the tiny dense
 * model's FSDP2 fp32 trainer layout and TP2 bf16 rollout layout, plans rollout
 * rank 1, and prints the rank's receive-buffer bytes, its work counts and the
 * canonical plan dump. Built with a C compiler and run by tests/test_abi_cpu.py,
 * which compares the output with the Python binding's. */
#include <stdio.h>
#include <stdlib.h>

#include "wb.h"

static void check(int rc, const char* what) {
  if (rc != WB_OK) {
    fprintf(stderr, "%s: status %d: %s\n", what, rc, wb_last_error());
    exit(1);
  }
}

int main(void) {
  const wb_model_shapes model = {WB_FAMILY_DENSE, 2, 256, 4, 4, 64, 1024, 1024, 0, 0};
  const wb_parallelism trainer = {WB_STYLE_FSDP_FLAT, WB_F32, 1, 1, 2, 1, 0, WB_DTYPE_NONE, 0};
  const wb_parallelism rollout = {WB_STYLE_SERVING, WB_BF16, 2, 1, 1, 1, 0, WB_DTYPE_NONE, 0};
  wb_layout_t* lt = NULL;
  wb_layout_t* lr = NULL;
  wb_plan_t* plan = NULL;
  int64_t bytes = 0, tasks = 0, blocks = 0, pieces = 0;
  size_t need = 0;
  char* text;

  check(wb_describe_layout(&model, &trainer, &lt), "trainer layout");
  check(wb_describe_layout(&model, &rollout, &lr), "rollout layout");
  check(wb_plan(lt, lr, WB_RECEIVER, 1, &plan), "plan");
  check(wb_plan_buffer_bytes(plan, &bytes), "buffer bytes");
  check(wb_plan_work_counts(plan, &tasks, &blocks, &pieces), "work counts");
  if (wb_plan_dump(plan, NULL, 0, &need) != WB_ESIZE || need == 0) {
    fprintf(stderr, "dump size query failed\n");
    return 1;
  }
  text = malloc(need);
  if (!text) return 1;
  check(wb_plan_dump(plan, text, need, &need), "dump");
  printf("%s\n%lld %lld %lld %lld\n%s", wb_version(), (long long)bytes, (long long)tasks, (long long)blocks,
         (long long)pieces, text);
  free(text);
  wb_plan_destroy(plan);
  wb_layout_destroy(lr);
  wb_layout_destroy(lt);
  return 0;
}
