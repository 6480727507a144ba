/* The C ABI from a C11 program: ppas.h compiles as C under strict warnings, the
 * library links, and its host-only entry points behave as declared (no GPU needed:
 * validation, status strings, planning, workspace sizing, tuning hooks). */
#include <stdio.h>
#include <string.h>

#include "ppas.h"

#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) {                                                    \
      printf("FAIL %s:%d %s\n", __FILE__, __LINE__, #c);           \
      return 1;                                                    \
    }                                                              \
  } while (0)

int main(void) {
  ppas_shape sh = {16, 2, 128, 16, 100, 0.08838834764831845f};
  ppas_seq seqs[2] = {{0, 1, 30}, {1, 20, 5}};
  int32_t bt[2][3] = {{0, 1, -1}, {2, 3, -1}};
  ppas_seq bad[1] = {{0, 0, 1}};
  int32_t items[64][8];
  int32_t n, i, decode = 0;
  ppas_plan_opts opts = {64, 64, 0, 0};
  ppas_plan_opts bad_opts = {0, 0, 0, 0};
  ppas_step_plan* plan = NULL;

  CHECK(ppas_validate_step(&sh, seqs, 2, &bt[0][0], 3) == PPAS_OK);
  CHECK(ppas_validate_step(&sh, bad, 1, NULL, 3) == PPAS_EINVAL);
  CHECK(ppas_validate_step(&sh, seqs, 0, NULL, 1) == PPAS_OK);
  CHECK(strncmp(ppas_status_string(PPAS_ERANGE), "PPAS_ERANGE", 11) == 0);

  n = ppas_plan_items(&sh, seqs, 2, NULL, NULL, 0);
  CHECK(n > 0 && n <= 64);
  CHECK(ppas_plan_items(&sh, seqs, 2, NULL, &items[0][0], n) == n);
  CHECK(ppas_plan_items(&sh, seqs, 2, &opts, NULL, 0) >= n);   /* 64-key splits: at least as many items */
  for (i = 0; i < n; ++i) decode += items[i][0] == 1;
  CHECK(decode >= 1);
  CHECK(ppas_attn_workspace_bytes(&sh, seqs, 2) >= 256);
  CHECK(ppas_attn_workspace_bytes(&sh, bad, 1) == 0);

  bad_opts.tile_positions = 24;
  CHECK(ppas_plan_items(&sh, seqs, 2, &bad_opts, NULL, 0) == PPAS_EINVAL);
  bad_opts.tile_positions = 0;
  bad_opts.prefill_split = -1;
  CHECK(ppas_plan_items(&sh, seqs, 2, &bad_opts, NULL, 0) == PPAS_EINVAL);
  /* planned calls refuse a NULL plan, and half-set event pairs, before any device work */
  CHECK(ppas_attn_step_planned(NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0, NULL, NULL) == PPAS_EINVAL);
  CHECK(ppas_kv_append_planned(NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL) == PPAS_EINVAL);
  CHECK(ppas_step_plan_create(&sh, bad, 1, NULL, 3, NULL, &plan) == PPAS_EINVAL && plan == NULL);
  CHECK(ppas_step_plan_info(NULL, NULL) == PPAS_EINVAL);
  ppas_step_plan_destroy(NULL);
  /* a device call with a bad step is refused before any device work */
  CHECK(ppas_attn_step(&sh, NULL, NULL, NULL, NULL, bad, 1, NULL, 3, NULL, NULL, 0, NULL) == PPAS_EINVAL);
  printf("ok\n");
  return 0;
}
