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

  CHECK(ppas_validate_step(&sh, seqs, 2, &bt[0][0], 3) == PPAS_OK);
  CHECK(ppas_validate_step(&sh, bad, 1, NULL, 3) == PPAS_EINVAL);
  CHECK(ppas_validate_step(&sh, seqs, 0, NULL, 1) == PPAS_OK);
  CHECK(strncmp(ppas_status_string(PPAS_ERANGE), "PPAS_ERANGE", 11) == 0);

  n = ppas_plan_items(&sh, seqs, 2, 256, NULL, 0);
  CHECK(n > 0 && n <= 64);
  CHECK(ppas_plan_items(&sh, seqs, 2, 256, &items[0][0], n) == n);
  for (i = 0; i < n; ++i) decode += items[i][0] == 1;
  CHECK(decode >= 1);
  CHECK(ppas_attn_workspace_bytes(&sh, seqs, 2) >= 256);
  CHECK(ppas_attn_workspace_bytes(&sh, bad, 1) == 0);

  CHECK(ppas_set_tile_positions(24) == PPAS_EINVAL);
  CHECK(ppas_set_split_keys(-1, 0) == PPAS_EINVAL);
  CHECK(ppas_set_profile_events(&sh, NULL) == PPAS_EINVAL);
  CHECK(ppas_set_profile_events(NULL, NULL) == PPAS_OK);
  /* a device call with a bad step is refused before any device work */
  CHECK(ppas_attn_step(&sh, NULL, NULL, NULL, NULL, bad, 1, NULL, 3, NULL, NULL, 0, NULL) == PPAS_EINVAL);
  printf("ok\n");
  return 0;
}
