/* Host-only use of libepic_link from C: plan a small LegoLink-2 request and print
 * the selected positions and the private blocks (checked by tests/test_c_abi.py). */
#include <stdio.h>
#include <stdlib.h>

#include "epic_link.h"

int main(void) {
  const int32_t lens[3] = {20, 18, 5};
  const int32_t off[4] = {0, 2, 4, 5};
  const int32_t blocks[5] = {0, 1, 2, 3, 4};
  epic_link_request req = {3, lens, off, blocks, 3, 2, 0};
  epic_attn_cfg cfg = {8, 2, 64, 16, 0.0f, 0, 0, 0.0f};
  int32_t free_blocks[8] = {5, 6, 7, 8, 9, 10, 11, 12};
  epic_plan_sizes sizes;
  if (epic_plan_sizes_get(&req, 1, &cfg, 8, &sizes) != EPIC_OK) {
    fprintf(stderr, "sizes: %s\n", epic_last_error());
    return 1;
  }
  int32_t* buf = calloc((size_t)sizes.total_ints, sizeof(int32_t));
  epic_plan plan;
  if (!buf || epic_plan_layout(&sizes, buf, &plan) != EPIC_OK ||
      epic_plan_link(&req, 1, &cfg, free_blocks, 8, 13, &sizes, &plan) != EPIC_OK) {
    fprintf(stderr, "plan: %s\n", epic_last_error());
    return 1;
  }
  printf("n_s %d n_private %d\n", sizes.n_s, sizes.n_private);
  for (int i = 0; i < sizes.n_s; ++i) printf("%d%c", plan.s_pos[i], i + 1 < sizes.n_s ? ' ' : '\n');
  for (int i = 0; i < sizes.n_private; ++i)
    printf("%d:%d%c", plan.priv_block[i], plan.priv_src[i], i + 1 < sizes.n_private ? ' ' : '\n');
  /* an invalid request is refused with a status, not a crash */
  epic_link_request bad = req;
  bad.suffix_len = -1;
  const epic_status st = epic_plan_sizes_get(&bad, 1, &cfg, 8, &sizes);
  printf("bad %d %s\n", (int)st, epic_status_string(st));
  free(buf);
  return 0;
}
