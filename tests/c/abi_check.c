/* Plain-C use of the library's ABI (host-only calls): the header must compile as C,
 * and the query-group, key-group, pair-count and tile calls must agree with values
 * derived here by hand for a teacher-forcing layout of 3 chunks of 4 tokens. */
#include <stdio.h>

#include "attn_jvp.h"

int main(void) {
  const int32_t offs[4] = {0, 4, 8, 12};
  attn_chunk_layout lay = {ATTN_MASK_TEACHER_FORCING, 3, offs, NULL};
  const int L = 24;
  int fails = 0;
  /* pairs: C^2 N (N + 1) = 16 * 3 * 4 */
  if (attn_count_unmasked_pairs(&lay, L) != 192) { printf("pairs\n"); ++fails; }
  int32_t g[6 * 8];
  if (attn_query_groups(&lay, L, g, 8) != 6) { printf("groups\n"); ++fails; }
  /* noisy chunk 1 (rows 16..20) sees clean chunk 0 and its own noisy chunk */
  if (g[6 * 4 + 0] != 16 || g[6 * 4 + 1] != 20 || g[6 * 4 + 2] != 0 || g[6 * 4 + 3] != 4 ||
      g[6 * 4 + 4] != 16 || g[6 * 4 + 5] != 20) { printf("group 4\n"); ++fails; }
  if (attn_key_groups(&lay, L, g, 8) != 6) { printf("key groups\n"); ++fails; }
  /* clean chunk 0 keys are seen by clean rows 0..11 and noisy rows 16..23 */
  if (g[0] != 0 || g[1] != 4 || g[2] != 0 || g[3] != 12 || g[4] != 16 || g[5] != 24) {
    printf("key group 0\n"); ++fails;
  }
  int rows = 0, keys = 0;
  attn_tile_shape(&rows, &keys);
  if (rows <= 0 || keys <= 0) { printf("tile shape\n"); ++fails; }
  /* an invalid layout is reported, with a message */
  const int32_t bad[3] = {0, 5, 3};
  attn_chunk_layout badlay = {ATTN_MASK_TEACHER_FORCING, 2, bad, NULL};
  if (attn_count_unmasked_pairs(&badlay, 10) != -1 || attn_last_error()[0] == '\0') {
    printf("bad layout\n"); ++fails;
  }
  printf(fails ? "FAIL\n" : "OK\n");
  return fails;
}
