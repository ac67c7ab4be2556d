/* Plain-C use of the library's ABI (host-only calls): the header must compile as C,
 * and the query-group, pair-count and tile-plan calls must agree with values
 * derived here by hand for a teacher-forcing layout of 3 chunks of 4 tokens and for a
 * range list with three key ranges in one group. */
#include <stdio.h>

#include "attn_jvp.h"

int main(void) {
  const int32_t offs[4] = {0, 4, 8, 12};
  attn_chunk_layout lay = {ATTN_MASK_TEACHER_FORCING, 3, offs, NULL, NULL};
  const int L = 24;
  int fails = 0;
  /* pairs: C^2 N (N + 1) = 16 * 3 * 4 */
  if (attn_count_unmasked_pairs(&lay, L) != 192) { printf("pairs\n"); ++fails; }
  int32_t b[9], ro[9], r[2 * 16];
  if (attn_query_groups(&lay, L, b, ro, r, 8, 16) != 6) { printf("groups\n"); ++fails; }
  /* noisy chunk 1 (group 4, rows 16..20) sees clean chunk 0 and its own noisy chunk */
  if (b[4] != 16 || b[5] != 20 || ro[5] - ro[4] != 2 || r[2 * ro[4]] != 0 || r[2 * ro[4] + 1] != 4 ||
      r[2 * ro[4] + 2] != 16 || r[2 * ro[4] + 3] != 20) { printf("group 4\n"); ++fails; }
  /* the one key tile (keys 0..23) is seen by every query: one 64-row block, partial */
  int32_t blk[4], full[4];
  if (attn_key_tile_plan(&lay, L, 0, blk, full, 4) != 1 || blk[0] != 0 || full[0] != 0) {
    printf("key tile plan\n"); ++fails;
  }
  /* range list over 10 tokens: rows 0..3 see keys {0, 4..5, 8}, given out of order with
     an empty range; rows 4..9 see keys 0..9 (two touching ranges) */
  const int32_t qb[3] = {0, 4, 10}, rofs[3] = {0, 4, 6};
  const int32_t rk[12] = {8, 9, 4, 6, 3, 3, 0, 1, 0, 5, 5, 10};
  attn_chunk_layout rl = {ATTN_MASK_RANGES, 2, qb, rofs, rk};
  if (attn_count_unmasked_pairs(&rl, 10) != 4 * 4 + 6 * 10) { printf("range pairs\n"); ++fails; }
  if (attn_query_groups(&rl, 10, b, ro, r, 8, 16) != 2 || ro[1] != 3 || ro[2] != 4 || r[0] != 0 || r[1] != 1 ||
      r[2] != 4 || r[3] != 6 || r[4] != 8 || r[5] != 9 || r[6] != 0 || r[7] != 10) {
    printf("range table\n"); ++fails;
  }
  int rows = 0, keys = 0;
  attn_tile_shape(&rows, &keys);
  if (rows <= 0 || keys <= 0) { printf("tile shape\n"); ++fails; }
  /* an invalid layout is reported, with a message */
  const int32_t bad[3] = {0, 5, 3};
  attn_chunk_layout badlay = {ATTN_MASK_TEACHER_FORCING, 2, bad, NULL, NULL};
  if (attn_count_unmasked_pairs(&badlay, 10) != -1 || attn_last_error()[0] == '\0') {
    printf("bad layout\n"); ++fails;
  }
  printf(fails ? "FAIL\n" : "OK\n");
  return fails;
}
