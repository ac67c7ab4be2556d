// layout.cpp -- host side of the mask: chunk-layout validation, the query-group
// table, pair counts and the work-group tile order.  Plain C++17, no HIP.
#include "layout.hpp"

#include <cstdio>
#include <string>

namespace attn {

namespace {
bool fail(std::string* err, const std::string& msg) {
  if (err) *err = msg;
  return false;
}
void add_group(GroupTable* gt, int q_end, int a0, int a1, int b0, int b1) {
  const int g = gt->n++;
  gt->q_end[g] = q_end;
  gt->a0[g] = a0; gt->a1[g] = a1;
  gt->b0[g] = b0; gt->b1[g] = b1;
}
}  // namespace

bool build_groups(const attn_chunk_layout* layout, int L, GroupTable* gt, std::string* err) {
  if (!layout) return fail(err, "layout is NULL");
  if (L <= 0) return fail(err, "sequence length L must be positive, got " + std::to_string(L));
  gt->n = 0;
  const int kind = layout->kind;
  if (kind == ATTN_MASK_FULL) {
    add_group(gt, L, 0, L, 0, 0);
    return true;
  }
  if (kind == ATTN_MASK_RANGES) {
    const int G = layout->num_chunks;
    if (G < 1 || G > ATTN_MAX_GROUPS)
      return fail(err, "number of query groups must be in [1, " + std::to_string(ATTN_MAX_GROUPS) +
                           "], got " + std::to_string(G));
    const int32_t* r = layout->ranges;
    if (!r) return fail(err, "ranges is NULL");
    int prev = 0;
    for (int g = 0; g < G; ++g) {
      const int qe = r[5 * g], a0 = r[5 * g + 1], a1 = r[5 * g + 2], b0 = r[5 * g + 3], b1 = r[5 * g + 4];
      const std::string at = " (group " + std::to_string(g) + ")";
      if (qe <= prev) return fail(err, "query group ends must be strictly increasing" + at);
      if (a0 < 0 || a0 > a1 || a1 > L || b0 < 0 || b0 > b1 || b1 > L)
        return fail(err, "key ranges must satisfy 0 <= begin <= end <= L" + at);
      if (a1 > a0 && b1 > b0 && a0 < b1 && b0 < a1) return fail(err, "key ranges overlap" + at);
      add_group(gt, qe, a0, a1, b0, b1);
      prev = qe;
    }
    if (prev != L)
      return fail(err, "query groups cover " + std::to_string(prev) + " rows but L = " + std::to_string(L));
    return true;
  }
  if (kind != ATTN_MASK_BLOCK_CAUSAL && kind != ATTN_MASK_TEACHER_FORCING)
    return fail(err, "unknown mask kind " + std::to_string(kind));
  const int N = layout->num_chunks;
  if (N < 1 || N > ATTN_MAX_CHUNKS)
    return fail(err, "num_chunks must be in [1, " + std::to_string(ATTN_MAX_CHUNKS) + "], got " +
                         std::to_string(N));
  const int32_t* o = layout->chunk_offsets;
  if (!o) return fail(err, "chunk_offsets is NULL");
  if (o[0] != 0) return fail(err, "chunk_offsets[0] must be 0");
  for (int i = 0; i < N; ++i)
    if (o[i + 1] <= o[i]) return fail(err, "chunk_offsets must be strictly increasing (index " +
                                               std::to_string(i + 1) + ")");
  const int half = o[N];
  if (kind == ATTN_MASK_BLOCK_CAUSAL) {
    if (L != half)
      return fail(err, "block-causal layout covers " + std::to_string(half) + " tokens but L = " +
                           std::to_string(L));
    for (int j = 0; j < N; ++j) add_group(gt, o[j + 1], 0, o[j + 1], 0, 0);
    return true;
  }
  if ((int64_t)L != 2 * (int64_t)half)
    return fail(err, "teacher-forcing layout needs L = 2 * chunk_offsets[N] = " +
                         std::to_string(2 * (int64_t)half) + ", got L = " + std::to_string(L));
  // clean chunk j: clean chunks <= j
  for (int j = 0; j < N; ++j) add_group(gt, o[j + 1], 0, o[j + 1], 0, 0);
  // noisy chunk i: clean chunks < i, then its own noisy chunk
  for (int i = 0; i < N; ++i) add_group(gt, half + o[i + 1], 0, o[i], half + o[i], half + o[i + 1]);
  return true;
}

int64_t count_pairs(const GroupTable& gt) {
  int64_t total = 0;
  for (int g = 0; g < gt.n; ++g) {
    const int64_t rows = gt.q_end[g] - group_q_begin(gt, g);
    total += rows * ((int64_t)(gt.a1[g] - gt.a0[g]) + (gt.b1[g] - gt.b0[g]));
  }
  return total;
}

int64_t count_computed_pairs(const GroupTable& gt, int L, int br, int bc) {
  int64_t total = 0;
  for (int q0 = 0; q0 < L; q0 += br) {
    const int q1 = q0 + br < L ? q0 + br : L;
    const TilePlan p = plan_tile(gt, q0, q1, bc);
    const int nb = plan_num_blocks(p);
    for (int i = 0; i < nb; ++i) {
      const int k0 = plan_block(p, i) * bc;
      const int k1 = k0 + bc < L ? k0 + bc : L;
      total += (int64_t)(q1 - q0) * (k1 - k0);
    }
  }
  return total;
}

TileOrder make_tile_order(const attn_chunk_layout* layout, int L, int br) {
  TileOrder o;
  o.nt = (L + br - 1) / br;
  o.split = o.nt;
  o.mode = 0;
  if (layout->kind == ATTN_MASK_BLOCK_CAUSAL) o.mode = 1;
  if (layout->kind == ATTN_MASK_TEACHER_FORCING) {
    o.mode = 2;
    const int half = L / 2;
    o.split = (half + br - 1) / br;  // the tile holding the clean/noisy boundary counts as clean
  }
  return o;
}

}  // namespace attn
