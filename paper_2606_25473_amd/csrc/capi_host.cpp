// capi_host.cpp -- the host-only extern "C" entry points of include/attn_jvp.h: the mask
// table, pair counts, tile plans and orders, and the error message.  Plain C++17.
#include <cstdint>
#include <string>

#include "attn_jvp.h"
#include "args.hpp"
#include "layout.hpp"
#include "validate.hpp"

namespace {

// Write a group table in the CSR form of attn_query_groups.
int write_table(const attn::GroupTable& gt, int32_t* bounds, int32_t* range_offsets, int32_t* ranges,
                int max_groups, int max_ranges) {
  const int nr = gt.r_begin[gt.n];
  if (!bounds || !range_offsets || max_groups < gt.n || max_ranges < nr || (nr > 0 && !ranges))
    return attn::set_error(ATTN_ERR_INVALID, "output buffer too small"), -1;
  bounds[0] = 0;
  range_offsets[0] = 0;
  for (int g = 0; g < gt.n; ++g) {
    bounds[g + 1] = gt.q_end[g];
    range_offsets[g + 1] = gt.r_begin[g + 1];
  }
  for (int r = 0; r < nr; ++r) {
    ranges[2 * r] = gt.k[2 * r];
    ranges[2 * r + 1] = gt.k[2 * r + 1];
  }
  return gt.n;
}

}  // namespace

extern "C" {

int attn_query_groups(const attn_chunk_layout* layout, int L, int32_t* bounds, int32_t* range_offsets,
                      int32_t* ranges, int max_groups, int max_ranges) {
  attn::GroupTable gt;
  std::string err;
  if (!attn::build_groups(layout, L, &gt, &err)) return attn::set_error(ATTN_ERR_INVALID, err), -1;
  return write_table(gt, bounds, range_offsets, ranges, max_groups, max_ranges);
}

int attn_key_tile_plan(const attn_chunk_layout* layout, int L, int ktile, int32_t* blocks, int32_t* full, int cap) {
  attn::GroupTable gt;
  std::string err;
  if (!attn::build_groups(layout, L, &gt, &err)) return attn::set_error(ATTN_ERR_INVALID, err), -1;
  const int kt = attn::kBwdKeysPerTile, qb = attn::kBwdRowsPerBlock;
  if (ktile < 0 || (int64_t)ktile * kt >= L) return attn::set_error(ATTN_ERR_INVALID, "key tile out of range"), -1;
  const int k0 = ktile * kt;
  const int k1 = k0 + kt < L ? k0 + kt : L;
  const attn::TilePlan p = attn::plan_key_tile(gt, k0, k1, qb);
  const int nb = attn::plan_num_blocks(p);
  if (!blocks || !full || cap < nb) return attn::set_error(ATTN_ERR_INVALID, "output buffer too small"), -1;
  for (int i = 0; i < nb; ++i) {
    blocks[i] = attn::plan_block(p, i);
    full[i] = attn::block_is_full(p, blocks[i] * qb, qb, L) ? 1 : 0;
  }
  return nb;
}

int64_t attn_count_unmasked_pairs(const attn_chunk_layout* layout, int L) {
  attn::GroupTable gt;
  std::string err;
  if (!attn::build_groups(layout, L, &gt, &err)) return attn::set_error(ATTN_ERR_INVALID, err), -1;
  return attn::count_pairs(gt);
}

int64_t attn_count_computed_pairs(const attn_chunk_layout* layout, int L, int D) {
  if (D != 64 && D != 128) return attn::set_error(ATTN_ERR_UNSUPPORTED, "unsupported head_dim " + std::to_string(D)), -1;
  attn::GroupTable gt;
  std::string err;
  if (!attn::build_groups(layout, L, &gt, &err)) return attn::set_error(ATTN_ERR_INVALID, err), -1;
  return attn::count_computed_pairs(gt, L, attn::kMfmaBr, attn::kMfmaBc);
}

void attn_tile_shape(int* rows_per_tile, int* keys_per_block) {
  if (rows_per_tile) *rows_per_tile = attn::kMfmaBr;
  if (keys_per_block) *keys_per_block = attn::kMfmaBc;
}

int attn_tile_plan(const attn_chunk_layout* layout, int L, int qtile, int32_t* blocks, int32_t* full, int cap) {
  attn::GroupTable gt;
  std::string err;
  if (!attn::build_groups(layout, L, &gt, &err)) return attn::set_error(ATTN_ERR_INVALID, err), -1;
  const int br = attn::kMfmaBr, bc = attn::kMfmaBc;
  if (qtile < 0 || (int64_t)qtile * br >= L) return attn::set_error(ATTN_ERR_INVALID, "query tile out of range"), -1;
  const int q0 = qtile * br;
  const int q1 = q0 + br < L ? q0 + br : L;
  const attn::TilePlan p = attn::plan_tile(gt, q0, q1, bc);
  const int nb = attn::plan_num_blocks(p);
  if (!blocks || !full || cap < nb) return attn::set_error(ATTN_ERR_INVALID, "output buffer too small"), -1;
  for (int i = 0; i < nb; ++i) {
    blocks[i] = attn::plan_block(p, i);
    full[i] = attn::block_is_full(p, blocks[i] * bc, bc, L) ? 1 : 0;
  }
  return nb;
}

int attn_tile_order(const attn_chunk_layout* layout, int L, int zero_clean, int32_t* order, int cap) {
  attn::GroupTable gt;
  std::string err;
  if (!attn::build_groups(layout, L, &gt, &err)) return attn::set_error(ATTN_ERR_INVALID, err), -1;
  if (zero_clean && layout->kind != ATTN_MASK_TEACHER_FORCING)
    return attn::set_error(ATTN_ERR_INVALID, "the zero-clean-tangent JVP needs a teacher-forcing layout"), -1;
  const attn::TileOrder o =
      zero_clean ? attn::make_tile_order_zero_clean(gt, L, attn::kMfmaBr, attn::kMfmaBc, L / 2)
                 : attn::make_tile_order(layout, L, attn::kMfmaBr);
  if (!order || cap < o.nt) return attn::set_error(ATTN_ERR_INVALID, "output buffer too small"), -1;
  for (int t = 0; t < o.nt; ++t) order[t] = attn::tile_of(o, t);
  return o.nt;
}

const char* attn_last_error(void) { return attn::last_error_message(); }

}  // extern "C"
