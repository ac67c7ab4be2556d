// layout.cpp -- host side of the mask: chunk-layout validation, the query-group
// table, pair counts and the work-group tile order.  Plain C++17, no HIP.
#include "layout.hpp"

#include <algorithm>
#include <cstdio>
#include <string>
#include <utility>
#include <vector>

namespace attn {

namespace {
bool fail(std::string* err, const std::string& msg) {
  if (err) *err = msg;
  return false;
}

// Open group n of the table: it owns rows up to q_end and has no key range yet.
void begin_group(GroupTable* gt, int q_end) {
  const int g = gt->n++;
  gt->q_end[g] = q_end;
  gt->r_begin[g + 1] = gt->r_begin[g];
}

// Append key range [k0, k1) (non-empty, after the group's last range and not touching
// it) to the last group.
bool add_range(GroupTable* gt, int k0, int k1, std::string* err) {
  const int r = gt->r_begin[gt->n];
  if (r == kMaxRanges)
    return fail(err, "more than " + std::to_string(kMaxRanges) + " key ranges in all (ATTN_MAX_RANGES)");
  gt->k[2 * r] = k0;
  gt->k[2 * r + 1] = k1;
  gt->r_begin[gt->n] = (uint16_t)(r + 1);
  return true;
}

std::string at_group(int g) { return " (group " + std::to_string(g) + ")"; }

// ATTN_MASK_RANGES: query-group bounds, per-group range offsets and key ranges.
bool build_range_list(const attn_chunk_layout* layout, int L, GroupTable* gt, std::string* err) {
  const int G = layout->num_chunks;
  if (G < 1 || G > ATTN_MAX_GROUPS)
    return fail(err, "number of query groups must be in [1, " + std::to_string(ATTN_MAX_GROUPS) + "], got " +
                         std::to_string(G));
  const int32_t* qb = layout->chunk_offsets;
  const int32_t* ro = layout->range_offsets;
  if (!qb) return fail(err, "chunk_offsets (the query-group bounds) is NULL");
  if (!ro) return fail(err, "range_offsets is NULL");
  if (qb[0] != 0) return fail(err, "the first query group must start at row 0");
  if (ro[0] != 0) return fail(err, "range_offsets[0] must be 0");
  for (int g = 0; g < G; ++g) {
    if (qb[g + 1] <= qb[g]) return fail(err, "query-group bounds must be strictly increasing" + at_group(g));
    if (ro[g + 1] < ro[g]) return fail(err, "range_offsets must not decrease" + at_group(g));
  }
  if (qb[G] != L)
    return fail(err, "query groups cover " + std::to_string(qb[G]) + " rows but L = " + std::to_string(L));
  const int32_t* rk = layout->ranges;
  if (ro[G] > 0 && !rk) return fail(err, "ranges is NULL");
  std::vector<std::pair<int, int>> K;
  for (int g = 0; g < G; ++g) {
    K.clear();
    for (int64_t r = ro[g]; r < ro[g + 1]; ++r) {
      const int k0 = rk[2 * r], k1 = rk[2 * r + 1];
      if (k0 < 0 || k0 > k1 || k1 > L)
        return fail(err, "key ranges must satisfy 0 <= begin <= end <= L" + at_group(g));
      if (k1 > k0) K.emplace_back(k0, k1);
    }
    std::sort(K.begin(), K.end());
    begin_group(gt, qb[g + 1]);
    for (size_t i = 0; i < K.size(); ++i) {
      if (i > 0 && K[i].first < K[i - 1].second) return fail(err, "key ranges overlap" + at_group(g));
      const int r = gt->r_begin[gt->n];
      if (i > 0 && K[i].first == K[i - 1].second) {
        gt->k[2 * r - 1] = K[i].second;  // touches the previous range: extend it
        continue;
      }
      if (!add_range(gt, K[i].first, K[i].second, err)) return false;
    }
  }
  return true;
}
}  // namespace

bool build_groups(const attn_chunk_layout* layout, int L, GroupTable* gt, std::string* err) {
  if (!layout) return fail(err, "layout is NULL");
  if (L <= 0) return fail(err, "sequence length L must be positive, got " + std::to_string(L));
  gt->n = 0;
  gt->r_begin[0] = 0;
  const int kind = layout->kind;
  if (kind == ATTN_MASK_FULL) {
    begin_group(gt, L);
    return add_range(gt, 0, L, err);
  }
  if (kind == ATTN_MASK_RANGES) return build_range_list(layout, L, gt, err);
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
    for (int j = 0; j < N; ++j) {
      begin_group(gt, o[j + 1]);
      add_range(gt, 0, o[j + 1], err);
    }
    return true;
  }
  if ((int64_t)L != 2 * (int64_t)half)
    return fail(err, "teacher-forcing layout needs L = 2 * chunk_offsets[N] = " +
                         std::to_string(2 * (int64_t)half) + ", got L = " + std::to_string(L));
  // clean chunk j: clean chunks <= j (N ranges)
  for (int j = 0; j < N; ++j) {
    begin_group(gt, o[j + 1]);
    add_range(gt, 0, o[j + 1], err);
  }
  // noisy chunk i: clean chunks < i, then its own noisy chunk (2N - 1 ranges; 3N - 1 <=
  // kMaxRanges for N <= ATTN_MAX_CHUNKS)
  for (int i = 0; i < N; ++i) {
    begin_group(gt, half + o[i + 1]);
    if (i > 0) add_range(gt, 0, o[i], err);
    add_range(gt, half + o[i], half + o[i + 1], err);
  }
  return true;
}

int64_t count_pairs(const GroupTable& gt) {
  int64_t total = 0;
  for (int g = 0; g < gt.n; ++g) {
    const int64_t rows = gt.q_end[g] - group_q_begin(gt, g);
    int64_t keys = 0;
    for (int r = gt.r_begin[g]; r < gt.r_begin[g + 1]; ++r) keys += gt.k[2 * r + 1] - gt.k[2 * r];
    total += rows * keys;
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
  TileOrder o{};
  o.nt = (L + br - 1) / br;
  o.split = o.nt;
  o.first = -1;
  o.mode = 0;
  if (layout->kind == ATTN_MASK_BLOCK_CAUSAL) o.mode = 1;
  if (layout->kind == ATTN_MASK_TEACHER_FORCING) {
    o.mode = 2;
    const int half = L / 2;
    o.split = (half + br - 1) / br;  // the tile holding the clean/noisy boundary counts as clean
  }
  return o;
}

TileOrder make_tile_order_zero_clean(const GroupTable& gt, int L, int br, int bc, int t0) {
  TileOrder o{};
  o.nt = (L + br - 1) / br;
  o.split = t0 / br;  // tiles wholly below t0 need the primal only; the boundary tile is upper
  o.first = -1;
  o.mode = 2;
  const bool straddle = t0 % br != 0;
  if (o.nt - (straddle ? 1 : 0) > kMaxMergeTiles) return o;  // merge bits for at most this many
  // Cost of a tile in key-block contractions: 2 per block (scores, output) for a tile
  // without tangent rows, 4 per block of keys without tangents (+ the dQ term of the
  // score tangent and the H~ term of the output tangent), 6 per block with tangent keys.
  auto cost = [&](int t) {
    const int q0 = t * br, q1 = q0 + br < L ? q0 + br : L;
    const TilePlan p = plan_tile(gt, q0, q1, bc);
    const int nb = plan_num_blocks(p);
    int64_t c = 0;
    for (int i = 0; i < nb; ++i) {
      const int k0 = plan_block(p, i) * bc;
      c += q1 <= t0 ? 2 : (k0 + bc > t0 ? 6 : 4);
    }
    return c;
  };
  o.mode = 3;
  // A tile straddling t0 holds the last clean chunk, which sees every clean key with
  // the dQ term: one of the heaviest tiles, and out of place at the low end of the
  // upper half.  It goes first.
  int lo = o.split - 1, hi = o.nt - 1, stop = o.split;
  if (straddle) {
    o.first = o.split;
    stop = o.split + 1;
  }
  int64_t clo = lo >= 0 ? cost(lo) : 0, chi = hi >= stop ? cost(hi) : 0;
  for (int t = 0; t < o.nt - (o.first >= 0 ? 1 : 0); ++t) {
    const bool take_hi = lo < 0 || (hi >= stop && chi >= clo);
    if (take_hi) {
      o.merge[t >> 5] |= 1u << (t & 31);
      --hi;
      chi = hi >= stop ? cost(hi) : 0;
    } else {
      --lo;
      clo = lo >= 0 ? cost(lo) : 0;
    }
  }
  return o;
}

}  // namespace attn
