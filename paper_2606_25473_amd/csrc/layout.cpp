// layout.cpp -- host side of the mask: chunk-layout validation, the query-group
// table, pair counts and the work-group tile order.  Plain C++17, no HIP.
#include "layout.hpp"

#include <algorithm>
#include <cstdio>
#include <string>
#include <vector>

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

bool transpose_groups(const GroupTable& gt, int L, GroupTable* kt, std::string* err) {
  // key breakpoints: every range end point; between two of them the admitting groups are fixed
  std::vector<int> cuts = {0, L};
  for (int g = 0; g < gt.n; ++g) {
    if (gt.a1[g] > gt.a0[g]) { cuts.push_back(gt.a0[g]); cuts.push_back(gt.a1[g]); }
    if (gt.b1[g] > gt.b0[g]) { cuts.push_back(gt.b0[g]); cuts.push_back(gt.b1[g]); }
  }
  std::sort(cuts.begin(), cuts.end());
  cuts.erase(std::unique(cuts.begin(), cuts.end()), cuts.end());
  kt->n = 0;
  for (size_t c = 0; c + 1 < cuts.size(); ++c) {
    const int k = cuts[c];  // representative key of [cuts[c], cuts[c+1])
    int runs[2][2] = {{0, 0}, {0, 0}};
    int nr = 0;
    for (int g = 0; g < gt.n; ++g) {
      const bool hit = (k >= gt.a0[g] && k < gt.a1[g]) || (k >= gt.b0[g] && k < gt.b1[g]);
      if (!hit) continue;
      const int q0 = group_q_begin(gt, g), q1 = gt.q_end[g];
      if (nr > 0 && runs[nr - 1][1] == q0) {
        runs[nr - 1][1] = q1;  // adjacent query groups form one run
        continue;
      }
      if (nr == 2)
        return fail(err, "the transposed mask needs more than two query ranges for key " + std::to_string(k));
      runs[nr][0] = q0; runs[nr][1] = q1;
      ++nr;
    }
    const int e = cuts[c + 1];
    const int n = kt->n;
    if (n > 0 && kt->a0[n - 1] == runs[0][0] && kt->a1[n - 1] == runs[0][1] && kt->b0[n - 1] == runs[1][0] &&
        kt->b1[n - 1] == runs[1][1]) {
      kt->q_end[n - 1] = e;  // same query ranges as the previous key interval: extend it
      continue;
    }
    if (n == kMaxGroups)
      return fail(err, "the transposed mask needs more than " + std::to_string(kMaxGroups) + " key groups");
    add_group(kt, e, runs[0][0], runs[0][1], runs[1][0], runs[1][1]);
  }
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
