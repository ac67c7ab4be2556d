// Seeded fuzz of the library's host code, built with g++ -fsanitize=address,undefined
// (tests/test_host_sanitized.py): layout validation and the query-group table, pair
// counts, the query-tile and key-tile plans and their per-row / per-key mask bits (also
// for windows past the end of the sequence), the tile orders, and the argument
// validation of every compute entry point with fake, never dereferenced pointers.
// Every derived quantity is checked against a brute-force mask taken from the layout's
// own definition (chunk ids, or the caller's raw range arrays), not from the table.
#include <algorithm>
#include <cstdint>
#include <cstdlib>
#include <cstdio>
#include <random>
#include <set>
#include <string>
#include <vector>

#include "args.hpp"
#include "attn_jvp.h"
#include "layout.hpp"
#include "validate.hpp"

namespace {

int fails = 0;
#define CHECK(c, ...)                 \
  do {                                \
    if (!(c)) {                       \
      if (fails < 20) {               \
        std::printf(__VA_ARGS__);     \
        std::printf("\n");            \
      }                               \
      ++fails;                        \
    }                                 \
  } while (0)

struct Layout {
  int kind = ATTN_MASK_FULL, n = 0, L = 0;
  std::vector<int32_t> offs, roffs, ranges;
  attn_chunk_layout c() const {
    return {kind, n, offs.empty() ? nullptr : offs.data(), roffs.empty() ? nullptr : roffs.data(),
            ranges.empty() ? nullptr : ranges.data()};
  }
  // the mask from the definition of the layout kind
  bool allowed(int q, int k) const {
    if (kind == ATTN_MASK_FULL) return true;
    if (kind == ATTN_MASK_RANGES) {
      int g = 0;
      while (offs[g + 1] <= q) ++g;
      for (int r = roffs[g]; r < roffs[g + 1]; ++r)
        if (k >= ranges[2 * r] && k < ranges[2 * r + 1]) return true;
      return false;
    }
    auto chunk = [&](int t) {
      int c = 0;
      while (offs[c + 1] <= t) ++c;
      return c;
    };
    if (kind == ATTN_MASK_BLOCK_CAUSAL) return chunk(k) <= chunk(q);
    const int half = offs[n];
    const bool qn = q >= half, kn = k >= half;
    const int cq = chunk(qn ? q - half : q), ck = chunk(kn ? k - half : k);
    return (!qn && !kn && ck <= cq) || (qn && !kn && ck < cq) || (qn && kn && ck == cq);
  }
};

Layout random_layout(std::mt19937& rng) {
  Layout l;
  auto uni = [&](int a, int b) { return std::uniform_int_distribution<int>(a, b)(rng); };
  l.kind = uni(0, 3);
  if (l.kind == ATTN_MASK_FULL) {
    l.L = uni(1, 1500);
    return l;
  }
  if (l.kind == ATTN_MASK_RANGES) {
    l.L = uni(1, 1500);
    const int G = uni(1, std::min(l.L, 40));
    std::set<int> cut;
    while ((int)cut.size() < G - 1) cut.insert(uni(1, l.L - 1));
    l.offs = {0};
    l.offs.insert(l.offs.end(), cut.begin(), cut.end());
    l.offs.push_back(l.L);
    l.n = G;
    l.roffs = {0};
    for (int g = 0; g < G; ++g) {
      // disjoint ranges: sorted random points paired up, some touching, some empty, shuffled
      const int R = uni(0, 6);
      std::vector<int> pts;
      for (int i = 0; i < 2 * R; ++i) pts.push_back(uni(0, l.L));
      std::sort(pts.begin(), pts.end());
      std::vector<std::pair<int, int>> ks;
      for (int i = 0; i < R; ++i) ks.push_back({pts[2 * i], pts[2 * i + 1]});
      if (R >= 2 && uni(0, 2) == 0) ks[1].first = ks[0].second;
      std::shuffle(ks.begin(), ks.end(), rng);
      for (auto& k : ks) {
        l.ranges.push_back(k.first);
        l.ranges.push_back(k.second);
      }
      l.roffs.push_back((int)l.ranges.size() / 2);
    }
    return l;
  }
  const int N = uni(1, 12);
  l.n = N;
  l.offs = {0};
  for (int i = 0; i < N; ++i) l.offs.push_back(l.offs.back() + uni(1, 90));
  l.L = l.kind == ATTN_MASK_TEACHER_FORCING ? 2 * l.offs[N] : l.offs[N];
  return l;
}

void check_layout(const Layout& l) {
  const attn_chunk_layout c = l.c();
  attn::GroupTable gt;
  std::string err;
  CHECK(attn::build_groups(&c, l.L, &gt, &err), "valid layout rejected: %s", err.c_str());
  const int L = l.L;
  // the table reproduces the mask, in normal form
  int64_t pairs = 0;
  for (int g = 0; g < gt.n; ++g)
    for (int r = gt.r_begin[g]; r < gt.r_begin[g + 1]; ++r) {
      CHECK(gt.k[2 * r] < gt.k[2 * r + 1], "empty range in the table");
      if (r > gt.r_begin[g]) CHECK(gt.k[2 * r - 1] < gt.k[2 * r], "unsorted or touching ranges");
    }
  std::vector<std::vector<char>> m(L, std::vector<char>(L));
  for (int q = 0; q < L; ++q)
    for (int k = 0; k < L; ++k) {
      m[q][k] = l.allowed(q, k);
      pairs += m[q][k];
    }
  CHECK(attn::count_pairs(gt) == pairs, "pair count %lld vs %lld", (long long)attn::count_pairs(gt),
        (long long)pairs);
  // query-tile plans (both tile heights) and the per-row bits
  for (int br : {attn::kMfmaBr, attn::kMfmaBrFwd}) {
    for (int q0 = 0; q0 < L; q0 += br) {
      const int q1 = std::min(L, q0 + br);
      const attn::TilePlan p = attn::plan_tile(gt, q0, q1, attn::kMfmaBc);
      const int nb = attn::plan_num_blocks(p);
      std::vector<char> vis((L + 31) / 32 + 1);
      int prev = -1;
      for (int i = 0; i < nb; ++i) {
        const int b = attn::plan_block(p, i);
        CHECK(b > prev && b * 32 < L, "plan block order / range");
        prev = b;
        vis[b] = 1;
        if (attn::block_is_full(p, b * 32, 32, L))
          for (int q = q0; q < q1; ++q)
            for (int k = b * 32; k < b * 32 + 32; ++k) CHECK(m[q][k], "full block with a masked pair");
      }
      for (int q = q0; q < q1; ++q)
        for (int k = 0; k < L; ++k)
          if (m[q][k]) CHECK(vis[k / 32], "admissible pair in an unvisited block");
      CHECK(attn::plan_blocks_below(p, (L / 2) / 32) <= nb, "blocks below");
      // per-row bits over every window of the tile's plan, and past the end
      for (int w = q0; w < q1; w += 32) {
        const int g0 = attn::find_group(gt, std::min(w, L - 1)), g1 = attn::find_group(gt, std::min(w + 31, L - 1));
        for (int kb = 0; kb < L + 64; kb += 32)
          for (int row = w; row < std::min(w + 32, L); ++row) {
            const uint32_t bits = attn::row_bits(gt, g0, g1, row, kb);
            for (int j = 0; j < 32; ++j) {
              const int k = kb + j;
              CHECK(((bits >> j) & 1u) == (k < L && m[row][k] ? 1u : 0u), "row bits row %d key %d", row, k);
            }
          }
      }
    }
  }
  // key-tile plans and per-key bits, windows past the end included
  const int KT = attn::kBwdKeysPerTile, QB = attn::kBwdRowsPerBlock;
  for (int k0 = 0; k0 < L; k0 += KT) {
    const int k1 = std::min(L, k0 + KT);
    const attn::TilePlan p = attn::plan_key_tile(gt, k0, k1, QB);
    const int nb = attn::plan_num_blocks(p);
    std::vector<char> vis((L + QB - 1) / QB + 1);
    int prev = -1;
    for (int i = 0; i < nb; ++i) {
      const int b = attn::plan_block(p, i);
      CHECK(b > prev && b * QB < L, "key plan block order / range");
      prev = b;
      vis[b] = 1;
      if (attn::block_is_full(p, b * QB, QB, L))
        for (int q = b * QB; q < b * QB + QB; ++q)
          for (int k = k0; k < k1; ++k) CHECK(m[q][k], "full query block with a masked pair");
      for (int half = 0; half < 2; ++half) {
        const int qb = b * QB + 32 * half;
        for (int k = k0; k < k1; ++k) {
          const uint32_t bits = attn::key_bits(gt, k, qb, L);
          for (int j = 0; j < 32; ++j) {
            const int q = qb + j;
            CHECK(((bits >> j) & 1u) == (q < L && m[q][k] ? 1u : 0u), "key bits key %d query %d", k, q);
          }
        }
      }
    }
    for (int q = 0; q < L; ++q)
      for (int k = k0; k < k1; ++k)
        if (m[q][k]) CHECK(vis[q / QB], "admissible pair in an unvisited query block");
  }
  // tile orders are permutations
  auto perm = [&](const attn::TileOrder& o) {
    std::set<int> s;
    for (int t = 0; t < o.nt; ++t) s.insert(attn::tile_of(o, t));
    return (int)s.size() == o.nt && *s.begin() == 0 && *s.rbegin() == o.nt - 1;
  };
  CHECK(perm(attn::make_tile_order(&c, L, attn::kMfmaBr)), "tile order");
  CHECK(perm(attn::make_tile_order(&c, L, attn::kMfmaBrFwd)), "forward tile order");
  if (l.kind == ATTN_MASK_TEACHER_FORCING)
    CHECK(perm(attn::make_tile_order_zero_clean(gt, L, attn::kMfmaBr, attn::kMfmaBc, L / 2)), "zero-clean order");
  // the host entry points on this layout
  std::vector<int32_t> bounds(ATTN_MAX_GROUPS + 1), ro(ATTN_MAX_GROUPS + 1), rk(2 * ATTN_MAX_RANGES);
  CHECK(attn_query_groups(&c, L, bounds.data(), ro.data(), rk.data(), ATTN_MAX_GROUPS, ATTN_MAX_RANGES) == gt.n,
        "attn_query_groups");
  CHECK(attn_query_groups(&c, L, bounds.data(), ro.data(), rk.data(), gt.n - 1, ATTN_MAX_RANGES) == -1,
        "attn_query_groups with a short buffer");
  CHECK(attn_count_unmasked_pairs(&c, L) == pairs, "attn_count_unmasked_pairs");
  std::vector<int32_t> blk(L / 16 + 8), full(L / 16 + 8);
  for (int t = 0; t * attn::kMfmaBr < L; ++t)
    CHECK(attn_tile_plan(&c, L, t, blk.data(), full.data(), (int)blk.size()) >= 0, "attn_tile_plan");
  for (int t = 0; t * KT < L; ++t)
    CHECK(attn_key_tile_plan(&c, L, t, blk.data(), full.data(), (int)blk.size()) >= 0, "attn_key_tile_plan");
  CHECK(attn_tile_plan(&c, L, (L + attn::kMfmaBr - 1) / attn::kMfmaBr, blk.data(), full.data(), 8) == -1,
        "tile index past the end");
  std::vector<int32_t> order(L / 64 + 8);
  CHECK(attn_tile_order(&c, L, 0, order.data(), (int)order.size()) >= 0, "attn_tile_order");
}

// Corrupt a valid layout in one random way; the library must reject it or accept it
// consistently, never read out of bounds.
void check_corrupt(const Layout& l0, std::mt19937& rng) {
  Layout l = l0;
  auto uni = [&](int a, int b) { return std::uniform_int_distribution<int>(a, b)(rng); };
  int L = l.L;
  switch (uni(0, 5)) {
    case 0: L += uni(-3, 3); break;
    case 1: if (!l.offs.empty()) l.offs[uni(0, (int)l.offs.size() - 1)] += uni(-5, 5); break;
    case 2: if (!l.ranges.empty()) l.ranges[uni(0, (int)l.ranges.size() - 1)] += uni(-30, 30); break;
    case 3: if (!l.roffs.empty()) { const int i = uni(1, (int)l.roffs.size() - 1); l.roffs[i] = std::max(0, std::min(l.roffs[i] + uni(-1, 1), (int)l.ranges.size() / 2)); } break;
    case 4: l.kind = uni(-1, 5); if (l.kind == ATTN_MASK_RANGES && l.roffs.empty()) l.kind = ATTN_MASK_FULL; break;
    default: if (l.kind != ATTN_MASK_RANGES && l.kind != ATTN_MASK_FULL) l.n = uni(0, (int)l.offs.size() - 1); break;
  }
  const attn_chunk_layout c = l.c();
  attn::GroupTable gt;
  std::string err;
  const bool ok = attn::build_groups(&c, L, &gt, &err);
  CHECK(ok || !err.empty(), "rejection without a message");
  if (ok && L > 0) {
    CHECK(attn_count_unmasked_pairs(&c, L) >= 0, "accepted layout without a pair count");
  }
}

// Argument validation with fake pointers (never dereferenced).
void check_prepare(std::mt19937& rng) {
  auto uni = [&](int a, int b) { return std::uniform_int_distribution<int>(a, b)(rng); };
  const int dtype = uni(-1, 2), B = uni(-1, 3), H = uni(-1, 3), L = uni(-2, 700), D = uni(0, 3) * 64;
  std::vector<uintptr_t> p(10);
  uintptr_t base = (uintptr_t)1 << 40;
  for (auto& x : p) {
    x = base + (uintptr_t)uni(0, 3) * (uintptr_t)uni(0, 1 << 20) * 16 + (uintptr_t)uni(0, 1) * (uintptr_t)uni(0, 8);
    if (uni(0, 30) == 0) x = 0;
    base += (uintptr_t)1 << 32;
  }
  if (uni(0, 4) == 0) p[uni(0, 9)] = p[uni(0, 9)];
  const int32_t offs[3] = {0, 100, 350};
  const attn_chunk_layout lay = {uni(0, 1) ? ATTN_MASK_TEACHER_FORCING : ATTN_MASK_FULL, 2, offs, nullptr, nullptr};
  attn::AttnArgs a;
  for (attn::Pass pass : {attn::Pass::kFwd, attn::Pass::kJvp, attn::Pass::kJvpZeroClean}) {
    const int rc = attn::prepare(pass, dtype, B, H, L, D, (void*)p[0], (void*)p[1], (void*)p[2], (void*)p[3],
                                 (void*)p[4], (void*)p[5], &lay, 0.f, (void*)p[6], (void*)p[7], (float*)p[8], &a);
    CHECK(rc == ATTN_OK || attn::last_error_message()[0] != '\0', "error without a message");
    if (rc == ATTN_OK) CHECK(a.L == L && a.B == B && a.H == H && a.gt.n >= 1, "prepared arguments");
  }
  attn::BwdArgs qa, ka;
  const int rc = attn::prepare_bwd(dtype, B, H, L, D, (void*)p[0], (void*)p[1], (void*)p[2], (void*)p[3],
                                   (void*)p[4], (const float*)p[5], &lay, 0.f, (void*)p[6], (void*)p[7],
                                   (void*)p[8], (float*)p[9], &qa, &ka);
  CHECK(rc == ATTN_OK || attn::last_error_message()[0] != '\0', "backward error without a message");
}

}  // namespace

int main(int argc, char** argv) {
  const int iters = argc > 1 ? std::atoi(argv[1]) : 150;
  std::mt19937 rng(20261202);
  for (int it = 0; it < iters; ++it) {
    const Layout l = random_layout(rng);
    check_layout(l);
    for (int j = 0; j < 4; ++j) check_corrupt(l, rng);
    for (int j = 0; j < 20; ++j) check_prepare(rng);
  }
  // fixed cases: the largest tables, and one range past the table
  {
    Layout l;
    l.kind = ATTN_MASK_TEACHER_FORCING;
    l.n = ATTN_MAX_CHUNKS;
    for (int i = 0; i <= l.n; ++i) l.offs.push_back(3 * i);
    l.L = 2 * l.offs.back();
    check_layout(l);
    Layout r;
    r.kind = ATTN_MASK_RANGES;
    r.n = 1;
    r.L = 2 * (ATTN_MAX_RANGES + 1);
    r.offs = {0, r.L};
    r.roffs = {0, ATTN_MAX_RANGES + 1};
    for (int i = 0; i <= ATTN_MAX_RANGES; ++i) {
      r.ranges.push_back(2 * i);
      r.ranges.push_back(2 * i + 1);
    }
    const attn_chunk_layout c = r.c();
    attn::GroupTable gt;
    std::string err;
    CHECK(!attn::build_groups(&c, r.L, &gt, &err) && err.find("ATTN_MAX_RANGES") != std::string::npos,
          "range table overflow not rejected");
    r.roffs[1] = ATTN_MAX_RANGES;
    r.ranges.resize(2 * ATTN_MAX_RANGES);
    check_layout(r);
  }
  std::printf(fails ? "FAIL %d\n" : "OK\n", fails);
  return fails ? 1 : 0;
}
