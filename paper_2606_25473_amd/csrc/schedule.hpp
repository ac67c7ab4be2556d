// schedule.hpp -- mask -> query groups -> per-query-tile key-block plan.
//
// Shared by the host code (layout validation, pair counts) and the kernels
// (which evaluate the same plan on scalar registers), so that both always agree
// on which key blocks a query tile visits.
//
// Representation (paper App. B, "Sparse custom-mask representation"): the mask
// is a list of query groups; group g owns the contiguous query interval
// [q_begin(g), q_end[g]) and admits the keys of its list of key ranges
// [k0, k1) (any number, possibly none).  The groups tile [0, L) in order; the
// ranges of a group are stored sorted, disjoint and not touching (the host
// merges adjacent ones and drops empty ones).  The TF mask of the packed
// [clean | noisy] sequence (paper Sec. 3.1.1) gives 2N groups: clean chunk j
// admits [0, o_{j+1}); noisy chunk i admits [0, o_i) and its own noisy chunk
// [half + o_i, half + o_{i+1}).  Block-causal gives N groups with one range,
// full attention one group with one range.
//
// Where Algorithm 1 launches one task per (group, query tile) and recomputes a
// tile that straddles a group boundary once per group, here a query tile is
// one task whatever groups it spans: it visits the union of its rows' key
// blocks once, and applies the per-row mask only on blocks that are not
// admissible for every row of the tile.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define ATTN_HD __host__ __device__ __forceinline__
#define ATTN_UNROLL _Pragma("unroll")
#else
#define ATTN_HD inline
#define ATTN_UNROLL
#endif

namespace attn {

constexpr int kMaxGroups = 128;  // ATTN_MAX_GROUPS (and 2 * ATTN_MAX_CHUNKS)
constexpr int kMaxRanges = 256;  // ATTN_MAX_RANGES

struct GroupTable {
  int32_t n;                         // number of groups
  int32_t q_end[kMaxGroups];         // group g owns rows [q_end[g - 1], q_end[g])
  uint16_t r_begin[kMaxGroups + 1];  // its key ranges are r_begin[g] .. r_begin[g + 1] - 1
  int32_t k[2 * kMaxRanges];         // key range r is [k[2 r], k[2 r + 1])
};

ATTN_HD int32_t group_q_begin(const GroupTable& gt, int g) { return g == 0 ? 0 : gt.q_end[g - 1]; }

// index of the group containing query row q (groups are sorted by q_end)
ATTN_HD int find_group(const GroupTable& gt, int q) {
  int lo = 0, hi = gt.n - 1;
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if (gt.q_end[mid] > q) hi = mid; else lo = mid + 1;
  }
  return lo;
}

ATTN_HD int imin(int a, int b) { return a < b ? a : b; }
ATTN_HD int imax(int a, int b) { return a > b ? a : b; }

// Key-block plan of a query tile: the visited key blocks form at most kPlanSegs
// segments in increasing order; the i-th visited block is i + off[s] for the segment s
// with cend[s - 1] <= i < cend[s].  When the tile's rows admit keys in more separate
// block runs, the runs with the smallest gaps are merged (the blocks in between are
// visited too and masked per row).  flo/fhi: key intervals that EVERY row of the tile
// admits (at most kPlanFull of them, a subset of that set).  Every field is a scalar:
// the plan lives in registers.
constexpr int kPlanSegs = 4;
constexpr int kPlanFull = 2;

struct TilePlan {
  int cend[kPlanSegs];
  int off[kPlanSegs];
  int flo[kPlanFull], fhi[kPlanFull];
  int g_first, g_last;          // groups overlapping the tile
};

namespace detail {
constexpr int kBig = 0x7fffffff;

// Add block run [b, e) to the increasing, disjoint, non-touching segments sb/se (slots
// holding kBig are unused; slot kPlanSegs is spare).
ATTN_HD void plan_insert(int (&sb)[kPlanSegs + 1], int (&se)[kPlanSegs + 1], int b, int e) {
  // absorb every segment that overlaps or touches [b, e); one pass suffices, since the
  // segments do not touch one another
ATTN_UNROLL
  for (int s = 0; s < kPlanSegs; ++s) {
    const bool t = sb[s] <= e && b <= se[s];
    b = t ? imin(b, sb[s]) : b;
    e = t ? imax(e, se[s]) : e;
    sb[s] = t ? kBig : sb[s];
    se[s] = t ? kBig : se[s];
  }
  // append, then restore increasing order (unused slots sort last)
  sb[kPlanSegs] = b;
  se[kPlanSegs] = e;
ATTN_UNROLL
  for (int i = 0; i < kPlanSegs; ++i) {
ATTN_UNROLL
    for (int j = 0; j < kPlanSegs - i; ++j) {
      const bool sw = sb[j] > sb[j + 1];
      const int tb = sb[j], te = se[j];
      sb[j] = sw ? sb[j + 1] : tb;
      se[j] = sw ? se[j + 1] : te;
      sb[j + 1] = sw ? tb : sb[j + 1];
      se[j + 1] = sw ? te : se[j + 1];
    }
  }
  // one segment too many: merge the neighbours with the smallest gap
  if (sb[kPlanSegs] != kBig) {
    int best = 0, bg = sb[1] - se[0];
ATTN_UNROLL
    for (int i = 1; i < kPlanSegs; ++i) {
      const int gap = sb[i + 1] - se[i];
      best = gap < bg ? i : best;
      bg = gap < bg ? gap : bg;
    }
ATTN_UNROLL
    for (int i = 0; i < kPlanSegs; ++i) {
      const int nb = i <= best ? sb[i] : sb[i + 1];
      const int ne = i < best ? se[i] : se[i + 1];
      sb[i] = nb;
      se[i] = ne;
    }
    sb[kPlanSegs] = kBig;
    se[kPlanSegs] = kBig;
  }
}

// Keep the kPlanFull longest intervals: insert [lo, hi) (ignored when empty).
ATTN_HD void keep_longest(int (&lo)[kPlanFull], int (&hi)[kPlanFull], int a, int b) {
  static_assert(kPlanFull == 2, "two full intervals");
  const int len = b - a;
  if (len <= 0) return;
  const bool first = len > hi[0] - lo[0];
  const bool second = !first && len > hi[1] - lo[1];
  lo[1] = first ? lo[0] : (second ? a : lo[1]);
  hi[1] = first ? hi[0] : (second ? b : hi[1]);
  lo[0] = first ? a : lo[0];
  hi[0] = first ? b : hi[0];
}
}  // namespace detail

ATTN_HD TilePlan plan_tile(const GroupTable& gt, int q0, int q1, int bc) {
  using detail::kBig;
  TilePlan p;
  int sb[kPlanSegs + 1], se[kPlanSegs + 1];
ATTN_UNROLL
  for (int s = 0; s <= kPlanSegs; ++s) sb[s] = se[s] = kBig;
  // keys admitted by every row so far: start from everything, intersect group by group
  int flo[kPlanFull] = {0, 0}, fhi[kPlanFull] = {kBig, 0};
  p.g_first = find_group(gt, q0);
  int g = p.g_first;
  for (; g < gt.n && group_q_begin(gt, g) < q1; ++g) {
    int nlo[kPlanFull] = {0, 0}, nhi[kPlanFull] = {0, 0};
    const int r1 = gt.r_begin[g + 1];
    for (int r = gt.r_begin[g]; r < r1; ++r) {
      const int k0 = gt.k[2 * r], k1 = gt.k[2 * r + 1];
      detail::plan_insert(sb, se, k0 / bc, (k1 + bc - 1) / bc);
ATTN_UNROLL
      for (int f = 0; f < kPlanFull; ++f) detail::keep_longest(nlo, nhi, imax(flo[f], k0), imin(fhi[f], k1));
    }
ATTN_UNROLL
    for (int f = 0; f < kPlanFull; ++f) {
      flo[f] = nlo[f];
      fhi[f] = nhi[f];
    }
  }
  p.g_last = g - 1;
  int acc = 0;
ATTN_UNROLL
  for (int s = 0; s < kPlanSegs; ++s) {
    const bool used = sb[s] != kBig;
    p.off[s] = used ? sb[s] - acc : 0;
    acc += used ? se[s] - sb[s] : 0;
    p.cend[s] = acc;
  }
ATTN_UNROLL
  for (int f = 0; f < kPlanFull; ++f) {
    p.flo[f] = flo[f];
    p.fhi[f] = fhi[f] > flo[f] ? fhi[f] : flo[f];
  }
  return p;
}

// Plan of the backward's key tile [k0, k1) over the query-group table: the query blocks
// (of qb rows) of every group that admits some key of the tile, and as full intervals
// the longest runs of consecutive groups that admit every key of the tile.  Loops over
// all groups once per tile; consecutive admitting groups enter the segments as one run.
ATTN_HD TilePlan plan_key_tile(const GroupTable& gt, int k0, int k1, int qb) {
  using detail::kBig;
  TilePlan p;
  int sb[kPlanSegs + 1], se[kPlanSegs + 1];
ATTN_UNROLL
  for (int s = 0; s <= kPlanSegs; ++s) sb[s] = se[s] = kBig;
  int flo[kPlanFull] = {0, 0}, fhi[kPlanFull] = {0, 0};
  int arun0 = 0, arun1 = 0;  // current run of groups admitting some key of the tile
  int frun0 = 0, frun1 = 0;  // current run of groups admitting every key of the tile
  for (int g = 0; g < gt.n; ++g) {
    bool any = false, all = false;
    const int r1 = gt.r_begin[g + 1];
    for (int r = gt.r_begin[g]; r < r1; ++r) {
      const int a = gt.k[2 * r], b = gt.k[2 * r + 1];
      any |= a < k1 && k0 < b;
      all |= a <= k0 && k1 <= b;
    }
    const int q0 = group_q_begin(gt, g), q1 = gt.q_end[g];
    if (any) {
      if (arun1 != q0 || arun1 == arun0) {  // not adjacent to the current run: flush it
        if (arun1 > arun0) detail::plan_insert(sb, se, arun0 / qb, (arun1 + qb - 1) / qb);
        arun0 = q0;
      }
      arun1 = q1;
    }
    if (all) {
      if (frun1 != q0 || frun1 == frun0) {
        detail::keep_longest(flo, fhi, frun0, frun1);
        frun0 = q0;
      }
      frun1 = q1;
    }
  }
  if (arun1 > arun0) detail::plan_insert(sb, se, arun0 / qb, (arun1 + qb - 1) / qb);
  detail::keep_longest(flo, fhi, frun0, frun1);
  p.g_first = 0;
  p.g_last = gt.n - 1;
  int acc = 0;
ATTN_UNROLL
  for (int s = 0; s < kPlanSegs; ++s) {
    const bool used = sb[s] != kBig;
    p.off[s] = used ? sb[s] - acc : 0;
    acc += used ? se[s] - sb[s] : 0;
    p.cend[s] = acc;
  }
ATTN_UNROLL
  for (int f = 0; f < kPlanFull; ++f) {
    p.flo[f] = flo[f];
    p.fhi[f] = fhi[f];
  }
  return p;
}

ATTN_HD int plan_num_blocks(const TilePlan& p) { return p.cend[kPlanSegs - 1]; }

// i-th visited key block of the plan (0 <= i < plan_num_blocks).  Written as a sum of
// selects against zero: a select between two fields lets the compiler turn the plan into
// memory indexed by the selected address (scratch), where these stay in scalar registers.
ATTN_HD int plan_block(const TilePlan& p, int i) {
  static_assert(kPlanSegs == 4, "segment sum below");
  return i + p.off[0] + (i >= p.cend[0] ? p.off[1] - p.off[0] : 0) + (i >= p.cend[1] ? p.off[2] - p.off[1] : 0) +
         (i >= p.cend[2] ? p.off[3] - p.off[2] : 0);
}

// number of visited blocks with index below kc (they come first: blocks increase)
ATTN_HD int plan_blocks_below(const TilePlan& p, int kc) {
  int n = 0, prev = 0;
ATTN_UNROLL
  for (int s = 0; s < kPlanSegs; ++s) {
    const int len = p.cend[s] - prev;
    n += imin(imax(kc - (p.off[s] + prev), 0), len);
    prev = p.cend[s];
  }
  return n;
}

// true if every key of block [k0, k0 + bc) exists and is admitted for every row of the tile
ATTN_HD bool block_is_full(const TilePlan& p, int k0, int bc, int L) {
  static_assert(kPlanFull == 2, "two full intervals");
  const int k1 = k0 + bc;
  if (k1 > L) return false;
  return (k0 >= p.flo[0] && k1 <= p.fhi[0]) || (k0 >= p.flo[1] && k1 <= p.fhi[1]);
}

// Bit j set: key kb + j (0 <= j < 32) lies in one of group g's key ranges.
ATTN_HD uint32_t group_bits(const GroupTable& gt, int g, int kb) {
  uint32_t bits = 0;
  const int r1 = gt.r_begin[g + 1];
  for (int r = gt.r_begin[g]; r < r1; ++r) {
    const int lo = imax(gt.k[2 * r] - kb, 0), hi = imin(gt.k[2 * r + 1] - kb, 32);
    if (hi > lo) bits |= (hi == 32 ? ~0u : (1u << hi) - 1u) & ~((1u << lo) - 1u);
  }
  return bits;
}

// The keys kb .. kb + 31 admitted for query `row`, as bits, given groups g0 .. g1 that
// contain the row (the row lies in the last of them whose first row is <= row).  With
// g0 and g1 uniform across a wave the range loop is scalar; only the final choice is
// per lane.
ATTN_HD uint32_t row_bits(const GroupTable& gt, int g0, int g1, int row, int kb) {
  uint32_t bits = 0;
  for (int g = g0; g <= g1; ++g) {
    const uint32_t b = group_bits(gt, g, kb);
    bits = row >= group_q_begin(gt, g) ? b : bits;
  }
  return bits;
}

// The queries qb .. qb + 31 that admit key `key`, as bits (backward key-tile pass).  The
// group loop is uniform across a wave; the membership of the lane's key in a group's
// ranges is per lane.
ATTN_HD uint32_t key_bits(const GroupTable& gt, int key, int qb, int L) {
  uint32_t bits = 0;
  const int qe = imin(qb + 32, L);
  for (int g = find_group(gt, imin(qb, L - 1)); g < gt.n && group_q_begin(gt, g) < qe; ++g) {
    bool hit = false;
    const int r1 = gt.r_begin[g + 1];
    for (int r = gt.r_begin[g]; r < r1; ++r)
      hit |= (unsigned)(key - gt.k[2 * r]) < (unsigned)(gt.k[2 * r + 1] - gt.k[2 * r]);
    // the group's rows within the window (none when the window lies past the end of the
    // sequence, where the last group ends before qb)
    const int lo = imax(group_q_begin(gt, g) - qb, 0), hi = imin(gt.q_end[g] - qb, 32);
    const uint32_t span = hi > lo ? (hi == 32 ? ~0u : (1u << hi) - 1u) & ~((1u << lo) - 1u) : 0u;
    bits |= hit ? span : 0u;
  }
  return bits;
}

// Order in which work-groups take query tiles: heaviest first where the mask
// makes per-tile work predictable.
//   mode 0: tile = t                         (full mask: equal work)
//   mode 1: tile = nt - 1 - t                (block-causal: work grows with the tile index)
//   mode 2: two halves [0, split) and [split, nt), each taken from its end,
//           interleaved (teacher forcing: work grows with the chunk index in
//           both the clean and the noisy half)
//   mode 3: tile `first` (if >= 0; it is then tile `split`), followed by the two
//           halves [0, split) and [split + (first >= 0), nt), each taken from its
//           end and merged by the bit string `merge` (bit t set: the t-th tile after
//           `first` is the next one of the upper half).  The host merges by
//           estimated tile cost, for layouts whose halves cost different amounts
//           per tile.
constexpr int kMaxMergeTiles = 1024;

struct TileOrder {
  int mode, nt, split, first;
  uint32_t merge[kMaxMergeTiles / 32];
};

ATTN_HD int popc32(uint32_t x) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __popc(x);
#else
  return __builtin_popcount(x);
#endif
}

ATTN_HD int tile_of(const TileOrder& o, int t) {
  if (o.mode == 1) return o.nt - 1 - t;
  if (o.mode == 2) {
    const int na = o.split, nb = o.nt - o.split;
    const int m = imin(na, nb);
    if (t < 2 * m) return (t & 1) ? (o.nt - 1 - (t >> 1)) : (na - 1 - (t >> 1));
    const int r = t - 2 * m;
    return na > nb ? (na - 1 - m - r) : (o.nt - 1 - m - r);
  }
  if (o.mode == 3) {
    if (o.first >= 0) {
      if (t == 0) return o.first;
      --t;
    }
    int upper = 0;  // upper-half tiles taken before position t
    for (int w = 0; w < (t >> 5); ++w) upper += popc32(o.merge[w]);
    const uint32_t word = o.merge[t >> 5];
    upper += popc32(word & ((1u << (t & 31)) - 1u));
    return ((word >> (t & 31)) & 1u) ? o.nt - 1 - upper : o.split - 1 - (t - upper);
  }
  return t;
}

// Work-group b of a launch over nbh (batch, head) pairs and nt tiles per pair: the pairs
// form groups of hg, taken one group after another; inside a group, work-groups go
// position-major (every pair's first tile of the order, then every pair's second, ...).
// So the heaviest tiles of a group's heads are dispatched first, before any light one,
// and a run never ends on a few long tiles of the last head (heads one after another
// leave such a tail); and only about hg heads' keys and values are in flight at once,
// which keeps the caches useful (all heads at once slowed launches over many heads).
// Work-group b runs on XCD b mod 8, so inside a full group of hg = 4 or 8 heads each XCD
// works on one head.  A partial last group (B * H not a multiple of hg) of gsz heads,
// gsz not dividing 8, spreads each of its heads over every XCD.
// Measured: groups of 4 for the JVP, forward and backward query-tile kernels, 8 for the
// zero-clean JVP and the backward key-tile pass.
constexpr int kHeadGroup = 4;      // JVP, forward, backward query-tile pass
constexpr int kHeadGroupWide = 8;  // zero-clean JVP, backward key-tile pass

struct TileSlot {
  int bh, pos;
};

ATTN_HD TileSlot slot_of(int b, int nbh, int nt, int hg) {
  const int grp = b / (hg * nt);
  const int gsz = imin(hg, nbh - grp * hg);
  const int r = b - grp * hg * nt;
  TileSlot s;
  s.pos = r / gsz;
  s.bh = grp * hg + (r - s.pos * gsz);
  return s;
}

}  // namespace attn
