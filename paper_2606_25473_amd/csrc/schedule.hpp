// schedule.hpp -- mask -> query groups -> per-query-tile key-block plan.
//
// Shared by the host code (layout validation, pair counts) and the kernels
// (which evaluate the same plan on scalar registers), so that both always agree
// on which key blocks a query tile visits.
//
// Representation (paper App. B, "Sparse custom-mask representation"): the mask
// is a list of query groups; group g owns the contiguous query interval
// [q_begin(g), q_end[g]) and admits keys in at most two intervals
// [a0, a1) and [b0, b1).  The groups tile [0, L) in order.  The TF mask of the
// packed [clean | noisy] sequence (paper Sec. 3.1.1) gives 2N groups: clean
// chunk j admits [0, o_{j+1}); noisy chunk i admits [0, o_i) and its own noisy
// chunk [half + o_i, half + o_{i+1}).  Block-causal gives N groups with one
// range, full attention one group with one range.
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
#else
#define ATTN_HD inline
#endif

namespace attn {

constexpr int kMaxGroups = 128;  // 2 * ATTN_MAX_CHUNKS = ATTN_MAX_GROUPS

struct GroupTable {
  int32_t n;
  int32_t q_end[kMaxGroups];
  int32_t a0[kMaxGroups], a1[kMaxGroups];
  int32_t b0[kMaxGroups], b1[kMaxGroups];
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

// Key-block plan of the query tile [q0, q1) with key blocks of bc keys.
struct TilePlan {
  int nseg;                     // 0, 1 or 2 block segments, in increasing key order
  int blk_begin0, blk_end0;     // scalar fields (no arrays): the plan lives in registers
  int blk_begin1, blk_end1;
  int afull_lo, afull_hi;       // keys admitted via range a for EVERY row of the tile
  int bfull_lo, bfull_hi;       // keys admitted via range b for EVERY row of the tile
  int g_first, g_last;          // groups overlapping the tile
};

ATTN_HD int imin(int a, int b) { return a < b ? a : b; }
ATTN_HD int imax(int a, int b) { return a > b ? a : b; }

ATTN_HD TilePlan plan_tile(const GroupTable& gt, int q0, int q1, int bc) {
  TilePlan p;
  const int big = 0x7fffffff;
  int alo = big, ahi = 0, blo = big, bhi = 0;
  int afl = 0, afh = big, bfl = 0, bfh = big;
  p.g_first = find_group(gt, q0);
  int g = p.g_first;
  for (; g < gt.n; ++g) {
    if (group_q_begin(gt, g) >= q1) break;
    const int a0 = gt.a0[g], a1 = gt.a1[g], b0 = gt.b0[g], b1 = gt.b1[g];
    if (a1 > a0) { alo = imin(alo, a0); ahi = imax(ahi, a1); afl = imax(afl, a0); afh = imin(afh, a1); }
    else { afh = 0; afl = 0; }
    if (b1 > b0) { blo = imin(blo, b0); bhi = imax(bhi, b1); bfl = imax(bfl, b0); bfh = imin(bfh, b1); }
    else { bfh = 0; bfl = 0; }
  }
  p.g_last = g - 1;
  p.afull_lo = afl; p.afull_hi = afh > afl ? afh : afl;
  p.bfull_lo = bfl; p.bfull_hi = bfh > bfl ? bfh : bfl;
  int n = 0;
  int sb[2], se[2];
  if (ahi > alo) { sb[n] = alo / bc; se[n] = (ahi + bc - 1) / bc; ++n; }
  if (bhi > blo) { sb[n] = blo / bc; se[n] = (bhi + bc - 1) / bc; ++n; }
  if (n == 2) {
    if (sb[1] < sb[0]) { int t = sb[0]; sb[0] = sb[1]; sb[1] = t; t = se[0]; se[0] = se[1]; se[1] = t; }
    if (se[0] >= sb[1]) { se[0] = imax(se[0], se[1]); n = 1; }  // blocks touch or overlap: merge
  }
  p.nseg = n;
  p.blk_begin0 = n > 0 ? sb[0] : 0;
  p.blk_end0 = n > 0 ? se[0] : 0;
  p.blk_begin1 = n > 1 ? sb[1] : 0;
  p.blk_end1 = n > 1 ? se[1] : 0;
  return p;
}

ATTN_HD int plan_num_blocks(const TilePlan& p) {
  return (p.blk_end0 - p.blk_begin0) + (p.blk_end1 - p.blk_begin1);
}

// i-th visited key block of the plan
ATTN_HD int plan_block(const TilePlan& p, int i) {
  const int n0 = p.blk_end0 - p.blk_begin0;
  return i < n0 ? p.blk_begin0 + i : p.blk_begin1 + (i - n0);
}

// true if every key of block [k0, k0 + bc) exists and is admitted for every row of the tile
ATTN_HD bool block_is_full(const TilePlan& p, int k0, int bc, int L) {
  const int k1 = k0 + bc;
  if (k1 > L) return false;
  return (k0 >= p.afull_lo && k1 <= p.afull_hi) || (k0 >= p.bfull_lo && k1 <= p.bfull_hi);
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
// Work-group b runs on XCD b mod 8, so with hg = 4 or 8 each XCD works on one head.
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
