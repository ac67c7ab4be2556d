// Host checks of the scheduling helpers the kernels evaluate on the device
// (paper_2606_25473_amd/csrc/schedule.hpp is shared by host and device code):
// every work-group of a launch gets a distinct (batch-head, tile) slot, and every
// tile order is a permutation.
#include <cstdio>
#include <set>
#include <utility>

#include "schedule.hpp"

int main() {
  int fails = 0;
  for (int hg : {attn::kHeadGroup, attn::kHeadGroupWide}) {
    for (int nbh : {1, 2, 11, 12, 13, 24, 80}) {
      for (int nt : {1, 7, 256, 1025}) {
        std::set<std::pair<int, int>> seen;
        for (int b = 0; b < nbh * nt; ++b) {
          const attn::TileSlot s = attn::slot_of(b, nbh, nt, hg);
          if (s.bh < 0 || s.bh >= nbh || s.pos < 0 || s.pos >= nt) ++fails;
          seen.insert({s.bh, s.pos});
        }
        if ((int)seen.size() != nbh * nt) { std::printf("slot_of hg=%d nbh=%d nt=%d\n", hg, nbh, nt); ++fails; }
        // inside a group, position-major: the first group's first nbh' slots are position 0
        const int g0 = nbh < hg ? nbh : hg;
        for (int b = 0; b < g0; ++b)
          if (attn::slot_of(b, nbh, nt, hg).pos != 0) { std::printf("position-major\n"); ++fails; break; }
        // each XCD (work-group b mod 8) sees one head of the first group while it lasts
        if (nbh >= hg && nt >= 8)
          for (int b = 0; b + 8 < hg * nt; ++b)
            if (attn::slot_of(b, nbh, nt, hg).bh != attn::slot_of(b + 8, nbh, nt, hg).bh) {
              std::printf("one head per XCD hg=%d nbh=%d nt=%d\n", hg, nbh, nt); ++fails; break;
            }
      }
    }
  }
  for (int mode : {0, 1, 2}) {
    for (int nt : {1, 2, 9, 256}) {
      for (int split : {0, 1, nt / 2, nt}) {
        attn::TileOrder o{};
        o.mode = mode; o.nt = nt; o.split = split; o.first = -1;
        std::set<int> seen;
        for (int t = 0; t < nt; ++t) seen.insert(attn::tile_of(o, t));
        if ((int)seen.size() != nt || *seen.begin() != 0 || *seen.rbegin() != nt - 1) {
          std::printf("tile_of mode=%d nt=%d split=%d\n", mode, nt, split); ++fails;
        }
      }
    }
  }
  std::printf(fails ? "FAIL\n" : "OK\n");
  return fails;
}
