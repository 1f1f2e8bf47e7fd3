// Host check of the persistent kernels' workgroup placement (wr_layout.h):
// for every plan shape and each of the 64 candidates (heads on XCD hx, units
// on XCD ux, or spread over all when ux == hx), every head, mirror and unit
// role is taken by exactly one block of the grid, heads and then mirrors sit
// on blocks 8 i + hx, units only on admitted XCDs, the last block of the grid
// is busy (the grid is no larger than needed) and the default candidate 0 is
// the original dealing (lead i at block 8 i, units on the remaining blocks in
// order).
#include <cstdio>
#include <vector>
#include "wr_layout.h"

static int check(const char* what, PersistPlan P) {
  int bad = 0;
  for (int i = 0; i < 64; ++i) {
    const int hx = i / 8, ux = i % 8, uxm = ux == hx ? 255 : 1 << ux;
    wr_place(&P, hx, uxm);
    const int NL = P.NH + P.NM;   // heads, then mirrors
    std::vector<int> seen(NL + P.NU, 0);
    for (int b = 0; b < P.grid; ++b) {
      const int r = wr_role(P, b);
      if (r < 0) continue;
      if (r >= NL + P.NU) { ++bad; continue; }
      ++seen[r];
      if (r < NL && (b % 8 != hx || b / 8 != r)) ++bad;
      if (r >= NL && (!(uxm >> (b % 8) & 1) || (b % 8 == hx && b / 8 < NL))) ++bad;
      if (i == 0 && r >= NL) {   // original dealing: unit k at block k + leads below it
        const int before = (b + 7) / 8 < NL ? (b + 7) / 8 : NL;
        if (r - NL != b - before) ++bad;
      }
    }
    for (int r = 0; r < NL + P.NU; ++r) bad += seen[r] != 1;
    if (wr_role(P, P.grid - 1) < 0) ++bad;
  }
  if (bad) printf("%s: %d violations\n", what, bad);
  return bad;
}

// Side-by-side launches of a dense plan (n = 2 .. 4 utterances, launch i's
// heads and mirrors on XCD 8 i / n, units spread, as the library places them):
// every XCD of 32 CUs holds the busy blocks of all n grids.
static int check_fan(PersistPlan P) {
  int bad = 0;
  for (int n = 2; n <= 4; ++n) {
    int busy[8] = {};
    for (int i = 0; i < n; ++i) {
      wr_place(&P, 8 * i / n, 255);
      for (int b = 0; b < P.grid; ++b)
        if (wr_role(P, b) >= 0) ++busy[b % 8];
    }
    for (int x = 0; x < 8; ++x)
      if (busy[x] > 32) {
        printf("H=%d: %d launches put %d workgroups on XCD %d\n", P.H, n, busy[x], x);
        ++bad;
      }
  }
  return bad;
}

int main() {
  int bad = 0, plans = 0;
  PersistPlan P;
  for (int H = 128; H <= 896; H += 128) {
    if (persist_plan(H, &P)) {
      if (P.NM != P.NH || P.NM * WR_MTILES != P.NCT) ++bad;   // the mirrors cover every coarse row tile
      bad += check("dense", P);
      bad += check_fan(P);
      ++plans;
    }
    if (fused_plan(H, &P)) { bad += check("fused", P); ++plans; }
  }
  for (int H : {256, 512, 1024, 2048})
    for (int SR : {16, 32, 64, 128})
      for (int bh : {4, 16})
        if (sparse_plan(H, SR, bh, bh == 4 ? 4 : 1, 8, 8, &P)) { bad += check("sparse", P); ++plans; }
  printf("%d plans, %d violations\n", plans, bad);
  return bad != 0 || plans < 20;
}
