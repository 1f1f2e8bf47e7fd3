// Host check of the persistent kernels' workgroup placement (wr_layout.h):
// for every plan shape and each of the 64 candidates (heads on XCD hx, units
// on XCD ux, or spread over all when ux == hx), every head and unit role is
// taken by exactly one block of the grid, heads sit on blocks 8 j + hx, units
// only on admitted XCDs, the last block of the grid is busy (the grid is no
// larger than needed) and the default candidate 0 is the original dealing
// (head j at block 8 j, units on the remaining blocks in order).
#include <cstdio>
#include <vector>
#include "wr_layout.h"

static int check(const char* what, PersistPlan P) {
  int bad = 0;
  for (int i = 0; i < 64; ++i) {
    const int hx = i / 8, ux = i % 8, uxm = ux == hx ? 255 : 1 << ux;
    wr_place(&P, hx, uxm);
    std::vector<int> seen(P.NH + P.NU, 0);
    for (int b = 0; b < P.grid; ++b) {
      const int r = wr_role(P, b);
      if (r < 0) continue;
      if (r >= P.NH + P.NU) { ++bad; continue; }
      ++seen[r];
      if (r < P.NH && (b % 8 != hx || b / 8 != r)) ++bad;
      if (r >= P.NH && (!(uxm >> (b % 8) & 1) || (b % 8 == hx && b / 8 < P.NH))) ++bad;
      if (i == 0 && r >= P.NH) {   // original dealing: unit k at block k + heads below it
        const int before = (b + 7) / 8 < P.NH ? (b + 7) / 8 : P.NH;
        if (r - P.NH != b - before) ++bad;
      }
    }
    for (int r = 0; r < P.NH + P.NU; ++r) bad += seen[r] != 1;
    if (wr_role(P, P.grid - 1) < 0) ++bad;
  }
  if (bad) printf("%s: %d violations\n", what, bad);
  return bad;
}

int main() {
  int bad = 0, plans = 0;
  PersistPlan P;
  for (int H = 128; H <= 896; H += 128) {
    if (persist_plan(H, &P)) { bad += check("dense", P); ++plans; }
    if (fused_plan(H, &P)) { bad += check("fused", P); ++plans; }
  }
  for (int H : {256, 512, 1024, 2048})
    for (int SR : {16, 32, 64, 128})
      for (int bh : {4, 16})
        if (sparse_plan(H, SR, bh, bh == 4 ? 4 : 1, 8, 8, &P)) { bad += check("sparse", P); ++plans; }
  printf("%d plans, %d violations\n", plans, bad);
  return bad != 0 || plans < 20;
}
