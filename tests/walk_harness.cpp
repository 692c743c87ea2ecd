// Host harness for the scheduled dK/dV kernel's walk (walk_plan, walk_step in
// common.hpp): reads "a0 b0 a1 b1 npairs" lines from stdin and prints, per
// line, the step count and then "q s hp" for every step, followed by the live
// flags of the steps just past either end.
#include <cstdio>

#include "common.hpp"

int main() {
  int a0, b0, a1, b1, np;
  while (std::scanf("%d %d %d %d %d", &a0, &b0, &a1, &b1, &np) == 5) {
    const bdlm::WalkPlan w = bdlm::walk_plan(a0, b0, a1, b1, np);
    std::printf("%d\n", w.nsteps);
    for (int i = 0; i < w.nsteps; ++i) {
      const bdlm::WalkStep s = bdlm::walk_step(w, i);
      std::printf("%d %d %d %d\n", s.q, s.s, s.hp, s.live ? 1 : 0);
    }
    std::printf("%d %d\n", bdlm::walk_step(w, w.nsteps).live ? 1 : 0, bdlm::walk_step(w, -1).live ? 1 : 0);
  }
  return 0;
}
