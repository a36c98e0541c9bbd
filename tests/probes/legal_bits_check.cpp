// Host check of the bit-mask forms of the window rule against legal32 itself:
// random windows (clamped as the kernels clamp them), random queries and key
// or query offsets around every boundary; prints the number of mismatches.
// Build: hipcc -x hip --offload-arch=gfx950 -O1 -I include legal_bits_check.cpp
#include "../../paper_2609_32704_amd/csrc/window_rule.h"
#include <stdio.h>
#include <random>
using namespace cowa;
int main() {
  std::mt19937 rng(2609);
  auto pick = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  long checked = 0, bad = 0;
  for (int t = 0; t < 20000; ++t) {
    HeadGeo hg;
    hg.n_k = pick(1, 600);
    hg.n_q = pick(1, hg.n_k);
    hg.w_sink = pick(0, 3) == 0 ? 0 : pick(0, 200);
    hg.w_near = pick(0, 3) == 0 ? 0 : pick(0, 300);
    hg.lo = pick(0, 700);
    hg.hi = pick(0, 3) == 0 ? hg.lo : hg.lo + pick(0, 400);
    hg.tile_q = hg.tile_k = 64;
    const Geo32 g = geo32(hg);
    for (int r = 0; r < 20; ++r) {
      const int q = pick(0, hg.n_q + 40), key0 = pick(0, hg.n_k + 40);
      const uint32_t m = legal_keys32(g, q, key0);
      for (int j = 0; j < 32; ++j) {
        const bool want = q < g.n_q && key0 + j < g.n_k && legal32(g, q, key0 + j);
        bad += want != (bool)((m >> j) & 1u);
        ++checked;
      }
      const int q0 = pick(0, hg.n_q + 40), k = pick(0, hg.n_k + 40);
      const uint32_t mq = legal_queries32(g, q0, k);
      for (int i = 0; i < 32; ++i) {
        const bool want = q0 + i < g.n_q && k < g.n_k && legal32(g, q0 + i, k);
        bad += want != (bool)((mq >> i) & 1u);
        ++checked;
      }
    }
  }
  printf("checked %ld mismatches %ld\n", checked, bad);
  return bad == 0 ? 0 : 1;
}
