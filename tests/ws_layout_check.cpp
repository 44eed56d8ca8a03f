// Host-side check of the evaluation workspace's control block against what include/hedgespec.h
// states: the epoch (uint32) at byte 0, the fail word at 8, the two tagged counters at 16 and
// 24, the mailbox rings from byte 64, every region 256-byte aligned and disjoint, and the size
// hs_eval_alpha_workspace_size reports. Built with hipcc and run on the CPU (no HIP call).
#include <cstdio>
#include <cstdlib>

#include "hs_internal.h"

static int fails = 0;
#define CHECK(c)                                              \
  do {                                                        \
    if (!(c)) {                                               \
      std::printf("FAIL %s:%d %s\n", __FILE__, __LINE__, #c); \
      ++fails;                                                \
    }                                                         \
  } while (0)

int main() {
  const int shapes[][5] = {{1, 8, 8, 151936, HS_BF16}, {32, 64, 8, 151936, HS_BF16},
                           {16, 16, 64, 151936, HS_BF16}, {1, 4, 4, 32000, HS_F32},
                           {3, 1, 1, 1, HS_F32}};
  for (const auto& s : shapes) {
    hs::TeamGeom g;
    CHECK(hs::team_geom(s[0], s[1], s[2], s[3], s[4], &g));
    const hs::TeamWs L = hs::team_ws(g);
    CHECK(L.epoch == 0);
    // control block: epoch 0..3, fail 8..15, row-set count 16..23, finished count 24..31,
    // mailboxes 64 .. 64 + 32 * kMaxTeams
    CHECK(L.stat >= 64 + 32 * (size_t)hs::kMaxTeams);
    const size_t regions[] = {L.stat, L.norm, L.part, L.gw, L.total};
    for (size_t r : regions) CHECK(r % 256 == 0);
    const size_t sets = (size_t)g.G * g.nsub, rows = (size_t)g.D + 1;
    CHECK(L.norm >= L.stat + 24 * sets * rows * g.S);
    // the normaliser words, and kNormCopies - 1 more copies after the gamma words (the
    // single-item kernel's), each 256-byte aligned and large enough
    CHECK(L.norm_copy % 256 == 0 && L.norm_copy >= 24 * sets * rows);
    CHECK(L.part >= L.norm + L.norm_copy);
    CHECK(L.gw >= L.part + 8 * (size_t)g.G * g.N * g.S);
    CHECK(L.total >= hs::align256(L.gw + 8 * (size_t)g.B * g.N * g.K) +
                         (size_t)(hs::kNormCopies - 1) * L.norm_copy);
    // the tag of every epoch is 31-bit and never 0 (the content of a zeroed workspace)
    const unsigned eps[] = {0u, 1u, 0x7FFFFFFEu, 0x7FFFFFFFu, 0x80000000u, 0xFFFFFFFFu};
    for (unsigned e : eps) {
      const uint32_t t = hs::tag_of_epoch(e);
      CHECK(t != 0 && (t & 0x80000000u) == 0);
    }
    CHECK(hs::tag_of_epoch(0xFFFFFFFFu) != hs::tag_of_epoch(0u));
  }
  std::printf(fails ? "layout check: %d failures\n" : "layout check: ok\n", fails);
  return fails ? 1 : 0;
}
