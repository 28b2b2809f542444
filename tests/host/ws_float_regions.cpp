// Host-only helper of the workspace tests: prints the byte ranges of the
// floating-point regions of mita_backward's (which = 0) or mita_forward's
// (which = 1) workspace, one "kind begin end" line each (kind f32 or io, the
// io type), for the configuration given on the command line:
//   B H grid_h grid_w d lm_h lm_w k use_shared use_routed dtype(0 fp32, 1 bf16) s which
#include <cstdio>
#include <cstdlib>

#include "../../paper_2602_01219_amd/csrc/check.hpp"

int main(int argc, char **argv) {
  if (argc != 14) return 2;
  mita_cfg_t c{};
  c.B = atoi(argv[1]); c.H = atoi(argv[2]); c.grid_h = atoi(argv[3]); c.grid_w = atoi(argv[4]);
  c.N = c.grid_h * c.grid_w; c.d = atoi(argv[5]); c.lm_h = atoi(argv[6]); c.lm_w = atoi(argv[7]);
  c.M = c.lm_h * c.lm_w; c.k = atoi(argv[8]); c.use_shared = atoi(argv[9]); c.use_routed = atoi(argv[10]);
  c.dtype = atoi(argv[11]) ? MITA_BF16 : MITA_F32; c.s = atoi(argv[12]); c.scale = 0.f; c.flags = 0;
  const bool fwd = atoi(argv[13]) != 0;
  std::string err;
  if (mita::check_cfg(&c, &err) != MITA_OK) return 3;
  const mita::BwdLayout L = mita::backward_layout(c);
  const mita::FwdLayout &F = L.f;
  if (fwd) {
    // landmark rows and expert tiles (io type), score rows and partials,
    // the pairs' partial outputs and log-sum-exps (s > 1)
    std::printf("io %zu %zu\n", F.q_lm, F.scores);
    std::printf("f32 %zu %zu\n", F.scores, F.idx);
    std::printf("io %zu %zu\n", F.kx, F.expert);
    std::printf("f32 %zu %zu\n", F.pair_o, F.plo);
    std::printf("total %zu\n", F.total);
    return 0;
  }
  // [begin, end) of each float region: the score rows and partials, and the
  // backward's accumulators, log-sum-exps and staging rows, which lie
  // between lse_lm and the inverse index
  std::printf("f32 %zu %zu\n", F.scores, F.idx);
  std::printf("f32 %zu %zu\n", L.lse_lm, L.inv_start);
  std::printf("f32 %zu %zu\n", L.D_lm, L.total);
  std::printf("io %zu %zu\n", F.q_lm, F.scores);
  std::printf("total %zu\n", L.total);
  return 0;
}
