// Host-only check of the split-K workspace sizing against the dispatch
// heuristic, through the library's own workspace carving: for the block and
// LM-head shapes of every workload and reduction lengths up to the
// workspace's capacity, the split-K factor gemm() is given never needs more
// partial floats than the carved workspace holds (block: the four
// weight-gradient products; LM head: the full and the last group of vocab
// chunks, the width its weight-gradient product runs on).
// Built with the library sources included (host compilation only; nothing
// is launched).  Exit status 1 on a violation.
#include <cstdio>
#include <algorithm>
#include "loss.hip"
// the two sources each define these helpers in their own unnamed namespace
#define check_cfg block_check_cfg
#define carve_saved block_carve_saved
#include "block.hip"
#undef check_cfg
#undef carve_saved
using namespace aj;
int main() {
  struct C { const char *name; int d, Hq, Hkv, hd, F, V, chunk, cap; } cs[] = {
    {"tiny", 128, 4, 4, 32, 512, 1024, 1024, 131072},
    {"1.5b", 1536, 12, 2, 128, 8960, 151936, 32768, 131072},
    {"7b", 3584, 28, 4, 128, 18944, 152064, 32768, 131072},
    {"7b-8192", 3584, 28, 4, 128, 18944, 152064, 8192, 131072},
    {"32b", 5120, 40, 8, 128, 27648, 152064, 8192, 131072},
    {"32b-32768", 5120, 40, 8, 128, 27648, 152064, 32768, 131072},
  };
  int bad = 0;
  for (auto &c : cs) {
    aj_block_cfg b{};
    b.d_model = c.d; b.n_q_heads = c.Hq; b.n_kv_heads = c.Hkv; b.head_dim = c.hd; b.d_ff = c.F;
    b.dtype = AJ_BF16;
    aj_loss_cfg l{};
    l.d_model = c.d; l.vocab = c.V; l.vocab_chunk = c.chunk; l.dtype = AJ_BF16;
    const size_t blk = carve_bwd(b, c.cap, nullptr).splitk_floats;
    const size_t los = carve_ws(l, c.cap, nullptr).splitk_floats;
    const int q = (c.Hq + 2 * c.Hkv) * c.hd, hq = c.Hq * c.hd;
    int64_t gfull = 0, glast = 0;
    group_widths(l, &gfull, &glast);
    for (int K = 1; K <= c.cap; K += (K < 20000 ? 7 : 61)) {
      const int shp[4][2] = {{c.d, c.F}, {2 * c.F, c.d}, {c.d, hq}, {q, c.d}};
      for (auto &s : shp) {
        const int S = gemm_split_k(s[0], s[1], K);
        if (S > 1 && (size_t)S * s[0] * s[1] > blk) {
          if (++bad < 10) printf("block %s %dx%d K=%d S=%d\n", c.name, s[0], s[1], K, S);
        }
      }
      for (int cw : {(int)gfull, (int)glast}) {
        const int S = gemm_split_k(cw, c.d, K);
        if (S > 1 && (size_t)S * cw * c.d > los) {
          if (++bad < 10) printf("loss %s %dx%d K=%d S=%d\n", c.name, cw, c.d, K, S);
        }
      }
    }
    printf("%-10s block %zu floats, LM head %zu floats\n", c.name, blk, los);
  }
  printf("violations: %d\n", bad);
  return bad != 0;
}
