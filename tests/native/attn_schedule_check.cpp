// Host check of the attention launch's workgroup -> (query head, query block)
// map, compiled against the kernel source: over head layouts whose KV-head
// count does and does not divide the XCD count and query-block counts from 1
// to 200, every (head, block) pair is served by exactly one workgroup of the
// grid, padding workgroups are reported as such, each XCD serves only the query
// heads of its KV head (when the KV-head count divides 8), and along one XCD's
// list the blocks come longest causal rows first.  The key-split launch (a few
// query rows, one block) is checked per unit: each KV head once when packed,
// each query head once otherwise.  Prints "ok <cases>" or the first failure.
#include "../../paper_2609_30884_amd/csrc/attn_bf16.hip"

#include <cstdio>
#include <vector>

namespace crf {
namespace {

int fail(const char *what, int nq, int nkv, int nqb) {
  std::printf("FAIL %s (nq=%d nkv=%d nqb=%d)\n", what, nq, nkv, nqb);
  return 1;
}

int check_window(int nq, int nkv, int nqb) {
  int xcd_r = -1;
  const int grid = attn_window_grid(nq, nkv, nqb, xcd_r);
  if (xcd_r < 0 || (8 % nkv == 0) != (xcd_r > 0)) return fail("per-XCD order chosen", nq, nkv, nqb);
  const int group = nq / nkv;
  std::vector<int> cover((size_t)nq * nqb, 0);
  std::vector<int> last(8, 1 << 30);
  for (int bid = 0; bid < grid; ++bid) {
    int head = -1, qblk = -1;
    if (!attn_block(bid, nq, nkv, nqb, xcd_r, 0, head, qblk)) {
      if (xcd_r == 0) return fail("padding without the per-XCD order", nq, nkv, nqb);
      continue;
    }
    if (head < 0 || head >= nq || qblk < 0 || qblk >= nqb) return fail("head or block out of range", nq, nkv, nqb);
    ++cover[(size_t)head * nqb + qblk];
    if (xcd_r > 0) {
      const int x = bid % 8;
      if (head / group != x / xcd_r) return fail("XCD serves another KV head", nq, nkv, nqb);
      if (qblk > last[x]) return fail("longest rows first along an XCD", nq, nkv, nqb);
      last[x] = qblk;
    }
  }
  for (size_t i = 0; i < cover.size(); ++i)
    if (cover[i] != 1) return fail("(head, block) not served exactly once", nq, nkv, nqb);
  return 0;
}

int check_split(int nq, int nkv, int packed) {
  const int units = packed ? nkv : nq, group = nq / nkv;
  std::vector<int> cover(nq, 0);
  for (int bid = 0; bid < units; ++bid) {
    int head = -1, qblk = -1;
    if (!attn_block(bid, nq, nkv, 1, 0, packed, head, qblk) || qblk != 0 || head < 0 || head >= nq)
      return fail("key-split unit", nq, nkv, 1);
    for (int h = head; h < head + (packed ? group : 1); ++h) ++cover[h];
  }
  for (int h = 0; h < nq; ++h)
    if (cover[h] != 1) return fail("key-split head not served exactly once", nq, nkv, 1);
  return 0;
}

}  // namespace
}  // namespace crf

int main() {
  using namespace crf;
  const int layouts[][2] = {{28, 4}, {12, 2}, {4, 2}, {8, 2}, {12, 6}, {16, 8}, {14, 7}, {9, 3}, {28, 28}, {5, 5},
                            {6, 1}, {32, 8}, {40, 10}};
  int cases = 0;
  for (const auto &l : layouts) {
    for (int nqb = 1; nqb <= 200; ++nqb) {
      if (check_window(l[0], l[1], nqb)) return 1;
      ++cases;
    }
    for (int packed = 0; packed < 2; ++packed) {
      if (check_split(l[0], l[1], packed)) return 1;
      ++cases;
    }
  }
  std::printf("ok %d\n", cases);
  return 0;
}
