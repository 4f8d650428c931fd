// Host check of the persistent bf16 GEMM's work decomposition, compiled
// against the kernel source itself (the scheduler is host/device code there).
// For each shape: every (256x256 tile, 64-wide K slice) pair is computed by
// exactly one work item; whole tiles come first and K-parts split their tile's
// slices into consecutive, non-overlapping ranges; no workgroup repeats an
// item (also when odd workgroups take their last item first); and with a
// whole number of tiles per XCD, the tiles run by XCD x are the x-th
// contiguous eighth of the whole-tile range.
// Prints "ok <cases>" and exits 0, or prints the first failure and exits 1.
#include "../../paper_2609_30884_amd/csrc/gemm_bf16.hip"

#include <cstdio>
#include <cstdlib>
#include <set>
#include <vector>

namespace crf {
namespace {

int fail(const char *what, int M, int N, int K, int n_cu, int epi) {
  std::printf("FAIL %s (M=%d N=%d K=%d n_cu=%d epi=%d)\n", what, M, N, K, n_cu, epi);
  return 1;
}

int check(GemmEpi epi, int M, int N, int K, int n_cu, int64_t split_cap) {
  static float dummy;
  GemmParams p{};
  p.M = M;
  p.N = N;
  p.K = K;
  p.n_cu = n_cu;
  p.split_part = &dummy;
  p.split_cap = split_cap;
  const Sched sc = schedule(epi, p);
  const int tiles = sc.tiles_m * sc.tiles_n;
  if (sc.tiles_m != (M + BM - 1) / BM || sc.tiles_n != (N + BN - 1) / BN || sc.nk != K / BK)
    return fail("tile counts", M, N, K, n_cu, epi);
  if (sc.split_first < 0 || sc.split_first > tiles || sc.split_s < 1)
    return fail("split range", M, N, K, n_cu, epi);
  if (epi == EPI_SWIGLU && sc.split_s != 1) return fail("SwiGLU tiles are never split", M, N, K, n_cu, epi);
  if (sc.split_s > 1 && (int64_t)(tiles - sc.split_first) * sc.split_s * BM * BN > split_cap)
    return fail("partials exceed their buffer", M, N, K, n_cu, epi);
  if (sc.n_items != sc.split_first + (tiles - sc.split_first) * sc.split_s)
    return fail("item count", M, N, K, n_cu, epi);
  if (sc.grid < 1 || sc.grid > sc.n_items || (n_cu > 0 && sc.grid > n_cu))
    return fail("grid", M, N, K, n_cu, epi);
  std::vector<int> cover((size_t)tiles * sc.nk, 0);
  std::vector<int> seen(sc.n_items, 0);
  int total = 0;
  for (int b = 0; b < sc.grid; ++b) {
    std::set<int> mine;
    const int n = n_mine(sc, b);
    for (int i = 0; i < n; ++i) {
      const WorkItem it = work_item(sc, b, i);
      if (it.w < 0 || it.w >= sc.n_items) return fail("item index", M, N, K, n_cu, epi);
      if (!mine.insert(it.w).second) return fail("item repeated in a workgroup", M, N, K, n_cu, epi);
      ++seen[it.w];
      int tm, tn;
      tile_coords(it.t, sc.tiles_m, sc.tiles_n, tm, tn);
      if (tm != it.tm || tn != it.tn || tm < 0 || tm >= sc.tiles_m || tn < 0 || tn >= sc.tiles_n)
        return fail("tile coordinates", M, N, K, n_cu, epi);
      if ((it.part < 0) != (it.t < sc.split_first)) return fail("whole tiles before K-parts", M, N, K, n_cu, epi);
      if (it.part < 0 && (it.kb != 0 || it.ke != sc.nk)) return fail("whole tile K range", M, N, K, n_cu, epi);
      if (it.part >= 0 && (it.part >= sc.split_s || it.kb != it.part * sc.nk / sc.split_s ||
                           it.ke != (it.part + 1) * sc.nk / sc.split_s || it.kb >= it.ke))
        return fail("K-part range", M, N, K, n_cu, epi);
      for (int k = it.kb; k < it.ke; ++k) ++cover[(size_t)(tm * sc.tiles_n + tn) * sc.nk + k];
      ++total;
    }
  }
  if (total != sc.n_items) return fail("items over all workgroups", M, N, K, n_cu, epi);
  for (int w = 0; w < sc.n_items; ++w)
    if (seen[w] != 1) return fail("item not run exactly once", M, N, K, n_cu, epi);
  for (size_t i = 0; i < cover.size(); ++i)
    if (cover[i] != 1) return fail("tile slice not computed exactly once", M, N, K, n_cu, epi);
  // XCD shares of the whole tiles: workgroup b runs on XCD b % 8
  const int whole = sc.split_s > 1 ? sc.split_first : sc.n_items;
  if (sc.grid % 8 == 0 && whole % 8 == 0 && whole > 0) {
    for (int b = 0; b < sc.grid; ++b)
      for (int i = 0; i < n_mine(sc, b); ++i) {
        const WorkItem it = work_item(sc, b, i);
        if (it.part >= 0) continue;
        const int x = b % 8;
        if (it.t < x * (whole / 8) || it.t >= (x + 1) * (whole / 8)) return fail("XCD share", M, N, K, n_cu, epi);
      }
  }
  return 0;
}

}  // namespace
}  // namespace crf

int main() {
  using namespace crf;
  struct Shape {
    int M, N, K;
  };
  std::vector<Shape> shapes = {
      // 7B window projections: QKV, O, gate/up, down
      {16384, 4608, 3584}, {16384, 3584, 3584}, {16384, 37888, 3584}, {16384, 3584, 18944},
      // 1.5B window projections
      {4096, 2048, 1536}, {4096, 1536, 1536}, {4096, 17920, 1536}, {4096, 1536, 8960},
      // ragged and small
      {333, 4608, 3584}, {1, 256, 64}, {257, 257, 128}, {1000, 700, 512}, {2048, 1536, 8960}, {300, 1024, 640},
  };
  std::srand(7);
  for (int r = 0; r < 200; ++r)
    shapes.push_back({1 + std::rand() % 9000, 1 + std::rand() % 6000, 64 * (1 + std::rand() % 120)});
  int cases = 0;
  for (const Shape &s : shapes)
    for (GemmEpi epi : {EPI_QKV, EPI_RESID, EPI_SWIGLU})
      for (int n_cu : {256, 80, 8, 0})
        for (int64_t cap : {(int64_t)1 << 40, (int64_t)64 << 20}) {
          if (check(epi, s.M, s.N, s.K, n_cu, cap)) return 1;
          ++cases;
        }
  std::printf("ok %d\n", cases);
  return 0;
}
