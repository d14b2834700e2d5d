// Exact-cover checks of the tiled launches' work lists (tile_order.h), run on
// the CPU: every upper tile (i <= j) of every matrix appears exactly once in
// a Gram list (bf16, and the fp32 grouped upper list), every tile once in an
// update list, and the XCD reordering is a permutation.  Prints "ok <n>" per
// case and "FAIL ..." otherwise.
#include <cstdio>
#include <map>
#include <random>
#include <tuple>
#include <vector>

#include "../../paper_2601_13776_amd/csrc/tile_order.h"

namespace {
int g_fail = 0;

void fail(const char* what, int c) {
  std::printf("FAIL case %d: %s\n", c, what);
  ++g_fail;
}

void check_gram(const std::vector<std::pair<int, int>>& mats, int gp, int c) {
  std::vector<orth::TileItem> out = orth::bf16_gram_tiles(mats, gp);
#ifdef PLANT_MISTAKE
  // the checks' own check: a list with its last tile dealt twice must fail
  if (!out.empty()) out.push_back(out.back());
#endif
  std::map<std::tuple<int, int, int>, int> seen;
  for (const auto& t : out) ++seen[std::make_tuple(t.mat, t.ti, t.tj)];
  size_t want = 0;
  for (const auto& m : mats) {
    for (int j = 0; j < m.second; ++j)
      for (int i = 0; i <= j; ++i)
        if (seen[std::make_tuple(m.first, i, j)] != 1) return fail("Gram tile missing or repeated", c);
    want += (size_t)m.second * (m.second + 1) / 2;
  }
  if (out.size() != want) return fail("Gram list holds tiles outside the upper triangles", c);
  for (const auto& t : out)
    if (t.flags != 0) return fail("Gram item with flags set", c);
  std::printf("ok %d\n", c);
}

void check_update(int mat, int tm, int tn, int c) {
  std::vector<orth::TileItem> out;
  orth::bf16_update_tiles(mat, tm, tn, out);
  std::map<std::pair<int, int>, int> seen;
  for (const auto& t : out) {
    if (t.mat != mat || t.ti < 0 || t.ti >= tm || t.tj < 0 || t.tj >= tn) return fail("update tile out of range", c);
    ++seen[{t.ti, t.tj}];
  }
  if (out.size() != (size_t)tm * tn || seen.size() != (size_t)tm * tn) return fail("update tile missing or repeated", c);
  std::printf("ok %d\n", c);
}

// the fp32 Gram list: grouped tiles of the upper triangle
void check_grouped_upper(int tn, int gm, int c) {
  std::vector<orth::TileItem> out;
  orth::grouped_tiles(5, tn, tn, gm, true, out);
  std::map<std::pair<int, int>, int> seen;
  for (const auto& t : out) {
    if (t.mat != 5 || t.ti > t.tj || t.tj >= tn || t.ti < 0) return fail("grouped upper tile out of range", c);
    ++seen[{t.ti, t.tj}];
  }
  if (out.size() != (size_t)tn * (tn + 1) / 2 || seen.size() != out.size())
    return fail("grouped upper tile missing or repeated", c);
  std::printf("ok %d\n", c);
}

void check_xcd(size_t n, int c) {
  std::vector<int> v(n);
  for (size_t i = 0; i < n; ++i) v[i] = (int)i;
  const std::vector<int> p = orth::xcd_order(v);
  std::vector<int> cnt(n, 0);
  for (int x : p) {
    if (x < 0 || (size_t)x >= n) return fail("xcd_order value out of range", c);
    ++cnt[x];
  }
  for (int k : cnt)
    if (k != 1) return fail("xcd_order is not a permutation", c);
  std::printf("ok %d\n", c);
}
}  // namespace

int main() {
  int c = 0;
  // the workloads' tile columns: the stress batch on 256-tiles, the
  // ImageNet-like stack on 128-tiles, and edge cases
  {
    std::vector<std::pair<int, int>> m(64);
    for (int i = 0; i < 64; ++i) m[i] = {i, 16};
    check_gram(m, 4, ++c);
  }
  check_gram({{0, 16}, {1, 16}, {2, 16}, {3, 16}, {4, 8}, {5, 8}, {6, 4}, {7, 2}, {8, 1}}, 4, ++c);
  check_gram({{0, 1}}, 4, ++c);
  check_gram({{0, 5}, {1, 3}, {2, 7}}, 4, ++c);
  check_gram({{0, 9}, {1, 1}}, 3, ++c);
  std::mt19937 rng(7);
  for (int r = 0; r < 50; ++r) {
    std::vector<std::pair<int, int>> m(1 + rng() % 12);
    for (size_t i = 0; i < m.size(); ++i) m[i] = {(int)i, 1 + (int)(rng() % 20)};
    check_gram(m, 1 + (int)(rng() % 5), ++c);
    check_update((int)(rng() % 9), 1 + (int)(rng() % 24), 1 + (int)(rng() % 24), ++c);
    check_xcd(rng() % 300, ++c);
    check_grouped_upper(1 + (int)(rng() % 40), 1 + (int)(rng() % 6), ++c);
  }
  check_update(3, 16, 16, ++c);
  check_update(0, 1, 1, ++c);
  check_xcd(0, ++c);
  check_xcd(8704, ++c);
  std::printf("cases %d failures %d\n", c, g_fail);
  return g_fail ? 1 : 0;
}
