// Work-list orders of the tiled launches (host side).  The order in which
// tiles are dispatched decides which operand panels are shared through the
// caches, so it is part of a kernel's measured HBM traffic.
#pragma once

#include <algorithm>
#include <cstdint>
#include <utility>
#include <vector>

#include "internal.h"

namespace orth {

// Reorders a logical work list so that physical block p (dispatched to XCD
// p % 8) gets consecutive logical items: XCD x owns one contiguous chunk.
template <typename T>
inline std::vector<T> xcd_order(const std::vector<T>& logical) {
  const size_t n = logical.size();
  std::vector<T> phys(n);
  size_t start = 0;
  for (size_t x = 0; x < 8; ++x) {
    const size_t cnt = n > x ? (n - x + 7) / 8 : 0;
    for (size_t slot = 0; slot < cnt; ++slot) phys[x + 8 * slot] = logical[start + slot];
    start += cnt;
  }
  return phys;
}

// Tiles of a tr x tc grid in groups of `gm` tile rows (column-major inside a
// group), so concurrently running tiles share operand panels.
inline void grouped_tiles(int mat, int tr, int tc, int gm, bool upper_only, std::vector<TileItem>& out) {
  for (int r0 = 0; r0 < tr; r0 += gm) {
    const int r1 = std::min(tr, r0 + gm);
    for (int j = 0; j < tc; ++j)
      for (int i = r0; i < r1; ++i)
        if (!upper_only || i <= j) out.push_back(TileItem{mat, i, j, 0});
  }
}

// The Gram (upper tiles) and update work lists of one matrix of a bf16 tile
// class, tn x tn and tm x tn tiles.  The lists are dispatched in this order
// itself (block b runs on XCD b % 8), so all XCDs work on the same matrix
// and its operand panels are shared through the memory-side cache; measured
// 7% faster for update launches than giving each XCD its own contiguous
// chunk of matrices.
inline void bf16_matrix_tiles(int mat, int tm, int tn, std::vector<TileItem>& gram, std::vector<TileItem>& upd) {
  grouped_tiles(mat, tn, tn, 4, true, gram);
  grouped_tiles(mat, tm, tn, 4, false, upd);
}

// Size class of the bf16 tiles: matrices with N >= 1024 use 256 x 256 tiles
// only when those tiles fill at least four waves of the 256 compute units
// (update tiles of the whole batch); otherwise the 128 x 128 tiles keep more
// units busy (measured on the ImageNet-like stack: 8 x 1024^2 + 4 x 2048^2
// gives 384 update tiles of 256, 1536 of 128).
constexpr int64_t kBigTileMinTiles = 4 * 256;
inline bool use_big_tiles(const std::vector<std::pair<int, int>>& tall_dims, int forced = 0) {
  if (forced) return forced == 256;
  int64_t tiles = 0;
  for (const auto& d : tall_dims)
    if (d.second >= 1024) tiles += (int64_t)((d.first + 255) / 256) * ((d.second + 255) / 256);
  return tiles >= kBigTileMinTiles;
}

}  // namespace orth
