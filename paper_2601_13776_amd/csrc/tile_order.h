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

// The update work list of one matrix of a bf16 tile class (tm x tn
// tiles).  The list is dispatched in this order itself (block b runs on
// XCD b % 8), so all XCDs work on the same matrix and its operand panels
// are shared through the memory-side cache, while each XCD's concurrent
// tiles cover 4 tile rows x 8 tile columns (12 operand panels for 32
// tiles); measured 7% faster than giving each XCD its own contiguous chunk
// of matrices.
inline void bf16_update_tiles(int mat, int tm, int tn, std::vector<TileItem>& upd) {
  grouped_tiles(mat, tm, tn, 4, false, upd);
}

// The Gram (upper-tile) work list of a batch of matrices of one bf16 tile
// class, for a launch whose blocks are dealt to the 8 XCDs round-robin.
// Tile (I, J) reads column panels I and J of the iterate, so every matrix's
// upper tiles are cut into chunks of panel blocks: blocks of gp panels,
// a diagonal pair of blocks holding gp (gp + 1) / 2 tiles on gp panels, an
// off-diagonal pair gp^2 tiles on 2 gp panels.  Each chunk goes whole to
// the XCD with the fewest tiles so far (matrices in the given order,
// largest chunks first), and the XCD queues are dealt round-robin into the
// physical order: the compute units of one XCD run neighbouring chunks of
// one matrix, whose few panels its L2 serves, and all XCDs stay on the
// same matrices, whose panels the memory-side cache serves.  `mats` holds
// (matrix index, tile columns) in dispatch order.
inline std::vector<TileItem> bf16_gram_tiles(const std::vector<std::pair<int, int>>& mats, int gp = 4) {
  std::vector<TileItem> q[8];
  for (const auto& m : mats) {
    const int mat = m.first, tn = m.second;
    std::vector<std::vector<TileItem>> chunks;
    for (int p0 = 0; p0 < tn; p0 += gp)
      for (int q0 = p0; q0 < tn; q0 += gp) {
        std::vector<TileItem> c;
        for (int j = q0; j < std::min(tn, q0 + gp); ++j)
          for (int i = p0; i < std::min(tn, p0 + gp); ++i)
            if (i <= j) c.push_back(TileItem{mat, i, j, 0});
        chunks.push_back(std::move(c));
      }
    std::stable_sort(chunks.begin(), chunks.end(),
                     [](const std::vector<TileItem>& a, const std::vector<TileItem>& b) { return a.size() > b.size(); });
    for (auto& c : chunks) {
      int x = 0;
      for (int y = 1; y < 8; ++y)
        if (q[y].size() < q[x].size()) x = y;
      q[x].insert(q[x].end(), c.begin(), c.end());
    }
  }
  // deal the queues: block 8 k + x takes the k-th tile of XCD x's queue;
  // past the end of the shortest queues the rest follow round-robin
  std::vector<TileItem> out;
  size_t total = 0, longest = 0;
  for (auto& v : q) {
    total += v.size();
    longest = std::max(longest, v.size());
  }
  out.reserve(total);
  for (size_t k = 0; k < longest; ++k)
    for (int x = 0; x < 8; ++x)
      if (k < q[x].size()) out.push_back(q[x][k]);
  return out;
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
