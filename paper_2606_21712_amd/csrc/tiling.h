// Tiling constants shared by the grouped GEMMs (device) and the workspace
// layout (host).  Plain C++: no HIP dependency.
#pragma once

namespace moe {

// Output tiles of the grouped GEMMs are 256 x 256 (GEMM-1: 256 rows x 128
// features of both gate and up).
constexpr int kTileRows = 256;
constexpr int kTileCols = 256;

// Tail split of the down projection.  A persistent grid of G workgroups runs
// n output tiles in ceil(n / G) rounds; the last holds only r = n mod G tiles.
// When r <= G / 2 each of those tiles is cut into s >= 2 pieces of consecutive
// k steps, at most kMaxTailPieces pieces in all, at most kMaxTailSplit per tile
// and at least kMinPieceSteps k steps each; a piece writes fp32 partial sums
// of its tile, and a reduction adds a tile's pieces in piece order.
constexpr int kMaxTailPieces = 256;
constexpr int kMaxTailSplit = 8;
constexpr int kMinPieceSteps = 8;

}  // namespace moe
