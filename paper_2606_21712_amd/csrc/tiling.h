// Tiling constants shared by the grouped GEMMs (device) and the workspace
// layout (host).  Plain C++: no HIP dependency.
#pragma once

namespace moe {

// Output tiles of the grouped GEMMs are 256 x 256 (GEMM-1: 256 rows x 128
// features of both gate and up).  An expert's rows are cut into m-tiles of
// kTileRows; in the bf16 GEMMs the last one may hold up to kTileRows +
// kTileExtraRows rows, so that a remainder of at most kTileExtraRows rows joins
// the tile before it instead of costing a tile of its own.
constexpr int kTileRows = 256;
constexpr int kTileCols = 256;
constexpr int kTileExtraRows = 64;
constexpr int kTileRowsMax = kTileRows + kTileExtraRows;

// Tail split of the down projection.  A persistent grid of G workgroups runs
// n output tiles in ceil(n / G) rounds; the last holds only r = n mod G tiles.
// When r <= G / 2 each of those tiles is cut into s >= 2 pieces of consecutive
// k steps, at most kMaxTailPieces pieces in all, at most kMaxTailSplit per tile
// and at least kMinPieceSteps k steps each; a piece writes fp32 partial sums
// of its tile, and a reduction adds a tile's pieces in piece order.
constexpr int kMaxTailPieces = 256;
constexpr int kMaxTailSplit = 8;
constexpr int kMinPieceSteps = 8;

// moe_permute_static keeps its per-expert counts of blocks of assignments (the
// moe_permute workspace) in a static device array of this size instead of a
// caller workspace: calls whose moe_permute_workspace_bytes() exceeds it are refused.
constexpr unsigned long kPermuteStaticScratchBytes = 4ul << 20;

}  // namespace moe
