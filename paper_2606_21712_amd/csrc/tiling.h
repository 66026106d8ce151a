// Tiling constants shared by the grouped GEMMs (device) and the workspace
// layout (host).  Plain C++: no HIP dependency.
#pragma once

namespace moe {

// Output tiles of the grouped GEMMs are m-tiles of an expert's rows x 256
// columns (GEMM-1: 128 features of both gate and up).  The bf16 GEMMs cut an
// expert of c rows into ceil(c / kTileRowsMax) m-tiles whose edges fall on
// 32-row blocks, the blocks shared out evenly, so every m-tile holds up to
// kTileRowsMax rows and only the expert's last block is partly filled.  The
// MXFP8 GEMMs cut it into m-tiles of kTileRows rows, the last one shorter.
constexpr int kTileRows = 256;
constexpr int kTileCols = 256;
constexpr int kTileRowsMax = 320;
constexpr int kTileRowBlock = 32;

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
