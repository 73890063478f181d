// Epilogue modes of the convolution kernels and the chunk-mode row tiling,
// shared by the planner, the executor and the kernels.
#pragma once

namespace st {

// State: P += dP in place, emit f(P_new) - f(P_old).  Defer: write the f32
// update rows (applied later).  Linear: emit dP itself.  ChunkState (chunk
// mode, rows grouped by site in frame order, tiles aligned to those runs):
// walk each site's frames in order with the state in registers and emit
// every frame's f(P_t) - f(P_{t-1}).  StateOnly (dense reference pass of a
// layer whose emitted rows come from elsewhere -- a pool -- or go nowhere --
// the net's output): store P, emit nothing.  ChunkPool (chunk mode, a
// max-pooled layer, tiles as for ChunkState): walk each site's frames in
// order and write every frame's state P_t to the row's update row, and
// the frames that updated the site to a bit mask; the pool emission reads
// them and the commit stores the last state.
enum {
  kModeState = 0,
  kModeDefer = 1,
  kModeLinear = 2,
  kModeChunkState = 3,
  kModeStateOnly = 4,
  kModeChunkPool = 5
};

constexpr bool chunk_tiled(int mode) {
  return mode == kModeChunkState || mode == kModeChunkPool;
}

// Rows per tile step of the run-aligned tiling: a tile starts at the first
// row of the site run that holds row j * step, so with runs of at most nf
// rows (nf <= 32) no tile exceeds 64 rows and none is empty.
constexpr int chunk_tile_step(int nf) { return 65 - nf; }

// Tiles of one compaction pass at most (the look-back statuses of a set;
// compactions alternate between two sets).
constexpr int kCompactMaxTiles = 4096;

// Partial counters per layer for the sites a chunk's fused epilogue
// updated (blocks add to slot blockIdx % kSiteSlots; the host sums them).
constexpr int kSiteSlots = 8;

}  // namespace st
