// Internal plan of a diff-computation net: shapes, workspace layout and
// host-side state shared by the planner (st_plan.cpp) and the executor
// (st_exec.hip).  Not part of the public ABI.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <utility>
#include <vector>

#include "../../include/sparsetem.h"
#include "st_modes.h"

namespace st {

constexpr int kChanAlign = 8;       // delta rows / weights padded to 8 channels
constexpr int kMaxChunkFrames = 32; // diff frames per chunk (frame bit masks)
constexpr int kChunkMaxInC = 16;    // input channels of a chunk's frame scan
constexpr int kMaxTiles = kCompactMaxTiles;  // compaction tiles per pass
constexpr int64_t kMaxGrid = (int64_t)kMaxTiles * 8192;  // sites per grid
constexpr size_t kAlign = 256;      // workspace sub-buffer alignment

// Squeeze-excitation row mapping: each site is handled by a power-of-two
// group of threads (at most one wave), each thread owning 8-channel vectors;
// a 256-thread block covers 256 / tps sites side by side.  The squeeze
// splits each image into about kSePartialFloats / cp site ranges (4..256),
// so that the partial sums one excitation block reduces stay near
// kSePartialFloats floats.
// Reduction splits of the gather-GEMM: a layer with at least
// kSplitMinLayerStages reduction stages may split each output tile into up
// to stages / 8 (at most kSplitMax) parts when a frame has few tiles.
constexpr int kSplitMinLayerStages = 32;
constexpr int kSplitMax = 8;

constexpr int kSeMaxChannels = 2048;
constexpr int kSePartialFloats = 16384;
inline int se_threads_per_site(int cp) {
  int t = 1;
  while (t < cp / 8 && t < 64) t <<= 1;
  return t;
}

inline int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Counter block layout (uint64 each).
struct CounterIdx {
  int rows;   // candidate rows of a tensor / affected outputs of a layer
  int act;    // kept rows of a tensor
  int pairs;  // rulebook pairs of a layer
};

// An emitted delta tensor: t = 0 is the frame delta, t = j + 1 is layer j's
// output (after its pool, if any).
struct TensorPlan {
  int N = 0, H = 0, W = 0, C = 0, Cp = 0;
  int64_t grid = 0;                 // N*H*W
  size_t off_rows = 0;              // storage dtype [grid][Cp]
  size_t off_rowpix = 0;            // int32 [grid]  row -> pixel (ascending)
  size_t off_act = 0;               // int32 [grid]  kept pixels (ascending)
  size_t off_map = 0;               // int32 [grid]  pixel -> row or -1
  size_t off_rowmax = 0;            // uint32 [grid] bits of max|delta| per row
  int cnt_rows = 0, cnt_act = 0;    // counter indices
  float last_thr = 0.f;             // threshold used by the last encode
  // layers reading this tensor: (layer, 0 = as conv input, 1 = as residual)
  std::vector<std::pair<int, int>> consumers;
};

struct LayerPlan {
  st_layer_desc d{};
  int Hi = 0, Wi = 0, Ho = 0, Wo = 0, Hp = 0, Wp = 0;
  int K = 0, cin_p = 0, cout_p = 0;
  int64_t ktot = 0, ktot_p = 0;     // K*cin_p and its padding to the GEMM chunk
  int64_t conv_grid = 0;            // N*Ho*Wo
  bool stateful = false, pool = false, dw = false, ident = false;
  bool se = false;                  // squeeze-excitation after the act
  int se_mid = 0, se_chunk = 0, se_nchunk = 0, se_tps = 0;
  int mode = 0;                     // epilogue mode (kMode*, st_kernels.h)
  int split_max = 1;                // most reduction splits per output tile
  // workspace offsets
  size_t off_P = 0;                 // f32 [conv_grid][cout_p]
  size_t off_O = 0;                 // int32 [conv_grid] affected conv outputs
  size_t off_Mo = 0;                // int32 [conv_grid] pixel -> O index
  size_t off_nbr = 0;               // int32 [K][conv_grid]
  size_t off_dP = 0;                // f32 [conv_grid][cout_p] (pooled layers)
  size_t off_w = 0;                 // GEMM: dtype [cout_p][ktot_p]; dw: f32 [K][cout_p]
  size_t off_bias = 0;              // f32 [cout_p]
  size_t off_sew1 = 0, off_seb1 = 0, off_sew2 = 0, off_seb2 = 0;  // f32
  size_t off_ses = 0;               // f32 [2][N][cout_p] gates, two slots
  size_t off_sesum = 0;             // f64 [N][cout_p] channel sums of f(P)
  size_t off_separt = 0;            // f32 [N][se_nchunk][cout_p]
  size_t off_flags = 0;             // uint8 [conv_grid] affected-output flags
  size_t off_pflags = 0;            // uint8 [pooled grid] (pooled layers)
  int cnt_O = 0, cnt_pairs = 0;
  size_t off_yhat = 0;              // residual carry: f32 [out grid][cout_p]
  int cnt_sites = 0;                // chunk mode: sites whose state a fused
                                    // GEMM updated (site runs)
  size_t off_tstart = 0;            // chunk mode: uint32 run-aligned GEMM
                                    // row tiles (fused-state layers)
  int64_t dense_pairs = 0;          // rulebook pairs with every pixel active
};

struct Recorder;  // executor-side profiling state

}  // namespace st

struct st_net {
  int dtype = 0, esize = 4;
  int N = 0, H = 0, W = 0, C = 0;
  int F = 1;                               // diff frames per chunk (capacity)
  int last_nf = 1;                         // frames of the last encode
  std::vector<st::LayerPlan> layers;
  std::vector<st::TensorPlan> tensors;     // n_layers + 1
  size_t ws_bytes = 0;
  size_t off_xhat = 0;                     // storage dtype [N*H*W*C]
  size_t off_flags = 0;                    // uint8 [input grid] keep bytes
  size_t off_tiles = 0;                    // uint32 [2][kMaxTiles] statuses
  int cpar = 0;                            // status set of the next compaction
  size_t off_zero = 0;                     // 256 zero bytes
  size_t off_part = 0;                     // f32 split partials (shared)
  // online threshold adjustment, per produced tensor
  size_t off_ibst_theta = 0, off_ibst_lo = 0, off_ibst_hi = 0;  // f64
  size_t off_ibst_thr = 0;                 // f32 thresholds the kernels read
  size_t off_ibst_ctl = 0;                 // uint8 controlled flags
  size_t off_ibst_sites = 0;               // int64 sites per tensor
  bool ibst_on = false;
  bool carry = false;                      // residual-carry semantics
  bool frozen_se = false;                  // frozen squeeze-excitation gates
  bool bf16_state = false;                 // pre-activation state in bf16
  bool has_se = false;                     // any squeeze-excitation layer
  size_t off_se_par = 0;                   // int: gate slot of the last gates
  double ibst_target = 0.9, ibst_eps = 0.025, ibst_theta_max = 1.0;
  // a cycle spans this many reference frames; reference frames seen since
  // the control was set
  int ibst_cycle_refs = 1;
  int64_t ibst_refs = 0;
  // chunk mode (F > 1): f32 deferred updates of the current layer (shared),
  // per input item the frame whose value X_hat held (0xFF: the X_hat of
  // the chunk's start), per input site the last kept frame, per conv site
  // the frames that updated it (bit mask)
  size_t off_chunk_dp = 0, off_chunk_base = 0, off_chunk_last = 0;
  size_t off_chunk_aff = 0;
  // chunk mode, exact squeeze-excitation: per-frame squeeze partials
  // [F][N][nchunk][cp] and per-frame gates [F][N][cp] (shared by the
  // layers, sized for the largest)
  size_t off_chunk_separt = 0, off_chunk_gates = 0;
  size_t off_cnt = 0;                      // uint64 [n_counters]
  size_t off_cleanup = 0;                  // cleanup descriptor table
  // dense reference pass (nets without squeeze-excitation or residual
  // carry): the counters a reference frame leaves (uint64 [n_counters]),
  // each layer's dense rulebook pair count, and the {offset, length} table
  // of the kept lists it writes as identities
  bool dense_ref = false;
  size_t off_refcnt = 0, off_iota = 0;
  size_t off_dens = 0;                     // uint64 [batch] per-image counts
  int n_counters = 0;
  int n_cleanup = 0;
  int n_iota = 0;
  int64_t max_grid = 0;
  // runtime
  char* ws = nullptr;
  bool bound = false, have_ref = false;
  // bound to the library's static workspace on device static_dev (-1: a
  // caller's workspace) as its static_gen-th binding there
  int static_dev = -1;
  uint64_t static_gen = 0;
  void* last_stream = nullptr;
  std::string err;
  st::Recorder* rec = nullptr;
};

namespace st {
st_status fail(st_net* net, st_status s, const std::string& msg);
}
