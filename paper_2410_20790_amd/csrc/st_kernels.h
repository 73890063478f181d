// Launch interface of the gfx950 kernels of the diff-computation path.
// Each launcher enqueues one kernel on `s`; counts that depend on the frame
// live in device memory (uint64 counters), so no launcher reads data back
// and the per-frame launch sequence is fixed.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "st_modes.h"

namespace st {

struct Geo {  // sliding-window geometry from an input grid to an output grid
  int Hi, Wi, Ho, Wo, kh, kw, sh, sw, ph, pw;
};

struct CleanEntry {  // map[list[r]] = -1 for r < counter[cnt]
  int64_t map_off, list_off;
  int32_t cnt, pad;
  int64_t pad2;
};

using u64 = unsigned long long;

// Profiling hook (defined by the executor): records an event pair around
// a launch when recording is enabled.
struct Prof {
  void* net;
  int layer;
};
void prof_begin(const Prof& p, int cls, hipStream_t s);
void prof_end(const Prof& p, int cls, hipStream_t s);

// ---- per-frame bookkeeping
// counters to zero, and the first look-back status set (kCompactMaxTiles)
void launch_reset(const Prof& pf, hipStream_t s, u64* cnt, int n,
                  uint32_t* status);
// dense reference pass: the frame's rows (pixel-ordered, padded to Cp
// channels) and X_hat = frame; identity kept lists of the tensors (a table
// of {list offset, length} in the workspace); the frame's counters from a
// precomputed block
void launch_dense_input(const Prof& pf, hipStream_t s, int dtype,
                        const void* x, void* xhat, void* rows, int C, int Cp,
                        int64_t npix);
struct IotaEntry {  // list[r] = r for r < n
  int64_t off, n;
};
void launch_iota_lists(const Prof& pf, hipStream_t s, const IotaEntry* tab,
                       int n_tab, char* ws, int64_t max_n);
void launch_copy_u64(hipStream_t s, u64* dst, const u64* src, int n);
// dense max-pool emission of the reference pass: pooled row q (pixel
// order) = max over the window of f(P) (the state of the conv grid)
void launch_pool_dense(const Prof& pf, hipStream_t s, int dtype,
                       const float* P, int p16, void* dout, Geo g, int cp,
                       int act, int64_t nq);
void launch_cleanup(const Prof& pf, hipStream_t s, const CleanEntry* tab,
                    int n_tab, char* ws, const u64* cnt, int64_t max_rows);

// ---- consumer-side rulebook preparation (done while a tensor's kept rows
// are emitted)
enum { kConsNone = 0, kConsIdent = 1, kConsMark = 2, kConsMarkSame = 3 };
constexpr int kMaxCons = 4;
struct Cons {
  int kind;
  int* O;             // ident: affected list, map, one-entry neighbour table
  int* Mo;
  int* nbr;
  uint32_t* rowmax;   // ident: row maxima of the consumer's output to clear
  u64* cnt_O;
  u64* pairs;
  uint8_t* flags;     // mark: the consumer's affected-output flags,
                      // site-major (site * nf + frame)
  Geo g;              // mark: the consumer's window geometry
  int nf, nimg;       // mark / ident: frames of the pass, images per frame
  int64_t per;        // mark-same / ident: sites per frame
  // ident, chunk mode: the consumer's run-aligned GEMM row tiles (as
  // launch_run_tiles writes them), cut by the list compaction, or NULL
  uint32_t* tstart;
};
struct ConsList {
  Cons c[kMaxCons];
  int n;
};

// ---- (a) subtraction + truncation + compaction of the frame delta
struct ScanArgs {
  const void* x;
  void* xhat;
  int C, Cp;
  int64_t npix;
  float thr;
  const float* thr_dev;  // threshold in device memory (or NULL: thr)
  int ref;
  uint32_t* tiles;     // look-back statuses of the compaction
  uint32_t* tiles_clear;  // the other status set, cleared for the next one
  void* rows;
  int* rowpix;
  int* act;
  int* map;
  u64* cnt_rows;
  u64* cnt_act;
  ConsList cons;
};
void launch_scan(const Prof& pf, hipStream_t s, int dtype, const ScanArgs& a);

// ---- (b) rulebook: affected-output compaction with the neighbour table
struct FlagArgs {
  uint8_t* flags;
  int64_t npix;       // sites of the output grid
  uint32_t* tiles;
  uint32_t* tiles_clear;
  int* list;
  int* map;
  uint32_t* rowmax;   // or NULL
  int* nbr;           // or NULL (pool windows)
  const int* map_in;
  int64_t stride;
  Geo g;
  u64* pairs;
  u64* cnt;
  // chunk mode: nf frames of `per` sites each (item = frame * per + site);
  // items are compacted site-major (a site's frames adjacent, in frame
  // order).  nf <= 1: item order.
  int nf;
  int64_t per;
  // chunk mode, or NULL: the emitted list's run-aligned GEMM row tiles (as
  // launch_run_tiles writes them); the pass's tiles then hold whole sites,
  // which needs compact_runs_fit(npix, nf)
  uint32_t* tstart;
};
bool compact_runs_fit(int64_t cap, int run);
void launch_flag_compact(const Prof& pf, int cls, hipStream_t s,
                         const FlagArgs& a);
// flags: site-major (site * nf + frame) over nf frames of nimg images.
void launch_mark(const Prof& pf, int cls, hipStream_t s, const int* list,
                 const u64* n_list, int64_t max_items, Geo g, uint8_t* flags,
                 int nimg, int nf);
// Run-aligned row tiles of a site-major affected list O (chunk mode):
// tstart[j] = first row of the run (same site) holding row j * step, for
// j < ceil(nO / step), and tstart[ceil(nO / step)] = nO.
void launch_run_tiles(const Prof& pf, hipStream_t s, const int* O,
                      const u64* nO, int64_t capO, int64_t per, int nf,
                      uint32_t* tstart);

// ---- (c)+(d) delta convolution with the fused state update / emission
// Most splits of one reduction (the split epilogue requests them all at
// once).
constexpr int kEpiSplits = 8;
struct ConvArgs {
  int p16;             // state stored as bf16 (P points to bf16 values)
  const void* din;     // input delta rows [*, cin_p]
  const int* nbr;      // [K][stride] input row or -1
  int64_t stride;
  int K, cin_p, cout_p;
  int64_t ktot_p;
  const void* w;       // GEMM: [cout_p][ktot_p] storage dtype; dw: [K][cout_p] f32
  const float* bias;   // [cout_p]
  const int* O;        // affected output pixels (row -> pixel)
  const u64* nO;
  int64_t capO;
  float* P;            // [grid][cout_p] pixel-indexed state
  float* dP;           // [capO][cout_p] deferred update (pooled layers)
  void* dout;          // [capO][cout_p] emitted delta rows
  uint32_t* rowmax;    // [capO]
  const void* dskip;   // residual delta rows [*, cout_p] or NULL
  const int* mskip;    // residual pixel -> row map
  int mode, act, ref;
  float keep_thr;      // threshold of the emitted tensor
  const float* keep_thr_dev;  // in device memory (or NULL: keep_thr)
  const void* zero;    // 16 zero bytes (16-byte aligned)
  // split reduction: up to split_max splits of the reduction stages per
  // output tile (chosen per frame from the tile count), their f32 partial
  // tiles in part [split][capO][cout_p]; split_max = 1: no split;
  // split_max <= kEpiSplits
  float* part;
  int split_max;
  // residual carry: the consumers' view of the emitted tensor ([grid]
  // [cout_p] f32, pixel-indexed) or NULL; diff-pass state-mode emissions
  // are f(P_new) - view instead of f(P_new) - f(P_old)
  const float* yhat;
  // kModeChunkState: row tile j is [tstart[j], tstart[j + 1]) (tiles step
  // chunk_tile_step(nf) rows); a row's site is its item modulo `per`; the
  // number of runs (distinct sites) is added to sites[0 .. kSiteSlots)
  // (partial counts)
  const uint32_t* tstart;
  u64* sites;
  int nf;
  int64_t per;
  // kModeChunkPool: per conv site, the frames that updated it (bit t)
  uint32_t* aff;
  // frozen squeeze-excitation: per-image gates [N][cout_p] scaling both
  // emitted values of a state-mode emission (image = site / gate_hw), or
  // NULL
  const float* gate;   // frozen gates: two slots [2][N][cout_p] (or NULL)
  const int* gpar;     // the slot in use (device parity word)
  int64_t gsz;         // floats per slot
  int64_t gate_hw;
  // dense reference pass: every conv output is a row (row = pixel, nO =
  // capO), every tensor's rows are pixel-ordered, so the neighbours follow
  // from the geometry g (input row of output o at offset k, or -1 in the
  // padding), the residual row of a pixel is the pixel itself, and no row
  // maximum is kept (rowmax NULL)
  int dense;
  Geo g;
};
// Returns false (and launches nothing) when a.zero is missing or misaligned.
bool launch_conv_gemm(const Prof& pf, hipStream_t s, int dtype,
                      const ConvArgs& a);
void launch_conv_dw(const Prof& pf, hipStream_t s, int dtype,
                    const ConvArgs& a);

// ---- non-linear post-op (max-pool) and state commit
struct PoolArgs {
  const int* Q;        // pooled rows -> pooled pixel
  const u64* nQ;
  int64_t capQ;
  Geo g;               // conv grid -> pooled grid (pool window)
  const float* P;
  const float* dP;
  const int* Mo;       // conv pixel -> O index or -1
  void* dout;
  uint32_t* rowmax;
  int cp, act, ref;
  const float* yhat;    // residual carry view (pooled grid) or NULL
};
void launch_pool_emit(const Prof& pf, hipStream_t s, int dtype,
                      const PoolArgs& a);
void launch_commit(const Prof& pf, hipStream_t s, const int* O, const u64* nO,
                   int64_t capO, float* P, const float* dP, int cp, int ref);

// ---- truncation of an emitted tensor (list-mode compaction)
struct ListArgs {
  const uint32_t* rowmax;
  const u64* n_rows;
  int64_t cap;
  float thr;
  const float* thr_dev;  // threshold in device memory (or NULL: thr)
  const int* rowpix;
  int* act;
  int* map;
  uint32_t* tiles;       // look-back statuses of the compaction
  uint32_t* tiles_clear;  // the other status set, cleared for the next one
  u64* cnt_act;
  ConsList cons;
};
void launch_list_compact(const Prof& pf, hipStream_t s, const ListArgs& a);

// ---- squeeze-excitation on a deferred layer
struct SeArgs {
  int p16;             // state stored as bf16
  const float* P;      // state [npix][cp] (updated in place by the emission)
  const float* dP;     // deferred update rows
  const int* Mo;       // site -> dP row or -1 (every site in the reference)
  float* part;         // [N][nchunk][cp] partial sums of this frame's change
  double* S;           // [N][cp] channel sums of f(P), kept across frames
  const float* w1;     // [mid][cp]
  const float* b1;     // [mid]
  const float* w2t;    // [mid][cp] (second excitation layer, transposed)
  const float* b2;     // [cp]
  float* gates;        // two gate slots [2][N][cp]: the previous frame's
                       // gates in slot *gpar, this frame's in the other
  const int* gpar;     // device parity word
  int64_t gsz;         // floats per slot
  void* dout;          // emitted rows [npix][cp] (row = site)
  uint32_t* rowmax;
  int* rowpix;
  int* map;
  u64* cnt_rows;
  int64_t npix, hw;
  int N, cp, c, mid, act, ref, chunk, nchunk, tps;
  float keep_thr;
  const float* keep_thr_dev;  // in device memory (or NULL: keep_thr)
  const float* yhat;          // residual carry view or NULL
  float* gout;                // excitation: gates to [N][cp] here instead
                              // of the new slot (or NULL)
  // excitation of a chunk's frames in one launch (nfr frames in order,
  // frame t's partials at part + t * part_stride, its gates at gout +
  // t * gout_stride); nfr 0 or 1: one frame
  int nfr;
  int64_t part_stride, gout_stride;
};
void launch_se(const Prof& pf, hipStream_t s, int dtype, const SeArgs& a);

// ---- exact squeeze-excitation in a chunk (frames t = 0 .. nf - 1): the
// chunk update has left each updated item's state after its frame in Pt
// (rows of the layer's affected list, Mo: conv item -> row) and each
// site's updating frames in aff.  Per frame t the squeeze sums
// f(P_t) - f(P_{t-1}) over the sites frame t updated into
// part[t][N][nchunk][cp] (the frame-by-frame squeeze's partials, in its
// order), the excitation moves S frame by frame and leaves frame t's gates
// in gates[t][N][cp], and the emission writes, for every site and frame,
// f(P_t) * s_t - f(P_{t-1}) * s_{t-1} (s_{-1}: the gates before the chunk,
// slot *gpar of the two-slot gate buffer) as candidate row
// site * nf + t.  Finally the last frame's gates go to the new gate slot.
struct ChunkSeArgs {
  int p16;
  const float* P;       // state before the chunk [npix][cp]
  const float* Pt;      // per-item states after their frame's update
  const int* Mo;        // conv item (frame * npix + site) -> Pt row or -1
  const uint32_t* aff;  // [npix] frames that updated each site
  float* part;          // [nf][N][nchunk][cp]
  float* gates;         // [nf][N][cp]
  float* slots;         // the layer's two gate slots [2][N][cp]
  const int* gpar;
  int64_t gsz;          // floats per slot
  void* dout;           // candidate rows [npix * nf][cp] (site-major)
  uint32_t* rowmax;
  int* rowpix;
  int* map;
  u64* cnt_rows;
  int64_t npix, hw;
  int N, nf, cp, act, chunk, nchunk, tps;
};
void launch_chunk_se(const Prof& pf, hipStream_t s, int dtype,
                     const ChunkSeArgs& c, const SeArgs& excite);
// Storage-dtype matrix src [rows][cols] (or, transposed, src [cols][rows])
// to f32 dst [rows_p][cols_p], zero padded; src may be NULL (zeros).
void launch_to_f32_pad(hipStream_t s, int dtype, const void* src, float* dst,
                       int rows, int cols, int rows_p, int cols_p,
                       bool transposed = false);

// ---- chunk mode: the diff frames of a chunk encoded layer-major
// Items: frame t's sites follow frame t-1's (item = t * sites + site).
struct ChunkScanArgs {
  const void* x;       // frames [nf][npix][C] (storage dtype)
  void* xhat;          // [npix][C]
  int C, Cp, nf;
  int64_t npix;        // input sites per frame
  float thr;
  const float* thr_dev;  // threshold in device memory (or NULL: thr)
  uint8_t* keep;       // [npix * nf] keep bytes, site-major
  uint8_t* base;       // [nf * npix] frame X_hat held (0xFF: chunk start)
  uint8_t* last;       // [npix] last kept frame (0xFF: none)
  uint32_t* tiles;
  uint32_t* tiles_clear;
  void* rows;
  int* rowpix;
  int* act;
  int* map;
  u64* cnt_rows;
  u64* cnt_act;
  ConsList cons;
};
void launch_chunk_scan(const Prof& pf, hipStream_t s, int dtype,
                       const ChunkScanArgs& a);

struct ChunkUpdArgs {
  int p16;             // state stored as bf16
  float* P;            // state [npix][cp] (physical sites)
  float* dP;           // deferred update rows [*][cp] (pool mode: P_t)
  const int* Mo;       // conv item -> dP row or -1
  const int* O;        // affected conv items (site-major), dP row = index
  const u64* nO;
  u64* sites;          // partial counts [kSiteSlots] of the sites updated
                       // (list mode), or NULL
  void* dout;          // emitted rows [*][cp] (not in pool mode)
  uint32_t* rowmax;    // [rows]
  uint32_t* aff;       // [npix] frames that updated each site (pool mode)
  float* out;          // dense output [nf][npix][c] or NULL
  int64_t npix;        // conv sites per frame
  int nf, cp, c, act, pool_mode, tps;
  const float* gate;    // frozen squeeze-excitation gates, two slots
                        // [2][N][cp] (slot *gpar in use), or NULL
  const int* gpar;
  int64_t gsz;
  int64_t gate_hw;      // sites per image of the conv grid
  // residual carry (not in pool mode): the consumers' view [npix][cp] and
  // the emitted tensor's threshold, or yhat NULL
  float* yhat;
  float keep_thr;
  const float* keep_thr_dev;  // in device memory (or NULL: keep_thr)
};
void launch_chunk_update(const Prof& pf, hipStream_t s, int dtype,
                         const ChunkUpdArgs& a);

struct ChunkPoolArgs {
  const int* Q;        // pooled rows -> pooled item
  const u64* nQ;
  int64_t capQ;
  Geo g;               // conv grid -> pooled grid (one frame)
  const float* P;      // state at the chunk's start [conv sites][cp]
  const float* Pt;     // P after frame t, per conv row
  const int* Mo;       // conv item -> row or -1
  const uint32_t* aff; // [conv sites] frames that updated each site
  void* dout;          // pooled rows [*][cp]
  uint32_t* rowmax;
  int64_t nconv, npool;  // conv / pooled sites per frame
  int cp, act, tps;
  // residual carry: the consumers' view of the pooled tensor [npool][cp]
  // and its threshold, or yhat NULL
  float* yhat;
  float keep_thr;
  const float* keep_thr_dev;
};
void launch_chunk_pool_emit(const Prof& pf, hipStream_t s, int dtype,
                            const ChunkPoolArgs& a);
// P[w] = P after the last frame that updated w, for the sites of the
// affected list O (site-major items, capacity capO), whose frame bits
// aff[w] are then cleared (pooled layers)
void launch_chunk_commit(const Prof& pf, hipStream_t s, int p16, float* P,
                         const float* Pt, const int* O, const u64* nO,
                         uint32_t* aff, int64_t capO, int64_t nconv, int cp);

// ---- dense network output (Accumulation)
// p16: the state is stored as bf16.  se: the last layer's two gate slots
// [2][N][cp] (or NULL), of which slot (*se_par ^ se_flip) applies.
void launch_output(const Prof& pf, hipStream_t s, const float* P, int p16,
                   int cp, int C, int N, Geo pool, int has_pool, int act,
                   const float* se, const int* se_par, int se_flip,
                   float* out);
// Flips the net's gate-slot parity word (end of a frame whose
// squeeze-excitation layers computed new gates).
void launch_flip_parity(hipStream_t s, int* par);

// ---- setup / introspection helpers
void launch_fill_u32(hipStream_t s, void* p, int64_t n, uint32_t v);
void launch_repack_dense(hipStream_t s, int dtype, const void* w, void* wt,
                         int cout, int cin, int kh, int kw, int cin_p,
                         int cout_p, int64_t ktot_p);
void launch_repack_dw(hipStream_t s, int dtype, const void* w, float* wdw,
                      int c, int kh, int kw, int cp);
void launch_bias(hipStream_t s, int dtype, const void* b, float* out,
                 int cout, int cout_p);
// ---- residual carry: the kept rows of an emitted tensor reach the
// consumers, so they join the view: view[pix] += row (f32) for every kept
// row (act[k] = pix, map[pix] = its row).
void launch_carry_commit(const Prof& pf, hipStream_t s, int dtype,
                         const int* act, const u64* n_act, int64_t cap,
                         const int* map, const void* rows, float* view,
                         int cp);

// ---- online threshold adjustment on the device
// Per tensor t: bisection state theta/lo/hi (f64), the f32 threshold the
// kernels read, a controlled flag, and the tensor's site count.  After a
// diff frame, each controlled tensor's sparsity 1 - kept / sites (kept =
// counters[2 t + 1]) moves theta one bisection step toward
// [target - eps, target + eps].
struct IbstArgs {
  double* theta;
  double* lo;
  double* hi;
  float* thr;
  const uint8_t* ctl;
  const int64_t* sites;
  int n;
  double target, eps, theta_max;
};
// nf: frames the counters cover (a chunk's kept rows over sites * nf).
void launch_ibst_step(hipStream_t s, const u64* counters, int nf,
                      const IbstArgs& a);
// A new cycle: every controlled bracket back to [0, theta_max].
void launch_ibst_restart(hipStream_t s, const IbstArgs& a);

// Kept rows per image of a kept list (any order); cap bounds its length.
void launch_density(hipStream_t s, const int* act, const u64* n_act,
                    int64_t cap, int64_t hw, int images, u64* out);

}  // namespace st
