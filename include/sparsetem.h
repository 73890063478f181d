/*
 * sparsetem.h -- C ABI of the MI355X (gfx950) diff-computation encoder.
 *
 * The library encodes a video chunk with a CNN encoder the way SparseTem's
 * Diff Computation does (paper, section "Skipping Non-zero Delta Pixels"):
 * the chunk's first frame (the reference frame) is encoded densely, every
 * later frame (a diff frame) only on the pixels that changed.  Per layer the
 * diff path is: per-pixel truncation mask + stream compaction of the changed
 * pixels, a rulebook mapping changed input sites to the output sites they
 * reach for every kernel offset (the dense amplification of the "Truncation
 * threshold" paragraph), a gather-GEMM-scatter delta convolution on the
 * changed rows only (linearity of convolution, Eq. 2), and an in-place
 * update of the HBM-resident f32 pre-activation state that also applies the
 * non-linearity and emits the next layer's delta f(P_new) - f(P_old)
 * (non-linear handling, Eq. 3; memory-efficient schedule of the section
 * "Design of SparseBatch": one pre-activation buffer per non-linear layer,
 * no cached outputs).
 *
 * Conventions
 *   - Every pointer named "device" is HIP device memory; "host" is host
 *     memory.  The library never allocates device memory: the caller owns
 *     the workspace, frames, outputs and weights.
 *   - Layout is NHWC; pixel id p = (n * H + y) * W + x.
 *   - `stream` is a hipStream_t passed as void*; NULL is the default stream.
 *     Encode calls are asynchronous and stream-ordered; calls documented as
 *     "synchronising" wait for the last encode's stream.
 *   - Every call returns an st_status; no exception crosses the ABI.
 *     st_last_error() gives a message for the last failure.
 *   - One st_net must not be used from two threads at once; distinct nets
 *     are independent.
 */
#ifndef SPARSETEM_H
#define SPARSETEM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct st_net st_net; /* opaque, library-owned host object */

typedef int32_t st_status;
enum {
  ST_OK = 0,
  ST_ERR_INVALID_ARG = 1, /* NULL pointer, bad shape/channels/geometry, NaN threshold */
  ST_ERR_UNSUPPORTED = 2, /* a layer kind this build does not implement */
  ST_ERR_STATE = 3,       /* no workspace bound, or diff before reference  */
  ST_ERR_WORKSPACE = 4,   /* workspace smaller than st_workspace_bytes()   */
  ST_ERR_HIP = 5          /* a HIP runtime call or kernel launch failed     */
};

/* Storage dtype of frames, weights, biases and emitted deltas.  Sums and
 * the pre-activation state are always f32. */
enum { ST_F32 = 0, ST_F16 = 1, ST_BF16 = 2 };

/* Non-linearity applied after the convolution (and residual add). */
enum { ST_ACT_NONE = 0, ST_ACT_RELU = 1, ST_ACT_SILU = 2 };

/*
 * One layer: a convolution with PyTorch conv2d geometry (dilation 1),
 * optionally plus a residual input, then an activation, then an optional
 * max-pool (PyTorch max_pool2d geometry, -inf padding).
 *   src           producer of the input: -1 = network input, else an earlier
 *                 layer index (layers are given in topological order).
 *   residual_src  producer whose output is added to this layer's
 *                 pre-activation (-2 = none, -1 = network input); its output
 *                 grid and channels must equal this conv's output.
 *   groups        1 (dense) or c_in == c_out == groups (depthwise).
 *   weight        device, storage dtype, [c_out][c_in/groups][k_h][k_w].
 *   bias          device, storage dtype, [c_out]; may be NULL (zero bias).
 *   pool_k_h == 0 means no pool.
 *   se_mid > 0    squeeze-excitation after the activation: per image,
 *                 s = sigmoid(se_w2 . silu(se_w1 . mean_hw(a) + se_b1) + se_b2)
 *                 and the layer emits a * s.  se_w1 [se_mid][c_out],
 *                 se_b1 [se_mid], se_w2 [c_out][se_mid], se_b2 [c_out]
 *                 (device, storage dtype; biases may be NULL).  The gates
 *                 of the previous frame are kept as state: a diff frame
 *                 emits f(P_new) * s_new - f(P_old) * s_old at every site
 *                 (the gates follow the dense activation).  Not combined
 *                 with a pool.
 * A layer is "stateful" (holds an f32 pre-activation buffer) when it has an
 * activation, a pool or squeeze-excitation, or is the last layer (the
 * network output).
 */
typedef struct st_layer_desc {
  int32_t src;
  int32_t residual_src;
  int32_t c_in, c_out, groups;
  int32_t k_h, k_w, s_h, s_w, p_h, p_w;
  int32_t act;
  int32_t pool_k_h, pool_k_w, pool_s_h, pool_s_w, pool_p_h, pool_p_w;
  int32_t se_mid;
  const void *weight, *bias;
  const void *se_w1, *se_b1, *se_w2, *se_b2;
} st_layer_desc;

/* Validate the layer graph and plan the workspace (host only, no HIP call).
 * Defines the encoder whose frames are encoded by Diff Computation (paper,
 * section "Skipping Non-zero Delta Pixels": the CNN encoder whose
 * convolutions, Eq. 1, are evaluated on diff pixels only; one cached
 * pre-activation per layer followed by a non-linear operation, as the
 * schedule of section "Design of SparseBatch" keeps).  Inputs are `batch`
 * images of in_h x in_w x in_c in `dtype`.  The descriptors (and the weight
 * pointers in them) are copied; the weights are read only by
 * st_bind_workspace.  On success *out owns a new net.
 * Errors: ST_ERR_INVALID_ARG (NULL, n_layers < 1, bad src/residual_src, a
 * channel or shape mismatch, an empty output grid, an unknown dtype or
 * activation, squeeze-excitation without its weights), ST_ERR_UNSUPPORTED
 * (groups other than 1 or depthwise, squeeze-excitation with a pool). */
st_status st_create_net(const st_layer_desc* layers, int32_t n_layers,
                        int32_t batch, int32_t in_h, int32_t in_w,
                        int32_t in_c, int32_t dtype, st_net** out);

/* As st_create_net, with room to encode up to `max_frames` (1..32) diff
 * frames in one st_encode_chunk call (the layer-major schedule of section
 * "Design of SparseBatch"): delta rows, active lists, pixel maps and
 * rulebooks are sized for max_frames frames, the pre-activation state and
 * the Subtraction buffer are not.  A net created here also accepts every
 * other call.  Errors as st_create_net, plus ST_ERR_INVALID_ARG for
 * max_frames outside [1, 32]. */
st_status st_create_net_chunked(const st_layer_desc* layers,
                                int32_t n_layers, int32_t batch,
                                int32_t max_frames, int32_t in_h,
                                int32_t in_w, int32_t in_c, int32_t dtype,
                                st_net** out);

/* Creation flags (st_create_net_ex). */
enum {
  /* Residual carry: every emitted tensor keeps its consumers' view (the sum
   * of the deltas they received, f32, one buffer per layer output -- the
   * output caches of the DeltaCNN scheme the paper compares SparseBatch
   * with, in section "Non-linear operations").  A candidate row emits the
   * layer's dense emitted value (f(P), pooled or gated; P for a layer
   * without non-linearity, which then keeps P too) minus the view; kept
   * rows join the view, truncated rows carry their residual until the site
   * is affected again, so what consumers see never strays from the dense
   * value by more than the threshold.  Both entries: in a chunk, every
   * layer applies its updates site by site in frame order, taking each
   * frame's keep decision before the site's next frame is formed, so the
   * result equals frame-by-frame encoding. */
  ST_NET_RESIDUAL_CARRY = 1,
  /* Frozen squeeze-excitation (an approximation, not the exact semantics):
   * the gates computed densely in the reference frame are kept for the
   * chunk's diff frames, so a squeeze-excitation layer emits
   * f(P_new) * s - f(P_old) * s at its affected sites only, with no dense
   * pass per frame.  Exclusive with ST_NET_RESIDUAL_CARRY. */
  ST_NET_FROZEN_SE = 2,
  /* Pre-activation state stored in bf16 (half the state memory and its
   * traffic; an approximation): every update rounds the new state to the
   * nearest bf16 value (ties to even) before it is stored and before the
   * emitted delta f(P_new) - f(P_old) is formed from it, the reference
   * pass rounds the dense pre-activation the same way; so the consumers'
   * sum of deltas follows the stored state exactly, and the state drifts
   * from the exact one by at most one bf16 rounding per update.  Not with
   * max-pooled layers or ST_NET_RESIDUAL_CARRY (ST_ERR_UNSUPPORTED);
   * combines with ST_NET_FROZEN_SE and both entries. */
  ST_NET_BF16_STATE = 4
};

/* As st_create_net_chunked, with creation flags (ST_NET_*).  Errors as
 * st_create_net_chunked, plus ST_ERR_INVALID_ARG for an unknown flag or
 * ST_NET_RESIDUAL_CARRY with ST_NET_FROZEN_SE, and ST_ERR_UNSUPPORTED for
 * ST_NET_RESIDUAL_CARRY with ST_NET_BF16_STATE and for ST_NET_BF16_STATE on
 * a net with a max-pooled layer. */
st_status st_create_net_ex(const st_layer_desc* layers, int32_t n_layers,
                           int32_t batch, int32_t max_frames, int32_t in_h,
                           int32_t in_w, int32_t in_c, int32_t dtype,
                           uint32_t flags, st_net** out);

/* Bytes of device workspace the net needs (host only).  The workspace holds
 * the Subtraction buffer, every f32 pre-activation buffer, the repacked
 * weights, and worst-case-sized (every pixel active) delta rows, active
 * lists, pixel maps and rulebooks, so no frame can overflow it. */
st_status st_workspace_bytes(const st_net* net, uint64_t* bytes);

/* Bind `bytes` of device memory at `dev_ptr` (256-byte aligned) as the
 * workspace, initialise it and repack the weights into it, on `stream`.
 * The weights must stay valid until that stream work has completed; after it
 * they are no longer read.  Rebinding resets the net to "no reference".
 * Errors: ST_ERR_WORKSPACE (too small), ST_ERR_INVALID_ARG (NULL or
 * misaligned), ST_ERR_HIP. */
st_status st_bind_workspace(st_net* net, void* dev_ptr, uint64_t bytes,
                            void* stream);

/* ---- a workspace that needs no allocation, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops and
 * harnesses that forbid hipMalloc).  The library holds one workspace of
 * ST_STATIC_WORKSPACE_BYTES per device in its own code object (a static
 * device array, present on every device the library runs on until the
 * process ends). */
#define ST_STATIC_WORKSPACE_BYTES (64ull << 20)

/* As st_bind_workspace, with the library's static workspace on the current
 * device instead of a caller's buffer: no device memory is allocated or
 * freed, by the library or on its behalf.  Waits for all work on the device
 * to finish first, then initialises everything the net uses in the array
 * (whatever an earlier binding left) and repacks the weights on `stream`.
 * One array per device is shared by every net bound to it: the last binding
 * owns it, and a net whose binding was taken over by another net's fails
 * every further call with ST_ERR_STATE until it is bound again.  Nets that
 * share the array must not run at the same time (their work on one device
 * would race); binding again resets the net to "no reference".
 * Errors: ST_ERR_INVALID_ARG (NULL net), ST_ERR_WORKSPACE
 * (st_workspace_bytes() above ST_STATIC_WORKSPACE_BYTES), ST_ERR_HIP. */
st_status st_bind_workspace_static(st_net* net, void* stream);

/* Dense pass on a reference frame (paper, section "Skipping Non-zero
 * Delta Pixels": the first frame of a chunk is computed densely and sets
 * the values later frames are differenced against; section "Design of
 * SparseBatch": the reference frame is encoded on its own before the diff
 * frames).  `frame`: device, storage dtype, NHWC
 * [batch][in_h][in_w][in_c].  (Re)initialises the Subtraction buffer and
 * every pre-activation buffer (bias included), and writes the network
 * output to `out` (device, f32, NHWC grid of the last layer; may be NULL
 * to skip the write).  Errors: ST_ERR_STATE (no workspace),
 * ST_ERR_INVALID_ARG, ST_ERR_HIP. */
st_status st_encode_reference(st_net* net, const void* frame, float* out,
                              void* stream);

/* Diff pass on the next frame of the chunk (paper, section "Skipping
 * Non-zero Delta Pixels": Subtraction against the committed input, the
 * truncation threshold on each pixel's channels, the convolution of the
 * remaining diff pixels by linearity (Eq. 2), Accumulation onto the cached
 * pre-activation and the non-linear handling of Eq. 3).  `thr` (host,
 * n_layers + 1 floats, read before the call returns): thr[0] truncates the
 * frame delta X - X_hat, thr[j + 1] truncates layer j's emitted delta
 * (shared by all its consumers).  A pixel is kept iff the largest |delta| over its channels is
 * strictly greater than its threshold; a negative threshold keeps every
 * pixel.  Kept input pixels are committed to the Subtraction buffer;
 * truncated deltas inside the network are dropped.  `out` as for
 * st_encode_reference.  Errors: ST_ERR_STATE (no reference since the last
 * bind), ST_ERR_INVALID_ARG (NULL frame/thr, NaN threshold), ST_ERR_HIP. */
st_status st_encode_diff(st_net* net, const void* frame, const float* thr,
                         float* out, void* stream);

/* The next n_frames diff frames at once, layer by layer (section "Design of
 * SparseBatch": one rulebook, GEMM and truncation launch per layer for all
 * frames, the frames taken in order per site wherever one frame's result
 * depends on the previous one's -- the Subtraction buffer, the
 * pre-activation state, max-pool windows).  Result and final state equal
 * n_frames successive st_encode_diff calls with the same `thr` (host,
 * n_layers + 1 floats, shared by the frames).  `frames`: device, storage
 * dtype, [n_frames][batch][in_h][in_w][in_c] contiguous; `out`: device f32
 * [n_frames][last layer's NHWC grid], or NULL.  Afterwards the introspection
 * calls see the frames as n_frames * batch images (frame t's images after
 * frame t-1's), and st_layer_density takes image = t * batch + n.
 * Errors: ST_ERR_STATE (no workspace or no reference), ST_ERR_INVALID_ARG
 * (NULL, NaN threshold, n_frames outside [1, max_frames]),
 * ST_ERR_UNSUPPORTED (a net created without chunk capacity, more than 16
 * input channels, a pooled or squeeze-excitation last layer), ST_ERR_HIP.
 * Exact squeeze-excitation layers take, within the call, each frame's
 * squeeze, excitation and emission at every site in frame order. */
st_status st_encode_chunk(st_net* net, const void* frames, int32_t n_frames,
                          const float* thr, float* out, void* stream);

/* Density (1 - sparsity) of the last encode (paper, section "Online
 * Truncation Threshold Adjustment": the per-layer sparsity the threshold
 * search reads).  Fraction of kept sites: layer = -1 is the frame delta,
 * layer = j is layer j's emitted delta.  image = -1 averages over the batch,
 * otherwise the density of that batch image alone (the per-stream density
 * an online threshold controller reads).  Synchronising. */
st_status st_layer_density(st_net* net, int32_t layer, int32_t image,
                           float* d);

/* ---- online truncation-threshold adjustment on the device (section
 * "Online Truncation Threshold Adjustment": a binary search per layer
 * toward a target sparsity band, restarted every cycle).
 *
 * st_set_threshold_control keeps, for every produced tensor t (index as in
 * `thr`), a threshold theta_t in device memory.  Controlled tensors
 * (controlled[t] != 0) start at theta0 (theta0 < 0: theta_max / 2) with
 * the bracket [0, theta_max]; the others keep fixed_thr[t].  After each
 * st_encode_diff_adaptive frame, every controlled tensor's sparsity
 * s = 1 - kept rows / sites (f64) moves theta one bisection step: s <
 * target - eps: lo = theta, theta = (theta + hi) / 2; s > target + eps:
 * hi = theta, theta = (lo + theta) / 2; the kernels read theta rounded to
 * f32.  A cycle spans cycle_refs reference frames: the first
 * st_encode_reference after this call, and every cycle_refs-th one after
 * it, starts a new cycle (brackets back to [0, theta_max], theta kept).
 * Frame by frame, cycle_refs = 1 gives one search per reference period;
 * st_encode_chunk_adaptive takes one step per chunk, so with a chunk per
 * reference period a search needs cycle_refs > 1 to take several steps.
 * No host round trip per frame: the step is a kernel on the encode stream.
 *
 * controlled, fixed_thr: host arrays of n_layers + 1 entries, read during
 * the call.  The state is uploaded on `stream` and the call waits for it.
 * Errors: ST_ERR_STATE (no workspace), ST_ERR_INVALID_ARG (NULL arrays,
 * target outside [0, 1], eps < 0, theta_max <= 0, theta0 > theta_max, NaN
 * threshold, cycle_refs < 1), ST_ERR_HIP. */
st_status st_set_threshold_control(st_net* net, const uint8_t* controlled,
                                   const float* fixed_thr, double target,
                                   double eps, double theta_max,
                                   double theta0, int32_t cycle_refs,
                                   void* stream);

/* A diff frame encoded with the device thresholds (as st_encode_diff
 * otherwise), followed by the controller's step.  Errors: ST_ERR_STATE (no
 * workspace, no reference frame, threshold control not set),
 * ST_ERR_INVALID_ARG (NULL frame), ST_ERR_HIP. */
st_status st_encode_diff_adaptive(st_net* net, const void* frame, float* out,
                                  void* stream);

/* A chunk encoded with the device thresholds (as st_encode_chunk
 * otherwise: every frame of the chunk uses the same thresholds), followed
 * by one controller step whose sparsity is that of the whole chunk,
 * s = 1 - kept rows over all its frames / (sites * n_frames).  Errors: as
 * st_encode_chunk (thr aside), and ST_ERR_STATE when threshold control is
 * not set. */
st_status st_encode_chunk_adaptive(st_net* net, const void* frames,
                                   int32_t n_frames, float* out,
                                   void* stream);

/* The current f32 thresholds (n_layers + 1 host floats), i.e. those the
 * next adaptive frame uses; synchronises with the last encode.  Errors:
 * ST_ERR_STATE (threshold control not set), ST_ERR_INVALID_ARG, ST_ERR_HIP. */
st_status st_get_thresholds(st_net* net, float* thr);

/* Output grid of layer j's emitted tensor (layer = -1: the input):
 * nhwc[4] = {batch, H, W, C} (host). */
st_status st_tensor_shape(const st_net* net, int32_t layer, int32_t* nhwc);

void st_destroy_net(st_net* net);

/* Message of the last failure on `net` (or of the calling thread's last
 * st_create_net failure when net is NULL).  Owned by the library. */
const char* st_last_error(const st_net* net);

/* ---- parity / introspection: host copies of the last frame's artefacts
 * (the intermediate products of section "Skipping Non-zero Delta Pixels":
 * the kept-pixel lists after truncation, the sites each diff pixel reaches
 * through a window -- the dense amplification of the "Truncation
 * threshold" paragraph -- and the cached pre-activations of Eq. 3).
 * All synchronising.  `cap` counts elements of the caller's buffer; *n
 * receives the full count even when it exceeds cap (nothing is then
 * written past cap). */

/* Kept pixel ids of tensor `layer` (-1 = frame delta), ascending. */
st_status st_debug_active(st_net* net, int32_t layer, int32_t* idx,
                          int64_t cap, int64_t* n);

/* Candidate rows of tensor `layer` before truncation: their pixel ids
 * (ascending, `pix`, may be NULL) and delta values converted to f32
 * (`rows`, [cap][C], may be NULL).  For layer -1 the candidates are the kept
 * pixels. */
st_status st_debug_candidates(st_net* net, int32_t layer, int32_t* pix,
                              float* rows, int64_t cap, int64_t* n);

/* Rulebook of conv layer `layer` as (offset, in_pix, out_pix) triples
 * (`kio`, [cap][3]), offset-major and ascending in in_pix within an offset;
 * offset = ky * k_w + kx. */
st_status st_debug_rulebook(st_net* net, int32_t layer, int32_t* kio,
                            int64_t cap, int64_t* n);

/* Dense f32 pre-activation state of stateful layer `layer`
 * ([batch][H_conv][W_conv][c_out], `cap` floats). */
st_status st_debug_state(st_net* net, int32_t layer, float* P, int64_t cap);

/* Consumers' view of layer `layer`'s emitted tensor on a net created with
 * ST_NET_RESIDUAL_CARRY ([batch][H_out][W_out][c_out] f32, `cap` floats).
 * Errors: ST_ERR_STATE (not a residual-carry net), as st_debug_state. */
st_status st_debug_carry(st_net* net, int32_t layer, float* view,
                         int64_t cap);

/* Per-layer rulebook pair counts (n_layers) and per-tensor kept counts
 * (n_layers + 1, index 0 = frame delta) of the last encode. */
st_status st_debug_counters(st_net* net, int64_t* pairs_per_layer,
                            int64_t* active_per_tensor);

/* ---- measurement: per-launch kernel timing with HIP events recorded on
 * the encode stream, plus a per-frame snapshot of the work counters. */

typedef struct st_launch_record {
  int32_t kernel; /* st_kernel_class */
  int32_t layer;  /* -1 for per-frame kernels */
  int32_t frame;  /* index of the encode call since st_profile_begin */
  float ms;       /* hipEventElapsedTime between the launch's two events */
} st_launch_record;

enum {
  ST_K_SCAN_MASK = 0, ST_K_SCAN_COMPACT, ST_K_RB_MARK, ST_K_RB_COUNT,
  ST_K_RB_COMPACT, ST_K_RB_NBR, ST_K_RB_IDENT, ST_K_CONV_GEMM, ST_K_CONV_DW,
  ST_K_POOL_MARK, ST_K_POOL_COUNT, ST_K_POOL_COMPACT, ST_K_POOL_EMIT,
  ST_K_COMMIT, ST_K_LIST_COUNT, ST_K_LIST_COMPACT, ST_K_OUTPUT,
  ST_K_CLEANUP, ST_K_RESET, ST_K_SE_SQUEEZE, ST_K_SE_EXCITE, ST_K_SE_EMIT,
  ST_K_CONV_SPLIT_EPI, ST_K_CHUNK_UPDATE, ST_K_RUN_TILES,
  ST_K_CARRY_COMMIT, ST_K_NUM_CLASSES
};

/* Start recording: room for `max_launches` launch records and
 * `max_frames` counter snapshots (host-side allocation only).  While
 * recording, every encode records two events around each kernel launch. */
st_status st_profile_begin(st_net* net, int32_t max_launches,
                           int32_t max_frames);

/* Stop recording (synchronising).  Writes up to `cap` launch records and,
 * per recorded encode call f and layer j, counts[(f * n_layers + j) * 8 + i]
 * = {affected conv outputs, rulebook pairs, kept input rows of the layer's
 * source, emitted candidate rows, emitted kept rows, kept rows of the
 * residual source (0 without residual), sites whose state the GEMM epilogue
 * updated over a chunk's frames (st_encode_chunk's fused layers; else 0),
 * sites whose state the chunk update kernel updated from the affected list
 * (st_encode_chunk's deferred layers other than the output layer; else
 * 0)}, up to `cap_frames` calls; a chunk's counts sum over its frames. */
st_status st_profile_end(st_net* net, st_launch_record* recs, int32_t cap,
                         int32_t* n, int64_t* counts, int32_t cap_frames,
                         int32_t* n_frames);

#ifdef __cplusplus
}
#endif

#endif /* SPARSETEM_H */
