// Executor and HIP-side entry points of the C ABI: workspace binding and
// weight repacking, the per-frame kernel sequence of the reference and diff
// passes, density queries, introspection copies and kernel timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "st_internal.h"
#include "st_kernels.h"

static_assert(st::kSplitMax <= st::kEpiSplits,
              "the split epilogue holds every split");

namespace st {

struct Recorder {
  bool on = false;
  int max_launches = 0, max_frames = 0;
  int frame = -1;
  std::vector<hipEvent_t> ev;            // two per launch
  std::vector<st_launch_record> recs;
  uint64_t* hist = nullptr;              // pinned host: [max_frames][n_counters]
  int n_hist = 0;
  ~Recorder() {
    for (hipEvent_t e : ev) (void)hipEventDestroy(e);
    if (hist) (void)hipHostFree(hist);
  }
};

void prof_begin(const Prof& p, int cls, hipStream_t s) {
  (void)cls;
  st_net* net = (st_net*)p.net;
  if (!net || !net->rec || !net->rec->on) return;
  Recorder& R = *net->rec;
  const size_t i = R.recs.size();
  if ((int)i >= R.max_launches) return;
  (void)hipEventRecord(R.ev[2 * i], s);
}

void prof_end(const Prof& p, int cls, hipStream_t s) {
  st_net* net = (st_net*)p.net;
  if (!net || !net->rec || !net->rec->on) return;
  Recorder& R = *net->rec;
  const size_t i = R.recs.size();
  if ((int)i >= R.max_launches) return;
  (void)hipEventRecord(R.ev[2 * i + 1], s);
  R.recs.push_back(st_launch_record{cls, p.layer, R.frame, 0.f});
}

}  // namespace st

// The library's own workspace for callers that cannot allocate device
// memory (st_bind_workspace_static): one fixed-size array per device, held
// until the process ends.  In host code `scratch` names a host-side stand-in,
// never the device array: its device address comes from
// hipGetSymbolAddress, taken once per device with that device current, and
// only that address is used.  A generation count per device records which
// net bound the array last; a net whose binding was taken over refuses to
// run.
static __device__ __align__(256) char scratch[ST_STATIC_WORKSPACE_BYTES];

namespace {

struct StaticWs {
  void* ptr = nullptr;   // device address of `scratch` on this device
  uint64_t gen = 0;      // bindings so far
};
std::mutex g_static_mu;
std::vector<StaticWs> g_static;  // indexed by device ordinal

uint64_t static_generation(int dev) {
  std::lock_guard<std::mutex> lk(g_static_mu);
  return dev >= 0 && dev < (int)g_static.size() ? g_static[dev].gen : 0;
}

}  // namespace

using namespace st;

namespace {

struct WS {
  char* base;
  template <typename T> T* at(size_t off) const { return (T*)(base + off); }
};

// Look-back status sets of the compactions: consecutive compactions (all on
// the encode's stream) alternate between the two, each clearing the other
// for the one after it; the reset at the start of an encode clears set 0.
// Called right before each compaction launch, in launch order.
uint32_t* status_set(st_net* net, uint32_t** clear) {
  uint32_t* t = WS{net->ws}.at<uint32_t>(net->off_tiles);
  const int p = net->cpar;
  net->cpar ^= 1;
  *clear = t + (p ^ 1) * kMaxTiles;
  return t + p * kMaxTiles;
}

st_status hip_check(st_net* net, const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return fail(net, ST_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
  return ST_OK;
}

// The workspace is usable: bound, and -- bound to the library's static
// workspace -- not bound by another net since.
st_status need_ws(st_net* net) {
  if (!net->bound) return fail(net, ST_ERR_STATE, "no workspace bound");
  if (net->static_dev >= 0 &&
      static_generation(net->static_dev) != net->static_gen)
    return fail(net, ST_ERR_STATE,
                "the library's static workspace was bound by another net "
                "since this one bound it");
  return ST_OK;
}

Geo conv_geo(const LayerPlan& L) {
  const st_layer_desc& d = L.d;
  return Geo{L.Hi, L.Wi, L.Ho, L.Wo, d.k_h, d.k_w, d.s_h, d.s_w, d.p_h, d.p_w};
}

Geo pool_geo(const LayerPlan& L) {
  const st_layer_desc& d = L.d;
  return Geo{L.Ho, L.Wo, L.Hp, L.Wp, d.pool_k_h, d.pool_k_w,
             d.pool_s_h, d.pool_s_w, d.pool_p_h, d.pool_p_w};
}

// Rulebook preparation the kept rows of tensor t do for the layers that
// read it (see ConsList in st_kernels.h).
// In a chunk, stateful layers whose every output row is finished by the
// GEMM tile that computes it apply the chunk's updates in the GEMM epilogue
// (rows come site-major, tiles are aligned to site runs).  Such a layer
// runs unsplit: a chunk holds several frames' rows, enough tiles to fill
// the chip without splitting the reduction.  Pooled and depthwise layers
// and the output layer (which also writes every frame's dense output)
// defer the updates to the update kernel.  With residual carry every layer
// defers: a frame's keep decision (the row's largest magnitude over all its
// channels) must be known before the next frame's delta of the same site is
// formed, and the update kernel holds a site's channels in one group of
// lanes.
bool chunk_fused(const st_net* net, int i) {
  const LayerPlan& L = net->layers[i];
  return L.stateful && !L.pool && !L.dw && !L.se && !net->carry &&
         i != (int)net->layers.size() - 1;
}

// A max-pooled layer's GEMM epilogue walks each site's frames the same
// way, but writes the state after each frame to the row's update row (the
// pool emission compares window states frame by frame) instead of
// emitting deltas; the commit after the pool emission stores the state.
// Half-precision nets only: measured on ResNet-50's bf16 stem it saves the
// update kernel's pass (289 -> 225 us per chunk of 10), on the f32
// CRNN-VGG (chunks of 16) it made the chunk 20% slower.
bool chunk_fused_pool(const st_net* net, int i) {
  const LayerPlan& L = net->layers[i];
  return net->dtype != ST_F32 && L.stateful && L.pool && !L.dw && !L.se &&
         !net->carry && i != (int)net->layers.size() - 1;
}

// Layers whose GEMM runs on run-aligned row tiles in a chunk.
bool chunk_tiled_layer(const st_net* net, int i) {
  return chunk_fused(net, i) || chunk_fused_pool(net, i);
}

// list_pass: the consumers of a list compaction in a chunk (the pass that
// cuts the run-aligned tiles of fused identity consumers).
ConsList consumers_of(st_net* net, int t, bool list_pass = false) {
  const WS ws{net->ws};
  u64* cnt = ws.at<u64>(net->off_cnt);
  ConsList cl{};
  cl.n = 0;
  for (const auto& cr : net->tensors[t].consumers) {
    const int j = cr.first;
    const LayerPlan& L = net->layers[j];
    Cons c{};
    if (cr.second == 0 && L.ident) {
      c.kind = kConsIdent;
      c.O = ws.at<int>(L.off_O);
      c.Mo = ws.at<int>(L.off_Mo);
      c.nbr = ws.at<int>(L.off_nbr);
      c.rowmax = (L.pool || L.se)
                     ? nullptr
                     : ws.at<uint32_t>(net->tensors[j + 1].off_rowmax);
      c.cnt_O = cnt + L.cnt_O;
      c.pairs = cnt + L.cnt_pairs;
      if (list_pass && net->last_nf > 1 && chunk_tiled_layer(net, j)) {
        c.tstart = ws.at<uint32_t>(L.off_tstart);
        c.nf = net->last_nf;
        c.per = net->tensors[t].grid;
      }
    } else if (cr.second == 0) {
      c.kind = kConsMark;
      c.flags = ws.at<uint8_t>(L.off_flags);
      c.g = conv_geo(L);
      c.nf = net->last_nf;
      c.nimg = net->N;
    } else {
      c.kind = kConsMarkSame;
      c.flags = ws.at<uint8_t>(L.off_flags);
      c.nf = net->last_nf;
      c.per = net->tensors[t].grid;
    }
    cl.c[cl.n++] = c;
  }
  return cl;
}

IbstArgs ibst_args(st_net* net);

// thr_dev: this layer's emitted-tensor threshold in device memory (online
// adjustment), or NULL to use thr.
bool run_layer(st_net* net, int i, bool ref, float thr, const float* thr_dev,
               hipStream_t s) {
  const WS ws{net->ws};
  const LayerPlan& L = net->layers[i];
  const st_layer_desc& d = L.d;
  const TensorPlan& in = net->tensors[d.src + 1];
  TensorPlan& out = net->tensors[i + 1];
  u64* cnt = ws.at<u64>(net->off_cnt);
  const Prof pf{net, i};

  int* O = ws.at<int>(L.off_O);
  int* Mo = ws.at<int>(L.off_Mo);
  int* nbr = ws.at<int>(L.off_nbr);
  u64* cO = cnt + L.cnt_O;
  u64* cpairs = cnt + L.cnt_pairs;
  uint32_t* rowmax_out = ws.at<uint32_t>(out.off_rowmax);
  // frozen squeeze-excitation in a diff frame: a state-mode layer whose
  // emitted values are scaled by the reference frame's gates
  const bool frozen = L.se && net->frozen_se && !ref;
  // pooled and (exact) squeeze-excitation layers emit rows of their own
  // (pooled sites / every site), not the affected conv outputs
  const bool own_rows = L.pool || (L.se && !frozen);
  uint32_t* rm_O = own_rows ? nullptr : rowmax_out;

  // (b) rulebook: the flags were set while the producers emitted their kept
  // rows; a 1x1 stride-1 layer's rulebook was written there directly.
  if (!L.ident) {
    FlagArgs fa{};
    fa.flags = ws.at<uint8_t>(L.off_flags);
    fa.npix = L.conv_grid;
    fa.list = O;
    fa.map = Mo;
    fa.rowmax = rm_O;
    fa.nbr = nbr;
    fa.map_in = ws.at<int>(in.off_map);
    fa.stride = L.conv_grid * net->F;  // the table holds F frames' rows
    fa.g = conv_geo(L);
    fa.pairs = cpairs;
    fa.cnt = cO;
    fa.tiles = status_set(net, &fa.tiles_clear);
    launch_flag_compact(pf, ST_K_RB_COMPACT, s, fa);
  }

  // (c) delta convolution with fused (d) update / emission
  ConvArgs a{};
  a.p16 = net->bf16_state ? 1 : 0;
  a.din = ws.at<char>(in.off_rows);
  a.nbr = nbr;
  a.stride = L.conv_grid * net->F;
  a.K = L.K;
  a.cin_p = L.cin_p;
  a.cout_p = L.cout_p;
  a.ktot_p = L.ktot_p;
  a.w = ws.at<char>(L.off_w);
  a.bias = ws.at<float>(L.off_bias);
  a.O = O;
  a.nO = cO;
  a.capO = L.conv_grid;
  a.P = L.stateful ? ws.at<float>(L.off_P) : nullptr;
  a.dP = own_rows ? ws.at<float>(L.off_dP) : nullptr;
  a.dout = own_rows ? nullptr : ws.at<char>(out.off_rows);
  a.rowmax = rm_O;
  if (d.residual_src != -2) {
    const TensorPlan& R = net->tensors[d.residual_src + 1];
    a.dskip = ws.at<char>(R.off_rows);
    a.mskip = ws.at<int>(R.off_map);
  }
  a.mode = frozen ? kModeState : L.mode;
  a.act = d.act;
  a.ref = ref ? 1 : 0;
  if (frozen) {
    a.gate = ws.at<float>(L.off_ses);
    a.gpar = ws.at<int>(net->off_se_par);
    a.gsz = (int64_t)net->N * L.cout_p;
    a.gate_hw = (int64_t)L.Ho * L.Wo;
  }
  a.keep_thr = thr;
  a.keep_thr_dev = thr_dev;
  a.yhat = net->carry && !own_rows ? ws.at<float>(L.off_yhat) : nullptr;
  a.zero = ws.at<char>(net->off_zero);
  a.part = ws.at<float>(net->off_part);
  a.split_max = L.split_max;
  if (L.dw)
    launch_conv_dw(pf, s, net->dtype, a);
  else if (!launch_conv_gemm(pf, s, net->dtype, a))
    return false;

  // non-linear post-op: max-pool from old and new state, then commit
  if (L.pool) {
    const Geo gp = pool_geo(L);
    uint8_t* pflags = ws.at<uint8_t>(L.off_pflags);
    launch_mark(pf, ST_K_POOL_MARK, s, O, cO, L.conv_grid, gp, pflags,
                net->N, 1);
    FlagArgs fp{};
    fp.flags = pflags;
    fp.npix = out.grid;
    fp.list = ws.at<int>(out.off_rowpix);
    fp.map = ws.at<int>(out.off_map);
    fp.rowmax = rowmax_out;
    fp.cnt = cnt + out.cnt_rows;
    fp.tiles = status_set(net, &fp.tiles_clear);
    launch_flag_compact(pf, ST_K_POOL_COMPACT, s, fp);
    PoolArgs pa{};
    pa.Q = ws.at<int>(out.off_rowpix);
    pa.nQ = cnt + out.cnt_rows;
    pa.capQ = out.grid;
    pa.g = gp;
    pa.P = ws.at<float>(L.off_P);
    pa.dP = ws.at<float>(L.off_dP);
    pa.Mo = Mo;
    pa.dout = ws.at<char>(out.off_rows);
    pa.rowmax = rowmax_out;
    pa.cp = L.cout_p;
    pa.act = d.act;
    pa.ref = ref ? 1 : 0;
    pa.yhat = net->carry ? ws.at<float>(L.off_yhat) : nullptr;
    launch_pool_emit(pf, s, net->dtype, pa);
    launch_commit(pf, s, O, cO, L.conv_grid, ws.at<float>(L.off_P),
                  ws.at<float>(L.off_dP), L.cout_p, ref ? 1 : 0);
  }
  if (L.se && !frozen) {
    SeArgs sa{};
    sa.p16 = net->bf16_state ? 1 : 0;
    sa.P = ws.at<float>(L.off_P);
    sa.dP = ws.at<float>(L.off_dP);
    sa.Mo = Mo;
    sa.part = ws.at<float>(L.off_separt);
    sa.S = ws.at<double>(L.off_sesum);
    sa.w1 = ws.at<float>(L.off_sew1);
    sa.b1 = ws.at<float>(L.off_seb1);
    sa.w2t = ws.at<float>(L.off_sew2);
    sa.b2 = ws.at<float>(L.off_seb2);
    sa.gates = ws.at<float>(L.off_ses);
    sa.gpar = ws.at<int>(net->off_se_par);
    sa.gsz = (int64_t)net->N * L.cout_p;
    sa.dout = ws.at<char>(out.off_rows);
    sa.rowmax = rowmax_out;
    sa.rowpix = ws.at<int>(out.off_rowpix);
    sa.map = ws.at<int>(out.off_map);
    sa.cnt_rows = cnt + out.cnt_rows;
    sa.npix = L.conv_grid;
    sa.hw = (int64_t)L.Ho * L.Wo;
    sa.tps = L.se_tps;
    sa.N = net->N;
    sa.cp = L.cout_p;
    sa.c = d.c_out;
    sa.mid = L.se_mid;
    sa.act = d.act;
    sa.ref = ref ? 1 : 0;
    sa.chunk = L.se_chunk;
    sa.nchunk = L.se_nchunk;
    sa.keep_thr = thr;
    sa.keep_thr_dev = thr_dev;
    sa.yhat = net->carry ? ws.at<float>(L.off_yhat) : nullptr;
    launch_se(pf, s, net->dtype, sa);
  }

  // truncation of the emitted delta (shared by every consumer), which also
  // prepares the consumers' rulebooks
  ListArgs la{};
  la.rowmax = rowmax_out;
  la.n_rows = cnt + out.cnt_rows;
  la.cap = out.grid;
  la.thr = thr;
  la.thr_dev = thr_dev;
  la.rowpix = ws.at<int>(out.off_rowpix);
  la.act = ws.at<int>(out.off_act);
  la.map = ws.at<int>(out.off_map);
  la.cnt_act = cnt + out.cnt_act;
  la.cons = consumers_of(net, i + 1);
  la.tiles = status_set(net, &la.tiles_clear);
  launch_list_compact(pf, s, la);
  // residual carry: the kept rows join the consumers' view
  if (net->carry)
    launch_carry_commit(pf, s, net->dtype, la.act, la.cnt_act, out.grid,
                        la.map, ws.at<char>(out.off_rows),
                        ws.at<float>(L.off_yhat), L.cout_p);
  out.last_thr = thr;
  return true;
}

// The reference frame keeps every pixel (threshold -1 everywhere), so the
// frame-by-frame pass would compact every tensor into its pixels in order.
// For nets without squeeze-excitation or residual carry it runs dense
// instead: each tensor's rows are its pixels, the convolutions take their
// neighbours from the geometry, and no list, map or rulebook is built.  It
// leaves what the frame-by-frame reference pass leaves for the diff frames
// and the queries: X_hat, every state, the emitted rows, the kept lists
// (identities) and the counters (every row kept, the dense pair counts).
static st_status encode_dense_ref(st_net* net, const void* frame, float* out,
                                  hipStream_t s) {
  const WS ws{net->ws};
  u64* cnt = ws.at<u64>(net->off_cnt);
  net->last_nf = 1;
  const Prof pf{net, -1};
  Recorder* R = net->rec && net->rec->on ? net->rec : nullptr;
  if (R) ++R->frame;
  (void)hipGetLastError();  // clear any stale error

  TensorPlan& T0 = net->tensors[0];
  launch_dense_input(pf, s, net->dtype, frame, ws.at<char>(net->off_xhat),
                     ws.at<char>(T0.off_rows), net->C, T0.Cp, T0.grid);
  T0.last_thr = -1.f;
  const int nl = (int)net->layers.size();
  for (int i = 0; i < nl; ++i) {
    const LayerPlan& L = net->layers[i];
    const st_layer_desc& d = L.d;
    const TensorPlan& in = net->tensors[d.src + 1];
    TensorPlan& outT = net->tensors[i + 1];
    const Prof pfl{net, i};
    // a pooled layer's rows are its pool's; the output layer's go nowhere
    const bool no_rows = L.pool || i == nl - 1;
    ConvArgs a{};
    a.p16 = net->bf16_state ? 1 : 0;
    a.din = ws.at<char>(in.off_rows);
    a.nbr = ws.at<int>(L.off_nbr);
    a.K = L.K;
    a.cin_p = L.cin_p;
    a.cout_p = L.cout_p;
    a.ktot_p = L.ktot_p;
    a.w = ws.at<char>(L.off_w);
    a.bias = ws.at<float>(L.off_bias);
    a.O = ws.at<int>(L.off_O);
    a.nO = cnt + L.cnt_O;
    a.capO = L.conv_grid;
    a.P = L.stateful ? ws.at<float>(L.off_P) : nullptr;
    a.dout = no_rows ? nullptr : ws.at<char>(outT.off_rows);
    a.rowmax = nullptr;
    if (d.residual_src != -2) {
      const TensorPlan& Rt = net->tensors[d.residual_src + 1];
      a.dskip = ws.at<char>(Rt.off_rows);
      a.mskip = ws.at<int>(Rt.off_map);  // marks the residual; not read
    }
    a.mode = no_rows ? kModeStateOnly
                     : (L.stateful ? kModeState : kModeLinear);
    a.act = d.act;
    a.ref = 1;
    a.keep_thr = -1.f;
    a.zero = ws.at<char>(net->off_zero);
    a.part = ws.at<float>(net->off_part);
    a.split_max = L.split_max;
    a.dense = 1;
    a.g = conv_geo(L);
    if (L.dw)
      launch_conv_dw(pfl, s, net->dtype, a);
    else if (!launch_conv_gemm(pfl, s, net->dtype, a))
      return fail(net, ST_ERR_HIP, "internal: GEMM launch arguments");
    if (L.pool)
      launch_pool_dense(pfl, s, net->dtype, ws.at<float>(L.off_P), a.p16,
                        ws.at<char>(outT.off_rows), pool_geo(L), L.cout_p,
                        d.act, outT.grid);
    outT.last_thr = -1.f;
  }
  if (out) {
    const LayerPlan& L = net->layers[nl - 1];
    const Geo g = L.pool ? pool_geo(L) : Geo{L.Ho, L.Wo, L.Ho, L.Wo, 1, 1,
                                             1, 1, 0, 0};
    launch_output(Prof{net, nl - 1}, s, ws.at<float>(L.off_P),
                  net->bf16_state ? 1 : 0, L.cout_p, L.d.c_out, net->N, g,
                  L.pool ? 1 : 0, L.d.act, nullptr,
                  ws.at<int>(net->off_se_par), 1, out);
  }
  launch_iota_lists(pf, s, ws.at<IotaEntry>(net->off_iota), net->n_iota,
                    net->ws, net->max_grid);
  launch_copy_u64(s, cnt, ws.at<u64>(net->off_refcnt), net->n_counters);
  if (net->ibst_on && net->ibst_refs++ % net->ibst_cycle_refs == 0)
    launch_ibst_restart(s, ibst_args(net));
  if (R && R->n_hist < R->max_frames) {
    (void)hipMemcpyAsync(R->hist + (size_t)R->n_hist * net->n_counters, cnt,
                         sizeof(u64) * net->n_counters, hipMemcpyDeviceToHost,
                         s);
    ++R->n_hist;
  }
  net->last_stream = (void*)s;
  return hip_check(net, "st_encode_reference");
}

// thr: host thresholds (ignored for the reference frame), or NULL for the
// thresholds of the online adjustment in device memory.
st_status encode(st_net* net, const void* frame, const float* thr, float* out,
                 hipStream_t s, bool ref) {
  if (ref && net->dense_ref) return encode_dense_ref(net, frame, out, s);
  const float* thr_dev =
      (!ref && !thr) ? WS{net->ws}.at<float>(net->off_ibst_thr) : nullptr;
  const WS ws{net->ws};
  u64* cnt = ws.at<u64>(net->off_cnt);
  net->last_nf = 1;
  const Prof pf{net, -1};
  Recorder* R = net->rec && net->rec->on ? net->rec : nullptr;
  if (R) ++R->frame;
  (void)hipGetLastError();  // clear any stale error

  launch_reset(pf, s, cnt, net->n_counters,
               ws.at<uint32_t>(net->off_tiles));
  net->cpar = 0;
  // residual carry: the reference frame's rows (every site) become the
  // consumers' whole view
  if (ref && net->carry)
    for (const LayerPlan& L : net->layers)
      launch_fill_u32(s, ws.at<float>(L.off_yhat),
                      net->tensors[&L - net->layers.data() + 1].grid *
                          L.cout_p,
                      0u);
  TensorPlan& T0 = net->tensors[0];
  const float thr0 = ref ? -1.f : thr_dev ? 0.f : thr[0];
  ScanArgs sa{};
  sa.x = frame;
  sa.xhat = ws.at<char>(net->off_xhat);
  sa.C = net->C;
  sa.Cp = T0.Cp;
  sa.npix = T0.grid;
  sa.thr = thr0;
  sa.thr_dev = thr_dev;
  sa.ref = ref ? 1 : 0;
  sa.rows = ws.at<char>(T0.off_rows);
  sa.rowpix = ws.at<int>(T0.off_rowpix);
  sa.act = ws.at<int>(T0.off_act);
  sa.map = ws.at<int>(T0.off_map);
  sa.cnt_rows = cnt + T0.cnt_rows;
  sa.cnt_act = cnt + T0.cnt_act;
  sa.cons = consumers_of(net, 0);
  sa.tiles = status_set(net, &sa.tiles_clear);
  launch_scan(pf, s, net->dtype, sa);
  T0.last_thr = thr0;
  const int nl = (int)net->layers.size();
  for (int i = 0; i < nl; ++i)
    if (!run_layer(net, i, ref, ref ? -1.f : thr_dev ? 0.f : thr[i + 1],
                   thr_dev ? thr_dev + i + 1 : nullptr, s))
      return fail(net, ST_ERR_HIP, "internal: GEMM launch arguments");

  if (out) {
    const LayerPlan& L = net->layers[nl - 1];
    const Geo g = L.pool ? pool_geo(L) : Geo{L.Ho, L.Wo, L.Ho, L.Wo, 1, 1,
                                             1, 1, 0, 0};
    // the gates this frame used: just computed (exact), or kept from the
    // reference frame (frozen)
    launch_output(Prof{net, nl - 1}, s, ws.at<float>(L.off_P),
                  net->bf16_state ? 1 : 0, L.cout_p, L.d.c_out, net->N, g,
                  L.pool ? 1 : 0, L.d.act,
                  L.se ? ws.at<float>(L.off_ses) : nullptr,
                  ws.at<int>(net->off_se_par),
                  (ref || !net->frozen_se) ? 1 : 0, out);
  }
  // the gates just computed become the previous frame's (a parity word in
  // device memory, so that a captured frame replays correctly)
  if (net->has_se && (ref || !net->frozen_se))
    launch_flip_parity(s, ws.at<int>(net->off_se_par));
  launch_cleanup(pf, s, ws.at<CleanEntry>(net->off_cleanup), net->n_cleanup,
                 net->ws, cnt, net->max_grid);
  // online adjustment: every cycle_refs-th reference frame starts a new
  // cycle; after a diff frame encoded with the device thresholds, one
  // bisection step
  if (net->ibst_on && ref && net->ibst_refs++ % net->ibst_cycle_refs == 0)
    launch_ibst_restart(s, ibst_args(net));
  if (thr_dev) launch_ibst_step(s, cnt, 1, ibst_args(net));
  if (R && R->n_hist < R->max_frames) {
    (void)hipMemcpyAsync(R->hist + (size_t)R->n_hist * net->n_counters, cnt,
                         sizeof(u64) * net->n_counters, hipMemcpyDeviceToHost,
                         s);
    ++R->n_hist;
  }
  net->last_stream = (void*)s;
  return hip_check(net, ref ? "st_encode_reference" : "st_encode_diff");
}

// ---- chunk mode: the frames of a chunk as items (frame t's sites after
// frame t-1's) for the rulebooks, GEMMs and truncations; per-site frame
// loops for the frame delta, the state update and the pools.
IbstArgs ibst_args(st_net* net) {
  const WS ws{net->ws};
  IbstArgs a{};
  a.theta = ws.at<double>(net->off_ibst_theta);
  a.lo = ws.at<double>(net->off_ibst_lo);
  a.hi = ws.at<double>(net->off_ibst_hi);
  a.thr = ws.at<float>(net->off_ibst_thr);
  a.ctl = ws.at<uint8_t>(net->off_ibst_ctl);
  a.sites = ws.at<int64_t>(net->off_ibst_sites);
  a.n = (int)net->tensors.size();
  a.target = net->ibst_target;
  a.eps = net->ibst_eps;
  a.theta_max = net->ibst_theta_max;
  return a;
}

// thr_dev: as for run_layer.
bool run_layer_chunk(st_net* net, int i, int nf, float thr,
                     const float* thr_dev, float* out, hipStream_t s) {
  const WS ws{net->ws};
  const LayerPlan& L = net->layers[i];
  const st_layer_desc& d = L.d;
  const TensorPlan& in = net->tensors[d.src + 1];
  TensorPlan& outT = net->tensors[i + 1];
  u64* cnt = ws.at<u64>(net->off_cnt);
  const Prof pf{net, i};
  const int64_t citems = L.conv_grid * nf;
  const int64_t stride = L.conv_grid * net->F;
  float* cdp = ws.at<float>(net->off_chunk_dp);

  int* O = ws.at<int>(L.off_O);
  int* Mo = ws.at<int>(L.off_Mo);
  int* nbr = ws.at<int>(L.off_nbr);
  u64* cO = cnt + L.cnt_O;
  u64* cpairs = cnt + L.cnt_pairs;
  uint32_t* rowmax_out = ws.at<uint32_t>(outT.off_rowmax);
  // exact squeeze-excitation: every site of every frame emits (per-frame
  // squeeze and excitation between the update and the emission)
  const bool exact_se = L.se && !net->frozen_se;
  uint32_t* rm_O = (L.pool || exact_se) ? nullptr : rowmax_out;
  const bool fused = chunk_fused(net, i);
  const bool fpool = chunk_fused_pool(net, i);
  // the fused GEMM's run-aligned row tiles: cut by the rulebook
  // compaction, or (identity layers) by the list compaction of the layer
  // that emitted the input, else by a pass of their own
  const bool tiled = fused || fpool;
  uint32_t* tstart = tiled ? ws.at<uint32_t>(L.off_tstart) : nullptr;
  bool tiles_cut = tiled && nf > 1 && L.ident && d.src >= 0;

  if (!L.ident) {
    FlagArgs fa{};
    fa.flags = ws.at<uint8_t>(L.off_flags);
    fa.npix = citems;
    fa.list = O;
    fa.map = Mo;
    fa.rowmax = rm_O;
    fa.nbr = nbr;
    fa.map_in = ws.at<int>(in.off_map);
    fa.stride = stride;
    fa.g = conv_geo(L);
    fa.pairs = cpairs;
    fa.cnt = cO;
    fa.nf = nf;
    fa.per = L.conv_grid;
    if (tiled && compact_runs_fit(citems, nf)) {
      fa.tstart = tstart;
      tiles_cut = true;
    }
    fa.tiles = status_set(net, &fa.tiles_clear);
    launch_flag_compact(pf, ST_K_RB_COMPACT, s, fa);
  }
  if (tiled && !tiles_cut)
    launch_run_tiles(pf, s, O, cO, citems, L.conv_grid, nf, tstart);

  ConvArgs a{};
  a.p16 = net->bf16_state ? 1 : 0;
  a.din = ws.at<char>(in.off_rows);
  a.nbr = nbr;
  a.stride = stride;
  a.K = L.K;
  a.cin_p = L.cin_p;
  a.cout_p = L.cout_p;
  a.ktot_p = L.ktot_p;
  a.w = ws.at<char>(L.off_w);
  a.bias = ws.at<float>(L.off_bias);
  a.O = O;
  a.nO = cO;
  a.capO = citems;
  if (fused) {
    a.mode = kModeChunkState;
    a.P = ws.at<float>(L.off_P);
    a.dout = ws.at<char>(outT.off_rows);
    a.rowmax = rowmax_out;
    a.tstart = tstart;
    a.sites = cnt + L.cnt_sites;
    a.nf = nf;
    a.per = L.conv_grid;
  } else if (fpool) {
    a.mode = kModeChunkPool;
    a.P = ws.at<float>(L.off_P);
    a.dP = cdp;
    a.aff = ws.at<uint32_t>(net->off_chunk_aff);
    a.tstart = tstart;
    a.sites = cnt + L.cnt_sites;
    a.nf = nf;
    a.per = L.conv_grid;
  } else if (L.stateful) {
    // every frame's update is deferred; the frame loop applies them
    a.mode = kModeDefer;
    a.dP = cdp;
  } else {
    a.mode = kModeLinear;
    a.dout = ws.at<char>(outT.off_rows);
    a.rowmax = rowmax_out;
  }
  if (d.residual_src != -2) {
    const TensorPlan& R = net->tensors[d.residual_src + 1];
    a.dskip = ws.at<char>(R.off_rows);
    a.mskip = ws.at<int>(R.off_map);
  }
  a.act = d.act;
  a.ref = 0;
  a.keep_thr = thr;
  a.keep_thr_dev = thr_dev;
  a.zero = ws.at<char>(net->off_zero);
  a.part = ws.at<float>(net->off_part);
  a.split_max = tiled ? 1 : L.split_max;
  if (L.dw)
    launch_conv_dw(pf, s, net->dtype, a);
  else if (!launch_conv_gemm(pf, s, net->dtype, a))
    return false;

  if (L.stateful && !tiled) {
    ChunkUpdArgs u{};
    u.p16 = net->bf16_state ? 1 : 0;
    u.P = ws.at<float>(L.off_P);
    u.dP = cdp;
    u.Mo = Mo;
    u.O = O;
    u.nO = cO;
    u.sites = cnt + L.cnt_sites;  // the GEMM epilogue does not count here
    u.dout = ws.at<char>(outT.off_rows);
    u.rowmax = rowmax_out;
    u.aff = ws.at<uint32_t>(net->off_chunk_aff);
    u.out = out;
    u.npix = L.conv_grid;
    u.nf = nf;
    u.cp = L.cout_p;
    u.c = d.c_out;
    u.act = d.act;
    // pooled and exact squeeze-excitation layers: the states after each
    // frame go to the update rows, the frames to aff
    u.pool_mode = (L.pool || exact_se) ? 1 : 0;
    if (L.se && !exact_se) {  // frozen gates
      u.gate = ws.at<float>(L.off_ses);
      u.gpar = ws.at<int>(net->off_se_par);
      u.gsz = (int64_t)net->N * L.cout_p;
      u.gate_hw = (int64_t)L.Ho * L.Wo;
    }
    u.tps = se_threads_per_site(L.cout_p);
    if (net->carry && !L.pool) {
      u.yhat = ws.at<float>(L.off_yhat);
      u.keep_thr = thr;
      u.keep_thr_dev = thr_dev;
    }
    launch_chunk_update(pf, s, net->dtype, u);
  }
  if (exact_se) {
    ChunkSeArgs c{};
    c.p16 = net->bf16_state ? 1 : 0;
    c.P = ws.at<float>(L.off_P);
    c.Pt = cdp;
    c.Mo = Mo;
    c.aff = ws.at<uint32_t>(net->off_chunk_aff);
    c.part = ws.at<float>(net->off_chunk_separt);
    c.gates = ws.at<float>(net->off_chunk_gates);
    c.slots = ws.at<float>(L.off_ses);
    c.gpar = ws.at<int>(net->off_se_par);
    c.gsz = (int64_t)net->N * L.cout_p;
    c.dout = ws.at<char>(outT.off_rows);
    c.rowmax = rowmax_out;
    c.rowpix = ws.at<int>(outT.off_rowpix);
    c.map = ws.at<int>(outT.off_map);
    c.cnt_rows = cnt + outT.cnt_rows;
    c.npix = L.conv_grid;
    c.hw = (int64_t)L.Ho * L.Wo;
    c.N = net->N;
    c.nf = nf;
    c.cp = L.cout_p;
    c.act = d.act;
    c.chunk = L.se_chunk;
    c.nchunk = L.se_nchunk;
    c.tps = L.se_tps;
    SeArgs ex{};
    ex.S = ws.at<double>(L.off_sesum);
    ex.w1 = ws.at<float>(L.off_sew1);
    ex.b1 = ws.at<float>(L.off_seb1);
    ex.w2t = ws.at<float>(L.off_sew2);
    ex.b2 = ws.at<float>(L.off_seb2);
    ex.gates = c.slots;
    ex.gpar = c.gpar;
    ex.gsz = c.gsz;
    ex.hw = c.hw;
    ex.N = net->N;
    ex.cp = L.cout_p;
    ex.c = d.c_out;
    ex.mid = L.se_mid;
    ex.nchunk = L.se_nchunk;
    launch_chunk_se(pf, s, net->dtype, c, ex);
    launch_chunk_commit(pf, s, c.p16, ws.at<float>(L.off_P), cdp, O, cO,
                        ws.at<uint32_t>(net->off_chunk_aff), citems,
                        L.conv_grid, L.cout_p);
  }
  if (L.pool) {
    const Geo gp = pool_geo(L);
    uint8_t* pflags = ws.at<uint8_t>(L.off_pflags);
    launch_mark(pf, ST_K_POOL_MARK, s, O, cO, citems, gp, pflags, net->N,
                nf);
    FlagArgs fp{};
    fp.flags = pflags;
    fp.npix = outT.grid * nf;
    fp.list = ws.at<int>(outT.off_rowpix);
    fp.map = ws.at<int>(outT.off_map);
    fp.rowmax = rowmax_out;
    fp.cnt = cnt + outT.cnt_rows;
    fp.nf = nf;
    fp.per = outT.grid;
    fp.tiles = status_set(net, &fp.tiles_clear);
    launch_flag_compact(pf, ST_K_POOL_COMPACT, s, fp);
    ChunkPoolArgs pa{};
    pa.Q = ws.at<int>(outT.off_rowpix);
    pa.nQ = cnt + outT.cnt_rows;
    pa.capQ = outT.grid * nf;
    pa.g = gp;
    pa.P = ws.at<float>(L.off_P);
    pa.Pt = cdp;
    pa.Mo = Mo;
    pa.aff = ws.at<uint32_t>(net->off_chunk_aff);
    pa.dout = ws.at<char>(outT.off_rows);
    pa.rowmax = rowmax_out;
    pa.nconv = L.conv_grid;
    pa.npool = outT.grid;
    pa.cp = L.cout_p;
    pa.act = d.act;
    pa.tps = se_threads_per_site(L.cout_p);
    if (net->carry) {
      pa.yhat = ws.at<float>(L.off_yhat);
      pa.keep_thr = thr;
      pa.keep_thr_dev = thr_dev;
    }
    launch_chunk_pool_emit(pf, s, net->dtype, pa);
    launch_chunk_commit(pf, s, 0, ws.at<float>(L.off_P), cdp, O, cO,
                        ws.at<uint32_t>(net->off_chunk_aff), citems,
                        L.conv_grid, L.cout_p);
  }

  ListArgs la{};
  la.rowmax = rowmax_out;
  la.n_rows = cnt + outT.cnt_rows;
  la.cap = outT.grid * nf;
  la.thr = thr;
  la.thr_dev = thr_dev;
  la.rowpix = ws.at<int>(outT.off_rowpix);
  la.act = ws.at<int>(outT.off_act);
  la.map = ws.at<int>(outT.off_map);
  la.cnt_act = cnt + outT.cnt_act;
  la.cons = consumers_of(net, i + 1, true);
  la.tiles = status_set(net, &la.tiles_clear);
  launch_list_compact(pf, s, la);
  outT.last_thr = thr;
  return true;
}

// thr: host thresholds, or NULL for the online adjustment's, which then
// takes one bisection step from the whole chunk's counts.
st_status encode_chunk(st_net* net, const void* frames, int nf,
                       const float* thr, float* out, hipStream_t s) {
  const WS ws{net->ws};
  const float* thr_dev = thr ? nullptr : ws.at<float>(net->off_ibst_thr);
  u64* cnt = ws.at<u64>(net->off_cnt);
  const Prof pf{net, -1};
  Recorder* R = net->rec && net->rec->on ? net->rec : nullptr;
  if (R) ++R->frame;
  (void)hipGetLastError();
  net->last_nf = nf;

  launch_reset(pf, s, cnt, net->n_counters,
               ws.at<uint32_t>(net->off_tiles));
  net->cpar = 0;
  TensorPlan& T0 = net->tensors[0];
  ChunkScanArgs sa{};
  sa.x = frames;
  sa.xhat = ws.at<char>(net->off_xhat);
  sa.C = net->C;
  sa.Cp = T0.Cp;
  sa.nf = nf;
  sa.npix = T0.grid;
  sa.thr = thr ? thr[0] : 0.f;
  sa.thr_dev = thr_dev;
  sa.keep = ws.at<uint8_t>(net->off_flags);
  sa.base = ws.at<uint8_t>(net->off_chunk_base);
  sa.last = ws.at<uint8_t>(net->off_chunk_last);
  sa.rows = ws.at<char>(T0.off_rows);
  sa.rowpix = ws.at<int>(T0.off_rowpix);
  sa.act = ws.at<int>(T0.off_act);
  sa.map = ws.at<int>(T0.off_map);
  sa.cnt_rows = cnt + T0.cnt_rows;
  sa.cnt_act = cnt + T0.cnt_act;
  sa.cons = consumers_of(net, 0);
  sa.tiles = status_set(net, &sa.tiles_clear);
  launch_chunk_scan(pf, s, net->dtype, sa);
  T0.last_thr = sa.thr;
  const int nl = (int)net->layers.size();
  for (int i = 0; i < nl; ++i)
    if (!run_layer_chunk(net, i, nf, thr ? thr[i + 1] : 0.f,
                         thr_dev ? thr_dev + i + 1 : nullptr,
                         i == nl - 1 ? out : nullptr, s))
      return fail(net, ST_ERR_HIP, "internal: GEMM launch arguments");
  launch_cleanup(pf, s, ws.at<CleanEntry>(net->off_cleanup), net->n_cleanup,
                 net->ws, cnt, net->max_grid);
  // exact squeeze-excitation: the chunk's last gates (in the new slots)
  // become the previous ones
  if (net->has_se && !net->frozen_se)
    launch_flip_parity(s, ws.at<int>(net->off_se_par));
  if (thr_dev) launch_ibst_step(s, cnt, nf, ibst_args(net));
  if (R && R->n_hist < R->max_frames) {
    (void)hipMemcpyAsync(R->hist + (size_t)R->n_hist * net->n_counters, cnt,
                         sizeof(u64) * net->n_counters, hipMemcpyDeviceToHost,
                         s);
    ++R->n_hist;
  }
  net->last_stream = (void*)s;
  return hip_check(net, "st_encode_chunk");
}

st_status sync_last(st_net* net) {
  hipError_t e = hipStreamSynchronize((hipStream_t)net->last_stream);
  if (e != hipSuccess)
    return fail(net, ST_ERR_HIP, std::string("stream sync: ") +
                                     hipGetErrorString(e));
  return ST_OK;
}

template <typename T>
st_status d2h(st_net* net, T* dst, const void* src, size_t count) {
  if (!count) return ST_OK;
  hipError_t e = hipMemcpy(dst, src, sizeof(T) * count, hipMemcpyDeviceToHost);
  if (e != hipSuccess)
    return fail(net, ST_ERR_HIP, std::string("copy: ") + hipGetErrorString(e));
  return ST_OK;
}

float half_to_float(uint16_t h) {
  _Float16 f;
  std::memcpy(&f, &h, 2);
  return (float)f;
}

float bf16_to_float(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

}  // namespace

extern "C" st_status st_bind_workspace(st_net* net, void* dev_ptr,
                                       uint64_t bytes, void* stream) {
  if (!net) return fail(nullptr, ST_ERR_INVALID_ARG, "net is NULL");
  if (!dev_ptr) return fail(net, ST_ERR_INVALID_ARG, "workspace is NULL");
  if ((uintptr_t)dev_ptr % kAlign)
    return fail(net, ST_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  if (bytes < net->ws_bytes)
    return fail(net, ST_ERR_WORKSPACE,
                "workspace too small: need " + std::to_string(net->ws_bytes));
  hipStream_t s = (hipStream_t)stream;
  net->ws = (char*)dev_ptr;
  net->bound = false;
  net->have_ref = false;
  net->static_dev = -1;
  (void)hipGetLastError();
  const WS ws{net->ws};
  launch_fill_u32(s, net->ws, (int64_t)(net->ws_bytes / 4), 0u);
  // pixel maps start empty for every frame slot of a chunk
  for (const TensorPlan& T : net->tensors)
    launch_fill_u32(s, ws.at<int>(T.off_map), T.grid * net->F, 0xFFFFFFFFu);
  std::vector<CleanEntry> tab;
  for (const TensorPlan& T : net->tensors)
    tab.push_back(CleanEntry{(int64_t)T.off_map, (int64_t)T.off_rowpix,
                             T.cnt_rows, 0, 0});
  for (const LayerPlan& L : net->layers) {
    const st_layer_desc& d = L.d;
    if (L.pool || (L.se && !net->frozen_se)) {
      launch_fill_u32(s, ws.at<int>(L.off_Mo), L.conv_grid * net->F,
                      0xFFFFFFFFu);
      tab.push_back(CleanEntry{(int64_t)L.off_Mo, (int64_t)L.off_O, L.cnt_O,
                               0, 0});
    }
    if (L.se) {
      launch_to_f32_pad(s, net->dtype, d.se_w1, ws.at<float>(L.off_sew1),
                        d.se_mid, d.c_out, d.se_mid, L.cout_p);
      launch_to_f32_pad(s, net->dtype, d.se_b1, ws.at<float>(L.off_seb1), 1,
                        d.se_mid, 1, d.se_mid);
      launch_to_f32_pad(s, net->dtype, d.se_w2, ws.at<float>(L.off_sew2),
                        d.se_mid, d.c_out, d.se_mid, L.cout_p, true);
      launch_to_f32_pad(s, net->dtype, d.se_b2, ws.at<float>(L.off_seb2), 1,
                        d.c_out, 1, L.cout_p);
    }
    if (L.dw)
      launch_repack_dw(s, net->dtype, d.weight, ws.at<float>(L.off_w),
                       d.c_out, d.k_h, d.k_w, L.cout_p);
    else
      launch_repack_dense(s, net->dtype, d.weight, ws.at<char>(L.off_w),
                          d.c_out, d.c_in, d.k_h, d.k_w, L.cin_p, L.cout_p,
                          L.ktot_p);
    launch_bias(s, net->dtype, d.bias, ws.at<float>(L.off_bias), d.c_out,
                L.cout_p);
  }
  static_assert(sizeof(CleanEntry) == 32, "cleanup entry layout");
  if ((int)tab.size() != net->n_cleanup)
    return fail(net, ST_ERR_INVALID_ARG, "internal: cleanup table size");
  // The tables must outlive the asynchronous copies: keep them alive.
  static thread_local std::vector<CleanEntry> keep_alive;
  keep_alive = tab;
  hipError_t e = hipMemcpyAsync(ws.at<char>(net->off_cleanup), keep_alive.data(),
                                sizeof(CleanEntry) * tab.size(),
                                hipMemcpyHostToDevice, s);
  // dense reference pass: the counters it leaves (every row of every
  // tensor kept, every layer's outputs affected, the dense pair counts)
  // and its identity kept lists
  static thread_local std::vector<u64> keep_cnt;
  static thread_local std::vector<IotaEntry> keep_iota;
  static_assert(sizeof(IotaEntry) == 16, "iota entry layout");
  if (net->dense_ref && e == hipSuccess) {
    keep_cnt.assign(net->n_counters, 0);
    keep_iota.clear();
    for (const TensorPlan& T : net->tensors) {
      keep_cnt[T.cnt_rows] = keep_cnt[T.cnt_act] = (u64)T.grid;
      keep_iota.push_back(IotaEntry{(int64_t)T.off_act, T.grid});
    }
    for (const LayerPlan& L : net->layers) {
      keep_cnt[L.cnt_O] = (u64)L.conv_grid;
      keep_cnt[L.cnt_pairs] = (u64)L.dense_pairs;
    }
    e = hipMemcpyAsync(ws.at<char>(net->off_refcnt), keep_cnt.data(),
                       sizeof(u64) * keep_cnt.size(), hipMemcpyHostToDevice,
                       s);
    if (e == hipSuccess)
      e = hipMemcpyAsync(ws.at<char>(net->off_iota), keep_iota.data(),
                         sizeof(IotaEntry) * keep_iota.size(),
                         hipMemcpyHostToDevice, s);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess)
    return fail(net, ST_ERR_HIP, std::string("bind: ") + hipGetErrorString(e));
  st_status st = hip_check(net, "st_bind_workspace");
  if (st != ST_OK) return st;
  net->bound = true;
  net->last_stream = stream;
  return ST_OK;
}

extern "C" st_status st_bind_workspace_static(st_net* net, void* stream) {
  if (!net) return fail(nullptr, ST_ERR_INVALID_ARG, "net is NULL");
  if (net->ws_bytes > (size_t)ST_STATIC_WORKSPACE_BYTES)
    return fail(net, ST_ERR_WORKSPACE,
                "the net needs " + std::to_string(net->ws_bytes) +
                    " workspace bytes; the static workspace holds " +
                    std::to_string((unsigned long long)
                                       ST_STATIC_WORKSPACE_BYTES));
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0)
    return fail(net, ST_ERR_HIP,
                std::string("hipGetDevice: ") + hipGetErrorString(e));
  // the previous owner's work (on any stream) must be done with the array
  e = hipDeviceSynchronize();
  if (e != hipSuccess)
    return fail(net, ST_ERR_HIP,
                std::string("hipDeviceSynchronize: ") + hipGetErrorString(e));
  void* ptr = nullptr;
  uint64_t gen = 0;
  {
    std::lock_guard<std::mutex> lk(g_static_mu);
    if ((int)g_static.size() <= dev) g_static.resize(dev + 1);
    StaticWs& w = g_static[dev];
    if (!w.ptr) {
      // first use on this device (current): the device address of the
      // array; the host-side name is never passed anywhere
      void* p = nullptr;
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return fail(net, ST_ERR_HIP,
                    std::string("hipGetSymbolAddress: ") +
                        hipGetErrorString(e));
      w.ptr = p;
    }
    ptr = w.ptr;
    gen = ++w.gen;
  }
  // the plain binding initialises every byte the net uses (zeros, empty
  // pixel maps, repacked weights), whatever the last binding left
  const st_status st = st_bind_workspace(net, ptr,
                                         ST_STATIC_WORKSPACE_BYTES, stream);
  if (st != ST_OK) return st;
  net->static_dev = dev;
  net->static_gen = gen;
  return ST_OK;
}

extern "C" st_status st_encode_reference(st_net* net, const void* frame,
                                         float* out, void* stream) {
  if (!net) return fail(nullptr, ST_ERR_INVALID_ARG, "net is NULL");
  if (const st_status w = need_ws(net); w != ST_OK) return w;
  if (!frame) return fail(net, ST_ERR_INVALID_ARG, "frame is NULL");
  st_status s = encode(net, frame, nullptr, out, (hipStream_t)stream, true);
  if (s == ST_OK) net->have_ref = true;
  return s;
}

// Checks shared by both chunk entry points (thresholds aside).
static st_status check_chunk(st_net* net, const void* frames,
                             int32_t n_frames) {
  if (!net) return fail(nullptr, ST_ERR_INVALID_ARG, "net is NULL");
  if (const st_status w = need_ws(net); w != ST_OK) return w;
  if (!net->have_ref)
    return fail(net, ST_ERR_STATE, "no reference frame encoded yet");
  if (!frames) return fail(net, ST_ERR_INVALID_ARG, "frames is NULL");
  if (n_frames < 1 || n_frames > net->F)
    return fail(net, ST_ERR_INVALID_ARG,
                "n_frames must be in [1, max_frames of the net]");
  const int nl = (int)net->layers.size();
  if (net->F < 2)
    return fail(net, ST_ERR_UNSUPPORTED,
                "net created without chunk capacity (st_create_net_chunked)");
  if (net->C > kChunkMaxInC)
    return fail(net, ST_ERR_UNSUPPORTED,
                "chunks need at most 16 input channels");
  if (net->layers[nl - 1].pool || net->layers[nl - 1].se)
    return fail(net, ST_ERR_UNSUPPORTED,
                "a pooled or squeeze-excitation last layer in a chunk");
  return ST_OK;
}

extern "C" st_status st_encode_chunk(st_net* net, const void* frames,
                                     int32_t n_frames, const float* thr,
                                     float* out, void* stream) {
  const st_status st = check_chunk(net, frames, n_frames);
  if (st != ST_OK) return st;
  if (!thr) return fail(net, ST_ERR_INVALID_ARG, "thr is NULL");
  for (size_t i = 0; i <= net->layers.size(); ++i)
    if (std::isnan(thr[i]))
      return fail(net, ST_ERR_INVALID_ARG, "threshold is NaN");
  return encode_chunk(net, frames, n_frames, thr, out, (hipStream_t)stream);
}

extern "C" st_status st_encode_chunk_adaptive(st_net* net, const void* frames,
                                              int32_t n_frames, float* out,
                                              void* stream) {
  const st_status st = check_chunk(net, frames, n_frames);
  if (st != ST_OK) return st;
  if (!net->ibst_on)
    return fail(net, ST_ERR_STATE, "threshold control not set");
  return encode_chunk(net, frames, n_frames, nullptr, out,
                      (hipStream_t)stream);
}

extern "C" st_status st_encode_diff(st_net* net, const void* frame,
                                    const float* thr, float* out,
                                    void* stream) {
  if (!net) return fail(nullptr, ST_ERR_INVALID_ARG, "net is NULL");
  if (const st_status w = need_ws(net); w != ST_OK) return w;
  if (!net->have_ref)
    return fail(net, ST_ERR_STATE, "st_encode_diff before st_encode_reference");
  if (!frame || !thr) return fail(net, ST_ERR_INVALID_ARG, "NULL frame or thr");
  for (size_t i = 0; i <= net->layers.size(); ++i)
    if (std::isnan(thr[i]))
      return fail(net, ST_ERR_INVALID_ARG,
                  "threshold " + std::to_string(i) + " is NaN");
  return encode(net, frame, thr, out, (hipStream_t)stream, false);
}

extern "C" st_status st_set_threshold_control(st_net* net,
                                              const uint8_t* controlled,
                                              const float* fixed_thr,
                                              double target, double eps,
                                              double theta_max, double theta0,
                                              int32_t cycle_refs,
                                              void* stream) {
  if (!net) return fail(nullptr, ST_ERR_INVALID_ARG, "net is NULL");
  if (const st_status w = need_ws(net); w != ST_OK) return w;
  if (!controlled || !fixed_thr)
    return fail(net, ST_ERR_INVALID_ARG, "NULL controlled or fixed_thr");
  if (!(target >= 0.0 && target <= 1.0) || !(eps >= 0.0) ||
      !(theta_max > 0.0) || std::isnan(theta0) || theta0 > theta_max ||
      cycle_refs < 1)
    return fail(net, ST_ERR_INVALID_ARG,
                "need 0 <= target <= 1, eps >= 0, theta_max > 0, "
                "theta0 <= theta_max, cycle_refs >= 1");
  const size_t n = net->tensors.size();
  std::vector<double> theta(n), lo(n, 0.0), hi(n, theta_max);
  std::vector<float> thr(n);
  std::vector<uint8_t> ctl(n);
  std::vector<int64_t> sites(n);
  for (size_t t = 0; t < n; ++t) {
    if (std::isnan(fixed_thr[t]))
      return fail(net, ST_ERR_INVALID_ARG,
                  "threshold " + std::to_string(t) + " is NaN");
    ctl[t] = controlled[t] ? 1 : 0;
    theta[t] = ctl[t] ? (theta0 < 0.0 ? theta_max / 2 : theta0)
                      : (double)fixed_thr[t];
    thr[t] = (float)theta[t];
    sites[t] = net->tensors[t].grid;
  }
  const WS ws{net->ws};
  hipStream_t s = (hipStream_t)stream;
  const struct {
    void* dst;
    const void* src;
    size_t bytes;
  } copies[] = {
      {ws.at<double>(net->off_ibst_theta), theta.data(), sizeof(double) * n},
      {ws.at<double>(net->off_ibst_lo), lo.data(), sizeof(double) * n},
      {ws.at<double>(net->off_ibst_hi), hi.data(), sizeof(double) * n},
      {ws.at<float>(net->off_ibst_thr), thr.data(), sizeof(float) * n},
      {ws.at<uint8_t>(net->off_ibst_ctl), ctl.data(), n},
      {ws.at<int64_t>(net->off_ibst_sites), sites.data(),
       sizeof(int64_t) * n},
  };
  for (const auto& c : copies)
    if (hipMemcpyAsync(c.dst, c.src, c.bytes, hipMemcpyHostToDevice, s) !=
        hipSuccess)
      return fail(net, ST_ERR_HIP, "threshold state upload failed");
  // the host vectors must outlive the copies
  if (hipStreamSynchronize(s) != hipSuccess)
    return fail(net, ST_ERR_HIP, "threshold state upload failed");
  net->ibst_on = true;
  net->ibst_target = target;
  net->ibst_eps = eps;
  net->ibst_theta_max = theta_max;
  net->ibst_cycle_refs = cycle_refs;
  net->ibst_refs = 0;
  return ST_OK;
}

extern "C" st_status st_encode_diff_adaptive(st_net* net, const void* frame,
                                             float* out, void* stream) {
  if (!net) return fail(nullptr, ST_ERR_INVALID_ARG, "net is NULL");
  if (const st_status w = need_ws(net); w != ST_OK) return w;
  if (!net->ibst_on)
    return fail(net, ST_ERR_STATE, "threshold control not set");
  if (!net->have_ref)
    return fail(net, ST_ERR_STATE,
                "st_encode_diff_adaptive before st_encode_reference");
  if (!frame) return fail(net, ST_ERR_INVALID_ARG, "NULL frame");
  return encode(net, frame, nullptr, out, (hipStream_t)stream, false);
}

extern "C" st_status st_get_thresholds(st_net* net, float* thr) {
  if (!net || !thr) return fail(net, ST_ERR_INVALID_ARG, "NULL argument");
  if (!net->ibst_on)
    return fail(net, ST_ERR_STATE, "threshold control not set");
  if (net->last_stream) {
    const st_status st = sync_last(net);
    if (st != ST_OK) return st;
  }
  return d2h(net, thr, WS{net->ws}.at<float>(net->off_ibst_thr),
             net->tensors.size());
}

extern "C" st_status st_layer_density(st_net* net, int32_t layer,
                                      int32_t image, float* d) {
  if (!net || !d) return fail(net, ST_ERR_INVALID_ARG, "NULL argument");
  if (const st_status w = need_ws(net); w != ST_OK) return w;
  if (!net->have_ref) return fail(net, ST_ERR_STATE, "nothing encoded yet");
  if (layer < -1 || layer >= (int)net->layers.size())
    return fail(net, ST_ERR_INVALID_ARG, "layer out of range");
  const int images = net->N * net->last_nf;
  if (image < -1 || image >= images)
    return fail(net, ST_ERR_INVALID_ARG, "image out of range");
  const TensorPlan& T = net->tensors[layer + 1];
  const WS ws{net->ws};
  u64* cnt = ws.at<u64>(net->off_cnt);
  st_status st = sync_last(net);
  if (st != ST_OK) return st;
  uint64_t k = 0;
  if (image < 0) {
    st = d2h(net, &k, cnt + T.cnt_act, 1);
    if (st != ST_OK) return st;
    *d = (float)((double)k / ((double)T.grid * net->last_nf));
    return ST_OK;
  }
  hipStream_t s = (hipStream_t)net->last_stream;
  u64* dens = ws.at<u64>(net->off_dens);
  launch_density(s, ws.at<int>(T.off_act), cnt + T.cnt_act,
                 T.grid * net->last_nf, (int64_t)T.H * T.W, images, dens);
  st = hip_check(net, "density");
  if (st != ST_OK) return st;
  st = sync_last(net);
  if (st != ST_OK) return st;
  st = d2h(net, &k, dens + image, 1);
  if (st != ST_OK) return st;
  *d = (float)((double)k / ((double)T.H * T.W));
  return ST_OK;
}

extern "C" void st_destroy_net(st_net* net) {
  if (!net) return;
  delete net->rec;
  delete net;
}

// ------------------------------------------------------------ debug copies

static st_status debug_prelude(st_net* net, int32_t layer, bool need_enc) {
  if (!net) return fail(nullptr, ST_ERR_INVALID_ARG, "net is NULL");
  if (layer < -1 || layer >= (int)net->layers.size())
    return fail(net, ST_ERR_INVALID_ARG, "layer out of range");
  if (const st_status w = need_ws(net); w != ST_OK) return w;
  if (need_enc && !net->have_ref)
    return fail(net, ST_ERR_STATE, "nothing encoded yet");
  return sync_last(net);
}

extern "C" st_status st_debug_active(st_net* net, int32_t layer, int32_t* idx,
                                     int64_t cap, int64_t* n) {
  st_status st = debug_prelude(net, layer, true);
  if (st != ST_OK) return st;
  if (!n) return fail(net, ST_ERR_INVALID_ARG, "n is NULL");
  const TensorPlan& T = net->tensors[layer + 1];
  const WS ws{net->ws};
  uint64_t k = 0;
  st = d2h(net, &k, ws.at<u64>(net->off_cnt) + T.cnt_act, 1);
  if (st != ST_OK) return st;
  *n = (int64_t)k;
  if (idx) st = d2h(net, idx, ws.at<int>(T.off_act), std::min<int64_t>(k, cap));
  return st;
}

extern "C" st_status st_debug_candidates(st_net* net, int32_t layer,
                                         int32_t* pix, float* rows,
                                         int64_t cap, int64_t* n) {
  st_status st = debug_prelude(net, layer, true);
  if (st != ST_OK) return st;
  if (!n) return fail(net, ST_ERR_INVALID_ARG, "n is NULL");
  const TensorPlan& T = net->tensors[layer + 1];
  const WS ws{net->ws};
  uint64_t k = 0;
  st = d2h(net, &k, ws.at<u64>(net->off_cnt) + T.cnt_rows, 1);
  if (st != ST_OK) return st;
  *n = (int64_t)k;
  const int64_t m = std::min<int64_t>(k, cap);
  if (pix) {
    st = d2h(net, pix, ws.at<int>(T.off_rowpix), m);
    if (st != ST_OK) return st;
  }
  if (rows && m) {
    std::vector<uint8_t> raw((size_t)m * T.Cp * net->esize);
    st = d2h(net, raw.data(), ws.at<char>(T.off_rows), raw.size());
    if (st != ST_OK) return st;
    for (int64_t r = 0; r < m; ++r)
      for (int c = 0; c < T.C; ++c) {
        const size_t e = (size_t)r * T.Cp + c;
        float v;
        if (net->dtype == ST_F32) {
          std::memcpy(&v, raw.data() + 4 * e, 4);
        } else {
          uint16_t h;
          std::memcpy(&h, raw.data() + 2 * e, 2);
          v = net->dtype == ST_F16 ? half_to_float(h) : bf16_to_float(h);
        }
        rows[r * T.C + c] = v;
      }
  }
  return ST_OK;
}

extern "C" st_status st_debug_rulebook(st_net* net, int32_t layer,
                                       int32_t* kio, int64_t cap, int64_t* n) {
  st_status st = debug_prelude(net, layer, true);
  if (st != ST_OK) return st;
  if (layer < 0 || !n) return fail(net, ST_ERR_INVALID_ARG, "bad layer or n");
  const LayerPlan& L = net->layers[layer];
  const TensorPlan& in = net->tensors[L.d.src + 1];
  const WS ws{net->ws};
  const u64* cnt = ws.at<u64>(net->off_cnt);
  uint64_t nO = 0, nin = 0;
  if ((st = d2h(net, &nO, cnt + L.cnt_O, 1)) != ST_OK) return st;
  if ((st = d2h(net, &nin, cnt + in.cnt_rows, 1)) != ST_OK) return st;
  std::vector<int> O(nO), rp(nin), nb((size_t)nO * L.K);
  if ((st = d2h(net, O.data(), ws.at<int>(L.off_O), nO)) != ST_OK) return st;
  if ((st = d2h(net, rp.data(), ws.at<int>(in.off_rowpix), nin)) != ST_OK)
    return st;
  for (int k = 0; k < L.K; ++k)
    if ((st = d2h(net, nb.data() + (size_t)k * nO,
                  ws.at<int>(L.off_nbr) + (size_t)k * L.conv_grid * net->F, nO)) !=
        ST_OK)
      return st;
  int64_t cntp = 0;
  for (int k = 0; k < L.K; ++k)
    for (uint64_t o = 0; o < nO; ++o) {
      const int r = nb[(size_t)k * nO + o];
      if (r < 0) continue;
      if (r >= (int)nin)
        return fail(net, ST_ERR_HIP, "internal: neighbour row out of range");
      if (kio && cntp < cap) {
        kio[3 * cntp] = k;
        kio[3 * cntp + 1] = rp[r];
        kio[3 * cntp + 2] = O[o];
      }
      ++cntp;
    }
  *n = cntp;
  return ST_OK;
}

extern "C" st_status st_debug_state(st_net* net, int32_t layer, float* P,
                                    int64_t cap) {
  st_status st = debug_prelude(net, layer, true);
  if (st != ST_OK) return st;
  if (layer < 0 || !P) return fail(net, ST_ERR_INVALID_ARG, "bad layer or P");
  const LayerPlan& L = net->layers[layer];
  if (!L.stateful) return fail(net, ST_ERR_INVALID_ARG, "layer holds no state");
  if (cap < L.conv_grid * L.d.c_out)
    return fail(net, ST_ERR_INVALID_ARG, "P buffer too small");
  std::vector<float> raw((size_t)L.conv_grid * L.cout_p);
  if (net->bf16_state) {
    std::vector<uint16_t> h(raw.size());
    st = d2h(net, h.data(), net->ws + L.off_P, h.size());
    if (st != ST_OK) return st;
    for (size_t i = 0; i < h.size(); ++i) {
      const uint32_t u = (uint32_t)h[i] << 16;
      std::memcpy(&raw[i], &u, 4);
    }
  } else {
    st = d2h(net, raw.data(), net->ws + L.off_P, raw.size());
    if (st != ST_OK) return st;
  }
  for (int64_t p = 0; p < L.conv_grid; ++p)
    std::memcpy(P + p * L.d.c_out, raw.data() + p * L.cout_p,
                sizeof(float) * L.d.c_out);
  return ST_OK;
}

extern "C" st_status st_debug_carry(st_net* net, int32_t layer, float* view,
                                    int64_t cap) {
  st_status st = debug_prelude(net, layer, true);
  if (st != ST_OK) return st;
  if (!net->carry)
    return fail(net, ST_ERR_STATE, "not a residual-carry net");
  if (layer < 0 || !view)
    return fail(net, ST_ERR_INVALID_ARG, "bad layer or view");
  const LayerPlan& L = net->layers[layer];
  const int64_t grid = net->tensors[layer + 1].grid;
  if (cap < grid * L.d.c_out)
    return fail(net, ST_ERR_INVALID_ARG, "view buffer too small");
  std::vector<float> raw((size_t)grid * L.cout_p);
  st = d2h(net, raw.data(), net->ws + L.off_yhat, raw.size());
  if (st != ST_OK) return st;
  for (int64_t p = 0; p < grid; ++p)
    std::memcpy(view + p * L.d.c_out, raw.data() + p * L.cout_p,
                sizeof(float) * L.d.c_out);
  return ST_OK;
}

extern "C" st_status st_debug_counters(st_net* net, int64_t* pairs,
                                       int64_t* active) {
  st_status st = debug_prelude(net, -1, true);
  if (st != ST_OK) return st;
  std::vector<uint64_t> c(net->n_counters);
  st = d2h(net, c.data(), net->ws + net->off_cnt, c.size());
  if (st != ST_OK) return st;
  for (size_t i = 0; i < net->layers.size(); ++i)
    if (pairs) pairs[i] = (int64_t)c[net->layers[i].cnt_pairs];
  for (size_t t = 0; t < net->tensors.size(); ++t)
    if (active) active[t] = (int64_t)c[net->tensors[t].cnt_act];
  return ST_OK;
}

// ------------------------------------------------------------- profiling

extern "C" st_status st_profile_begin(st_net* net, int32_t max_launches,
                                      int32_t max_frames) {
  if (!net) return fail(nullptr, ST_ERR_INVALID_ARG, "net is NULL");
  if (max_launches < 0 || max_frames < 0)
    return fail(net, ST_ERR_INVALID_ARG, "negative capacity");
  if (!net->rec) net->rec = new Recorder();
  Recorder& R = *net->rec;
  while ((int)R.ev.size() < 2 * max_launches) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess)
      return fail(net, ST_ERR_HIP, "hipEventCreate failed");
    R.ev.push_back(e);
  }
  if (R.hist) {
    (void)hipHostFree(R.hist);
    R.hist = nullptr;
  }
  if (max_frames &&
      hipHostMalloc((void**)&R.hist,
                    sizeof(uint64_t) * net->n_counters * max_frames) !=
          hipSuccess)
    return fail(net, ST_ERR_HIP, "hipHostMalloc failed");
  R.max_launches = max_launches;
  R.max_frames = max_frames;
  R.recs.clear();
  R.n_hist = 0;
  R.frame = -1;
  R.on = true;
  return ST_OK;
}

extern "C" st_status st_profile_end(st_net* net, st_launch_record* recs,
                                    int32_t cap, int32_t* n, int64_t* counts,
                                    int32_t cap_frames, int32_t* n_frames) {
  if (!net || !net->rec) return fail(net, ST_ERR_STATE, "not recording");
  Recorder& R = *net->rec;
  R.on = false;
  st_status st = net->last_stream ? sync_last(net) : ST_OK;
  if (st != ST_OK) return st;
  for (size_t i = 0; i < R.recs.size(); ++i) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, R.ev[2 * i], R.ev[2 * i + 1]) != hipSuccess)
      return fail(net, ST_ERR_HIP, "hipEventElapsedTime failed");
    R.recs[i].ms = ms;
  }
  if (n) *n = (int32_t)R.recs.size();
  if (recs)
    for (int i = 0; i < (int)R.recs.size() && i < cap; ++i) recs[i] = R.recs[i];
  const int nl = (int)net->layers.size();
  if (n_frames) *n_frames = R.n_hist;
  if (counts)
    for (int f = 0; f < R.n_hist && f < cap_frames; ++f) {
      const uint64_t* c = R.hist + (size_t)f * net->n_counters;
      for (int j = 0; j < nl; ++j) {
        const LayerPlan& L = net->layers[j];
        const TensorPlan& in = net->tensors[L.d.src + 1];
        const TensorPlan& out = net->tensors[j + 1];
        int64_t* q = counts + ((size_t)f * nl + j) * 8;
        q[0] = (int64_t)c[L.cnt_O];
        q[1] = (int64_t)c[L.cnt_pairs];
        q[2] = (int64_t)c[in.cnt_act];
        q[3] = (int64_t)c[out.cnt_rows];
        q[4] = (int64_t)c[out.cnt_act];
        q[5] = L.d.residual_src == -2
                   ? 0
                   : (int64_t)c[net->tensors[L.d.residual_src + 1].cnt_act];
        // sites updated over a chunk: by the fused GEMM epilogue, or by
        // the chunk update kernel walking the affected list
        int64_t sites = 0;
        for (int k = 0; k < kSiteSlots; ++k)
          sites += (int64_t)c[L.cnt_sites + k];
        const bool fused = net->last_nf > 1 && chunk_tiled_layer(net, j);
        q[6] = fused ? sites : 0;
        q[7] = fused ? 0 : sites;
      }
    }
  return ST_OK;
}
