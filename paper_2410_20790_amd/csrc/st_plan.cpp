// Host-side planning of a diff-computation net: descriptor validation,
// per-layer shapes and the workspace layout.  No HIP call is made here, so
// the graph checks of st_create_net run on any host.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <string>

#include "st_internal.h"

namespace {
thread_local std::string g_create_err;

int esize_of(int dtype) { return dtype == ST_F32 ? 4 : 2; }

// GEMM reduction chunk: must match the kernel's stage depth per dtype.
int gemm_chunk(int dtype) { return dtype == ST_F32 ? 16 : 64; }

int64_t out_size(int64_t n, int k, int s, int p) {
  return (n + 2 * (int64_t)p - k) / s + 1;
}

struct Alloc {
  size_t top = 0;
  size_t take(size_t bytes) {
    size_t off = st::round_up((int64_t)top, (int64_t)st::kAlign);
    top = off + bytes;
    return off;
  }
};
}  // namespace

namespace st {
st_status fail(st_net* net, st_status s, const std::string& msg) {
  if (net) net->err = msg; else g_create_err = msg;
  return s;
}
}  // namespace st

using namespace st;

static st_status create_fail(st_status s, const std::string& msg) {
  g_create_err = msg;
  return s;
}

static st_status create_impl(const st_layer_desc* layers, int32_t n_layers,
                             int32_t batch, int32_t max_frames, int32_t in_h,
                             int32_t in_w, int32_t in_c, int32_t dtype,
                             uint32_t flags, st_net** out) {
  if (!out) return create_fail(ST_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  if (!layers || n_layers < 1)
    return create_fail(ST_ERR_INVALID_ARG, "no layers");
  if (batch < 1 || in_h < 1 || in_w < 1 || in_c < 1)
    return create_fail(ST_ERR_INVALID_ARG, "input shape must be positive");
  if (max_frames < 1 || max_frames > kMaxChunkFrames)
    return create_fail(ST_ERR_INVALID_ARG, "max_frames must be in [1, 32]");
  if (dtype != ST_F32 && dtype != ST_F16 && dtype != ST_BF16)
    return create_fail(ST_ERR_INVALID_ARG, "unknown dtype");
  if (flags & ~(uint32_t)(ST_NET_RESIDUAL_CARRY | ST_NET_FROZEN_SE |
                          ST_NET_BF16_STATE))
    return create_fail(ST_ERR_INVALID_ARG, "unknown flag");
  const bool carry = (flags & ST_NET_RESIDUAL_CARRY) != 0;
  const bool frozen_se = (flags & ST_NET_FROZEN_SE) != 0;
  const bool bf16_state = (flags & ST_NET_BF16_STATE) != 0;
  if (carry && bf16_state)
    return create_fail(ST_ERR_UNSUPPORTED,
                       "a bf16 state with residual carry is not supported");
  if (carry && frozen_se)
    return create_fail(ST_ERR_INVALID_ARG,
                       "residual carry and frozen squeeze-excitation are "
                       "exclusive");
  const int64_t F = max_frames;
  if ((int64_t)batch * in_h * in_w * F >= (int64_t)1 << 31)
    return create_fail(ST_ERR_INVALID_ARG, "input grid exceeds 2^31 pixels");
  if ((int64_t)batch * in_h * in_w * F > kMaxGrid)
    return create_fail(ST_ERR_UNSUPPORTED, "input grid above the compaction "
                                           "limit");

  st_net* net = new (std::nothrow) st_net();
  if (!net) return create_fail(ST_ERR_INVALID_ARG, "out of host memory");
  net->dtype = dtype;
  net->esize = esize_of(dtype);
  net->N = batch; net->H = in_h; net->W = in_w; net->C = in_c;
  net->F = max_frames;
  net->carry = carry;
  net->frozen_se = frozen_se;
  net->bf16_state = bf16_state;
  net->layers.resize(n_layers);
  net->tensors.resize(n_layers + 1);

  auto bad = [&](st_status s, int i, const std::string& m) {
    delete net;
    return create_fail(s, "layer " + std::to_string(i) + ": " + m);
  };

  TensorPlan& t0 = net->tensors[0];
  t0.N = batch; t0.H = in_h; t0.W = in_w; t0.C = in_c;
  t0.Cp = (int)round_up(in_c, kChanAlign);
  // a frame of at most 4 channels (RGB) is padded to 4 only: the first
  // convolution's reduction then packs two kernel offsets per 16-byte
  // half-precision vector instead of one offset and 5 zero channels --
  // when only dense convolutions read the frame delta as their input (a
  // depthwise layer or a residual add would read it at the output's
  // 8-channel padding)
  bool input_packable = in_c <= 4;
  for (int i = 0; i < n_layers; ++i)
    if ((layers[i].src == -1 && layers[i].groups > 1) ||
        layers[i].residual_src == -1)
      input_packable = false;
  if (input_packable) t0.Cp = 4;
  t0.grid = (int64_t)batch * in_h * in_w;
  const int kc = gemm_chunk(dtype);

  for (int i = 0; i < n_layers; ++i) {
    const st_layer_desc& d = layers[i];
    LayerPlan& L = net->layers[i];
    L.d = d;
    if (d.src < -1 || d.src >= i)
      return bad(ST_ERR_INVALID_ARG, i, "src must be -1 or an earlier layer");
    const TensorPlan& in = net->tensors[d.src + 1];
    if (d.c_in != in.C)
      return bad(ST_ERR_INVALID_ARG, i, "c_in does not match the producer");
    if (d.c_out < 1) return bad(ST_ERR_INVALID_ARG, i, "c_out < 1");
    if (d.k_h < 1 || d.k_w < 1 || d.s_h < 1 || d.s_w < 1 || d.p_h < 0 ||
        d.p_w < 0)
      return bad(ST_ERR_INVALID_ARG, i, "bad conv geometry");
    if (d.groups < 1) return bad(ST_ERR_INVALID_ARG, i, "groups < 1");
    if (d.groups != 1 && !(d.groups == d.c_in && d.groups == d.c_out))
      return bad(ST_ERR_UNSUPPORTED, i,
                 "only dense (groups=1) and depthwise convolutions");
    if (d.act < ST_ACT_NONE || d.act > ST_ACT_SILU)
      return bad(ST_ERR_INVALID_ARG, i, "unknown activation");
    if (d.se_mid < 0) return bad(ST_ERR_INVALID_ARG, i, "se_mid < 0");
    if (d.se_mid > 0 && (!d.se_w1 || !d.se_w2))
      return bad(ST_ERR_INVALID_ARG, i, "squeeze-excitation weights missing");
    if (d.se_mid > 0 && (d.pool_k_h > 0 || d.pool_k_w > 0))
      return bad(ST_ERR_UNSUPPORTED, i, "squeeze-excitation with a pool");
    if (!d.weight) return bad(ST_ERR_INVALID_ARG, i, "weight is NULL");
    L.Hi = in.H; L.Wi = in.W;
    int64_t ho = out_size(in.H, d.k_h, d.s_h, d.p_h);
    int64_t wo = out_size(in.W, d.k_w, d.s_w, d.p_w);
    if (ho < 1 || wo < 1)
      return bad(ST_ERR_INVALID_ARG, i, "empty conv output");
    L.Ho = (int)ho; L.Wo = (int)wo;
    L.pool = d.pool_k_h > 0 || d.pool_k_w > 0;
    if (L.pool && bf16_state)
      return bad(ST_ERR_UNSUPPORTED, i,
                 "a bf16 state is not supported for max-pooled layers");
    if (L.pool) {
      if (d.pool_k_h < 1 || d.pool_k_w < 1 || d.pool_s_h < 1 ||
          d.pool_s_w < 1 || d.pool_p_h < 0 || d.pool_p_w < 0 ||
          2 * d.pool_p_h > d.pool_k_h || 2 * d.pool_p_w > d.pool_k_w)
        return bad(ST_ERR_INVALID_ARG, i, "bad pool geometry");
      int64_t hp = out_size(ho, d.pool_k_h, d.pool_s_h, d.pool_p_h);
      int64_t wp = out_size(wo, d.pool_k_w, d.pool_s_w, d.pool_p_w);
      if (hp < 1 || wp < 1)
        return bad(ST_ERR_INVALID_ARG, i, "empty pool output");
      L.Hp = (int)hp; L.Wp = (int)wp;
    } else {
      L.Hp = L.Ho; L.Wp = L.Wo;
    }
    if (d.residual_src != -2) {
      if (d.residual_src < -1 || d.residual_src >= i)
        return bad(ST_ERR_INVALID_ARG, i, "bad residual_src");
      const TensorPlan& r = net->tensors[d.residual_src + 1];
      if (r.H != L.Ho || r.W != L.Wo || r.C != d.c_out)
        return bad(ST_ERR_INVALID_ARG, i,
                   "residual shape differs from the conv output");
    }
    L.K = d.k_h * d.k_w;
    if (L.K > 64)
      return bad(ST_ERR_UNSUPPORTED, i, "kernels with more than 64 offsets");
    L.cin_p = in.Cp;
    L.cout_p = (int)round_up(d.c_out, kChanAlign);
    L.dw = d.groups > 1;
    L.ktot = (int64_t)L.K * L.cin_p;
    L.ktot_p = round_up(L.ktot, kc);
    L.conv_grid = (int64_t)batch * L.Ho * L.Wo;
    L.se = d.se_mid > 0;
    L.se_mid = d.se_mid;
    if (L.se && L.cout_p > kSeMaxChannels)
      return bad(ST_ERR_UNSUPPORTED, i,
                 "squeeze-excitation on more than 2048 channels");
    // with residual carry every layer keeps its pre-activation (a layer
    // without non-linearity emits P_new minus the consumers' view)
    L.stateful = d.act != ST_ACT_NONE || L.pool || L.se ||
                 i == n_layers - 1 || carry;
    L.mode = (L.pool || L.se) ? kModeDefer
                              : (L.stateful ? kModeState : kModeLinear);
    L.ident = d.k_h == 1 && d.k_w == 1 && d.s_h == 1 && d.s_w == 1 &&
              d.p_h == 0 && d.p_w == 0 && d.residual_src == -2;
    net->tensors[d.src + 1].consumers.push_back({i, 0});
    if (d.residual_src != -2)
      net->tensors[d.residual_src + 1].consumers.push_back({i, 1});
    TensorPlan& t = net->tensors[i + 1];
    t.N = batch; t.H = L.Hp; t.W = L.Wp; t.C = d.c_out; t.Cp = L.cout_p;
    t.grid = (int64_t)batch * L.Hp * L.Wp;
    if (L.conv_grid * F >= ((int64_t)1 << 31) / std::max(L.K, 1))
      return bad(ST_ERR_INVALID_ARG, i, "rulebook exceeds 2^31 entries");
    if (L.conv_grid * F > kMaxGrid || t.grid * F > kMaxGrid)
      return bad(ST_ERR_UNSUPPORTED, i, "grid above the compaction limit");
  }

  for (int t = 0; t <= n_layers; ++t)
    if (net->tensors[t].consumers.size() > 4) {
      delete net;
      return create_fail(ST_ERR_UNSUPPORTED,
                         "a tensor read by more than 4 layers");
    }

  // ---- workspace layout
  Alloc a;
  const int L_n = n_layers;
  // per tensor: candidate and kept rows; per layer: pairs, own affected
  // list (pooled / SE layers), and kSiteSlots partial counts of the sites
  // a chunk's fused epilogue updated
  net->n_counters = 2 * (L_n + 1) + (2 + kSiteSlots) * L_n;
  net->off_cnt = a.take(sizeof(uint64_t) * net->n_counters);
  net->off_dens = a.take(sizeof(uint64_t) * batch * F);
  // the two sets of compaction look-back statuses
  net->off_tiles = a.take(sizeof(uint32_t) * 2 * kMaxTiles);
  net->off_se_par = a.take(sizeof(int));
  net->off_xhat = a.take((size_t)t0.grid * in_c * net->esize);
  // Per-site buffers of the emitted tensors and rulebooks hold F frames
  // (chunk items: frame t's sites follow frame t-1's); the state, X_hat and
  // squeeze-excitation buffers are per physical site.
  int64_t max_grid = t0.grid * F;
  for (int t = 0; t <= L_n; ++t) {
    TensorPlan& T = net->tensors[t];
    const int64_t items = T.grid * F;
    T.cnt_rows = 2 * t;
    T.cnt_act = 2 * t + 1;
    T.off_rows = a.take((size_t)items * T.Cp * net->esize);
    T.off_rowpix = a.take(sizeof(int32_t) * items);
    T.off_act = a.take(sizeof(int32_t) * items);
    T.off_map = a.take(sizeof(int32_t) * items);
    T.off_rowmax = a.take(sizeof(uint32_t) * items);
    max_grid = std::max(max_grid, items);
  }
  int n_cleanup = L_n + 1;
  size_t part_bytes = 0, chunk_dp_bytes = 0;
  size_t chunk_separt_bytes = 0, chunk_gates_bytes = 0;
  int64_t max_conv_phys = 0;
  for (int i = 0; i < L_n; ++i) {
    LayerPlan& L = net->layers[i];
    TensorPlan& T = net->tensors[i + 1];
    const int64_t citems = L.conv_grid * F;
    L.cnt_pairs = 2 * (L_n + 1) + i;
    L.cnt_sites = 2 * (L_n + 1) + 2 * L_n + kSiteSlots * i;
    max_grid = std::max(max_grid, citems);
    max_conv_phys = std::max(max_conv_phys, L.conv_grid);
    if (F > 1 && L.stateful)
      chunk_dp_bytes = std::max<size_t>(chunk_dp_bytes,
                                        sizeof(float) * citems * L.cout_p);
    // pooled and (exact) squeeze-excitation layers keep their affected
    // list apart from their emitted rows; with frozen gates a
    // squeeze-excitation layer emits at its affected sites like any other
    // (its reference pass still defers the update, so it keeps dP)
    if (L.pool || (L.se && !frozen_se)) {
      L.cnt_O = 2 * (L_n + 1) + L_n + i;
      L.off_O = a.take(sizeof(int32_t) * citems);
      L.off_Mo = a.take(sizeof(int32_t) * citems);
      L.off_dP = a.take(sizeof(float) * L.conv_grid * L.cout_p);
      ++n_cleanup;
    } else {
      L.cnt_O = T.cnt_rows;
      L.off_O = T.off_rowpix;
      L.off_Mo = T.off_map;
      if (L.se) L.off_dP = a.take(sizeof(float) * L.conv_grid * L.cout_p);
    }
    L.off_nbr = a.take(sizeof(int32_t) * citems * L.K);
    if (L.stateful)
      L.off_P = a.take((bf16_state ? 2 : sizeof(float)) * L.conv_grid *
                       L.cout_p);
    if (carry) L.off_yhat = a.take(sizeof(float) * T.grid * L.cout_p);
    if (L.dw)
      L.off_w = a.take(sizeof(float) * L.K * L.cout_p);
    else
      L.off_w = a.take((size_t)L.cout_p * L.ktot_p * net->esize);
    L.off_bias = a.take(sizeof(float) * L.cout_p);
    if (!L.dw) {
      const int64_t stages = L.ktot_p / kc;
      if (stages >= kSplitMinLayerStages)
        L.split_max = (int)std::min<int64_t>(kSplitMax, stages / 8);
      part_bytes = std::max<size_t>(
          part_bytes, L.split_max > 1 ? sizeof(float) * L.split_max *
                                            citems * L.cout_p
                                      : 0);
    }
    if (!L.ident) L.off_flags = a.take(round_up(citems, 16));
    if (F > 1 && L.stateful && !L.dw && !L.se)
      L.off_tstart = a.take(sizeof(uint32_t) *
                            (citems / chunk_tile_step(F) + 2));
    if (L.pool) L.off_pflags = a.take(round_up(T.grid * F, 16));
    if (L.se) {
      const int64_t hw = (int64_t)L.Ho * L.Wo;
      L.se_tps = se_threads_per_site(L.cout_p);
      const int64_t lanes = 256 / L.se_tps;
      const int64_t parts =
          std::min<int64_t>(256, std::max<int64_t>(4, kSePartialFloats /
                                                          L.cout_p));
      L.se_chunk = (int)round_up(ceil_div(hw, parts), lanes);
      L.se_nchunk = (int)ceil_div(hw, L.se_chunk);
      L.off_sew1 = a.take(sizeof(float) * L.se_mid * L.cout_p);
      L.off_seb1 = a.take(sizeof(float) * L.se_mid);
      L.off_sew2 = a.take(sizeof(float) * L.cout_p * L.se_mid);
      L.off_seb2 = a.take(sizeof(float) * L.cout_p);
      L.off_ses = a.take(sizeof(float) * 2 * batch * L.cout_p);
      net->has_se = true;
      L.off_sesum = a.take(sizeof(double) * batch * L.cout_p);
      L.off_separt = a.take(sizeof(float) * batch * L.se_nchunk * L.cout_p);
      if (F > 1 && !frozen_se) {
        chunk_separt_bytes = std::max<size_t>(
            chunk_separt_bytes,
            sizeof(float) * F * batch * L.se_nchunk * L.cout_p);
        chunk_gates_bytes = std::max<size_t>(
            chunk_gates_bytes, sizeof(float) * F * batch * L.cout_p);
      }
    }
  }
  net->max_grid = max_grid;
  net->off_flags = a.take(round_up(t0.grid * F, 16));
  if (F > 1) {
    net->off_chunk_dp = a.take(std::max<size_t>(chunk_dp_bytes, 256));
    net->off_chunk_base = a.take(round_up(t0.grid * F, 16));
    net->off_chunk_last = a.take(round_up(t0.grid, 16));
    net->off_chunk_aff = a.take(sizeof(uint32_t) * max_conv_phys);
    if (chunk_separt_bytes) {
      net->off_chunk_separt = a.take(chunk_separt_bytes);
      net->off_chunk_gates = a.take(chunk_gates_bytes);
    }
  }
  net->off_zero = a.take(256);
  const size_t n_t = (size_t)L_n + 1;
  net->off_ibst_theta = a.take(sizeof(double) * n_t);
  net->off_ibst_lo = a.take(sizeof(double) * n_t);
  net->off_ibst_hi = a.take(sizeof(double) * n_t);
  net->off_ibst_thr = a.take(sizeof(float) * n_t);
  net->off_ibst_ctl = a.take(n_t);
  net->off_ibst_sites = a.take(sizeof(int64_t) * n_t);
  net->off_part = a.take(std::max<size_t>(part_bytes, 256));
  net->n_cleanup = n_cleanup;
  net->off_cleanup = a.take(32 * n_cleanup);
  // the reference frame keeps every pixel; without squeeze-excitation
  // (whose gates need the per-image sums its own pass keeps) or residual
  // carry (whose views its list pass rebuilds) it runs dense
  net->dense_ref = !net->has_se && !carry;
  if (net->dense_ref) {
    net->off_refcnt = a.take(sizeof(uint64_t) * net->n_counters);
    net->n_iota = L_n + 1;
    net->off_iota = a.take(16 * (size_t)net->n_iota);
  }
  for (LayerPlan& L : net->layers) {
    // (output, offset) pairs whose input site lies inside the input grid
    const st_layer_desc& d = L.d;
    int64_t pairs = 0;
    for (int ky = 0; ky < d.k_h; ++ky) {
      int64_t ny = 0, nx = 0;
      for (int oy = 0; oy < L.Ho; ++oy) {
        const int64_t iy = (int64_t)oy * d.s_h - d.p_h + ky;
        ny += iy >= 0 && iy < L.Hi;
      }
      for (int kx = 0; kx < d.k_w; ++kx) {
        nx = 0;
        for (int ox = 0; ox < L.Wo; ++ox) {
          const int64_t ix = (int64_t)ox * d.s_w - d.p_w + kx;
          nx += ix >= 0 && ix < L.Wi;
        }
        pairs += ny * nx;
      }
    }
    L.dense_pairs = pairs * batch;
  }
  net->ws_bytes = round_up(a.top, kAlign);
  *out = net;
  return ST_OK;
}

extern "C" st_status st_create_net(const st_layer_desc* layers,
                                   int32_t n_layers, int32_t batch,
                                   int32_t in_h, int32_t in_w, int32_t in_c,
                                   int32_t dtype, st_net** out) {
  return create_impl(layers, n_layers, batch, 1, in_h, in_w, in_c, dtype,
                     0u, out);
}

extern "C" st_status st_create_net_ex(const st_layer_desc* layers,
                                      int32_t n_layers, int32_t batch,
                                      int32_t max_frames, int32_t in_h,
                                      int32_t in_w, int32_t in_c,
                                      int32_t dtype, uint32_t flags,
                                      st_net** out) {
  return create_impl(layers, n_layers, batch, max_frames, in_h, in_w, in_c,
                     dtype, flags, out);
}

extern "C" st_status st_create_net_chunked(const st_layer_desc* layers,
                                           int32_t n_layers, int32_t batch,
                                           int32_t max_frames, int32_t in_h,
                                           int32_t in_w, int32_t in_c,
                                           int32_t dtype, st_net** out) {
  return create_impl(layers, n_layers, batch, max_frames, in_h, in_w, in_c,
                     dtype, 0u, out);
}

extern "C" st_status st_workspace_bytes(const st_net* net, uint64_t* bytes) {
  if (!net || !bytes) return create_fail(ST_ERR_INVALID_ARG, "NULL argument");
  *bytes = net->ws_bytes;
  return ST_OK;
}

extern "C" st_status st_tensor_shape(const st_net* net, int32_t layer,
                                     int32_t* nhwc) {
  if (!net || !nhwc) return create_fail(ST_ERR_INVALID_ARG, "NULL argument");
  if (layer < -1 || layer >= (int)net->layers.size())
    return create_fail(ST_ERR_INVALID_ARG, "layer out of range");
  const TensorPlan& t = net->tensors[layer + 1];
  nhwc[0] = t.N; nhwc[1] = t.H; nhwc[2] = t.W; nhwc[3] = t.C;
  return ST_OK;
}

extern "C" const char* st_last_error(const st_net* net) {
  return net ? net->err.c_str() : g_create_err.c_str();
}
