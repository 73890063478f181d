// gfx950 kernels of the diff-computation path (wave64, MFMA, LDS).
//
//   scan      subtraction X - X_hat, per-pixel truncation mask, ascending
//             compaction with wave ballot + mbcnt prefixes, commit of X_hat
//   rulebook  affected-output marking, compaction, output-major neighbour
//             table (the dense amplification of a sliding window)
//   conv      gather-GEMM-scatter on MFMA over affected output rows, with
//             the state update / non-linearity / delta emission fused into
//             the epilogue; a vector-ALU path for depthwise layers
//   pool      max-pool non-linear handling from old and new state
//   list      truncation of an emitted delta tensor
//
// Determinism: every output row is owned by one tile and its offsets are
// summed in a fixed order; the only atomics are integer counters and an
// unsigned max on the bit pattern of non-negative floats, both
// order-independent.
#include <hip/hip_runtime.h>

#include <mutex>
#include <type_traits>
#include <vector>

#include <cstdint>

#include "st_kernels.h"

namespace st {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

struct bf16_t {
  uint16_t v;
};

// ------------------------------------------------------------ conversions
__device__ __forceinline__ float to_f(float x) { return x; }
__device__ __forceinline__ float to_f(_Float16 x) { return (float)x; }
__device__ __forceinline__ float to_f(bf16_t x) {
  return __uint_as_float((uint32_t)x.v << 16);
}
template <typename T> __device__ __forceinline__ T from_f(float x);
template <> __device__ __forceinline__ float from_f<float>(float x) {
  return x;
}
template <> __device__ __forceinline__ _Float16 from_f<_Float16>(float x) {
  return (_Float16)x;  // hardware conversion, round to nearest even
}
template <> __device__ __forceinline__ bf16_t from_f<bf16_t>(float x) {
  // hardware conversion (gfx950), round to nearest even
  return bf16_t{__builtin_bit_cast(uint16_t, (__bf16)x)};
}
template <typename T> __device__ __forceinline__ T zero_v() {
  return from_f<T>(0.f);
}

// Activation f: 0 identity, 1 ReLU, 2 SiLU (x / (1 + e^-x)).
template <int ACT>
__device__ __forceinline__ float act_c(float x) {
  if constexpr (ACT == 1)
    return __builtin_amdgcn_fmed3f(x, 0.f, __builtin_inff());  // max(x, 0)
  else if constexpr (ACT == 2)
    return x / (1.f + expf(-x));
  else
    return x;
}
__device__ __forceinline__ float act_f(float x, int a) {
  if (a == 1) return act_c<1>(x);
  if (a == 2) return act_c<2>(x);
  return x;
}
// Calls f(std::integral_constant<int, ACT>{}) for the activation act, so
// that f's body is built once per activation.
template <class F>
__device__ __forceinline__ void with_act(int act, F&& f) {
  if (act == 1)
    f(std::integral_constant<int, 1>{});
  else if (act == 2)
    f(std::integral_constant<int, 2>{});
  else
    f(std::integral_constant<int, 0>{});
}

// ------------------------------------------------------------ reductions
__device__ __forceinline__ unsigned wave_sum(unsigned v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Sum over a 256-thread block; every thread receives the total.
__device__ __forceinline__ unsigned block_sum(unsigned v) {
  __shared__ unsigned red[4];
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

__device__ __forceinline__ unsigned lane_prefix(u64 ballot) {
  return __builtin_amdgcn_mbcnt_hi((unsigned)(ballot >> 32),
                                   __builtin_amdgcn_mbcnt_lo((unsigned)ballot,
                                                             0u));
}

__device__ __forceinline__ int64_t read_count(const u64* dev, int64_t host) {
  return dev ? (int64_t)*dev : host;
}

// ============================================================ compaction
// Ascending stream compaction in one pass.  Items are split into tiles of
// `tile` consecutive indices (at most 256 * kMaxItemsPerThread), one block
// per tile.  Each thread owns ceil(tile / 256) consecutive items and
// evaluates them; one block scan gives every kept item its position in the
// tile.  The tile's offset in the output comes from the tiles before it,
// in the same launch: a tile publishes its own count as soon as it has
// evaluated its items, then sums the published counts of its predecessors
// (lookback_offset).  Blocks are dispatched in index order, so every tile a
// block waits for has been dispatched before it, and it publishes without
// waiting on anything.  The statuses start at zero: compactions use two
// status sets in turn, and each one's blocks clear the set it does not use
// (a slice each), for the next compaction; the per-encode reset clears the
// first set.  No block waits for the others to finish.
//
// The predicate's item data (P::Item, from P::load) is requested together
// with the item count -- all loads stay within the capacity `cap`, and which
// items are real is decided once the count has arrived.  With IPT > 0
// (items per thread known at compile time) the items are kept in registers
// until the keep decision.  Dropped items are handed to pred.drop by their
// owner; the kept ones are listed in LDS in position order and emitted by
// the whole block, consecutive threads taking consecutive positions, so
// every lane of a wave runs an emit (emits are the expensive part: rows
// gathered, windows marked, neighbour tables built) and their stores are
// contiguous.  pred.emit re-loads its item (predicates whose emit ignores
// the item let the compiler drop that load); it returns a work count that
// is summed over the block and handed to pred.block_done; pred.finish
// receives the total.
constexpr int kMaxItemsPerThread = 32;
constexpr int kLoadBatch = 8;  // item loads issued together (generic path)
constexpr uint32_t kLbAgg = 1u << 30;  // status: the tile's count is set
constexpr uint32_t kLbVal = kLbAgg - 1;
// Exclusive prefix of a per-thread count over a 256-thread block (wave
// scan with DPP-free shuffles, wave totals through LDS); also returns the
// block total.
__device__ __forceinline__ unsigned block_exclusive_scan(unsigned v,
                                                         unsigned* total) {
  __shared__ unsigned wsum[4];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const unsigned t = __shfl_up(incl, o, 64);
    if (lane >= o) incl += t;
  }
  __syncthreads();
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  unsigned wpre = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    wpre += (w < wave) ? wsum[w] : 0u;
    tot += wsum[w];
  }
  *total = tot;
  return wpre + incl - v;
}

// Bound on a look-back wait, in sleeps of ~128 cycles (~1 s in all): a
// wait never runs that long, as the waited-for tile is already dispatched
// and publishes before it waits for anything; the bound only guarantees
// that every wave exits (a wait that expired would leave its tile's offset
// short of the counts it did not see).
constexpr int kLbSpinLimit = 1 << 23;

// Predicates with P::kRanked cut run-aligned row tiles while they emit: the
// items form runs of pred.run_len() consecutive indices (a chunk's frames of
// one site), the pass's tiles hold whole runs, and where pred.rank_needed
// asks for it the emit hands pred.emit_ranked the number of kept items of
// the same run before the item.
template <class P, class = void>
struct IsRanked : std::false_type {};
template <class P>
struct IsRanked<P, std::void_t<decltype(P::kRanked)>> : std::true_type {};

// Exclusive output offset of tile t of this block (every thread of the
// block must call it; all receive it): publishes the tile's count in
// status[t], then sums the counts of all the tiles before it, which the
// block's threads read side by side (each thread every 256th tile), waiting
// only for counts not yet published.  A tile publishes its count as soon
// as it has evaluated its items, before it waits for anything, so no wait
// depends on another (a chain of published prefixes would make the last
// tile wait for every earlier one in turn).
// The look-back is split in two: lookback_request reads this thread's
// share of the earlier tiles' statuses as soon as the kernel starts (most
// earlier tiles have published by the time they arrive, so the look-back
// costs no round trip of its own); lookback_offset publishes the tile's
// count and polls again only the statuses that were not yet published.
constexpr int kLbQ = kCompactMaxTiles / 256;
__device__ __forceinline__ void lookback_request(const uint32_t* status,
                                                 unsigned t,
                                                 uint32_t (&v)[kLbQ]) {
#pragma unroll
  for (int q = 0; q < kLbQ; ++q) {
    const unsigned j = threadIdx.x + 256u * q;
    v[q] = j < t ? __hip_atomic_load(status + j, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT)
                 : kLbAgg;
  }
}

__device__ __forceinline__ unsigned lookback_offset(uint32_t* status,
                                                    unsigned t,
                                                    unsigned count,
                                                    uint32_t (&v)[kLbQ]) {
  constexpr int Q = kLbQ;
  if (threadIdx.x == 0)
    __hip_atomic_store(status + t, kLbAgg | count, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  unsigned sum = 0;
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const unsigned j = threadIdx.x + 256u * q;
    for (int spins = 0; v[q] == 0u && spins < kLbSpinLimit; ++spins) {
      __builtin_amdgcn_s_sleep(2);
      v[q] = __hip_atomic_load(status + j, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
    }
    sum += v[q] & kLbVal;
  }
  return block_sum(sum);
}

template <class P, int IPT>
__global__ __launch_bounds__(256) void k_compact(const u64* n_dev,
                                                 int64_t n_host, int64_t cap,
                                                 int tile, uint32_t* status,
                                                 uint32_t* clear, u64* out_cnt,
                                                 u64* out_cnt2, P pred) {
  using Item = typename P::Item;
  // tile offsets of the kept items (tile <= kMaxItemsPerThread * 256)
  __shared__ uint16_t kept[kMaxItemsPerThread * 256];
  // IPT > 0: the kept items themselves, in position order (their emit
  // reads them here instead of loading them again)
  __shared__ Item kitem[IPT > 0 ? 256 * IPT : 1];
  const int64_t base = (int64_t)blockIdx.x * tile;
  {
    // this block's slice of the other status set, for the next compaction
    const unsigned per = (kCompactMaxTiles + gridDim.x - 1) / gridDim.x;
    const unsigned lo = blockIdx.x * per;
    const unsigned hi = min(lo + per, (unsigned)kCompactMaxTiles);
    for (unsigned j = lo + threadIdx.x; j < hi; j += 256) clear[j] = 0u;
  }
  const int ipt = IPT > 0 ? IPT : (tile + 255) / 256;
  const int64_t first = base + (int64_t)threadIdx.x * ipt;
  Item it[IPT > 0 ? IPT : 1];
  if constexpr (IPT > 0) {
#pragma unroll
    for (int j = 0; j < IPT; ++j)
      if (first + j < cap) it[j] = pred.load(first + j);
  }
  uint32_t lbv[kLbQ];
  lookback_request(status, blockIdx.x, lbv);
  const int64_t n = read_count(n_dev, n_host);
  if (base >= n) {
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      *out_cnt = 0;
      if (out_cnt2) *out_cnt2 = 0;
      pred.finish(0u);
    }
    return;
  }
  const int64_t end = min(base + (int64_t)tile, n);
  uint32_t keepbits = 0;
  unsigned mine = 0;
  if constexpr (IPT > 0) {
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
      if (first + j < end && pred.keep(it[j])) {
        keepbits |= 1u << j;
        ++mine;
      }
    }
  } else {
    // kLoadBatch items at a time: their loads are issued together
    for (int j0 = 0; j0 < ipt; j0 += kLoadBatch) {
      Item b[kLoadBatch];
#pragma unroll
      for (int u = 0; u < kLoadBatch; ++u)
        if (j0 + u < ipt && first + j0 + u < end)
          b[u] = pred.load(first + j0 + u);
#pragma unroll
      for (int u = 0; u < kLoadBatch; ++u) {
        if (j0 + u < ipt && first + j0 + u < end && pred.keep(b[u])) {
          keepbits |= 1u << (j0 + u);
          ++mine;
        }
      }
    }
  }
  unsigned tile_total = 0;
  unsigned lp = block_exclusive_scan(mine, &tile_total);
  const unsigned off =
      lookback_offset(status, blockIdx.x, tile_total, lbv);
  for (int j = 0; j < ipt; ++j) {
    const int64_t i = first + j;
    if (i >= end) break;
    if (keepbits & (1u << j)) {
      if constexpr (IPT > 0) kitem[lp] = it[j < IPT ? j : 0];
      kept[lp++] = (uint16_t)(i - base);
    } else {
      if constexpr (IPT > 0)
        pred.drop(i, it[j < IPT ? j : 0]);
      else
        pred.drop(i, pred.load(i));
    }
  }
  __syncthreads();
  unsigned work = 0;
  for (unsigned k = threadIdx.x; k < tile_total; k += 256) {
    const int64_t i = base + kept[k];
    Item itm;
    if constexpr (IPT > 0)
      itm = kitem[k];
    else
      itm = pred.load(i);
    if constexpr (IsRanked<P>::value) {
      const unsigned pos = off + k;
      unsigned rank = 0;
      if (pred.rank_needed(pos)) {
        // tiles start on run boundaries, so tile offsets group like items
        const unsigned R = pred.run_len(), g = kept[k] / R;
        while (rank < k && kept[k - 1 - rank] / R == g) ++rank;
      }
      work += pred.emit_ranked(i, pos, itm, rank);
    } else {
      work += pred.emit(i, off + k, itm);
    }
  }
  work = block_sum(work);
  if (threadIdx.x == 0) {
    pred.block_done(work);
    if (end == n) {
      const unsigned total = off + tile_total;
      *out_cnt = total;
      if (out_cnt2) *out_cnt2 = total;
      pred.finish(total);
    }
  }
}

// Tile of a compaction pass: a multiple of 256 items, at least 512, with at
// most `max_tiles` tiles and at most 32 items per thread (the keep bitmask
// of k_compact) -- more tiles (up to kCompactMaxTiles, the status buffer)
// only where 32 items per thread would not cover the capacity.  run > 1: a
// multiple of run instead (whole runs per tile), which may take one item
// per thread more than k_compact holds (compact_runs_fit).
//
// A tile's look-back reads the status of every live tile before it, so
// the reads grow with the square of the live tiles.  The rulebook and
// pooled-site compactions, whose flag arrays keep every tile live and
// whose items are mostly dropped, take fewer, larger tiles
// (kSparseCompactTiles; measured on ResNet-50 chunks: -14% of their time).
// The truncation pass (only the candidates' tiles live) and the frame-delta
// passes (whose per-item loads and emits gain from more blocks) keep up to
// kCompactMaxTiles small tiles.
constexpr int kSparseCompactTiles = 1024;
static int64_t compact_tile(int64_t cap, int run, int max_tiles) {
  int64_t t = (cap + max_tiles - 1) / max_tiles;
  t = (t + 255) / 256 * 256;
  if (t < 512) t = 512;
  const int64_t tmax = 256 * kMaxItemsPerThread;
  if (t > tmax) {
    t = (cap + kCompactMaxTiles - 1) / kCompactMaxTiles;
    t = (t + 255) / 256 * 256;
    if (t < tmax) t = tmax;
  }
  if (run > 1) {
    // the largest multiple of run not above t, unless that takes more
    // than kCompactMaxTiles tiles
    const int64_t d = t - t % run;
    t = (cap + d - 1) / d <= kCompactMaxTiles ? d : d + run;
  }
  return t;
}

static int compact_tiles(int64_t cap, int run, int max_tiles) {
  const int64_t tile = compact_tile(cap, run, max_tiles);
  const int nt = (int)((cap + tile - 1) / tile);
  return nt < 1 ? 1 : nt;
}

bool compact_runs_fit(int64_t cap, int run) {
  return compact_tile(cap, run, kSparseCompactTiles) <=
         256 * kMaxItemsPerThread;
}

// One compaction launch on the kCompactMaxTiles look-back statuses `tiles`;
// it clears the other set, `clear`, for the next compaction.
template <class P>
static void run_compact(const Prof& pf, int cls, hipStream_t s,
                        const u64* n_dev, int64_t n_host, int64_t cap,
                        uint32_t* tiles, uint32_t* clear, u64* out_cnt,
                        u64* out_cnt2, P pred, int run = 0,
                        int max_tiles = kCompactMaxTiles) {
  const int tile = (int)compact_tile(cap, run, max_tiles);
  const int nt = compact_tiles(cap, run, max_tiles);
  prof_begin(pf, cls, s);
  if ((tile + 255) / 256 == 2)
    k_compact<P, 2><<<nt, 256, 0, s>>>(n_dev, n_host, cap, tile, tiles, clear,
                                       out_cnt, out_cnt2, pred);
  else
    k_compact<P, 0><<<nt, 256, 0, s>>>(n_dev, n_host, cap, tile, tiles, clear,
                                       out_cnt, out_cnt2, pred);
  prof_end(pf, cls, s);
}

// Input row of output pixel o at kernel offset k in a dense pass, where
// every tensor's rows are its pixels in order: the input pixel the offset
// reads, or -1 in the padding.
__device__ __forceinline__ int dense_src(const Geo& g, int64_t o, int k) {
  const int64_t hwo = (int64_t)g.Ho * g.Wo;
  const int n = (int)(o / hwo);
  const int rem = (int)(o - n * hwo);
  const int oy = rem / g.Wo, ox = rem - (rem / g.Wo) * g.Wo;
  const int ky = k / g.kw, kx = k - (k / g.kw) * g.kw;
  const int iy = oy * g.sh - g.ph + ky, ix = ox * g.sw - g.pw + kx;
  if (iy < 0 || iy >= g.Hi || ix < 0 || ix >= g.Wi) return -1;
  return (int)(((int64_t)n * g.Hi + iy) * g.Wi + ix);
}

// ------------------------------------------- consumer-side rulebook prep
// When a tensor's kept rows are emitted, the rulebooks of the layers that
// read it are prepared in the same pass: a 1x1 stride-1 convolution gets its
// affected list, map and one-entry neighbour table directly (its affected
// outputs are exactly the kept inputs); any other consumer gets its
// affected output sites marked through its window geometry (or, for a
// residual input, at the same site).
// Marks the outputs whose window holds input item p (n = frame * nimg +
// image); the output flags are site-major over nf frames (site * nf +
// frame), so the compactions that visit items site-major read them in
// order.
__device__ __forceinline__ void mark_window(uint8_t* flags, int p,
                                            const Geo& g, int nimg, int nf) {
  const unsigned hwi = (unsigned)g.Hi * (unsigned)g.Wi;
  const unsigned nn = (unsigned)p / hwi;
  const unsigned rem = (unsigned)p - nn * hwi;
  const int t = (int)(nn / (unsigned)nimg), n = (int)nn - t * nimg;
  const int iy = (int)(rem / (unsigned)g.Wi), ix = (int)rem - iy * g.Wi;
  // outputs o whose window o * s - pad + [0, k) holds the input: o * s in
  // [i + pad - k + 1, i + pad], 0 <= o < Ho (the lower bound by ceiling
  // division, which is 0 or less when the bound is)
  const int ty = iy + g.ph, tx = ix + g.pw;
  const int ly = ty - g.kh + 1, lx = tx - g.kw + 1;
  const int oy0 = ly > 0 ? (ly + g.sh - 1) / g.sh : 0;
  const int ox0 = lx > 0 ? (lx + g.sw - 1) / g.sw : 0;
  const int oy1 = min(ty / g.sh, g.Ho - 1), ox1 = min(tx / g.sw, g.Wo - 1);
  for (int oy = oy0; oy <= oy1; ++oy) {
    const int64_t rowo = ((int64_t)n * g.Ho + oy) * g.Wo;
    for (int ox = ox0; ox <= ox1; ++ox) flags[(rowo + ox) * nf + t] = 1;
  }
}

__device__ __forceinline__ void cons_emit(const ConsList& cl, int p,
                                          unsigned pos, int row) {
  for (int i = 0; i < cl.n; ++i) {
    const Cons& c = cl.c[i];
    if (c.kind == kConsIdent) {
      c.O[pos] = p;
      c.Mo[p] = (int)pos;
      c.nbr[pos] = row;
      if (c.rowmax) c.rowmax[pos] = 0u;
    } else if (c.kind == kConsMark) {
      mark_window(c.flags, p, c.g, c.nimg, c.nf);
    } else if (c.kind == kConsMarkSame) {
      c.flags[(p % c.per) * c.nf + p / c.per] = 1;
    }
  }
}

__device__ __forceinline__ void cons_finish(const ConsList& cl,
                                            unsigned total) {
  for (int i = 0; i < cl.n; ++i)
    if (cl.c[i].kind == kConsIdent) {
      *cl.c[i].cnt_O = total;
      *cl.c[i].pairs = total;
      if (cl.c[i].tstart) {
        const unsigned step = (unsigned)chunk_tile_step(cl.c[i].nf);
        cl.c[i].tstart[(total + step - 1) / step] = total;
      }
    }
}

// ------------------------------------------------------- (a) frame delta
template <typename T>
struct ScanPred {
  const T* x;
  T* xhat;
  T* rows;
  int* rowpix;
  int* act;
  int* map;
  int C, Cp, ref;
  float thr;
  const float* thr_dev;
  ConsList cons;
  // the truncation rule on the pixel's largest |X - X_hat| over channels
  struct Item {
    uint8_t k;
  };
  __device__ Item load(int64_t i) const {
    const float thr = thr_dev ? *thr_dev : this->thr;
    float m = 0.f;
    for (int c = 0; c < C; ++c) {
      float d = to_f(x[i * C + c]) - (ref ? 0.f : to_f(xhat[i * C + c]));
      m = fmaxf(m, fabsf(d));
    }
    return Item{(uint8_t)(m > thr ? 1 : 0)};
  }
  __device__ bool keep(const Item& it) const { return it.k != 0; }
  // kept pixels: gather the delta row, commit the pixel to X_hat
  __device__ unsigned emit(int64_t i, unsigned pos, const Item&) const {
    rowpix[pos] = (int)i;
    act[pos] = (int)i;
    map[i] = (int)pos;
    T* r = rows + (int64_t)pos * Cp;
    for (int c = 0; c < Cp; ++c) {
      if (c < C) {
        const T xv = x[i * C + c];
        const float d = to_f(xv) - (ref ? 0.f : to_f(xhat[i * C + c]));
        r[c] = from_f<T>(d);
        xhat[i * C + c] = xv;
      } else {
        r[c] = zero_v<T>();
      }
    }
    cons_emit(cons, (int)i, pos, (int)pos);
    return 0u;
  }
  __device__ void drop(int64_t, const Item&) const {}
  __device__ void block_done(unsigned) const {}
  __device__ void finish(unsigned total) const { cons_finish(cons, total); }
};

template <typename T>
static void scan_t(const Prof& pf, hipStream_t s, const ScanArgs& a) {
  ScanPred<T> p{(const T*)a.x, (T*)a.xhat, (T*)a.rows, a.rowpix, a.act,
                a.map, a.C, a.Cp, a.ref, a.thr, a.thr_dev, a.cons};
  run_compact(pf, 1 /*ST_K_SCAN_COMPACT*/, s, nullptr, a.npix, a.npix,
              a.tiles, a.tiles_clear, a.cnt_rows, a.cnt_act, p);
}

void launch_scan(const Prof& pf, hipStream_t s, int dtype,
                 const ScanArgs& a) {
  if (dtype == 0)
    scan_t<float>(pf, s, a);
  else if (dtype == 1)
    scan_t<_Float16>(pf, s, a);
  else
    scan_t<bf16_t>(pf, s, a);
}

// ---------------------------------------------------------- (b) rulebook
static int grid_for(int64_t items, int cap_blocks = 4096) {
  int64_t b = (items + 255) / 256;
  if (b < 1) b = 1;
  return (int)(b > cap_blocks ? cap_blocks : b);
}

// Mark every output site reached by an active site through the window
// (used for the pool windows of pooled layers).
__global__ __launch_bounds__(256) void k_mark(const int* list, const u64* n1p,
                                              Geo g, uint8_t* flags, int nimg,
                                              int nf) {
  const int64_t n1 = (int64_t)*n1p;
  for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n1;
       j += (int64_t)gridDim.x * 256)
    mark_window(flags, list[j], g, nimg, nf);
}

void launch_mark(const Prof& pf, int cls, hipStream_t s, const int* list,
                 const u64* n_list, int64_t max_items, Geo g, uint8_t* flags,
                 int nimg, int nf) {
  prof_begin(pf, cls, s);
  k_mark<<<grid_for(max_items), 256, 0, s>>>(list, n_list, g, flags, nimg,
                                              nf);
  prof_end(pf, cls, s);
}

// Run-aligned row tiles (chunk mode): the run holding row x starts at most
// nf - 1 rows earlier; the nf - 1 preceding entries are requested together
// (one round trip) and the run is the unbroken stretch of the same site
// ending at x.
__global__ __launch_bounds__(256) void k_run_tiles(const int* O,
                                                   const u64* nOp,
                                                   int64_t per, int nf,
                                                   uint32_t* tstart) {
  constexpr int kMaxBack = 31;  // nf <= 32
  const int64_t nO = (int64_t)*nOp;
  const int step = chunk_tile_step(nf);
  const int64_t nt = (nO + step - 1) / step;
  const unsigned pu = (unsigned)per;
  for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j <= nt;
       j += (int64_t)gridDim.x * 256) {
    int64_t r = nO;
    if (j < nt) {
      const int64_t x = j * step;
      // rows x - q for q < nb; past that the address is clamped (the loads
      // stay unconditional) and the value ignored
      const int nb = (int)min((int64_t)nf, x + 1);
      int v[kMaxBack + 1];
#pragma unroll
      for (int q = 0; q <= kMaxBack; ++q) v[q] = O[x - min(q, nb - 1)];
      const unsigned site = (unsigned)v[0] % pu;
      int len = 1;
      bool alive = true;
#pragma unroll
      for (int q = 1; q <= kMaxBack; ++q) {
        alive = alive && q < nb && (unsigned)v[q] % pu == site;
        len += alive ? 1 : 0;
      }
      r = x - len + 1;
    }
    tstart[j] = (uint32_t)r;
  }
}

void launch_run_tiles(const Prof& pf, hipStream_t s, const int* O,
                      const u64* nO, int64_t capO, int64_t per, int nf,
                      uint32_t* tstart) {
  prof_begin(pf, 24 /*ST_K_RUN_TILES*/, s);
  k_run_tiles<<<grid_for(capO / chunk_tile_step(nf) + 1, 512), 256, 0, s>>>(
      O, nO, per, nf, tstart);
  prof_end(pf, 24, s);
}

// Compaction order of chunk-mode items (item = frame * per + site): the
// j-th item visited is site j / nf, frame j % nf, so a site's frames come
// out adjacent and in frame order.  nf <= 1: item order.
__device__ __forceinline__ int64_t site_major(int64_t j, int nf,
                                              int64_t per) {
  if (nf <= 1) return j;
  // items stay below 2^31 (grids times frames are bounded at plan time)
  const unsigned jj = (unsigned)j, site = jj / (unsigned)nf;
  return (int64_t)(jj - site * (unsigned)nf) * per + site;
}

// Affected-output compaction.  With `nbr` set, each emitted output also gets
// its output-major neighbour entries nbr[k][o] = row of the input delta at
// the site offset k reads (or -1: padding or inactive site), and the block
// adds its number of valid entries to `pairs`.
struct FlagPred {
  uint8_t* flags;
  int* list;
  int* map;
  uint32_t* rowmax;
  int* nbr;
  const int* map_in;
  int64_t stride;
  Geo g;  // conv geometry: input grid -> this (output) grid
  u64* pairs;
  int nf;
  int64_t per;
  uint32_t* tstart;  // run-aligned row tiles of the emitted list, or NULL
  static constexpr bool kRanked = true;
  struct Item {
    uint8_t f;
  };
  // a run: one site's nf frames (items site * nf + frame)
  __device__ unsigned run_len() const { return (unsigned)nf; }
  __device__ bool rank_needed(unsigned pos) const {
    return tstart && pos % (unsigned)chunk_tile_step(nf) == 0u;
  }
  // tile pos / step starts where the run holding row pos starts
  __device__ unsigned emit_ranked(int64_t j, unsigned pos, const Item& it,
                                  unsigned rank) const {
    if (rank_needed(pos))
      tstart[pos / (unsigned)chunk_tile_step(nf)] = pos - rank;
    return emit(j, pos, it);
  }
  // the flags are site-major: item j's flag is flags[j]
  __device__ Item load(int64_t j) const { return Item{flags[j]}; }
  __device__ bool keep(const Item& it) const { return it.f != 0; }
  __device__ unsigned emit(int64_t j, unsigned pos, const Item&) const {
    const int64_t i = site_major(j, nf, per);
    list[pos] = (int)i;
    map[i] = (int)pos;
    flags[j] = 0;
    if (rowmax) rowmax[pos] = 0u;
    if (!nbr) return 0u;
    // items stay below 2^31 (grids times frames are bounded at plan time)
    const unsigned hwo = (unsigned)g.Ho * (unsigned)g.Wo;
    const unsigned n = (unsigned)i / hwo;
    const unsigned rem = (unsigned)i - n * hwo;
    const int oy = (int)(rem / (unsigned)g.Wo), ox = (int)rem - oy * g.Wo;
    const int K = g.kh * g.kw;
    const int64_t nrow = (int64_t)n * g.Hi;
    unsigned valid = 0;
    // up to 16 window entries at a time: all their loads are issued before
    // any neighbour-table store (the two may alias for the compiler); the
    // offsets' (ky, kx) advance without divisions
    int ky = 0, kx = 0;
    for (int k0 = 0; k0 < K; k0 += 16) {
      int v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int k = k0 + u;
        const int iy = oy * g.sh - g.ph + ky, ix = ox * g.sw - g.pw + kx;
        v[u] = -1;
        if (k < K && iy >= 0 && iy < g.Hi && ix >= 0 && ix < g.Wi)
          v[u] = map_in[(nrow + iy) * g.Wi + ix];
        if (++kx == g.kw) {
          kx = 0;
          ++ky;
        }
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        if (k0 + u < K) {
          nbr[(int64_t)(k0 + u) * stride + pos] = v[u];
          valid += v[u] >= 0 ? 1u : 0u;
        }
      }
    }
    return valid;
  }
  __device__ void drop(int64_t, const Item&) const {}
  __device__ void block_done(unsigned w) const {
    if (pairs && w) atomicAdd(pairs, (u64)w);
  }
  __device__ void finish(unsigned total) const {
    if (!tstart) return;
    const unsigned step = (unsigned)chunk_tile_step(nf);
    tstart[(total + step - 1) / step] = total;
  }
};

void launch_flag_compact(const Prof& pf, int cls, hipStream_t s,
                         const FlagArgs& a) {
  FlagPred p{a.flags, a.list, a.map, a.rowmax, a.nbr, a.map_in, a.stride,
             a.g, a.pairs, a.nf, a.per, a.tstart};
  run_compact(pf, cls, s, nullptr, a.npix, a.npix, a.tiles, a.tiles_clear,
              a.cnt, nullptr,
              p, a.tstart ? a.nf : 0, kSparseCompactTiles);
}

// ------------------------------------------- (c)+(d) convolution epilogue
// --------------------------------------------------- (c) gather-GEMM MFMA
// Output-stationary tile of BM=64 affected rows x BN=64 output channels,
// four waves in a 2x2 arrangement, each owning a 32x32 sub-tile (2x2 MFMA
// 16x16 blocks).  The reduction index r = k * cin_p + ci runs over kernel
// offsets and input channels; per stage KC reduction columns of the
// gathered input rows (A) and of the repacked weights (B, [cout_p][ktot_p])
// are staged through LDS.
//
// Latency hiding: the tile's neighbour indices are staged in LDS once, so a
// stage's gather is a single global round trip; the next active stage's A
// and B vectors are loaded into registers while the MFMAs of the current
// stage run, and the LDS tiles are double buffered (one barrier per stage).
// Stages whose offsets have no active neighbour in the tile are skipped
// (adding exact zeros would not change the sum).  Tiles are assigned so that
// the blocks of one XCD (blocks are dealt round-robin over the 8 XCDs) work
// on consecutive tiles, which share gathered rows in that XCD's L2.
template <typename T> struct MmaCfg;
template <> struct MmaCfg<float> {
  static constexpr int KC = 16, LD = 17;  // scalar LDS rows, conflict-free
};
template <> struct MmaCfg<_Float16> {
  static constexpr int KC = 64, LD = 72;  // 16-byte aligned LDS rows
};
template <> struct MmaCfg<bf16_t> {
  static constexpr int KC = 64, LD = 72;
};

template <typename T>
__device__ __forceinline__ void lds_store16(T* dst, uint4 v);
template <>
__device__ __forceinline__ void lds_store16<float>(float* dst, uint4 v) {
  dst[0] = __uint_as_float(v.x);
  dst[1] = __uint_as_float(v.y);
  dst[2] = __uint_as_float(v.z);
  dst[3] = __uint_as_float(v.w);
}
template <>
__device__ __forceinline__ void lds_store16<_Float16>(_Float16* dst, uint4 v) {
  *(uint4*)dst = v;
}
template <>
__device__ __forceinline__ void lds_store16<bf16_t>(bf16_t* dst, uint4 v) {
  *(uint4*)dst = v;
}

constexpr int kGemmBM = 64, kGemmBN = 64, kXcd = 8, kCUs = 256;

// 8 consecutive storage elements <-> 8 floats (16- or 32-byte aligned).
template <typename T> struct Vec8;
template <> struct Vec8<float> {
  __device__ __forceinline__ static void load(const float* p, float* f) {
    const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
    f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
  // stores the rounded values, returns their largest magnitude
  __device__ __forceinline__ static float store(float* p, const float* f) {
    *(float4*)p = make_float4(f[0], f[1], f[2], f[3]);
    *(float4*)(p + 4) = make_float4(f[4], f[5], f[6], f[7]);
    float m = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) m = fmaxf(m, fabsf(f[e]));
    return m;
  }
};
template <typename T> struct Vec8Half {
  __device__ __forceinline__ static void load(const T* p, float* f) {
    const uint4 v = *(const uint4*)p;
    const T* h = (const T*)&v;
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = to_f(h[e]);
  }
  // stores the rounded values, returns their largest magnitude: rounding
  // to nearest is monotone and odd, so that is the rounded largest
  // magnitude of the unrounded values (one conversion instead of eight)
  __device__ __forceinline__ static float store(T* p, const float* f) {
    uint4 v;
    T* h = (T*)&v;
    float m = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      h[e] = from_f<T>(f[e]);
      m = fmaxf(m, fabsf(f[e]));
    }
    *(uint4*)p = v;
    return to_f(from_f<T>(m));
  }
};
template <> struct Vec8<_Float16> : Vec8Half<_Float16> {};
template <> struct Vec8<bf16_t> : Vec8Half<bf16_t> {};


__device__ __forceinline__ void load8f(const float* p, float* f) {
  Vec8<float>::load(p, f);
}
__device__ __forceinline__ void store8f(float* p, const float* f) {
  *(float4*)p = make_float4(f[0], f[1], f[2], f[3]);
  *(float4*)(p + 4) = make_float4(f[4], f[5], f[6], f[7]);
}

// Pre-activation state storage: f32, or bf16 (nets created with a bf16
// state), which holds every value rounded to nearest even.  `half` is the
// net's choice (uniform); indices count values, not bytes.
__device__ __forceinline__ float state_round(bool half, float x) {
  return half ? to_f(from_f<bf16_t>(x)) : x;
}
__device__ __forceinline__ void state_load8(const float* P, bool half,
                                            int64_t i, float* f) {
  if (half)
    Vec8<bf16_t>::load((const bf16_t*)P + i, f);
  else
    load8f(P + i, f);
}
__device__ __forceinline__ void state_store8(float* P, bool half, int64_t i,
                                             const float* f) {
  if (half)
    (void)Vec8<bf16_t>::store((bf16_t*)P + i, f);
  else
    store8f(P + i, f);
}
__device__ __forceinline__ float4 state_load4(const float* P, bool half,
                                              int64_t i) {
  if (!half) return *(const float4*)(P + i);
  const uint2 v = *(const uint2*)((const bf16_t*)P + i);
  const bf16_t* h = (const bf16_t*)&v;
  return make_float4(to_f(h[0]), to_f(h[1]), to_f(h[2]), to_f(h[3]));
}
__device__ __forceinline__ void state_store4(float* P, bool half, int64_t i,
                                             float4 f) {
  if (!half) {
    *(float4*)(P + i) = f;
    return;
  }
  uint2 v;
  bf16_t* h = (bf16_t*)&v;
  h[0] = from_f<bf16_t>(f.x);
  h[1] = from_f<bf16_t>(f.y);
  h[2] = from_f<bf16_t>(f.z);
  h[3] = from_f<bf16_t>(f.w);
  *(uint2*)((bf16_t*)P + i) = v;
}
// The gate slot in use: base + (*par ^ flip) * sz (two slots of one
// squeeze-excitation layer's per-image gates, chosen by a parity word in
// device memory so that a captured frame replays with either).
__device__ __forceinline__ const float* gate_slot(const float* base,
                                                  const int* par, int64_t sz,
                                                  int flip) {
  return base + (int64_t)((*par) ^ flip) * sz;
}
__device__ __forceinline__ float state_load1(const float* P, bool half,
                                             int64_t i) {
  return half ? to_f(((const bf16_t*)P)[i]) : P[i];
}

// Reduction stages of a layer that hold real (not padding) columns.
template <typename T>
__device__ __forceinline__ int gemm_stages(const ConvArgs& a) {
  constexpr int KC = MmaCfg<T>::KC;
  return min((int)a.ktot_p, (a.K * a.cin_p + KC - 1) / KC * KC) / KC;
}

// Splits of the reduction per output tile for this frame: enough work units
// (tiles x splits) to give every CU several, at most split_max, and at
// least kSplitMinStages stages per split.  The GEMM and its split epilogue
// both derive it from the same device count.
constexpr int kSplitTarget = 1024, kSplitMinStages = 4;
__device__ __forceinline__ int split_count(int64_t ntiles, int nst, int smax) {
  if (smax <= 1 || ntiles <= 0) return 1;
  int64_t sp = (kSplitTarget + ntiles - 1) / ntiles;
  sp = min(sp, (int64_t)smax);
  sp = min(sp, (int64_t)max(1, nst / kSplitMinStages));
  return (int)max(sp, (int64_t)1);
}

// Finishes one thread's share of an output tile -- row eo of the tile,
// columns n0 + ec + [0, 16) -- from the reduced values v: adds the bias
// (reference pass) and the residual delta, then either defers the update
// (mode 1), or updates the f32 state in place and emits f(P_new) - f(P_old)
// (mode 0), or passes the linear delta on (mode 2).  Row maxima are merged
// with device-scope atomics; the last block to finish a row tile (over its
// column tiles) counts the tile's kept rows for the truncation pass.  Every
// thread of the block must call it (it synchronises).
//
// finish_cols does the per-column work of one thread (16 columns of 64) and
// returns the largest magnitude it emitted; finish_rows merges the row
// maxima and counts kept rows.
template <typename T, bool REF, int ACT, class LoadV, class LoadPo,
          class LoadSk>
__device__ __forceinline__ float finish_cols(const ConvArgs& a, LoadV load_v,
                                             LoadPo load_po, LoadSk load_sk,
                                             const bool (&hv)[2], int64_t eo,
                                             int epix, int n0, int ec) {
  const int cout_p = a.cout_p;
  T* dout = (T*)a.dout;
  float rm = 0.f;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (!hv[h]) continue;
    const int n = n0 + ec + 8 * h;
    float v[8], sk[8];
    load_v(h, v);
    load_sk(h, sk);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (REF) v[e] += a.bias[n + e];
      v[e] += sk[e];
    }
    if (a.mode == 1) {
      store8f(a.dP + eo * cout_p + n, v);
      continue;
    }
    if (a.mode == kModeState || a.mode == kModeStateOnly) {
      float po[8], pn[8];
      load_po(h, po);
      if (a.gate) {
        // frozen squeeze-excitation: both values scaled by the gates
        float g[8];
        load8f(gate_slot(a.gate, a.gpar, a.gsz, 0) + (epix / a.gate_hw) *
                   cout_p + n,
               g);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          pn[e] = state_round(a.p16, po[e] + v[e]);
          v[e] = act_c<ACT>(pn[e]) * g[e] - act_c<ACT>(po[e]) * g[e];
        }
      } else if (!REF && a.yhat) {
        // residual carry: against what the consumers received
        float yh[8];
        load8f(a.yhat + (int64_t)epix * cout_p + n, yh);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          pn[e] = state_round(a.p16, po[e] + v[e]);
          v[e] = act_c<ACT>(pn[e]) - yh[e];
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          pn[e] = state_round(a.p16, po[e] + v[e]);
          v[e] = act_c<ACT>(pn[e]) - act_c<ACT>(po[e]);
        }
      }
      state_store8(a.P, a.p16, (int64_t)epix * cout_p + n, pn);
      if (a.mode == kModeStateOnly) continue;
    }
    rm = fmaxf(rm, Vec8<T>::store(dout + eo * cout_p + n, v));
  }
  return rm;
}

// Row maxima of an output tile (rm: this thread's largest emitted
// magnitude over its columns), merged with device-scope atomics.
__device__ __forceinline__ void finish_rows(const ConvArgs& a, float rm,
                                            int64_t eo, bool eok) {
  const int tid = threadIdx.x;
  // the four threads of a row are adjacent lanes
  rm = fmaxf(rm, __shfl_xor(rm, 1, 64));
  rm = fmaxf(rm, __shfl_xor(rm, 2, 64));
  if (eok && (tid & 3) == 0 && a.mode != 1 && rm > 0.f && a.rowmax)
    atomicMax(a.rowmax + eo, __float_as_uint(rm));
}

template <typename T, bool REF, int ACT, class LoadV, class LoadPo,
          class LoadSk>
__device__ __forceinline__ void finish_tile(const ConvArgs& a, LoadV load_v,
                                            LoadPo load_po, LoadSk load_sk,
                                            const bool (&hv)[2], int64_t eo,
                                            bool eok, int epix, int n0,
                                            int ec) {
  const float rm = finish_cols<T, REF, ACT>(a, load_v, load_po, load_sk, hv,
                                            eo, epix, n0, ec);
  finish_rows(a, rm, eo, eok);
}

// Four channels of a delta row stored in the storage type; returns the
// largest magnitude of the rounded values (the rounded largest magnitude,
// as rounding to nearest is monotone and odd).
template <typename T>
__device__ __forceinline__ float store4(T* p, const float* f) {
  float m = 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e) m = fmaxf(m, fabsf(f[e]));
  if constexpr (sizeof(T) == 4) {
    *(float4*)p = make_float4(f[0], f[1], f[2], f[3]);
    return m;
  } else {
    uint2 v;
    T* h = (T*)&v;
#pragma unroll
    for (int e = 0; e < 4; ++e) h[e] = from_f<T>(f[e]);
    *(uint2*)p = v;
    return to_f(from_f<T>(m));
  }
}

// Chunk-state epilogue, for CPT columns per thread (64 / CPT threads per
// run, adjacent lanes).  The runs' states and the rows' residual deltas are
// requested together; the residual deltas are added into Cs (four threads
// per row, 16 columns each); then each run's threads apply its frames in
// order from LDS -- P_t = P_{t-1} + update, emit f(P_t) - f(P_{t-1}) -- and
// store the state once.  Row maxima are merged in LDS (s_rmax, one LDS
// atomic per thread and row, no cross-lane reduction in the frame loop)
// and then with one device atomic per row and column tile.  With an
// active WriteCs, Cs is written by write_cs() once the loads are issued
// (the accumulators go to LDS while the states and residual rows are on
// their way), followed by a barrier.
struct NoCs {
  static constexpr bool kActive = false;
  __device__ void operator()() const {}
};
template <class F>
struct ActiveCs {
  static constexpr bool kActive = true;
  F& f;
  __device__ void operator()() const { f(); }
};

template <typename T, int CPT, bool POOL, class WriteCs>
__device__ __forceinline__ void chunk_tile_runs(const ConvArgs& a, float* Cs,
                                                int cld, const int* s_run,
                                                int nruns, int64_t m0,
                                                int rows, int n0,
                                                const int* s_site,
                                                const int* s_rsk,
                                                unsigned* s_rmax,
                                                const int* s_frm,
                                                WriteCs write_cs) {
  constexpr int TPR = 64 / CPT, Q = CPT / 4;
  const int tid = threadIdx.x;
  const int cout_p = a.cout_p;
  T* dout = (T*)a.dout;
  const T* dskip = (const T*)a.dskip;
  // this thread's run and columns
  const int g = tid / TPR, j = tid - (tid / TPR) * TPR;
  const int c0 = n0 + j * CPT;
  const bool run = g < nruns;
  const int64_t site = run ? s_site[s_run[g]] : 0;
  float P[CPT];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (run && c0 + 4 * q < cout_p)
      v = state_load4(a.P, a.p16, site * cout_p + c0 + 4 * q);
    P[4 * q] = v.x;
    P[4 * q + 1] = v.y;
    P[4 * q + 2] = v.z;
    P[4 * q + 3] = v.w;
  }
  // residual rows: four threads per row, 16 columns each, kept in their
  // storage type until added
  {
    constexpr int SKV = (int)sizeof(T) / 2;  // 16-byte vectors / 8 channels
    const int er = tid >> 2, ec = (tid & 3) * 16;
    const int rsk = er < rows ? s_rsk[er] : -1;
    uint4 sk[2][SKV];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c = n0 + ec + 8 * h;
#pragma unroll
      for (int v = 0; v < SKV; ++v)
        sk[h][v] =
            (rsk >= 0 && c < cout_p)
                ? ((const uint4*)(dskip + (int64_t)rsk * cout_p + c))[v]
                : make_uint4(0u, 0u, 0u, 0u);
    }
    if constexpr (WriteCs::kActive) {
      write_cs();
      __syncthreads();
    }
    if (rsk >= 0) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float f[8];
        Vec8<T>::load((const T*)sk[h], f);
#pragma unroll
        for (int e = 0; e < 8; ++e) Cs[er * cld + ec + 8 * h + e] += f[e];
      }
    }
  }
  __syncthreads();
  const int r0 = run ? s_run[g] : 0, r1 = run ? s_run[g + 1] : 0;
  if constexpr (POOL) {
    // the states after each frame go to the rows' update rows (f32), the
    // run's frames to the site's bit mask; the state itself is committed
    // after the pool emission
    uint32_t bits = 0u;
    for (int r = r0; r < r1; ++r) {
      bits |= 1u << s_frm[r];
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        if (c0 + 4 * q >= cout_p) continue;
        const float4 u = *(const float4*)(Cs + r * cld + (c0 - n0) + 4 * q);
        const float uv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          P[4 * q + e] = state_round(a.p16, P[4 * q + e] + uv[e]);
        *(float4*)(a.dP + (m0 + r) * cout_p + c0 + 4 * q) =
            make_float4(P[4 * q], P[4 * q + 1], P[4 * q + 2], P[4 * q + 3]);
      }
    }
    if (run && j == 0) a.aff[site] = bits;
    return;
  } else {
  // the frames of the run, with the activation fixed at compile time
  auto frames = [&](auto act_tag) {
    constexpr int ACT = decltype(act_tag)::value;
    // four columns at a time; the delta stores take eight (16 bytes) where
    // the thread owns at least eight (the padded width is a multiple of 8)
    constexpr int SV = Q % 2 == 0 ? 8 : 4;
    for (int r = r0; r < r1; ++r) {
      float rm = 0.f;
#pragma unroll
      for (int q2 = 0; q2 < CPT / SV; ++q2) {
        if (c0 + SV * q2 >= cout_p) continue;
        float d[SV];
#pragma unroll
        for (int h = 0; h < SV / 4; ++h) {
          const int q = (SV / 4) * q2 + h;
          const float4 u =
              *(const float4*)(Cs + r * cld + (c0 - n0) + 4 * q);
          const float uv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float po = P[4 * q + e];
            const float pn = state_round(a.p16, po + uv[e]);
            d[4 * h + e] = act_c<ACT>(pn) - act_c<ACT>(po);
            P[4 * q + e] = pn;
          }
        }
        T* dst = dout + (m0 + r) * cout_p + c0 + SV * q2;
        if constexpr (SV == 8)
          rm = fmaxf(rm, Vec8<T>::store(dst, d));
        else
          rm = fmaxf(rm, store4<T>(dst, d));
      }
      if (rm > 0.f) atomicMax(s_rmax + r, __float_as_uint(rm));
    }
  };
  with_act(a.act, frames);
  if (run) {
#pragma unroll
    for (int q = 0; q < Q; ++q)
      if (c0 + 4 * q < cout_p)
        state_store4(a.P, a.p16, site * cout_p + c0 + 4 * q,
                     make_float4(P[4 * q], P[4 * q + 1], P[4 * q + 2],
                                 P[4 * q + 3]));
  }
  }
}

// Chunk-state epilogue: the tile's rows [m0, m0 + rows) are whole site
// runs (a site's frames, in frame order), the f32 accumulators of 64 of
// its columns (from n0) in Cs (row stride cld), the rows' sites and
// residual rows in s_site / s_rsk.  The runs are listed (first call of a
// tile), then each run gets 4, 8 or 16 threads (16, 8 or 4 columns each)
// -- as many as the tile's run count leaves -- so that long runs (sites
// that changed in most frames) still keep the block busy.  A tile of
// several 64-column quarters calls it once per quarter; its row maxima
// gather in s_rmax and the last call merges them into the device row
// maxima.  Every thread of the block must call it.  POOL (a max-pooled
// layer, kModeChunkPool): s_frm holds the rows' frames, and the states
// after each frame go to the rows' update rows instead of deltas.
template <typename T, bool POOL = false, class WriteCs = NoCs>
__device__ __forceinline__ void finish_chunk_tile(const ConvArgs& a,
                                                  float* Cs, int cld,
                                                  int* s_run, int64_t m0,
                                                  int rows, int n0,
                                                  const int* s_site,
                                                  const int* s_rsk,
                                                  unsigned* s_rmax,
                                                  const int* s_frm,
                                                  bool first = true,
                                                  bool last = true,
                                                  WriteCs write_cs = {}) {
  constexpr int BM = kGemmBM;
  const int tid = threadIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // run starts: s_run[0..nruns) (wave 0 lists them), s_run[nruns] = rows,
  // s_run[BM + 1] = nruns
  if (first && tid < BM) s_rmax[tid] = 0u;
  if (first && wave == 0) {
    const bool opens =
        lane < rows && (lane == 0 || s_site[lane] != s_site[lane - 1]);
    const u64 starts = __ballot(opens);
    const int nr = __popcll(starts);
    if (opens) s_run[lane_prefix(starts)] = lane;
    if (lane == 0) {
      s_run[nr] = rows;
      s_run[BM + 1] = nr;
      // every run lies in one row tile: its first column tile counts it
      if (n0 == 0 && nr)
        atomicAdd(a.sites + blockIdx.x % kSiteSlots, (u64)nr);
    }
  }
  __syncthreads();
  const int nruns = s_run[BM + 1];
  if (nruns > 32)
    chunk_tile_runs<T, 16, POOL>(a, Cs, cld, s_run, nruns, m0, rows, n0,
                                 s_site, s_rsk, s_rmax, s_frm, write_cs);
  else if (nruns > 16)
    chunk_tile_runs<T, 8, POOL>(a, Cs, cld, s_run, nruns, m0, rows, n0,
                                s_site, s_rsk, s_rmax, s_frm, write_cs);
  else
    chunk_tile_runs<T, 4, POOL>(a, Cs, cld, s_run, nruns, m0, rows, n0,
                                s_site, s_rsk, s_rmax, s_frm, write_cs);
  if (last) {
    __syncthreads();
    if (tid < rows && s_rmax[tid])
      atomicMax(a.rowmax + m0 + tid, s_rmax[tid]);
  }
}

// Tile shape of the gather-GEMM: 64 affected rows by 64 output channels,
// four waves (256 threads) in a 2x2 arrangement, each a 32x32 sub-tile;
// reduction stages of MmaCfg<T>::KC columns; four blocks per CU.
template <typename T> struct GemmTile {
  static constexpr int BM = kGemmBM, BN = kGemmBN;
  static constexpr int KC = MmaCfg<T>::KC, LD = MmaCfg<T>::LD;
  static constexpr int WAVES_M = 2, WAVES_N = 2;
  static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;
  static constexpr int IM = WM / 16, JN = WN / 16;
  static constexpr int BLOCKS_PER_CU = 4;
};

// Reduction stages of a layer that hold real (not padding) columns, for
// stages of KC columns.
template <int KC>
__device__ __forceinline__ int gemm_stages_kc(const ConvArgs& a) {
  return min((int)a.ktot_p, (a.K * a.cin_p + KC - 1) / KC * KC) / KC;
}

// SPLIT: the layer's reduction may be split (split_max > 1); every unit
// then writes its partial tile (even when this frame needs one split) and
// the split epilogue finishes the tiles, so no epilogue state is held
// through the reduction.
// The register budget follows the blocks each CU holds: four waves per
// SIMD.
template <typename T, bool REF, bool ALIGNED, bool SPLIT, bool CHUNK,
          bool POOL = false>
__global__ __launch_bounds__(256)
__attribute__((amdgpu_waves_per_eu(GemmTile<T>::BLOCKS_PER_CU)))
void k_conv_gemm(ConvArgs a) {
  using G = GemmTile<T>;
  constexpr int BM = G::BM, BN = G::BN;
  constexpr int KC = G::KC, LD = G::LD;
  constexpr int IM = G::IM, JN = G::JN;
  constexpr int VEC = 16 / (int)sizeof(T);
  constexpr int VPR = KC / VEC;           // 16-byte vectors per staged row
  constexpr int AV = BM * VPR / 256;      // A vectors per thread per stage
  constexpr int BV = BN * VPR / 256;      // B vectors per thread per stage
  constexpr int NQ = BN / kGemmBN;        // 64-column quarters per tile
  constexpr int CLD = kGemmBN + 4;        // f32 accumulator row (a quarter)
  constexpr size_t AB_BYTES = 2ull * (BM + BN) * LD * sizeof(T);
  constexpr size_t C_BYTES = (size_t)BM * CLD * sizeof(float);
  static_assert(AV >= 1 && BV >= 1, "stage vectors");
  __shared__ __align__(16) char smem[AB_BYTES > C_BYTES ? AB_BYTES : C_BYTES];
  // the units' kernel-offset masks, two in turn: a unit clears the one
  // the next unit fills, so no barrier orders the clearing
  __shared__ u64 s_kmask[2];
  __shared__ int s_site[BM], s_rsk[BM], s_run[BM + 2], s_frm[POOL ? BM : 1];
  __shared__ unsigned s_rmax[BM];
  // dense pass: window origin of each row of the tile (n * Hi, oy * sh - ph,
  // ox * sw - pw) and each kernel offset's (ky, kx), so that a neighbour
  // costs no division
  __shared__ int s_dorg[REF ? 3 * BM : 1], s_koff[REF ? 64 : 1];
  extern __shared__ int s_nbr[];          // [K][BM]
  // LDS carve-up: A[2][BM][LD], B[2][BN][LD]; the f32 accumulator tile of
  // the epilogue (one 64-column quarter at a time) reuses the same bytes
  T* const sA = (T*)smem;
  T* const sB = (T*)smem + 2 * BM * LD;
  float* const Cs = (float*)smem;

  const T* din = (const T*)a.din;
  const T* wt = (const T*)a.w;
  const T* zvec = (const T*)a.zero;
  const T* dskip = (const T*)a.dskip;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l16 = lane & 15, lg = lane >> 4;
  const int64_t nO = a.dense ? a.capO : (int64_t)*a.nO;
  // row tiles: 64 rows each, or (chunk-state mode) aligned to site runs
  const bool runs = CHUNK;  // the launcher pairs tstart with this mode
  const int rstep = runs ? chunk_tile_step(a.nf) : BM;
  const int64_t tiles_m = (nO + rstep - 1) / rstep;
  const int tiles_n = (a.cout_p + BN - 1) / BN;
  const int64_t ntiles = tiles_m * tiles_n;
  const int K = a.K, cin_p = a.cin_p, cout_p = a.cout_p;
  const int ktot_p = (int)a.ktot_p;
  // reduction stages that hold real (not padding) columns; with ALIGNED
  // (cin_p a multiple of KC) every stage lies within one kernel offset and
  // offset k covers stages [k * spk, (k + 1) * spk)
  const int nst = gemm_stages_kc<KC>(a);
  const int spk = ALIGNED ? cin_p / KC : 1;
  // work units: (split, tile) pairs, split-major, so that neighbouring
  // tiles of one split (which gather the same input rows) stay together
  const int S = SPLIT ? split_count(ntiles, nst, a.split_max) : 1;
  const int64_t nunits = ntiles * S;
  // XCD-aware order: blocks are dealt round-robin over the kXcd XCDs
  // (gridDim.x is a multiple of kXcd); the unit range is cut into kXcd
  // contiguous chunks, one per XCD, and the XCD's blocks stride through
  // their chunk, so neighbouring tiles (which share gathered rows) meet in
  // one L2 and every XCD gets work however few units there are.
  const int chunk = (int)((nunits + kXcd - 1) / kXcd);
  const int xcd = blockIdx.x % kXcd;
  const int u_end = (int)min(nunits, (int64_t)(xcd + 1) * chunk);
  const int per_xcd = gridDim.x / kXcd;
  // epilogue ownership: thread -> row em, columns [ec, ec + 16) of a
  // 64-column quarter
  const int em = tid >> 2, ec = (tid & 3) * 16;
  if (REF && a.dense && tid < K) {
    const int ky = tid / a.g.kw;
    s_koff[tid] = (ky << 16) | (tid - ky * a.g.kw);
  }

  // run-aligned row tiles (chunk-state mode): a unit's bounds are fetched
  // during the previous unit, so they have arrived when it starts
  const int u_first = xcd * chunk + blockIdx.x / kXcd;
  unsigned nb_lo = 0u, nb_hi = 0u;
  if (CHUNK && u_first < u_end) {
    const int tm = (int)((unsigned)u_first / (unsigned)tiles_n);
    nb_lo = a.tstart[tm];
    nb_hi = a.tstart[tm + 1];
  }
  if (tid == 0) s_kmask[0] = 0ull;
  int kp = 0;  // this unit's offset mask
  for (int u = u_first; u < u_end; u += per_xcd, kp ^= 1) {
    // this unit's split and tile, and its reduction stages [st_lo, st_hi)
    const int sp = SPLIT ? (int)((unsigned)u / (unsigned)ntiles) : 0;
    const int t = SPLIT ? u - sp * (int)ntiles : u;
    const int st_lo = SPLIT ? (int)((int64_t)sp * nst / S) : 0;
    const int st_hi = SPLIT ? (int)((int64_t)(sp + 1) * nst / S) : nst;
    const int tm_i = (int)((unsigned)t / (unsigned)tiles_n);
    const int64_t m0 =
        runs ? (int64_t)(unsigned)__builtin_amdgcn_readfirstlane((int)nb_lo)
             : (int64_t)tm_i * BM;
    const int64_t m1 =
        runs ? (int64_t)(unsigned)__builtin_amdgcn_readfirstlane((int)nb_hi)
             : min(m0 + BM, nO);
    const int n0 = (t - tm_i * tiles_n) * BN;

    __syncthreads();  // previous tile's LDS reads are complete
    if (tid == 0) s_kmask[kp ^ 1] = 0ull;
    // this thread's epilogue row; its old state and residual are fetched
    // now so that they arrive while the reduction runs
    const int64_t eo = m0 + em;
    const bool eok = eo < m1;
    const int epix = !eok ? 0 : a.dense ? (int)eo : a.O[eo];
    if (REF && a.dense && tid < BM) {
      const int64_t o = m0 + tid;
      const unsigned op = o < m1 ? (unsigned)o : 0u;
      const unsigned hwo = (unsigned)a.g.Ho * (unsigned)a.g.Wo;
      const unsigned n = op / hwo, rem = op - n * hwo;
      const unsigned oy = rem / (unsigned)a.g.Wo;
      const unsigned ox = rem - oy * (unsigned)a.g.Wo;
      s_dorg[tid] = (int)n * a.g.Hi;
      s_dorg[BM + tid] = (int)oy * a.g.sh - a.g.ph;
      s_dorg[2 * BM + tid] = (int)ox * a.g.sw - a.g.pw;
    }
    if (REF) __syncthreads();  // the window origins are written
    u64 my = 0ull;
    for (int e = tid; e < BM * K; e += 256) {
      const int k = e / BM, m = e - (e / BM) * BM;
      const int64_t o = m0 + m;
      int src = -1;
      if (o < m1) {
        if (REF && a.dense) {
          const int ko = s_koff[k];
          const int iy = s_dorg[BM + m] + (ko >> 16);
          const int ix = s_dorg[2 * BM + m] + (ko & 0xffff);
          if (iy >= 0 && iy < a.g.Hi && ix >= 0 && ix < a.g.Wi)
            src = (s_dorg[m] + iy) * a.g.Wi + ix;
        } else {
          src = a.nbr[(int64_t)k * a.stride + o];
        }
      }
      s_nbr[e] = src;
      if (src >= 0) my |= 1ull << k;
    }
    if (my) atomicOr(&s_kmask[kp], my);
    __syncthreads();
    const u64 kmask = s_kmask[kp];
    if (CHUNK && u + per_xcd < u_end) {
      const int tm = (int)((unsigned)(u + per_xcd) / (unsigned)tiles_n);
      nb_lo = a.tstart[tm];
      nb_hi = a.tstart[tm + 1];
    }

    auto stage_active = [&](int st) {
      const int klo = (st * KC) / cin_p;
      int khi = (st * KC + KC - 1) / cin_p;
      if (khi > K - 1) khi = K - 1;
      const int span = khi - klo + 1;
      const u64 bits = (span >= 64 ? ~0ull : ((1ull << span) - 1)) << klo;
      return (kmask & bits) != 0ull;
    };
    auto next_k = [&](int k) {
      if (k >= K) return K;
      const u64 mk = kmask >> k;
      return mk ? k + __builtin_ctzll(mk) : K;
    };
    // Stage iterator.  ALIGNED: stages are walked as (offset kc, sub-stage)
    // pairs, jumping over offsets without active neighbours by a bit scan of
    // the offset mask; otherwise stage by stage with the span test.
    struct It {
      int kc, sub, st;
    };
    auto first_stage = [&]() {
      It it{0, 0, st_lo};
      if (ALIGNED && !SPLIT) {
        it.kc = next_k(0);
        it.st = it.kc < K ? it.kc * spk : st_hi;
      } else if (ALIGNED) {
        it.kc = st_lo / spk;
        it.sub = st_lo - it.kc * spk;
        if (!((kmask >> it.kc) & 1ull)) {
          it.kc = next_k(it.kc + 1);
          it.sub = 0;
        }
        it.st = it.kc < K ? min(it.kc * spk + it.sub, st_hi) : st_hi;
      } else {
        while (it.st < st_hi && !stage_active(it.st)) ++it.st;
      }
      return it;
    };
    auto advance = [&](It it) {
      if (it.st >= st_hi) return it;
      if (ALIGNED) {
        if (++it.sub == spk) {
          it.kc = next_k(it.kc + 1);
          it.sub = 0;
        }
        if (SPLIT)
          it.st = it.kc < K ? min(it.kc * spk + it.sub, st_hi) : st_hi;
        else
          it.st = it.kc < K ? it.kc * spk + it.sub : st_hi;
      } else {
        ++it.st;
        while (it.st < st_hi && !stage_active(it.st)) ++it.st;
      }
      return it;
    };

    // Loads of one stage into a register slot.  Every lane always issues
    // its loads (inactive neighbours, columns past cout_p and stages past
    // the end read a zero vector), so the loads of the next two stages can
    // stay in flight while the current one is staged and multiplied.
    // ALIGNED: the gathered rows of this thread's A vectors (row pointers,
    // NULL for an inactive neighbour) are kept for the current kernel
    // offset, so a stage within it neither reads the neighbour table nor
    // rebuilds the row addresses.
    const T* arow[AV];
    int arow_kc = -1;
    auto load_stage = [&](const It& it, uint4 (&ra)[AV], uint4 (&rb)[BV]) {
      const bool live = it.st < st_hi;
      const int r0 = it.st * KC;
      if (ALIGNED && live && it.kc != arow_kc) {
        arow_kc = it.kc;
#pragma unroll
        for (int q = 0; q < AV; ++q) {
          const int m = (tid + q * 256) / VPR;
          const int src = s_nbr[arow_kc * BM + m];
          arow[q] = src >= 0 ? din + (int64_t)src * cin_p : nullptr;
        }
      }
#pragma unroll
      for (int q = 0; q < AV; ++q) {
        const int v = tid + q * 256;
        const int m = v / VPR, cv = v - (v / VPR) * VPR;
        if (ALIGNED) {
          const T* row = live ? arow[q] : nullptr;
          ra[q] = *(const uint4*)(row ? row + it.sub * KC + cv * VEC : zvec);
          continue;
        }
        int k, ci;
        {
          const int r = r0 + cv * VEC;
          k = r / cin_p;
          ci = r - k * cin_p;
        }
        if (!ALIGNED && VEC == 8 && cin_p == 4) {
          // a frame of 4 (padded) channels: the vector holds offsets k and
          // k + 1, four channels each, from two gathered rows
          const int s0 = (live && k < K) ? s_nbr[k * BM + m] : -1;
          const int s1 = (live && k + 1 < K) ? s_nbr[(k + 1) * BM + m] : -1;
          const T* p0 = s0 >= 0 ? din + (int64_t)s0 * 4 : zvec;
          const T* p1 = s1 >= 0 ? din + (int64_t)s1 * 4 : zvec;
          const uint2 lo = *(const uint2*)p0, hi = *(const uint2*)p1;
          ra[q] = make_uint4(lo.x, lo.y, hi.x, hi.y);
          continue;
        }
        const int src = (live && k < K) ? s_nbr[k * BM + m] : -1;
        const T* pa = src >= 0 ? din + (int64_t)src * cin_p + ci : zvec;
        ra[q] = *(const uint4*)pa;
      }
#pragma unroll
      for (int q = 0; q < BV; ++q) {
        const int v = tid + q * 256;
        const int nn = v / VPR, cv = v - (v / VPR) * VPR;
        const int n = n0 + nn;
        const T* pb = (live && n < cout_p)
                          ? wt + (int64_t)n * ktot_p + r0 + cv * VEC
                          : zvec;
        rb[q] = *(const uint4*)pb;
      }
    };
    auto store_stage = [&](int buf, const uint4 (&ra)[AV],
                           const uint4 (&rb)[BV]) {
#pragma unroll
      for (int q = 0; q < AV; ++q) {
        const int v = tid + q * 256;
        const int m = v / VPR, cv = v - (v / VPR) * VPR;
        lds_store16<T>(sA + buf * BM * LD + m * LD + cv * VEC, ra[q]);
      }
#pragma unroll
      for (int q = 0; q < BV; ++q) {
        const int v = tid + q * 256;
        const int nn = v / VPR, cv = v - (v / VPR) * VPR;
        lds_store16<T>(sB + buf * BN * LD + nn * LD + cv * VEC, rb[q]);
      }
    };

    v4f acc[IM][JN];
#pragma unroll
    for (int i = 0; i < IM; ++i)
#pragma unroll
      for (int j = 0; j < JN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](int buf) {
      const T* Ab = sA + buf * BM * LD + wm * G::WM * LD;
      const T* Bb = sB + buf * BN * LD + wn * G::WN * LD;
      if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int kk = 0; kk < KC; kk += 4) {
          float af[IM], bf[JN];
#pragma unroll
          for (int i = 0; i < IM; ++i)
            af[i] = Ab[(i * 16 + l16) * LD + kk + lg];
#pragma unroll
          for (int j = 0; j < JN; ++j)
            bf[j] = Bb[(j * 16 + l16) * LD + kk + lg];
#pragma unroll
          for (int i = 0; i < IM; ++i)
#pragma unroll
            for (int j = 0; j < JN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                  af[i], bf[j], acc[i][j], 0, 0, 0);
        }
      } else {
#pragma unroll
        for (int kk = 0; kk < KC; kk += 32) {
          uint4 av[IM], bv[JN];
#pragma unroll
          for (int i = 0; i < IM; ++i)
            av[i] = *(const uint4*)(Ab + (i * 16 + l16) * LD + kk + 8 * lg);
#pragma unroll
          for (int j = 0; j < JN; ++j)
            bv[j] = *(const uint4*)(Bb + (j * 16 + l16) * LD + kk + 8 * lg);
#pragma unroll
          for (int i = 0; i < IM; ++i) {
#pragma unroll
            for (int j = 0; j < JN; ++j) {
              if constexpr (__is_same(T, _Float16)) {
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                    __builtin_bit_cast(v8h, av[i]),
                    __builtin_bit_cast(v8h, bv[j]), acc[i][j], 0, 0, 0);
              } else {
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    __builtin_bit_cast(v8bf, av[i]),
                    __builtin_bit_cast(v8bf, bv[j]), acc[i][j], 0, 0, 0);
              }
            }
          }
        }
      }
    };

    // this thread's output row's residual row, requested now so that it
    // arrives during the reduction; (chunk-state mode) the row's site
    const int rsk = (!SPLIT && a.mskip && eok)
                        ? (a.dense ? epix : a.mskip[epix])
                        : -1;
    if (CHUNK && (tid & 3) == 0) {
      s_site[em] = eok ? (int)((unsigned)epix % (unsigned)a.per) : -1;
      if (POOL) s_frm[em] = eok ? (int)((unsigned)epix / (unsigned)a.per) : 0;
    }

    // two stages in flight: slot 0 / slot 1 alternate
    uint4 ra0[AV], rb0[BV], ra1[AV], rb1[BV];
    It ia = first_stage();
    load_stage(ia, ra0, rb0);
    It ib = advance(ia);
    load_stage(ib, ra1, rb1);
    int buf = 0;
    while (ia.st < st_hi) {
      store_stage(buf, ra0, rb0);
      __syncthreads();
      const It ic = advance(ib);
      load_stage(ic, ra0, rb0);
      compute(buf);
      buf ^= 1;
      if (ib.st >= st_hi) break;
      store_stage(buf, ra1, rb1);
      __syncthreads();
      const It id = advance(ic);
      load_stage(id, ra1, rb1);
      compute(buf);
      buf ^= 1;
      ia = ic;
      ib = id;
    }

    // ---- fused epilogue.  The accumulator tile goes through LDS, one
    // 64-column quarter at a time, so that each thread finishes 16
    // contiguous columns of one row: full-width state loads/stores and
    // 16-byte delta stores.  MFMA 16x16 block layout: D[row = 4*lg + r]
    // [col = l16]; the four waves' 32x32 sub-tiles make the 64x64 tile.
    if (CHUNK && (tid & 3) == 0) s_rsk[em] = rsk;
    // (reference pass, half storage) the residual row's 16 columns of this
    // thread are requested before the accumulators go through LDS, so that
    // they arrive meanwhile; a missing row reads as +0, which adds exactly
    // what the zero residual adds
    constexpr bool kSkPre = REF && !SPLIT && !CHUNK && sizeof(T) == 2;
    uint4 skr[kSkPre ? 2 : 1] = {};
    if constexpr (kSkPre) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
        if (rsk >= 0 && n0 + ec + 8 * h < cout_p)
          skr[h] = *(const uint4*)(dskip + (int64_t)rsk * cout_p + n0 + ec +
                                   8 * h);
    }
    auto write_acc = [&]() {
#pragma unroll
      for (int i = 0; i < IM; ++i)
#pragma unroll
        for (int j = 0; j < JN; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            Cs[(wm * G::WM + i * 16 + 4 * lg + r) * CLD + wn * G::WN +
               j * 16 + l16] = acc[i][j][r];
    };
    if constexpr (CHUNK && NQ == 1) {
      // the run listing's barrier also ends the reduction's LDS reads;
      // the accumulators go to LDS while the states and residual rows
      // are requested
      finish_chunk_tile<T, POOL>(a, Cs, CLD, s_run, m0, (int)(m1 - m0), n0,
                                 s_site, s_rsk, s_rmax, s_frm, true, true,
                                 ActiveCs<decltype(write_acc)>{write_acc});
      continue;
    }
    float rm_all = 0.f;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      __syncthreads();  // the staged tiles are read
      write_acc();
      __syncthreads();
      const int nq = n0 + q * kGemmBN;
      const float* crow = Cs + em * CLD + ec;
      bool hv[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) hv[h] = eok && nq + ec + 8 * h < cout_p;
      if constexpr (SPLIT) {
        // partial tile of split sp, reduced by the split epilogue
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          if (!hv[h]) continue;
          float v[8];
          load8f(crow + 8 * h, v);
          store8f(a.part + ((int64_t)sp * a.capO + eo) * cout_p + nq + ec +
                      8 * h,
                  v);
        }
      } else if constexpr (CHUNK) {
        finish_chunk_tile<T, POOL>(a, Cs, CLD, s_run, m0, (int)(m1 - m0),
                                   nq, s_site, s_rsk, s_rmax, s_frm, q == 0,
                                   q == NQ - 1);
      } else {
        auto load_v = [&](int h, float* v) { load8f(crow + 8 * h, v); };
        auto load_po = [&](int h, float* po) {
          if (REF) {
#pragma unroll
            for (int e = 0; e < 8; ++e) po[e] = 0.f;
          } else {
            state_load8(a.P, a.p16, (int64_t)epix * cout_p + nq + ec + 8 * h,
                        po);
          }
        };
        auto load_sk = [&](int h, float* sk) {
          if constexpr (kSkPre) {
            const T* hp = (const T*)&skr[h];
#pragma unroll
            for (int e = 0; e < 8; ++e) sk[e] = to_f(hp[e]);
          } else if (rsk >= 0) {
            Vec8<T>::load(dskip + (int64_t)rsk * cout_p + nq + ec + 8 * h,
                          sk);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) sk[e] = 0.f;
          }
        };
        with_act(a.act, [&](auto act_tag) {
          rm_all = fmaxf(rm_all,
                         finish_cols<T, REF, decltype(act_tag)::value>(
                             a, load_v, load_po, load_sk, hv, eo, epix, nq,
                             ec));
        });
      }
    }
    if constexpr (!SPLIT && !CHUNK) finish_rows(a, rm_all, eo, eok);
  }
}

// Split epilogue: sums the partial tiles of this frame's splits in split
// order and finishes each output tile as the unsplit GEMM does.
template <typename T, bool REF>
__global__ __launch_bounds__(256) void k_split_epi(ConvArgs a) {
  constexpr int BM = kGemmBM, BN = kGemmBN;
  const int64_t nO = a.dense ? a.capO : (int64_t)*a.nO;
  const int64_t tiles_m = (nO + BM - 1) / BM;
  const int tiles_n = (a.cout_p + BN - 1) / BN;
  const int64_t ntiles = tiles_m * tiles_n;
  const int S = split_count(ntiles, gemm_stages<T>(a), a.split_max);
  const int tid = threadIdx.x, cout_p = a.cout_p;
  const int em = tid >> 2, ec = (tid & 3) * 16;
  const T* dskip = (const T*)a.dskip;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t tm_i = t / tiles_n;
    const int64_t m0 = tm_i * BM;
    const int n0 = (int)(t - tm_i * tiles_n) * BN;
    const int64_t eo = m0 + em;
    const bool eok = eo < nO;
    const int epix = !eok ? 0 : a.dense ? (int)eo : a.O[eo];
    bool hv[2];
    float po[2][8], sk[2][8];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int n = n0 + ec + 8 * h;
      hv[h] = eok && n < cout_p;
#pragma unroll
      for (int e = 0; e < 8; ++e) po[h][e] = sk[h][e] = 0.f;
      if (hv[h] && a.mode == 0 && !REF)
        state_load8(a.P, a.p16, (int64_t)epix * cout_p + n, po[h]);
    }
    const int rsk =
        (a.mskip && eok) ? (a.dense ? epix : a.mskip[epix]) : -1;
#pragma unroll
    for (int h = 0; h < 2; ++h)
      if (hv[h] && rsk >= 0)
        Vec8<T>::load(dskip + (int64_t)rsk * cout_p + n0 + ec + 8 * h, sk[h]);
    const float* prow = a.part + eo * cout_p + n0 + ec;
    const int64_t pstride = a.capO * cout_p;
    // every split's partial row is requested before any is summed (one
    // round trip instead of one per split); the sum is in split order
    float4 q[kEpiSplits][2][2];
#pragma unroll
    for (int sp = 0; sp < kEpiSplits; ++sp) {
      if (sp >= S) break;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float* pp = prow + sp * pstride + 8 * h;
        q[sp][h][0] = hv[h] ? *(const float4*)pp : make_float4(0, 0, 0, 0);
        q[sp][h][1] =
            hv[h] ? *(const float4*)(pp + 4) : make_float4(0, 0, 0, 0);
      }
    }
    float vs[2][8];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int e = 0; e < 8; ++e) vs[h][e] = 0.f;
#pragma unroll
      for (int sp = 0; sp < kEpiSplits; ++sp) {
        if (sp >= S) break;
        const float4 lo = q[sp][h][0], hi = q[sp][h][1];
        vs[h][0] += lo.x; vs[h][1] += lo.y; vs[h][2] += lo.z;
        vs[h][3] += lo.w; vs[h][4] += hi.x; vs[h][5] += hi.y;
        vs[h][6] += hi.z; vs[h][7] += hi.w;
      }
    }
    auto load_v = [&](int h, float* v) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = vs[h][e];
    };
    auto load_po = [&](int h, float* o) {
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = po[h][e];
    };
    auto load_sk = [&](int h, float* o) {
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = sk[h][e];
    };
    with_act(a.act, [&](auto act_tag) {
      finish_tile<T, REF, decltype(act_tag)::value>(
          a, load_v, load_po, load_sk, hv, eo, eok, epix, n0, ec);
    });
  }
}

// ---------------------------------------------------------- big tiles
// 128 rows by 128 output channels per tile, four waves in a 2x2
// arrangement (64x64 each: 4x4 MFMA 16x16 blocks), reduction stages of 64
// columns staged through two LDS buffers, two stages of loads in flight in
// registers.  A staged byte feeds twice the products it feeds in a 64x64
// tile, but a CU holds two such blocks instead of four; as each wave's
// gathers are bound by their latency, the two effects nearly cancel, and
// only the layers with the longest reductions gain (use_big).  LDS rows
// are unpadded: the eight 16-byte vectors of a staged row are XOR-swizzled
// (big_swz), so the rows a group of lanes reads at one vector column fall
// in distinct banks.  Half-precision layers whose input channels are a
// multiple of 64 only; never split.  The epilogue is the chunk-state one:
// a tile is two consecutive run-aligned row tiles (at most 64 rows each),
// finished one after the other.
constexpr int kBigBM = 128, kBigBN = 128;
// Vector-column swizzle of staged row r, a function of r's low four bits:
// distinct for any eight consecutive rows from a multiple of eight, and,
// among sixteen consecutive rows from a multiple of sixteen, distinct over
// the even rows and over the odd rows.
__device__ __forceinline__ int big_swz(int r) {
  return (r & 7) ^ ((r >> 3) & 1);
}

template <typename T>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2)))
void k_conv_gemm_big(ConvArgs a) {
  static_assert(sizeof(T) == 2, "big tiles are half-precision");
  constexpr int BM = kBigBM, BN = kBigBN, KC = 64, VEC = 8;
  constexpr int VPR = KC / VEC;           // 16-byte vectors per staged row
  constexpr int AV = BM * VPR / 256;      // A vectors per thread per stage
  constexpr int BV = BN * VPR / 256;      // B vectors per thread per stage
  constexpr int IM = 4, JN = 4;           // 16x16 blocks per wave
  constexpr int CLD = BN + 4;             // f32 accumulator row
  constexpr int HM = kGemmBM;             // rows of an epilogue half
  constexpr size_t AB_BYTES = 2ull * (BM + BN) * KC * sizeof(T);
  constexpr size_t C_BYTES = (size_t)BM * CLD * sizeof(float);
  __shared__ __align__(16) char smem[AB_BYTES > C_BYTES ? AB_BYTES : C_BYTES];
  // the units' kernel-offset masks, two in turn: a unit clears the one
  // the next unit fills, so no barrier orders the clearing
  __shared__ u64 s_kmask[2];
  __shared__ int s_site[BM], s_rsk[BM], s_run[2][HM + 2];
  __shared__ unsigned s_rmax[2][HM];
  extern __shared__ int s_nbr[];          // [K][BM]
  T* const sA = (T*)smem;
  T* const sB = (T*)smem + 2 * BM * KC;
  float* const Cs = (float*)smem;

  const T* din = (const T*)a.din;
  const T* wt = (const T*)a.w;
  const T* zvec = (const T*)a.zero;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l16 = lane & 15, lg = lane >> 4;
  const int64_t nO = (int64_t)*a.nO;
  // row tiles: run-aligned halves, two per tile
  const int rstep = chunk_tile_step(a.nf);
  const int64_t tiles_r = (nO + rstep - 1) / rstep;
  const int64_t tiles_m = (tiles_r + 1) / 2;
  const int tiles_n = (a.cout_p + BN - 1) / BN;
  const int64_t ntiles = tiles_m * tiles_n;
  const int K = a.K, cin_p = a.cin_p, cout_p = a.cout_p;
  const int ktot_p = (int)a.ktot_p;
  const int spk = cin_p / KC;             // stages per kernel offset
  const int nst = K * spk;
  // XCD-aware order, as in k_conv_gemm
  const int chunk = (int)((ntiles + kXcd - 1) / kXcd);
  const int xcd = blockIdx.x % kXcd;
  const int u_end = (int)min(ntiles, (int64_t)(xcd + 1) * chunk);
  const int per_xcd = gridDim.x / kXcd;
  const int em = tid >> 2, ec = (tid & 3) * 16;

  // a unit's row bounds, fetched during the previous unit
  unsigned nb0 = 0u, nb1 = 0u, nb2 = 0u;
  auto fetch_bounds = [&](int u) __attribute__((always_inline)) {
    const int64_t j = 2 * (int64_t)((unsigned)u / (unsigned)tiles_n);
    nb0 = a.tstart[j];
    nb1 = a.tstart[min(j + 1, tiles_r)];
    nb2 = a.tstart[min(j + 2, tiles_r)];
  };
  const int u_first = xcd * chunk + blockIdx.x / kXcd;
  if (u_first < u_end) fetch_bounds(u_first);

  if (tid == 0) s_kmask[0] = 0ull;
  int kp = 0;  // this unit's offset mask
  for (int u = u_first; u < u_end; u += per_xcd, kp ^= 1) {
    const int tm = (int)((unsigned)u / (unsigned)tiles_n);
    const int n0 = (u - tm * tiles_n) * BN;
    // the tile's rows: halves [m0, mh) and [mh, m1)
    const int64_t m0 =
        (int64_t)(unsigned)__builtin_amdgcn_readfirstlane((int)nb0);
    const int64_t mh =
        (int64_t)(unsigned)__builtin_amdgcn_readfirstlane((int)nb1);
    const int64_t m1 =
        (int64_t)(unsigned)__builtin_amdgcn_readfirstlane((int)nb2);

    __syncthreads();  // the previous unit's LDS reads are complete
    if (tid == 0) s_kmask[kp ^ 1] = 0ull;
    // this thread's epilogue row in each half and its pixel
    const int64_t eo0 = m0 + em, eo1 = mh + em;
    const bool eok0 = eo0 < mh, eok1 = eo1 < m1;
    const int epix0 = eok0 ? a.O[eo0] : 0;
    const int epix1 = eok1 ? a.O[eo1] : 0;
    u64 my = 0ull;
    for (int e = tid; e < BM * K; e += 256) {
      const int k = e / BM, m = e - (e / BM) * BM;
      const int64_t o = m0 + m;
      const int src = o < m1 ? a.nbr[(int64_t)k * a.stride + o] : -1;
      s_nbr[e] = src;
      if (src >= 0) my |= 1ull << k;
    }
    if (my) atomicOr(&s_kmask[kp], my);
    __syncthreads();
    const u64 kmask = s_kmask[kp];
    if (u + per_xcd < u_end) fetch_bounds(u + per_xcd);

    auto next_k = [&](int k) __attribute__((always_inline)) {
      if (k >= K) return K;
      const u64 mk = kmask >> k;
      return mk ? k + __builtin_ctzll(mk) : K;
    };
    // stages walked as (offset kc, sub-stage) pairs, offsets without any
    // active neighbour in the tile skipped by a bit scan of the offset mask
    struct It {
      int kc, sub, st;
    };
    auto first_stage = [&]() __attribute__((always_inline)) {
      It it{next_k(0), 0, 0};
      it.st = it.kc < K ? it.kc * spk : nst;
      return it;
    };
    auto advance = [&](It it) __attribute__((always_inline)) {
      if (it.st >= nst) return it;
      if (++it.sub == spk) {
        it.kc = next_k(it.kc + 1);
        it.sub = 0;
      }
      it.st = it.kc < K ? it.kc * spk + it.sub : nst;
      return it;
    };
    // the gathered rows of this thread's A vectors, kept for the current
    // kernel offset (NULL: inactive neighbour)
    const T* arow[AV];
    int arow_kc = -1;
    auto load_stage = [&](const It& it, uint4 (&ra)[AV], uint4 (&rb)[BV]) __attribute__((always_inline)) {
      const bool live = it.st < nst;
      const int r0 = it.st * KC;
      if (live && it.kc != arow_kc) {
        arow_kc = it.kc;
#pragma unroll
        for (int q = 0; q < AV; ++q) {
          const int m = (tid + q * 256) / VPR;
          const int src = s_nbr[arow_kc * BM + m];
          arow[q] = src >= 0 ? din + (int64_t)src * cin_p : nullptr;
        }
      }
#pragma unroll
      for (int q = 0; q < AV; ++q) {
        const int v = tid + q * 256;
        const int cv = v - (v / VPR) * VPR;
        const T* row = live ? arow[q] : nullptr;
        ra[q] = *(const uint4*)(row ? row + it.sub * KC + cv * VEC : zvec);
      }
#pragma unroll
      for (int q = 0; q < BV; ++q) {
        const int v = tid + q * 256;
        const int nn = v / VPR, cv = v - (v / VPR) * VPR;
        const int n = n0 + nn;
        const T* pb = (live && n < cout_p)
                          ? wt + (int64_t)n * ktot_p + r0 + cv * VEC
                          : zvec;
        rb[q] = *(const uint4*)pb;
      }
    };
    auto store_stage = [&](int buf, const uint4 (&ra)[AV],
                           const uint4 (&rb)[BV]) __attribute__((always_inline)) {
#pragma unroll
      for (int q = 0; q < AV; ++q) {
        const int v = tid + q * 256;
        const int m = v / VPR, cv = v - (v / VPR) * VPR;
        lds_store16<T>(sA + buf * BM * KC + m * KC + ((cv ^ big_swz(m)) * VEC),
                       ra[q]);
      }
#pragma unroll
      for (int q = 0; q < BV; ++q) {
        const int v = tid + q * 256;
        const int nn = v / VPR, cv = v - (v / VPR) * VPR;
        lds_store16<T>(sB + buf * BN * KC + nn * KC +
                           ((cv ^ big_swz(nn)) * VEC),
                       rb[q]);
      }
    };

    v4f acc[IM][JN];
#pragma unroll
    for (int i = 0; i < IM; ++i)
#pragma unroll
      for (int j = 0; j < JN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

    // a lane reads row (or column) 16 i + l16 of its wave's 64, vector
    // column kk / 8 + lg; the row's swizzle is that of l16
    auto compute = [&](int buf) __attribute__((always_inline)) {
      const T* Ab = sA + buf * BM * KC + wm * 64 * KC;
      const T* Bb = sB + buf * BN * KC + wn * 64 * KC;
#pragma unroll
      for (int kk = 0; kk < KC; kk += 32) {
        const int vc = ((kk / VEC + lg) ^ big_swz(l16)) * VEC;
        uint4 av[IM], bv[JN];
#pragma unroll
        for (int i = 0; i < IM; ++i)
          av[i] = *(const uint4*)(Ab + (i * 16 + l16) * KC + vc);
#pragma unroll
        for (int j = 0; j < JN; ++j)
          bv[j] = *(const uint4*)(Bb + (j * 16 + l16) * KC + vc);
#pragma unroll
        for (int i = 0; i < IM; ++i) {
#pragma unroll
          for (int j = 0; j < JN; ++j) {
            if constexpr (__is_same(T, _Float16)) {
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                  __builtin_bit_cast(v8h, av[i]),
                  __builtin_bit_cast(v8h, bv[j]), acc[i][j], 0, 0, 0);
            } else {
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  __builtin_bit_cast(v8bf, av[i]),
                  __builtin_bit_cast(v8bf, bv[j]), acc[i][j], 0, 0, 0);
            }
          }
        }
      }
    };

    // residual rows of this thread's epilogue rows, requested now so that
    // they arrive during the reduction, and the rows' sites
    const int rsk0 = (a.mskip && eok0) ? a.mskip[epix0] : -1;
    const int rsk1 = (a.mskip && eok1) ? a.mskip[epix1] : -1;
    if ((tid & 3) == 0) {
      if (eok0) s_site[em] = (int)((unsigned)epix0 % (unsigned)a.per);
      if (eok1)
        s_site[mh - m0 + em] = (int)((unsigned)epix1 % (unsigned)a.per);
    }

    // stages go in pairs: a pair's loads are issued together as soon as
    // the pair before is staged in LDS, and waited for together when the
    // pair is staged, two reductions later (one wait per pair, whose
    // count the compiler cannot get wrong)
    uint4 ra0[AV], rb0[BV], ra1[AV], rb1[BV];
    It ia = first_stage();
    It ib = advance(ia);
    load_stage(ia, ra0, rb0);
    load_stage(ib, ra1, rb1);
    while (ia.st < nst) {
      __syncthreads();  // every wave has read both buffers
      store_stage(0, ra0, rb0);
      store_stage(1, ra1, rb1);
      __syncthreads();
      const bool two = ib.st < nst;
      const It ic = advance(ib);
      const It id = advance(ic);
      load_stage(ic, ra0, rb0);
      load_stage(id, ra1, rb1);
      compute(0);
      if (two) compute(1);
      ia = ic;
      ib = id;
    }

    // ---- epilogue: the whole accumulator tile to LDS (MFMA 16x16 block
    // layout: D[row = 4 lg + r][col = l16]), then per half and 64-column
    // quarter as the 64x64 tile finishes it
    __syncthreads();  // every wave's last stage is read
    if ((tid & 3) == 0) {
      if (eok0) s_rsk[em] = rsk0;
      if (eok1) s_rsk[mh - m0 + em] = rsk1;
    }
#pragma unroll
    for (int i = 0; i < IM; ++i)
#pragma unroll
      for (int j = 0; j < JN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          Cs[(wm * 64 + i * 16 + 4 * lg + r) * CLD + wn * 64 + j * 16 +
             l16] = acc[i][j][r];
    __syncthreads();
    // one pass per (half, 64-column quarter), kept rolled: a copy of the
    // epilogue per pass would not fit the instruction cache
#pragma unroll 1
    for (int hq = 0; hq < 2 * (BN / kGemmBN); ++hq) {
      const int h = hq / (BN / kGemmBN), q = hq - h * (BN / kGemmBN);
      const int64_t hm0 = h ? mh : m0;              // the half's first row
      const int hb0 = (int)(hm0 - m0);
      const int rows = (int)((h ? m1 : mh) - hm0);
      finish_chunk_tile<T>(a, Cs + hb0 * CLD + q * kGemmBN, CLD, s_run[h],
                           hm0, rows, n0 + q * kGemmBN, s_site + hb0,
                           s_rsk + hb0, s_rmax[h], nullptr, q == 0,
                           q == BN / kGemmBN - 1);
    }
  }
}

template <typename T>
static void gemm_big_t(hipStream_t s, int grid, size_t lds,
                       const ConvArgs& a) {
  k_conv_gemm_big<T><<<grid, 256, lds, s>>>(a);
}

template <typename T>
static void split_epi_t(hipStream_t s, int grid, const ConvArgs& a) {
  if (a.ref)
    k_split_epi<T, true><<<grid, 256, 0, s>>>(a);
  else
    k_split_epi<T, false><<<grid, 256, 0, s>>>(a);
}

// ------------------------------------------------ dense stem (reference)
// Dense reference pass of a 7x7 stride-2 convolution over rows of at most
// four channels (a ResNet stem) with at most 64 output channels.  A tile is
// 64 consecutive output pixels of one output row.  The tile's input window
// -- 7 rows by 136 pixels of 4 channels, zeros outside the image -- is
// staged once in LDS, and each 32-wide reduction step is one kernel row:
// offsets kx = 0..7 of 4 channels, kx = 7 against a zero weight, so a
// lane's eight values (offsets 2 lg and 2 lg + 1) are two adjacent staged
// pixels.  The weights are staged once per block in that order.  A tile's
// window is requested before the previous tile's epilogue, so that it
// arrives while that epilogue runs.  Tiles are finished as the reference
// build finishes its tiles.
constexpr int kStemBM = 64, kStemPW = 136;  // tile pixels, staged row pixels

template <typename T>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3)))
void k_stem_dense(ConvArgs a) {
  static_assert(sizeof(T) == 2, "half-precision stem");
  constexpr int BM = kStemBM, BN = 64, KS = 7, KR = 32;  // 7 steps of 32
  constexpr int BLD = KS * KR + 8;  // staged weight row
  constexpr int CLD = BN + 4;       // f32 accumulator row
  constexpr size_t PATCH_BYTES = (size_t)KS * kStemPW * 4 * sizeof(T);
  constexpr size_t C_BYTES = (size_t)BM * CLD * sizeof(float);
  __shared__ __align__(16) T sB[BN * BLD];
  // the staged window, and (after the products) the accumulator tile
  __shared__ __align__(16) char smem[PATCH_BYTES > C_BYTES ? PATCH_BYTES
                                                           : C_BYTES];
  T* const sP = (T*)smem;          // [KS][kStemPW][4]
  float* const Cs = (float*)smem;  // [BM][CLD]
  const T* din = (const T*)a.din;
  const T* wt = (const T*)a.w;
  const T* dskip = (const T*)a.dskip;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l16 = lane & 15, lg = lane >> 4;
  const int cout_p = a.cout_p;
  const Geo g = a.g;
  // B[n][ky*32 + kx*4 + c] = w[n][(ky*7 + kx)*4 + c] for kx < 7, else 0
  for (int e = tid; e < BN * KS * KR; e += 256) {
    const int n = e / (KS * KR), r = e - n * (KS * KR);
    const int ky = r / KR, q = r - ky * KR, kx = q >> 2, c = q & 3;
    T v = zero_v<T>();
    if (n < cout_p && kx < 7)
      v = wt[(int64_t)n * a.ktot_p + (ky * 7 + kx) * 4 + c];
    sB[n * BLD + r] = v;
  }
  const int tiles_x = (g.Wo + BM - 1) / BM;
  const int64_t ntiles = a.capO / g.Wo * tiles_x;  // output rows x tiles
  // XCD-aware order, as in k_conv_gemm
  const int chunk = (int)((ntiles + kXcd - 1) / kXcd);
  const int xcd = blockIdx.x % kXcd;
  const int u_end = (int)min(ntiles, (int64_t)(xcd + 1) * chunk);
  const int per_xcd = gridDim.x / kXcd;
  const int em = tid >> 2, ec = (tid & 3) * 16;
  // this thread's share of a tile's window: entries tid + 256 q
  constexpr int WQ = (KS * kStemPW + 255) / 256;
  auto fetch_window = [&](int u, uint2 (&w)[WQ]) {
    const int row = u / tiles_x;
    const int ox0 = (u - row * tiles_x) * BM;
    const int img = row / g.Ho, oy = row - img * g.Ho;
    const int iy0 = oy * 2 - g.ph, ix0 = ox0 * 2 - g.pw;
#pragma unroll
    for (int q = 0; q < WQ; ++q) {
      const int e = tid + 256 * q;
      const int ky = e / kStemPW, px = e - ky * kStemPW;
      const int iy = iy0 + ky, ix = ix0 + px;
      w[q] = make_uint2(0u, 0u);
      if (e < KS * kStemPW && iy >= 0 && iy < g.Hi && ix >= 0 && ix < g.Wi)
        w[q] = *(const uint2*)(din +
                               ((int64_t)(img * g.Hi + iy) * g.Wi + ix) * 4);
    }
  };
  uint2 win[WQ];
  const int u0 = xcd * chunk + blockIdx.x / kXcd;
  if (u0 < u_end) fetch_window(u0, win);
  for (int u = u0; u < u_end; u += per_xcd) {
    const int row = u / tiles_x;  // image * Ho + output row
    const int ox0 = (u - row * tiles_x) * BM;
    __syncthreads();  // the weights are staged; the last tile's reads done
#pragma unroll
    for (int q = 0; q < WQ; ++q) {
      const int e = tid + 256 * q;
      if (e < KS * kStemPW) *(uint2*)(sP + e * 4) = win[q];
    }
    __syncthreads();
    v4f acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ky = 0; ky < KS; ++ky) {
      uint4 av[2], bv[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int m = wm * 32 + i * 16 + l16;
        av[i] = *(const uint4*)(sP + (ky * kStemPW + 2 * m + 2 * lg) * 4);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int nn = wn * 32 + j * 16 + l16;
        bv[j] = *(const uint4*)(sB + nn * BLD + ky * KR + 8 * lg);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          if constexpr (__is_same(T, _Float16)) {
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                __builtin_bit_cast(v8h, av[i]), __builtin_bit_cast(v8h, bv[j]),
                acc[i][j], 0, 0, 0);
          } else {
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(v8bf, av[i]),
                __builtin_bit_cast(v8bf, bv[j]), acc[i][j], 0, 0, 0);
          }
        }
      }
    }
    if (u + per_xcd < u_end) fetch_window(u + per_xcd, win);
    __syncthreads();  // every wave has read the window (Cs reuses it)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          Cs[(wm * 32 + i * 16 + 4 * lg + r) * CLD + wn * 32 + j * 16 + l16] =
              acc[i][j][r];
    __syncthreads();
    // thread -> pixel em of the tile, columns [ec, ec + 16)
    const int ox = ox0 + em;
    const bool eok = ox < g.Wo;
    const int64_t eo = (int64_t)row * g.Wo + ox;
    const int epix = eok ? (int)eo : 0;
    const int rsk = (a.mskip && eok) ? epix : -1;
    const float* crow = Cs + em * CLD + ec;
    bool hv[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) hv[h] = eok && ec + 8 * h < cout_p;
    auto load_v = [&](int h, float* v) { load8f(crow + 8 * h, v); };
    auto load_po = [&](int, float* po) {
#pragma unroll
      for (int e = 0; e < 8; ++e) po[e] = 0.f;
    };
    auto load_sk = [&](int h, float* sk) {
      if (rsk >= 0) {
        Vec8<T>::load(dskip + (int64_t)rsk * cout_p + ec + 8 * h, sk);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) sk[e] = 0.f;
      }
    };
    float rm = 0.f;
    with_act(a.act, [&](auto act_tag) {
      rm = finish_cols<T, true, decltype(act_tag)::value>(
          a, load_v, load_po, load_sk, hv, eo, epix, 0, ec);
    });
    finish_rows(a, rm, eo, eok);
  }
}

// The dense reference pass's stem takes k_stem_dense: half precision, 7x7
// stride 2 over rows of 4 (padded) channels, at most 64 output channels.
static bool stem_dense(int dtype, const ConvArgs& a) {
  return dtype != 0 && a.ref && a.dense && a.K == 49 && a.cin_p == 4 &&
         a.cout_p <= 64 && a.g.kh == 7 && a.g.kw == 7 && a.g.sh == 2 &&
         a.g.sw == 2 && a.split_max <= 1 && a.g.Wo > 0;
}

using GemmFn = void (*)(ConvArgs);

// The gather-GEMM build for a launch.
template <typename T, bool SPLIT>
static GemmFn pick_gemm(const ConvArgs& a) {
  const bool aligned = a.cin_p % GemmTile<T>::KC == 0;
  if (a.ref)
    return aligned ? k_conv_gemm<T, true, true, SPLIT, false>
                   : k_conv_gemm<T, true, false, SPLIT, false>;
  if (!SPLIT && a.mode == kModeChunkState)  // builds of their own
    return aligned ? k_conv_gemm<T, false, true, false, true>
                   : k_conv_gemm<T, false, false, false, true>;
  if (!SPLIT && a.mode == kModeChunkPool)
    return aligned ? k_conv_gemm<T, false, true, false, true, true>
                   : k_conv_gemm<T, false, false, false, true, true>;
  return aligned ? k_conv_gemm<T, false, true, SPLIT, false>
                 : k_conv_gemm<T, false, false, SPLIT, false>;
}

template <typename T>
static GemmFn pick_gemm(const ConvArgs& a) {
  return a.split_max > 1 ? pick_gemm<T, true>(a) : pick_gemm<T, false>(a);
}

// Blocks of a persistent kernel that one CU holds at once with `lds`
// bytes of dynamic LDS (its registers and static LDS decide too; at most
// `cap`); asked of the runtime once per kernel and size.
static int blocks_per_cu(const void* fn, size_t lds, int cap) {
  struct Entry {
    const void* fn;
    size_t lds;
    int n;
  };
  static std::mutex mu;
  static std::vector<Entry> cache;
  std::lock_guard<std::mutex> lock(mu);
  for (const Entry& e : cache)
    if (e.fn == fn && e.lds == lds) return e.n;
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, 256, lds) !=
          hipSuccess ||
      n < 1)
    n = 1;
  n = n < cap ? n : cap;
  cache.push_back({fn, lds, n});
  return n;
}

// A persistent grid: the units, at most what the CUs hold at once, a
// multiple of the XCD count.
static int persistent_grid(int64_t units, const void* fn, size_t lds,
                           int cap) {
  const int64_t resident = (int64_t)kCUs * blocks_per_cu(fn, lds, cap);
  int64_t grid = units < resident ? units : resident;
  grid = (grid + kXcd - 1) / kXcd * kXcd;
  return (int)grid;
}

// Big tiles for the chunk-state layers where they measured faster than
// the 64x64 ones (ResNet-50 at 1024x2048, 10% change, chunks of 10): the
// 3x3 layers with 256 or 512 input channels (-3% to -23%) and the 1x1
// layers with 2048 input channels (-4% to -15%); a 3x3 layer with 128
// input channels, or a 1x1 layer with 1024, is 2% to 25% slower with them
// (half the resident waves, and row tiles of half the count).
static bool use_big(int dtype, const ConvArgs& a) {
  return dtype != 0 && a.mode == kModeChunkState && !a.ref &&
         a.split_max <= 1 && a.cout_p % kBigBN == 0 && a.cin_p % 64 == 0 &&
         a.K <= 64 && ((a.K > 1 && a.cin_p >= 256) || a.cin_p >= 2048);
}

bool launch_conv_gemm(const Prof& pf, hipStream_t s, int dtype,
                      const ConvArgs& a) {
  // inactive lanes read the zero vector: never launch without it
  if (!a.zero || ((uintptr_t)a.zero & 15)) return false;
  if (a.split_max > 1 && !a.part) return false;
  // run-aligned tiles belong to the chunk-state epilogue, which finishes
  // whole tiles itself (no split)
  if ((a.tstart != nullptr) != chunk_tiled(a.mode)) return false;
  if (a.mode == kModeChunkPool && (!a.dP || !a.aff)) return false;
  if (a.tstart && (a.split_max > 1 || a.nf < 1 || a.nf > 32 || a.per < 1 ||
                   !a.sites))
    return false;
  if (stem_dense(dtype, a)) {
    const int64_t units =
        a.capO / a.g.Wo * ((a.g.Wo + kStemBM - 1) / kStemBM);
    const GemmFn fn = dtype == 1 ? (GemmFn)k_stem_dense<_Float16>
                                 : (GemmFn)k_stem_dense<bf16_t>;
    const int grid = persistent_grid(units, (const void*)fn, 0, 3);
    prof_begin(pf, 7 /*ST_K_CONV_GEMM*/, s);
    fn<<<grid, 256, 0, s>>>(a);
    prof_end(pf, 7, s);
    return true;
  }
  if (use_big(dtype, a)) {
    const int64_t halves =
        (a.capO + chunk_tile_step(a.nf) - 1) / chunk_tile_step(a.nf);
    const int64_t units = (halves + 1) / 2 * (a.cout_p / kBigBN);
    const size_t lds = sizeof(int) * (size_t)a.K * kBigBM;
    const GemmFn fn = dtype == 1 ? (GemmFn)k_conv_gemm_big<_Float16>
                                 : (GemmFn)k_conv_gemm_big<bf16_t>;
    const int grid = persistent_grid(units, (const void*)fn, lds, 2);
    prof_begin(pf, 7 /*ST_K_CONV_GEMM*/, s);
    fn<<<grid, 256, lds, s>>>(a);
    prof_end(pf, 7, s);
    return true;
  }
  const int rstep = a.tstart ? chunk_tile_step(a.nf) : kGemmBM;
  const int64_t worst =
      ((a.capO + rstep - 1) / rstep) * ((a.cout_p + kGemmBN - 1) / kGemmBN);
  const int64_t units = worst * (a.split_max > 1 ? a.split_max : 1);
  const size_t lds = sizeof(int) * (size_t)a.K * kGemmBM;
  const GemmFn fn = dtype == 0   ? pick_gemm<float>(a)
                    : dtype == 1 ? pick_gemm<_Float16>(a)
                                 : pick_gemm<bf16_t>(a);
  // persistent blocks: what the CUs hold at once (a large window's
  // neighbour table can leave room for fewer than four)
  const int grid = persistent_grid(units, (const void*)fn, lds,
                                   GemmTile<bf16_t>::BLOCKS_PER_CU);
  prof_begin(pf, 7 /*ST_K_CONV_GEMM*/, s);
  fn<<<grid, 256, lds, s>>>(a);
  prof_end(pf, 7, s);
  if (a.split_max > 1) {
    const int egrid = (int)(worst < 1024 ? worst : 1024);
    prof_begin(pf, 22 /*ST_K_CONV_SPLIT_EPI*/, s);
    if (dtype == 0)
      split_epi_t<float>(s, egrid, a);
    else if (dtype == 1)
      split_epi_t<_Float16>(s, egrid, a);
    else
      split_epi_t<bf16_t>(s, egrid, a);
    prof_end(pf, 22, s);
  }
  return true;
}

// ---------------------------------------------------- (c') depthwise path
// Memory-bound: each thread owns 8 channels of one affected row.  The
// row's neighbour indices are read up to eight offsets at a time and their
// input rows requested together, then summed in offset order on the vector
// ALU (the same order as one offset at a time); the epilogue reads and
// writes whole 8-channel vectors.
template <typename T, bool REF, int ACT>
__device__ __forceinline__ void conv_dw_rows(const ConvArgs& a) {
  constexpr int KB = 8;                       // offsets per batch of loads
  constexpr int RV = (int)sizeof(T) / 2;      // 16-byte vectors per 8 channels
  const T* din = (const T*)a.din;
  const float* w = (const float*)a.w;
  const T* dskip = (const T*)a.dskip;
  T* dout = (T*)a.dout;
  const int cout_p = a.cout_p, cin_p = a.cin_p;
  const int64_t nO = a.dense ? a.capO : (int64_t)*a.nO;
  const int cpr = cout_p / 8;
  const int64_t total = nO * cpr;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * 256) {
    const int64_t o = idx / cpr;
    const int c0 = (int)(idx - o * cpr) * 8;
    const int pix = a.dense ? (int)o : a.O[o];
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    for (int k0 = 0; k0 < a.K; k0 += KB) {
      int src[KB];
#pragma unroll
      for (int j = 0; j < KB; ++j)
        src[j] = k0 + j >= a.K ? -1
                 : a.dense     ? dense_src(a.g, o, k0 + j)
                               : a.nbr[(int64_t)(k0 + j) * a.stride + o];
      uint4 raw[KB][RV];
#pragma unroll
      for (int j = 0; j < KB; ++j)
#pragma unroll
        for (int v = 0; v < RV; ++v)
          raw[j][v] = src[j] >= 0
                          ? ((const uint4*)(din + (int64_t)src[j] * cin_p +
                                            c0))[v]
                          : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
      for (int j = 0; j < KB; ++j) {
        if (src[j] < 0) continue;
        float x[8], wk[8];
        Vec8<T>::load((const T*)raw[j], x);
        load8f(w + (int64_t)(k0 + j) * cout_p + c0, wk);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += wk[e] * x[e];
      }
    }
    // every load of the epilogue before its stores
    const int rsk = !a.mskip ? -1 : a.dense ? pix : a.mskip[pix];
    float sk[8], po[8], ex[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) sk[e] = po[e] = 0.f;
    if (rsk >= 0) Vec8<T>::load(dskip + (int64_t)rsk * cout_p + c0, sk);
    const bool state = a.mode == kModeState || a.mode == kModeStateOnly;
    if (state && !REF) state_load8(a.P, a.p16, (int64_t)pix * cout_p + c0, po);
    if (state && a.gate)
      load8f(gate_slot(a.gate, a.gpar, a.gsz, 0) + (pix / a.gate_hw) *
                 cout_p + c0,
             ex);
    else if (state && !REF && a.yhat)
      load8f(a.yhat + (int64_t)pix * cout_p + c0, ex);
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      v[e] = acc[e];
      if (REF) v[e] += a.bias[c0 + e];
      v[e] += sk[e];
    }
    if (a.mode == kModeDefer) {
      store8f(a.dP + o * cout_p + c0, v);
      continue;
    }
    if (state) {
      float pn[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) pn[e] = state_round(a.p16, po[e] + v[e]);
      state_store8(a.P, a.p16, (int64_t)pix * cout_p + c0, pn);
      if (a.mode == kModeStateOnly) continue;
      if (a.gate) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          v[e] = act_c<ACT>(pn[e]) * ex[e] - act_c<ACT>(po[e]) * ex[e];
      } else if (!REF && a.yhat) {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = act_c<ACT>(pn[e]) - ex[e];
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          v[e] = act_c<ACT>(pn[e]) - act_c<ACT>(po[e]);
      }
    }
    const float rm = Vec8<T>::store(dout + o * cout_p + c0, v);
    if (rm > 0.f && a.rowmax) atomicMax(a.rowmax + o, __float_as_uint(rm));
  }
}

template <typename T, bool REF>
__global__ __launch_bounds__(256) void k_conv_dw(ConvArgs a) {
  with_act(a.act, [&](auto act_tag) {
    conv_dw_rows<T, REF, decltype(act_tag)::value>(a);
  });
}

template <typename T>
static void dw_t(hipStream_t s, int grid, const ConvArgs& a) {
  if (a.ref)
    k_conv_dw<T, true><<<grid, 256, 0, s>>>(a);
  else
    k_conv_dw<T, false><<<grid, 256, 0, s>>>(a);
}

void launch_conv_dw(const Prof& pf, hipStream_t s, int dtype,
                    const ConvArgs& a) {
  const int grid = grid_for(a.capO * (a.cout_p / 8), 8192);
  prof_begin(pf, 8 /*ST_K_CONV_DW*/, s);
  if (dtype == 0)
    dw_t<float>(s, grid, a);
  else if (dtype == 1)
    dw_t<_Float16>(s, grid, a);
  else
    dw_t<bf16_t>(s, grid, a);
  prof_end(pf, 8, s);
}

// ----------------------------------------------------------- max-pool
// Delta of a pooled output = max over its window of f(P_new) minus the
// same max of f(P_old); P_new = P_old + dP on affected conv outputs.
template <typename T>
__global__ __launch_bounds__(256) void k_pool_emit(PoolArgs a) {
  T* dout = (T*)a.dout;
  const int64_t nQ = (int64_t)*a.nQ;
  const int64_t total = nQ * a.cp;
  const Geo& g = a.g;  // Hi/Wi: conv grid, Ho/Wo: pooled grid
  const int64_t hwq = (int64_t)g.Ho * g.Wo;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * 256) {
    const int64_t q = idx / a.cp;
    const int c = (int)(idx - q * a.cp);
    const int p = a.Q[q];
    const int n = (int)(p / hwq);
    const int rem = (int)(p - n * hwq);
    const int qy = rem / g.Wo, qx = rem - (rem / g.Wo) * g.Wo;
    float mo = -INFINITY, mn = -INFINITY;
    for (int ky = 0; ky < g.kh; ++ky) {
      const int iy = qy * g.sh - g.ph + ky;
      if (iy < 0 || iy >= g.Hi) continue;
      for (int kx = 0; kx < g.kw; ++kx) {
        const int ix = qx * g.sw - g.pw + kx;
        if (ix < 0 || ix >= g.Wi) continue;
        const int64_t w = ((int64_t)n * g.Hi + iy) * g.Wi + ix;
        const float po = a.ref ? 0.f : a.P[w * a.cp + c];
        const int r = a.Mo[w];
        const float pn = r >= 0 ? po + a.dP[(int64_t)r * a.cp + c] : po;
        mo = fmaxf(mo, act_f(po, a.act));
        mn = fmaxf(mn, act_f(pn, a.act));
      }
    }
    // residual carry: against what the consumers received
    if (a.yhat && !a.ref) mo = a.yhat[(int64_t)p * a.cp + c];
    const T qv = from_f<T>(mn - mo);
    dout[q * a.cp + c] = qv;
    const float ab = fabsf(to_f(qv));
    if (ab > 0.f) atomicMax(a.rowmax + q, __float_as_uint(ab));
  }
}

void launch_pool_emit(const Prof& pf, hipStream_t s, int dtype,
                      const PoolArgs& a) {
  const int grid = grid_for(a.capQ * a.cp, 8192);
  prof_begin(pf, 12 /*ST_K_POOL_EMIT*/, s);
  if (dtype == 0)
    k_pool_emit<float><<<grid, 256, 0, s>>>(a);
  else if (dtype == 1)
    k_pool_emit<_Float16><<<grid, 256, 0, s>>>(a);
  else
    k_pool_emit<bf16_t><<<grid, 256, 0, s>>>(a);
  prof_end(pf, 12, s);
}

__global__ __launch_bounds__(256) void k_commit(const int* O, const u64* nOp,
                                                float* P, const float* dP,
                                                int cp, int ref) {
  const int64_t nO = (int64_t)*nOp;
  const int c4 = cp / 4;
  const int64_t total = nO * c4;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * 256) {
    const int64_t o = idx / c4;
    const int c = (int)(idx - o * c4) * 4;
    float4* pp = (float4*)(P + (int64_t)O[o] * cp + c);
    const float4 d = *(const float4*)(dP + o * cp + c);
    float4 v = ref ? make_float4(0.f, 0.f, 0.f, 0.f) : *pp;
    v.x += d.x; v.y += d.y; v.z += d.z; v.w += d.w;
    *pp = v;
  }
}

void launch_commit(const Prof& pf, hipStream_t s, const int* O, const u64* nO,
                   int64_t capO, float* P, const float* dP, int cp, int ref) {
  prof_begin(pf, 13 /*ST_K_COMMIT*/, s);
  k_commit<<<grid_for(capO * (cp / 4), 8192), 256, 0, s>>>(O, nO, P, dP, cp,
                                                           ref);
  prof_end(pf, 13, s);
}

// ------------------------------------------------ truncation (list mode)
// Keeps the rows of an emitted tensor whose max |delta| exceeds the
// threshold (ascending kept list), removes dropped rows from the pixel map
// and prepares the consumers' rulebooks.
struct ListPred {
  const uint32_t* rowmax;
  const int* rowpix;
  int* act;
  int* map;
  float thr;
  const float* thr_dev;  // or NULL: thr
  ConsList cons;
  struct Item {
    uint32_t rm;
    int pix;
  };
  __device__ float th() const { return thr_dev ? *thr_dev : thr; }
  __device__ Item load(int64_t r) const { return Item{rowmax[r], rowpix[r]}; }
  __device__ bool keep(const Item& it) const {
    return __uint_as_float(it.rm) > th();
  }
  __device__ unsigned emit(int64_t r, unsigned pos, const Item& it) const {
    act[pos] = it.pix;
    cons_emit(cons, it.pix, pos, (int)r);
    // an identity consumer's affected list is this list: where its GEMM
    // tile starts (pos a multiple of the tile step), the tile is moved back
    // to the start of the site's run.  The rows of a site are adjacent
    // (the list is site-major); the kept ones among the rows before r give
    // the rank.  rowmax and rowpix are not written by this pass.
    for (int i = 0; i < cons.n; ++i) {
      const Cons& c = cons.c[i];
      if (c.kind != kConsIdent || !c.tstart) continue;
      const unsigned step = (unsigned)chunk_tile_step(c.nf);
      if (pos % step) continue;
      const unsigned pu = (unsigned)c.per, site = (unsigned)it.pix % pu;
      unsigned rank = 0;
      for (int q = 1; q < c.nf && r - q >= 0; ++q) {
        if ((unsigned)rowpix[r - q] % pu != site) break;
        rank += __uint_as_float(rowmax[r - q]) > th() ? 1u : 0u;
      }
      c.tstart[pos / step] = pos - rank;
    }
    return 0u;
  }
  __device__ void drop(int64_t, const Item& it) const { map[it.pix] = -1; }
  __device__ void block_done(unsigned) const {}
  __device__ void finish(unsigned total) const { cons_finish(cons, total); }
};

void launch_list_compact(const Prof& pf, hipStream_t s, const ListArgs& a) {
  ListPred p{a.rowmax, a.rowpix, a.act, a.map, a.thr, a.thr_dev, a.cons};
  run_compact(pf, 15 /*ST_K_LIST_COMPACT*/, s, a.n_rows, 0, a.cap, a.tiles,
              a.tiles_clear,
              a.cnt_act, nullptr, p);
}

// ------------------------------------------------- squeeze-excitation
__host__ __device__ __forceinline__ int round_up8(int x) {
  return (x + 7) & ~7;
}

// Exact squeeze-excitation on a deferred layer (state P, update rows dP of
// the affected sites, Mo: site -> dP row).  The pooled mean of f(P) is kept
// as per-image f64 channel sums S that each frame moves by
// sum over affected sites of f(P_new) - f(P_old) (in the reference pass:
// by f(P) over every site, from S = 0).  Squeeze: partial sums of that
// change over fixed site ranges; excite: S, mean and gates per image;
// emit: delta = f(P_new) * s_new - f(P_old) * s_old at every site, the state
// commit, row maxima and the 64-site kept counts.  Every sum runs in a fixed
// order, so results do not depend on scheduling.
//
// Row mapping: TPS threads per site (a power of two up to one wave), each
// owning the 8-channel vectors lane, lane + TPS, ... (at most 4 of them for
// up to 2048 channels); 256 / TPS sites side by side per block.
template <int TPS>
__global__ __launch_bounds__(256) void k_se_squeeze(SeArgs a) {
  constexpr int R = 256 / TPS, IT = TPS == 64 ? 4 : 1;
  __shared__ float sm[256 * IT * 8];  // [R][cp] per-lane partials
  const int n = blockIdx.y, g = blockIdx.x;
  const int lane = threadIdx.x % TPS, rl = threadIdx.x / TPS;
  const int cp = a.cp, V = cp / 8;
  float acc[IT][8];
#pragma unroll
  for (int k = 0; k < IT; ++k)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[k][e] = 0.f;
  const int64_t base = (int64_t)n * a.hw;
  const int64_t s0 = (int64_t)g * a.chunk;
  const int64_t s1 = min(s0 + (int64_t)a.chunk, a.hw);
  for (int64_t si = s0 + rl; si < s1; si += R) {
    const int64_t p = base + si;
    const int r = a.Mo[p];
    if (r < 0) continue;
#pragma unroll
    for (int k = 0; k < IT; ++k) {
      const int v = lane + k * TPS;
      if (v >= V) break;
      float po[8], dp[8];
      if (a.ref) {
#pragma unroll
        for (int e = 0; e < 8; ++e) po[e] = 0.f;
      } else {
        state_load8(a.P, a.p16, p * cp + v * 8, po);
      }
      load8f(a.dP + (int64_t)r * cp + v * 8, dp);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        acc[k][e] += act_f(state_round(a.p16, po[e] + dp[e]), a.act) -
                     act_f(po[e], a.act);
    }
  }
#pragma unroll
  for (int k = 0; k < IT; ++k) {
    const int v = lane + k * TPS;
    if (v < V) {
#pragma unroll
      for (int e = 0; e < 8; ++e) sm[rl * cp + v * 8 + e] = acc[k][e];
    }
  }
  __syncthreads();
  // pairwise tree over the R row lanes (fixed pairing)
  for (int h = R / 2; h > 0; h >>= 1) {
    for (int i = threadIdx.x; i < h * cp; i += 256) {
      const int j = i / cp, c = i - j * cp;
      sm[j * cp + c] += sm[(j + h) * cp + c];
    }
    __syncthreads();
  }
  for (int c = threadIdx.x; c < cp; c += 256)
    a.part[((int64_t)n * a.nchunk + g) * cp + c] = sm[c];
}

// Excitation of one image per block (1024 threads): the frame's partial
// sums over the site chunks (Lc lanes per 4-channel column, then the Lc
// results in lane order) move the f64 channel sums S; the means feed the
// hidden units (one wave per unit, two units per pass) and the gates
// (each 4-channel output split over Lg thread groups of the hidden units,
// then summed in group order).
constexpr int kSeExciteThreads = 1024;
__global__ __launch_bounds__(kSeExciteThreads) void k_se_excite(SeArgs a) {
  constexpr int NT = kSeExciteThreads;
  extern __shared__ __align__(16) float sm[];  // [cp] means, [mid], [NT] x4
  float* m = sm;
  float* z = sm + a.cp;
  float4* red = (float4*)(sm + a.cp + round_up8(a.mid));
  const int n = blockIdx.x, cp = a.cp, V4 = cp / 4, t = threadIdx.x;
  const int nfr = a.nfr > 1 ? a.nfr : 1;
  // frames in order: frame fr + 1 starts from the sums frame fr left
  for (int fr = 0; fr < nfr; ++fr) {
    float* s_new = a.gout ? a.gout + fr * a.gout_stride
                          : const_cast<float*>(gate_slot(a.gates, a.gpar,
                                                         a.gsz, 1));
    const int Lc = V4 <= NT ? NT / V4 : 1;
    const float4* part = (const float4*)(a.part + fr * a.part_stride +
                                         (int64_t)n * a.nchunk * cp);
    for (int v0 = 0; v0 < V4; v0 += NT) {
      const int v = v0 + (Lc > 1 ? t % V4 : t), l = Lc > 1 ? t / V4 : 0;
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
      if (v < V4 && l < Lc) {
        for (int g = l; g < a.nchunk; g += Lc) {
          const float4 q = part[(int64_t)g * V4 + v];
          acc.x += q.x; acc.y += q.y; acc.z += q.z; acc.w += q.w;
        }
      }
      red[t] = acc;
      __syncthreads();
      if (v < V4 && l == 0) {
        float4 tot = red[t];
        for (int j = 1; j < Lc; ++j) {
          const float4 q = red[t + j * V4];
          tot.x += q.x; tot.y += q.y; tot.z += q.z; tot.w += q.w;
        }
        const float tv[4] = {tot.x, tot.y, tot.z, tot.w};
  #pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int c = 4 * v + k;
          double* S = a.S + (int64_t)n * cp + c;
          const double sv = (a.ref ? 0.0 : *S) + (double)tv[k];
          *S = sv;
          m[c] = (float)(sv / (double)a.hw);
        }
      }
      __syncthreads();
    }
    // hidden units z = silu(w1 . m + b1)
    const int lane = t & 63, wave = t >> 6, nw = NT / 64;
    const float4* m4 = (const float4*)m;
    for (int j0 = wave; j0 < a.mid; j0 += 2 * nw) {
      const int j1 = j0 + nw;
      const float4* w0 = (const float4*)(a.w1 + (int64_t)j0 * cp);
      const float4* w1 = (const float4*)(a.w1 + (int64_t)(j1 < a.mid ? j1 : j0)
                                         * cp);
      float d0 = 0.f, d1 = 0.f;
  #pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int v = lane + 64 * i;
        if (v < V4) {
          const float4 x = m4[v], p = w0[v], q = w1[v];
          d0 += p.x * x.x + p.y * x.y + p.z * x.z + p.w * x.w;
          d1 += q.x * x.x + q.y * x.y + q.z * x.z + q.w * x.w;
        }
      }
  #pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        d0 += __shfl_xor(d0, o, 64);
        d1 += __shfl_xor(d1, o, 64);
      }
      if (lane == 0) {
        z[j0] = act_f(d0 + a.b1[j0], 2);
        if (j1 < a.mid) z[j1] = act_f(d1 + a.b1[j1], 2);
      }
    }
    __syncthreads();
    // gates: output vector v, hidden units split over Lg groups
    const int Lg = V4 <= NT ? NT / V4 : 1;
    for (int v0 = 0; v0 < V4; v0 += NT) {
      const int v = v0 + (Lg > 1 ? t % V4 : t), l = Lg > 1 ? t / V4 : 0;
      float4 e = make_float4(0.f, 0.f, 0.f, 0.f);
      if (v < V4 && l < Lg) {
        const float4* w = (const float4*)a.w2t + v;
  #pragma unroll 4
        for (int j = l; j < a.mid; j += Lg) {
          const float4 q = w[(int64_t)j * V4];
          const float zj = z[j];
          e.x += q.x * zj; e.y += q.y * zj; e.z += q.z * zj; e.w += q.w * zj;
        }
      }
      red[t] = e;
      __syncthreads();
      if (v < V4 && l == 0) {
        float4 tot = ((const float4*)a.b2)[v];
        for (int j = 0; j < Lg; ++j) {
          const float4 q = red[t + j * V4];
          tot.x += q.x; tot.y += q.y; tot.z += q.z; tot.w += q.w;
        }
        const float ev[4] = {tot.x, tot.y, tot.z, tot.w};
  #pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int c = 4 * v + k;
          s_new[(int64_t)n * cp + c] =
              c < a.c ? 1.f / (1.f + expf(-ev[k])) : 0.f;
        }
      }
      __syncthreads();
    }
  }
}


template <typename T, int TPS>
__global__ __launch_bounds__(256) void k_se_emit(SeArgs a) {
  constexpr int R = 256 / TPS, IT = TPS == 64 ? 4 : 1;
  T* dout = (T*)a.dout;
  const int lane = threadIdx.x % TPS;
  const int64_t row = (int64_t)blockIdx.x * R + threadIdx.x / TPS;
  const int cp = a.cp, V = cp / 8;
  const bool in = row < a.npix;
  float rm = 0.f;
  if (in) {
    const int n = (int)(row / a.hw);
    const int r = a.Mo[row];
    const float* sn = gate_slot(a.gates, a.gpar, a.gsz, 1) + (int64_t)n * cp;
    const float* so = gate_slot(a.gates, a.gpar, a.gsz, 0) + (int64_t)n * cp;
#pragma unroll
    for (int k = 0; k < IT; ++k) {
      const int v = lane + k * TPS;
      if (v >= V) break;
      const int c0 = v * 8;
      float po[8], dp[8], gn[8], go[8], pn[8], d[8];
      if (a.ref) {
#pragma unroll
        for (int e = 0; e < 8; ++e) po[e] = 0.f;
      } else {
        state_load8(a.P, a.p16, row * cp + c0, po);
      }
      if (r >= 0) {
        load8f(a.dP + (int64_t)r * cp + c0, dp);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) dp[e] = 0.f;
      }
      load8f(sn + c0, gn);
      const bool carry = a.yhat && !a.ref;
      // residual carry: against what the consumers received
      load8f(carry ? a.yhat + row * cp + c0 : so + c0, go);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        pn[e] = state_round(a.p16, po[e] + dp[e]);
        const float en = act_f(pn[e], a.act) * gn[e];
        const float eo = a.ref     ? 0.f
                         : carry   ? go[e]
                                   : act_f(po[e], a.act) * go[e];
        d[e] = en - eo;
      }
      rm = fmaxf(rm, Vec8<T>::store(dout + row * cp + c0, d));
      if (r >= 0) state_store8(const_cast<float*>(a.P), a.p16, row * cp + c0, pn);
    }
  }
#pragma unroll
  for (int o = 1; o < TPS; o <<= 1) rm = fmaxf(rm, __shfl_xor(rm, o, 64));
  if (in && lane == 0) {
    a.rowmax[row] = __float_as_uint(rm);
    a.rowpix[row] = (int)row;
    a.map[row] = (int)row;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *a.cnt_rows = (u64)a.npix;
}

template <int TPS>
static void se_t(const Prof& pf, hipStream_t s, int dtype, const SeArgs& a) {
  prof_begin(pf, 19 /*ST_K_SE_SQUEEZE*/, s);
  k_se_squeeze<TPS><<<dim3(a.nchunk, a.N), 256, 0, s>>>(a);
  prof_end(pf, 19, s);
  prof_begin(pf, 20 /*ST_K_SE_EXCITE*/, s);
  k_se_excite<<<a.N, kSeExciteThreads,
                sizeof(float) * (a.cp + round_up8(a.mid) +
                                 4 * kSeExciteThreads),
                s>>>(a);
  prof_end(pf, 20, s);
  constexpr int R = 256 / TPS;
  const int blocks = (int)((a.npix + R - 1) / R);
  prof_begin(pf, 21 /*ST_K_SE_EMIT*/, s);
  if (dtype == 0)
    k_se_emit<float, TPS><<<blocks, 256, 0, s>>>(a);
  else if (dtype == 1)
    k_se_emit<_Float16, TPS><<<blocks, 256, 0, s>>>(a);
  else
    k_se_emit<bf16_t, TPS><<<blocks, 256, 0, s>>>(a);
  prof_end(pf, 21, s);
}

void launch_se(const Prof& pf, hipStream_t s, int dtype, const SeArgs& a) {
  switch (a.tps) {
    case 1: se_t<1>(pf, s, dtype, a); break;
    case 2: se_t<2>(pf, s, dtype, a); break;
    case 4: se_t<4>(pf, s, dtype, a); break;
    case 8: se_t<8>(pf, s, dtype, a); break;
    case 16: se_t<16>(pf, s, dtype, a); break;
    case 32: se_t<32>(pf, s, dtype, a); break;
    default: se_t<64>(pf, s, dtype, a); break;
  }
}

// ---- exact squeeze-excitation in a chunk
// Row in Pt of site p's state before frame t: the latest frame below t
// that updated it, or -1 (the chunk's starting state).
__device__ __forceinline__ int chunk_prev_row(const int* Mo, uint32_t bits,
                                              int t, int64_t npix,
                                              int64_t p) {
  const uint32_t below = t > 0 ? bits & ((1u << t) - 1u) : 0u;
  if (!below) return -1;
  const int tp = 31 - __builtin_clz(below);
  return Mo[(int64_t)tp * npix + p];
}

// Frame blockIdx.z's squeeze: the partial sums of f(P_t) - f(P_{t-1}) over
// the sites it updated, with the frame-by-frame squeeze's site chunks,
// lanes and reduction tree (so its sums, and the gates, come out the same).
template <int TPS>
__global__ __launch_bounds__(256) void k_chunk_se_squeeze(ChunkSeArgs a) {
  constexpr int R = 256 / TPS, IT = TPS == 64 ? 4 : 1;
  __shared__ float sm[256 * IT * 8];  // [R][cp] per-lane partials
  const int n = blockIdx.y, g = blockIdx.x, t = blockIdx.z;
  const int lane = threadIdx.x % TPS, rl = threadIdx.x / TPS;
  const int cp = a.cp, V = cp / 8;
  float acc[IT][8];
#pragma unroll
  for (int k = 0; k < IT; ++k)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[k][e] = 0.f;
  const int64_t base = (int64_t)n * a.hw;
  const int64_t s0 = (int64_t)g * a.chunk;
  const int64_t s1 = min(s0 + (int64_t)a.chunk, a.hw);
  for (int64_t si = s0 + rl; si < s1; si += R) {
    const int64_t p = base + si;
    const uint32_t bits = a.aff[p];
    if (!((bits >> t) & 1u)) continue;
    const int r = a.Mo[(int64_t)t * a.npix + p];
    const int rp = chunk_prev_row(a.Mo, bits, t, a.npix, p);
#pragma unroll
    for (int k = 0; k < IT; ++k) {
      const int v = lane + k * TPS;
      if (v >= V) break;
      float po[8], pn[8];
      if (rp >= 0)
        load8f(a.Pt + (int64_t)rp * cp + v * 8, po);
      else
        state_load8(a.P, a.p16, p * cp + v * 8, po);
      load8f(a.Pt + (int64_t)r * cp + v * 8, pn);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        acc[k][e] += act_f(pn[e], a.act) - act_f(po[e], a.act);
    }
  }
#pragma unroll
  for (int k = 0; k < IT; ++k) {
    const int v = lane + k * TPS;
    if (v < V) {
#pragma unroll
      for (int e = 0; e < 8; ++e) sm[rl * cp + v * 8 + e] = acc[k][e];
    }
  }
  __syncthreads();
  for (int h = R / 2; h > 0; h >>= 1) {
    for (int i = threadIdx.x; i < h * cp; i += 256) {
      const int j = i / cp, c = i - j * cp;
      sm[j * cp + c] += sm[(j + h) * cp + c];
    }
    __syncthreads();
  }
  float* part = a.part + (((int64_t)t * a.N + n) * a.nchunk + g) * cp;
  for (int c = threadIdx.x; c < cp; c += 256) part[c] = sm[c];
}

// Every site's frames in order (TPS lanes per site, its state in
// registers): frame t's candidate row site * nf + t is
// f(P_t) * s_t - f(P_{t-1}) * s_{t-1}.
template <typename T, int TPS>
__global__ __launch_bounds__(256) void k_chunk_se_emit(ChunkSeArgs a) {
  constexpr int R = 256 / TPS, IT = TPS == 64 ? 4 : 1;
  T* dout = (T*)a.dout;
  const int lane = threadIdx.x % TPS;
  const int64_t p = (int64_t)blockIdx.x * R + threadIdx.x / TPS;
  const int cp = a.cp, V = cp / 8;
  if (p < a.npix) {
    const int n = (int)(p / a.hw);
    const uint32_t bits = a.aff[p];
    const float* g_first = gate_slot(a.slots, a.gpar, a.gsz, 0) +
                           (int64_t)n * cp;
    float pv[IT][8];
#pragma unroll
    for (int k = 0; k < IT; ++k) {
      const int v = lane + k * TPS;
      if (v < V) state_load8(a.P, a.p16, p * cp + v * 8, pv[k]);
    }
    for (int t = 0; t < a.nf; ++t) {
      const int r = ((bits >> t) & 1u) ? a.Mo[(int64_t)t * a.npix + p] : -1;
      const float* gn = a.gates + ((int64_t)t * a.N + n) * cp;
      const float* go =
          t ? a.gates + ((int64_t)(t - 1) * a.N + n) * cp : g_first;
      const int64_t j = p * a.nf + t;
      float rm = 0.f;
#pragma unroll
      for (int k = 0; k < IT; ++k) {
        const int v = lane + k * TPS;
        if (v >= V) break;
        float pn[8], g1[8], g0[8], d[8];
        if (r >= 0) {
          load8f(a.Pt + (int64_t)r * cp + v * 8, pn);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) pn[e] = pv[k][e];
        }
        load8f(gn + v * 8, g1);
        load8f(go + v * 8, g0);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          d[e] = act_f(pn[e], a.act) * g1[e] - act_f(pv[k][e], a.act) * g0[e];
          pv[k][e] = pn[e];
        }
        rm = fmaxf(rm, Vec8<T>::store(dout + j * cp + v * 8, d));
      }
#pragma unroll
      for (int o = 1; o < TPS; o <<= 1) rm = fmaxf(rm, __shfl_xor(rm, o, 64));
      if (lane == 0) {
        a.rowmax[j] = __float_as_uint(rm);
        a.rowpix[j] = (int)((int64_t)t * a.npix + p);
        a.map[(int64_t)t * a.npix + p] = (int)j;
      }
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0)
    *a.cnt_rows = (u64)(a.npix * a.nf);
}

// The chunk's last gates become the new slot's (the slots flip after the
// chunk).
__global__ void k_gate_copy(const float* src, float* slots, const int* gpar,
                            int64_t gsz, int64_t n) {
  float* dst = const_cast<float*>(gate_slot(slots, gpar, gsz, 1));
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * 256)
    dst[i] = src[i];
}

template <int TPS>
static void chunk_se_t(const Prof& pf, hipStream_t s, int dtype,
                       const ChunkSeArgs& c, const SeArgs& ex) {
  prof_begin(pf, 19 /*ST_K_SE_SQUEEZE*/, s);
  k_chunk_se_squeeze<TPS><<<dim3(c.nchunk, c.N, c.nf), 256, 0, s>>>(c);
  prof_end(pf, 19, s);
  prof_begin(pf, 20 /*ST_K_SE_EXCITE*/, s);
  SeArgs e = ex;
  e.part = c.part;
  e.gout = c.gates;
  e.nfr = c.nf;
  e.part_stride = (int64_t)c.N * c.nchunk * c.cp;
  e.gout_stride = (int64_t)c.N * c.cp;
  e.ref = 0;
  k_se_excite<<<c.N, kSeExciteThreads,
                sizeof(float) * (c.cp + round_up8(e.mid) +
                                 4 * kSeExciteThreads),
                s>>>(e);
  prof_end(pf, 20, s);
  constexpr int R = 256 / TPS;
  const int blocks = (int)((c.npix + R - 1) / R);
  prof_begin(pf, 21 /*ST_K_SE_EMIT*/, s);
  if (dtype == 0)
    k_chunk_se_emit<float, TPS><<<blocks, 256, 0, s>>>(c);
  else if (dtype == 1)
    k_chunk_se_emit<_Float16, TPS><<<blocks, 256, 0, s>>>(c);
  else
    k_chunk_se_emit<bf16_t, TPS><<<blocks, 256, 0, s>>>(c);
  const int64_t ng = (int64_t)c.N * c.cp;
  k_gate_copy<<<grid_for(ng, 256), 256, 0, s>>>(
      c.gates + (int64_t)(c.nf - 1) * ng, c.slots, c.gpar, c.gsz, ng);
  prof_end(pf, 21, s);
}

void launch_chunk_se(const Prof& pf, hipStream_t s, int dtype,
                     const ChunkSeArgs& c, const SeArgs& ex) {
  switch (c.tps) {
    case 1: chunk_se_t<1>(pf, s, dtype, c, ex); break;
    case 2: chunk_se_t<2>(pf, s, dtype, c, ex); break;
    case 4: chunk_se_t<4>(pf, s, dtype, c, ex); break;
    case 8: chunk_se_t<8>(pf, s, dtype, c, ex); break;
    case 16: chunk_se_t<16>(pf, s, dtype, c, ex); break;
    case 32: chunk_se_t<32>(pf, s, dtype, c, ex); break;
    default: chunk_se_t<64>(pf, s, dtype, c, ex); break;
  }
}

template <typename T>
__global__ void k_to_f32_pad(const T* src, float* dst, int rows, int cols,
                             int rows_p, int cols_p, int transposed) {
  const int64_t total = (int64_t)rows_p * cols_p;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * 256) {
    const int r = (int)(idx / cols_p), c = (int)(idx - (int64_t)r * cols_p);
    float v = 0.f;
    if (src && r < rows && c < cols)
      v = to_f(transposed ? src[(int64_t)c * rows + r]
                          : src[(int64_t)r * cols + c]);
    dst[idx] = v;
  }
}

void launch_to_f32_pad(hipStream_t s, int dtype, const void* src, float* dst,
                       int rows, int cols, int rows_p, int cols_p,
                       bool transposed) {
  const int grid = grid_for((int64_t)rows_p * cols_p, 1024);
  const int tr = transposed ? 1 : 0;
  if (dtype == 0)
    k_to_f32_pad<float><<<grid, 256, 0, s>>>((const float*)src, dst, rows,
                                             cols, rows_p, cols_p, tr);
  else if (dtype == 1)
    k_to_f32_pad<_Float16><<<grid, 256, 0, s>>>((const _Float16*)src, dst,
                                                rows, cols, rows_p, cols_p,
                                                tr);
  else
    k_to_f32_pad<bf16_t><<<grid, 256, 0, s>>>((const bf16_t*)src, dst, rows,
                                              cols, rows_p, cols_p, tr);
}

// ------------------------------------------------------------ chunk mode
// The diff frames of a chunk encoded layer-major (the SparseBatch schedule):
// rulebooks, gather-GEMMs and truncations treat the frames as extra images
// ("items", frame t's sites after frame t-1's); the steps that couple
// frames -- the frame delta against the evolving X_hat, the state update,
// the max-pool over states -- loop over the frames per site in order, so
// every frame sees exactly the state the previous one left.

// Frame-delta decisions: per input site, in frame order, the keep bit and
// the frame whose value X_hat holds at that point; X_hat itself is only
// committed after the deltas are gathered.
template <typename T>
__global__ __launch_bounds__(256) void k_chunk_scan_prep(ChunkScanArgs a) {
  const T* x = (const T*)a.x;
  const T* xhat = (const T*)a.xhat;
  const float thr = a.thr_dev ? *a.thr_dev : a.thr;
  for (int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x; p < a.npix;
       p += (int64_t)gridDim.x * 256) {
    float xh[16];
    for (int c = 0; c < a.C; ++c) xh[c] = to_f(xhat[p * a.C + c]);
    uint8_t cur = 0xFF;
    for (int t = 0; t < a.nf; ++t) {
      const int64_t i = (int64_t)t * a.npix + p;
      const T* xt = x + i * a.C;
      float m = 0.f;
      for (int c = 0; c < a.C; ++c) m = fmaxf(m, fabsf(to_f(xt[c]) - xh[c]));
      const bool k = m > thr;
      a.keep[p * a.nf + t] = k ? 1 : 0;
      a.base[i] = cur;
      if (k) {
        for (int c = 0; c < a.C; ++c) xh[c] = to_f(xt[c]);
        cur = (uint8_t)t;
      }
    }
    a.last[p] = cur;
  }
}

// The same decisions for three-channel (RGB) half-precision frames, eight
// sites per thread: a frame's 24 values of the eight sites arrive as three
// 16-byte loads, and the base bytes of each frame, the sites' keep bytes
// (8·nf consecutive bytes, site-major) and their last bytes leave as 8-byte
// words.  Requires npix a multiple of 8 and aligned buffers (the launcher
// checks).
template <typename T>
__global__ __launch_bounds__(256) void k_chunk_scan_prep_rgb8(
    ChunkScanArgs a) {
  static_assert(sizeof(T) == 2, "half-precision frames");
  const T* x = (const T*)a.x;
  const T* xhat = (const T*)a.xhat;
  const float thr = a.thr_dev ? *a.thr_dev : a.thr;
  const int64_t groups = a.npix / 8;
  for (int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x; g < groups;
       g += (int64_t)gridDim.x * 256) {
    const int64_t p0 = g * 8;
    float xh[24];
#pragma unroll
    for (int v = 0; v < 3; ++v)
      Vec8Half<T>::load(xhat + p0 * 3 + 8 * v, xh + 8 * v);
    uint32_t kb[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) kb[j] = 0u;
    uint64_t cur = ~0ull;  // byte j: the frame X_hat of site j holds
    for (int t = 0; t < a.nf; ++t) {
      const T* xt = x + ((int64_t)t * a.npix + p0) * 3;
      float xv[24];
#pragma unroll
      for (int v = 0; v < 3; ++v) Vec8Half<T>::load(xt + 8 * v, xv + 8 * v);
      *(uint64_t*)(a.base + (int64_t)t * a.npix + p0) = cur;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float m = 0.f;
#pragma unroll
        for (int c = 0; c < 3; ++c)
          m = fmaxf(m, fabsf(xv[3 * j + c] - xh[3 * j + c]));
        if (m > thr) {
          kb[j] |= 1u << t;
#pragma unroll
          for (int c = 0; c < 3; ++c) xh[3 * j + c] = xv[3 * j + c];
          cur = (cur & ~(0xFFull << (8 * j))) | ((uint64_t)t << (8 * j));
        }
      }
    }
    *(uint64_t*)(a.last + p0) = cur;
    // keep bytes of the eight sites, site-major: 8·nf bytes from p0·nf
    uint64_t* kp = (uint64_t*)(a.keep + p0 * a.nf);
    uint64_t w = 0ull;
    int nb = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      for (int t = 0; t < a.nf; ++t) {
        w |= (uint64_t)((kb[j] >> t) & 1u) << (8 * nb);
        if (++nb == 8) {
          *kp++ = w;
          w = 0ull;
          nb = 0;
        }
      }
    }
  }
}

template <typename T>
struct ChunkScanPred {
  const T* x;
  const T* xhat;
  uint8_t* keepb;
  const uint8_t* base;
  T* rows;
  int* rowpix;
  int* act;
  int* map;
  int C, Cp, nf;
  int64_t npix;
  ConsList cons;
  struct Item {
    uint8_t k;
  };
  // items are visited site-major (a site's kept frames adjacent); the
  // keep bytes are stored in that order
  __device__ Item load(int64_t j) const { return Item{keepb[j]}; }
  __device__ bool keep(const Item& it) const { return it.k != 0; }
  // delta against the value X_hat held when frame t arrived
  __device__ unsigned emit(int64_t j, unsigned pos, const Item&) const {
    const int64_t i = site_major(j, nf, npix);
    const int64_t p = i % npix;
    const uint8_t b = base[i];
    const T* xt = x + i * C;
    const T* xb = b == 0xFF ? xhat + p * C : x + ((int64_t)b * npix + p) * C;
    T* r = rows + (int64_t)pos * Cp;
    for (int c = 0; c < Cp; ++c)
      r[c] = c < C ? from_f<T>(to_f(xt[c]) - to_f(xb[c])) : zero_v<T>();
    rowpix[pos] = (int)i;
    act[pos] = (int)i;
    map[i] = (int)pos;
    keepb[j] = 0;
    cons_emit(cons, (int)i, pos, (int)pos);
    return 0u;
  }
  __device__ void drop(int64_t, const Item&) const {}
  __device__ void block_done(unsigned) const {}
  __device__ void finish(unsigned total) const { cons_finish(cons, total); }
};

template <typename T>
__global__ __launch_bounds__(256) void k_chunk_xhat_commit(ChunkScanArgs a) {
  const T* x = (const T*)a.x;
  T* xhat = (T*)a.xhat;
  for (int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x; p < a.npix;
       p += (int64_t)gridDim.x * 256) {
    const uint8_t b = a.last[p];
    if (b == 0xFF) continue;
    for (int c = 0; c < a.C; ++c)
      xhat[p * a.C + c] = x[((int64_t)b * a.npix + p) * a.C + c];
  }
}

template <typename T>
static void chunk_scan_t(const Prof& pf, hipStream_t s,
                         const ChunkScanArgs& a) {
  prof_begin(pf, 0 /*ST_K_SCAN_MASK*/, s);
  bool rgb8 = false;
  if constexpr (sizeof(T) == 2) {
    rgb8 = a.C == 3 && a.npix % 8 == 0 &&
           (((uintptr_t)a.x | (uintptr_t)a.xhat) & 15) == 0 &&
           (((uintptr_t)a.keep | (uintptr_t)a.base | (uintptr_t)a.last) &
            7) == 0;
    if (rgb8)
      k_chunk_scan_prep_rgb8<T>
          <<<grid_for(a.npix / 8, 4096), 256, 0, s>>>(a);
  }
  if (!rgb8)
    k_chunk_scan_prep<T><<<grid_for(a.npix, 4096), 256, 0, s>>>(a);
  prof_end(pf, 0, s);
  ChunkScanPred<T> p{(const T*)a.x, (const T*)a.xhat, a.keep, a.base,
                     (T*)a.rows, a.rowpix, a.act, a.map, a.C, a.Cp, a.nf,
                     a.npix, a.cons};
  const int64_t items = (int64_t)a.nf * a.npix;
  run_compact(pf, 1 /*ST_K_SCAN_COMPACT*/, s, nullptr, items, items, a.tiles,
              a.tiles_clear,
              a.cnt_rows, a.cnt_act, p);
  prof_begin(pf, 1 /*ST_K_SCAN_COMPACT*/, s);
  k_chunk_xhat_commit<T><<<grid_for(a.npix, 4096), 256, 0, s>>>(a);
  prof_end(pf, 1, s);
}

void launch_chunk_scan(const Prof& pf, hipStream_t s, int dtype,
                       const ChunkScanArgs& a) {
  if (dtype == 0)
    chunk_scan_t<float>(pf, s, a);
  else if (dtype == 1)
    chunk_scan_t<_Float16>(pf, s, a);
  else
    chunk_scan_t<bf16_t>(pf, s, a);
}

// State update of a stateful layer over the chunk's frames: per conv site
// (a group of TPS threads, 8 channels each, as in the squeeze-excitation
// kernels), the state stays in registers while the frames that updated the
// site are applied in order; each frame's row gets
// f(P_t) - f(P_{t-1}) and its max |delta|.  Pool mode: the rows get P_t
// instead (the pool compares window states per frame) and the frames that
// updated each site are recorded; the state is committed afterwards.
// CARRY (residual carry, not in pool mode): the site's consumers' view
// stays in registers across the frames; frame t emits f(P_t) - view, and
// if the row is kept (its largest rounded magnitude, over all the site's
// channels -- one group of TPS lanes holds them all -- above the
// threshold) the rounded delta joins the view.
//
// LIST: the sites are those of the affected list O (item = frame * npix +
// site, site-major, so a site's frames are adjacent rows in frame order):
// the group whose row opens a site's run walks the run, the others return;
// untouched sites are not read.  Otherwise (the output layer, whose dense
// output f(P) after every frame is written to `out` for every site) every
// conv site is visited and its rows are found through the map Mo.
template <typename T, int TPS, bool GATE, bool CARRY, bool LIST>
__global__ __launch_bounds__(256) void k_chunk_update(ChunkUpdArgs a) {
  constexpr int R = 256 / TPS, IT = TPS == 64 ? 4 : 1;
  T* dout = (T*)a.dout;
  const int lane = threadIdx.x % TPS;
  const int cp = a.cp, V = cp / 8;
  const uint32_t pu = (uint32_t)a.npix;
  // site p; LIST: j0 is the first row of its run
  auto site_work = [&](int64_t p, int64_t j0) {
  float pv[IT][8], yh[IT][8];
#pragma unroll
  for (int k = 0; k < IT; ++k) {
    const int v = lane + k * TPS;
    if (v < V) state_load8(a.P, a.p16, p * cp + v * 8, pv[k]);
    if (CARRY && v < V) load8f(a.yhat + p * cp + v * 8, yh[k]);
  }
  const float kthr =
      CARRY ? (a.keep_thr_dev ? *a.keep_thr_dev : a.keep_thr) : 0.f;
  uint32_t bits = 0;
  // one frame's row r of this site
  auto apply = [&](int t, int64_t r) {
    bits |= 1u << t;
    float rm = 0.f;
    float dr[IT][8];  // the rounded deltas (residual carry)
#pragma unroll
    for (int k = 0; k < IT; ++k) {
      const int v = lane + k * TPS;
      if (v < V) {
        float dp[8], pn[8];
        float* row = a.dP + r * cp + v * 8;
        load8f(row, dp);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          pn[e] = state_round(a.p16, pv[k][e] + dp[e]);
        if (a.pool_mode) {
          store8f(row, pn);
        } else {
          float d[8];
          if constexpr (GATE) {
            // frozen squeeze-excitation: both values scaled by the gates
            float g[8];
            load8f(gate_slot(a.gate, a.gpar, a.gsz, 0) +
                       (p / a.gate_hw) * cp + v * 8,
                   g);
#pragma unroll
            for (int e = 0; e < 8; ++e)
              d[e] = act_f(pn[e], a.act) * g[e] -
                     act_f(pv[k][e], a.act) * g[e];
          } else if constexpr (CARRY) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              d[e] = act_f(pn[e], a.act) - yh[k][e];
              dr[k][e] = to_f(from_f<T>(d[e]));
            }
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              d[e] = act_f(pn[e], a.act) - act_f(pv[k][e], a.act);
          }
          rm = fmaxf(rm, Vec8<T>::store(dout + r * cp + v * 8, d));
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) pv[k][e] = pn[e];
      }
    }
    if (!a.pool_mode) {
#pragma unroll
      for (int o = 1; o < TPS; o <<= 1) rm = fmaxf(rm, __shfl_xor(rm, o, 64));
      if (lane == 0) a.rowmax[r] = __float_as_uint(rm);
      if (CARRY && rm > kthr) {
        // kept: the consumers receive the rounded delta
#pragma unroll
        for (int k = 0; k < IT; ++k)
#pragma unroll
          for (int e = 0; e < 8; ++e) yh[k][e] += dr[k][e];
      }
    }
  };
  if constexpr (LIST) {
    const int64_t nO = (int64_t)*a.nO;
    for (int64_t r = j0; r < nO; ++r) {
      const uint32_t it = (uint32_t)a.O[r];
      if ((int64_t)(it % pu) != p) break;
      apply((int)(it / pu), r);
    }
  } else {
    for (int t = 0; t < a.nf; ++t) {
      const int r = a.Mo[(int64_t)t * a.npix + p];
      if (r >= 0) apply(t, r);
      if (a.out) {
        float* o = a.out + ((int64_t)t * a.npix + p) * a.c;
#pragma unroll
        for (int k = 0; k < IT; ++k) {
          const int v = lane + k * TPS;
          if (v < V && (a.c & 7) == 0 && ((uintptr_t)a.out & 15) == 0) {
            // whole 8-channel vectors (rows of c floats, c a multiple of
            // 8, on a 16-byte aligned output)
            if (v * 8 < a.c) {
              float f[8];
#pragma unroll
              for (int e = 0; e < 8; ++e) f[e] = act_f(pv[k][e], a.act);
              store8f(o + v * 8, f);
            }
          } else if (v < V) {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              if (v * 8 + e < a.c) o[v * 8 + e] = act_f(pv[k][e], a.act);
          }
        }
      }
    }
  }
  if (a.pool_mode) {
    // LIST: only touched sites get bits; the others stay 0 (the commit
    // clears what it consumed)
    if (lane == 0 && (!LIST || bits)) a.aff[p] = bits;
  } else if (bits) {
#pragma unroll
    for (int k = 0; k < IT; ++k) {
      const int v = lane + k * TPS;
      if (v < V) state_store8(a.P, a.p16, p * cp + v * 8, pv[k]);
      if (CARRY && v < V) store8f(a.yhat + p * cp + v * 8, yh[k]);
    }
  }
  };
  if constexpr (LIST) {
    // every group of TPS lanes strides over the rows; a row's group works
    // only if the row opens its site's run (all lanes of a group agree).
    // The sites are counted (one atomic per block).
    const int64_t nO = (int64_t)*a.nO;
    unsigned nsites = 0;
    for (int64_t j = (int64_t)blockIdx.x * R + threadIdx.x / TPS; j < nO;
         j += (int64_t)gridDim.x * R) {
      const int64_t p = (int64_t)((uint32_t)a.O[j] % pu);
      if (j > 0 && (int64_t)((uint32_t)a.O[j - 1] % pu) == p) continue;
      site_work(p, j);
      nsites += lane == 0 ? 1u : 0u;
    }
    nsites = block_sum(nsites);
    if (threadIdx.x == 0 && nsites && a.sites)
      atomicAdd(a.sites + blockIdx.x % kSiteSlots, (u64)nsites);
  } else {
    const int64_t p = (int64_t)blockIdx.x * R + threadIdx.x / TPS;
    if (p < a.npix) site_work(p, 0);
  }
}

// P of conv site w after frame t (the latest frame <= t that updated it,
// else the chunk's starting state); t < 0: the starting state.
__device__ __forceinline__ const float* state_at(const ChunkPoolArgs& a,
                                                 int64_t w, int t) {
  if (t >= 0) {
    const uint32_t b = a.aff[w] & (uint32_t)((2ull << t) - 1);
    if (b) {
      const int tl = 31 - __clz((int)b);
      const int r = a.Mo[(int64_t)tl * a.nconv + w];
      return a.Pt + (int64_t)r * a.cp;
    }
  }
  return a.P + w * a.cp;
}

// Pooled rows of frame t: max_window f(P after t) - max_window f(P after
// t - 1), as the streaming pool does with its old and new states.
// CARRY (residual carry): the entry that opens a pooled site's run (the
// kept lists are site-major, so a site's frames are adjacent entries)
// walks the run in frame order with the site's consumers' view in
// registers: each frame emits max_win f(P_t) - view, and a kept row (its
// largest rounded magnitude above the threshold) adds its rounded delta to
// the view.
template <typename T, int TPS, bool CARRY>
__global__ __launch_bounds__(256) void k_chunk_pool_emit(ChunkPoolArgs a) {
  constexpr int R = 256 / TPS, IT = TPS == 64 ? 4 : 1;
  T* dout = (T*)a.dout;
  const int lane = threadIdx.x % TPS;
  const int64_t j = (int64_t)blockIdx.x * R + threadIdx.x / TPS;
  const int64_t nQ = (int64_t)*a.nQ;
  if (j >= nQ) return;
  const Geo& g = a.g;
  const int64_t qi = a.Q[j];
  const int64_t q = qi % a.npool;
  if (CARRY && j > 0 && (int64_t)a.Q[j - 1] % a.npool == q) return;
  const int64_t hwq = (int64_t)g.Ho * g.Wo;
  const int n = (int)(q / hwq);
  const int rem = (int)(q - n * hwq);
  const int qy = rem / g.Wo, qx = rem - (rem / g.Wo) * g.Wo;
  const int cp = a.cp, V = cp / 8;
  // max over the window of f(P after frame t), 8 channels from v * 8
  auto pooled = [&](int t, int v, float* mx) {
#pragma unroll
    for (int e = 0; e < 8; ++e) mx[e] = -INFINITY;
    for (int ky = 0; ky < g.kh; ++ky) {
      const int iy = qy * g.sh - g.ph + ky;
      if (iy < 0 || iy >= g.Hi) continue;
      for (int kx = 0; kx < g.kw; ++kx) {
        const int ix = qx * g.sw - g.pw + kx;
        if (ix < 0 || ix >= g.Wi) continue;
        const int64_t w = ((int64_t)n * g.Hi + iy) * g.Wi + ix;
        float vv[8];
        load8f(state_at(a, w, t) + v * 8, vv);
#pragma unroll
        for (int e = 0; e < 8; ++e) mx[e] = fmaxf(mx[e], act_f(vv[e], a.act));
      }
    }
  };
  if constexpr (!CARRY) {
    const int t = (int)(qi / a.npool);
    float rm = 0.f;
#pragma unroll
    for (int k = 0; k < IT; ++k) {
      const int v = lane + k * TPS;
      if (v >= V) continue;
      float mn[8], mo[8], d[8];
      pooled(t, v, mn);
      pooled(t - 1, v, mo);
#pragma unroll
      for (int e = 0; e < 8; ++e) d[e] = mn[e] - mo[e];
      rm = fmaxf(rm, Vec8<T>::store(dout + j * cp + v * 8, d));
    }
#pragma unroll
    for (int o = 1; o < TPS; o <<= 1) rm = fmaxf(rm, __shfl_xor(rm, o, 64));
    if (lane == 0) a.rowmax[j] = __float_as_uint(rm);
  } else {
    const float kthr = a.keep_thr_dev ? *a.keep_thr_dev : a.keep_thr;
    float yh[IT][8];
#pragma unroll
    for (int k = 0; k < IT; ++k) {
      const int v = lane + k * TPS;
      if (v < V) load8f(a.yhat + q * cp + v * 8, yh[k]);
    }
    for (int64_t jj = j; jj < nQ; ++jj) {
      const int64_t qj = a.Q[jj];
      if (qj % a.npool != q) break;
      const int t = (int)(qj / a.npool);
      float rm = 0.f, dr[IT][8];
#pragma unroll
      for (int k = 0; k < IT; ++k) {
        const int v = lane + k * TPS;
        if (v >= V) continue;
        float mn[8], d[8];
        pooled(t, v, mn);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          d[e] = mn[e] - yh[k][e];
          dr[k][e] = to_f(from_f<T>(d[e]));
        }
        rm = fmaxf(rm, Vec8<T>::store(dout + jj * cp + v * 8, d));
      }
#pragma unroll
      for (int o = 1; o < TPS; o <<= 1) rm = fmaxf(rm, __shfl_xor(rm, o, 64));
      if (lane == 0) a.rowmax[jj] = __float_as_uint(rm);
      if (rm > kthr) {
#pragma unroll
        for (int k = 0; k < IT; ++k)
#pragma unroll
          for (int e = 0; e < 8; ++e) yh[k][e] += dr[k][e];
      }
    }
#pragma unroll
    for (int k = 0; k < IT; ++k) {
      const int v = lane + k * TPS;
      if (v < V) store8f(a.yhat + q * cp + v * 8, yh[k]);
    }
  }
}

// P[w] = P after the last frame that updated w, for the sites of the
// affected list O (run openers; 4 channels per thread of a group of cp / 4
// threads), and the site's frame bits cleared for the next pooled layer.
__global__ __launch_bounds__(256) void k_chunk_commit(int p16, float* P,
                                                      const float* Pt,
                                                      const int* O,
                                                      const u64* nOp,
                                                      uint32_t* aff,
                                                      int64_t nconv, int cp) {
  const int c4 = cp / 4;
  const int64_t nO = (int64_t)*nOp;
  const int64_t total = nO * c4;
  const uint32_t pu = (uint32_t)nconv;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * 256) {
    const int64_t j = idx / c4;
    const int c = (int)(idx - j * c4) * 4;
    const uint32_t w = (uint32_t)O[j] % pu;
    if (j > 0 && (uint32_t)O[j - 1] % pu == w) continue;  // not the opener
    // the run's last row holds the state after its last frame
    int64_t r = j;
    while (r + 1 < nO && (uint32_t)O[r + 1] % pu == w) ++r;
    state_store4(P, p16 != 0, (int64_t)w * cp + c,
                 *(const float4*)(Pt + r * cp + c));
    if (c == 0) aff[w] = 0u;
  }
}

template <typename T, int TPS, bool LIST>
static void chunk_upd_t(hipStream_t s, const ChunkUpdArgs& a, int grid) {
  if (a.gate)
    k_chunk_update<T, TPS, true, false, LIST><<<grid, 256, 0, s>>>(a);
  else if (a.yhat && !a.pool_mode)
    k_chunk_update<T, TPS, false, true, LIST><<<grid, 256, 0, s>>>(a);
  else
    k_chunk_update<T, TPS, false, false, LIST><<<grid, 256, 0, s>>>(a);
}

// Without a dense output the update walks the affected list (a group per
// row, its run's opener working); with one, every conv site.
template <typename T, int TPS>
static void chunk_upd_t(hipStream_t s, const ChunkUpdArgs& a) {
  constexpr int R = 256 / TPS;
  if (a.out) {
    chunk_upd_t<T, TPS, false>(s, a, (int)((a.npix + R - 1) / R));
  } else {
    const int64_t cap = a.npix * a.nf;
    chunk_upd_t<T, TPS, true>(s, a, grid_for(cap * TPS, 8192));
  }
}

template <typename T>
static void chunk_upd_d(hipStream_t s, const ChunkUpdArgs& a) {
  switch (a.tps) {
    case 1: chunk_upd_t<T, 1>(s, a); break;
    case 2: chunk_upd_t<T, 2>(s, a); break;
    case 4: chunk_upd_t<T, 4>(s, a); break;
    case 8: chunk_upd_t<T, 8>(s, a); break;
    case 16: chunk_upd_t<T, 16>(s, a); break;
    case 32: chunk_upd_t<T, 32>(s, a); break;
    default: chunk_upd_t<T, 64>(s, a); break;
  }
}

void launch_chunk_update(const Prof& pf, hipStream_t s, int dtype,
                         const ChunkUpdArgs& a) {
  prof_begin(pf, 23 /*ST_K_CHUNK_UPDATE*/, s);
  if (dtype == 0)
    chunk_upd_d<float>(s, a);
  else if (dtype == 1)
    chunk_upd_d<_Float16>(s, a);
  else
    chunk_upd_d<bf16_t>(s, a);
  prof_end(pf, 23, s);
}

template <typename T, int TPS>
static void chunk_pool_t(hipStream_t s, const ChunkPoolArgs& a) {
  constexpr int R = 256 / TPS;
  const int grid = (int)((a.capQ + R - 1) / R);
  if (a.yhat)
    k_chunk_pool_emit<T, TPS, true><<<grid, 256, 0, s>>>(a);
  else
    k_chunk_pool_emit<T, TPS, false><<<grid, 256, 0, s>>>(a);
}

template <typename T>
static void chunk_pool_d(hipStream_t s, const ChunkPoolArgs& a) {
  switch (a.tps) {
    case 1: chunk_pool_t<T, 1>(s, a); break;
    case 2: chunk_pool_t<T, 2>(s, a); break;
    case 4: chunk_pool_t<T, 4>(s, a); break;
    case 8: chunk_pool_t<T, 8>(s, a); break;
    case 16: chunk_pool_t<T, 16>(s, a); break;
    case 32: chunk_pool_t<T, 32>(s, a); break;
    default: chunk_pool_t<T, 64>(s, a); break;
  }
}

void launch_chunk_pool_emit(const Prof& pf, hipStream_t s, int dtype,
                            const ChunkPoolArgs& a) {
  prof_begin(pf, 12 /*ST_K_POOL_EMIT*/, s);
  if (dtype == 0)
    chunk_pool_d<float>(s, a);
  else if (dtype == 1)
    chunk_pool_d<_Float16>(s, a);
  else
    chunk_pool_d<bf16_t>(s, a);
  prof_end(pf, 12, s);
}

void launch_chunk_commit(const Prof& pf, hipStream_t s, int p16, float* P,
                         const float* Pt, const int* O, const u64* nO,
                         uint32_t* aff, int64_t capO, int64_t nconv, int cp) {
  prof_begin(pf, 13 /*ST_K_COMMIT*/, s);
  k_chunk_commit<<<grid_for(capO * (cp / 4), 8192), 256, 0, s>>>(
      p16, P, Pt, O, nO, aff, nconv, cp);
  prof_end(pf, 13, s);
}

// ------------------------------------------------------- dense output
__global__ __launch_bounds__(256) void k_output(const float* P, int p16,
                                                int cp, int C, int N, Geo g,
                                                int has_pool, int act,
                                                const float* se_base,
                                                const int* se_par,
                                                int se_flip, float* out) {
  const float* se =
      se_base ? gate_slot(se_base, se_par, (int64_t)N * cp, se_flip)
              : nullptr;
  // g.Hi/Wi: conv grid; g.Ho/Wo: output grid (== conv grid without pool)
  const int64_t total = (int64_t)N * g.Ho * g.Wo * C;
  const int64_t hwo = (int64_t)g.Ho * g.Wo;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * 256) {
    const int64_t q = idx / C;
    const int c = (int)(idx - q * C);
    if (!has_pool) {
      const float v = act_f(state_load1(P, p16, q * cp + c), act);
      out[idx] = se ? v * se[(q / hwo) * cp + c] : v;
      continue;
    }
    const int n = (int)(q / hwo);
    const int rem = (int)(q - n * hwo);
    const int qy = rem / g.Wo, qx = rem - (rem / g.Wo) * g.Wo;
    float m = -INFINITY;
    for (int ky = 0; ky < g.kh; ++ky) {
      const int iy = qy * g.sh - g.ph + ky;
      if (iy < 0 || iy >= g.Hi) continue;
      for (int kx = 0; kx < g.kw; ++kx) {
        const int ix = qx * g.sw - g.pw + kx;
        if (ix < 0 || ix >= g.Wi) continue;
        m = fmaxf(m, act_f(state_load1(
                               P, p16,
                               (((int64_t)n * g.Hi + iy) * g.Wi + ix) * cp + c),
                           act));
      }
    }
    out[idx] = m;
  }
}

void launch_output(const Prof& pf, hipStream_t s, const float* P, int p16,
                   int cp, int C, int N, Geo g, int has_pool, int act,
                   const float* se, const int* se_par, int se_flip,
                   float* out) {
  prof_begin(pf, 16 /*ST_K_OUTPUT*/, s);
  k_output<<<grid_for((int64_t)N * g.Ho * g.Wo * C, 8192), 256, 0, s>>>(
      P, p16, cp, C, N, g, has_pool, act, se, se_par, se_flip, out);
  prof_end(pf, 16, s);
}

__global__ void k_flip_parity(int* par) {
  if (threadIdx.x == 0) *par ^= 1;
}

void launch_flip_parity(hipStream_t s, int* par) {
  k_flip_parity<<<1, 64, 0, s>>>(par);
}

// ------------------------------------------------------- bookkeeping
__global__ void k_reset(u64* cnt, int n, uint32_t* status) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) cnt[i] = 0ull;
  for (int i = threadIdx.x; i < kCompactMaxTiles; i += blockDim.x)
    status[i] = 0u;
}

void launch_reset(const Prof& pf, hipStream_t s, u64* cnt, int n,
                  uint32_t* status) {
  prof_begin(pf, 18 /*ST_K_RESET*/, s);
  k_reset<<<1, 256, 0, s>>>(cnt, n, status);
  prof_end(pf, 18, s);
}

__global__ __launch_bounds__(256) void k_cleanup(const CleanEntry* tab,
                                                 char* ws, const u64* cnt) {
  const CleanEntry e = tab[blockIdx.y];
  int* map = (int*)(ws + e.map_off);
  const int* list = (const int*)(ws + e.list_off);
  const int64_t n = (int64_t)cnt[e.cnt];
  for (int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x; r < n;
       r += (int64_t)gridDim.x * 256)
    map[list[r]] = -1;
}

void launch_cleanup(const Prof& pf, hipStream_t s, const CleanEntry* tab,
                    int n_tab, char* ws, const u64* cnt, int64_t max_rows) {
  prof_begin(pf, 17 /*ST_K_CLEANUP*/, s);
  dim3 grid(grid_for(max_rows, 512), n_tab);
  k_cleanup<<<grid, 256, 0, s>>>(tab, ws, cnt);
  prof_end(pf, 17, s);
}

// ----------------------------------------------- dense reference pass
// The reference frame encodes every pixel (every delta kept, the state
// treated as zero), so its rows need no compaction: each tensor's rows are
// its pixels in order.
template <typename T>
__global__ __launch_bounds__(256) void k_dense_input(const T* x, T* xhat,
                                                     T* rows, int C, int Cp,
                                                     int64_t npix) {
  for (int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x; p < npix;
       p += (int64_t)gridDim.x * 256) {
    for (int c = 0; c < Cp; ++c) {
      T v = zero_v<T>();
      if (c < C) {
        v = x[p * C + c];
        xhat[p * C + c] = v;
      }
      rows[p * Cp + c] = v;
    }
  }
}

void launch_dense_input(const Prof& pf, hipStream_t s, int dtype,
                        const void* x, void* xhat, void* rows, int C, int Cp,
                        int64_t npix) {
  const int grid = grid_for(npix, 8192);
  prof_begin(pf, 1 /*ST_K_SCAN_COMPACT*/, s);
  if (dtype == 0)
    k_dense_input<float><<<grid, 256, 0, s>>>(
        (const float*)x, (float*)xhat, (float*)rows, C, Cp, npix);
  else if (dtype == 1)
    k_dense_input<_Float16><<<grid, 256, 0, s>>>(
        (const _Float16*)x, (_Float16*)xhat, (_Float16*)rows, C, Cp, npix);
  else
    k_dense_input<bf16_t><<<grid, 256, 0, s>>>(
        (const bf16_t*)x, (bf16_t*)xhat, (bf16_t*)rows, C, Cp, npix);
  prof_end(pf, 1, s);
}

__global__ __launch_bounds__(256) void k_iota_lists(const IotaEntry* tab,
                                                    char* ws) {
  const IotaEntry e = tab[blockIdx.y];
  int* list = (int*)(ws + e.off);
  for (int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x; r < e.n;
       r += (int64_t)gridDim.x * 256)
    list[r] = (int)r;
}

void launch_iota_lists(const Prof& pf, hipStream_t s, const IotaEntry* tab,
                       int n_tab, char* ws, int64_t max_n) {
  if (n_tab < 1) return;
  const dim3 grid(grid_for(max_n, 1024), n_tab);
  prof_begin(pf, 17 /*ST_K_CLEANUP*/, s);
  k_iota_lists<<<grid, 256, 0, s>>>(tab, ws);
  prof_end(pf, 17, s);
}

__global__ void k_copy_u64(u64* dst, const u64* src, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) dst[i] = src[i];
}

void launch_copy_u64(hipStream_t s, u64* dst, const u64* src, int n) {
  k_copy_u64<<<1, 256, 0, s>>>(dst, src, n);
}

// One thread per 8 channels of a pooled pixel: the largest f(P) over the
// window's conv sites (g: Hi/Wi the conv grid, Ho/Wo the pooled grid), as
// the frame-by-frame pool emission computes it with an all-zero previous
// state (max f(P) - max f(0), f(0) = 0).
template <typename T, int ACT>
__device__ __forceinline__ void pool_dense_rows(const float* P, int p16,
                                                T* dout, const Geo& g,
                                                int cp, int64_t nq) {
  const int cpr = cp / 8;
  const int64_t hwq = (int64_t)g.Ho * g.Wo;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
       idx < nq * cpr; idx += (int64_t)gridDim.x * 256) {
    const int64_t q = idx / cpr;
    const int c0 = (int)(idx - q * cpr) * 8;
    const int n = (int)(q / hwq);
    const int rem = (int)(q - n * hwq);
    const int qy = rem / g.Wo, qx = rem - (rem / g.Wo) * g.Wo;
    float m[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) m[e] = -INFINITY;
    for (int ky = 0; ky < g.kh; ++ky) {
      const int iy = qy * g.sh - g.ph + ky;
      if (iy < 0 || iy >= g.Hi) continue;
      for (int kx = 0; kx < g.kw; ++kx) {
        const int ix = qx * g.sw - g.pw + kx;
        if (ix < 0 || ix >= g.Wi) continue;
        const int64_t w = ((int64_t)n * g.Hi + iy) * g.Wi + ix;
        float v[8];
        state_load8(P, p16 != 0, w * cp + c0, v);
#pragma unroll
        for (int e = 0; e < 8; ++e) m[e] = fmaxf(m[e], act_c<ACT>(v[e]));
      }
    }
    (void)Vec8<T>::store(dout + q * cp + c0, m);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_pool_dense(const float* P, int p16,
                                                    T* dout, Geo g, int cp,
                                                    int act, int64_t nq) {
  with_act(act, [&](auto act_tag) {
    pool_dense_rows<T, decltype(act_tag)::value>(P, p16, dout, g, cp, nq);
  });
}

void launch_pool_dense(const Prof& pf, hipStream_t s, int dtype,
                       const float* P, int p16, void* dout, Geo g, int cp,
                       int act, int64_t nq) {
  const int grid = grid_for(nq * (cp / 8), 8192);
  prof_begin(pf, 12 /*ST_K_POOL_EMIT*/, s);
  if (dtype == 0)
    k_pool_dense<float><<<grid, 256, 0, s>>>(P, p16, (float*)dout, g, cp,
                                             act, nq);
  else if (dtype == 1)
    k_pool_dense<_Float16><<<grid, 256, 0, s>>>(P, p16, (_Float16*)dout, g,
                                                cp, act, nq);
  else
    k_pool_dense<bf16_t><<<grid, 256, 0, s>>>(P, p16, (bf16_t*)dout, g, cp,
                                              act, nq);
  prof_end(pf, 12, s);
}

__global__ void k_fill_u32(uint32_t* p, int64_t n, uint32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * 256)
    p[i] = v;
}

void launch_fill_u32(hipStream_t s, void* p, int64_t n, uint32_t v) {
  k_fill_u32<<<grid_for(n, 8192), 256, 0, s>>>((uint32_t*)p, n, v);
}

// Weight repack: PyTorch [cout][cin][kh][kw] -> [cout_p][ktot_p] with the
// reduction index r = (ky * kw + kx) * cin_p + ci, zero padded.
template <typename T>
__global__ void k_repack_dense(const T* w, T* wt, int cout, int cin, int kh,
                               int kw, int cin_p, int cout_p, int64_t ktot_p) {
  const int64_t total = (int64_t)cout_p * ktot_p;
  const int K = kh * kw;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * 256) {
    const int n = (int)(idx / ktot_p);
    const int64_t r = idx - (int64_t)n * ktot_p;
    const int k = (int)(r / cin_p);
    const int ci = (int)(r - (int64_t)k * cin_p);
    T v = zero_v<T>();
    if (n < cout && k < K && ci < cin) {
      const int ky = k / kw, kx = k - (k / kw) * kw;
      v = w[(((int64_t)n * cin + ci) * kh + ky) * kw + kx];
    }
    wt[idx] = v;
  }
}

void launch_repack_dense(hipStream_t s, int dtype, const void* w, void* wt,
                         int cout, int cin, int kh, int kw, int cin_p,
                         int cout_p, int64_t ktot_p) {
  const int grid = grid_for((int64_t)cout_p * ktot_p, 8192);
  if (dtype == 0)
    k_repack_dense<float><<<grid, 256, 0, s>>>((const float*)w, (float*)wt,
                                               cout, cin, kh, kw, cin_p,
                                               cout_p, ktot_p);
  else if (dtype == 1)
    k_repack_dense<_Float16><<<grid, 256, 0, s>>>(
        (const _Float16*)w, (_Float16*)wt, cout, cin, kh, kw, cin_p, cout_p,
        ktot_p);
  else
    k_repack_dense<bf16_t><<<grid, 256, 0, s>>>((const bf16_t*)w, (bf16_t*)wt,
                                                cout, cin, kh, kw, cin_p,
                                                cout_p, ktot_p);
}

template <typename T>
__global__ void k_repack_dw(const T* w, float* wdw, int c, int kh, int kw,
                            int cp) {
  const int K = kh * kw;
  const int64_t total = (int64_t)K * cp;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * 256) {
    const int k = (int)(idx / cp);
    const int ch = (int)(idx - (int64_t)k * cp);
    wdw[idx] = ch < c ? to_f(w[(int64_t)ch * K + k]) : 0.f;
  }
}

void launch_repack_dw(hipStream_t s, int dtype, const void* w, float* wdw,
                      int c, int kh, int kw, int cp) {
  const int grid = grid_for((int64_t)kh * kw * cp);
  if (dtype == 0)
    k_repack_dw<float><<<grid, 256, 0, s>>>((const float*)w, wdw, c, kh, kw,
                                            cp);
  else if (dtype == 1)
    k_repack_dw<_Float16><<<grid, 256, 0, s>>>((const _Float16*)w, wdw, c, kh,
                                               kw, cp);
  else
    k_repack_dw<bf16_t><<<grid, 256, 0, s>>>((const bf16_t*)w, wdw, c, kh, kw,
                                             cp);
}

template <typename T>
__global__ void k_bias(const T* b, float* out, int cout, int cout_p) {
  for (int i = threadIdx.x; i < cout_p; i += blockDim.x)
    out[i] = (b && i < cout) ? to_f(b[i]) : 0.f;
}

void launch_bias(hipStream_t s, int dtype, const void* b, float* out,
                 int cout, int cout_p) {
  if (dtype == 0)
    k_bias<float><<<1, 256, 0, s>>>((const float*)b, out, cout, cout_p);
  else if (dtype == 1)
    k_bias<_Float16><<<1, 256, 0, s>>>((const _Float16*)b, out, cout, cout_p);
  else
    k_bias<bf16_t><<<1, 256, 0, s>>>((const bf16_t*)b, out, cout, cout_p);
}

// Per-image kept counts of an ascending pixel list (binary search of the
// image boundaries).
// ------------------------------------------------------- residual carry
template <typename T>
__global__ __launch_bounds__(256) void k_carry_commit(const int* act,
                                                     const u64* n_act,
                                                     const int* map,
                                                     const T* rows,
                                                     float* view, int cp) {
  const int64_t n = (int64_t)*n_act;
  const int c4 = cp / 4;
  const int64_t total = n * c4;
  for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * 256) {
    const int64_t k = idx / c4;
    const int c = (int)(idx - k * c4) * 4;
    const int pix = act[k];
    const T* rv = rows + (int64_t)map[pix] * cp + c;
    float4* vp = (float4*)(view + (int64_t)pix * cp + c);
    float4 v = *vp;
    v.x += to_f(rv[0]);
    v.y += to_f(rv[1]);
    v.z += to_f(rv[2]);
    v.w += to_f(rv[3]);
    *vp = v;
  }
}

void launch_carry_commit(const Prof& pf, hipStream_t s, int dtype,
                         const int* act, const u64* n_act, int64_t cap,
                         const int* map, const void* rows, float* view,
                         int cp) {
  const int grid = grid_for(cap * (cp / 4), 8192);
  prof_begin(pf, 25 /*ST_K_CARRY_COMMIT*/, s);
  if (dtype == 0)
    k_carry_commit<float><<<grid, 256, 0, s>>>(act, n_act, map,
                                              (const float*)rows, view, cp);
  else if (dtype == 1)
    k_carry_commit<_Float16><<<grid, 256, 0, s>>>(
        act, n_act, map, (const _Float16*)rows, view, cp);
  else
    k_carry_commit<bf16_t><<<grid, 256, 0, s>>>(act, n_act, map,
                                               (const bf16_t*)rows, view, cp);
  prof_end(pf, 25, s);
}

// ------------------------------------------- online threshold adjustment
// One bisection step per controlled tensor, in f64 as the host controller
// takes it; the f32 threshold is theta rounded to nearest.
__global__ void k_ibst_step(const u64* counters, int nf, IbstArgs a) {
  for (int t = threadIdx.x; t < a.n; t += blockDim.x) {
    if (!a.ctl[t]) continue;
    const double sp = 1.0 - (double)counters[2 * t + 1] /
                                ((double)a.sites[t] * (double)nf);
    double th = a.theta[t];
    if (sp < a.target - a.eps) {
      a.lo[t] = th;
      th = 0.5 * (th + a.hi[t]);
    } else if (sp > a.target + a.eps) {
      a.hi[t] = th;
      th = 0.5 * (a.lo[t] + th);
    }
    a.theta[t] = th;
    a.thr[t] = (float)th;
  }
}

__global__ void k_ibst_restart(IbstArgs a) {
  for (int t = threadIdx.x; t < a.n; t += blockDim.x)
    if (a.ctl[t]) {
      a.lo[t] = 0.0;
      a.hi[t] = a.theta_max;
    }
}

void launch_ibst_step(hipStream_t s, const u64* counters, int nf,
                      const IbstArgs& a) {
  k_ibst_step<<<1, 256, 0, s>>>(counters, nf, a);
}

void launch_ibst_restart(hipStream_t s, const IbstArgs& a) {
  k_ibst_restart<<<1, 256, 0, s>>>(a);
}

// Kept rows per image (image = item / hw) of a kept list in any order: a
// per-block histogram in LDS (up to kDensityLdsImages images; beyond that,
// device atomics directly), added to `out` (zeroed first).
constexpr int kDensityLdsImages = 4096;

__global__ __launch_bounds__(256) void k_density(const int* act,
                                                 const u64* n_act,
                                                 int64_t hw, int images,
                                                 u64* out) {
  __shared__ unsigned h[kDensityLdsImages];
  const bool lds = images <= kDensityLdsImages;
  if (lds)
    for (int b = threadIdx.x; b < images; b += 256) h[b] = 0u;
  __syncthreads();
  const int64_t n = (int64_t)*n_act;
  for (int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x; r < n;
       r += (int64_t)gridDim.x * 256) {
    const int b = (int)((int64_t)act[r] / hw);
    if (lds)
      atomicAdd(&h[b], 1u);
    else
      atomicAdd(out + b, (u64)1);
  }
  __syncthreads();
  if (lds)
    for (int b = threadIdx.x; b < images; b += 256)
      if (h[b]) atomicAdd(out + b, (u64)h[b]);
}

void launch_density(hipStream_t s, const int* act, const u64* n_act,
                    int64_t cap, int64_t hw, int images, u64* out) {
  launch_fill_u32(s, out, 2 * (int64_t)images, 0u);
  k_density<<<grid_for(cap, 1024), 256, 0, s>>>(act, n_act, hw, images,
                                                 out);
}

}  // namespace st
