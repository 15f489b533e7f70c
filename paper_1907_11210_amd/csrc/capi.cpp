// capi.cpp -- the C ABI of libhuge2 (declared in include/huge2.h).
//
// plan_create runs the host-side decomposition (plan.cpp), lays the
// segments, taps and GEMM work list out for the device, and packs the
// weights; plan_execute enqueues the phase GEMM (preceded by an input
// re-layout when the input is NCHW or has a ragged channel count).  No
// exception crosses the ABI.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <queue>
#include <vector>

#include "huge2.h"
#include "kernels.hpp"
#include "plan.hpp"

using namespace huge2;

// Where a plan's device buffers come from: hipMalloc, hipMallocAsync on the
// plan's stream (stream_ordered, the one-shot entry points), or a bump
// allocation from a caller-provided region (arena, the no-allocation entry
// point), which the plan never frees.
struct Arena {
  char* base;
  size_t cap, used;
};
struct Mem {
  bool stream_ordered = false;
  Arena* arena = nullptr;
};

struct huge2_plan {
  huge2_conv_desc desc;
  int transposed;
  int ho, wo;
  int cfg;
  bool staged;    // input re-laid out into xs first
  int c_stride;   // channels per pixel of the GEMM's input
  int cin_pad, cout_pad;
  size_t x_bytes, wp_bytes;  // extents of the GEMM's input and packed weights
  int n_works;
  void* wp;    // packed weights
  void* meta;  // segments, taps, work list
  void* xs;    // staged input (or null)
  SegDev* d_segs;
  TapDev* d_taps;
  WorkDev* d_works;
  const uint32_t* d_ptab;  // pixel table of a listed plan (or null)
  Mem mem;  // where the buffers came from (see Mem)
  hipStream_t alloc_stream;
  int64_t nonzero_macs, issued_macs;
  bool ztile;   // all-taps form for few output channels (no GEMM work list)
  ZArgs zargs;  // its launch shape (pointers filled per call)
  bool rowphase;  // output-stationary form for large strides
  RpArgs rpargs;
  bool colphase;  // column-phase form for a column stride of 32
  CpArgs cpargs;
  bool grouped;   // grouped / depthwise: the direct kernel over a copy of w
  GrArgs grargs;
  bool quad;      // all-phase form of the stride-2, 4x4, padding-1 layer
  QArgs qargs;
  int bias_div;   // GEMM columns per bias entry (r * s for the 1x1-input product form)
  int bias_mod;   // > 0: bias entries repeat every bias_mod columns (its NHWC form)
  int prod_rs;    // > 0: the NHWC product form's weights are packed tap-major
  int ksplit;     // K slices across workgroups (1: none)
  void* part;     // their fp32 partial outputs, ksplit x |y| (or null)
  huge2_plan* inner;  // two-pass all-taps form: the per-tap pointwise GEMM; gather form: the
                      // pointwise GEMM over the gathered receptive fields (or null)
  bool gather;        // gather form: staging = the receptive-field gather into inner->xs
  void* zbuf;         // its output, the per-tap products (fp32 NCHW)
  char kernel_name[64];
  // host copies of the GEMM metadata, for grouped launches (huge2_group)
  std::vector<SegDev> h_segs;
  std::vector<TapDev> h_taps;
  std::vector<WorkDev> h_works;
  std::vector<uint32_t> h_ptab;
};

// Several GEMM plans of one input run as one launch: their segments, taps,
// works and pixel tables concatenated (each segment naming its plan), the
// works ordered by image and, inside an image, by decreasing cost.
struct huge2_group {
  int count;
  const huge2_plan* plans[huge2::kMaxGroup];
  void* meta;
  huge2::SegDev* d_segs;
  huge2::TapDev* d_taps;
  huge2::WorkDev* d_works;
  const uint32_t* d_ptab;
  int n_works;
  int cfg;  // launch tile: the plans' own, or its two-per-CU form for long lists
  char kernel_name[64];
};

namespace {

int elem_size(int dtype) { return dtype == HUGE2_BF16 ? 2 : 4; }
int round_up(int v, int m) { return (v + m - 1) / m * m; }

// Fault injection for host-side tests of the error paths: HUGE2_FAULT=alloc
// makes the next device allocation fail, HUGE2_FAULT=launch the next launch.
bool fault(const char* what) {
  const char* f = std::getenv("HUGE2_FAULT");
  return f && std::strcmp(f, what) == 0;
}

int env_int(const char* name, int dflt) {
  const char* v = std::getenv(name);
  if (!v || !*v) return dflt;
  return std::atoi(v);
}

long long count_works(const huge2_conv_desc& d, bool transposed, int class_split, int cfg) {
  PlanShape shape;
  const int bm = tile_bm(cfg), bn = tile_bn(cfg);
  if (!build_shape(d, transposed, class_split, bm, &shape)) return 0;
  long long works = 0;
  const long long ntiles = (d.c_out + bn - 1) / bn;
  for (const huge2_segment& s : shape.segs) {
    long long m = (long long)d.n * s.nphase_h * s.nphase_w * s.qn_h * s.qn_w;
    works += (m + bm - 1) / bm * ntiles;
  }
  return works;
}

// Tile choice, from measurements on MI355X.  bf16: many pixels and at most
// 128 output channels take the pipelined 4-wave 128 x 128 tile for
// transposed convs (the odd-kernel layer 20.4 against 23.0 us, the NHWC
// generator's third layer 33.4 against 37.9 us) and the two-operand 8-wave
// tile of that shape for convs (the gathered data gradient of the
// generator's last layer, one short K stage: 25.8 against 33.1 us); 256 or
// more output
// channels take the pipelined 8-wave 128 x 256 tile when every CU gets one
// (the atrous pyramid: twice the pixels per weight fetch of 64 x 256, which
// its L2 traffic needs; its three-buffer pipeline measured 1090 against 955
// TFLOP/s for the split-wave kernel of the same tile on the grouped pyramid),
// else the 64 x 256 one with plenty of its tiles; otherwise the split-wave
// tiles with two K groups per workgroup, 128 x 128 when that still gives
// every CU a tile, else 64 x 128 (few pixels and long K: the first DCGAN
// layers).  A pointwise GEMM of at most 64 pixel rows and many channels (a
// generator's projection of z) takes the 4-wave 32 x 256 tile: two row tiles,
// and no second K group idling on its single K stage.  Few output channels
// take the narrow 128 x 32 tile.  fp32 keeps the two-operand-LDS tiles.
int choose_cfg(const huge2_conv_desc& d, bool transposed, int class_split) {
  int forced = env_int("HUGE2_TILE", -1);
  if (forced >= 0 && forced < TILE_COUNT) return forced;
  if (d.c_out <= 32) return TILE_128x32;
  const bool large = count_works(d, transposed, class_split, TILE_128x128) >= 512;
  if (d.dtype != HUGE2_BF16) return large ? TILE_128x128 : TILE_64x128;
  if (large && d.c_out <= 128) return transposed ? TILE_P3_128x128 : TILE_128x128;
  if (d.r == 1 && d.s == 1 && (long long)d.n * d.h * d.w <= 64 && d.c_out >= 256)
    return TILE_SW_32x256;  // a pointwise GEMM of at most 64 rows (the 1x1-input product form)
  if (d.c_out >= 256) {
    const long long w3 = count_works(d, transposed, class_split, TILE_P3_128x256);
    // two workgroups per CU (its fallback for tap lists, the 128 x 256
    // split-wave tile, takes 128-byte K blocks)
    if (w3 >= 2 * kComputeUnits && d.c_in % (tile_kb(TILE_SW_128x256) / elem_size(d.dtype)) == 0)
      return TILE_P3_128x256_W4;
    if (w3 >= kComputeUnits) return TILE_P3_128x256;
  }
  if (d.c_out >= 256 && count_works(d, transposed, class_split, TILE_SW_64x256) >= 384)
    return TILE_SW_64x256;
  if (count_works(d, transposed, class_split, TILE_SW_128x128_K2) >= kComputeUnits)
    return TILE_SW_128x128_K2;
  return TILE_SW_64x128_K2;
}

// Order the work list for the eight XCDs.  The kernel hands work index
// chunk x (contiguous, works/8 long) to the workgroups that the dispatcher
// places on XCD x, and each XCD has its own L2.  The works are split into
// eight cells, a ranges of spatial position (image, then output row of the
// phase) times b ranges of output-channel tiles (a * b = 8), choosing the
// split that minimises the bytes every XCD must fetch (input / a + packed
// weights / b).  All phases and border classes of one region land in the same
// cell, so the input rows they share are read into one L2 and each output
// cache line is completed by one XCD.  Inside a cell the works run in order of
// position, then segment, then tile.
void order_works_for_xcds(std::vector<WorkDev>& works, const std::vector<SegDev>& segs, int nimg,
                          int ho, int bn, int ntiles_n, double x_bytes, double w_bytes) {
  if (works.size() < 16) return;
  int best_b = 1;
  double best = 1e300;
  for (int b = 1; b <= 8; b *= 2) {
    if (b > ntiles_n) break;
    const double cost = x_bytes / (8 / b) + w_bytes / b;
    if (cost < best) {
      best = cost;
      best_b = b;
    }
  }
  const int b = best_b, a = 8 / best_b;
  struct Key {
    int64_t cell, pos;
    WorkDev w;
  };
  std::vector<Key> keys;
  keys.reserve(works.size());
  for (const WorkDev& w : works) {
    const SegDev& sg = segs[w.seg];
    int64_t j = w.m0;
    j /= sg.qn_w;
    const int64_t a_h = j % sg.qn_h;
    j /= sg.qn_h;
    const int64_t img = std::min<int64_t>(j / sg.nphase, nimg - 1);
    const int64_t qt = std::max<int64_t>(1, (ho + sg.out_step_h - 1) / sg.out_step_h);
    const int64_t qh = std::min<int64_t>(sg.q0_h + a_h, qt - 1);
    const int64_t pos = img * qt + qh;  // in [0, nimg * qt)
    const int64_t row = pos * a / ((int64_t)nimg * qt);
    const int64_t col = (int64_t)(w.n0 / bn) * b / ntiles_n;
    Key k;
    k.cell = row * b + col;
    k.pos = pos;
    k.w = w;
    keys.push_back(k);
  }
  std::stable_sort(keys.begin(), keys.end(), [](const Key& x, const Key& y) {
    if (x.cell != y.cell) return x.cell < y.cell;
    if (x.pos != y.pos) return x.pos < y.pos;
    if (x.w.seg != y.w.seg) return x.w.seg < y.w.seg;
    if (x.w.m0 != y.w.m0) return x.w.m0 < y.w.m0;
    if (x.w.n0 != y.w.n0) return x.w.n0 < y.w.n0;
    return x.w.ks < y.w.ks;
  });
  for (size_t i = 0; i < works.size(); ++i) works[i] = keys[i].w;
}

// Works that are all resident at once (at most 32 x wg_per_cu per XCD).  The
// y-th workgroup of an XCD's run then lands on compute unit y mod 32 of that
// XCD (measured: workgroups y and y + 32 of a run share a unit), and
// co-resident workgroups share the unit's MFMA, LDS and load pipes, so a unit
// finishes after about the sum of its works' stages.  Inside each XCD's run
// (the contiguous chunk of the list that xcd_remap gives it), the works are
// dealt longest first to the least loaded unit with a free slot, and placed
// so that unit k's works sit at run positions k, k + 32, ...  Works beyond
// the resident slots (a few, from ragged segments) go last, shortest first:
// they start on the units that free first.  Only the placement inside a run
// changes, so an XCD keeps its share of the input and weights.
void order_works_resident(std::vector<WorkDev>& works, int cblocks, int ksplit, int wg_per_cu) {
  const int g = (int)works.size();
  if (g < 16) return;
  const int g8 = (g + 7) / 8, r = g % 8;
  constexpr int kUnits = kComputeUnits / 8;
  if (g8 > kUnits * wg_per_cu + kUnits) return;  // several rounds: the dispatcher balances
  auto cost = [&](const WorkDev& w) {
    const int cb = (w.ks + 1) * cblocks / ksplit - w.ks * cblocks / ksplit;
    return (int64_t)w.tap_count * cb + 2;
  };
  std::vector<WorkDev> out(works.size());
  for (int x = 0; x < 8; ++x) {
    const int start = (r == 0 || x < r) ? x * g8 : r * g8 + (x - r) * (g8 - 1);
    const int len = (r == 0 || x < r) ? g8 : g8 - 1;
    std::vector<int> idx(len);
    for (int i = 0; i < len; ++i) idx[i] = start + i;
    std::stable_sort(idx.begin(), idx.end(),
                     [&](int a, int b) { return cost(works[a]) > cost(works[b]); });
    const int resident = std::min(len, kUnits * wg_per_cu);
    const int units = std::min(len, kUnits);
    std::vector<int64_t> load(units, 0);
    std::vector<std::vector<int>> held(units);
    for (int i = 0; i < resident; ++i) {
      int best = -1;
      for (int u = 0; u < units; ++u)
        if ((int)held[u].size() < wg_per_cu && (best < 0 || load[u] < load[best])) best = u;
      held[best].push_back(idx[i]);
      load[best] += cost(works[idx[i]]);
    }
    // units holding more works first, so that every level is a prefix
    std::stable_sort(held.begin(), held.end(), [](const std::vector<int>& a,
                                                  const std::vector<int>& b) {
      return a.size() > b.size();
    });
    int pos = start;
    for (int level = 0; level < wg_per_cu; ++level)
      for (int u = 0; u < units; ++u)
        if ((int)held[u].size() > level) out[pos++] = works[held[u][level]];
    for (int i = len - 1; i >= resident; --i) out[pos++] = works[idx[i]];
  }
  works.swap(out);
}

// Schedule model: the dispatcher hands the works, in list order, to the first
// free workgroup slot (kComputeUnits x wg_per_cu slots); a work costs its K
// stages plus about two stages of prologue and epilogue.  Returns the model's
// makespan in stages.  A work count just above the slot count doubles the
// makespan, which a finer split into border classes can cause.
int64_t makespan_of(const std::vector<int64_t>& costs, int cfg) {
  const int64_t slots = (int64_t)kComputeUnits * kTiles[cfg].wg_per_cu;
  std::priority_queue<int64_t, std::vector<int64_t>, std::greater<int64_t>> free_at;
  int64_t used = 0, end = 0;
  for (int64_t cost : costs) {
    int64_t t = 0;
    if (used < slots) {
      ++used;
    } else {
      t = free_at.top();
      free_at.pop();
    }
    free_at.push(t + cost);
    end = std::max(end, t + cost);
  }
  return end;
}

int64_t cblocks_of(const huge2_conv_desc& d, int cfg) {
  const int64_t kc = tile_kb(cfg) / elem_size(d.dtype);
  return (d.c_in + kc - 1) / kc;
}

int64_t makespan_stages(const huge2_conv_desc& d, const PlanShape& shape, int cfg) {
  const int bm = tile_bm(cfg), bn = tile_bn(cfg);
  const int64_t cblocks = cblocks_of(d, cfg);
  const int64_t ntn = (d.c_out + bn - 1) / bn;
  std::vector<int64_t> costs;
  for (const huge2_segment& s : shape.segs) {
    const int64_t m = (int64_t)d.n * s.nphase_h * s.nphase_w * s.qn_h * s.qn_w;
    const int64_t works = (m + bm - 1) / bm * ntn;
    costs.insert(costs.end(), works, (int64_t)s.tap_count * cblocks + 2);
  }
  return makespan_of(costs, cfg);
}

// The same model for the listed form: per image, its tiles in list order.
int64_t makespan_listed(const huge2_conv_desc& d, const ListedShape& ls, int cfg) {
  const int bn = tile_bn(cfg);
  const int64_t cblocks = cblocks_of(d, cfg);
  const int64_t ntn = (d.c_out + bn - 1) / bn;
  std::vector<int64_t> costs;
  for (int img = 0; img < d.n; ++img)
    for (const auto& taps : ls.tile_taps)
      costs.insert(costs.end(), ntn, (int64_t)taps.size() * cblocks + 2);
  return makespan_of(costs, cfg);
}

int floor_div_i(int a, int b) { return a >= 0 ? a / b : -((-a + b - 1) / b); }
int ceil_div_i(int a, int b) { return -floor_div_i(-a, b); }

// The all-taps form (ztile_kernel) applies to bf16 transposed convs whose
// taps x output channels fit one 64-column MFMA tile, NCHW with an even input
// width or NHWC with a multiple of 8 input channels, strides up to 4, at
// most 4 taps of an axis reaching one output phase and output rows of at most
// 256 columns.
// The block of output rows per workgroup is the largest multiple of the
// stride whose input tile fits the LDS budget while the grid still has two
// workgroups per CU (else one); small problems take the largest block that
// fits.
// Returns false when the form does not apply (or HUGE2_ZTILE=0, or a GEMM
// tile is forced through HUGE2_TILE).
bool ztile_shape(const huge2_conv_desc& d, bool transposed, ZArgs* z, int64_t* issued) {
  // bf16 only: in fp32 the phase GEMM measured faster.  NHWC reads each
  // pixel's channels as 16-byte groups (c_in a multiple of 8)
  if (!transposed || d.dtype != HUGE2_BF16) return false;
  const bool nhwc = d.layout == HUGE2_NHWC;
  if (nhwc ? d.c_in % 8 != 0 : d.w % 2 != 0) return false;
  if (env_int("HUGE2_ZTILE", 1) == 0 || env_int("HUGE2_TILE", -1) >= 0) return false;
  if ((long long)d.c_out * d.r * d.s > 64) return false;
  if (d.stride_h > kZtileMaxStride || d.stride_w > kZtileMaxStride || d.r > kZtileMaxTaps ||
      d.s > kZtileMaxTaps || d.dil_h > 16 || d.dil_w > 16)
    return false;
  int ho, wo;
  if (!output_dims(d, true, &ho, &wo)) return false;
  const long long x_bytes = (long long)d.n * d.c_in * d.h * d.w * 2;
  if (x_bytes >= (1ll << 31) || wo > 256) return false;
  // tile columns: every input column an output reads, and every input column
  const int j_lo = std::min(0, ceil_div_i(d.pad_w - (d.s - 1) * d.dil_w, d.stride_w));
  const int j_hi = std::max(d.w - 1, floor_div_i(wo - 1 + d.pad_w, d.stride_w));
  const int tcw = j_hi - j_lo + 1;
  const int cin_pad = round_up(d.c_in, 64);
  const int i_off = ceil_div_i(d.pad_h - (d.r - 1) * d.dil_h, d.stride_h);
  // output rows per workgroup: the tile (and its Z) must fit, and the input
  // items of a pass must fit the threads; prefer two workgroups per compute
  // unit, then one
  int best2 = -1, best1 = -1, fallback = -1;
  for (int q = (ho + d.stride_h - 1) / d.stride_h; q >= 1; --q) {
    const int ob = std::min(q * d.stride_h, ho);
    const int tr = floor_div_i(ob - 1 + d.pad_h, d.stride_h) - i_off + 1;
    const long long np = (long long)tr * tcw;
    if (np > kZtileMaxPixels) continue;
    if ((long long)std::min(tr, d.h) * d.w * 4 > (long long)kZtileMaxItems * kZtileThreads) continue;
    const long long blocks = (long long)d.n * ((ho + ob - 1) / ob);
    if (fallback < 0) fallback = ob;
    if (best1 < 0 && blocks >= kComputeUnits) best1 = ob;
    if (best2 < 0 && blocks >= 2 * kComputeUnits) best2 = ob;
  }
  // two workgroups share a compute unit only if their LDS fits twice
  const bool two_per_cu = 2 * kZtileLds <= 160 * 1024;
  const int ob = (two_per_cu && best2 >= 0) ? best2 : best1 >= 0 ? best1 : fallback;
  if (ob < 0) return false;
  std::memset(z, 0, sizeof(*z));
  z->x_bytes = (uint32_t)x_bytes;
  z->n = d.n;
  z->cin = d.c_in;
  z->h = d.h;
  z->w = d.w;
  z->cout = d.c_out;
  z->r = d.r;
  z->s = d.s;
  z->cin_pad = cin_pad;
  z->cout_pad = d.c_out;
  z->stride_h = d.stride_h;
  z->stride_w = d.stride_w;
  z->pad_h = d.pad_h;
  z->pad_w = d.pad_w;
  z->dil_h = d.dil_h;
  z->dil_w = d.dil_w;
  z->ho = ho;
  z->wo = wo;
  z->ob = ob;
  z->tr = floor_div_i(ob - 1 + d.pad_h, d.stride_h) - i_off + 1;
  z->tcw = tcw;
  z->j_lo = j_lo;
  z->cchunk = 64;
  z->nhwc = nhwc ? 1 : 0;
  // per-phase tap tables: output o with o + pad = stride*Q + rho reads input
  // Q + delta through kernel tap k when rho - k*dil = stride*delta
  const int strides[2] = {d.stride_h, d.stride_w}, ks[2] = {d.r, d.s}, dils[2] = {d.dil_h, d.dil_w};
  for (int ax = 0; ax < 2; ++ax)
    for (int rho = 0; rho < strides[ax]; ++rho) {
      int cnt = 0;
      for (int k = 0; k < ks[ax]; ++k) {
        const int num = rho - k * dils[ax];
        if (((num % strides[ax]) + strides[ax]) % strides[ax] != 0) continue;
        if (cnt == kZtilePhaseTaps) return false;
        z->tap_k[ax][rho][cnt] = (int8_t)k;
        z->tap_d[ax][rho][cnt] = (int8_t)(num / strides[ax]);
        ++cnt;
      }
      z->tap_n[ax][rho] = (int8_t)cnt;
      int& mx = ax == 0 ? z->max_th : z->max_tw;
      mx = std::max(mx, cnt);
    }
  const int64_t np = (int64_t)z->tr * tcw;
  *issued = (int64_t)d.n * ((ho + ob - 1) / ob) * ((np + 31) / 32 * 32) * 64 * z->cin_pad;
  return true;
}

// The output-stationary form (rowphase_kernel) applies to NCHW bf16
// transposed convs with strides of at least 4, dilation 1, at most 32 input
// and output channels, kernel extents at most twice the stride, input rows
// of at most 64 and output rows a multiple of 8 elements (at most 2048).  Returns false
// otherwise (or with HUGE2_ROWPHASE=0, or a GEMM tile forced).
bool rowphase_shape(const huge2_conv_desc& d, bool transposed, RpArgs* z, int64_t* issued) {
  if (!transposed || d.layout != HUGE2_NCHW || d.dtype != HUGE2_BF16) return false;
  if (env_int("HUGE2_ROWPHASE", 1) == 0 || env_int("HUGE2_TILE", -1) >= 0) return false;
  if (d.stride_h < 4 || d.stride_w < 4 || d.dil_h != 1 || d.dil_w != 1) return false;
  if (d.stride_w > (kRpThreads / 64) * kRpMaxColPhasesPerWave) return false;
  if (d.c_in > kRpCh || d.c_out > kRpCh || d.r > 2 * d.stride_h || d.s > 2 * d.stride_w)
    return false;
  if (d.w > kRpMaxW) return false;
  int ho, wo;
  if (!output_dims(d, true, &ho, &wo) || wo % 8 != 0 || wo > 64 * 4 * 8) return false;
  if ((long long)kRpMaxRb * (d.w + 2) >= 4096) return false;  // pixel index range of a phase
  // input columns read: Q_w - t for t < 2 must stay within [-1, w]
  int max_rows = 0;
  for (int rho = 0; rho < d.stride_w; ++rho) {
    const int qhi = floor_div_i(wo - 1 + d.pad_w - rho, d.stride_w);
    if (qhi > d.w) return false;
  }
  for (int rho = 0; rho < d.stride_h; ++rho) {
    const int qlo = ceil_div_i(d.pad_h - rho, d.stride_h);
    const int qhi = floor_div_i(ho - 1 + d.pad_h - rho, d.stride_h);
    max_rows = std::max(max_rows, qhi - qlo + 1);
  }
  if (max_rows <= 0) return false;
  // LDS rows are column-phase major: stride_w phases x nq slots per row
  int nq = d.w + 1;
  while ((d.stride_w * nq) % 8 != 0) ++nq;
  const long long row_elems = (long long)d.stride_w * nq;
  int rb = std::min(kRpMaxRb, max_rows);
  while (rb > 1 && d.c_out * (rb * row_elems + 2) > kRpOutElems) --rb;
  if (d.c_out * (rb * row_elems + 2) > kRpOutElems) return false;
  std::memset(z, 0, sizeof(*z));
  z->n = d.n;
  z->cin = d.c_in;
  z->h = d.h;
  z->w = d.w;
  z->cout = d.c_out;
  z->r = d.r;
  z->s = d.s;
  z->stride_h = d.stride_h;
  z->stride_w = d.stride_w;
  z->pad_h = d.pad_h;
  z->pad_w = d.pad_w;
  z->ho = ho;
  z->wo = wo;
  z->rb = rb;
  z->qblocks = (max_rows + rb - 1) / rb;
  z->nq = nq;
  // issued multiply-adds: per workgroup and column phase, 32-pixel blocks x
  // 32 channels x (taps x 32 input channels)
  int64_t iss = 0;
  for (int rh = 0; rh < d.stride_h; ++rh) {
    const int tnh = rh < d.r ? std::min(2, (d.r - 1 - rh) / d.stride_h + 1) : 0;
    const int rows = floor_div_i(ho - 1 + d.pad_h - rh, d.stride_h) - ceil_div_i(d.pad_h - rh, d.stride_h) + 1;
    for (int rw = 0; rw < d.stride_w; ++rw) {
      const int tnw = rw < d.s ? std::min(2, (d.s - 1 - rw) / d.stride_w + 1) : 0;
      const int nqw = floor_div_i(wo - 1 + d.pad_w - rw, d.stride_w) - ceil_div_i(d.pad_w - rw, d.stride_w) + 1;
      for (int q0 = 0; q0 < rows; q0 += rb) {
        const int64_t npix = (int64_t)std::min(rb, rows - q0) * std::max(nqw, 0);
        iss += (npix + 31) / 32 * 32 * 32 * (int64_t)tnh * tnw * 32;
      }
    }
  }
  *issued = iss * d.n;
  return true;
}

// The column-phase form (colphase_kernel) applies to NCHW bf16 transposed
// convs with column stride 32, dilation 1, at most 32 input channels, kernel
// width at most 64 and height at most twice the row stride, output padding
// and width multiples of 8 (16-byte output pieces), every output row and
// column reaching back into the input or its one-pixel border, and the
// staged input within 64 KiB of LDS.  Returns false otherwise (or with
// HUGE2_COLPHASE=0, or a GEMM tile forced).
bool colphase_shape(const huge2_conv_desc& d, bool transposed, CpArgs* z, int64_t* issued) {
  if (!transposed || d.layout != HUGE2_NCHW || d.dtype != HUGE2_BF16) return false;
  if (env_int("HUGE2_COLPHASE", 1) == 0 || env_int("HUGE2_TILE", -1) >= 0) return false;
  if (d.stride_w != 32 || d.dil_h != 1 || d.dil_w != 1 || d.c_in > 32 || d.s > 64 ||
      d.r > 2 * d.stride_h || d.pad_w % 8 != 0)
    return false;
  int ho, wo;
  if (!output_dims(d, true, &ho, &wo) || wo % 8 != 0) return false;
  const int cp = round_up(d.c_in, 8);
  if (((long long)(d.h + 2) * (d.w + 2) * cp + (long long)kCpWaves * kCpRows * round_up(wo, 32)) *
          2 > kCpMaxLds)
    return false;
  const int qw_lo = ceil_div_i(d.pad_w - 31, 32), qw_hi = floor_div_i(wo - 1 + d.pad_w, 32);
  if (qw_lo < 0 || qw_hi > d.w || qw_hi < qw_lo) return false;
  // issued: the kernel's column tiles, kCpRows rows of a row phase at a time
  int64_t cols = 0;
  for (int rho = 0; rho < d.stride_h; ++rho) {
    const int q_lo = ceil_div_i(d.pad_h - rho, d.stride_h);
    const int q_hi = floor_div_i(ho - 1 + d.pad_h - rho, d.stride_h);
    if (q_hi < q_lo) continue;
    if (q_lo < 0 || q_hi > d.h) return false;
    for (int q0 = 0; q0 < q_hi - q_lo + 1; q0 += kCpRows) {
      const int nr = std::min(kCpRows, q_hi - q_lo + 1 - q0);
      cols += ((int64_t)nr * (qw_hi - qw_lo + 1) + 31) / 32 * 32;
    }
  }
  std::memset(z, 0, sizeof(*z));
  z->n = d.n;
  z->cin = d.c_in;
  z->h = d.h;
  z->w = d.w;
  z->cout = d.c_out;
  z->r = d.r;
  z->s = d.s;
  z->stride_h = d.stride_h;
  z->pad_h = d.pad_h;
  z->pad_w = d.pad_w;
  z->ho = ho;
  z->wo = wo;
  z->cp = cp;
  z->qw_lo = qw_lo;
  z->nqw = qw_hi - qw_lo + 1;
  const uint32_t dv[6] = {(uint32_t)(d.w + 2), (uint32_t)(d.h + 2), (uint32_t)z->nqw,
                          (uint32_t)(cp / 8), (uint32_t)d.c_in, (uint32_t)std::max(1, d.w / 8)};
  for (int k = 0; k < 6; ++k) division_magic(dv[k], &z->dv_mul[k], &z->dv_shift[k]);
  // per (image, output channel) and row phase: 32 column phases x the
  // padded columns x K = 4 taps x cp
  *issued = (int64_t)d.n * d.c_out * cols * 32 * 4 * cp;
  return true;
}

// The all-phase form (quad_kernel) applies to bf16 transposed convs, NCHW
// or NHWC (then with output channels a multiple of 8), with stride 2, a 4x4
// kernel, padding 1, dilation 1 and no output padding
// (so every phase has 2x2 taps at input offsets in [-1, 1] and the input's
// pixel grid), input channels a multiple of 64, and a width of at least 4
// that tiles P = 64 (or 128) positions per workgroup: whole images of
// h*w <= P pixels (h*w dividing P, a multiple of 8), or P/w full rows (w
// dividing P, h a multiple of P/w).  Returns false otherwise (or with
// HUGE2_QUAD=0, or a GEMM tile forced).
//
// 128 positions per workgroup (np = 4) halve the weight bytes per
// multiply-add; they are taken when they still give every compute unit a
// workgroup of 64 channels (DCGAN L3: 32.5 -> 29.4 us).
bool quad_shape(const huge2_conv_desc& d, bool transposed, QArgs* q, int64_t* issued) {
  if (!transposed || d.dtype != HUGE2_BF16) return false;
  const bool nhwc = d.layout == HUGE2_NHWC;
  if (nhwc && (d.c_out % 8 != 0 || env_int("HUGE2_QUAD_NHWC", 1) == 0)) return false;
  if (env_int("HUGE2_QUAD", 1) == 0 || env_int("HUGE2_TILE", -1) >= 0) return false;
  if (d.stride_h != 2 || d.stride_w != 2 || d.r != 4 || d.s != 4 || d.pad_h != 1 ||
      d.pad_w != 1 || d.dil_h != 1 || d.dil_w != 1 || d.out_pad_h != 0 || d.out_pad_w != 0)
    return false;
  if (d.c_in % 64 != 0 || d.w < 4) return false;
  const long long hw = (long long)d.h * d.w;
  const bool keven = (d.c_in / 64) % 2 == 0;
  // images and rows per workgroup for pix positions; false if the shape
  // does not tile or the halo tile or the input items per thread overflow
  auto tiling = [&](int pix, int ks, int* ni, int* qbh) {
    if (hw <= pix) {
      if (pix % hw != 0 || hw % 8 != 0) return false;
      *ni = (int)(pix / hw);
      *qbh = d.h;
    } else {
      if (d.w > pix || pix % d.w != 0) return false;
      *ni = 1;
      *qbh = pix / d.w;
      if (d.h % *qbh != 0) return false;
    }
    if (*ni * (*qbh + 2) * (d.w + 2) > kQuadHaloRows) return false;
    // loaded rows per block: at most min(h, qbh + 2)
    const long long items = (long long)*ni * std::min(d.h, *qbh + 2) * d.w / 2 * 8;
    return items <= (long long)kQuadMaxPieces * (kQuadThreads / ks);
  };
  auto wgs_for = [&](int ni, int qbh, int nch) {
    return (long long)((d.n + ni - 1) / ni) * (d.h / qbh) * ((d.c_out + 32 * nch - 1) / (32 * nch));
  };
  int ni = 0, qbh = 0, np = 0, nch = 2, ks = 1;
  const int np_env = env_int("HUGE2_QUAD_NP", 0);  // 0: by shape; 2 or 4: forced
  const int ks_env = env_int("HUGE2_QUAD_KS", 0);  // 128 positions: K groups forced
  if (np_env != 2) {
    // 128 positions: 64-channel tiles (two waves of 32 channels per phase)
    // if every compute unit gets one.  32-channel tiles in two K groups are
    // taken only when forced (measured slower than 64 positions on DCGAN L2)
    for (int cand = 0; cand < 2 && np == 0; ++cand) {
      const int cks = cand == 0 ? 1 : 2, cnch = cand == 0 ? 2 : 1;
      if ((cks == 2 && (!keven || np_env != 4)) || (ks_env != 0 && ks_env != cks)) continue;
      if (!tiling(128, cks, &ni, &qbh)) continue;
      if (np_env != 4 && wgs_for(ni, qbh, cnch) < kComputeUnits) continue;
      np = 4;
      nch = cnch;
      ks = cks;
    }
    if (np == 0 && np_env == 4) return false;
  }
  if (np == 0) {
    // 64 positions.  64-channel tiles: two waves of 32 channels per phase,
    // or (HUGE2_QUAD_WCH=2, an even number of 64-channel K blocks) two K
    // groups of one wave of 64 channels per phase; 32-channel tiles in two K
    // groups when 64-channel tiles would leave compute units idle
    np = 2;
    if (!tiling(64, 1, &ni, &qbh)) return false;
    if (wgs_for(ni, qbh, 2) < kComputeUnits && keven) {
      nch = 1;
      ks = 2;
    } else if (keven && env_int("HUGE2_QUAD_WCH", 1) == 2) {
      ks = 2;
    }
    if (!tiling(64, ks, &ni, &qbh)) return false;
  }
  const int igroups = (d.n + ni - 1) / ni, hblocks = d.h / qbh;
  const long long x_bytes = (long long)d.n * d.c_in * hw * 2;
  if (x_bytes >= (1ll << 31)) return false;
  std::memset(q, 0, sizeof(*q));
  q->x_bytes = (uint32_t)x_bytes;
  q->nhwc = nhwc ? 1 : 0;
  q->n = d.n;
  q->cin = d.c_in;
  q->h = d.h;
  q->w = d.w;
  q->cout = d.c_out;
  q->cout_pad = round_up(d.c_out, 32 * nch);
  q->ni = ni;
  q->qbh = qbh;
  q->np = np;
  q->nch = nch;
  q->ks = ks;
  q->igroups = igroups;
  q->hblocks = hblocks;
  q->ntiles = q->cout_pad / (32 * nch);
  const long long wgs = (long long)q->ntiles * igroups * hblocks;
  // Few workgroups over a long K: each runs its K blocks one after another,
  // where the phase GEMM splits K across workgroups.  Measured on the batch-1
  // DCGAN L1 (16 workgroups, 8 K blocks per group): 19.8 us here, 14.7 us on
  // the phase GEMM with an 8-way K split; with 4 K blocks per group (batch-1
  // L2) this kernel is still the faster (12.8 against 14.5 us).
  if (wgs < kComputeUnits / 4 && d.c_in / (64 * ks) >= 8) return false;
  q->depth = env_int("HUGE2_QUAD_DEPTH", 2);
  // (eight stages spill the registers: measured 4x slower)
  if ((q->depth != 2 && q->depth != 4) || (nch == 2 && ks == 2) ||
      np == 4)
    q->depth = 2;
  const long long wp_bytes = 16ll * q->cout_pad * d.c_in * 2;
  if (wp_bytes >= (1ll << 31)) return false;
  q->wp_bytes = (uint32_t)wp_bytes;
  // output o = 2 q + rho takes kernel tap k with (rho + pad - k) even, reading
  // input q + (rho + pad - k) / 2
  for (int rh = 0; rh < 2; ++rh)
    for (int rw = 0; rw < 2; ++rw)
      for (int th = 0; th < 2; ++th)
        for (int tw = 0; tw < 2; ++tw) {
          const int kh = (rh + d.pad_h) % 2 + 2 * th, kw = (rw + d.pad_w) % 2 + 2 * tw;
          q->slot[2 * rh + rw][2 * th + tw] = (int8_t)(kh * 4 + kw);
          q->dh[2 * rh + rw][2 * th + tw] = (int8_t)((rh + d.pad_h - kh) / 2);
          q->dw[2 * rh + rw][2 * th + tw] = (int8_t)((rw + d.pad_w - kw) / 2);
        }
  // issued multiply-adds: per workgroup 4 phases x 32*np positions x 32*nch
  // channels x 4 taps x c_in
  *issued = wgs * 4 * (32 * np) * 32 * nch * 4 * (long long)d.c_in;
  return true;
}

// Whether a segment's taps are the product of two arithmetic progressions
// (the order build_shape emits: h outer, w inner), verified tap by tap; fills
// the progression fields of sd when they are.
bool tap_progressions(const huge2_tap* tl, int count, SegDev* sd) {
  if (count <= 0) return false;
  int ntw = 1;
  while (ntw < count && tl[ntw].kh == tl[0].kh) ++ntw;
  if (count % ntw != 0) return false;
  const int nth = count / ntw;
  sd->ntw = ntw;
  sd->off0_h = tl[0].off_h;
  sd->off0_w = tl[0].off_w;
  sd->kh0 = tl[0].kh;
  sd->kw0 = tl[0].kw;
  sd->doff_h = nth > 1 ? tl[ntw].off_h - tl[0].off_h : 0;
  sd->dkh = nth > 1 ? tl[ntw].kh - tl[0].kh : 0;
  sd->doff_w = ntw > 1 ? tl[1].off_w - tl[0].off_w : 0;
  sd->dkw = ntw > 1 ? tl[1].kw - tl[0].kw : 0;
  for (int t = 0; t < count; ++t) {
    const int th = t / ntw, tw = t % ntw;
    if (tl[t].kh != sd->kh0 + th * sd->dkh || tl[t].kw != sd->kw0 + tw * sd->dkw ||
        tl[t].off_h != sd->off0_h + th * sd->doff_h || tl[t].off_w != sd->off0_w + tw * sd->doff_w)
      return false;
  }
  return true;
}

// The same check for a work's own tap list, into the work's progression
// fields (ap_ntw = 0 when the taps are no such product).
void work_progressions(const TapDev* tl, int count, int s_width, WorkDev* w) {
  w->ap_ntw = 0;
  if (count <= 0) return;
  std::vector<huge2_tap> t(count);
  for (int i = 0; i < count; ++i) {
    t[i].kh = tl[i].slot / s_width;
    t[i].kw = tl[i].slot % s_width;
    t[i].off_h = tl[i].off_h;
    t[i].off_w = tl[i].off_w;
  }
  SegDev sd;
  std::memset(&sd, 0, sizeof(sd));
  if (!tap_progressions(t.data(), count, &sd)) return;
  w->ap_ntw = sd.ntw;
  w->ap_kh0 = sd.kh0;
  w->ap_dkh = sd.dkh;
  w->ap_kw0 = sd.kw0;
  w->ap_dkw = sd.dkw;
  w->ap_off0_h = sd.off0_h;
  w->ap_doff_h = sd.doff_h;
  w->ap_off0_w = sd.off0_w;
  w->ap_doff_w = sd.doff_w;
}

// Border-class splitting of a plan: HUGE2_CLASS_SPLIT (0, 1, 2) forces it;
// otherwise 0 (one segment per phase group, out-of-range taps read zeros) or
// 2 (per group, the form that issues fewer tile-taps), whichever the schedule
// model finishes first (ties: 2).  When the works of form 0 are all resident
// at once and the split's ragged segments add works beyond the resident
// slots, form 0 wins: such a straggler starts only when a unit frees and
// adds its whole latency (measured on the odd-kernel layer, 512 against 514
// works: 21.3 against 25.1 us).
int choose_split(const huge2_conv_desc& d, bool transposed, int cfg) {
  const int forced = env_int("HUGE2_CLASS_SPLIT", -1);
  if (forced >= 0 && forced <= 2) return forced;
  PlanShape s0, s2;
  if (!build_shape(d, transposed, 0, tile_bm(cfg), &s0) ||
      !build_shape(d, transposed, 2, tile_bm(cfg), &s2))
    return 2;
  const long long slots = (long long)kComputeUnits * kTiles[cfg].wg_per_cu;
  const long long w0 = count_works(d, transposed, 0, cfg), w2 = count_works(d, transposed, 2, cfg);
  if (w0 <= slots && w2 > slots) return 0;
  return makespan_stages(d, s0, cfg) < makespan_stages(d, s2, cfg) ? 0 : 2;
}

// Tile configuration, border-class form and decomposition of a GEMM plan
// (shared by plan creation and the MAC report).  A stride-1 dilated conv
// takes the listed form (*listed true, ls filled) when the schedule model
// finishes it no later than the segment form (HUGE2_LISTED=0/1 forces the
// choice).  Returns -1 if the shape cannot be built.
int plan_gemm_shape(const huge2_conv_desc& d, bool tr, PlanShape* shape, bool* listed,
                    ListedShape* ls) {
  const int cfg = choose_cfg(d, tr, 2);
  const int split = choose_split(d, tr, cfg);
  if (!build_shape(d, tr, split, tile_bm(cfg), shape)) return -1;
  *listed = false;
  const int force = env_int("HUGE2_LISTED", -1);
  if (!tr && force != 0 && build_listed(d, tile_bm(cfg), ls))
    *listed = force == 1 || makespan_listed(d, *ls, cfg) <= makespan_stages(d, *shape, cfg);
  return cfg;
}


void free_buffers(huge2_plan* p) {
  void* bufs[5] = {p->wp, p->meta, p->xs, p->part, p->zbuf};
  for (void* b : bufs) {
    if (!b) continue;
    if (p->mem.arena)
      continue;  // a region the plan does not own
    if (p->mem.stream_ordered)
      (void)hipFreeAsync(b, p->alloc_stream);
    else
      (void)hipFree(b);
  }
  p->wp = p->meta = p->xs = p->part = p->zbuf = nullptr;
  if (p->inner) {
    free_buffers(p->inner);
    delete p->inner;
    p->inner = nullptr;
  }
}

huge2_status dev_alloc(huge2_plan* p, void** out, size_t bytes) {
  *out = nullptr;
  if (bytes == 0) return HUGE2_OK;
  if (p->mem.arena) {
    Arena& a = *p->mem.arena;
    const size_t at = (a.used + 255) / 256 * 256;
    if (at > a.cap || bytes > a.cap - at) return HUGE2_ERR_UNSUPPORTED;
    *out = a.base + at;
    a.used = at + bytes;
    return HUGE2_OK;
  }
  if (fault("alloc")) return HUGE2_ERR_ALLOC;
  hipError_t e = p->mem.stream_ordered ? hipMallocAsync(out, bytes, p->alloc_stream)
                                   : hipMalloc(out, bytes);
  if (e != hipSuccess) {
    *out = nullptr;
    (void)hipGetLastError();
    return HUGE2_ERR_ALLOC;
  }
  return HUGE2_OK;
}

// Plan of the all-taps form (zp), the output-stationary form (rp) or the
// all-phase form (qp): packed weights only (K-contiguous, or in the lane order
// of 128-byte K stages for qp); the three kernels read the NCHW input
// directly, so nothing is staged.
huge2_status create_direct(huge2_plan** out, const huge2_conv_desc& d, int transposed,
                          const void* w, hipStream_t stream, Mem mem, const ZArgs* zp,
                          const RpArgs* rp, const QArgs* qp, int64_t issued,
                          const CpArgs* cpa = nullptr) {
  PlanShape shape;
  if (!build_shape(d, true, 2, 128, &shape)) return HUGE2_ERR_INVALID_ARG;
  huge2_plan* p = new (std::nothrow) huge2_plan();
  if (!p) return HUGE2_ERR_ALLOC;
  const int esz = elem_size(d.dtype);
  p->desc = d;
  p->transposed = transposed;
  p->bias_div = 1;
  p->ksplit = 1;
  output_dims(d, true, &p->ho, &p->wo);
  p->cfg = -1;
  p->staged = false;
  p->c_stride = d.c_in;
  p->cin_pad = zp ? zp->cin_pad : qp ? d.c_in : kRpCh;
  p->cout_pad = zp ? zp->cout_pad : qp ? qp->cout_pad : kRpCh;
  p->x_bytes = (size_t)d.n * d.c_in * d.h * d.w * esz;
  p->wp_bytes = (size_t)d.r * d.s * p->cout_pad * p->cin_pad * esz;
  if (cpa) {
    p->cin_pad = cpa->cp;
    p->cout_pad = d.c_out;
    p->wp_bytes = (size_t)d.c_out * d.stride_h * (cpa->cp / 4) * 64 * 8 * esz;
  }
  p->mem = mem;
  p->alloc_stream = stream;
  p->nonzero_macs = shape.nonzero_macs;
  p->issued_macs = issued;
  if (cpa) {
    p->colphase = true;
    p->cpargs = *cpa;
    std::snprintf(p->kernel_name, sizeof(p->kernel_name), "colphase_kernel cp%d", cpa->cp);
  } else if (zp) {
    p->ztile = true;
    p->zargs = *zp;
    std::snprintf(p->kernel_name, sizeof(p->kernel_name), "ztile_kernel ob%d", zp->ob);
  } else if (rp) {
    p->rowphase = true;
    p->rpargs = *rp;
    std::snprintf(p->kernel_name, sizeof(p->kernel_name), "rowphase_kernel rb%d", rp->rb);
  } else {
    p->quad = true;
    p->qargs = *qp;
    std::snprintf(p->kernel_name, sizeof(p->kernel_name), "quad_kernel %dx%dx%d c%d k%d d%d",
                  qp->ni, qp->qbh, d.w, 32 * qp->nch, qp->ks, qp->depth);
  }
  huge2_status st = dev_alloc(p, &p->wp, p->wp_bytes);
  if (st != HUGE2_OK) {
    free_buffers(p);
    delete p;
    return st;
  }
  bool ok = !fault("launch");
  if (ok && cpa)
    ok = launch_pack_colphase(w, p->wp, d.c_in, d.c_out, d.r, d.s, d.stride_h, cpa->cp, stream) ==
         hipSuccess;
  else if (ok)
    ok = launch_pack_weights(w, p->wp, d.dtype, true, d.c_in, d.c_out, d.r, d.s, p->cin_pad,
                             p->cout_pad, qp ? 128 : 0, stream) == hipSuccess;
  if (ok) ok = hipStreamSynchronize(stream) == hipSuccess;
  if (!ok) {
    (void)hipGetLastError();
    free_buffers(p);
    delete p;
    return HUGE2_ERR_HIP;
  }
  *out = p;
  return HUGE2_OK;
}

// A transposed conv of a 1x1 input with no padding and unit dilation is the
// plain product y[n][k][m][q] = sum_c x[n][c] w[c][k][m][q] (section 3.1
// with a single input pixel: every tap its own phase and output pixel): one
// dense GEMM of n rows, run as a 1x1 conv to c_out*r*s channels on the same
// memory.  NCHW: y is [n][c_out*r*s] with column k*r*s + m*s + q, w read
// as it lies ([c_in][c_out*r*s]), bias k over r*s consecutive columns.  NHWC:
// y is [n][r*s*c_out] with column (m*s + q)*c_out + k, the weights packed
// tap-major, bias k repeating every c_out columns.  Writes the descriptor
// the plan runs to *dd and the GEMM's bias mapping and packing to the
// outputs (1, 0, 0 when the form does not apply).
void product_form(const huge2_conv_desc& d, bool transposed, huge2_conv_desc* dd, int* bias_div,
                  int* bias_mod, int* prod_rs) {
  *dd = d;
  *bias_div = 1;
  *bias_mod = 0;
  *prod_rs = 0;
  if (!transposed || d.h != 1 || d.w != 1 || d.pad_h != 0 || d.pad_w != 0 ||
      d.out_pad_h != 0 || d.out_pad_w != 0 || d.dil_h != 1 || d.dil_w != 1 ||
      (d.r == 1 && d.s == 1) || (long long)d.c_out * d.r * d.s > INT32_MAX / 2)
    return;
  if (d.layout == HUGE2_NHWC && env_int("HUGE2_PRODUCT_NHWC", 1) == 0) return;
  dd->c_out = d.c_out * d.r * d.s;
  dd->r = dd->s = 1;
  dd->stride_h = dd->stride_w = 1;
  dd->layout = HUGE2_NHWC;
  if (d.layout == HUGE2_NCHW) {
    *bias_div = d.r * d.s;
  } else {
    *bias_mod = d.c_out;
    *prod_rs = d.r * d.s;
  }
}

// The two-pass all-taps form applies to fp32 NCHW transposed convs whose
// taps x output channels fit one 64-wide tile (the fp32 counterpart of the
// all-taps kernel): pass 1 is the pointwise GEMM of every input pixel with
// all taps, z = x . w read as [c_in][c_out*r*s] (a 1x1 transposed conv, on
// the phase GEMM), pass 2 gathers each output's taps from z.  The phase
// GEMM would pad the few output channels to a 32-wide MFMA tile per phase.
bool two_pass_shape(const huge2_conv_desc& d, bool transposed, huge2_conv_desc* d1) {
  if (!transposed || d.dtype != HUGE2_F32 || d.layout != HUGE2_NCHW) return false;
  if (env_int("HUGE2_TWOPASS", 1) == 0 || env_int("HUGE2_TILE", -1) >= 0) return false;
  if ((long long)d.c_out * d.r * d.s > 64 || (d.r == 1 && d.s == 1)) return false;
  *d1 = d;
  d1->c_out = d.c_out * d.r * d.s;
  d1->r = d1->s = 1;
  d1->stride_h = d1->stride_w = 1;
  d1->pad_h = d1->pad_w = 0;
  d1->out_pad_h = d1->out_pad_w = 0;
  d1->dil_h = d1->dil_w = 1;
  d1->activation = HUGE2_ACT_NONE;
  return (long long)d.n * d1->c_out * d.h * d.w < (1ll << 31);
}

huge2_status create_impl(huge2_plan** out, const huge2_conv_desc* desc, int transposed,
                         const void* w, hipStream_t stream, Mem mem);

// The gather form applies to NCHW convs (dilated or strided) with few input
// channels, c_in*r*s <= 64 and r*s > 1 (a discriminator's RGB input layer,
// the last layer of a generator's backward pass): the phase GEMM would pad
// each tap's few channels to a 64-channel K stage.  Instead each output
// pixel's receptive field (c_in*r*s values, Algorithm 2's gather) is gathered
// into one GEMM row, in the staged layout of a pointwise conv whose weights
// are w read in place as [c_out][c_in*r*s].
bool gather_shape(const huge2_conv_desc& d, bool transposed, huge2_conv_desc* d1) {
  if (transposed || d.layout != HUGE2_NCHW) return false;
  if (env_int("HUGE2_GATHER", 1) == 0 || env_int("HUGE2_TILE", -1) >= 0) return false;
  if ((long long)d.c_in * d.r * d.s > 64 || (d.r == 1 && d.s == 1)) return false;
  int ho, wo;
  if (!output_dims(d, false, &ho, &wo)) return false;
  *d1 = d;
  d1->c_in = d.c_in * d.r * d.s;
  d1->h = ho;
  d1->w = wo;
  d1->r = d1->s = 1;
  d1->stride_h = d1->stride_w = 1;
  d1->pad_h = d1->pad_w = 0;
  d1->dil_h = d1->dil_w = 1;
  return true;
}

huge2_status create_gather(huge2_plan** out, const huge2_conv_desc& d, const huge2_conv_desc& d1,
                           const void* w, hipStream_t stream, Mem mem) {
  huge2_plan* inner = nullptr;
  huge2_status st = create_impl(&inner, &d1, 0, w, stream, mem);
  if (st != HUGE2_OK) return st;
  if (!inner->staged || inner->inner) {  // the pointwise GEMM must read a staged input
    free_buffers(inner);
    delete inner;
    return HUGE2_ERR_UNSUPPORTED;
  }
  huge2_plan* p = new (std::nothrow) huge2_plan();
  if (!p) {
    free_buffers(inner);
    delete inner;
    return HUGE2_ERR_ALLOC;
  }
  p->desc = d;
  p->transposed = 0;
  p->bias_div = 1;
  p->ksplit = 1;
  p->mem = mem;
  p->alloc_stream = stream;
  output_dims(d, false, &p->ho, &p->wo);
  p->inner = inner;
  p->gather = true;
  p->staged = true;
  p->issued_macs = inner->issued_macs;
  PlanShape shape;
  p->nonzero_macs = build_shape(d, false, 2, 128, &shape) ? shape.nonzero_macs : 0;
  std::snprintf(p->kernel_name, sizeof(p->kernel_name), "gather_taps + %.48s", inner->kernel_name);
  *out = p;
  return HUGE2_OK;
}

huge2_status create_two_pass(huge2_plan** out, const huge2_conv_desc& d, const huge2_conv_desc& d1,
                             const void* w, hipStream_t stream, Mem mem) {
  huge2_plan* inner = nullptr;
  huge2_status st = create_impl(&inner, &d1, 1, w, stream, mem);
  if (st != HUGE2_OK) return st;
  huge2_plan* p = new (std::nothrow) huge2_plan();
  if (!p) {
    free_buffers(inner);
    delete inner;
    return HUGE2_ERR_ALLOC;
  }
  p->desc = d;
  p->transposed = 1;
  p->bias_div = 1;
  p->ksplit = 1;
  p->mem = mem;
  p->alloc_stream = stream;
  output_dims(d, true, &p->ho, &p->wo);
  p->inner = inner;
  p->staged = inner->staged;
  p->issued_macs = inner->issued_macs;
  PlanShape shape;
  p->nonzero_macs = build_shape(d, true, 2, 128, &shape) ? shape.nonzero_macs : 0;
  std::snprintf(p->kernel_name, sizeof(p->kernel_name), "two-pass: %.40s + taps_combine",
                inner->kernel_name);
  if ((st = dev_alloc(p, &p->zbuf, (size_t)d.n * d1.c_out * d.h * d.w * sizeof(float))) != HUGE2_OK) {
    free_buffers(p);
    delete p;
    return st;
  }
  *out = p;
  return HUGE2_OK;
}

// A grouped (or depthwise) layer: the weight copied into the plan (the caller
// may free w after plan creation), the direct kernel at execute.
huge2_status create_grouped(huge2_plan** out, const huge2_conv_desc& d, int transposed,
                            const void* w, hipStream_t stream, Mem mem) {
  huge2_plan* p = new (std::nothrow) huge2_plan();
  if (!p) return HUGE2_ERR_ALLOC;
  const bool tr = transposed != 0;
  const int esz = elem_size(d.dtype);
  p->desc = d;
  p->transposed = transposed;
  p->bias_div = 1;
  p->ksplit = 1;
  p->cfg = -1;
  p->staged = false;
  output_dims(d, tr, &p->ho, &p->wo);
  p->mem = mem;
  p->alloc_stream = stream;
  p->grouped = true;
  p->wp_bytes = (size_t)d.c_in * (d.c_out / d.groups) * d.r * d.s * esz;
  PlanShape shape;
  p->nonzero_macs = build_shape(d, tr, 2, 128, &shape) ? shape.nonzero_macs / d.groups : 0;
  p->issued_macs = p->nonzero_macs;
  GrArgs& g = p->grargs;
  std::memset(&g, 0, sizeof(g));
  g.n = d.n;
  g.cin = d.c_in;
  g.h = d.h;
  g.w_ = d.w;
  g.cout = d.c_out;
  g.r = d.r;
  g.s = d.s;
  g.stride_h = d.stride_h;
  g.stride_w = d.stride_w;
  g.pad_h = d.pad_h;
  g.pad_w = d.pad_w;
  g.dil_h = d.dil_h;
  g.dil_w = d.dil_w;
  g.ho = p->ho;
  g.wo = p->wo;
  g.groups = d.groups;
  g.transposed = transposed;
  g.nhwc = d.layout == HUGE2_NHWC;
  g.act = d.activation;
  std::snprintf(p->kernel_name, sizeof(p->kernel_name), "grouped_kernel g%d", d.groups);
  huge2_status st = dev_alloc(p, &p->wp, p->wp_bytes);
  if (st != HUGE2_OK) {
    free_buffers(p);
    delete p;
    return st;
  }
  bool ok = !fault("launch") &&
            hipMemcpyAsync(p->wp, w, p->wp_bytes, hipMemcpyDeviceToDevice, stream) == hipSuccess;
  if (ok) ok = hipStreamSynchronize(stream) == hipSuccess;
  if (!ok) {
    (void)hipGetLastError();
    free_buffers(p);
    delete p;
    return HUGE2_ERR_HIP;
  }
  *out = p;
  return HUGE2_OK;
}

huge2_status create_impl(huge2_plan** out, const huge2_conv_desc* desc, int transposed,
                         const void* w, hipStream_t stream, Mem mem) {
  if (!out) return HUGE2_ERR_INVALID_ARG;
  *out = nullptr;
  if (transposed != 0 && transposed != 1) return HUGE2_ERR_INVALID_ARG;
  huge2_status st = validate_desc(desc, transposed != 0);
  if (st != HUGE2_OK) return st;
  if (!w) return HUGE2_ERR_INVALID_ARG;
  const bool tr = transposed != 0;
  if (desc->groups > 1) return create_grouped(out, *desc, transposed, w, stream, mem);
  // the 1x1-input product form: bias k then covers r*s consecutive columns
  huge2_conv_desc dd;
  int bias_div, bias_mod, prod_rs;
  product_form(*desc, tr, &dd, &bias_div, &bias_mod, &prod_rs);
  const huge2_conv_desc& d = dd;
  {
    huge2_conv_desc d1;
    if (two_pass_shape(d, tr, &d1)) return create_two_pass(out, d, d1, w, stream, mem);
    if (gather_shape(d, tr, &d1)) return create_gather(out, d, d1, w, stream, mem);
  }

  {
    ZArgs z;
    int64_t z_issued = 0;
    if (ztile_shape(d, tr, &z, &z_issued))
      return create_direct(out, d, transposed, w, stream, mem, &z, nullptr, nullptr,
                           z_issued);
    CpArgs cpa;
    if (colphase_shape(d, tr, &cpa, &z_issued))
      return create_direct(out, d, transposed, w, stream, mem, nullptr, nullptr, nullptr,
                           z_issued, &cpa);
    RpArgs rp;
    if (rowphase_shape(d, tr, &rp, &z_issued))
      return create_direct(out, d, transposed, w, stream, mem, nullptr, &rp, nullptr,
                           z_issued);
    QArgs q;
    if (quad_shape(d, tr, &q, &z_issued))
      return create_direct(out, d, transposed, w, stream, mem, nullptr, nullptr, &q,
                           z_issued);
  }

  PlanShape shape;
  ListedShape ls;
  bool listed = false;
  const int cfg = plan_gemm_shape(d, tr, &shape, &listed, &ls);
  if (cfg < 0) return HUGE2_ERR_INVALID_ARG;
  const int bm = tile_bm(cfg), bn = tile_bn(cfg);

  huge2_plan* p = new (std::nothrow) huge2_plan();
  if (!p) return HUGE2_ERR_ALLOC;
  p->desc = d;
  p->transposed = transposed;
  output_dims(d, tr, &p->ho, &p->wo);
  p->cfg = cfg;
  p->bias_div = bias_div;
  p->bias_mod = bias_mod;
  p->prod_rs = prod_rs;
  {
    const TileShape& t = kTiles[cfg];
    if (t.kind == 0)
      std::snprintf(p->kernel_name, sizeof(p->kernel_name), "phase_gemm_kernel %dx%d w%dx%d",
                    t.bm, t.bn, t.pw, t.cw);
    else
      std::snprintf(p->kernel_name, sizeof(p->kernel_name), "phase_gemm%d_kernel %dx%d w%d k%d",
                    t.kind == 3 ? 3 : 2, t.bm, t.bn, t.pw * t.cw, t.ksplit);
    if (listed) {
      const size_t len = std::strlen(p->kernel_name);
      std::snprintf(p->kernel_name + len, sizeof(p->kernel_name) - len, " listed");
    }
  }
  const int esz = elem_size(d.dtype);
  const int vec = 16 / esz;
  const int bk = tile_kb(cfg) / esz;
  // NCHW inputs and ragged channel counts are re-laid out to channel-
  // contiguous pixels (channel count padded to 16 bytes) by a staging kernel.
  p->staged = !(d.layout == HUGE2_NHWC && d.c_in % vec == 0);
  p->c_stride = p->staged ? round_up(d.c_in, vec) : d.c_in;
  p->x_bytes = (size_t)d.n * d.h * d.w * p->c_stride * esz;
  p->cin_pad = round_up(d.c_in, bk);
  p->cout_pad = round_up(d.c_out, bn);
  p->mem = mem;
  p->alloc_stream = stream;
  p->nonzero_macs = shape.nonzero_macs;

  // Device views of the decomposition, and the work list.
  std::vector<SegDev> segs;
  std::vector<TapDev> taps;
  std::vector<WorkDev> works;
  const int ntiles_n = p->cout_pad / bn;
  int64_t issued = 0;
  std::vector<uint32_t> ptab;
  if (listed) {
    // one segment over every image; each tile of bm listed pixels of one image
    // runs its own tap set (the taps of equal sets are stored once)
    SegDev sd;
    std::memset(&sd, 0, sizeof(sd));
    const int per_img = (int)ls.pix.size();
    sd.nphase_w = sd.nphase = 1;
    sd.m_total = d.n * per_img;
    sd.out_step_h = sd.out_step_w = 1;
    sd.in0_h = -d.pad_h;
    sd.in0_w = -d.pad_w;
    sd.in_step_h = sd.in_step_w = 1;
    sd.ptab = 0;
    sd.per_img = per_img;
    sd.ntw = 1;
    const uint32_t divisors[4] = {1, 1, (uint32_t)per_img, 1};
    for (int k = 0; k < 4; ++k) division_magic(divisors[k], &sd.div_mul[k], &sd.div_shift[k]);
    segs.push_back(sd);
    ptab = ls.pix;
    std::vector<std::pair<int, int>> tile_range;  // (tap_begin, tap_count) per tile
    for (const auto& tl : ls.tile_taps) {
      int found = -1;
      for (size_t u = 0; u < tile_range.size() && found < 0; ++u) {
        const auto& prev = ls.tile_taps[u];
        if (prev.size() != tl.size()) continue;
        bool same = true;
        for (size_t k = 0; k < tl.size() && same; ++k)
          same = prev[k].kh == tl[k].kh && prev[k].kw == tl[k].kw;
        if (same) found = (int)u;
      }
      if (found >= 0) {
        tile_range.push_back(tile_range[found]);
        continue;
      }
      tile_range.emplace_back((int)taps.size(), (int)tl.size());
      for (const huge2_tap& t : tl) {
        TapDev td;
        td.slot = t.kh * d.s + t.kw;
        td.off_h = t.off_h;
        td.off_w = t.off_w;
        td.pad = 0;
        taps.push_back(td);
      }
    }
    for (int img = 0; img < d.n; ++img)
      for (size_t t = 0; t < ls.tile_taps.size(); ++t) {
        const int m0 = img * per_img + (int)t * bm;
        for (int nt = 0; nt < ntiles_n; ++nt) {
          WorkDev wd;
          std::memset(&wd, 0, sizeof(wd));
          wd.seg = 0;
          wd.m0 = m0;
          wd.m1 = std::min(m0 + bm, (img + 1) * per_img);
          wd.n0 = nt * bn;
          wd.tap_begin = tile_range[t].first;
          wd.tap_count = tile_range[t].second;
          works.push_back(wd);
          issued += (int64_t)bm * bn * wd.tap_count * p->cin_pad;
        }
      }
  }
  for (const huge2_tap& t : shape.taps) {
    if (listed) break;
    TapDev td;
    td.slot = t.kh * d.s + t.kw;
    td.off_h = t.off_h;
    td.off_w = t.off_w;
    td.pad = 0;
    taps.push_back(td);
  }
  for (size_t i = 0; i < shape.segs.size() && !listed; ++i) {
    const huge2_segment& s = shape.segs[i];
    SegDev sd;
    std::memset(&sd, 0, sizeof(sd));
    sd.ptab = -1;
    sd.phase0_h = s.phase0_h;
    sd.phase0_w = s.phase0_w;
    sd.nphase_w = s.nphase_w;
    sd.m_total = d.n * s.nphase_h * s.nphase_w * s.qn_h * s.qn_w;
    sd.out_step_h = s.out_step_h;
    sd.out_step_w = s.out_step_w;
    sd.q0_h = s.q0_h;
    sd.q0_w = s.q0_w;
    sd.qn_h = s.qn_h;
    sd.qn_w = s.qn_w;
    sd.in0_h = s.in0_h;
    sd.in0_w = s.in0_w;
    sd.in_dphase_h = s.in_dphase_h;
    sd.in_dphase_w = s.in_dphase_w;
    sd.in_step_h = s.in_step_h;
    sd.in_step_w = s.in_step_w;
    sd.tap_begin = s.tap_begin;
    sd.tap_count = s.tap_count;
    sd.nphase = s.nphase_h * s.nphase_w;
    const uint32_t divisors[4] = {(uint32_t)s.qn_w, (uint32_t)s.qn_h, (uint32_t)sd.nphase,
                                  (uint32_t)s.nphase_w};
    for (int k = 0; k < 4; ++k) division_magic(divisors[k], &sd.div_mul[k], &sd.div_shift[k]);
    // exact: every tap's read is in range for every pixel of the segment (the
    // input coordinate is affine and non-decreasing in phase and q, so the
    // extremes are at the segment's corners)
    sd.exact = 1;
    for (int t = s.tap_begin; t < s.tap_begin + s.tap_count; ++t) {
      const huge2_tap& tp = shape.taps[t];
      const long long h_lo = s.in0_h + (long long)s.in_step_h * s.q0_h + tp.off_h;
      const long long h_hi = s.in0_h + (long long)s.in_dphase_h * (s.nphase_h - 1) +
                             (long long)s.in_step_h * (s.q0_h + s.qn_h - 1) + tp.off_h;
      const long long w_lo = s.in0_w + (long long)s.in_step_w * s.q0_w + tp.off_w;
      const long long w_hi = s.in0_w + (long long)s.in_dphase_w * (s.nphase_w - 1) +
                             (long long)s.in_step_w * (s.q0_w + s.qn_w - 1) + tp.off_w;
      if (h_lo < 0 || h_hi >= d.h || w_lo < 0 || w_hi >= d.w) sd.exact = 0;
    }
    sd.tap_ap = tap_progressions(&shape.taps[s.tap_begin], s.tap_count, &sd) ? 1 : 0;
    if (!sd.tap_ap) sd.ntw = 1;
    segs.push_back(sd);
    for (int m0 = 0; m0 < sd.m_total; m0 += bm)
      for (int nt = 0; nt < ntiles_n; ++nt) {
        WorkDev wd;
        std::memset(&wd, 0, sizeof(wd));
        wd.seg = (int32_t)i;
        wd.m0 = m0;
        wd.m1 = std::min(m0 + bm, sd.m_total);
        wd.n0 = nt * bn;
        wd.ks = 0;
        wd.tap_begin = s.tap_begin;
        wd.tap_count = s.tap_count;
        works.push_back(wd);
        issued += (int64_t)bm * bn * s.tap_count * p->cin_pad;
      }
  }
  p->issued_macs = issued;
  bool all_ap = true;
  for (WorkDev& wd : works) {
    work_progressions(taps.data() + wd.tap_begin, wd.tap_count, d.s, &wd);
    all_ap = all_ap && wd.ap_ntw > 0;
  }
  if (kTiles[p->cfg].kind == 3 && !all_ap) {
    // the pipelined kernel steps through progressions only: the split-wave
    // kernel of the same tile and packing takes tap lists
    // (the same works and lane-ordered packing; its K block must divide the
    // padded channel count; one with the same K groups first)
    const int from = p->cfg;
    for (int pass = 0; pass < 2 && kTiles[p->cfg].kind == 3; ++pass)
      for (int c = 0; c < TILE_COUNT; ++c) {
        const TileShape &t = kTiles[c], &u = kTiles[from];
        if (t.kind == 1 && t.bm == u.bm && t.bn == u.bn && (pass == 1 || t.ksplit == u.ksplit) &&
            p->cin_pad % (t.kb / esz) == 0) {
          p->cfg = c;
          break;
        }
      }
    if (kTiles[p->cfg].kind == 3) {
      free_buffers(p);
      delete p;
      return HUGE2_ERR_UNSUPPORTED;
    }
    const TileShape& t = kTiles[p->cfg];
    std::snprintf(p->kernel_name, sizeof(p->kernel_name), "phase_gemm2_kernel %dx%d w%d k%d%s",
                  t.bm, t.bn, t.pw * t.cw, t.ksplit, listed ? " listed" : "");
  }
  // Too few tiles to give every compute unit one: split the input channel
  // blocks into ksplit slices, one workgroup per (tile, slice), whose fp32
  // partials a second kernel adds in slice order (deterministic), with the
  // bias and activation.  The partials cost 2 x 4 x ksplit bytes per output.
  // (HUGE2_SPLITK forces a count, up to the channel blocks.)
  {
    const int cblocks = p->cin_pad / bk;
    int max_taps = 1;
    for (const SegDev& sd : segs) max_taps = std::max(max_taps, (int)sd.tap_count);
    // at least 8 K stages per slice: shorter slices lose more to the second
    // launch than they gain (measured on a 2-block, 1-tap GEMM)
    int ks = std::min({cblocks, kComputeUnits / std::max(1, (int)works.size()), 8,
                       std::max(1, cblocks * max_taps / 8)});
    const int forced = env_int("HUGE2_SPLITK", -1);
    if (forced >= 1) ks = std::min(forced, cblocks);
    const size_t ny = (size_t)d.n * d.c_out * p->ho * p->wo;
    while (ks > 1 && (ks * ny * 4 > ((size_t)1 << 28) || ny >= ((size_t)1 << 31))) --ks;
    p->ksplit = std::max(1, ks);
    // With four or more slices per tile, the two K groups inside a workgroup
    // of the 64 x 128 tile only halve work that is already short: its
    // one-group form (same tile, same work list and packing, three
    // workgroups per compute unit) measured faster on the batch-1 5x5
    // DCGAN layers (17.3 against 20.1 us, 16.1 against 18.9 us).
    if (p->ksplit >= 4 && p->cfg == TILE_SW_64x128_K2 && env_int("HUGE2_TILE", -1) < 0) {
      p->cfg = TILE_SW_64x128;
      const TileShape& t = kTiles[TILE_SW_64x128];
      std::snprintf(p->kernel_name, sizeof(p->kernel_name), "phase_gemm2_kernel %dx%d w%d k%d",
                    t.bm, t.bn, t.pw * t.cw, t.ksplit);
    }
    if (p->ksplit > 1) {
      const size_t nw = works.size();
      for (int k = 1; k < p->ksplit; ++k)
        for (size_t i = 0; i < nw; ++i) {
          WorkDev wd = works[i];
          wd.ks = k;
          works.push_back(wd);
        }
    }
  }
  p->n_works = (int)works.size();
  // NCHW outputs of transposed convs with few phases: the phases of a
  // region share input rows and output cache lines (measured: fewer bytes and
  // faster); elsewhere the segment-major order measured as fast or faster,
  // except for works that are all resident at once: their XCDs then finish
  // when their own works do, so every XCD takes a cell of every phase, and
  // inside the cell long works share compute units with short ones.
  // (HUGE2_WORK_ORDER=0 forces segment-major order, 1 the cells alone.)
  const int order = env_int("HUGE2_WORK_ORDER", -1);
  const bool resident =
      (int64_t)works.size() <= (int64_t)kComputeUnits * kTiles[p->cfg].wg_per_cu + 8;
  if (order == 1 || (order < 0 && tr && (d.layout == HUGE2_NCHW || resident) &&
                     d.stride_h * d.stride_w <= 16))
    order_works_for_xcds(works, segs, d.n, p->ho, bn, ntiles_n, (double)p->x_bytes,
                         (double)d.r * d.s * p->cout_pad * p->cin_pad * esz);
  if (order != 0 && order != 1 && resident)
    order_works_resident(works, p->cin_pad / bk, p->ksplit, kTiles[p->cfg].wg_per_cu);

  const size_t seg_b = segs.size() * sizeof(SegDev);
  const size_t tap_b = taps.size() * sizeof(TapDev);
  const size_t work_b = works.size() * sizeof(WorkDev);
  const size_t ptab_b = ptab.size() * sizeof(uint32_t);
  const size_t meta_b = seg_b + tap_b + work_b + ptab_b;
  const size_t wp_b = (size_t)d.r * d.s * p->cout_pad * p->cin_pad * esz;
  const size_t xs_b = p->staged ? p->x_bytes : 0;
  p->wp_bytes = wp_b;

  const size_t part_b =
      p->ksplit > 1 ? (size_t)p->ksplit * d.n * d.c_out * p->ho * p->wo * sizeof(float) : 0;
  if ((st = dev_alloc(p, &p->meta, meta_b)) != HUGE2_OK ||
      (st = dev_alloc(p, &p->wp, wp_b)) != HUGE2_OK ||
      (st = dev_alloc(p, &p->xs, xs_b)) != HUGE2_OK ||
      (st = dev_alloc(p, &p->part, part_b)) != HUGE2_OK) {
    free_buffers(p);
    delete p;
    return st;
  }
  p->d_segs = (SegDev*)p->meta;
  p->d_taps = (TapDev*)((char*)p->meta + seg_b);
  p->d_works = (WorkDev*)((char*)p->meta + seg_b + tap_b);
  p->d_ptab = ptab_b ? (const uint32_t*)((char*)p->meta + seg_b + tap_b + work_b) : nullptr;

  std::vector<char> host(meta_b);
  if (seg_b) std::memcpy(host.data(), segs.data(), seg_b);
  if (tap_b) std::memcpy(host.data() + seg_b, taps.data(), tap_b);
  if (work_b) std::memcpy(host.data() + seg_b + tap_b, works.data(), work_b);
  if (ptab_b) std::memcpy(host.data() + seg_b + tap_b + work_b, ptab.data(), ptab_b);

  bool ok = !fault("launch");
  if (ok && meta_b)
    ok = hipMemcpyAsync(p->meta, host.data(), meta_b, hipMemcpyHostToDevice, stream) == hipSuccess;
  if (ok)
    ok = launch_pack_weights(w, p->wp, d.dtype, tr, d.c_in, d.c_out, d.r, d.s, p->cin_pad,
                             p->cout_pad, kTiles[p->cfg].kind != 0 ? kPackKB : 0, stream,
                             p->prod_rs) == hipSuccess;
  // the host copy of the metadata must outlive the transfer
  if (ok) ok = hipStreamSynchronize(stream) == hipSuccess;
  if (ok) {
    p->h_segs = std::move(segs);
    p->h_taps = std::move(taps);
    p->h_works = std::move(works);
    p->h_ptab = std::move(ptab);
  }
  if (!ok) {
    (void)hipGetLastError();
    free_buffers(p);
    delete p;
    return HUGE2_ERR_HIP;
  }
  *out = p;
  return HUGE2_OK;
}

huge2_status stage_impl(const huge2_plan* p, const void* x, hipStream_t stream) {
  if (!p) return HUGE2_ERR_INVALID_ARG;
  if (p->gather) {
    if (!x) return HUGE2_ERR_INVALID_ARG;
    if (fault("launch")) return HUGE2_ERR_HIP;
    const huge2_conv_desc& d = p->desc;
    GatherArgs g;
    g.x = x;
    g.xs = p->inner->xs;
    g.n = d.n;
    g.cin = d.c_in;
    g.h = d.h;
    g.w = d.w;
    g.r = d.r;
    g.s = d.s;
    g.stride_h = d.stride_h;
    g.stride_w = d.stride_w;
    g.pad_h = d.pad_h;
    g.pad_w = d.pad_w;
    g.dil_h = d.dil_h;
    g.dil_w = d.dil_w;
    g.ho = p->ho;
    g.wo = p->wo;
    g.c_stride = p->inner->c_stride;
    if (launch_gather_taps(g, d.dtype, stream) != hipSuccess) {
      (void)hipGetLastError();
      return HUGE2_ERR_HIP;
    }
    return HUGE2_OK;
  }
  if (p->inner) return stage_impl(p->inner, x, stream);
  if (!p->staged) return HUGE2_OK;
  if (!x) return HUGE2_ERR_INVALID_ARG;
  const huge2_conv_desc& d = p->desc;
  if (fault("launch")) return HUGE2_ERR_HIP;
  if (launch_stage_input(x, p->xs, d.dtype, d.layout == HUGE2_NCHW, d.n, d.c_in, d.h * d.w,
                         p->c_stride, stream) != hipSuccess) {
    (void)hipGetLastError();
    return HUGE2_ERR_HIP;
  }
  return HUGE2_OK;
}

huge2_status gemm_impl(const huge2_plan* p, const void* x, const float* bias, void* y,
                       hipStream_t stream) {
  if (!p || !y || (!p->staged && !x) || x == y) return HUGE2_ERR_INVALID_ARG;
  const huge2_conv_desc& d = p->desc;
  if (fault("launch")) return HUGE2_ERR_HIP;
  if (p->gather) return gemm_impl(p->inner, x, bias, y, stream);
  if (p->inner) {
    huge2_status st = gemm_impl(p->inner, x, nullptr, p->zbuf, stream);
    if (st != HUGE2_OK) return st;
    CombArgs c;
    c.z = (const float*)p->zbuf;
    c.bias = bias;
    c.y = (float*)y;
    c.n = d.n;
    c.h = d.h;
    c.w = d.w;
    c.cout = d.c_out;
    c.r = d.r;
    c.s = d.s;
    c.stride_h = d.stride_h;
    c.stride_w = d.stride_w;
    c.pad_h = d.pad_h;
    c.pad_w = d.pad_w;
    c.dil_h = d.dil_h;
    c.dil_w = d.dil_w;
    c.ho = p->ho;
    c.wo = p->wo;
    c.act = d.activation;
    if (launch_taps_combine(c, stream) != hipSuccess) {
      (void)hipGetLastError();
      return HUGE2_ERR_HIP;
    }
    return HUGE2_OK;
  }
  if (p->ztile) {
    ZArgs z = p->zargs;
    z.x = x;
    z.wp = p->wp;
    z.bias = bias;
    z.y = y;
    z.act = d.activation;
    if (launch_ztile(z, d.dtype, stream) != hipSuccess) {
      (void)hipGetLastError();
      return HUGE2_ERR_HIP;
    }
    return HUGE2_OK;
  }
  if (p->grouped) {
    GrArgs g = p->grargs;
    g.x = x;
    g.w = p->wp;
    g.bias = bias;
    g.y = y;
    if (launch_grouped(g, d.dtype, stream) != hipSuccess) {
      (void)hipGetLastError();
      return HUGE2_ERR_HIP;
    }
    return HUGE2_OK;
  }
  if (p->colphase) {
    CpArgs z = p->cpargs;
    z.x = x;
    z.wp = p->wp;
    z.bias = bias;
    z.y = y;
    z.act = d.activation;
    if (launch_colphase(z, stream) != hipSuccess) {
      (void)hipGetLastError();
      return HUGE2_ERR_HIP;
    }
    return HUGE2_OK;
  }
  if (p->rowphase) {
    RpArgs z = p->rpargs;
    z.x = x;
    z.wp = p->wp;
    z.bias = bias;
    z.y = y;
    z.act = d.activation;
    if (launch_rowphase(z, stream) != hipSuccess) {
      (void)hipGetLastError();
      return HUGE2_ERR_HIP;
    }
    return HUGE2_OK;
  }
  if (p->quad) {
    QArgs z = p->qargs;
    z.x = x;
    z.wp = p->wp;
    z.bias = bias;
    z.y = y;
    z.act = d.activation;
    if (launch_quad(z, stream) != hipSuccess) {
      (void)hipGetLastError();
      return HUGE2_ERR_HIP;
    }
    return HUGE2_OK;
  }
  GemmArgs a;
  std::memset(&a, 0, sizeof(a));
  a.x = p->staged ? p->xs : x;
  a.wp[0] = p->wp;
  a.bias[0] = bias;
  a.y[0] = y;
  a.bias_div = p->bias_div;
  a.bias_mod = p->bias_mod;
  a.act = d.activation;
  a.ksplit = p->ksplit;
  a.part = (float*)p->part;
  a.part_stride = (uint32_t)((size_t)d.n * d.c_out * p->ho * p->wo);
  if (p->ksplit > 1) {
    // the slices write partials; bias and activation come with the sum
    a.bias[0] = nullptr;
    a.act = HUGE2_ACT_NONE;
  }
  a.segs = p->d_segs;
  a.taps = p->d_taps;
  a.works = p->d_works;
  a.ptab = p->d_ptab;
  a.n_works = p->n_works;
  a.n = d.n;
  a.h = d.h;
  a.w = d.w;
  a.cin = p->c_stride;
  a.ks = d.s;
  a.x_bytes = (uint32_t)p->x_bytes;
  a.wp_bytes = (uint32_t)p->wp_bytes;
  a.cin_pad = p->cin_pad;
  a.cout = d.c_out;
  a.cout_pad = p->cout_pad;
  a.ho = p->ho;
  a.wo = p->wo;
  if (launch_phase_gemm(a, d.dtype, p->cfg, d.layout == HUGE2_NCHW, stream) != hipSuccess) {
    (void)hipGetLastError();
    return HUGE2_ERR_HIP;
  }
  if (p->ksplit > 1) {
    SplitKArgs r;
    r.part = (const float*)p->part;
    r.bias = bias;
    r.y = y;
    r.stride = a.part_stride;
    r.total = a.part_stride;
    r.ksplit = p->ksplit;
    r.cout = d.c_out;
    r.hw = p->ho * p->wo;
    r.nchw = d.layout == HUGE2_NCHW ? 1 : 0;
    r.bias_div = p->bias_div;
    r.bias_mod = p->bias_mod;
    r.act = d.activation;
    if (launch_splitk_reduce(r, d.dtype, stream) != hipSuccess) {
      (void)hipGetLastError();
      return HUGE2_ERR_HIP;
    }
  }
  return HUGE2_OK;
}

huge2_status execute_impl(const huge2_plan* p, const void* x, const float* bias, void* y,
                          hipStream_t stream) {
  if (!p || !x || !y || x == y) return HUGE2_ERR_INVALID_ARG;
  huge2_status st = stage_impl(p, x, stream);
  if (st != HUGE2_OK) return st;
  return gemm_impl(p, x, bias, y, stream);
}

huge2_status one_shot(const huge2_conv_desc* desc, int transposed, const void* x, const void* w,
                      const float* bias, void* y, hipStream_t stream) {
  huge2_status st = validate_desc(desc, transposed != 0);
  if (st != HUGE2_OK) return st;
  if (!x || !w || !y || x == y) return HUGE2_ERR_INVALID_ARG;
  huge2_plan* p = nullptr;
  Mem mem;
  mem.stream_ordered = true;
  st = create_impl(&p, desc, transposed, w, stream, mem);
  if (st != HUGE2_OK) return st;
  st = execute_impl(p, x, bias, y, stream);
  free_buffers(p);  // stream-ordered: released after the enqueued work
  delete p;
  return st;
}

// The no-allocation form of the one-shot transposed conv: every device
// buffer the plan needs (packed weights, work list, staging, K-slice
// partials) is carved from this device's copy of `scratch`, whose device
// address hipGetSymbolAddress gives once per device (in host code the
// array's name is not a device address).
constexpr size_t kScratchBytes = (size_t)64 << 20;
constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void* g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];

}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

huge2_status scratch_region(void** ptr) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return HUGE2_ERR_HIP;
  }
  std::call_once(g_scratch_once[dev], [dev] {
    void* p = nullptr;
    g_scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch_ptr[dev] = g_scratch_err[dev] == hipSuccess ? p : nullptr;
  });
  if (g_scratch_err[dev] != hipSuccess || !g_scratch_ptr[dev]) return HUGE2_ERR_HIP;
  *ptr = g_scratch_ptr[dev];
  return HUGE2_OK;
}

huge2_status one_shot_noalloc(const huge2_conv_desc* desc, const void* x, const void* w,
                              const float* bias, void* y, hipStream_t stream) {
  huge2_status st = validate_desc(desc, true);
  if (st != HUGE2_OK) return st;
  if (!x || !w || !y || x == y) return HUGE2_ERR_INVALID_ARG;
  void* base = nullptr;
  if ((st = scratch_region(&base)) != HUGE2_OK) return st;
  Arena arena{(char*)base, kScratchBytes, 0};
  Mem mem;
  mem.arena = &arena;
  huge2_plan* p = nullptr;
  st = create_impl(&p, desc, 1, w, stream, mem);
  if (st != HUGE2_OK) return st;
  st = execute_impl(p, x, bias, y, stream);
  free_buffers(p);  // nothing to release: the buffers lie in the scratch region
  delete p;
  return st;
}

}  // namespace

// ---------------------------------------------------------------------------
// Weight gradients (section 3.2.3).

struct huge2_wgrad_plan {
  huge2_conv_desc desc;
  int transposed;
  int ms, nb;          // small / big tensor channels
  int hs, ws, hb, wb;  // small / big pixel grids
  int chunk;           // images per chunk
  int kp;              // padded K of a full chunk
  int ksplit;          // K slices of the GEMM (workgroups along K)
  int groups;          // > 1: grouped conv (direct per-plane sums, no workspace)
  int direct_out;      // the GEMM writes dw (WgArgs::direct_out)
  int gather_ib;       // images per LDS-gather workgroup (0: the staging kernel gathers)
  int bt_phase;        // Bt in phase planes (WgArgs::bt_phase)
  int hr, sh_min;
  int direct;          // St read in place from the small tensor (WgArgs::direct)
  void* st;
  void* bt;
  float* g;
};

namespace {

constexpr long long kWgradStageBudget = 256ll << 20;  // staged operands of one chunk

void wgrad_free(huge2_wgrad_plan* p) {
  void* bufs[3] = {p->st, p->bt, p->g};
  for (void* b : bufs)
    if (b) (void)hipFree(b);
  p->st = p->bt = nullptr;
  p->g = nullptr;
}

huge2_status wgrad_create(huge2_wgrad_plan** out, const huge2_conv_desc* desc, int transposed) {
  if (!out) return HUGE2_ERR_INVALID_ARG;
  *out = nullptr;
  if (transposed != 0 && transposed != 1) return HUGE2_ERR_INVALID_ARG;
  huge2_status st = validate_desc(desc, transposed != 0);
  if (st != HUGE2_OK) return st;
  const huge2_conv_desc& d = *desc;
  if (d.layout != HUGE2_NCHW || d.activation != HUGE2_ACT_NONE) return HUGE2_ERR_UNSUPPORTED;
  int ho, wo;
  if (!output_dims(d, transposed != 0, &ho, &wo)) return HUGE2_ERR_INVALID_ARG;
  huge2_wgrad_plan* p = new (std::nothrow) huge2_wgrad_plan();
  if (!p) return HUGE2_ERR_ALLOC;
  p->desc = d;
  p->transposed = transposed;
  if (transposed) {  // small = x, big = dy
    p->ms = d.c_in, p->nb = d.c_out, p->hs = d.h, p->ws = d.w, p->hb = ho, p->wb = wo;
  } else {           // small = dy, big = x
    p->ms = d.c_out, p->nb = d.c_in, p->hs = ho, p->ws = wo, p->hb = d.h, p->wb = d.w;
  }
  const long long esz = elem_size(d.dtype), taps = (long long)d.r * d.s;
  if (d.groups > 1) {
    // grouped: one plane per (small channel, big channel of its group), no
    // staged operands and no fp32 gradient (wgrad_grouped_kernel)
    const long long big_b = (long long)d.n * p->nb * p->hb * p->wb * esz;
    const long long small_b = (long long)d.n * p->ms * p->hs * p->ws * esz;
    if (big_b >= (1ll << 40) || small_b >= (1ll << 40) || taps > 65535 ||
        (long long)p->ms * (p->nb / d.groups) >= (1ll << 31)) {
      delete p;
      return HUGE2_ERR_UNSUPPORTED;
    }
    p->groups = d.groups;
    p->chunk = d.n;
    p->ksplit = 1;
    *out = p;
    return HUGE2_OK;
  }
  const long long hws = (long long)p->hs * p->ws;
  const long long per_img = esz * (p->ms + taps * p->nb) * hws;
  long long chunk = std::max(1ll, std::min<long long>(d.n, kWgradStageBudget / std::max(1ll, per_img)));
  {
    // HUGE2_WGRAD_CHUNK: fewer images per chunk (tests of the chunk accumulation)
    const int forced = env_int("HUGE2_WGRAD_CHUNK", 0);
    if (forced > 0 && forced < chunk) chunk = forced;
  }
  const long long kp = (chunk * hws + 63) / 64 * 64;
  // St read in place where every 64-pixel K run lies in one channel plane
  // (HUGE2_WGRAD_DIRECT=0: always staged)
  p->direct = hws % 64 == 0 && env_int("HUGE2_WGRAD_DIRECT", 1) != 0;
  // the large tensor's copies through LDS where its planes fit
  // (HUGE2_WGRAD_GATHER=0: the plain staging kernel gathers them)
  p->gather_ib = env_int("HUGE2_WGRAD_GATHER", 1) != 0
                     ? wgrad_gather_images(p->hs, p->ws, p->hb, p->wb, (int)esz, (int)chunk, p->nb)
                     : 0;
  // phase planes instead of per-tap copies where a K stage lies in one image
  // and the planes (hr rows each) are smaller than the taps' copies
  // (HUGE2_WGRAD_PHASE=0: per-tap copies)
  {
    const int sh_lo = floor_div_i(-d.pad_h, d.stride_h);
    const int sh_hi = floor_div_i((d.r - 1) * d.dil_h - d.pad_h, d.stride_h);
    p->sh_min = sh_lo;
    p->hr = p->hs + sh_hi - sh_lo;
    p->bt_phase = p->gather_ib > 0 && hws % 64 == 0 && p->ws % 8 == 0 &&
                  (long long)d.stride_h * p->hr < (long long)d.r * p->hs &&
                  env_int("HUGE2_WGRAD_PHASE", 1) != 0;
  }
  // one GEMM of all taps: N = nb * taps columns (n, tap), dw's own order
  const long long nb_g = taps * p->nb;
  if (nb_g >= (1ll << 30)) {
    delete p;
    return HUGE2_ERR_UNSUPPORTED;
  }
  // split K so that the GEMM has about two workgroups per compute unit
  // (the 128 x 128 tiles run two per compute unit; the 64 x 64 ones four),
  // each split keeping at least 8 K stages
  const long long wt = wgrad_tile(p->ms, (int)nb_g);
  const long long tiles = ((p->ms + wt - 1) / wt) * ((nb_g + wt - 1) / wt);
  const long long stages = kp * esz / 128;
  const long long per_cu = wt == 128 ? 2 : 4;
  long long ksplit = std::max(1ll, (per_cu * kComputeUnits + tiles - 1) / tiles);
  ksplit = std::max(1ll, std::min(ksplit, stages / 8));
  // each slice's fp32 gradient is read back by the store: at most 32 MiB of
  // them (DCGAN's 512 -> 256 and 256 -> 128 layers measured fastest at 4 and
  // 16 slices, two workgroups per compute unit, despite the larger store)
  const long long g_slice = taps * p->ms * p->nb * 4;
  ksplit = std::min(ksplit, std::max(1ll, (32ll << 20) / g_slice));
  ksplit = std::min(ksplit, 256ll);
  {
    // HUGE2_WGRAD_KSPLIT: a given number of K slices (tests and tuning)
    const int forced = env_int("HUGE2_WGRAD_KSPLIT", 0);
    if (forced > 0) ksplit = std::min<long long>(forced, std::max(1ll, stages));
  }
  // one K slice over the whole batch: the GEMM writes dw itself, rounded
  // once, and there is no fp32 gradient (HUGE2_WGRAD_DIRECT_OUT=0: never)
  p->direct_out = ksplit == 1 && chunk >= d.n && env_int("HUGE2_WGRAD_DIRECT_OUT", 1) != 0;
  const long long st_b = p->direct ? 0 : p->ms * kp * esz;
  const long long bt_b = p->bt_phase
                             ? (long long)p->nb * d.stride_h * d.s * chunk * p->hr * p->ws * esz
                             : taps * p->nb * kp * esz;
  const long long g_b = p->direct_out ? 0 : ksplit * taps * p->ms * p->nb * 4;
  const long long big_b = (long long)d.n * p->nb * p->hb * p->wb * esz;
  const long long small_b = (long long)d.n * p->ms * hws * esz;
  if (st_b >= (1ll << 31) || bt_b >= (1ll << 31) || g_b >= (1ll << 31) || big_b >= (1ll << 40) ||
      small_b >= (1ll << 40) || taps > 65535 || (p->ms + wt - 1) / wt > 65535 ||
      (nb_g + wt - 1) / wt > 65535) {
    delete p;
    return HUGE2_ERR_UNSUPPORTED;
  }
  p->chunk = (int)chunk;
  p->kp = (int)kp;
  p->ksplit = (int)ksplit;
  if (fault("alloc") || (st_b > 0 && hipMalloc(&p->st, st_b) != hipSuccess) ||
      hipMalloc(&p->bt, bt_b) != hipSuccess ||
      (g_b > 0 && hipMalloc((void**)&p->g, g_b) != hipSuccess)) {
    (void)hipGetLastError();
    wgrad_free(p);
    delete p;
    return HUGE2_ERR_ALLOC;
  }
  *out = p;
  return HUGE2_OK;
}

huge2_status wgrad_execute(const huge2_wgrad_plan* p, const void* x, const void* dy, void* dw,
                           hipStream_t stream) {
  if (!p || !x || !dy || !dw || dw == x || dw == dy) return HUGE2_ERR_INVALID_ARG;
  const huge2_conv_desc& d = p->desc;
  if (fault("launch")) return HUGE2_ERR_HIP;
  WgArgs a;
  std::memset(&a, 0, sizeof(a));
  a.sm = p->transposed ? x : dy;
  a.bg = p->transposed ? dy : x;
  a.st = p->st;
  a.bt = p->bt;
  a.g = p->g;
  a.dw = dw;
  a.ms = p->ms, a.nb = p->nb, a.hs = p->hs, a.ws = p->ws, a.hb = p->hb, a.wb = p->wb;
  a.r = d.r, a.s = d.s;
  a.stride_h = d.stride_h, a.stride_w = d.stride_w, a.pad_h = d.pad_h, a.pad_w = d.pad_w;
  a.dil_h = d.dil_h, a.dil_w = d.dil_w;
  a.ksplit = p->ksplit;
  if (p->groups > 1) {
    a.groups = p->groups;
    a.img0 = 0;
    a.nimg = d.n;
    if (launch_wgrad_grouped(a, d.dtype, stream) != hipSuccess) {
      (void)hipGetLastError();
      return HUGE2_ERR_HIP;
    }
    return HUGE2_OK;
  }
  const long long hws = (long long)p->hs * p->ws;
  a.gather_ib = p->gather_ib;
  a.bt_phase = p->bt_phase;
  a.hr = p->hr;
  a.sh_min = p->sh_min;
  division_magic((uint32_t)p->ws, &a.ws_mul, &a.ws_shift);
  division_magic((uint32_t)hws, &a.hws_mul, &a.hws_shift);
  division_magic((uint32_t)(p->hr * p->ws), &a.hrws_mul, &a.hrws_shift);
  a.direct_out = p->direct_out;
  a.direct = p->direct;
  // chunks in order: the first writes the fp32 gradient, the rest add to it
  for (int img0 = 0; img0 < d.n; img0 += p->chunk) {
    a.img0 = img0;
    a.nimg = std::min(p->chunk, d.n - img0);
    a.kp = (int)((a.nimg * hws + 63) / 64 * 64);
    a.accumulate = img0 > 0;
    if (launch_wgrad_stage(a, d.dtype, stream) != hipSuccess ||
        launch_wgrad_gemm(a, d.dtype, stream) != hipSuccess) {
      (void)hipGetLastError();
      return HUGE2_ERR_HIP;
    }
  }
  if (!p->direct_out && launch_wgrad_store(a, d.dtype, stream) != hipSuccess) {
    (void)hipGetLastError();
    return HUGE2_ERR_HIP;
  }
  return HUGE2_OK;
}

huge2_status wgrad_one_shot(const huge2_conv_desc* desc, int transposed, const void* x,
                            const void* dy, void* dw, hipStream_t stream) {
  if (!x || !dy || !dw || dw == x || dw == dy) return HUGE2_ERR_INVALID_ARG;
  huge2_wgrad_plan* p = nullptr;
  huge2_status st = wgrad_create(&p, desc, transposed);
  if (st != HUGE2_OK) return st;
  st = wgrad_execute(p, x, dy, dw, stream);
  if (hipStreamSynchronize(stream) != hipSuccess && st == HUGE2_OK) st = HUGE2_ERR_HIP;
  wgrad_free(p);
  delete p;
  return st;
}

// ---------------------------------------------------------------------------
// Grouped launch of several GEMM plans that read one input.

bool groupable(const huge2_plan* p, const huge2_plan* q) {
  if (!p || !q || p->cfg < 0 || q->cfg < 0 || p->inner || q->inner || p->ztile || q->ztile ||
      p->rowphase || q->rowphase || p->quad || q->quad || p->colphase || q->colphase ||
      p->staged || q->staged ||
      p->ksplit != 1 || q->ksplit != 1 || p->h_works.empty() || q->h_works.empty())
    return false;
  const huge2_conv_desc &a = p->desc, &b = q->desc;
  return a.n == b.n && a.c_in == b.c_in && a.h == b.h && a.w == b.w && a.c_out == b.c_out &&
         a.layout == b.layout && a.dtype == b.dtype && a.activation == b.activation &&
         p->ho == q->ho && p->wo == q->wo && p->cfg == q->cfg && p->cin_pad == q->cin_pad &&
         p->cout_pad == q->cout_pad && p->c_stride == q->c_stride && p->x_bytes == q->x_bytes &&
         p->wp_bytes == q->wp_bytes && p->bias_div == q->bias_div &&
         p->bias_mod == q->bias_mod && a.r == b.r && a.s == b.s;
}

// Image of the first pixel of a work (the segment's pixels are image-major).
int work_image(const SegDev& sg, const WorkDev& w) {
  if (sg.ptab >= 0) return w.m0 / std::max(1, sg.per_img);
  const int64_t per_img = (int64_t)sg.qn_w * sg.qn_h * sg.nphase;
  return (int)(w.m0 / std::max<int64_t>(1, per_img));
}

huge2_status group_create(huge2_group** out, const huge2_plan* const* plans, int count,
                          hipStream_t stream) {
  if (!out) return HUGE2_ERR_INVALID_ARG;
  *out = nullptr;
  if (!plans || count < 1 || count > kMaxGroup) return HUGE2_ERR_INVALID_ARG;
  for (int i = 0; i < count; ++i)
    if (!plans[i]) return HUGE2_ERR_INVALID_ARG;
  for (int i = 0; i < count; ++i)
    if (!groupable(plans[0], plans[i])) return HUGE2_ERR_UNSUPPORTED;
  const huge2_plan* p0 = plans[0];
  const int64_t kc = tile_kb(p0->cfg) / elem_size(p0->desc.dtype);
  const int64_t cblocks = (p0->cin_pad + kc - 1) / kc;
  std::vector<SegDev> segs;
  std::vector<TapDev> taps;
  std::vector<uint32_t> ptab;
  struct Item {
    int img;
    int64_t cost;
    WorkDev w;
  };
  std::vector<Item> items;
  for (int i = 0; i < count; ++i) {
    const huge2_plan* p = plans[i];
    const int s0 = (int)segs.size(), t0 = (int)taps.size(), q0 = (int)ptab.size();
    for (SegDev sd : p->h_segs) {
      sd.plan = i;
      sd.tap_begin += t0;
      if (sd.ptab >= 0) sd.ptab += q0;
      segs.push_back(sd);
    }
    taps.insert(taps.end(), p->h_taps.begin(), p->h_taps.end());
    ptab.insert(ptab.end(), p->h_ptab.begin(), p->h_ptab.end());
    for (WorkDev w : p->h_works) {
      const int img = work_image(p->h_segs[w.seg], w);
      w.seg += s0;
      w.tap_begin += t0;
      items.push_back({img, (int64_t)w.tap_count * cblocks + 2, w});
    }
  }
  // image-major: the eight XCDs take contiguous runs of the list, so the
  // workgroups that run together on one XCD share one image's input rows in
  // its L2; inside an image the costliest works first, so that the
  // dispatcher's greedy placement balances the compute units
  std::stable_sort(items.begin(), items.end(), [](const Item& a, const Item& b) {
    if (a.img != b.img) return a.img < b.img;
    return a.cost > b.cost;
  });
  std::vector<WorkDev> works;
  works.reserve(items.size());
  for (const Item& it : items) works.push_back(it.w);
  huge2_group* g = new (std::nothrow) huge2_group();
  if (!g) return HUGE2_ERR_ALLOC;
  g->count = count;
  for (int i = 0; i < count; ++i) g->plans[i] = plans[i];
  g->n_works = (int)works.size();
  // Enough works for two workgroups on every compute unit: the 4-wave form of
  // the pipelined tile (the same 128 x 256 works and packed weights, a K
  // block of 64 bytes), two of which share a compute unit and hide each
  // other's barriers and epilogues.
  g->cfg = p0->cfg;
  const int64_t kc4 = tile_kb(TILE_P3_128x256_W4) / elem_size(p0->desc.dtype);
  if (p0->cfg == TILE_P3_128x256 && env_int("HUGE2_TILE", -1) < 0 &&
      g->n_works >= 2 * kComputeUnits && p0->cin_pad % kc4 == 0)
    g->cfg = TILE_P3_128x256_W4;
  if (g->cfg == p0->cfg) {
    std::snprintf(g->kernel_name, sizeof(g->kernel_name), "%s", p0->kernel_name);
  } else {
    const TileShape& t = kTiles[g->cfg];
    std::snprintf(g->kernel_name, sizeof(g->kernel_name), "phase_gemm3_kernel %dx%d w%d k%d%s", t.bm,
                  t.bn, t.pw * t.cw, t.ksplit, std::strstr(p0->kernel_name, " listed") ? " listed" : "");
  }
  const size_t seg_b = segs.size() * sizeof(SegDev), tap_b = taps.size() * sizeof(TapDev);
  const size_t work_b = works.size() * sizeof(WorkDev), ptab_b = ptab.size() * sizeof(uint32_t);
  const size_t meta_b = seg_b + tap_b + work_b + ptab_b;
  if (fault("alloc") || hipMalloc(&g->meta, meta_b) != hipSuccess) {
    (void)hipGetLastError();
    delete g;
    return HUGE2_ERR_ALLOC;
  }
  g->d_segs = (SegDev*)g->meta;
  g->d_taps = (TapDev*)((char*)g->meta + seg_b);
  g->d_works = (WorkDev*)((char*)g->meta + seg_b + tap_b);
  g->d_ptab = ptab_b ? (const uint32_t*)((char*)g->meta + seg_b + tap_b + work_b) : nullptr;
  std::vector<char> host(meta_b);
  std::memcpy(host.data(), segs.data(), seg_b);
  if (tap_b) std::memcpy(host.data() + seg_b, taps.data(), tap_b);
  std::memcpy(host.data() + seg_b + tap_b, works.data(), work_b);
  if (ptab_b) std::memcpy(host.data() + seg_b + tap_b + work_b, ptab.data(), ptab_b);
  bool ok = !fault("launch") &&
            hipMemcpyAsync(g->meta, host.data(), meta_b, hipMemcpyHostToDevice, stream) == hipSuccess;
  if (ok) ok = hipStreamSynchronize(stream) == hipSuccess;
  if (!ok) {
    (void)hipGetLastError();
    (void)hipFree(g->meta);
    delete g;
    return HUGE2_ERR_HIP;
  }
  *out = g;
  return HUGE2_OK;
}

huge2_status group_execute(const huge2_group* g, const void* x, const float* const* bias,
                           void* const* y, hipStream_t stream) {
  if (!g || !x || !y) return HUGE2_ERR_INVALID_ARG;
  for (int i = 0; i < g->count; ++i)
    if (!y[i] || y[i] == x) return HUGE2_ERR_INVALID_ARG;
  if (fault("launch")) return HUGE2_ERR_HIP;
  const huge2_plan* p = g->plans[0];
  const huge2_conv_desc& d = p->desc;
  GemmArgs a;
  std::memset(&a, 0, sizeof(a));
  a.x = x;
  for (int i = 0; i < g->count; ++i) {
    a.wp[i] = g->plans[i]->wp;
    a.bias[i] = bias ? bias[i] : nullptr;
    a.y[i] = y[i];
  }
  a.bias_div = p->bias_div;
  a.bias_mod = p->bias_mod;
  a.act = d.activation;
  a.ksplit = 1;
  a.segs = g->d_segs;
  a.taps = g->d_taps;
  a.works = g->d_works;
  a.ptab = g->d_ptab;
  a.n_works = g->n_works;
  a.n = d.n;
  a.h = d.h;
  a.w = d.w;
  a.cin = p->c_stride;
  a.ks = d.s;
  a.x_bytes = (uint32_t)p->x_bytes;
  a.wp_bytes = (uint32_t)p->wp_bytes;
  a.cin_pad = p->cin_pad;
  a.cout = d.c_out;
  a.cout_pad = p->cout_pad;
  a.ho = p->ho;
  a.wo = p->wo;
  if (launch_phase_gemm(a, d.dtype, g->cfg, d.layout == HUGE2_NCHW, stream) != hipSuccess) {
    (void)hipGetLastError();
    return HUGE2_ERR_HIP;
  }
  return HUGE2_OK;
}

}  // namespace

extern "C" {

const char* huge2_status_str(huge2_status status) {
  switch (status) {
    case HUGE2_OK: return "HUGE2_OK";
    case HUGE2_ERR_INVALID_ARG: return "HUGE2_ERR_INVALID_ARG";
    case HUGE2_ERR_UNSUPPORTED: return "HUGE2_ERR_UNSUPPORTED";
    case HUGE2_ERR_ALLOC: return "HUGE2_ERR_ALLOC";
    case HUGE2_ERR_HIP: return "HUGE2_ERR_HIP";
  }
  return "HUGE2_ERR_UNKNOWN";
}

huge2_status huge2_output_shape(const huge2_conv_desc* desc, int32_t transposed, int32_t* h_out,
                                int32_t* w_out) {
  if (!h_out || !w_out || (transposed != 0 && transposed != 1)) return HUGE2_ERR_INVALID_ARG;
  huge2_status st = validate_desc(desc, transposed != 0);
  if (st == HUGE2_ERR_UNSUPPORTED) st = HUGE2_OK;  // the shape itself is well defined
  if (st != HUGE2_OK) return st;
  int ho, wo;
  output_dims(*desc, transposed != 0, &ho, &wo);
  *h_out = ho;
  *w_out = wo;
  return HUGE2_OK;
}

huge2_status huge2_dgrad_output_padding(const huge2_conv_desc* conv_desc, int32_t* op_h,
                                        int32_t* op_w) {
  if (!op_h || !op_w) return HUGE2_ERR_INVALID_ARG;
  huge2_status st = validate_desc(conv_desc, false);
  if (st == HUGE2_ERR_UNSUPPORTED) st = HUGE2_OK;  // the shape itself is well defined
  if (st != HUGE2_OK) return st;
  const huge2_conv_desc& d = *conv_desc;
  int ho, wo;
  if (!output_dims(d, false, &ho, &wo)) return HUGE2_ERR_INVALID_ARG;
  // the transposed conv of an ho x wo input reaches (ho-1)*s - 2p + d(r-1) + 1
  *op_h = d.h - ((ho - 1) * d.stride_h - 2 * d.pad_h + d.dil_h * (d.r - 1) + 1);
  *op_w = d.w - ((wo - 1) * d.stride_w - 2 * d.pad_w + d.dil_w * (d.s - 1) + 1);
  return HUGE2_OK;
}

huge2_status huge2_plan_create(huge2_plan** out, const huge2_conv_desc* desc, int32_t transposed,
                               const void* w, void* hip_stream) {
  try {
    return create_impl(out, desc, transposed, w, (hipStream_t)hip_stream, Mem());
  } catch (...) {
    return HUGE2_ERR_ALLOC;
  }
}

huge2_status huge2_plan_execute(const huge2_plan* plan, const void* x, const float* bias, void* y,
                                void* hip_stream) {
  try {
    return execute_impl(plan, x, bias, y, (hipStream_t)hip_stream);
  } catch (...) {
    return HUGE2_ERR_HIP;
  }
}

huge2_status huge2_plan_stage_input(const huge2_plan* plan, const void* x, void* hip_stream) {
  try {
    return stage_impl(plan, x, (hipStream_t)hip_stream);
  } catch (...) {
    return HUGE2_ERR_HIP;
  }
}

huge2_status huge2_plan_run_gemm(const huge2_plan* plan, const void* x, const float* bias, void* y,
                                 void* hip_stream) {
  try {
    return gemm_impl(plan, x, bias, y, (hipStream_t)hip_stream);
  } catch (...) {
    return HUGE2_ERR_HIP;
  }
}

const char* huge2_plan_kernel(const huge2_plan* plan) {
  if (!plan) return "";
  return plan->kernel_name;
}

int32_t huge2_plan_stages_input(const huge2_plan* plan) {
  if (!plan) return -1;
  return plan->staged ? 1 : 0;
}

huge2_status huge2_plan_destroy(huge2_plan* plan) {
  if (!plan) return HUGE2_OK;
  free_buffers(plan);
  delete plan;
  return HUGE2_OK;
}

huge2_status huge2_conv2d_transpose(const huge2_conv_desc* desc, const void* x, const void* w,
                                    const float* bias, void* y, void* hip_stream) {
  try {
    return one_shot(desc, 1, x, w, bias, y, (hipStream_t)hip_stream);
  } catch (...) {
    return HUGE2_ERR_ALLOC;
  }
}

huge2_status huge2_conv2d_transpose_noalloc(const huge2_conv_desc* desc, const void* x,
                                            const void* w, const float* bias, void* y,
                                            void* hip_stream) {
  try {
    return one_shot_noalloc(desc, x, w, bias, y, (hipStream_t)hip_stream);
  } catch (...) {
    return HUGE2_ERR_HIP;
  }
}

huge2_status huge2_conv2d_dilated(const huge2_conv_desc* desc, const void* x, const void* w,
                                  const float* bias, void* y, void* hip_stream) {
  try {
    return one_shot(desc, 0, x, w, bias, y, (hipStream_t)hip_stream);
  } catch (...) {
    return HUGE2_ERR_ALLOC;
  }
}

huge2_status huge2_plan_describe(const huge2_conv_desc* desc, int32_t transposed,
                                 int32_t class_split, huge2_segment* segs, int32_t seg_cap,
                                 int32_t* n_segs, huge2_tap* taps, int32_t tap_cap,
                                 int32_t* n_taps) {
  if (!n_segs || !n_taps || seg_cap < 0 || tap_cap < 0 || (seg_cap > 0 && !segs) ||
      (tap_cap > 0 && !taps) || (transposed != 0 && transposed != 1) || class_split < 0 ||
      class_split > 2)
    return HUGE2_ERR_INVALID_ARG;
  huge2_status st = validate_desc(desc, transposed != 0);
  if (st != HUGE2_OK) return st;
  try {
    const int cfg = choose_cfg(*desc, transposed != 0, 2);
    PlanShape shape;
    if (!build_shape(*desc, transposed != 0, class_split, tile_bm(cfg), &shape))
      return HUGE2_ERR_INVALID_ARG;
    *n_segs = (int32_t)shape.segs.size();
    *n_taps = (int32_t)shape.taps.size();
    for (int i = 0; i < seg_cap && i < *n_segs; ++i) segs[i] = shape.segs[i];
    for (int i = 0; i < tap_cap && i < *n_taps; ++i) taps[i] = shape.taps[i];
    return HUGE2_OK;
  } catch (...) {
    return HUGE2_ERR_ALLOC;
  }
}

huge2_status huge2_plan_macs(const huge2_conv_desc* desc, int32_t transposed, int64_t* nonzero_macs,
                             int64_t* issued_macs) {
  if (!nonzero_macs || !issued_macs || (transposed != 0 && transposed != 1))
    return HUGE2_ERR_INVALID_ARG;
  huge2_status st = validate_desc(desc, transposed != 0);
  if (st != HUGE2_OK) return st;
  try {
    if (desc->groups > 1) {
      PlanShape shape;
      if (!build_shape(*desc, transposed != 0, 2, 128, &shape)) return HUGE2_ERR_INVALID_ARG;
      *nonzero_macs = *issued_macs = shape.nonzero_macs / desc->groups;
      return HUGE2_OK;
    }
    ZArgs z;
    int64_t z_issued = 0;
    RpArgs rp;
    QArgs q;
    // the same form choices, in the same order, as plan creation
    huge2_conv_desc dd;
    int bias_div, bias_mod, prod_rs;
    product_form(*desc, transposed != 0, &dd, &bias_div, &bias_mod, &prod_rs);
    huge2_conv_desc d1;
    if (two_pass_shape(dd, transposed != 0, &d1) || gather_shape(dd, transposed != 0, &d1)) {
      int64_t nz1 = 0;
      PlanShape shape;
      if (!build_shape(dd, transposed != 0, 2, 128, &shape)) return HUGE2_ERR_INVALID_ARG;
      *nonzero_macs = shape.nonzero_macs;
      return huge2_plan_macs(&d1, transposed != 0 ? 1 : 0, &nz1, issued_macs);
    }
    CpArgs cpa;
    if (ztile_shape(dd, transposed != 0, &z, &z_issued) ||
        colphase_shape(dd, transposed != 0, &cpa, &z_issued) ||
        rowphase_shape(dd, transposed != 0, &rp, &z_issued) ||
        quad_shape(dd, transposed != 0, &q, &z_issued)) {
      PlanShape shape;
      if (!build_shape(*desc, true, 2, 128, &shape)) return HUGE2_ERR_INVALID_ARG;
      *nonzero_macs = shape.nonzero_macs;
      *issued_macs = z_issued;
      return HUGE2_OK;
    }
    PlanShape shape;
    ListedShape ls;
    bool listed = false;
    const int cfg = plan_gemm_shape(dd, transposed != 0, &shape, &listed, &ls);
    if (cfg < 0) return HUGE2_ERR_INVALID_ARG;
    const int bm = tile_bm(cfg), bn = tile_bn(cfg);
    const int bk = tile_kb(cfg) / elem_size(dd.dtype);
    const int64_t cin_pad = round_up(dd.c_in, bk);
    const int64_t ntn = round_up(dd.c_out, bn) / bn;
    *nonzero_macs = shape.nonzero_macs;
    *issued_macs = listed ? ls.issued_rows_taps * bn * ntn * cin_pad
                          : shape.tile_taps * bm * bn * ntn * cin_pad;
    return HUGE2_OK;
  } catch (...) {
    return HUGE2_ERR_ALLOC;
  }
}

huge2_status huge2_wgrad_plan_create(huge2_wgrad_plan** out, const huge2_conv_desc* desc,
                                     int32_t transposed) {
  try {
    return wgrad_create(out, desc, transposed);
  } catch (...) {
    return HUGE2_ERR_ALLOC;
  }
}

huge2_status huge2_wgrad_execute(const huge2_wgrad_plan* plan, const void* x, const void* dy,
                                 void* dw, void* hip_stream) {
  try {
    return wgrad_execute(plan, x, dy, dw, (hipStream_t)hip_stream);
  } catch (...) {
    return HUGE2_ERR_ALLOC;
  }
}

huge2_status huge2_wgrad_plan_destroy(huge2_wgrad_plan* plan) {
  if (!plan) return HUGE2_OK;
  wgrad_free(plan);
  delete plan;
  return HUGE2_OK;
}

huge2_status huge2_conv2d_transpose_wgrad(const huge2_conv_desc* desc, const void* x,
                                          const void* dy, void* dw, void* hip_stream) {
  try {
    return wgrad_one_shot(desc, 1, x, dy, dw, (hipStream_t)hip_stream);
  } catch (...) {
    return HUGE2_ERR_ALLOC;
  }
}

huge2_status huge2_conv2d_dilated_wgrad(const huge2_conv_desc* desc, const void* x,
                                        const void* dy, void* dw, void* hip_stream) {
  try {
    return wgrad_one_shot(desc, 0, x, dy, dw, (hipStream_t)hip_stream);
  } catch (...) {
    return HUGE2_ERR_ALLOC;
  }
}

huge2_status huge2_group_create(huge2_group** out, const huge2_plan* const* plans, int32_t count,
                                void* hip_stream) {
  try {
    return group_create(out, plans, count, (hipStream_t)hip_stream);
  } catch (...) {
    return HUGE2_ERR_ALLOC;
  }
}

const char* huge2_group_kernel(const huge2_group* group) {
  return group ? group->kernel_name : "";
}

huge2_status huge2_group_execute(const huge2_group* group, const void* x, const float* const* bias,
                                 void* const* y, void* hip_stream) {
  try {
    return group_execute(group, x, bias, y, (hipStream_t)hip_stream);
  } catch (...) {
    return HUGE2_ERR_HIP;
  }
}

huge2_status huge2_group_destroy(huge2_group* group) {
  if (!group) return HUGE2_OK;
  const hipError_t e = hipFree(group->meta);  // waits for work that may still read it
  delete group;
  return e == hipSuccess ? HUGE2_OK : HUGE2_ERR_HIP;
}

}  // extern "C"
