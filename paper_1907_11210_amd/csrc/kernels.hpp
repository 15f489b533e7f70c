// kernels.hpp -- device-side data structures and kernel launchers of libhuge2.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace huge2 {

// A segment as the GEMM kernel reads it (mirrors huge2_segment, plus the
// flattened GEMM height m_total = n * nphase_h * nphase_w * qn_h * qn_w).
// Pixel index j of the segment decomposes, fastest first, as
// (a_w in [0,qn_w), a_h in [0,qn_h), phase index in [0, nphase), image n):
// the pixels of one image are contiguous, so that the workgroups that run at
// the same time read a compact region of the input.
struct SegDev {
  int32_t phase0_h, phase0_w, nphase_w, nphase, m_total;
  int32_t out_step_h, out_step_w, q0_h, q0_w;
  int32_t qn_h, qn_w, in0_h, in0_w;
  int32_t in_dphase_h, in_dphase_w, in_step_h, in_step_w;
  int32_t tap_begin, tap_count;
  int32_t exact;  // 1: every tap reads inside the input for every pixel (no bounds tests)
  // tap_ap = 1: the taps are the product of two arithmetic progressions, tap
  // t = (th, tw) = (t / ntw, t % ntw) with kernel tap (kh0 + th*dkh, kw0 + tw*dkw)
  // at input offset (off0_h + th*doff_h, off0_w + tw*doff_w); the kernel then
  // derives each tap from two counters instead of reading the tap list
  int32_t tap_ap;
  int32_t ntw, off0_h, doff_h, off0_w, doff_w, kh0, dkh, kw0, dkw;
  // floor(v / d) = (v * mul) >> shift for 0 <= v < 2^31, for the divisors
  // qn_w, qn_h, nphase (phases) and nphase_w of the pixel decomposition
  uint32_t div_mul[4];
  uint32_t div_shift[4];
  // ptab >= 0: a listed segment.  Pixel m is image m / per_img (divisor 2 of
  // the magic numbers above) and entry ptab + m mod per_img of the pixel
  // table, (oh << 16) | ow, reading input (in0_h + oh, in0_w + ow) + tap
  // offset (a stride-1 dilated conv with in0 = -pad).
  int32_t ptab, per_img;
  int32_t plan;  // entry of the per-plan pointers of GemmArgs (0 outside a group)
};

// Multiplier and shift of the division by d (1 <= d < 2^31) for dividends
// below 2^31: floor(v / d) = (v * mul) >> shift with l = ceil(log2 d),
// mul = floor(2^(31+l) / d) + 1, shift = 31 + l (Granlund and Montgomery,
// "Division by invariant integers using multiplication", 1994).
inline void division_magic(uint32_t d, uint32_t* mul, uint32_t* shift) {
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  *mul = (uint32_t)(((1ull << (31 + l)) / d) + 1);
  *shift = 31 + l;
}

// One tap of a segment: the packed sub-kernel block (slot = kh*s + kw) and
// the input offset it reads at.
struct TapDev {
  int32_t slot, off_h, off_w, pad;
};
constexpr int kMaxLdsTaps = 64;  // taps per segment staged in LDS (more: scalar loads)

// One workgroup's job: GEMM tile of pixels [m0, m1) (at most BM of them) and
// output channels from n0 of segment seg, over the input channel blocks of K
// slice ks (of GemmArgs::ksplit), with the taps [tap_begin, tap_begin +
// tap_count) of the tap list (the segment's taps, or a listed tile's own).
// When those taps are the product of two arithmetic progressions (ap_ntw >
// 0), tap t = (th, tw) = (t / ap_ntw, t % ap_ntw) is kernel tap (ap_kh0 +
// th*ap_dkh, ap_kw0 + tw*ap_dkw) at input offset (ap_off0_h + th*ap_doff_h,
// ap_off0_w + tw*ap_doff_w), so that a kernel can step through them with two
// counters and no memory reads.
struct WorkDev {
  int32_t seg, m0, m1, n0, ks, tap_begin, tap_count;
  int32_t ap_ntw, ap_kh0, ap_dkh, ap_kw0, ap_dkw, ap_off0_h, ap_doff_h, ap_off0_w, ap_doff_w;
};

constexpr int kMaxGroup = 8;  // plans of one grouped launch (huge2_group)
struct GemmArgs {
  const void* x;  // input, channel-contiguous: [n][h][w][cin]
  // Per plan of a grouped launch (entry 0 alone for a single plan); a
  // segment's `plan` field selects the entry.
  const void* wp[kMaxGroup];     // packed weights: [slot][cout_pad][cin_pad]
  // [cout / bias_div] or null: column ch takes bias[ch / bias_div], or with
  // bias_mod > 0 bias[(ch / bias_div) % bias_mod]
  const float* bias[kMaxGroup];
  void* y[kMaxGroup];            // output, NCHW or NHWC
  const SegDev* segs;
  const TapDev* taps;
  const WorkDev* works;
  const uint32_t* ptab;        // pixel table of listed segments
  uint32_t x_bytes, wp_bytes;  // buffer extents (< 2^31)
  int32_t n_works;
  int32_t n, h, w, cin;       // cin: channels per input pixel, a multiple of 16 bytes
  int32_t cin_pad;            // K stride of the packed weights (multiple of the K block)
  int32_t cout, cout_pad;
  int32_t ho, wo;
  int32_t ks;  // kernel width s: weight slot of tap (kh, kw) = kh * ks + kw
  int32_t bias_div, bias_mod;
  // K split across workgroups: ksplit > 1 writes each slice's fp32 partial
  // tile (no bias, no activation) to part + slice * part_stride, in the
  // output's layout; splitk_reduce then sums the slices in order
  int32_t ksplit;
  float* part;
  uint32_t part_stride;
  int act;           // huge2_activation, applied after the bias
};

// Tile configurations of the phase GEMM kernel: BM pixels x BN output
// channels per workgroup, PW x CW waves (64 threads each), KB bytes of K per
// LDS stage.
// depth: stages of global loads in flight ahead of the MFMAs (1 or 2; each
// in-flight stage costs one register buffer).
// wg_per_cu: workgroups of this shape that fit on one compute unit at once
// (the tighter of the register and LDS limits; the same for both dtypes and
// layouts), used by the host's schedule model.
// kind 0: both operands through LDS, PW x CW waves of (BM/PW) x (BN/CW).
// kind 1: split-wave form, the pixel tile through LDS, CW waves each loading
//         BN/CW weight rows itself (PW = 1) from lane-ordered packed weights.
// kind 3: the same tile and packing, pipelined over three LDS stage buffers
//         (phase_gemm3_kernel; depth = 10 x weight stages in flight + pixel
//         stages held in registers).
// ksplit (split-wave kinds): K groups of PW x CW waves per workgroup, each
// over its own share of the input-channel blocks, summed in LDS at the end.
struct TileShape {
  int bm, bn, pw, cw, kb, depth, wg_per_cu, kind, ksplit = 1;
};
// Every configuration here is one that the planner picks for some shape
// (choose_cfg and the split-K rewrite in capi.cpp).
enum TileCfg {
  TILE_128x128 = 0,      // two-operand LDS, 8 waves
  TILE_64x128 = 1,       // two-operand LDS, 4 waves
  TILE_128x32 = 2,       // narrow: few output channels, small LDS footprint
  TILE_SW_64x128 = 3,    // split-wave: 4 waves of 64 x 32 channels
  TILE_SW_64x256 = 4,    // split-wave: 4 waves of 64 x 64 channels
  TILE_SW_32x256 = 5,    // split-wave: 4 waves of 32 x 64 channels
  TILE_SW_64x128_K2 = 6,   // as TILE_SW_64x128, two K groups (8 waves)
  TILE_SW_128x128_K2 = 7,  // split-wave: 4 waves of 128 x 32 channels, two K groups
  TILE_SW_128x256 = 8,   // split-wave: 8 waves of 128 x 32 channels
  TILE_P3_128x256 = 9,   // pipelined split-wave: 8 waves of 128 x 32 channels
  TILE_P3_128x256_W4 = 10,  // pipelined split-wave: 4 waves of 128 x 64 channels, 64-byte K
  TILE_P3_128x128 = 11,  // pipelined split-wave: 4 waves of 128 x 32 channels
};
constexpr TileShape kTiles[] = {
    {128, 128, 4, 2, 128, 2, 2, 0},     // TILE_128x128
    {64, 128, 1, 4, 128, 2, 2, 0},      // TILE_64x128
    {128, 32, 4, 1, 64, 2, 6, 0},       // TILE_128x32
    {64, 128, 1, 4, 128, 4, 3, 1},      // TILE_SW_64x128
    {64, 256, 1, 4, 128, 3, 2, 1},      // TILE_SW_64x256
    {32, 256, 1, 4, 128, 4, 2, 1},      // TILE_SW_32x256
    {64, 128, 1, 4, 128, 4, 1, 1, 2},   // TILE_SW_64x128_K2
    {128, 128, 1, 4, 128, 3, 1, 1, 2},  // TILE_SW_128x128_K2
    {128, 256, 1, 8, 128, 3, 1, 1, 1},  // TILE_SW_128x256
    {128, 256, 1, 8, 128, 32, 1, 3, 1},  // TILE_P3_128x256
    {128, 256, 1, 4, 64, 32, 2, 3, 1},   // TILE_P3_128x256_W4
    {128, 128, 1, 4, 128, 32, 2, 3, 1},  // TILE_P3_128x128
};
// A split-K plan may switch from the two-K-group 64 x 128 tile to its
// one-group form after the work list and the weight packing were laid out for
// the first: both must share the tile, the K block and the packed layout.
static_assert(kTiles[TILE_SW_64x128].bm == kTiles[TILE_SW_64x128_K2].bm &&
                  kTiles[TILE_SW_64x128].bn == kTiles[TILE_SW_64x128_K2].bn &&
                  kTiles[TILE_SW_64x128].kb == kTiles[TILE_SW_64x128_K2].kb &&
                  kTiles[TILE_SW_64x128].kind == kTiles[TILE_SW_64x128_K2].kind,
              "the split-K tile switch keeps the work list and the packing");
constexpr int kComputeUnits = 256;  // MI355X
constexpr int TILE_COUNT = (int)(sizeof(kTiles) / sizeof(kTiles[0]));
// K bytes of one block of the lane-ordered weight packing (split-wave and
// pipelined kinds).  Inside a block, MFMA K chunk c takes bytes
// [16c, 16c + 16) of the block's first half in lanes 0-31 and of its second
// half in lanes 32-63; a K stage of KB bytes is KB / kPackKB such blocks.  One
// packing for every K block size, so that plans of different tiles share it.
constexpr int kPackKB = 64;
// Byte offset, inside a K stage, of MFMA K chunk c for lane half `half`.
__host__ __device__ constexpr int pack_chunk_byte(int c, int half) {
  return (c / (kPackKB / 32)) * kPackKB + half * (kPackKB / 2) + (c % (kPackKB / 32)) * 16;
}
inline int tile_bm(int cfg) { return kTiles[cfg].bm; }
inline int tile_bn(int cfg) { return kTiles[cfg].bn; }
inline int tile_threads(int cfg) {
  return kTiles[cfg].pw * kTiles[cfg].cw * (kTiles[cfg].kind ? kTiles[cfg].ksplit : 1) * 64;
}
inline int tile_kb(int cfg) { return kTiles[cfg].kb; }
// LDS bytes of a configuration (two stages of the rows that go through LDS,
// 16-byte row pad)
inline int tile_lds(int cfg) {
  const TileShape& t = kTiles[cfg];
  const int rows = t.kind == 0 ? t.bm + t.bn : t.bm;
  return (t.kind == 3 ? 3 : 2) * rows * (t.kb + 16);
}
constexpr int kMaxBlockK_bytes = 256;  // largest K block per stage: 128 bf16 or 64 fp32

// dtype: 0 fp32, 1 bf16; nchw_out selects the output layout.
hipError_t launch_phase_gemm(const GemmArgs& a, int dtype, int cfg, bool nchw_out,
                             hipStream_t stream);

// Gather w into [slot = kh*s + kw][cout_pad][cin_pad] (zero padded), in the
// layout the tile kind reads.
// transposed: w is [cin][cout][r][s]; otherwise [cout][cin][r][s].
// lane_kb: 0 for the K-contiguous layout; the stage size KB of a kind-1 tile
// for its lane-ordered layout (see pack_weights_kernel).
// prod_rs > 0: w is a transposed conv's [cin][cout / prod_rs][prod_rs] (its
// taps last) packed as a 1x1 conv to cout columns ordered tap-major (column
// t * (cout / prod_rs) + k): the NHWC form of the 1x1-input product.
hipError_t launch_pack_weights(const void* w, void* wp, int dtype, bool transposed, int cin,
                               int cout, int r, int s, int cin_pad, int cout_pad, int lane_kb,
                               hipStream_t stream, int prod_rs = 0);

// All-taps form of a transposed conv with few output channels (NCHW, bf16,
// c_out * r * s <= 64): workgroup (image, block of `ob` output rows) holds
// input rows [i_lo, i_lo + tr) (i_lo from the block's first output row) and
// input columns [j_lo, j_lo + tcw) in LDS, channel-contiguous per pixel
// (kZtileRowB bytes: 64 channels + pad), one 64-channel pass at a time in two
// buffers; Z (tile pixels x 64 fp32) then reuses the same LDS.
constexpr int kZtileZPitch = 65;      // Z row pitch, floats
constexpr int kZtileMaxPixels = 256;  // tile pixels (tr * tcw)
constexpr int kZtileRowB = 144;       // LDS bytes per tile pixel and pass
constexpr int kZtileLds = 2 * kZtileMaxPixels * kZtileRowB;  // two pass buffers, then Z
constexpr int kZtileMaxItems = 2;     // input items (pixel pair x 8 channels) per thread and pass
constexpr int kZtileMaxStride = 4;    // phases per axis of the tap tables
constexpr int kZtileMaxTaps = 8;      // kernel taps per axis
constexpr int kZtilePhaseTaps = 4;    // taps per axis reaching one output phase
constexpr int kZtileThreads = 512;    // 8 waves: two per SIMD hide each other's latency
struct ZArgs {
  const void* x;
  const void* wp;  // packed K-contiguous weights [slot][cout_pad][cin_pad]
  const float* bias;
  void* y;
  uint32_t x_bytes;
  int n, cin, h, w, cout, r, s, cin_pad, cout_pad;
  int stride_h, stride_w, pad_h, pad_w, dil_h, dil_w, ho, wo;
  int ob;        // output rows per workgroup
  int tr, tcw;   // tile rows, tile columns
  int j_lo;      // first tile column (input coordinate)
  int cchunk;    // K padding unit of the packed weights (channels)
  // per axis (0 = h, 1 = w) and phase rho = (o + pad) mod stride: the taps
  // k with (rho - k*dil) divisible by the stride, and delta = (rho - k*dil) /
  // stride, so that output o reads input (o + pad) div stride + delta
  int8_t tap_n[2][kZtileMaxStride];
  int max_th, max_tw;  // largest tap count of a phase, per axis
  int8_t tap_k[2][kZtileMaxStride][kZtileMaxTaps];
  int8_t tap_d[2][kZtileMaxStride][kZtileMaxTaps];
  int act;           // huge2_activation, applied after the bias
  int nhwc;          // 1: x and y NHWC (c_in a multiple of 8), else NCHW
};
hipError_t launch_ztile(const ZArgs& a, int dtype, hipStream_t stream);

// Output-stationary form for large strides and few channels (NCHW, bf16,
// dilation 1, c_in, c_out <= 32, kernel size <= 2 * stride): workgroup
// (image, row phase, block of rb rows of that phase) runs every column
// phase's small GEMM, collects its output rows in LDS and writes them whole.
constexpr int kRpCh = 32;                  // channel padding of input and weights
constexpr int kRpMaxW = 64;                // input width
constexpr int kRpMaxRb = 8;                // rows of one row phase per workgroup
constexpr int kRpOutElems = 48 * 1024;     // LDS output rows (bf16 elements)
constexpr int kRpThreads = 512;            // 8 waves: many column phases in flight
constexpr int kRpMaxColPhasesPerWave = 4;  // stride_w <= 8 waves x 4
struct RpArgs {
  const void* x;
  const void* wp;  // packed K-contiguous weights [slot][32][32]
  const float* bias;
  void* y;
  int n, cin, h, w, cout, r, s;
  int stride_h, stride_w, pad_h, pad_w, ho, wo;
  int rb;       // rows of one row phase per workgroup
  int qblocks;  // row blocks per (image, row phase)
  int nq;       // q_w slots per column phase in LDS (stride_w * nq a multiple of 8)
  int act;           // huge2_activation, applied after the bias
};
hipError_t launch_rowphase(const RpArgs& a, hipStream_t stream);

// Column-phase form for a column stride of 32 (NCHW, bf16, dilation 1, at
// most 32 input channels, kernel width <= 64, kernel height <= 2 * row
// stride): the 32 column phases rho_w of an output block are the 32 rows of
// one MFMA tile, so that its results are 32 consecutive output elements of
// one output row.  Wave (output channel k, image n, row phase rho_h) runs
//   C[rho_w][(Q, Q_w)] = sum over (th, tw, c) of
//       Wp[k][rho_h][rho_w][(th, tw, c)] * X[n][c][Q - th][Q_w - tw]
// (K = 4 taps x cp channels, cp = c_in padded to 8) with the input of image
// n staged in LDS (channel-contiguous, one pixel of zeros around it).  Each
// column's 32 results are output row rho_h + s_h*Q - pad_h, columns 32*Q_w -
// pad_w + [0, 32): they go to an LDS copy of kCpRows output rows, which are
// then written whole, 16 bytes per lane.
constexpr int kCpWaves = 4;              // row phases per workgroup
constexpr int kCpRows = 8;               // output rows per wave assembled in LDS at a time
constexpr int kCpMaxLds = 64 * 1024;     // LDS bytes of the staged input and the output rows
struct CpArgs {
  const void* x;
  const void* wp;  // [c_out][s_h][kblk][64 lanes][8 bf16] (pack_colphase_kernel)
  const float* bias;
  void* y;
  int n, cin, h, w, cout, r, s;
  int stride_h, pad_h, pad_w, ho, wo;
  int cp;        // c_in padded to 8
  int qw_lo, nqw;  // Q_w range of every row phase
  int act;
  // floor(v / d) = (v * mul) >> shift (division_magic) for d = w + 2, h + 2,
  // nqw, cp / 8, cin and w / 8: the kernel's index arithmetic has no integer
  // division
  uint32_t dv_mul[6], dv_shift[6];
};
hipError_t launch_colphase(const CpArgs& a, hipStream_t stream);
hipError_t launch_pack_colphase(const void* w, void* wp, int cin, int cout, int r, int s,
                                int stride_h, int cp, hipStream_t stream);

// All four phases per workgroup for the stride-2, 4x4, padding-1 transposed
// conv (NCHW, bf16): every phase has 2 x 2 taps with input offsets in
// [-1, 1] and the input's pixel grid.  Workgroup: 64 input positions (ni
// images x qbh rows x the full width w) x 32*nch output channels, 8 waves.
// Weights in the lane order of 128-byte K stages (pack_weights_kernel with
// lane_kb = 128).
constexpr int kQuadThreads = 512;
constexpr int kQuadPix = 64;         // input positions per workgroup (np = 2; 128 with np = 4)
constexpr int kQuadRowB = 128;       // LDS bytes per halo pixel: 64 channels (slot-swizzled; + 16-byte pad unswizzled)
constexpr int kQuadHaloRows = 200;   // halo pixels per LDS tile: ni * (qbh + 2) * (w + 2)
constexpr int kQuadMaxPieces = 2;    // input items (pixel pair x 8 channels) per thread and K block
struct QArgs {
  const void* x;     // input, NCHW or (nhwc) NHWC
  const void* wp;    // packed weights [slot][cout_pad/32][cin/64][4][64 lanes][16 bytes]
  const float* bias;
  void* y;           // output, 2h x 2w, the input's layout
  uint32_t x_bytes, wp_bytes;
  int n, cin, h, w, cout, cout_pad;
  int ni, qbh;       // images and input rows per workgroup (ni * qbh * w = 32 * np)
  int np;            // 32-position MFMA blocks per wave: 2, or 4 (one 32-channel block per wave)
  // 32-channel blocks and K groups per workgroup; the 8 waves are 4 phases x
  // (nch = 2, ks = 1: a 32-channel block each | nch = 1, ks = 2: a K group
  // each | nch = 2, ks = 2: a K group each, both 32-channel blocks per wave)
  int nch, ks;
  int igroups, hblocks, ntiles;  // grid = ntiles x igroups x hblocks
  int depth;         // weight stages in flight (2 or 4)
  // per phase (2 * rho_h + rho_w) and tap (2 * th + tw): weight slot kh*4+kw
  // and input offsets: output (2q_h + rho_h, 2q_w + rho_w) reads input q + (dh, dw)
  int8_t slot[4][4], dh[4][4], dw[4][4];
  int act;           // huge2_activation, applied after the bias
  int nhwc;          // 1: NHWC (c_out a multiple of 8: 16-byte output pieces)
};
hipError_t launch_quad(const QArgs& a, hipStream_t stream);

// Grouped (and depthwise) convolution, direct: one thread per output
// element, in the output's layout order.  Transposed (transposed = 1): output
// o with o + pad = i*stride + m*dil takes input i through kernel tap m (the
// taps of o's phase, section 3.1); dilated / strided: input o*stride - pad +
// m*dil.  The sum runs over the taps and the input channels of the output
// channel's group, in fp32, then bias, activation and rounding.
struct GrArgs {
  const void* x;
  const void* w;   // the plan's copy of the weight, the caller's layout
  const float* bias;
  void* y;
  int n, cin, h, w_, cout, r, s, stride_h, stride_w, pad_h, pad_w, dil_h, dil_w, ho, wo;
  int groups, transposed, nhwc, act;
};
hipError_t launch_grouped(const GrArgs& a, int dtype, hipStream_t stream);

// y[i] = act(bias[ch(i) / bias_div] + sum over s < ksplit, in order, of
// part[s * stride + i]) in the dtype; ch(i) = (i / hw) % cout for NCHW, i %
// cout for NHWC.
struct SplitKArgs {
  const float* part;
  const float* bias;
  void* y;
  uint32_t stride, total;
  int ksplit, cout, hw, nchw, bias_div, bias_mod, act;
};
hipError_t launch_splitk_reduce(const SplitKArgs& a, int dtype, hipStream_t stream);

// Second pass of the two-pass all-taps form of a transposed conv: z holds,
// per input pixel, every kernel tap's products, z[n][(k*r + m)*s + q][ih][iw]
// = sum_c x[n][c][ih][iw] * w[c][k][m][q] (fp32, NCHW); the output gathers
// y[n][k][oh][ow] = act(bias[k] + sum over the taps (m, q), in order, with
// oh + pad_h - m*dil_h = ih*stride_h and ow + pad_w - q*dil_w = iw*stride_w
// inside the input, of z[n][(k*r + m)*s + q][ih][iw]) (fp32, NCHW).
struct CombArgs {
  const float* z;
  const float* bias;
  float* y;
  int n, h, w, cout, r, s, stride_h, stride_w, pad_h, pad_w, dil_h, dil_w, ho, wo, act;
};
hipError_t launch_taps_combine(const CombArgs& a, hipStream_t stream);

// Weight gradient (training, section 3.2.3).  With the "small" tensor S on
// the tap's pixel grid and the "big" tensor B read at position
// q*stride - pad + k*dil of that grid (transposed conv: S = x, B = dy; strided
// or dilated conv: S = dy, B = x), dw[m][n][tap] = sum over (image, q) of
// S[m][q] * B[n][tap position of q].  For one chunk of images, with
// k = local image * hws + q (zero up to kp, a multiple of 64):
//  - St[m][k] = S[image][m][q], read in place by the GEMM (direct) or
//    staged by wgrad_stage;
//  - Bt, the untangled copies of the big tensor (zero outside): one row per
//    (n, tap) (wgrad_stage or wgrad_gather), or phase planes that the taps of
//    one kernel column and row phase share (bt_phase, wgrad_gather);
//  - wgrad_gemm: G[split][m][n * taps + tap] (fp32) = (or +=) St Bt^T over
//    the split's K range, all taps in one GEMM on MFMA (or, direct_out, dw
//    itself);
//  - wgrad_store: dw = the sum over the splits (in a fixed order), in the
//    dtype.
struct WgArgs {
  const void* sm;  // small tensor [n][ms][hs][ws] (NCHW)
  const void* bg;  // big tensor [n][nb][hb][wb]
  void* st;       // [ms][kp]
  void* bt;       // [nb][taps][kp]: row (n, tap)
  float* g;       // [ksplit][ms][nb][taps]: each K slice in dw's own layout
  void* dw;       // [ms][nb][r][s]
  int img0, nimg;  // image chunk
  int ms, nb, hs, ws, hb, wb, r, s;
  int stride_h, stride_w, pad_h, pad_w, dil_h, dil_w;
  int kp;          // padded K of the chunk (multiple of 64)
  int accumulate;  // 0: G = product, 1: G += product
  int ksplit;      // K slices of the GEMM, each with its own fp32 slice of G
  int groups;      // > 1: grouped conv (wgrad_grouped_kernel; st, bt and g unused)
  int gather_ib;   // > 0: Bt through LDS, workgroups of gather_ib images (wgrad_gather_kernel)
  uint32_t ws_mul, ws_shift;  // floor(v / ws) = (v * ws_mul) >> ws_shift (division_magic)
  // the GEMM writes dw itself, rounded once (one K slice and one image
  // chunk: no fp32 gradient and no store)
  int direct_out;
  // the GEMM reads its St operand in place from the small tensor (hs*ws a
  // multiple of 64: every K stage lies in one image's channel plane) and St
  // is not staged
  int direct;
  uint32_t hws_mul, hws_shift;  // floor(v / (hs*ws)) (division_magic)
  // Bt in phase planes (bt_phase): row (n, plane = ph * s + kw) holds, per
  // image of the chunk, hr rows of ws elements, element (i', j) = big[n][(i'
  // + sh_min) * stride_h + ph][j * stride_w + kw * dil_w - pad_w] (zero
  // outside).  Tap (kh, kw), whose big row for small row i is (i + sh) *
  // stride_h + ph with kh * dil_h - pad_h = sh * stride_h + ph, reads plane
  // (ph, kw) from row i + sh - sh_min: the taps that differ only in their row
  // shift share one copy, and a row shift is a whole-row offset in K.
  int bt_phase;
  int hr, sh_min;
  uint32_t hrws_mul, hrws_shift;  // floor(v / (hr*ws)) (division_magic)
  int g_taps, g_s;                // the layer's taps and kernel width (the
                                  // GEMM launch folds r, s into nb)
};
// Output tile of the weight-gradient GEMM (square, channels of the small x
// the large tensor): 128 x 128 when both channel counts reach 128, else 64.
inline int wgrad_tile(int ms, int nb) { return ms >= 128 && nb >= 128 ? 128 : 64; }
hipError_t launch_wgrad_stage(const WgArgs& a, int dtype, hipStream_t stream);
hipError_t launch_wgrad_gemm(const WgArgs& a, int dtype, hipStream_t stream);
hipError_t launch_wgrad_store(const WgArgs& a, int dtype, hipStream_t stream);
// K slices from which the store adds them with a workgroup per 64 entries
// (four waves over the slices) rather than a thread per entry
constexpr int kWgSplitStore = 16;
hipError_t launch_wgrad_grouped(const WgArgs& a, int dtype, hipStream_t stream);
// Images per workgroup of the LDS gather for a chunk (0: the plain staging
// kernel gathers Bt): each workgroup holds that many big-tensor planes, as
// many as fit and still leave about four workgroups per compute unit.
constexpr int kWgGatherLds = 32 * 1024;
inline int wgrad_gather_images(int hs, int ws, int hb, int wb, int esz, int nimg, int nb) {
  const long long plane = (long long)hb * wb * esz;
  if ((hs * ws) % 8 != 0 || plane > kWgGatherLds) return 0;
  long long ib = (long long)nimg * nb / 1024;
  if (ib > kWgGatherLds / plane) ib = kWgGatherLds / plane;
  if (ib > nimg) ib = nimg;
  return (int)(ib < 1 ? 1 : ib);
}

// Re-layout the input into [n][h*w][c_stride] with zero channel padding.
// nchw: source is NCHW; otherwise NHWC with cin channels per pixel.
hipError_t launch_stage_input(const void* x, void* xs, int dtype, bool nchw, int n, int cin,
                              int hw, int c_stride, hipStream_t stream);

// Gather form of a conv with few input channels: every output pixel's
// receptive field, xs[n][oh*wo + ow][(c*r + m)*s + q] = x[n][c][oh*stride_h -
// pad_h + m*dil_h][ow*stride_w - pad_w + q*dil_w] (NCHW x; zero outside the
// input and for j >= cin*r*s up to c_stride), in the channel-contiguous
// layout the phase GEMM reads.
struct GatherArgs {
  const void* x;
  void* xs;
  int n, cin, h, w, r, s, stride_h, stride_w, pad_h, pad_w, dil_h, dil_w, ho, wo, c_stride;
};
hipError_t launch_gather_taps(const GatherArgs& a, int dtype, hipStream_t stream);

}  // namespace huge2
