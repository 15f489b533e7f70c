// kernels.hpp -- device-side data structures and kernel launchers of libhuge2.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace huge2 {

// A segment as the GEMM kernel reads it (mirrors huge2_segment, plus the
// flattened GEMM height m_total = n * nphase_h * nphase_w * qn_h * qn_w).
// Pixel index j of the segment decomposes, fastest first, as
// (a_w in [0,qn_w), a_h in [0,qn_h), image n, phase index in [0, nphase_h*nphase_w)).
struct SegDev {
  int32_t phase0_h, phase0_w, nphase_w, m_total;
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
  // qn_w, qn_h, n (images) and nphase_w of the pixel decomposition
  uint32_t div_mul[4];
  uint32_t div_shift[4];
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

// One workgroup's job: GEMM tile (m0, n0) of segment seg.
struct WorkDev {
  int32_t seg, m0, n0, pad;
};

struct GemmArgs {
  const void* x;      // input, channel-contiguous: [n][h][w][cin]
  const void* wp;     // packed weights: [slot][cout_pad][cin_pad]
  const float* bias;  // [cout] or null
  void* y;            // output, NCHW or NHWC
  const SegDev* segs;
  const TapDev* taps;
  const WorkDev* works;
  uint32_t x_bytes, wp_bytes;  // buffer extents (< 2^31)
  int32_t n_works;
  int32_t n, h, w, cin;       // cin: channels per input pixel, a multiple of 16 bytes
  int32_t cin_pad;            // K stride of the packed weights (multiple of the K block)
  int32_t cout, cout_pad;
  int32_t ho, wo;
  int32_t ks;  // kernel width s: weight slot of tap (kh, kw) = kh * ks + kw
};

// Tile configurations of the phase GEMM kernel: BM pixels x BN output
// channels per workgroup, PW x CW waves (64 threads each), KB bytes of K per
// LDS stage.
// depth: stages of global loads in flight ahead of the MFMAs (1 or 2; each
// in-flight stage costs one register buffer).
// wg_per_cu: workgroups of this shape that fit on one compute unit at once
// (the tighter of the register and LDS limits; the same for both dtypes and
// layouts), used by the host's schedule model.
struct TileShape {
  int bm, bn, pw, cw, kb, depth, wg_per_cu;
};
constexpr TileShape kTiles[] = {
    {128, 128, 2, 2, 128, 2, 2},  // 0
    {256, 32, 4, 1, 128, 2, 1},   // 1  narrow: few output channels
    {64, 128, 1, 4, 128, 2, 2},   // 2
    {256, 128, 2, 2, 128, 2, 1},  // 3
    {128, 256, 2, 2, 128, 2, 1},  // 4
    {256, 256, 2, 4, 128, 2, 1},  // 5  8 waves
    {256, 128, 4, 2, 128, 2, 1},  // 6  8 waves
    {128, 256, 2, 4, 128, 2, 1},  // 7  8 waves
    {128, 128, 4, 2, 128, 2, 2},  // 8  8 waves
    {256, 256, 2, 2, 128, 1, 1},  // 9  4 waves of 128 x 128
    {128, 32, 4, 1, 64, 2, 6},    // 10 narrow, small LDS footprint
    {256, 32, 4, 1, 64, 2, 3},    // 11 narrow, small LDS footprint
    {64, 128, 1, 4, 64, 2, 5},    // 12 small LDS footprint
    {128, 128, 2, 2, 64, 2, 3},   // 13 small LDS footprint
    {256, 128, 2, 2, 128, 1, 1},  // 14 4 waves of 128 x 64, one buffer
    {128, 256, 2, 2, 128, 1, 1},  // 15 4 waves of 64 x 128, one buffer
};
constexpr int kComputeUnits = 256;  // MI355X
constexpr int TILE_COUNT = (int)(sizeof(kTiles) / sizeof(kTiles[0]));
inline int tile_bm(int cfg) { return kTiles[cfg].bm; }
inline int tile_bn(int cfg) { return kTiles[cfg].bn; }
inline int tile_threads(int cfg) { return kTiles[cfg].pw * kTiles[cfg].cw * 64; }
inline int tile_kb(int cfg) { return kTiles[cfg].kb; }
// LDS bytes of a configuration (two stages of BM + BN rows, 16-byte row pad)
inline int tile_lds(int cfg) { return 2 * (kTiles[cfg].bm + kTiles[cfg].bn) * (kTiles[cfg].kb + 16); }
constexpr int kMaxBlockK_bytes = 128;  // largest K block per stage: 64 bf16 or 32 fp32

// dtype: 0 fp32, 1 bf16; nchw_out selects the output layout.
hipError_t launch_phase_gemm(const GemmArgs& a, int dtype, int cfg, bool nchw_out,
                             hipStream_t stream);

// Gather w into [slot = kh*s + kw][cout_pad][cin_pad] (zero padded).
// transposed: w is [cin][cout][r][s]; otherwise [cout][cin][r][s].
hipError_t launch_pack_weights(const void* w, void* wp, int dtype, bool transposed, int cin,
                               int cout, int r, int s, int cin_pad, int cout_pad,
                               hipStream_t stream);

// Re-layout the input into [n][h*w][c_stride] with zero channel padding.
// nchw: source is NCHW; otherwise NHWC with cin channels per pixel.
hipError_t launch_stage_input(const void* x, void* xs, int dtype, bool nchw, int n, int cin,
                              int hw, int c_stride, hipStream_t stream);

}  // namespace huge2
