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
  int32_t pad0;
};

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
};

// Tile configurations of the phase GEMM kernel.
enum TileCfg : int32_t {
  TILE_128x128 = 0,  // 128 pixels x 128 output channels, 4 waves as 2x2
  TILE_256x32 = 1,   // 256 pixels x 32 output channels, 4 waves as 4x1
  TILE_64x128 = 2,   // 64 pixels x 128 output channels, 4 waves as 1x4
  TILE_256x128 = 3,  // 256 pixels x 128 output channels, 4 waves as 2x2
  TILE_128x256 = 4,  // 128 pixels x 256 output channels, 4 waves as 2x2
  TILE_256x256_W8 = 5,  // 256 x 256, 8 waves as 2x4
  TILE_256x128_W8 = 6,  // 256 x 128, 8 waves as 4x2
  TILE_128x256_W8 = 7,  // 128 x 256, 8 waves as 2x4
  TILE_128x128_W8 = 8,  // 128 x 128, 8 waves as 4x2
  TILE_COUNT = 9
};
int tile_bm(int cfg);
int tile_bn(int cfg);
int tile_threads(int cfg);
constexpr int kBlockK_bytes = 128;  // K block per LDS stage: 64 bf16 or 32 fp32

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
