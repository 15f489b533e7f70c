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
  int32_t tap_begin, tap_count, pad0, pad1;
};

// One tap of a segment: the packed sub-kernel block (slot = kh*s + kw) and
// the input offset it reads at.
struct TapDev {
  int32_t slot, off_h, off_w, pad;
};

// One workgroup's job: GEMM tile (m0, n0) of segment seg.
struct WorkDev {
  int32_t seg, m0, n0, pad;
};

struct GemmArgs {
  const void* x;      // input: [n][c][h][w] (NCHW) or [n][h][w][c] (NHWC)
  const void* wp;     // packed weights: [slot][cout_pad][cin_pad]
  const float* bias;  // [cout] or null
  void* y;            // output, NCHW or NHWC
  const SegDev* segs;
  const TapDev* taps;
  const WorkDev* works;
  int32_t n_works;
  int32_t n, h, w, cin;
  int32_t cin_pad;            // K stride of the packed weights (multiple of the K block)
  int32_t cout, cout_pad;
  int32_t ho, wo;
};

// Tile configurations of the phase GEMM kernel.
enum TileCfg : int32_t {
  TILE_128x128 = 0,  // 128 pixels x 128 output channels, 4 waves as 2x2
  TILE_256x32 = 1,   // 256 pixels x 32 output channels, 4 waves as 4x1
  TILE_64x128 = 2,   // 64 pixels x 128 output channels, 4 waves as 1x4
  TILE_COUNT = 3
};
int tile_bm(int cfg);
int tile_bn(int cfg);
constexpr int kBlockK_bytes = 64;  // K block per LDS stage: 32 bf16 or 16 fp32

// How the GEMM kernel gathers its input tile.
enum InputMode : int32_t {
  IN_NHWC_VEC = 0,   // NHWC, cin a multiple of 16 bytes: 16-byte loads per pixel
  IN_NCHW = 1,       // NCHW: per-element loads, consecutive lanes on consecutive pixels
  IN_NHWC_ELEM = 2,  // NHWC with a ragged channel count: per-element loads
};

// dtype: 0 fp32, 1 bf16.  The output layout follows the input layout
// (IN_NCHW -> NCHW output, otherwise NHWC).
hipError_t launch_phase_gemm(const GemmArgs& a, int dtype, int cfg, int in_mode,
                             hipStream_t stream);

// Gather w into [slot = kh*s + kw][cout_pad][cin_pad] (zero padded).
// transposed: w is [cin][cout][r][s]; otherwise [cout][cin][r][s].
hipError_t launch_pack_weights(const void* w, void* wp, int dtype, bool transposed, int cin,
                               int cout, int r, int s, int cin_pad, int cout_pad,
                               hipStream_t stream);

}  // namespace huge2
