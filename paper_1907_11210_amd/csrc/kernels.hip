// kernels.hip -- gfx950 (CDNA4) kernels of libhuge2.
//
//  phase_gemm_kernel   the untangled phase convolution (section 3.2.1 of the
//                      paper): per segment, an implicit GEMM
//                        Y[pixel, k] = sum_{tap, c} X[pixel + tap offset, c] * Wp[tap][k][c]
//                      on MFMA (fp32: v_mfma_f32_32x32x2_f32, bf16:
//                      v_mfma_f32_32x32x16_bf16, fp32 accumulation), with
//                      double-buffered LDS staging and an epilogue that writes
//                      each pixel straight to its interleaved output position
//                      (the scatter of section 3.1: disjoint, no atomics).
//  pack_weights_kernel the per-tap sub-kernel blocks (the N x C matrix of each
//                      kernel position, section 3.2.1), K-contiguous.
//  stage_*_kernel      input re-layout to channel-contiguous pixels.
#include <algorithm>
#include <type_traits>

#include "kernels.hpp"

namespace huge2 {

typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;

constexpr int cmax(int a, int b) { return a > b ? a : b; }
constexpr int gcd_c(int a, int b) { return b == 0 ? a : gcd_c(b, a % b); }
constexpr int lcm3(int a, int b, int c) {
  return (a / gcd_c(a, b) * b) / gcd_c(a / gcd_c(a, b) * b, c) * c;
}
// f(integral_constant<int, u>) for u = 0 .. N-1, unrolled at compile time.
template <int N, int I = 0, typename F>
__device__ __forceinline__ void unroll_stages(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>());
    unroll_stages<N, I + 1>(f);
  }
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// 16-byte store of output data that nothing in the kernel reads back, with
// the non-temporal (streaming) cache policy.
__device__ __forceinline__ void store_stream16(void* p, uint4 v) {
  const u32x4 t = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(t, (u32x4*)p);
}

// Workgroups are dealt to the 8 XCDs round-robin (id mod 8).  Map them so
// that each XCD runs one contiguous run of the work list: neighbouring
// tiles share input rows and weight blocks, which then stay in that XCD's L2.
__device__ __forceinline__ int xcd_remap(int b, int g) {
  const int g8 = (g + 7) >> 3, r = g & 7, x = b & 7, y = b >> 3;
  if (r == 0 || x < r) return x * g8 + y;
  return r * g8 + (x - r) * (g8 - 1) + y;
}

// The epilogue's elementwise function (huge2_activation): 0 none, 1 max(v, 0),
// 2 tanh(v).  act is uniform over the launch.
__device__ __forceinline__ float activate(float v, int act) {
  return act == 1 ? fmaxf(v, 0.f) : act == 2 ? tanhf(v) : v;
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  // v_cvt_pk_bf16_f32: round to nearest even, NaN stays a (quiet) NaN
  return __builtin_bit_cast(uint16_t, (__bf16)f);
}

// Two floats to bf16 (round to nearest even) in one 32-bit word, lo in the
// low half: one v_cvt_pk_bf16_f32 with both sources.
__device__ __forceinline__ uint32_t pack_bf16x2_rne(float lo, float hi) {
  typedef float f2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 b2_t __attribute__((ext_vector_type(2)));
  const f2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, b2_t));
}

// Decomposition of a segment pixel index into image, output and input coordinates.
struct PixelPos {
  int img, oh, ow, ih, iw;
};
// Bias entry of GEMM column ch (the 1x1-input product forms: bias_div
// columns per entry, or entries repeating every bias_mod columns).
__device__ __forceinline__ int bias_index(const GemmArgs& a, int ch) {
  const int bc = ch / a.bias_div;
  return a.bias_mod > 0 ? bc % a.bias_mod : bc;
}
__device__ __forceinline__ uint32_t fast_div(uint32_t v, uint32_t mul, uint32_t shift) {
  return (uint32_t)(((uint64_t)v * mul) >> shift);
}
__device__ __forceinline__ PixelPos pixel_pos(const SegDev& sg, const uint32_t* ptab, int m) {
  PixelPos p;
  uint32_t j = (uint32_t)m;
  if (sg.ptab >= 0) {
    const uint32_t img = fast_div(j, sg.div_mul[2], sg.div_shift[2]);
    const uint32_t e = ptab[sg.ptab + (int)(j - img * (uint32_t)sg.per_img)];
    p.img = (int)img;
    p.oh = (int)(e >> 16);
    p.ow = (int)(e & 0xffffu);
    p.ih = sg.in0_h + p.oh;
    p.iw = sg.in0_w + p.ow;
    return p;
  }
  uint32_t t = fast_div(j, sg.div_mul[0], sg.div_shift[0]);
  const int a_w = (int)(j - t * (uint32_t)sg.qn_w);
  j = t;
  t = fast_div(j, sg.div_mul[1], sg.div_shift[1]);
  const int a_h = (int)(j - t * (uint32_t)sg.qn_h);
  j = t;
  t = fast_div(j, sg.div_mul[2], sg.div_shift[2]);
  const uint32_t iph = j - t * (uint32_t)sg.nphase;
  p.img = (int)t;
  const uint32_t iph_h = fast_div(iph, sg.div_mul[3], sg.div_shift[3]);
  const int iph_w = (int)(iph - iph_h * (uint32_t)sg.nphase_w);
  const int qh = sg.q0_h + a_h, qw = sg.q0_w + a_w;
  p.oh = sg.phase0_h + (int)iph_h + sg.out_step_h * qh;
  p.ow = sg.phase0_w + iph_w + sg.out_step_w * qw;
  p.ih = sg.in0_h + sg.in_dphase_h * (int)iph_h + sg.in_step_h * qh;
  p.iw = sg.in0_w + sg.in_dphase_w * iph_w + sg.in_step_w * qw;
  return p;
}

// Epilogue: bias, rounding, and the scatter of a wave's TP x TC blocks of
// 32 x 32 results (pixels from pix0, output channels from ch0) to the
// interleaved output positions of their phase.  32x32 MFMA result layout:
// lane l holds column l % 32 and rows 8*(r/4) + 4*(l/32) + (r%4), r = 0..15.
// NCHW output puts pixels on the columns (a channel's stores coalesce along
// the lanes); NHWC output puts pixels on the rows.
// sb: bias by output channel (sb[ch], staged in LDS, zeros without bias):
// reading it from global memory between the stores would make every load
// wait for the stores issued before it.
template <bool BF16, bool NCHW_OUT, int TP, int TC>
__device__ __forceinline__ void store_tile(const GemmArgs& a, const SegDev& sg, int m_end, void* y,
                                           const f32x16 (&acc)[TP][TC], int pix0, int ch0,
                                           int lane, const float* sb) {
  const int hw_o = a.ho * a.wo;
  // the bias values are read from LDS up front: an LDS read between the
  // global stores would wait for its own latency element by element
  if constexpr (!NCHW_OUT) {
    float bv[TC];
#pragma unroll
    for (int j = 0; j < TC; ++j) {
      const int ch = ch0 + 32 * j + (lane & 31);
      bv[j] = ch < a.cout ? sb[ch] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < TP; ++i) {
      // the 16 rows' positions before their stores: a table lookup issued
      // behind stores would wait for them (the memory counter is in order)
      int pixr[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = pix0 + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const PixelPos p = pixel_pos(sg, a.ptab, m < m_end ? m : pix0);
        pixr[r] = m < m_end ? (p.img * a.ho + p.oh) * a.wo + p.ow : -1;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int pix = pixr[r];
        if (pix < 0) continue;
#pragma unroll
        for (int j = 0; j < TC; ++j) {
          const int ch = ch0 + 32 * j + (lane & 31);
          if (ch >= a.cout) continue;
          const float v = activate(acc[i][j][r] + bv[j], a.act);
          const size_t off = (size_t)pix * a.cout + ch;
          if constexpr (BF16)
            ((uint16_t*)y)[off] = f32_to_bf16_rne(v);
          else
            ((float*)y)[off] = v;
        }
      }
    }
  } else {
    size_t base[TP];
    bool ok[TP];
#pragma unroll
    for (int i = 0; i < TP; ++i) {
      const int m = pix0 + 32 * i + (lane & 31);
      ok[i] = m < m_end;
      const PixelPos p = pixel_pos(sg, a.ptab, ok[i] ? m : pix0);
      base[i] = (size_t)p.img * a.cout * hw_o + (size_t)p.oh * a.wo + p.ow;
    }
#pragma unroll
    for (int j = 0; j < TC; ++j) {
      float bv[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ch = ch0 + 32 * j + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        bv[r] = ch < a.cout ? sb[ch] : 0.f;
      }
#pragma unroll
      for (int i = 0; i < TP; ++i) {
        if (!ok[i]) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int ch = ch0 + 32 * j + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (ch >= a.cout) continue;
          const float v = activate(acc[i][j][r] + bv[r], a.act);
          const size_t off = base[i] + (size_t)ch * hw_o;
          if constexpr (BF16)
            ((uint16_t*)y)[off] = f32_to_bf16_rne(v);
          else
            ((float*)y)[off] = v;
        }
      }
    }
  }
}

// NHWC bf16 epilogue through LDS, for tiles whose output rows are whole
// 16-byte pieces (C_out a multiple of 8, a 16-byte aligned output).  The
// waves write their results (bias, activation, rounding) into a [BM][BN]
// tile in LDS; then every thread stores 16-byte pieces of output pixel
// rows: in NHWC a pixel's channels are contiguous, so each row of the tile
// is one run of BN * 2 bytes.  lds: at least BM * (2 * BN + 16) bytes, free
// once every wave passed the barrier at the start; row_off: each tile row's
// output pixel index (-1: past the end of the work), in LDS; sb: the tile's
// BN bias values (zeros without bias); wch0: the wave's first channel within
// the tile.
template <int TP, int TC, int BM, int BN, int NT, int ACT>
__device__ __forceinline__ void store_rows_nhwc(const GemmArgs& a, int n0, void* y,
                                                const f32x16 (&acc)[TP][TC], int wch0, int lane,
                                                int tid, char* lds, const int* row_off,
                                                const float* sb) {
  constexpr int PITCH = 2 * BN + 16;  // 16-byte pad: rows 4 apart on other banks
  constexpr int PIECES = 2 * BN / 16;
  constexpr int RSTEP = NT / PIECES;
  constexpr int PASSES = BM / RSTEP;
  static_assert(NT % PIECES == 0 && BM % RSTEP == 0, "epilogue shape");
  float bv[TC];
#pragma unroll
  for (int j = 0; j < TC; ++j) bv[j] = sb[wch0 + 32 * j + (lane & 31)];
  __syncthreads();  // every wave has finished with the stage buffers
#pragma unroll
  for (int i = 0; i < TP; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int px = 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
#pragma unroll
      for (int j = 0; j < TC; ++j) {
        float v = acc[i][j][r] + bv[j];
        if constexpr (ACT == 1) v = fmaxf(v, 0.f);
        if constexpr (ACT == 2) v = tanhf(v);
        *(uint16_t*)(lds + px * PITCH + 2 * (wch0 + 32 * j + (lane & 31))) = f32_to_bf16_rne(v);
      }
    }
  __syncthreads();
  // (streaming stores: the output is not read back by this launch)
  const int piece = tid % PIECES, row0 = tid / PIECES;
  if (n0 + 8 * piece >= a.cout) return;
  uint16_t* const yb = (uint16_t*)y + n0 + 8 * piece;
#pragma unroll
  for (int k = 0; k < PASSES; ++k) {
    const int row = row0 + RSTEP * k;
    const int off = row_off[row];
    if (off >= 0)
      store_stream16(yb + (size_t)off * a.cout, *(const uint4*)(lds + row * PITCH + 16 * piece));
  }
}

// ---------------------------------------------------------------------------
// Phase GEMM.  A workgroup of 256 threads (4 waves) computes a BM x BN tile
// (BM pixels of one segment, BN output channels).  The K loop runs over the
// segment's taps and, per tap, over KB-byte blocks of input channels (one
// "stage").  Each stage holds BM + BN rows of KB bytes in LDS with a 16-byte
// row pad (so that the 16-byte accesses of 8 consecutive rows hit distinct
// banks), double buffered.  Global loads run two stages ahead through two
// register buffers: while the MFMAs consume stage s from LDS, the loads of
// stage s+2 are in flight and stage s+1 is written to the other LDS buffer.
//
// The input is channel-contiguous ([n][h][w][cin], cin a multiple of 16
// bytes).  The tile row of a pixel at a tap is the run of channels
// [cb*KC, cb*KC + KC) of input pixel (ih, iw) = pixel base + tap offset,
// fetched as KB/16 buffer loads of 16 bytes by KB/16 neighbouring lanes.
// Rows outside the input get an out-of-range buffer offset, which the
// hardware returns as zeros: the loads are branch-free, so the compiler can
// keep the next stages' loads in flight while it waits for the current one.
//
// MFMA operands are K-contiguous per lane: lane l reads KB/2 bytes of its
// row at byte offset (KB/2)*(l/32).  The K order inside a stage is permuted
// identically for both operands, which leaves the contraction unchanged:
//   bf16: MFMA t uses row elements [h*KC/2 + 8t, h*KC/2 + 8t + 8), h = l/32
//   fp32: MFMA t uses row element h*KC/2 + t.
// NCHW output puts pixels on MFMA columns (lanes hold consecutive pixels, so
// a channel's stores coalesce); NHWC output puts pixels on MFMA rows (lanes
// hold consecutive channels of a pixel).
template <bool BF16, int BM, int BN, int PWAVES, int CWAVES, int KB, int DEPTH, bool NCHW_OUT>
__global__ __launch_bounds__(PWAVES * CWAVES * 64) void phase_gemm_kernel(GemmArgs a) {
  constexpr int NT = PWAVES * CWAVES * 64;  // threads per workgroup
  constexpr int ESZ = BF16 ? 2 : 4;
  constexpr int KC = KB / ESZ;    // K elements per stage
  constexpr int VE = 16 / ESZ;    // elements per 16-byte chunk
  constexpr int CPR = KB / 16;    // 16-byte chunks per row
  constexpr int ROWB = KB + 16;   // LDS row pitch
  constexpr int WP = BM / PWAVES, WC = BN / CWAVES;
  constexpr int TP = WP / 32, TC = WC / 32;
  constexpr int A_LD = BM * CPR / NT;
  constexpr int B_LD = (BN * CPR + NT - 1) / NT;  // the last may be partial
  constexpr int KSUB = BF16 ? KB / 32 : KB / 8;  // MFMAs per operand pair and stage
  static_assert(BM * CPR % NT == 0, "whole A loads per thread");
  static_assert(TP >= 1 && TC >= 1 && WP % 32 == 0 && WC % 32 == 0, "32x32 MFMA blocks");
  constexpr int STAGE_B = (BM + BN) * ROWB;
  constexpr uint32_t OOB = 0x80000000u;  // beyond every buffer: loads return 0
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE_B];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int work = xcd_remap(blockIdx.x, gridDim.x);
  const WorkDev wk = a.works[work];
  const SegDev sg = a.segs[wk.seg];
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.x, 0, a.x_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t wr =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.wp[sg.plan], 0, a.wp_bytes, 0x00020000);

  // This thread's A-tile rows (pixels) and its 16-byte chunk within a row.
  // Rows past the end of the segment repeat its last pixel: they compute
  // values the epilogue never stores.
  const int chunk = tid % CPR;
  int a_ih[A_LD], a_iw[A_LD];
  uint32_t a_base[A_LD];  // byte offset of (pixel, chunk) at tap offset (0, 0)
#pragma unroll
  for (int i = 0; i < A_LD; ++i) {
    const int m = min(wk.m0 + tid / CPR + (NT / CPR) * i, wk.m1 - 1);
    const PixelPos p = pixel_pos(sg, a.ptab, m);
    a_ih[i] = p.ih;
    a_iw[i] = p.iw;
    // unsigned (wrapping) arithmetic: the tap offset brings it back in range
    a_base[i] = (((uint32_t)p.img * (uint32_t)a.h + (uint32_t)p.ih) * (uint32_t)a.w +
                 (uint32_t)p.iw) * (uint32_t)a.cin * ESZ + (uint32_t)(chunk * VE * ESZ);
  }
  const int ntaps = wk.tap_count;
  const int cblocks = a.cin_pad / KC;
  // this workgroup's K slice of channel blocks, [cb_w0, cb_w1)
  const int cb_w0 = wk.ks * cblocks / a.ksplit, cb_w1 = (wk.ks + 1) * cblocks / a.ksplit;
  const int nsteps = ntaps * (cb_w1 - cb_w0);
  // channels of the last K block that exist (a partial block needs masking)
  const int tail_c = a.cin - (cblocks - 1) * KC;

  __shared__ float s_bias[BN];
  const float* const bias = a.bias[sg.plan];
  for (int t = tid; t < BN; t += NT)
    s_bias[t] = (bias && wk.n0 + t < a.cout) ? bias[bias_index(a, wk.n0 + t)] : 0.f;

  // The segment's taps in LDS: byte delta of the tapped pixel and byte
  // offset of the tap's weight block.
  __shared__ int4 s_taps[kMaxLdsTaps];
  const bool lds_taps = !sg.tap_ap && ntaps <= kMaxLdsTaps;
  if (lds_taps) {
    for (int t = tid; t < ntaps; t += NT) {
      const TapDev tp = a.taps[wk.tap_begin + t];
      s_taps[t] = make_int4((tp.off_h * a.w + tp.off_w) * a.cin * ESZ,
                            (int)((uint32_t)tp.slot * (uint32_t)a.cout_pad * (uint32_t)a.cin_pad * ESZ),
                            tp.off_h, tp.off_w);
    }
  }
  __syncthreads();

  struct Regs {
    uint4 a[A_LD];
    uint4 b[B_LD];
  };
  Regs r0;
  [[maybe_unused]] Regs r1;

  uint32_t voff_b[B_LD];  // per B row: byte offset within a tap's weight block
#pragma unroll
  for (int i = 0; i < B_LD; ++i)
    voff_b[i] = tid + NT * i < BN * CPR
                    ? (uint32_t)(((wk.n0 + tid / CPR + (NT / CPR) * i) * a.cin_pad + chunk * VE) * ESZ)
                    : OOB;

  // Resources with no records: every load through them returns zero.
  const __amdgpu_buffer_rsrc_t xr0 =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.x, 0, 0, 0x00020000);
  const __amdgpu_buffer_rsrc_t wr0 =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.wp[sg.plan], 0, 0, 0x00020000);

  // K order: channel block outer, tap inner, so that the taps of one channel
  // block re-read the same input rows while they are still in cache.  A load
  // past the last stage goes through the empty resources instead of
  // branching around the loads: the load sequence stays the same on every
  // path, which lets the compiler wait only for the stage it stores.
  int ld_tap = 0, ld_cb = cb_w0, ld_th = 0, ld_tw = 0;
  const uint32_t slot_bytes = (uint32_t)a.cout_pad * (uint32_t)a.cin_pad * ESZ;
  auto load_step = [&](Regs& R, bool valid) {
    const __amdgpu_buffer_rsrc_t xs = valid ? xr : xr0;
    const __amdgpu_buffer_rsrc_t ws = valid ? wr : wr0;
    int delta, off_h, off_w;
    uint32_t slot_b;
    if (sg.tap_ap) {
      // the tap from two counters, in scalar registers
      off_h = sg.off0_h + ld_th * sg.doff_h;
      off_w = sg.off0_w + ld_tw * sg.doff_w;
      delta = (off_h * a.w + off_w) * a.cin * ESZ;
      slot_b = (uint32_t)((sg.kh0 + ld_th * sg.dkh) * a.ks + sg.kw0 + ld_tw * sg.dkw) * slot_bytes;
    } else {
      int4 ti;
      if (lds_taps) {
        ti = s_taps[valid ? ld_tap : 0];
      } else {
        const TapDev tp = a.taps[wk.tap_begin + (valid ? ld_tap : 0)];
        ti = make_int4((tp.off_h * a.w + tp.off_w) * a.cin * ESZ, (int)((uint32_t)tp.slot * slot_bytes),
                       tp.off_h, tp.off_w);
      }
      delta = __builtin_amdgcn_readfirstlane(ti.x);
      slot_b = (uint32_t)__builtin_amdgcn_readfirstlane(ti.y);
      off_h = __builtin_amdgcn_readfirstlane(ti.z);
      off_w = __builtin_amdgcn_readfirstlane(ti.w);
    }
    const uint32_t kb = (uint32_t)ld_cb * KB;
    const bool tail = ld_cb == cblocks - 1 && tail_c < KC;
    const bool chunk_out = tail && chunk * VE >= tail_c;
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      uint32_t v = a_base[i] + (uint32_t)delta;
      if (!sg.exact) {
        const int ih = a_ih[i] + off_h, iw = a_iw[i] + off_w;
        const bool in = ((unsigned)ih < (unsigned)a.h) & ((unsigned)iw < (unsigned)a.w);
        v = in ? v : OOB;
      }
      v = chunk_out ? OOB : v;
      R.a[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xs, v, kb, 0));
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i)
      R.b[i] = __builtin_bit_cast(
          uint4, __builtin_amdgcn_raw_buffer_load_b128(ws, voff_b[i], slot_b + kb, 0));
    if (valid) {
      if (++ld_tw == sg.ntw) {
        ld_tw = 0;
        ++ld_th;
      }
      if (++ld_tap == ntaps) {
        ld_tap = 0;
        ld_th = 0;
        ld_tw = 0;
        ++ld_cb;
      }
    }
  };
  auto store_stage = [&](int buf, const Regs& R) {
    char* as = smem + buf * STAGE_B;
    char* bs = as + BM * ROWB;
#pragma unroll
    for (int i = 0; i < A_LD; ++i)
      *(uint4*)(as + (tid / CPR + (NT / CPR) * i) * ROWB + chunk * 16) = R.a[i];
#pragma unroll
    for (int i = 0; i < B_LD; ++i)
      if (BN * CPR % NT == 0 || tid + NT * i < BN * CPR)
        *(uint4*)(bs + (tid / CPR + (NT / CPR) * i) * ROWB + chunk * 16) = R.b[i];
  };

  f32x16 acc[TP][TC];
#pragma unroll
  for (int i = 0; i < TP; ++i)
#pragma unroll
    for (int j = 0; j < TC; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int wp_i = wave % PWAVES, wc_i = wave / PWAVES;
  auto compute = [&](int buf) {
    const char* as = smem + buf * STAGE_B + (wp_i * WP + (lane & 31)) * ROWB + (lane >> 5) * (KB / 2);
    const char* bs = smem + buf * STAGE_B + (BM + wc_i * WC + (lane & 31)) * ROWB + (lane >> 5) * (KB / 2);
    if constexpr (BF16) {
#pragma unroll
      for (int t = 0; t < KSUB; ++t) {
        uint4 fp[TP], fc[TC];
#pragma unroll
        for (int i = 0; i < TP; ++i) fp[i] = *(const uint4*)(as + 32 * i * ROWB + 16 * t);
#pragma unroll
        for (int j = 0; j < TC; ++j) fc[j] = *(const uint4*)(bs + 32 * j * ROWB + 16 * t);
#pragma unroll
        for (int i = 0; i < TP; ++i)
#pragma unroll
          for (int j = 0; j < TC; ++j) {
            const bf16x8 vp = __builtin_bit_cast(bf16x8, fp[i]);
            const bf16x8 vc = __builtin_bit_cast(bf16x8, fc[j]);
            if constexpr (NCHW_OUT)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vc, vp, acc[i][j], 0, 0, 0);
            else
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vp, vc, acc[i][j], 0, 0, 0);
          }
      }
    } else {
#pragma unroll
      for (int t4 = 0; t4 < KSUB / 4; ++t4) {
        uint4 fp[TP], fc[TC];
#pragma unroll
        for (int i = 0; i < TP; ++i) fp[i] = *(const uint4*)(as + 32 * i * ROWB + 16 * t4);
#pragma unroll
        for (int j = 0; j < TC; ++j) fc[j] = *(const uint4*)(bs + 32 * j * ROWB + 16 * t4);
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int i = 0; i < TP; ++i)
#pragma unroll
            for (int j = 0; j < TC; ++j) {
              const uint32_t bp = e == 0 ? fp[i].x : e == 1 ? fp[i].y : e == 2 ? fp[i].z : fp[i].w;
              const uint32_t bc = e == 0 ? fc[j].x : e == 1 ? fc[j].y : e == 2 ? fc[j].z : fc[j].w;
              const float vp = __uint_as_float(bp), vc = __uint_as_float(bc);
              if constexpr (NCHW_OUT)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(vc, vp, acc[i][j], 0, 0, 0);
              else
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(vp, vc, acc[i][j], 0, 0, 0);
            }
      }
    }
  };

  // Main loop, unrolled by two so that the two register buffers alternate
  // statically; an odd stage count is padded with one all-zero stage.
  // Invariant at the top of each half: LDS buffer (s & 1) holds stage s and
  // the other register buffer is receiving stage s+1.
  const int nsteps2 = (nsteps + 1) & ~1;
  if (nsteps2 > 0) {
    if constexpr (DEPTH == 2) {
      load_step(r0, true);
      store_stage(0, r0);
      load_step(r0, 1 < nsteps);
      __syncthreads();
      for (int s = 0; s < nsteps2; s += 2) {
        load_step(r1, s + 2 < nsteps);
        compute(0);  // s < nsteps always
        store_stage(1, r0);
        __syncthreads();
        load_step(r0, s + 3 < nsteps);
        if (s + 1 < nsteps) compute(1);  // the padding step of an odd count has no MFMAs
        store_stage(0, r1);
        __syncthreads();
      }
    } else {
      // one register buffer: the loads of stage s+1 overlap the MFMAs of stage s
      load_step(r0, true);
      store_stage(0, r0);
      __syncthreads();
      for (int s = 0; s < nsteps2; s += 2) {
        load_step(r0, s + 1 < nsteps);
        compute(0);
        store_stage(1, r0);
        __syncthreads();
        load_step(r0, s + 2 < nsteps);
        if (s + 1 < nsteps) compute(1);
        store_stage(0, r0);
        __syncthreads();
      }
    }
  }

  if (a.ksplit > 1) {
    store_tile<false, NCHW_OUT, TP, TC>(a, sg, wk.m1, a.part + (size_t)wk.ks * a.part_stride, acc,
                                        wk.m0 + wp_i * WP, wk.n0 + wc_i * WC, lane, s_bias - wk.n0);
  } else {
    store_tile<BF16, NCHW_OUT, TP, TC>(a, sg, wk.m1, a.y[sg.plan], acc, wk.m0 + wp_i * WP,
                                       wk.n0 + wc_i * WC, lane, s_bias - wk.n0);
  }
}

// ---------------------------------------------------------------------------
// Phase GEMM, split-wave form.  The W waves of a workgroup split its BM x BN
// tile along one dimension only.  The operand every wave needs (SHARE_A: the
// BM pixel rows; otherwise the BN weight rows) goes through LDS, written once
// and read once per wave per stage; each wave loads its own slice of the
// other operand straight from global memory into registers, already in the
// MFMA lane layout (lane l: row l % 32, bytes [(l/32)*KB/2, (l/32+1)*KB/2)
// of the stage).  Per K element, LDS then moves RS*(W+1) rows' bytes for
// 2*BM*BN flops, against (BM+BN) + W*(wave rows + wave columns) rows in the
// form above, which is what bounds the MFMA rate at small wave tiles.
// DEPTH register buffers hold the stages in flight; the loop is unrolled by
// U = lcm(DEPTH, 2) so that every buffer index is a compile-time constant.
template <bool BF16, int BM, int BN, int W, int KB, int DEPTH, bool SHARE_A, int KS, bool NCHW_OUT>
__global__ __launch_bounds__(W * 64 * KS) void phase_gemm2_kernel(GemmArgs a) {
  constexpr int NTA = W * 64 * KS;  // threads of the workgroup
  constexpr int NT = W * 64;        // threads of one K group
  constexpr int ESZ = BF16 ? 2 : 4;
  constexpr int KC = KB / ESZ;    // K elements per stage
  constexpr int VE = 16 / ESZ;    // elements per 16-byte chunk
  constexpr int CPR = KB / 16;    // 16-byte chunks per row and stage
  constexpr int HC = CPR / 2;     // chunks per lane half
  constexpr int ROWB = KB + 16;   // LDS row pitch
  constexpr int RS = SHARE_A ? BM : BN;        // rows through LDS
  constexpr int RD = (SHARE_A ? BN : BM) / W;  // rows each wave loads itself
  constexpr int TS = RS / 32, TD = RD / 32;
  constexpr int TP = SHARE_A ? TS : TD, TC = SHARE_A ? TD : TS;
  constexpr int S_LD = (RS * CPR + NT - 1) / NT;  // shared-operand loads per thread
  constexpr int U = DEPTH == 3 ? 6 : (DEPTH == 1 ? 2 : DEPTH);
  static_assert(RD % 32 == 0 && RS % 32 == 0 && HC >= 1, "32-row blocks, whole lane halves");
  static_assert(!SHARE_A || KB % kPackKB == 0, "K stages of whole packing blocks");
  static_assert(DEPTH >= 2 && DEPTH <= 4, "two to four stages in flight");
  constexpr int STAGE_B = RS * ROWB;
  constexpr uint32_t OOB = 0x80000000u;
  // KS K groups of W waves each run the pipeline below on their own range of
  // channel blocks, with their own LDS buffers; group 1 hands its partial sums
  // to group 0 through LDS at the end (a fixed order: the result does not
  // depend on timing).
  constexpr int ACC_B = KS > 1 ? W * 64 * TP * TC * 16 * 4 : 0;
  constexpr int SMEM_B = KS * 2 * STAGE_B > ACC_B ? KS * 2 * STAGE_B : ACC_B;
  __shared__ __attribute__((aligned(16))) char smem_all[SMEM_B];

  // wave indices are wave-uniform: keep them in scalar registers
  const int wave_all = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63, grp = KS > 1 ? wave_all / W : 0;
  const int wave = wave_all - grp * W;                       // within the K group
  const int tid = (int)threadIdx.x - grp * NT;
  char* const smem = smem_all + grp * 2 * STAGE_B;
  const int half = lane >> 5, row32 = lane & 31;
  const int work = xcd_remap(blockIdx.x, gridDim.x);
  const WorkDev wk = a.works[work];
  const SegDev sg = a.segs[wk.seg];
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.x, 0, a.x_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t wr =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.wp[sg.plan], 0, a.wp_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t xr0 =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.x, 0, 0, 0x00020000);
  const __amdgpu_buffer_rsrc_t wr0 =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.wp[sg.plan], 0, 0, 0x00020000);

  // Pixel rows this thread loads: the shared rows (SHARE_A, S_LD of them, as
  // chunk tid % CPR) or its wave's own rows (TD of them, as lane half).
  constexpr int NPIX = SHARE_A ? S_LD : TD;
  int p_ih[NPIX], p_iw[NPIX];
  uint32_t p_base[NPIX];
  const int s_chunk = tid % CPR;
#pragma unroll
  for (int i = 0; i < NPIX; ++i) {
    const int r = SHARE_A ? tid / CPR + (NT / CPR) * i : wave * RD + 32 * i + row32;
    const int m = min(wk.m0 + r, wk.m1 - 1);
    const PixelPos p = pixel_pos(sg, a.ptab, m);
    p_ih[i] = p.ih;
    p_iw[i] = p.iw;
    const uint32_t byte_in_row = SHARE_A ? (uint32_t)(s_chunk * 16) : (uint32_t)(half * (KB / 2));
    p_base[i] = (((uint32_t)p.img * (uint32_t)a.h + (uint32_t)p.ih) * (uint32_t)a.w +
                 (uint32_t)p.iw) * (uint32_t)a.cin * ESZ + byte_in_row;
  }
  // Weight rows (output channels) this thread loads, byte offset in a tap block.
  constexpr int NW = SHARE_A ? TD : S_LD;
  uint32_t w_off[NW];
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    if (SHARE_A) {
      // lane-ordered weights: 32-channel block (n0 + wave*RD)/32 + i
      w_off[i] = (uint32_t)(((wk.n0 + wave * RD) / 32 + i) * 32 * a.cin_pad * ESZ + lane * 16);
    } else {
      const int r = tid / CPR + (NT / CPR) * i;
      w_off[i] = tid + NT * i < RS * CPR
                     ? (uint32_t)(((wk.n0 + r) * a.cin_pad) * ESZ + s_chunk * 16)
                     : OOB;
    }
  }

  const int ntaps = wk.tap_count;
  const int cblocks = a.cin_pad / KC;
  // this workgroup's K slice of channel blocks [cb_w0, cb_w1), split over
  // its K groups
  const int cb_w0 = wk.ks * cblocks / a.ksplit, cb_w1 = (wk.ks + 1) * cblocks / a.ksplit;
  const int cb_per = (cb_w1 - cb_w0 + KS - 1) / KS;           // channel blocks per K group
  const int cb_lo = min(cb_w0 + grp * cb_per, cb_w1);
  const int nsteps = ntaps * (min(cb_lo + cb_per, cb_w1) - cb_lo);  // this group's stages
  const int nsteps_all = ntaps * cb_per;                      // the loop runs this many
  const int tail_c = a.cin - (cblocks - 1) * KC;

  __shared__ float s_bias[BN];
  const float* const bias = a.bias[sg.plan];
  for (int t = threadIdx.x; t < BN; t += NTA)
    s_bias[t] = (bias && wk.n0 + t < a.cout) ? bias[bias_index(a, wk.n0 + t)] : 0.f;
  __shared__ int4 s_taps[kMaxLdsTaps];
  const bool lds_taps = !sg.tap_ap && ntaps <= kMaxLdsTaps;
  if (lds_taps) {
    for (int t = threadIdx.x; t < ntaps; t += NTA) {
      const TapDev tp = a.taps[wk.tap_begin + t];
      s_taps[t] = make_int4((tp.off_h * a.w + tp.off_w) * a.cin * ESZ,
                            (int)((uint32_t)tp.slot * (uint32_t)a.cout_pad * (uint32_t)a.cin_pad * ESZ),
                            tp.off_h, tp.off_w);
    }
  }
  __syncthreads();

  struct Regs {
    uint4 s[S_LD];      // shared operand, this thread's chunks
    uint4 d[TD][HC];    // this wave's own operand, MFMA layout
  };
  Regs rb[DEPTH];

  int ld_tap = 0, ld_cb = cb_lo, ld_th = 0, ld_tw = 0;
  const uint32_t slot_bytes = (uint32_t)a.cout_pad * (uint32_t)a.cin_pad * ESZ;
  auto load_step = [&](Regs& R, bool valid) {
    const __amdgpu_buffer_rsrc_t xs = valid ? xr : xr0;
    const __amdgpu_buffer_rsrc_t ws = valid ? wr : wr0;
    int delta, off_h, off_w;
    uint32_t slot_b;
    if (sg.tap_ap) {
      off_h = sg.off0_h + ld_th * sg.doff_h;
      off_w = sg.off0_w + ld_tw * sg.doff_w;
      delta = (off_h * a.w + off_w) * a.cin * ESZ;
      slot_b = (uint32_t)((sg.kh0 + ld_th * sg.dkh) * a.ks + sg.kw0 + ld_tw * sg.dkw) * slot_bytes;
    } else {
      int4 ti;
      if (lds_taps) {
        ti = s_taps[valid ? ld_tap : 0];
      } else {
        const TapDev tp = a.taps[wk.tap_begin + (valid ? ld_tap : 0)];
        ti = make_int4((tp.off_h * a.w + tp.off_w) * a.cin * ESZ, (int)((uint32_t)tp.slot * slot_bytes),
                       tp.off_h, tp.off_w);
      }
      delta = __builtin_amdgcn_readfirstlane(ti.x);
      slot_b = (uint32_t)__builtin_amdgcn_readfirstlane(ti.y);
      off_h = __builtin_amdgcn_readfirstlane(ti.z);
      off_w = __builtin_amdgcn_readfirstlane(ti.w);
    }
    const uint32_t kb = (uint32_t)ld_cb * KB;
    const bool tail = ld_cb == cblocks - 1 && tail_c < KC;
    auto pix_off = [&](int i) {
      uint32_t v = p_base[i] + (uint32_t)delta;
      if (!sg.exact) {
        const int ih = p_ih[i] + off_h, iw = p_iw[i] + off_w;
        const bool in = ((unsigned)ih < (unsigned)a.h) & ((unsigned)iw < (unsigned)a.w);
        v = in ? v : OOB;
      }
      return v;
    };
    // the wave's own operand first: waiting for the shared chunks of a stage
    // then also covers these loads
    if constexpr (SHARE_A) {
#pragma unroll
      for (int i = 0; i < TD; ++i)
#pragma unroll
        for (int c = 0; c < HC; ++c)
          R.d[i][c] = __builtin_bit_cast(
              uint4, __builtin_amdgcn_raw_buffer_load_b128(ws, w_off[i], slot_b + 32 * kb + 1024 * c, 0));
#pragma unroll
      for (int i = 0; i < S_LD; ++i) {
        uint32_t v = pix_off(i);
        v = (tail && s_chunk * VE >= tail_c) ? OOB : v;
        R.s[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xs, v, kb, 0));
      }
    } else {
#pragma unroll
      for (int i = 0; i < TD; ++i) {
        const uint32_t v = pix_off(i);
#pragma unroll
        for (int c = 0; c < HC; ++c) {
          const bool out = tail && (half * HC + c) * VE >= tail_c;
          R.d[i][c] = __builtin_bit_cast(
              uint4, __builtin_amdgcn_raw_buffer_load_b128(xs, out ? OOB : v, kb + 16 * c, 0));
        }
      }
#pragma unroll
      for (int i = 0; i < S_LD; ++i)
        R.s[i] = __builtin_bit_cast(
            uint4, __builtin_amdgcn_raw_buffer_load_b128(ws, w_off[i], slot_b + kb, 0));
    }
    if (valid) {
      if (++ld_tw == sg.ntw) {
        ld_tw = 0;
        ++ld_th;
      }
      if (++ld_tap == ntaps) {
        ld_tap = 0;
        ld_th = 0;
        ld_tw = 0;
        ++ld_cb;
      }
    }
  };
  auto store_shared = [&](int buf, const Regs& R) {
    char* ss = smem + buf * STAGE_B;
#pragma unroll
    for (int i = 0; i < S_LD; ++i)
      if (RS * CPR % NT == 0 || tid + NT * i < RS * CPR)
        *(uint4*)(ss + (tid / CPR + (NT / CPR) * i) * ROWB + s_chunk * 16) = R.s[i];
  };

  f32x16 acc[TP][TC];
#pragma unroll
  for (int i = 0; i < TP; ++i)
#pragma unroll
    for (int j = 0; j < TC; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto compute = [&](int buf, const Regs& R) {
    const char* ss = smem + buf * STAGE_B + row32 * ROWB;
#pragma unroll
    for (int c = 0; c < HC; ++c) {
      uint4 fs[TS];
#pragma unroll
      for (int i = 0; i < TS; ++i)
        fs[i] = *(const uint4*)(ss + 32 * i * ROWB +
                                (SHARE_A ? pack_chunk_byte(c, half) : half * (KB / 2) + 16 * c));
      uint4 fp[TP], fc[TC];
#pragma unroll
      for (int i = 0; i < TP; ++i) fp[i] = SHARE_A ? fs[i] : R.d[i][c];
#pragma unroll
      for (int j = 0; j < TC; ++j) fc[j] = SHARE_A ? R.d[j][c] : fs[j];
      if constexpr (BF16) {
#pragma unroll
        for (int i = 0; i < TP; ++i)
#pragma unroll
          for (int j = 0; j < TC; ++j) {
            const bf16x8 vp = __builtin_bit_cast(bf16x8, fp[i]);
            const bf16x8 vc = __builtin_bit_cast(bf16x8, fc[j]);
            if constexpr (NCHW_OUT)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vc, vp, acc[i][j], 0, 0, 0);
            else
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vp, vc, acc[i][j], 0, 0, 0);
          }
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int i = 0; i < TP; ++i)
#pragma unroll
            for (int j = 0; j < TC; ++j) {
              const uint32_t bp = e == 0 ? fp[i].x : e == 1 ? fp[i].y : e == 2 ? fp[i].z : fp[i].w;
              const uint32_t bc = e == 0 ? fc[j].x : e == 1 ? fc[j].y : e == 2 ? fc[j].z : fc[j].w;
              const float vp = __uint_as_float(bp), vc = __uint_as_float(bc);
              if constexpr (NCHW_OUT)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(vc, vp, acc[i][j], 0, 0, 0);
              else
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(vp, vc, acc[i][j], 0, 0, 0);
            }
      }
    }
  };

  // Prologue: stages 0 .. DEPTH-1 in flight, stage 0 in LDS buffer 0.  Loop
  // invariant at the top of step u of an unrolled block starting at stage s:
  // LDS buffer (u & 1) holds stage s+u, register buffer (u % DEPTH) holds its
  // own-operand chunks, and the next DEPTH-1 stages are in flight.
  const int nsteps_u = (nsteps_all + U - 1) / U * U;
  if (nsteps_u > 0) {
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) load_step(rb[d], d < nsteps);
    store_shared(0, rb[0]);
    __syncthreads();
    for (int s = 0; s < nsteps_u; s += U) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        // the steps that round the loop up to U hold zeros: no MFMAs for them
        if (s + u < nsteps) compute(u & 1, rb[u % DEPTH]);
        store_shared((u + 1) & 1, rb[(u + 1) % DEPTH]);
        load_step(rb[u % DEPTH], s + u + DEPTH < nsteps);
        __syncthreads();
      }
    }
  }

  if constexpr (KS > 1) {
    // group 1's partial sums to LDS (lane-contiguous), group 0 adds them
    float* red = (float*)smem_all + wave * (TP * TC * 16 * 64) + lane;
    if (grp == 1) {
#pragma unroll
      for (int i = 0; i < TP; ++i)
#pragma unroll
        for (int j = 0; j < TC; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) red[((i * TC + j) * 16 + r) * 64] = acc[i][j][r];
    }
    __syncthreads();
    if (grp != 0) return;
#pragma unroll
    for (int i = 0; i < TP; ++i)
#pragma unroll
      for (int j = 0; j < TC; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] += red[((i * TC + j) * 16 + r) * 64];
  }
  const int pix0 = wk.m0 + (SHARE_A ? 0 : wave * RD);
  const int ch0 = wk.n0 + (SHARE_A ? wave * RD : 0);
  if (a.ksplit > 1) {
    store_tile<false, NCHW_OUT, TP, TC>(a, sg, wk.m1, a.part + (size_t)wk.ks * a.part_stride, acc,
                                        pix0, ch0, lane, s_bias - wk.n0);
  } else {
    store_tile<BF16, NCHW_OUT, TP, TC>(a, sg, wk.m1, a.y[sg.plan], acc, pix0, ch0, lane,
                                       s_bias - wk.n0);
  }
}

// ---------------------------------------------------------------------------
// Phase GEMM, pipelined split-wave form.  The same tile as phase_gemm2_kernel
// (BM pixel rows through LDS, each of the W waves of a K group loading its
// BN/W weight rows straight into registers in the MFMA lane layout), with
// the stage order rearranged so that LDS latency hides behind the MFMAs:
//  - three LDS stage buffers: stage s is written two stages ahead of its use
//    (while stage s-1's buffer may still be read), so one barrier per stage
//    separates every write from the reads it must not overtake;
//  - the 16-byte pixel fragments of K chunk c+1 are read while the MFMAs of
//    chunk c run, and the first chunk of stage s+1 while stage s finishes;
//  - pixel chunks are loaded DA = 2 stages before they are written to LDS,
//    weight fragments DB stages before their MFMAs, each with its own tap
//    and channel-block counter (a work's taps are a product of two
//    arithmetic progressions, read from the work item: no memory lookup per
//    stage; plans whose works have other tap lists take the unpipelined
//    kernel).
// The loop is unrolled by U = 6 (a multiple of the 3 LDS buffers and of DA
// and DB), so every buffer index is a compile-time constant.
template <bool BF16, int BM, int BN, int W, int KB, int DA, int DB, int KS, bool NCHW_OUT>
__global__ __launch_bounds__(W * 64 * KS, 2) void phase_gemm3_kernel(GemmArgs a) {
  constexpr int NTA = W * 64 * KS, NT = W * 64;
  constexpr int ESZ = BF16 ? 2 : 4;
  constexpr int KC = KB / ESZ;   // K elements per stage
  constexpr int VE = 16 / ESZ;   // elements per 16-byte chunk
  constexpr int CPR = KB / 16;   // 16-byte chunks per row and stage
  constexpr int HC = CPR / 2;    // K chunks per stage (one per lane half)
  constexpr int ROWB = KB + 16;  // LDS row pitch (16-byte pad: distinct banks)
  constexpr int RD = BN / W;     // weight rows (output channels) per wave
  constexpr int TP = BM / 32, TC = RD / 32;
  constexpr int S_LD = (BM * CPR + NT - 1) / NT;  // pixel chunks per thread and stage
  constexpr int NB = 3;
  constexpr int U = lcm3(NB, DA, DB);
  static_assert(RD % 32 == 0 && BM % 32 == 0 && HC >= 2 && HC % 2 == 0, "tile shape");
  static_assert(KB % kPackKB == 0, "K stages of whole packing blocks");
  static_assert(DA >= 2 && DA <= 4 && DB >= 2 && DB <= 4, "two to four stages in flight");
  constexpr int STAGE_B = BM * ROWB;
  constexpr uint32_t OOB = 0x80000000u;
  constexpr int ACC_B = KS > 1 ? W * 64 * TP * TC * 16 * 4 : 0;
  constexpr bool ROWS_OUT = BF16 && !NCHW_OUT && KS == 1;  // row epilogue through LDS
  constexpr int EPI_B = ROWS_OUT ? BM * (2 * BN + 16) : 0;
  constexpr int SMEM_B0 = KS * NB * STAGE_B > ACC_B ? KS * NB * STAGE_B : ACC_B;
  constexpr int SMEM_B = SMEM_B0 > EPI_B ? SMEM_B0 : EPI_B;
  __shared__ __attribute__((aligned(16))) char smem_all[SMEM_B];
  __shared__ float s_bias[BN];
  __shared__ int s_rowoff[ROWS_OUT ? BM : 1];  // output pixel index of each tile row

  const int wave_all = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63, grp = KS > 1 ? wave_all / W : 0;
  const int wave = wave_all - grp * W;
  const int tid = (int)threadIdx.x - grp * NT;
  char* const smem = smem_all + grp * NB * STAGE_B;
  const int half = lane >> 5, row32 = lane & 31;
  const int work = xcd_remap(blockIdx.x, gridDim.x);
  const WorkDev wk = a.works[work];
  const SegDev sg = a.segs[wk.seg];
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.x, 0, a.x_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t wr =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.wp[sg.plan], 0, a.wp_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t xr0 = __builtin_amdgcn_make_buffer_rsrc((void*)a.x, 0, 0, 0x00020000);
  const __amdgpu_buffer_rsrc_t wr0 =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.wp[sg.plan], 0, 0, 0x00020000);

  // this thread's pixel rows (chunk s_chunk of rows tid / CPR + (NT / CPR) * i)
  int p_ih[S_LD], p_iw[S_LD];
  uint32_t p_base[S_LD];
  const int s_chunk = tid % CPR;
#pragma unroll
  for (int i = 0; i < S_LD; ++i) {
    const int r = tid / CPR + (NT / CPR) * i;
    const int m = min(wk.m0 + r, wk.m1 - 1);
    const PixelPos p = pixel_pos(sg, a.ptab, m);
    p_ih[i] = p.ih;
    p_iw[i] = p.iw;
    p_base[i] = (((uint32_t)p.img * (uint32_t)a.h + (uint32_t)p.ih) * (uint32_t)a.w +
                 (uint32_t)p.iw) * (uint32_t)a.cin * ESZ + (uint32_t)(s_chunk * 16);
    if (ROWS_OUT && s_chunk == 0 && r < BM)
      s_rowoff[r] = wk.m0 + r < wk.m1 ? (p.img * a.ho + p.oh) * a.wo + p.ow : -1;
  }
  // lane-ordered weights: 32-channel block (n0 + wave * RD) / 32 + i
  uint32_t w_off[TC];
#pragma unroll
  for (int i = 0; i < TC; ++i)
    w_off[i] = (uint32_t)(((wk.n0 + wave * RD) / 32 + i) * 32 * a.cin_pad * ESZ + lane * 16);

  const int ntaps = wk.tap_count;
  const int cblocks = a.cin_pad / KC;
  const int cb_w0 = wk.ks * cblocks / a.ksplit, cb_w1 = (wk.ks + 1) * cblocks / a.ksplit;
  const int cb_per = (cb_w1 - cb_w0 + KS - 1) / KS;
  const int cb_lo = min(cb_w0 + grp * cb_per, cb_w1);
  const int nsteps = ntaps * (min(cb_lo + cb_per, cb_w1) - cb_lo);  // this group's stages
  const int nsteps_all = ntaps * cb_per;  // both groups run this many (shared barriers)
  const int tail_c = a.cin - (cblocks - 1) * KC;
  const uint32_t slot_bytes = (uint32_t)a.cout_pad * (uint32_t)a.cin_pad * ESZ;

  const float* const bias = a.bias[sg.plan];
  for (int t = threadIdx.x; t < BN; t += NTA)
    s_bias[t] = (bias && wk.n0 + t < a.cout) ? bias[bias_index(a, wk.n0 + t)] : 0.f;

  // Stage counters: tap (th, tw) inner, channel block outer.
  struct Iter {
    int th, tw, t, cb;
  };
  auto advance = [&](Iter& it) {
    if (++it.tw == wk.ap_ntw) {
      it.tw = 0;
      ++it.th;
    }
    if (++it.t == ntaps) {
      it.t = it.th = it.tw = 0;
      ++it.cb;
    }
  };
  // (the plan gives this kernel only works whose taps are progressions)
  auto tap_of = [&](const Iter& it, int* off_h, int* off_w, uint32_t* slot_b) {
    *off_h = wk.ap_off0_h + it.th * wk.ap_doff_h;
    *off_w = wk.ap_off0_w + it.tw * wk.ap_doff_w;
    *slot_b = (uint32_t)((wk.ap_kh0 + it.th * wk.ap_dkh) * a.ks + wk.ap_kw0 + it.tw * wk.ap_dkw) *
              slot_bytes;
  };
  Iter ia{0, 0, 0, cb_lo}, ib{0, 0, 0, cb_lo};

  struct RegA {
    uint4 v[S_LD];
  };
  struct RegB {
    uint4 v[TC][HC];
  };
  RegA ra[DA];
  RegB rb[DB];

  // Both loads are branch-free: a stage past the end reads through a
  // zero-size buffer (zeros), and a read outside the input gets an
  // out-of-range offset (zeros); the counters run on regardless.
  auto load_a = [&](RegA& R, bool valid) {
    const __amdgpu_buffer_rsrc_t xs = valid ? xr : xr0;
    int off_h, off_w;
    uint32_t slot_b;
    tap_of(ia, &off_h, &off_w, &slot_b);
    const int delta = (off_h * a.w + off_w) * a.cin * ESZ;
    const uint32_t kb = (uint32_t)ia.cb * KB;
    const bool tail = ia.cb == cblocks - 1 && tail_c < KC && s_chunk * VE >= tail_c;
#pragma unroll
    for (int i = 0; i < S_LD; ++i) {
      const int ih = p_ih[i] + off_h, iw = p_iw[i] + off_w;
      const bool in = ((unsigned)ih < (unsigned)a.h) & ((unsigned)iw < (unsigned)a.w) & !tail;
      const uint32_t v = in ? p_base[i] + (uint32_t)delta : OOB;
      R.v[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xs, v, kb, 0));
    }
    advance(ia);
  };
  auto load_b = [&](RegB& R, bool valid) {
    const __amdgpu_buffer_rsrc_t ws = valid ? wr : wr0;
    int off_h, off_w;
    uint32_t slot_b;
    tap_of(ib, &off_h, &off_w, &slot_b);
    const uint32_t kb = (uint32_t)ib.cb * KB;
#pragma unroll
    for (int i = 0; i < TC; ++i)
#pragma unroll
      for (int c = 0; c < HC; ++c)
        R.v[i][c] = __builtin_bit_cast(
            uint4, __builtin_amdgcn_raw_buffer_load_b128(ws, w_off[i], slot_b + 32 * kb + 1024 * c, 0));
    advance(ib);
  };
  auto store_a = [&](int buf, const RegA& R) {
    char* ss = smem + buf * STAGE_B;
#pragma unroll
    for (int i = 0; i < S_LD; ++i)
      if (BM * CPR % NT == 0 || tid + NT * i < BM * CPR)
        *(uint4*)(ss + (tid / CPR + (NT / CPR) * i) * ROWB + s_chunk * 16) = R.v[i];
  };
  auto read_f = [&](int buf, int c, uint4 (&f)[TP]) {
    const char* ss = smem + buf * STAGE_B + row32 * ROWB + pack_chunk_byte(c, half);
#pragma unroll
    for (int i = 0; i < TP; ++i) f[i] = *(const uint4*)(ss + 32 * i * ROWB);
  };

  f32x16 acc[TP][TC];
#pragma unroll
  for (int i = 0; i < TP; ++i)
#pragma unroll
    for (int j = 0; j < TC; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto mfma_chunk = [&](const uint4 (&fp)[TP], const RegB& R, int c) {
    if constexpr (BF16) {
#pragma unroll
      for (int i = 0; i < TP; ++i)
#pragma unroll
        for (int j = 0; j < TC; ++j) {
          const bf16x8 vp = __builtin_bit_cast(bf16x8, fp[i]);
          const bf16x8 vc = __builtin_bit_cast(bf16x8, R.v[j][c]);
          if constexpr (NCHW_OUT)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vc, vp, acc[i][j], 0, 0, 0);
          else
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vp, vc, acc[i][j], 0, 0, 0);
        }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int i = 0; i < TP; ++i)
#pragma unroll
          for (int j = 0; j < TC; ++j) {
            const uint4 x4 = fp[i], w4 = R.v[j][c];
            const uint32_t bp = e == 0 ? x4.x : e == 1 ? x4.y : e == 2 ? x4.z : x4.w;
            const uint32_t bc = e == 0 ? w4.x : e == 1 ? w4.y : e == 2 ? w4.z : w4.w;
            const float vp = __uint_as_float(bp), vc = __uint_as_float(bc);
            if constexpr (NCHW_OUT)
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(vc, vp, acc[i][j], 0, 0, 0);
            else
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(vp, vc, acc[i][j], 0, 0, 0);
          }
    }
  };

  // Prologue: stages 0 and 1 in LDS buffers 0 and 1, stages 2 and 3 in the
  // pixel registers, weight stages 0 .. DB-1 in flight, the first K chunk of
  // stage 0 being read.
  uint4 fr[2][TP];
  // One stage of the loop (u = stage mod U, a compile-time constant).  With
  // `checked`, the MFMAs of stages past this group's end are skipped (the
  // last, partial block of U stages); the full blocks run branch-free.
  auto stage = [&](auto u_c, auto checked, int st) {
    constexpr int u = decltype(u_c)::value;
#pragma unroll
    for (int c = 0; c < HC; ++c) {
      if (c + 1 < HC)
        read_f(u % NB, c + 1, fr[(c + 1) & 1]);
      else
        read_f((u + 1) % NB, 0, fr[(c + 1) & 1]);
      if constexpr (decltype(checked)::value) {
        if (st < nsteps) mfma_chunk(fr[c & 1], rb[u % DB], c);
      } else {
        mfma_chunk(fr[c & 1], rb[u % DB], c);
      }
      if (c == 0) {
        // stage st + 2 to LDS (its buffer last held stage st - 1, which
        // every wave finished reading before the previous barrier), and the
        // pixel loads of stage st + 2 + DA into the freed registers
        store_a((u + 2) % NB, ra[(u + 2) % DA]);
        load_a(ra[(u + 2) % DA], st + 2 + DA < nsteps);
      }
    }
    load_b(rb[u % DB], st + DB < nsteps);
    __syncthreads();
  };
  auto block = [&](auto checked, int s0) {
    unroll_stages<U>([&](auto u_c) { stage(u_c, checked, s0 + decltype(u_c)::value); });
  };
  if (nsteps_all > 0) {
    // stages 0, 1 through registers 0, 1 to LDS; then stages 2 .. DA+1 into
    // registers (stage j in register j mod DA: the loop stores stage st + 2
    // from register st mod DA and reloads it with stage st + 2 + DA)
    load_a(ra[0], 0 < nsteps);
    load_a(ra[1 % DA], 1 < nsteps);
    if constexpr (DA == 2) {
#pragma unroll
      for (int d = 0; d < DB; ++d) load_b(rb[d], d < nsteps);
      store_a(0, ra[0]);
      store_a(1, ra[1]);
    } else {
      store_a(0, ra[0]);
      store_a(1, ra[1]);
#pragma unroll
      for (int d = 0; d < DB; ++d) load_b(rb[d], d < nsteps);
    }
#pragma unroll
    for (int j = 2; j < 2 + DA; ++j) load_a(ra[j % DA], j < nsteps);
    __syncthreads();
    read_f(0, 0, fr[0]);
    // full blocks: every group has all of their stages when KS = 1 or the
    // groups' channel blocks split evenly; otherwise the shorter group's
    // extra stages multiply the zeros its loads returned
    const int nfull = (KS == 1 || nsteps == nsteps_all) ? nsteps_all / U * U : 0;
    for (int s = 0; s < nfull; s += U) block(std::false_type(), s);
    for (int s = nfull; s < nsteps_all; s += U) block(std::true_type(), s);
  } else {
    __syncthreads();
  }

  if constexpr (KS > 1) {
    float* red = (float*)smem_all + wave * (TP * TC * 16 * 64) + lane;
    if (grp == 1) {
#pragma unroll
      for (int i = 0; i < TP; ++i)
#pragma unroll
        for (int j = 0; j < TC; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) red[((i * TC + j) * 16 + r) * 64] = acc[i][j][r];
    }
    __syncthreads();
    if (grp != 0) return;
#pragma unroll
    for (int i = 0; i < TP; ++i)
#pragma unroll
      for (int j = 0; j < TC; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] += red[((i * TC + j) * 16 + r) * 64];
  }
  const int ch0 = wk.n0 + wave * RD;
  if constexpr (ROWS_OUT) {
    void* const yp = a.y[sg.plan];
    if (a.ksplit == 1 && (a.cout & 7) == 0 && ((uintptr_t)yp & 15) == 0) {
      if (a.act == 1)
        store_rows_nhwc<TP, TC, BM, BN, NT, 1>(a, wk.n0, yp, acc, wave * RD, lane, tid,
                                               smem_all, s_rowoff, s_bias);
      else if (a.act == 2)
        store_rows_nhwc<TP, TC, BM, BN, NT, 2>(a, wk.n0, yp, acc, wave * RD, lane, tid,
                                               smem_all, s_rowoff, s_bias);
      else
        store_rows_nhwc<TP, TC, BM, BN, NT, 0>(a, wk.n0, yp, acc, wave * RD, lane, tid,
                                               smem_all, s_rowoff, s_bias);
      return;
    }
  }
  if (a.ksplit > 1) {
    store_tile<false, NCHW_OUT, TP, TC>(a, sg, wk.m1, a.part + (size_t)wk.ks * a.part_stride, acc,
                                        wk.m0, ch0, lane, s_bias - wk.n0);
  } else {
    store_tile<BF16, NCHW_OUT, TP, TC>(a, sg, wk.m1, a.y[sg.plan], acc, wk.m0, ch0, lane,
                                       s_bias - wk.n0);
  }
}

template <bool BF16, bool NCHW_OUT, int CFG>
static void launch_one(const GemmArgs& a, hipStream_t stream) {
  constexpr TileShape t = kTiles[CFG];
  if constexpr (t.kind == 0)
    hipLaunchKernelGGL((phase_gemm_kernel<BF16, t.bm, t.bn, t.pw, t.cw, t.kb, t.depth, NCHW_OUT>),
                       dim3(a.n_works), dim3(t.pw * t.cw * 64), 0, stream, a);
  else if constexpr (t.kind == 3)
    hipLaunchKernelGGL((phase_gemm3_kernel<BF16, t.bm, t.bn, t.pw * t.cw, t.kb, t.depth % 10,
                                           t.depth / 10, t.ksplit, NCHW_OUT>),
                       dim3(a.n_works), dim3(t.pw * t.cw * t.ksplit * 64), 0, stream, a);
  else
    hipLaunchKernelGGL((phase_gemm2_kernel<BF16, t.bm, t.bn, t.pw * t.cw, t.kb, t.depth,
                                           t.kind == 1, t.ksplit, NCHW_OUT>),
                       dim3(a.n_works), dim3(t.pw * t.cw * t.ksplit * 64), 0, stream, a);
}

template <bool BF16, bool NCHW_OUT, int CFG = 0>
static hipError_t launch_cfg(const GemmArgs& a, int cfg, hipStream_t stream) {
  if constexpr (CFG < TILE_COUNT) {
    if (cfg == CFG) {
      launch_one<BF16, NCHW_OUT, CFG>(a, stream);
      return hipGetLastError();
    }
    return launch_cfg<BF16, NCHW_OUT, CFG + 1>(a, cfg, stream);
  } else {
    return hipErrorInvalidValue;
  }
}

hipError_t launch_phase_gemm(const GemmArgs& a, int dtype, int cfg, bool nchw_out,
                             hipStream_t stream) {
  if (a.n_works <= 0) return hipSuccess;
  if (dtype == 1)
    return nchw_out ? launch_cfg<true, true>(a, cfg, stream) : launch_cfg<true, false>(a, cfg, stream);
  return nchw_out ? launch_cfg<false, true>(a, cfg, stream) : launch_cfg<false, false>(a, cfg, stream);
}

// ---------------------------------------------------------------------------
// Transposed conv with few output channels (c_out * r * s <= 64), NCHW, bf16.
// The phase GEMM has N = c_out there, so its tiles are mostly padding and
// every input pixel is fetched once per (phase, tap).  This kernel instead
// keeps a block of input rows (full width, plus the halo its outputs need) in
// LDS, computes for every pixel of the block the products with all kernel
// taps at once on MFMA, Z[p][tap * c_out + k] = sum_c x[c][p] * w[c][k][tap]
// (section 3.2.1's per-tap 1x1 convolutions, all taps in one GEMM), and then
// forms each owned output as the sum of the Z entries of the input pixels and
// taps that reach it (the interleaved scatter of section 3.1, read side).
// Workgroup (image, block of OB output rows).  Input tile: rows [i_lo,
// i_lo + tr) and columns [j_lo, j_lo + tcw) of the input, zero outside it,
// stored channel-contiguous per pixel, 64 channels per pass (two LDS buffers:
// the next pass loads while this one multiplies).  A thread loads one pixel
// pair of 8 channels (8 dword loads, coalesced along the pixels) and writes
// each pixel's 8 channels with one 16-byte store.
__device__ __forceinline__ int floor_div_d(int a, int b) { return a >= 0 ? a / b : -((-a + b - 1) / b); }

template <bool NHWC>
__global__ __launch_bounds__(kZtileThreads) void ztile_kernel(ZArgs a) {
  constexpr int NT = kZtileThreads, NW = NT / 64;
  constexpr int RB = kZtileRowB;
  constexpr int BUF_B = kZtileMaxPixels * RB;
  // input items per thread and pass: NCHW (pixel pair, 8 channels) as 8
  // dword loads; NHWC (pixel, 8 channels) as one 16-byte load
  constexpr int MAXP = NHWC ? 2 * kZtileMaxItems : kZtileMaxItems;
  constexpr int MB_MAX = (kZtileMaxPixels / 32 + NW - 1) / NW;  // M blocks per wave
  constexpr uint32_t OOB = 0x80000000u;
  __shared__ __attribute__((aligned(16))) char zsm[kZtileLds];
  float* zs = (float*)zsm;  // [p][kZtileZPitch], after the GEMM
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int img = blockIdx.y, o0 = blockIdx.x * a.ob, o1 = min(o0 + a.ob, a.ho);
  const int i_lo = -floor_div_d(-(o0 + a.pad_h - (a.r - 1) * a.dil_h), a.stride_h);
  const int np = a.tr * a.tcw;
  const int mblocks = (np + 31) / 32;
  const int kx = a.r * a.s * a.cout;
  const uint32_t plane_b = (uint32_t)a.h * (uint32_t)a.w * 2u;
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc((void*)a.x, 0, a.x_bytes, 0x00020000);
  const uint32_t wp_bytes = (uint32_t)(a.r * a.s * a.cout_pad) * (uint32_t)a.cin_pad * 2u;
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc((void*)a.wp, 0, wp_bytes, 0x00020000);

  // weight fragments of one 64-channel pass, K permuted like the input tile
  // reads below: MFMA step t, lane half h takes channels c0 + 32h + 8t ..+8;
  // column col = nb*32 + lane%32 = tap*cout + k.  Branch-free: columns past
  // the taps read zeros (out-of-range offset).
  uint32_t w_off[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int col = nb * 32 + (lane & 31);
    const int tap = col / a.cout, k = col - tap * a.cout;
    w_off[nb] = col < kx ? ((uint32_t)(tap * a.cout_pad + k) * (uint32_t)a.cin_pad + 32u * (lane >> 5)) * 2u
                         : OOB;
  }
  auto load_w = [&](int c0, uint4 (&bfr)[4][2]) {
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        bfr[t][nb] = __builtin_bit_cast(
            uint4, __builtin_amdgcn_raw_buffer_load_b128(wr, w_off[nb], (uint32_t)(c0 + 8 * t) * 2u, 0));
  };
  uint4 bfr[4][2];
  load_w(0, bfr);
  // tap tables and bias for the final combine: read now into registers,
  // staged in LDS only before the combine, so nothing waits for them here
  __shared__ int8_t s_tap[3][2][kZtileMaxStride][kZtileMaxTaps];
  __shared__ int8_t s_tapn[2][kZtileMaxStride];
  __shared__ float s_zb[64];
  constexpr int NTAB = 2 * kZtileMaxStride * kZtileMaxTaps;
  static_assert(NTAB <= NT, "one tap-table entry per thread");
  const float zb_r = (a.bias && tid < a.cout) ? a.bias[tid] : 0.f;
  int8_t tk_r = 0, td_r = 0, tn_r = 0;
  if (tid < NTAB) {
    const int ax = tid / (kZtileMaxStride * kZtileMaxTaps), rem = tid % (kZtileMaxStride * kZtileMaxTaps);
    const int rho = rem / kZtileMaxTaps, t = rem % kZtileMaxTaps;
    tk_r = a.tap_k[ax][rho][t];
    td_r = a.tap_d[ax][rho][t];
    tn_r = a.tap_n[ax][rho];
  }
  // zero both tile buffers: halo columns and rows outside the input stay zero
  for (int e = tid; e < 2 * BUF_B / 16; e += NT) ((uint4*)zsm)[e] = make_uint4(0, 0, 0, 0);

  // This thread's input items of a pass: (pixel pair, 8-channel group), pairs
  // fastest, over the tile rows inside the input and the full input width
  // (w is even, so a pair never straddles a row).
  const int ir0 = max(0, i_lo), ir1 = min(a.h, i_lo + a.tr);
  const int npairs = max(0, ir1 - ir0) * a.w / 2;
  const int itotal = NHWC ? max(0, ir1 - ir0) * a.w * 8 : npairs * 8;
  uint32_t p_src[MAXP];
  int p_lds[MAXP], p_grp[MAXP];
#pragma unroll
  for (int j = 0; j < MAXP; ++j) {
    const int it = tid + NT * j;
    const bool ok = it < itotal;
    if constexpr (NHWC) {
      // the 8 channel groups of a pixel on neighbouring threads: each
      // pixel's 128 bytes of a pass are one run
      const int g = it & 7, px = it >> 3;
      const int rr = px / a.w, col = px - rr * a.w;
      p_grp[j] = g;
      p_src[j] = ok ? ((((uint32_t)img * (uint32_t)a.h + (uint32_t)(ir0 + rr)) * (uint32_t)a.w +
                        (uint32_t)col) * (uint32_t)a.cin + 8u * g) * 2u
                    : OOB;
      p_lds[j] = ok ? ((ir0 + rr - i_lo) * a.tcw + col - a.j_lo) * RB + 16 * g : -1;
    } else {
      const int g = it / max(npairs, 1), pp = it - g * npairs;
      const int rr = (2 * pp) / a.w, col = 2 * pp - rr * a.w;
      p_grp[j] = g;
      p_src[j] = ok ? ((((uint32_t)img * (uint32_t)a.cin + 8u * g) * (uint32_t)a.h + (uint32_t)(ir0 + rr)) *
                           (uint32_t)a.w + (uint32_t)col) * 2u
                    : OOB;
      p_lds[j] = ok ? ((ir0 + rr - i_lo) * a.tcw + col - a.j_lo) * RB + 16 * g : -1;
    }
  }
  // NCHW: P[j][k] is channel 8g + k of a pixel pair (two bf16); NHWC:
  // P[j][0..3] are the 8 channels of one pixel (c_in a multiple of 8)
  auto load_items = [&](int c0, uint32_t (&P)[MAXP][8]) {
    const uint32_t cbo = NHWC ? (uint32_t)c0 * 2u : (uint32_t)c0 * plane_b;
#pragma unroll
    for (int j = 0; j < MAXP; ++j) {
      if (j * NT >= itotal) break;  // the same for the whole workgroup
      // channels past c_in read zeros (out-of-range offset)
      if constexpr (NHWC) {
        const bool in = c0 + 8 * p_grp[j] < a.cin;
        const uint4 v = __builtin_bit_cast(
            uint4, __builtin_amdgcn_raw_buffer_load_b128(xr, in ? p_src[j] : OOB, cbo, 0));
        P[j][0] = v.x;
        P[j][1] = v.y;
        P[j][2] = v.z;
        P[j][3] = v.w;
      } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const bool in = c0 + 8 * p_grp[j] + k < a.cin;
          P[j][k] = __builtin_amdgcn_raw_buffer_load_b32(xr, in ? p_src[j] : OOB,
                                                         cbo + (uint32_t)k * plane_b, 0);
        }
      }
    }
  };
  auto store_items = [&](char* buf, const uint32_t (&P)[MAXP][8]) {
#pragma unroll
    for (int j = 0; j < MAXP; ++j) {
      if (j * NT >= itotal) break;
      if (p_lds[j] < 0) continue;
      if constexpr (NHWC) {
        *(uint4*)(buf + p_lds[j]) = make_uint4(P[j][0], P[j][1], P[j][2], P[j][3]);
      } else {
        uint32_t lo[4], hi[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          lo[e] = __builtin_amdgcn_perm(P[j][2 * e + 1], P[j][2 * e], 0x05040100u);
          hi[e] = __builtin_amdgcn_perm(P[j][2 * e + 1], P[j][2 * e], 0x07060302u);
        }
        *(uint4*)(buf + p_lds[j]) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
        *(uint4*)(buf + p_lds[j] + RB) = make_uint4(hi[0], hi[1], hi[2], hi[3]);
      }
    }
  };

  f32x16 acc[MB_MAX][2];
#pragma unroll
  for (int i = 0; i < MB_MAX; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[i][j][q] = 0.f;
  // LDS byte offset of each of this wave's M-block rows (pixels past np
  // repeat the last one: their Z rows are never read)
  int src_off[MB_MAX];
#pragma unroll
  for (int mi = 0; mi < MB_MAX; ++mi)
    src_off[mi] = min((wave + NW * mi) * 32 + (lane & 31), np - 1) * RB + (lane >> 5) * 64;

  uint32_t P[MAXP][8];
  load_items(0, P);  // registers only: issued before the barrier
  __syncthreads();  // tiles zeroed
  store_items(zsm, P);
  __syncthreads();
  const int npass = a.cin_pad / 64;
  if (npass > 1) load_items(64, P);
  for (int pass = 0; pass < npass; ++pass) {
    const char* buf = zsm + (pass & 1) * BUF_B;
#pragma unroll
    for (int mi = 0; mi < MB_MAX; ++mi) {
      if (wave + NW * mi >= mblocks) break;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const bf16x8 av = __builtin_bit_cast(bf16x8, *(const uint4*)(buf + src_off[mi] + 16 * t));
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
          acc[mi][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, __builtin_bit_cast(bf16x8, bfr[t][nb]),
                                                                acc[mi][nb], 0, 0, 0);
      }
    }
    // the next pass's weights into the registers just consumed
    __builtin_amdgcn_sched_barrier(0);
    if (pass + 1 < npass) load_w(64 * (pass + 1), bfr);
    __builtin_amdgcn_sched_barrier(0);
    if (pass + 1 < npass) store_items(zsm + ((pass + 1) & 1) * BUF_B, P);
    __syncthreads();
    if (pass + 2 < npass) load_items(64 * (pass + 2), P);
  }
  // Z to LDS (over the tile buffers): lane holds column lane%32 of rows
  // 8*(q/4) + 4*(lane/32) + q%4
#pragma unroll
  for (int mi = 0; mi < MB_MAX; ++mi) {
    const int mb = wave + NW * mi;
    if (mb >= mblocks) break;
    // rows past np land in the unused part of the buffer (mblocks * 32 rows
    // of Z fit in kZtileLds)
    float* zr = zs + (mb * 32 + 4 * (lane >> 5)) * kZtileZPitch + (lane & 31);
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int q = 0; q < 16; ++q)
        zr[(8 * (q >> 2) + (q & 3)) * kZtileZPitch + nb * 32] = acc[mi][nb][q];
  }
  if (tid < 64) s_zb[tid] = zb_r;
  if (tid < NTAB) {
    const int ax = tid / (kZtileMaxStride * kZtileMaxTaps), rem = tid % (kZtileMaxStride * kZtileMaxTaps);
    const int rho = rem / kZtileMaxTaps, t = rem % kZtileMaxTaps;
    s_tap[0][ax][rho][t] = tk_r;
    s_tap[1][ax][rho][t] = td_r;
    if (t == 0) s_tapn[ax][rho] = tn_r;
  }
  __syncthreads();
  // Owned outputs: rows [o0, o1), all columns, all channels.  Output row oh
  // with u = oh + pad = s*Q + rho takes the taps of phase rho, reading input
  // row Q + delta (the host's per-phase tap tables, staged in LDS).  Each
  // wave takes whole output rows, all channels; lane l takes columns
  // ow = l, l + 64, ...  The column part of every Z address depends only on
  // ow, so it is computed once per lane; the row part once per row.
  constexpr int PT = kZtilePhaseTaps;
  constexpr int OWL = 4;  // columns per lane held in registers (wo <= 256)
  int wpart[OWL][PT], ntw[OWL];
#pragma unroll
  for (int c = 0; c < OWL; ++c) {
    const int ow = lane + 64 * c;
    const int uw = ow + a.pad_w, qw = uw / a.stride_w, rw = uw - qw * a.stride_w;
    ntw[c] = ow < a.wo ? s_tapn[1][rw] : 0;
#pragma unroll
    for (int tw = 0; tw < PT; ++tw)
      wpart[c][tw] = (qw + s_tap[1][1][rw][tw] - a.j_lo) * kZtileZPitch + s_tap[0][1][rw][tw] * a.cout;
  }
  const int rows = o1 - o0;
  const int zmax = np * kZtileZPitch - 1;
  for (int orow = wave; orow < rows; orow += NW) {
    const int oh = o0 + orow;
    const int uh = oh + a.pad_h, qh = uh / a.stride_h, rh = uh - qh * a.stride_h;
    const int nth = s_tapn[0][rh];
    int hpart[PT];
#pragma unroll
    for (int th = 0; th < PT; ++th)
      hpart[th] = (qh + s_tap[1][0][rh][th] - i_lo) * a.tcw * kZtileZPitch +
                  s_tap[0][0][rh][th] * a.s * a.cout;
#pragma unroll
    for (int c = 0; c < OWL; ++c) {
      if (64 * c >= a.wo) break;
      const int ow = lane + 64 * c;
      // every tap pair up to the largest counts is read (addresses clamped
      // into Z) and the pairs this phase lacks are selected away, so that
      // the reads issue together instead of behind one branch each
      int addr[PT][PT];
      bool use[PT][PT];
#pragma unroll
      for (int th = 0; th < PT; ++th)
#pragma unroll
        for (int tw = 0; tw < PT; ++tw) {
          addr[th][tw] = min(max(hpart[th] + wpart[c][tw], 0), zmax - a.cout + 1);
          use[th][tw] = th < nth && tw < ntw[c];
        }
      // NCHW: channel k's plane; NHWC: the pixel's c_out consecutive channels
      size_t off = NHWC ? (((size_t)img * a.ho + oh) * a.wo + ow) * a.cout
                        : (((size_t)img * a.cout) * a.ho + oh) * a.wo + ow;
      const size_t kstep = NHWC ? 1 : (size_t)a.ho * a.wo;
      for (int k = 0; k < a.cout; ++k, off += kstep) {
        float v = s_zb[k];
#pragma unroll
        for (int th = 0; th < PT; ++th) {
          if (th >= a.max_th) break;
#pragma unroll
          for (int tw = 0; tw < PT; ++tw) {
            if (tw >= a.max_tw) break;
            const float z = zs[addr[th][tw] + k];
            v += use[th][tw] ? z : 0.f;
          }
        }
        if (ow < a.wo) ((uint16_t*)a.y)[off] = f32_to_bf16_rne(activate(v, a.act));
      }
    }
  }
}

hipError_t launch_ztile(const ZArgs& a, int dtype, hipStream_t stream) {
  if (dtype != 1) return hipErrorInvalidValue;  // the planner selects this form for bf16 only
  const dim3 grid((a.ho + a.ob - 1) / a.ob, a.n);
  if (a.nhwc)
    hipLaunchKernelGGL(ztile_kernel<true>, grid, dim3(kZtileThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(ztile_kernel<false>, grid, dim3(kZtileThreads), 0, stream, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Transposed conv with a large stride and few channels (NCHW, bf16, dilation
// 1, c_in and c_out <= 32, at most two taps of each axis per output phase):
// the segmentation-decoder upsampling shape.  Every output phase there is a
// GEMM of a few hundred pixels, and its pixels lie `stride` apart in the
// output, so the phase GEMM writes 2-byte elements that no store can
// combine.  This kernel is output-stationary instead: workgroup (image, row
// phase rho_h, block of RB rows of that phase) runs, for every column phase
// rho_w in turn, the small phase GEMM of section 3.1 (pixels x c_out, K =
// taps x c_in) on MFMA, scatters the results into an LDS copy of its output
// rows, and finally writes those rows whole with 16-byte stores.
// Output o with o + pad = s*Q + rho takes kernel taps k = rho + s*t and input
// Q - t (t = 0, 1 while k < kernel size).

__global__ __launch_bounds__(kRpThreads) void rowphase_kernel(RpArgs a) {
  constexpr int CH = kRpCh;
  constexpr int NT = kRpThreads, NW = NT / 64;
  constexpr int MRW = kRpMaxColPhasesPerWave;
  constexpr int PP = CH + 8;  // LDS elements per input pixel (16-byte pad: spreads the banks)
  __shared__ __attribute__((aligned(16))) uint16_t s_in[(kRpMaxRb + 1) * (kRpMaxW + 2) * PP];
  // output rows, column-phase major: [k][row][rho_w][q_w] (q_w < nq), so that
  // the lanes of one phase GEMM write consecutive elements
  __shared__ __attribute__((aligned(16))) uint16_t s_out[kRpOutElems];
  __shared__ float s_b[CH];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int b = blockIdx.x;
  const int qb = b % a.qblocks;
  b /= a.qblocks;
  const int rho_h = b % a.stride_h, img = b / a.stride_h;
  // rows of this row phase: oh = s*Q + rho_h - pad in [0, ho)
  const int q_lo = -floor_div_d(-(a.pad_h - rho_h), a.stride_h);
  const int q_hi = floor_div_d(a.ho - 1 + a.pad_h - rho_h, a.stride_h);
  const int Q0 = q_lo + qb * a.rb;
  const int nrows = min(a.rb, q_hi - Q0 + 1);
  if (nrows <= 0) return;  // the whole workgroup leaves together
  const int tnh = rho_h < a.r ? min(2, (a.r - 1 - rho_h) / a.stride_h + 1) : 0;
  const int wp2 = a.w + 2;
  const int nq = a.nq;  // q_w slots per column phase (>= largest q_w + 1)

  // weight fragments of all this wave's column phases rho_w = wave + NW*c,
  // issued first so that they arrive while the input is staged
  const int k = lane & 31, half = lane >> 5;
  uint4 bw[MRW][4][2];
#pragma unroll
  for (int c = 0; c < MRW; ++c) {
    const int rho_w = wave + NW * c;
    const int tnw = (rho_w < a.stride_w && rho_w < a.s) ? min(2, (a.s - 1 - rho_w) / a.stride_w + 1) : 0;
#pragma unroll
    for (int tp = 0; tp < 4; ++tp)
#pragma unroll
      for (int cs = 0; cs < 2; ++cs) {
        const int th = tp >> 1, tw = tp & 1;
        bw[c][tp][cs] = make_uint4(0, 0, 0, 0);
        if (th < tnh && tw < tnw) {
          const int slot = (rho_h + a.stride_h * th) * a.s + rho_w + a.stride_w * tw;
          bw[c][tp][cs] = *(const uint4*)((const uint16_t*)a.wp +
                                          ((size_t)slot * CH + k) * CH + cs * 16 + half * 8);
        }
      }
  }

  if (tid < CH) s_b[tid] = (a.bias && tid < a.cout) ? a.bias[tid] : 0.f;
  // input rows Q0-1 .. Q0+nrows-1, columns -1 .. w, channel-contiguous; zero outside
  const int in_elems = (nrows + 1) * wp2 * CH;
  for (int e = tid; e < in_elems; e += NT) {
    const int c = e % CH, pc = e / CH;
    const int lc = pc % wp2, lr = pc / wp2;
    const int i = Q0 - 1 + lr, j = lc - 1;
    uint16_t v = 0;
    if (c < a.cin && i >= 0 && i < a.h && j >= 0 && j < a.w)
      v = ((const uint16_t*)a.x)[(((size_t)img * a.cin + c) * a.h + i) * a.w + j];
    s_in[pc * PP + c] = v;
  }
  __syncthreads();
  // output rows start at the bias (phases no tap reaches keep it), two
  // elements at a time.  Channel k's rows start at k * cp: one dword more
  // than its rows need, so that the 32 channels one store instruction
  // writes fall in distinct LDS banks.
  const int blk = a.stride_w * nq;  // a multiple of 8 (host)
  const int cp = nrows * blk + 2;
  const int npair = a.cout * (cp / 2);
  for (int e = tid; e < npair; e += NT) {
    const int kk = e / (cp / 2);
    const uint32_t bb = f32_to_bf16_rne(activate(s_b[kk], a.act));
    *(uint32_t*)(s_out + (size_t)e * 2) = bb | (bb << 16);
  }
  __syncthreads();

#pragma unroll
  for (int c = 0; c < MRW; ++c) {
    const int rho_w = wave + NW * c;
    if (rho_w >= a.stride_w) break;
    const int tnw = rho_w < a.s ? min(2, (a.s - 1 - rho_w) / a.stride_w + 1) : 0;
    const int qw_lo = -floor_div_d(-(a.pad_w - rho_w), a.stride_w);
    const int qw_hi = floor_div_d(a.wo - 1 + a.pad_w - rho_w, a.stride_w);
    const int nqw = qw_hi - qw_lo + 1;
    const int npix = nrows * nqw;
    if (tnh == 0 || tnw == 0 || nqw <= 0) continue;
    // pixel m -> (row, column) by a float reciprocal: m < 2^12, so
    // (m + 0.5) / nqw never lands within rounding error of an integer
    const float inv_nqw = 1.0f / (float)nqw;
    for (int mb = 0; mb * 32 < npix; ++mb) {
      const int m = min(mb * 32 + (lane & 31), npix - 1);
      const int qrow = (int)(((float)m + 0.5f) * inv_nqw), qw = qw_lo + m - qrow * nqw;
      f32x16 acc;
#pragma unroll
      for (int q = 0; q < 16; ++q) acc[q] = 0.f;
#pragma unroll
      for (int tp = 0; tp < 4; ++tp) {
        const int th = tp >> 1, tw = tp & 1;
        if (th >= tnh || tw >= tnw) continue;
        const int lr = qrow + 1 - th, lc = qw - tw + 1;
#pragma unroll
        for (int cs = 0; cs < 2; ++cs) {
          const uint4 av = *(const uint4*)(s_in + (lr * wp2 + lc) * PP + cs * 16 + half * 8);
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, av),
                                                        __builtin_bit_cast(bf16x8, bw[c][tp][cs]),
                                                        acc, 0, 0, 0);
        }
      }
      // lane holds output channel k for pixels 8*(q/4) + 4*half + q%4 of the block
      if (k < a.cout) {
        const float bk = s_b[k];
#pragma unroll
        for (int q = 0; q < 16; ++q) {
          const int mm = mb * 32 + 8 * (q >> 2) + 4 * half + (q & 3);
          if (mm >= npix) continue;
          const int qr = (int)(((float)mm + 0.5f) * inv_nqw), qwv = qw_lo + mm - qr * nqw;
          s_out[k * cp + (qr * a.stride_w + rho_w) * nq + qwv] = f32_to_bf16_rne(activate(acc[q] + bk, a.act));
        }
      }
    }
  }
  __syncthreads();
  // whole output rows, 16 bytes per store: element ow of a row is phase
  // (ow + pad) mod stride, slot (ow + pad) div stride.  Lane l takes the
  // 8-element pieces v = l, l + 64, ... of every row its wave visits, so the
  // phase/slot decomposition is done once per piece.
  const int vpr = a.wo / 8;
  constexpr int VPL = 4;  // pieces per lane: rows of at most 2048 elements
  int q0[VPL], r0[VPL];
#pragma unroll
  for (int c = 0; c < VPL; ++c) {
    const int u = (lane + 64 * c) * 8 + a.pad_w;
    q0[c] = u / a.stride_w;
    r0[c] = u - q0[c] * a.stride_w;
  }
  for (int rr = wave; rr < a.cout * nrows; rr += NW) {
    const int kk = rr / nrows, qr = rr - kk * nrows;
    const int oh = a.stride_h * (Q0 + qr) + rho_h - a.pad_h;
    const uint16_t* row = s_out + kk * cp + qr * blk;
    uint16_t* yrow = (uint16_t*)a.y + (((size_t)img * a.cout + kk) * a.ho + oh) * a.wo;
#pragma unroll
    for (int c = 0; c < VPL; ++c) {
      const int v = lane + 64 * c;
      if (v >= vpr) break;
      int qw = q0[c], rw = r0[c];
      uint32_t wv[4];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const uint32_t h16 = row[rw * nq + qw];
        if (t & 1)
          wv[t >> 1] |= h16 << 16;
        else
          wv[t >> 1] = h16;
        if (++rw == a.stride_w) {
          rw = 0;
          ++qw;
        }
      }
      store_stream16(yrow + v * 8, make_uint4(wv[0], wv[1], wv[2], wv[3]));
    }
  }
}

// ---------------------------------------------------------------------------
// Column-phase form of a transposed conv with column stride 32 (the FCN-32s
// upsampling shape).  Output column o with o + pad_w = 32*Q_w + rho_w takes
// kernel columns rho_w + 32*tw from input column Q_w - tw (tw = 0, 1); row
// phase rho_h likewise takes kernel rows rho_h + s_h*th from input row Q - th.
// For one (k, rho_h) the 32 column phases share the input fragments, so they
// are the 32 rows of an MFMA tile whose columns are input positions (Q, Q_w):
// each result column is then 32 consecutive elements of one output row,
// which after one exchange between the wave halves go out as 16-byte pieces.

template <int KBLK, int ACT>
__global__ __launch_bounds__(kCpWaves * 64) void colphase_kernel(CpArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint16_t s_x[];  // [(h+2)*(w+2)][cp]
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rblocks = (a.stride_h + kCpWaves - 1) / kCpWaves;
  int b = blockIdx.x;
  const int rb = b % rblocks;
  b /= rblocks;
  const int img = b % a.n, k = b / a.n;
  const int rho_h = rb * kCpWaves + wave;
  constexpr int kblk = KBLK;  // K blocks of 16: 4 taps x CP channels
  constexpr int CP = 4 * KBLK;  // channel slots per staged pixel (CpArgs::cp)
  const int wp2 = a.w + 2;

  // this wave's weight fragments (row rho_w = lane % 32, K run 2*kb + lane/32)
  uint4 wa[KBLK];
  const bool live = rho_h < a.stride_h;
  {
    const uint4* src = (const uint4*)a.wp + ((size_t)(k * a.stride_h + (live ? rho_h : 0)) * kblk) * 64 + lane;
#pragma unroll
    for (int kb = 0; kb < kblk; ++kb) wa[kb] = src[kb * 64];
  }
  // image img's input, channel-contiguous, with a border of zeros; the
  // elements go 16 per thread at a time, all loads before the LDS stores,
  // so that their latencies overlap
  const int npix = (a.h + 2) * wp2;
  const int total = npix * CP;
  const uint16_t* xin = (const uint16_t*)a.x + (size_t)img * a.cin * a.h * a.w;
  constexpr int NT = kCpWaves * 64;
  if ((a.w & 7) == 0 && ((uintptr_t)a.x & 15) == 0) {
    // 16-byte pieces of input rows (8 pixels of one channel), four per
    // thread in flight, then spread to the pixels' channel slots over a
    // zeroed area (border and padding channels stay 0).  Piece q is channel
    // q mod C_in of pixel piece q div C_in: neighbouring lanes write
    // neighbouring channel slots (few LDS bank conflicts).
    const int wv = a.w / 8, nv = a.cin * a.h * wv;
    uint4 v[4];
    int dst[4];
    auto fetch = [&](int q0) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int q = q0 + u * NT;
        const int rest = (int)fast_div((uint32_t)q, a.dv_mul[4], a.dv_shift[4]);
        const int c = q - rest * a.cin;
        const int i = (int)fast_div((uint32_t)rest, a.dv_mul[5], a.dv_shift[5]);
        const int piece = rest - i * wv;
        v[u] = q < nv ? *(const uint4*)(xin + ((size_t)c * a.h + i) * a.w + 8 * piece)
                      : make_uint4(0, 0, 0, 0);
        dst[u] = ((i + 1) * wp2 + 8 * piece + 1) * CP + c;
      }
    };
    fetch(tid);  // the first pieces in flight during the zeroing pass
    for (int e = 8 * tid; e < total; e += 8 * NT) *(uint4*)(s_x + e) = make_uint4(0, 0, 0, 0);
    __syncthreads();
    for (int q0 = tid; q0 < nv; q0 += 4 * NT) {
      if (q0 != tid) fetch(q0);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (q0 + u * NT >= nv) break;
        uint16_t* d = s_x + dst[u];
        const uint32_t w4[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
        for (int t = 0; t < 8; ++t) d[t * CP] = (uint16_t)(w4[t >> 1] >> (16 * (t & 1)));
      }
    }
  } else {
  constexpr int SU = 16;
  for (int e0 = tid; e0 < total; e0 += SU * kCpWaves * 64) {
    uint16_t v[SU];
    int dst[SU];
#pragma unroll
    for (int u = 0; u < SU; ++u) {
      const int e = e0 + u * kCpWaves * 64;
      const int t = (int)fast_div((uint32_t)e, a.dv_mul[0], a.dv_shift[0]);
      const int pj = e - t * wp2;
      const int c = (int)fast_div((uint32_t)t, a.dv_mul[1], a.dv_shift[1]);
      const int pi = t - c * (a.h + 2);
      const int i = pi - 1, j = pj - 1;
      const bool in = e < total && c < a.cin && i >= 0 && i < a.h && j >= 0 && j < a.w;
      // branch-free: an element outside the input reads x[0] and keeps 0
      const uint16_t xv = xin[in ? ((size_t)c * a.h + i) * a.w + j : 0];
      v[u] = in ? xv : (uint16_t)0;
      dst[u] = e < total ? (pi * wp2 + pj) * CP + c : -1;
    }
#pragma unroll
    for (int u = 0; u < SU; ++u)
      if (dst[u] >= 0) s_x[dst[u]] = v[u];
  }
  }
  const float bk = a.bias ? a.bias[k] : 0.f;
  __syncthreads();
  if (!live) return;

  const int q_lo = -floor_div_d(-(a.pad_h - rho_h), a.stride_h);
  const int q_hi = floor_div_d(a.ho - 1 + a.pad_h - rho_h, a.stride_h);
  const int nq = q_hi - q_lo + 1;
  if (nq <= 0) return;
  const int half = lane >> 5, col32 = lane & 31;
  const int rpt = CP / 8;  // 8-channel runs per tap
  uint16_t* yk = (uint16_t*)a.y + ((size_t)img * a.cout + k) * a.ho * a.wo;
  // this wave's output rows, kCpRows at a time, assembled in LDS and then
  // written whole (16 bytes per lane, consecutive lanes consecutive pieces)
  // Row qi of the buffer holds 16-byte piece p of the output row at piece
  // p ^ ((p >> 4) & 3) (rows padded to whole groups of four pieces): the
  // lanes of one LDS write hold neighbouring 64-byte column blocks, which
  // unswizzled fall on four bank groups (8-way conflicts), swizzled on 16.
  const int wo_lds = (a.wo + 31) & ~31;
  uint16_t* s_o = s_x + (size_t)(a.h + 2) * wp2 * CP + (size_t)wave * kCpRows * wo_lds;
  auto swz = [](int piece) { return piece ^ ((piece >> 4) & 3); };
  const int vpr = a.wo / 8;  // 16-byte pieces per output row
  for (int q0 = 0; q0 < nq; q0 += kCpRows) {
    const int nr = min(kCpRows, nq - q0);
    const int ncol = nr * a.nqw;
    // column tiles two at a time (independent accumulators: their MFMA
    // chains and LDS reads interleave), then the odd one
    auto tiles = [&](int c0, auto two_c) {
      constexpr int NTL = decltype(two_c)::value ? 2 : 1;
      int qi[NTL], Qw[NTL], base[NTL];
#pragma unroll
      for (int u = 0; u < NTL; ++u) {
        const int col = min(c0 + 32 * u + col32, ncol - 1);
        qi[u] = (int)fast_div((uint32_t)col, a.dv_mul[2], a.dv_shift[2]);
        Qw[u] = a.qw_lo + col - qi[u] * a.nqw;
        base[u] = ((q_lo + q0 + qi[u] + 1) * wp2 + Qw[u] + 1) * CP;
      }
      f32x16 acc[NTL];  // the bias is the sums' starting value
#pragma unroll
      for (int u = 0; u < NTL; ++u)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[u][r] = bk;
#pragma unroll
      for (int kb = 0; kb < kblk; ++kb) {
        const int run = 2 * kb + half;
        const int t = (int)fast_div((uint32_t)run, a.dv_mul[3], a.dv_shift[3]);
        const int off = (-(t >> 1) * wp2 - (t & 1)) * CP + (run - t * rpt) * 8;
        uint4 xv[NTL];
#pragma unroll
        for (int u = 0; u < NTL; ++u) xv[u] = *(const uint4*)(s_x + base[u] + off);
#pragma unroll
        for (int u = 0; u < NTL; ++u)
          acc[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, wa[kb]),
                                                           __builtin_bit_cast(bf16x8, xv[u]), acc[u],
                                                           0, 0, 0);
      }
      // rows 8g + 4*half + (0..3) of a column are four consecutive output
      // elements of row qi: one 8-byte LDS write each (all four groups
      // without checks where the column's 32 outputs lie inside the row)
#pragma unroll
      for (int u = 0; u < NTL; ++u) {
        if (c0 + 32 * u + col32 >= ncol) continue;
        const int ow_b = 32 * Qw[u] + 4 * half - a.pad_w;
        uint16_t* const orow = s_o + qi[u] * wo_lds;
        auto put = [&](int g) {
          const int ow0 = ow_b + 8 * g;
          const uint32_t p0 = pack_bf16x2_rne(activate(acc[u][4 * g], ACT),
                                              activate(acc[u][4 * g + 1], ACT));
          const uint32_t p1 = pack_bf16x2_rne(activate(acc[u][4 * g + 2], ACT),
                                              activate(acc[u][4 * g + 3], ACT));
          *(uint2*)(orow + 8 * swz(ow0 >> 3) + (ow0 & 7)) = make_uint2(p0, p1);
        };
        if (ow_b >= 0 && ow_b + 24 < a.wo) {
#pragma unroll
          for (int g = 0; g < 4; ++g) put(g);
        } else {
#pragma unroll
          for (int g = 0; g < 4; ++g)
            if (ow_b + 8 * g >= 0 && ow_b + 8 * g < a.wo) put(g);
        }
      }
    };
    int c0 = 0;
    for (; c0 + 32 < ncol; c0 += 64) tiles(c0, std::true_type());
    if (c0 < ncol) tiles(c0, std::false_type());
    // the rows out: piece v of row qi from LDS to the output (streaming
    // stores: the output is written once and not read back here)
    for (int qi = 0; qi < nr; ++qi) {
      const int oh = a.stride_h * (q_lo + q0 + qi) + rho_h - a.pad_h;
      for (int v = lane; v < vpr; v += 64)
        store_stream16(yk + (size_t)oh * a.wo + 8 * v, *(const uint4*)(s_o + qi * wo_lds + 8 * swz(v)));
    }
  }
}

hipError_t launch_colphase(const CpArgs& a, hipStream_t stream) {
  const int rblocks = (a.stride_h + kCpWaves - 1) / kCpWaves;
  const dim3 grid(a.cout * a.n * rblocks);
  const size_t lds =
      ((size_t)(a.h + 2) * (a.w + 2) * a.cp + (size_t)kCpWaves * kCpRows * ((a.wo + 31) & ~31)) * 2;
  const int kblk = a.cp / 4;
#define HUGE2_CP_LAUNCH(KB, ACT)                                                            \
  if (kblk == KB && a.act == ACT)                                                           \
    hipLaunchKernelGGL((colphase_kernel<KB, ACT>), grid, dim3(kCpWaves * 64), lds, stream, a);
  HUGE2_CP_LAUNCH(2, 0) HUGE2_CP_LAUNCH(2, 1) HUGE2_CP_LAUNCH(2, 2)
  HUGE2_CP_LAUNCH(4, 0) HUGE2_CP_LAUNCH(4, 1) HUGE2_CP_LAUNCH(4, 2)
  HUGE2_CP_LAUNCH(6, 0) HUGE2_CP_LAUNCH(6, 1) HUGE2_CP_LAUNCH(6, 2)
  HUGE2_CP_LAUNCH(8, 0) HUGE2_CP_LAUNCH(8, 1) HUGE2_CP_LAUNCH(8, 2)
#undef HUGE2_CP_LAUNCH
  return hipGetLastError();
}

// Weights of the column-phase form: per (k, rho_h), K block kb and lane l the
// 8 values w[c, k, rho_h + s_h*th, rho_w + 32*tw] for c in [c0, c0 + 8), with
// rho_w = l % 32, K run 2*kb + l/32 = tap * (cp/8) + c0/8, tap = 2*th + tw
// (zero for c >= c_in or a kernel index past the kernel).
__global__ void pack_colphase_kernel(const uint16_t* __restrict__ w, uint16_t* __restrict__ wp,
                                     int cin, int cout, int r, int s, int stride_h, int cp,
                                     long long total) {
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int e = (int)(idx % 8);
    long long t = idx / 8;
    const int lane = (int)(t % 64);
    t /= 64;
    const int kblk = cp / 4;
    const int kb = (int)(t % kblk);
    t /= kblk;
    const int rho_h = (int)(t % stride_h);
    const int k = (int)(t / stride_h);
    const int rho_w = lane % 32, run = 2 * kb + lane / 32, rpt = cp / 8;
    const int tap = run / rpt, c = (run - tap * rpt) * 8 + e;
    const int kh = rho_h + stride_h * (tap >> 1), kw = rho_w + 32 * (tap & 1);
    uint16_t v = 0;
    if (c < cin && kh < r && kw < s) v = w[(((long long)c * cout + k) * r + kh) * s + kw];
    wp[idx] = v;
  }
}

hipError_t launch_pack_colphase(const void* w, void* wp, int cin, int cout, int r, int s,
                                int stride_h, int cp, hipStream_t stream) {
  const long long total = (long long)cout * stride_h * (cp / 4) * 64 * 8;
  const long long want = (total + 255) / 256;
  const int grid = (int)(want < 65536 ? want : 65536);
  hipLaunchKernelGGL(pack_colphase_kernel, dim3(grid), dim3(256), 0, stream, (const uint16_t*)w,
                     (uint16_t*)wp, cin, cout, r, s, stride_h, cp, total);
  return hipGetLastError();
}

hipError_t launch_rowphase(const RpArgs& a, hipStream_t stream) {
  const dim3 grid(a.n * a.stride_h * a.qblocks);
  hipLaunchKernelGGL(rowphase_kernel, grid, dim3(kRpThreads), 0, stream, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Stride-2 transposed conv with a 4x4 kernel and padding 1 (NCHW, bf16), the
// DCGAN/cGAN generator layer.  Each of its four output phases has 2x2 taps
// whose input offsets lie in [-1, 1], and each phase's pixel grid is the
// input grid (section 3.1).  A workgroup takes 32*NP input positions (ni
// images x qbh rows x the full width) and 32*nch output channels, and
// computes the four phases there.  Each weight fragment a wave loads feeds
// NP MFMAs, so NP = 4 halves the weight bytes per multiply-add that reach
// the compute unit from L2:
//  - per 64-channel K block, the input block plus a one-pixel halo is read
//    straight from the NCHW planes into an LDS tile of channel-contiguous
//    pixel rows: a thread loads one pixel pair of 8 channels (8 dword loads,
//    coalesced along the pixels), regroups the halves with byte permutes and
//    writes each pixel's 8 channels with one 16-byte store.  The four phases
//    and their taps all read that one tile, so there is one barrier per K
//    block rather than one per tap, and no separate re-layout pass;
//  - wave (phase, K group or channel block) runs its phase's GEMM over WCH
//    32-channel blocks with the four taps as K stages (the untangled 1x1
//    convolutions of section 3.2.1), the weights loaded straight into the
//    MFMA lane layout, DEPTH taps ahead; with WCH = 2 each 16-byte pixel
//    fragment read from LDS feeds two MFMAs;
//  - the four phases' results are interleaved in LDS into whole output rows
//    (the scatter of section 3.1) and written with 16-byte stores.
// With two K groups, group 1 hands its partial sums to group 0 through LDS in
// a fixed order (deterministic).
template <int KS, int WCH, int DEPTH, int NP, bool NHWC>
__global__ __launch_bounds__(kQuadThreads) void quad_kernel(QArgs a) {
  constexpr int NT = kQuadThreads;
  constexpr int NTG = NT / KS;  // threads of one K group
  // the slot swizzle (below); unswizzled rows are padded by 16 bytes
  constexpr bool SWZ = true;
  constexpr int RB = SWZ ? kQuadRowB : kQuadRowB + 16;
  constexpr int HALO_B = kQuadHaloRows * RB;
  // input items per thread and K block: NCHW (pixel pair, 8 channels) as 8
  // dword loads; NHWC (pixel, 8 channels) as one 16-byte load
  constexpr int MAXP = NHWC ? 2 * kQuadMaxPieces : kQuadMaxPieces;
  constexpr uint32_t OOB = 0x80000000u;
  static_assert(DEPTH == 2 || DEPTH == 4, "weight stages in flight");
  static_assert(KS == 2 || WCH == 1, "one K group: two waves of 32 channels per phase");
  static_assert(NP == 2 || (NP == 4 && WCH == 1), "32-position blocks per wave");
  // pixel fragments double-buffered across taps where the registers allow
  constexpr bool PF = NP == 2 && WCH == 1 && DEPTH == 2;
  constexpr int U = DEPTH > 4 ? DEPTH / 4 : 1;  // K blocks per unrolled loop step
  // LDS: the K groups' double-buffered halo tiles, reused after the main loop
  // for group 1's partial sums and then for the interleaved output block
  // (64 channels x 4 phases x 32*NP positions, rows padded by 16 bytes)
  constexpr int TILE_B = KS * 2 * HALO_B;
  constexpr int RED_B = KS > 1 ? 4 * WCH * NP * 16 * 64 * 4 : 0;
  // NCHW: [channel][4 * 32 * NP positions + 8]; NHWC: [pixel][64 + 8 channels]
  constexpr int OUT_B = NHWC ? 4 * 32 * NP * (64 + 8) * 2 : 64 * (4 * 32 * NP + 8) * 2;
  constexpr int SMEM_B = cmax(TILE_B, cmax(RED_B, OUT_B));
  __shared__ __attribute__((aligned(16))) char smem[SMEM_B];
  __shared__ __attribute__((aligned(16))) float s_bias[64];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int rho = wave & 3, rest = wave >> 2;
  const int grp = KS > 1 ? rest : 0, hc = KS > 1 ? 0 : rest;
  const int tg = tid - grp * NTG;  // thread index within the K group
  const int bn = 32 * a.nch;
  // output-channel tile slowest: each XCD's contiguous run of workgroups
  // shares one weight slice
  const int work = xcd_remap(blockIdx.x, gridDim.x);
  const int nsp = a.igroups * a.hblocks;
  const int ntile = work / nsp, sp = work - ntile * nsp;
  const int ig = sp / a.hblocks, hb = sp - ig * a.hblocks;
  const int img0 = ig * a.ni, qh0 = hb * a.qbh, n0 = ntile * bn;
  const int hww = a.w + 2, hrows = a.qbh + 2;  // halo tile: width, rows per image
  const uint32_t plane_b = (uint32_t)a.h * (uint32_t)a.w * 2u;

  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc((void*)a.x, 0, a.x_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc((void*)a.wp, 0, a.wp_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t wr0 = __builtin_amdgcn_make_buffer_rsrc((void*)a.wp, 0, 0, 0x00020000);

  // zero halo tiles: the halo ring, rows outside the image and images past
  // the batch are never written afterwards
  for (int e = tid; e < KS * 2 * HALO_B / 16; e += NT) ((uint4*)smem)[e] = make_uint4(0, 0, 0, 0);
  // the bias is needed in the epilogue only: its load is not waited for here
  const float bias_r = (a.bias && tid < bn && n0 + tid < a.cout) ? a.bias[n0 + tid] : 0.f;

  // This thread's input items of a K block: item = (pixel pair, group of 8
  // channels), pixel pairs fastest.  The loaded rows are [r0, r1) of each
  // image (the block's rows plus the halo rows inside the image); w is even,
  // so a pair never straddles a row.
  const int r0 = max(0, qh0 - 1), r1 = min(a.h, qh0 + a.qbh + 1);
  const int rows = r1 - r0;
  const int npairs = a.ni * rows * a.w / 2;
  const int itotal = NHWC ? a.ni * rows * a.w * 8 : npairs * 8;
  // LDS tile layout: halo pixel (il, rl, cl) (rl, cl counting the halo row
  // and column) is the RB-byte row p = (il * hrows + rl) * hww + cl, and its
  // eight 16-byte groups of 8 channels sit at slots g ^ sw(pv), where
  // sw(pv) = (pv >> 1) & 7 and pv = (il * qbh + rl - 1) * w + cl.  The 32
  // pixels that one fragment read takes (any tap) have consecutive pv, so
  // the XOR spreads them over all 64 banks (no padding needed; measured: two
  // rows of 16 or four rows of 8 such 144-byte rows conflict two-way).
  auto slot_sw = [](int pv) { return SWZ ? (pv >> 1) & 7 : 0; };
  uint32_t p_src[MAXP];
  int p_lds[MAXP], p_lds_hi[MAXP];
#pragma unroll
  for (int j = 0; j < MAXP; ++j) {
    const int it = tg + NTG * j;
    // NHWC: the 8 channel groups of a pixel on neighbouring threads (one
    // 128-byte run per pixel and K block); NCHW: pixel pairs fastest
    const int g = NHWC ? (it & 7) : it / max(npairs, 1);
    const int px = NHWC ? (it >> 3) : 2 * (it - g * npairs), per_img = rows * a.w;
    const int il = px / per_img, rem = px - il * per_img;
    const int pr = rem / a.w, col = rem - pr * a.w;
    const bool ok = it < itotal && img0 + il < a.n;
    if constexpr (NHWC)
      p_src[j] = ok ? ((((uint32_t)(img0 + il) * (uint32_t)a.h + (uint32_t)(r0 + pr)) * (uint32_t)a.w +
                        (uint32_t)col) * (uint32_t)a.cin + 8u * g) * 2u
                    : OOB;
    else
      p_src[j] = ok ? ((((uint32_t)(img0 + il) * (uint32_t)a.cin + 8u * g) * (uint32_t)a.h + (uint32_t)(r0 + pr)) *
                           (uint32_t)a.w + (uint32_t)col) * 2u
                    : OOB;
    const int rl = r0 + pr - qh0 + 1, cl = col + 1;
    const int prow = (il * hrows + rl) * hww + cl, pv = (il * a.qbh + rl - 1) * a.w + cl;
    p_lds[j] = ok ? prow * RB + 16 * (g ^ slot_sw(pv)) : -1;
    p_lds_hi[j] = (prow + 1) * RB + 16 * (g ^ slot_sw(pv + 1));
  }
  // NCHW: P[j][k] is channel 8g + k of a pixel pair; NHWC: P[j][0..3] the 8
  // channels of one pixel
  auto load_pieces = [&](int cb, uint32_t (&P)[MAXP][8]) {
    const uint32_t cbo = NHWC ? (uint32_t)cb * 128u : (uint32_t)cb * 64u * plane_b;
#pragma unroll
    for (int j = 0; j < MAXP; ++j) {
      if (j * NTG >= itotal) break;  // the same for the whole group
      if constexpr (NHWC) {
        const uint4 v = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(xr, p_src[j], cbo, 0));
        P[j][0] = v.x;
        P[j][1] = v.y;
        P[j][2] = v.z;
        P[j][3] = v.w;
      } else {
#pragma unroll
        for (int k = 0; k < 8; ++k)
          P[j][k] = __builtin_amdgcn_raw_buffer_load_b32(xr, p_src[j], cbo + (uint32_t)k * plane_b, 0);
      }
    }
  };
  auto store_pieces = [&](char* tile, const uint32_t (&P)[MAXP][8]) {
#pragma unroll
    for (int j = 0; j < MAXP; ++j) {
      if (j * NTG >= itotal) break;
      if (p_lds[j] < 0) continue;
      if constexpr (NHWC) {
        *(uint4*)(tile + p_lds[j]) = make_uint4(P[j][0], P[j][1], P[j][2], P[j][3]);
        continue;
      }
      // P[j][k] holds channel 8g + k of the pixel pair: low half the first
      // pixel, high half the second
      uint32_t lo[4], hi[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo[e] = __builtin_amdgcn_perm(P[j][2 * e + 1], P[j][2 * e], 0x05040100u);
        hi[e] = __builtin_amdgcn_perm(P[j][2 * e + 1], P[j][2 * e], 0x07060302u);
      }
      *(uint4*)(tile + p_lds[j]) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
      *(uint4*)(tile + p_lds_hi[j]) = make_uint4(hi[0], hi[1], hi[2], hi[3]);
    }
  };

  // This wave's pixels: q = 32 i + lane % 32; LDS byte offset and virtual
  // index pv of its halo pixel at tap offset (0, 0).  The lane half h reads
  // K groups 4h + c (c = 0..3), at slots (4h + c) ^ sw(pv + tap delta).
  int lrow[NP], lpv[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int q = 32 * i + (lane & 31);
    const int per_img = a.qbh * a.w;
    const int il = q / per_img, qr = q - il * per_img;
    const int qh = qr / a.w, qw = qr - qh * a.w;
    lrow[i] = ((il * hrows + qh + 1) * hww + qw + 1) * RB;
    lpv[i] = (il * a.qbh + qh) * a.w + qw + 1;
  }
  const int hk = 4 * (lane >> 5);
  int tdelta[4], tdv[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    tdelta[t] = (a.dh[rho][t] * hww + a.dw[rho][t]) * RB;
    tdv[t] = a.dh[rho][t] * a.w + a.dw[rho][t];
  }

  // weight stage (K block cb, tap t) of this wave's 32-channel blocks
  const int ncb = a.cin / 64;
  const int cbn = ncb / KS, cb_lo = grp * cbn;
  const uint32_t kb32 = (uint32_t)(n0 / 32 + hc * WCH), nkb32 = (uint32_t)(a.cout_pad / 32);
  auto load_w = [&](uint4 (&W)[WCH][4], bool valid, int cb, int t) {
    const __amdgpu_buffer_rsrc_t ws = valid ? wr : wr0;
#pragma unroll
    for (int j = 0; j < WCH; ++j) {
      const uint32_t base =
          (((uint32_t)a.slot[rho][t] * nkb32 + kb32 + j) * (uint32_t)ncb + (uint32_t)cb) * 4096u;
#pragma unroll
      for (int c = 0; c < 4; ++c)
        W[j][c] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(ws, lane * 16, base + 1024u * c, 0));
    }
  };

  f32x16 acc[WCH][NP];
#pragma unroll
  for (int j = 0; j < WCH; ++j)
#pragma unroll
    for (int i = 0; i < NP; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][i][r] = 0.f;
  // the pixel fragments of one tap: 4 K steps of 16 channels x NP blocks
  auto read_frags = [&](const char* tile, int t, bf16x8 (&f)[4][NP]) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int i = 0; i < NP; ++i)
        f[c][i] = __builtin_bit_cast(
            bf16x8, *(const uint4*)(tile + lrow[i] + tdelta[t] + 16 * ((hk + c) ^ slot_sw(lpv[i] + tdv[t]))));
  };
  // one K step (16 channels) of a tap
  auto read_step = [&](const char* tile, int t, int c, bf16x8 (&f)[NP]) {
#pragma unroll
    for (int i = 0; i < NP; ++i)
      f[i] = __builtin_bit_cast(
          bf16x8, *(const uint4*)(tile + lrow[i] + tdelta[t] + 16 * ((hk + c) ^ slot_sw(lpv[i] + tdv[t]))));
  };
  auto mfma_step = [&](int c, const bf16x8 (&f)[NP], const uint4 (&W)[WCH][4]) {
#pragma unroll
    for (int j = 0; j < WCH; ++j) {
      const bf16x8 wv = __builtin_bit_cast(bf16x8, W[j][c]);
#pragma unroll
      for (int i = 0; i < NP; ++i)
        acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wv, f[i], acc[j][i], 0, 0, 0);
    }
  };
  auto mfmas = [&](const bf16x8 (&f)[4][NP], const uint4 (&W)[WCH][4]) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int j = 0; j < WCH; ++j) {
        const bf16x8 wv = __builtin_bit_cast(bf16x8, W[j][c]);
#pragma unroll
        for (int i = 0; i < NP; ++i)
          acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wv, f[c][i], acc[j][i], 0, 0, 0);
      }
  };

  char* const tiles = smem + grp * 2 * HALO_B;
  uint32_t P[MAXP][8];
  uint4 W[DEPTH][WCH][4];
  // the first K block's loads go out before the barrier (they only fill
  // registers), so their latency overlaps the LDS clear and the launch of
  // the workgroup's other waves
  load_pieces(cb_lo, P);
#pragma unroll
  for (int d = 0; d < DEPTH; ++d) load_w(W[d], d / 4 < cbn, cb_lo + min(d / 4, cbn - 1), d % 4);
  __syncthreads();  // halo tiles zeroed
  store_pieces(tiles, P);
  __syncthreads();
  if (cbn > 1) load_pieces(cb_lo + 1, P);
  for (int cb0 = 0; cb0 < cbn; cb0 += U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int cbi = cb0 + u;
      if (U > 1 && cbi >= cbn) break;  // the same for the whole workgroup
      const char* tile = tiles + (cbi & 1) * HALO_B;
      if constexpr (!PF) {
        // recomputed per K block: hoisted, the 64 swizzled fragment
        // addresses would not fit the registers
#pragma unroll
        for (int i = 0; i < NP; ++i) __asm__ volatile("" : "+v"(lrow[i]), "+v"(lpv[i]));
      }
      auto next_w = [&](int t) {
        // the stage DEPTH taps later goes into the buffer just consumed,
        // issued here (not sunk below later taps' MFMAs by the scheduler)
        const int nb = cbi + (t + DEPTH) / 4;
        __builtin_amdgcn_sched_barrier(0);
        load_w(W[(4 * u + t) % DEPTH], nb < cbn, cb_lo + min(nb, cbn - 1), (t + DEPTH) % 4);
        __builtin_amdgcn_sched_barrier(0);
      };
      if constexpr (PF) {
        // Tap t's MFMAs run while tap t+1's pixel fragments are read from
        // LDS (two register sets): the LDS latency is exposed once per K
        // block rather than before every MFMA.
        auto step = [&](int t, const bf16x8 (&cur)[4][NP], bf16x8 (&nxt)[4][NP]) {
          if (t < 3) read_frags(tile, t + 1, nxt);
          __builtin_amdgcn_sched_barrier(0);
          mfmas(cur, W[(4 * u + t) % DEPTH]);
          next_w(t);
        };
        bf16x8 fa[4][NP], fb[4][NP];
        read_frags(tile, 0, fa);
        step(0, fa, fb);
        step(1, fb, fa);
        step(2, fa, fb);
        step(3, fb, fa);
      } else {
        // per tap, K step c+1's fragments are read while step c's MFMAs run
        // (two sets of NP fragments)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const uint4 (&Wt)[WCH][4] = W[(4 * u + t) % DEPTH];
          bf16x8 f0[NP], f1[NP];
          read_step(tile, t, 0, f0);
          read_step(tile, t, 1, f1);
          __builtin_amdgcn_sched_barrier(0);
          mfma_step(0, f0, Wt);
          read_step(tile, t, 2, f0);
          __builtin_amdgcn_sched_barrier(0);
          mfma_step(1, f1, Wt);
          read_step(tile, t, 3, f1);
          __builtin_amdgcn_sched_barrier(0);
          mfma_step(2, f0, Wt);
          mfma_step(3, f1, Wt);
          next_w(t);
        }
      }
      if (cbi + 1 < cbn) store_pieces(tiles + ((cbi + 1) & 1) * HALO_B, P);
      __syncthreads();
      if (cbi + 2 < cbn) load_pieces(cb_lo + cbi + 2, P);
    }
  }

  if constexpr (KS > 1) {
    // group 1's partial sums to LDS (lane-contiguous), group 0 adds them
    float* red = (float*)smem + rho * (WCH * NP * 16 * 64) + lane;
    if (grp == 1) {
#pragma unroll
      for (int j = 0; j < WCH; ++j)
#pragma unroll
        for (int i = 0; i < NP; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) red[((j * NP + i) * 16 + r) * 64] = acc[j][i][r];
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll
      for (int j = 0; j < WCH; ++j)
#pragma unroll
        for (int i = 0; i < NP; ++i)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[j][i][r] += red[((j * NP + i) * 16 + r) * 64];
    }
    __syncthreads();
  }

  // Interleave the phases in LDS: [channel][image][output row][output column]
  // of the workgroup's output block (2 qbh rows x 2w columns per image).
  const int obw = 2 * a.w, obh = 2 * a.qbh;
  // NCHW: [channel][position], cpo elements per channel (16-byte pad); NHWC:
  // [position][channel], 64 + 8 elements per position
  const int cpo = a.ni * obh * obw + 8;
  constexpr int PPITCH = 64 + 8;
  uint16_t* so = (uint16_t*)smem;
  if (tid < 64) s_bias[tid] = bias_r;
  __syncthreads();
  if (grp == 0) {
    const int rho_h = rho >> 1, rho_w = rho & 1;
    // this lane's bias values (channels 8g + 4 (lane / 32) + 0..3 of each
    // 32-channel block) and output positions, all read before any store
    float bv[WCH][16];
#pragma unroll
    for (int j = 0; j < WCH; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float4 b4 = *(const float4*)(s_bias + (hc * WCH + j) * 32 + 8 * g + 4 * (lane >> 5));
        bv[j][4 * g] = b4.x;
        bv[j][4 * g + 1] = b4.y;
        bv[j][4 * g + 2] = b4.z;
        bv[j][4 * g + 3] = b4.w;
      }
    int pos[NP];
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      const int q = 32 * i + (lane & 31);
      const int per_img = a.qbh * a.w;
      const int il = q / per_img, qr = q - il * per_img;
      const int qh = qr / a.w, qw = qr - qh * a.w;
      pos[i] = (il * obh + 2 * qh + rho_h) * obw + 2 * qw + rho_w;
    }
    if constexpr (NHWC) {
      // rows 4g .. 4g + 3 of a lane are four consecutive channels of one
      // output position: one 8-byte write of the packed pairs
#pragma unroll
      for (int j = 0; j < WCH; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int ch = (hc * WCH + j) * 32 + 8 * g + 4 * (lane >> 5);
#pragma unroll
          for (int i = 0; i < NP; ++i) {
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = activate(acc[j][i][4 * g + e] + bv[j][4 * g + e], a.act);
            *(uint2*)(so + pos[i] * PPITCH + ch) =
                make_uint2(pack_bf16x2_rne(v[0], v[1]), pack_bf16x2_rne(v[2], v[3]));
          }
        }
    } else {
#pragma unroll
      for (int j = 0; j < WCH; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int ch = (hc * WCH + j) * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
#pragma unroll
          for (int i = 0; i < NP; ++i)
            so[ch * cpo + pos[i]] = f32_to_bf16_rne(activate(acc[j][i][r] + bv[j][r], a.act));
        }
    }
  }
  __syncthreads();
  // Whole output rows: per (channel, image) the rows [2 qh0, 2 qh0 + obh)
  // are one contiguous run of obh * obw elements in y.
  if constexpr (NHWC) {
    // each output pixel's bn channels are one run of y: 16-byte pieces,
    // the pieces of a pixel on neighbouring threads
    const int pieces = bn / 8, npx = a.ni * obh * obw;
    for (int e = tid; e < npx * pieces; e += NT) {
      const int pc = e % pieces, px = e / pieces;
      const int il = px / (obh * obw), rem = px - il * (obh * obw);
      const int oy = rem / obw, ox = rem - oy * obw;
      if (n0 + 8 * pc >= a.cout || img0 + il >= a.n) continue;
      const uint4 v = *(const uint4*)(so + px * PPITCH + 8 * pc);
      uint16_t* dst = (uint16_t*)a.y +
                      (((size_t)(img0 + il) * (2 * a.h) + 2 * qh0 + oy) * obw + ox) * a.cout + n0 + 8 * pc;
      store_stream16(dst, v);
    }
    return;
  }
  const int run8 = obh * obw / 8;
  const int total = bn * a.ni * run8;
  const size_t plane_o = (size_t)(2 * a.h) * (size_t)obw;
  for (int e = tid; e < total; e += NT) {
    const int k8 = e % run8, t2 = e / run8;
    const int il = t2 % a.ni, ch = t2 / a.ni;
    if (n0 + ch >= a.cout || img0 + il >= a.n) continue;
    const uint4 v = *(const uint4*)(so + ch * cpo + il * obh * obw + 8 * k8);
    uint16_t* dst = (uint16_t*)a.y + ((size_t)(img0 + il) * a.cout + n0 + ch) * plane_o +
                    (size_t)(2 * qh0) * obw + 8 * k8;
    store_stream16(dst, v);
  }
}

// ---------------------------------------------------------------------------
// Split-K reduction: the K slices' fp32 partial outputs added in slice order
// (deterministic), then bias, activation and the output dtype.
template <bool BF16>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(SplitKArgs a) {
  for (uint32_t i = blockIdx.x * 256u + threadIdx.x; i < a.total; i += gridDim.x * 256u) {
    float v = 0.f;
    for (int s = 0; s < a.ksplit; ++s) v += a.part[(size_t)s * a.stride + i];
    const uint32_t ch = a.nchw ? (i / (uint32_t)a.hw) % (uint32_t)a.cout : i % (uint32_t)a.cout;
    if (a.bias) {
      const uint32_t bc = ch / (uint32_t)a.bias_div;
      v += a.bias[a.bias_mod > 0 ? bc % (uint32_t)a.bias_mod : bc];
    }
    v = activate(v, a.act);
    if constexpr (BF16)
      ((uint16_t*)a.y)[i] = f32_to_bf16_rne(v);
    else
      ((float*)a.y)[i] = v;
  }
}

hipError_t launch_splitk_reduce(const SplitKArgs& a, int dtype, hipStream_t stream) {
  const uint32_t blocks = std::min<uint32_t>((a.total + 255u) / 256u, 4096u);
  if (dtype == 1)
    hipLaunchKernelGGL(splitk_reduce_kernel<true>, dim3(blocks), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(splitk_reduce_kernel<false>, dim3(blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Gather of the per-tap products into the transposed-conv output (section
// 3.1's relation read from the output side: output o takes tap m iff
// o + pad - m*dil is a multiple of the stride, reading input (o + pad -
// m*dil) / stride).  One thread per output element, taps in a fixed order.
__global__ __launch_bounds__(256) void taps_combine_kernel(CombArgs a) {
  const uint32_t total = (uint32_t)a.n * a.cout * a.ho * a.wo;
  for (uint32_t i = blockIdx.x * 256u + threadIdx.x; i < total; i += gridDim.x * 256u) {
    const int ow = (int)(i % (uint32_t)a.wo);
    uint32_t t = i / (uint32_t)a.wo;
    const int oh = (int)(t % (uint32_t)a.ho);
    t /= (uint32_t)a.ho;
    const int k = (int)(t % (uint32_t)a.cout);
    const int img = (int)(t / (uint32_t)a.cout);
    float v = a.bias ? a.bias[k] : 0.f;
    for (int m = 0; m < a.r; ++m) {
      const int uh = oh + a.pad_h - m * a.dil_h;
      if (uh < 0 || uh % a.stride_h != 0) continue;
      const int ih = uh / a.stride_h;
      if (ih >= a.h) continue;
      for (int q = 0; q < a.s; ++q) {
        const int uw = ow + a.pad_w - q * a.dil_w;
        if (uw < 0 || uw % a.stride_w != 0) continue;
        const int iw = uw / a.stride_w;
        if (iw >= a.w) continue;
        const size_t zc = ((size_t)img * a.cout + k) * a.r * a.s + (size_t)m * a.s + q;
        v += a.z[(zc * a.h + ih) * a.w + iw];
      }
    }
    a.y[i] = activate(v, a.act);
  }
}

hipError_t launch_taps_combine(const CombArgs& a, hipStream_t stream) {
  const uint32_t total = (uint32_t)a.n * a.cout * a.ho * a.wo;
  const uint32_t blocks = std::min<uint32_t>((total + 255u) / 256u, 8192u);
  hipLaunchKernelGGL(taps_combine_kernel, dim3(blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Receptive-field gather for a conv with few input channels (Algorithm 2's
// gather, stored per output pixel as one GEMM row).  One thread per element
// of xs, so the stores are contiguous.
template <typename T>
__global__ __launch_bounds__(256) void gather_taps_kernel(GatherArgs a) {
  // 16 bytes of one pixel's row per thread (c_stride is a multiple of VEC)
  constexpr int VEC = 16 / (int)sizeof(T);
  const int cv = a.c_stride / VEC;
  const uint32_t total = (uint32_t)a.n * a.ho * a.wo * cv;
  const int rs = a.r * a.s, kk = a.cin * rs;
  for (uint32_t i = blockIdx.x * 256u + threadIdx.x; i < total; i += gridDim.x * 256u) {
    const int j0 = (int)(i % (uint32_t)cv) * VEC;
    const uint32_t pix = i / (uint32_t)cv;
    const int ow = (int)(pix % (uint32_t)a.wo);
    const uint32_t t = pix / (uint32_t)a.wo;
    const int oh = (int)(t % (uint32_t)a.ho), img = (int)(t / (uint32_t)a.ho);
    T v[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const int j = j0 + e;
      v[e] = T(0);
      if (j < kk) {
        const int c = j / rs, mq = j - c * rs, m = mq / a.s, q = mq - m * a.s;
        const int ih = oh * a.stride_h - a.pad_h + m * a.dil_h;
        const int iw = ow * a.stride_w - a.pad_w + q * a.dil_w;
        if (ih >= 0 && ih < a.h && iw >= 0 && iw < a.w)
          v[e] = ((const T*)a.x)[(((size_t)img * a.cin + c) * a.h + ih) * a.w + iw];
      }
    }
    *(uint4*)((T*)a.xs + (size_t)pix * a.c_stride + j0) = *(const uint4*)v;
  }
}

hipError_t launch_gather_taps(const GatherArgs& a, int dtype, hipStream_t stream) {
  const int vec = dtype == 1 ? 8 : 4;
  const uint32_t total = (uint32_t)a.n * a.ho * a.wo * (uint32_t)(a.c_stride / vec);
  const uint32_t blocks = std::min<uint32_t>((total + 255u) / 256u, 8192u);
  if (dtype == 1)
    hipLaunchKernelGGL(gather_taps_kernel<uint16_t>, dim3(blocks), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(gather_taps_kernel<uint32_t>, dim3(blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Grouped and depthwise convolutions (see GrArgs).
template <typename T>
__device__ __forceinline__ float to_f32(T v) {
  if constexpr (std::is_same<T, uint16_t>::value)
    return __uint_as_float((uint32_t)v << 16);
  else
    return __uint_as_float(v);
}

template <typename T>
__global__ __launch_bounds__(256) void grouped_kernel(GrArgs a, long long total) {
  const T* __restrict__ x = (const T*)a.x;
  const T* __restrict__ w = (const T*)a.w;
  const int cig = a.cin / a.groups, cog = a.cout / a.groups;
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    long long t = idx;
    int k, oh, ow, n;
    if (a.nhwc) {
      k = (int)(t % a.cout);
      t /= a.cout;
      ow = (int)(t % a.wo);
      t /= a.wo;
      oh = (int)(t % a.ho);
      n = (int)(t / a.ho);
    } else {
      ow = (int)(t % a.wo);
      t /= a.wo;
      oh = (int)(t % a.ho);
      t /= a.ho;
      k = (int)(t % a.cout);
      n = (int)(t / a.cout);
    }
    const int g = k / cog, kg = k - g * cog, c0 = g * cig;
    float acc = 0.f;
    for (int m = 0; m < a.r; ++m) {
      int ih;
      if (a.transposed) {
        const int num = oh + a.pad_h - m * a.dil_h;  // = ih * stride_h on the phase's taps
        if (num < 0 || num % a.stride_h != 0) continue;
        ih = num / a.stride_h;
      } else {
        ih = oh * a.stride_h - a.pad_h + m * a.dil_h;
      }
      if (ih < 0 || ih >= a.h) continue;
      for (int q = 0; q < a.s; ++q) {
        int iw;
        if (a.transposed) {
          const int num = ow + a.pad_w - q * a.dil_w;
          if (num < 0 || num % a.stride_w != 0) continue;
          iw = num / a.stride_w;
        } else {
          iw = ow * a.stride_w - a.pad_w + q * a.dil_w;
        }
        if (iw < 0 || iw >= a.w_) continue;
        for (int ci = 0; ci < cig; ++ci) {
          const int c = c0 + ci;
          const size_t xi = a.nhwc ? (((size_t)n * a.h + ih) * a.w_ + iw) * a.cin + c
                                   : (((size_t)n * a.cin + c) * a.h + ih) * a.w_ + iw;
          const size_t wi = a.transposed ? (((size_t)c * cog + kg) * a.r + m) * a.s + q
                                         : (((size_t)k * cig + ci) * a.r + m) * a.s + q;
          acc = fmaf(to_f32(x[xi]), to_f32(w[wi]), acc);
        }
      }
    }
    const float v = activate(acc + (a.bias ? a.bias[k] : 0.f), a.act);
    if constexpr (std::is_same<T, uint16_t>::value)
      ((uint16_t*)a.y)[idx] = f32_to_bf16_rne(v);
    else
      ((float*)a.y)[idx] = v;
  }
}

hipError_t launch_grouped(const GrArgs& a, int dtype, hipStream_t stream) {
  const long long total = (long long)a.n * a.cout * a.ho * a.wo;
  const long long want = (total + 255) / 256;
  const int grid = (int)(want < 1048576 ? want : 1048576);
  if (total == 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(grouped_kernel<uint16_t>, dim3(grid), dim3(256), 0, stream, a, total);
  else
    hipLaunchKernelGGL(grouped_kernel<uint32_t>, dim3(grid), dim3(256), 0, stream, a, total);
  return hipGetLastError();
}

hipError_t launch_quad(const QArgs& a, hipStream_t stream) {
  const dim3 grid(a.ntiles * a.igroups * a.hblocks);
#define HUGE2_QUAD_LAUNCH(KS_, WCH_, D_, NP_)                                                  \
  do {                                                                                        \
    if (a.nhwc)                                                                               \
      hipLaunchKernelGGL((quad_kernel<KS_, WCH_, D_, NP_, true>), grid, dim3(kQuadThreads), 0, \
                         stream, a);                                                          \
    else                                                                                      \
      hipLaunchKernelGGL((quad_kernel<KS_, WCH_, D_, NP_, false>), grid, dim3(kQuadThreads), 0, \
                         stream, a);                                                          \
  } while (0)
  if (a.np == 4) {
    // two weight stages in flight: the registers hold no more
    if (a.ks == 2) HUGE2_QUAD_LAUNCH(2, 1, 2, 4);
    else HUGE2_QUAD_LAUNCH(1, 1, 2, 4);
  } else if (a.ks == 2 && a.nch == 2) {
    HUGE2_QUAD_LAUNCH(2, 2, 2, 2);  // both channel blocks per wave: two stages fit the registers
  } else if (a.ks == 2) {
    if (a.depth == 2) HUGE2_QUAD_LAUNCH(2, 1, 2, 2);
    else HUGE2_QUAD_LAUNCH(2, 1, 4, 2);
  } else {
    if (a.depth == 2) HUGE2_QUAD_LAUNCH(1, 1, 2, 2);
    else HUGE2_QUAD_LAUNCH(1, 1, 4, 2);
  }
#undef HUGE2_QUAD_LAUNCH
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight packing: element (slot, k, c) = w at kernel tap slot = (kh, kw),
// output channel k, input channel c.
//   lane_kb = 0: K-contiguous rows, wp[slot][k][c].
//   lane_kb = kPackKB (or the all-phase kernel's 128): the lane order of the
//     split-wave GEMM's own-operand loads: per (slot, 32-channel block, K
//     block of lane_kb bytes) a block of 32 rows x lane_kb bytes stored as
//     [chunk c16 < lane_kb/32][lane < 64][16 bytes], lane = 32 * (byte /
//     (lane_kb/2)) + row, so that one 16-byte load per lane reads 1 KB
//     contiguous.

template <typename T>
__global__ void pack_weights_kernel(const T* __restrict__ w, T* __restrict__ wp, bool transposed,
                                    int cin, int cout, int r, int s, int cin_pad, int cout_pad,
                                    int lane_kb, long long total, int prod_rs) {
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(idx % cin_pad);
    const long long t = idx / cin_pad;
    const int k = (int)(t % cout_pad);
    const int slot = (int)(t / cout_pad);
    const int kh = slot / s, kw = slot - kh * s;
    T v = T(0);
    if (c < cin && k < cout) {
      long long src;
      if (prod_rs > 0) {  // column k = tap * (cout / prod_rs) + channel
        const int co = cout / prod_rs, tap = k / co;
        src = ((long long)c * co + (k - tap * co)) * prod_rs + tap;
      } else {
        src = transposed ? (((long long)c * cout + k) * r + kh) * s + kw
                         : (((long long)k * cin + c) * r + kh) * s + kw;
      }
      v = w[src];
    }
    long long dst = idx;
    if (lane_kb > 0) {
      const int kc = lane_kb / (int)sizeof(T);          // K elements per stage
      const int e = (c % kc) * (int)sizeof(T);          // byte within the stage row
      const int h = e / (lane_kb / 2), c16 = (e % (lane_kb / 2)) / 16, bo = e % 16;
      const long long blk = (long long)slot * (cout_pad / 32) + k / 32;
      const long long byte = ((blk * (cin_pad / kc) + c / kc) * (lane_kb / 32) + c16) * 1024 +
                             (h * 32 + k % 32) * 16 + bo;
      dst = byte / (long long)sizeof(T);
    }
    wp[dst] = v;
  }
}

hipError_t launch_pack_weights(const void* w, void* wp, int dtype, bool transposed, int cin,
                               int cout, int r, int s, int cin_pad, int cout_pad, int lane_kb,
                               hipStream_t stream, int prod_rs) {
  const long long total = (long long)r * s * cout_pad * cin_pad;
  const int block = 256;
  const long long want = (total + block - 1) / block;
  const int grid = (int)(want < 65536 ? want : 65536);
  if (total == 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(pack_weights_kernel<uint16_t>, dim3(grid), dim3(block), 0, stream,
                       (const uint16_t*)w, (uint16_t*)wp, transposed, cin, cout, r, s, cin_pad,
                       cout_pad, lane_kb, total, prod_rs);
  else
    hipLaunchKernelGGL(pack_weights_kernel<uint32_t>, dim3(grid), dim3(block), 0, stream,
                       (const uint32_t*)w, (uint32_t*)wp, transposed, cin, cout, r, s, cin_pad,
                       cout_pad, lane_kb, total, prod_rs);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight gradient (section 3.2.3).  The error maps (or, for a strided conv,
// the input) are untangled into copies on the small tensor's pixel grid, so
// that every tap's gradient is a dense product over pixels with no zero
// products; all taps run as one GEMM on MFMA with both operands K-contiguous.

// Staging of one image chunk: St (the image and channel axes exchanged) and
// Bt (the tap gather), zero up to kp.  A thread produces 8 consecutive k of
// one row and writes them with one 16-byte store (kp is a multiple of 64).
// When rows of the small grid are a multiple of 8 (the usual case), the 8 k
// lie in one row: St takes one 16-byte load, Bt one row of the big tensor at
// the stride; otherwise each element is located on its own.  Indices fit 32
// bits (the staged buffers stay below 2^31 bytes).
template <typename T>
__global__ __launch_bounds__(256) void wgrad_stage_kernel(WgArgs a) {
  constexpr int V = 8;
  const uint32_t hws = (uint32_t)a.hs * (uint32_t)a.ws;
  const uint32_t kreal = (uint32_t)a.nimg * hws;
  const uint32_t kv = (uint32_t)a.kp / V;
  const uint32_t st_total = a.direct ? 0u : (uint32_t)a.ms * kv;  // (read in place: no St)
  // (with the LDS gather, Bt is wgrad_gather_kernel's)
  const uint32_t total = st_total + (a.gather_ib > 0 ? 0u : (uint32_t)(a.r * a.s * a.nb) * kv);
  const bool rows8 = a.ws % V == 0;
  // the 8 k of a piece lie in one image (hws % 8 == 0): contiguous in the
  // small tensor; rows of 1, 2 or 4 pixels (8 % ws == 0) are whole rows of
  // the big tensor's gather
  const bool img8 = hws % V == 0;
  const bool short_rows = img8 && !rows8 && V % a.ws == 0;
  const int lg_ws = a.ws == 1 ? 0 : a.ws == 2 ? 1 : 2;
  const T* sm = (const T*)a.sm;
  const T* bg = (const T*)a.bg;
  for (uint32_t e = blockIdx.x * blockDim.x + threadIdx.x; e < total; e += gridDim.x * blockDim.x) {
    T v[V];
    const bool is_st = e < st_total;
    const uint32_t f = is_st ? e : e - st_total;
    const uint32_t row = f / kv, k0 = (f - row * kv) * V;
    T* dst = (is_st ? (T*)a.st : (T*)a.bt) + (size_t)row * a.kp + k0;
    const uint32_t il0 = k0 / hws, q0 = k0 - il0 * hws;
    const uint32_t qh0 = q0 / (uint32_t)a.ws, qw0 = q0 - qh0 * (uint32_t)a.ws;
    if (is_st) {
      const size_t base = ((size_t)(a.img0 + il0) * a.ms + row) * hws;
      if (img8 && k0 < kreal) {
        __builtin_memcpy(v, sm + base + q0, sizeof(v));
      } else {
#pragma unroll
        for (int t = 0; t < V; ++t) {
          const uint32_t k = k0 + t, il = k / hws, q = k - il * hws;
          v[t] = k < kreal ? sm[((size_t)(a.img0 + il) * a.ms + row) * hws + q] : T(0);
        }
      }
    } else {
      const int tap = (int)(row % (uint32_t)(a.r * a.s)), n = (int)(row / (uint32_t)(a.r * a.s));
      const int kh = tap / a.s, kw = tap - kh * a.s;
      if (rows8 && k0 < kreal) {
        const int ih = (int)qh0 * a.stride_h - a.pad_h + kh * a.dil_h;
        const int iw0 = (int)qw0 * a.stride_w - a.pad_w + kw * a.dil_w;
        const bool row_in = ih >= 0 && ih < a.hb;
        const T* src = bg + (((size_t)(a.img0 + il0) * a.nb + n) * a.hb + (row_in ? ih : 0)) * a.wb;
#pragma unroll
        for (int t = 0; t < V; ++t) {
          const int iw = iw0 + t * a.stride_w;
          v[t] = (row_in && iw >= 0 && iw < a.wb) ? src[iw] : T(0);
        }
      } else if (short_rows && k0 < kreal) {
        const T* src = bg + ((size_t)(a.img0 + il0) * a.nb + n) * a.hb * a.wb;
#pragma unroll
        for (int t = 0; t < V; ++t) {
          const int qh = (int)qh0 + (t >> lg_ws), qw = t & (a.ws - 1);
          const int ih = qh * a.stride_h - a.pad_h + kh * a.dil_h;
          const int iw = qw * a.stride_w - a.pad_w + kw * a.dil_w;
          const bool in = ih >= 0 && ih < a.hb && iw >= 0 && iw < a.wb;
          v[t] = in ? src[in ? ih * a.wb + iw : 0] : T(0);
        }
      } else {
#pragma unroll
        for (int t = 0; t < V; ++t) {
          const uint32_t k = k0 + t;
          v[t] = T(0);
          if (k < kreal) {
            const uint32_t il = k / hws, q = k - il * hws;
            const int qh = (int)(q / (uint32_t)a.ws), qw = (int)(q - (uint32_t)qh * (uint32_t)a.ws);
            const int ih = qh * a.stride_h - a.pad_h + kh * a.dil_h;
            const int iw = qw * a.stride_w - a.pad_w + kw * a.dil_w;
            if (ih >= 0 && ih < a.hb && iw >= 0 && iw < a.wb)
              v[t] = bg[(((size_t)(a.img0 + il) * a.nb + n) * a.hb + ih) * a.wb + iw];
          }
        }
      }
    }
#pragma unroll
    for (int t = 0; t < V; t += 16 / (int)sizeof(T)) {
      uint4 u;
      __builtin_memcpy(&u, &v[t], 16);
      *(uint4*)(dst + t) = u;
    }
  }
}

// Byte offsets of the GEMM's St operand: row m, and K stage ks of KC
// elements.  Staged, St is [ms][kp]; read in place (a.direct: hs*ws a
// multiple of 64, so a stage lies in one image) stage ks is image
// k / (hs*ws) of the chunk at pixel k mod (hs*ws) of channel m's plane.
__device__ __forceinline__ size_t wgrad_a_row(const WgArgs& a, int m, int esz) {
  const size_t hws = (size_t)a.hs * a.ws;
  return a.direct ? ((size_t)a.img0 * a.ms + m) * hws * esz : (size_t)m * a.kp * esz;
}
__device__ __forceinline__ size_t wgrad_a_stage(const WgArgs& a, int ks, int kc, int esz) {
  if (!a.direct) return (size_t)ks * kc * esz;
  const uint32_t k = (uint32_t)ks * kc, hws = (uint32_t)a.hs * a.ws;
  const uint32_t il = fast_div(k, a.hws_mul, a.hws_shift);
  return ((size_t)il * a.ms * hws + (k - il * hws)) * esz;
}

// Byte offsets of the GEMM's Bt operand: column c = (n, tap), and K stage
// ks.  Per-tap rows: row c of kp elements.  Phase planes (a.bt_phase, hs*ws
// a multiple of 64 so that a stage lies in one image): tap (kh, kw) of n
// reads plane (ph, kw) of n from row sh - sh_min of each image's hr rows.
__device__ __forceinline__ size_t wgrad_b_row(const WgArgs& a, int c, int esz) {
  if (!a.bt_phase) return (size_t)c * a.kp * esz;
  const int n = c / a.g_taps, tap = c - n * a.g_taps, kh = tap / a.g_s, kw = tap - kh * a.g_s;
  const int rs = kh * a.dil_h - a.pad_h;
  const int sh = floor_div_d(rs, a.stride_h), ph = rs - sh * a.stride_h;
  const size_t rowlen = (size_t)a.nimg * a.hr * a.ws;
  return (((size_t)n * a.stride_h * a.g_s + ph * a.g_s + kw) * rowlen + (size_t)(sh - a.sh_min) * a.ws) *
         esz;
}
__device__ __forceinline__ size_t wgrad_b_stage(const WgArgs& a, int ks, int kc, int esz) {
  if (!a.bt_phase) return (size_t)ks * kc * esz;
  const uint32_t k = (uint32_t)ks * kc, hws = (uint32_t)a.hs * a.ws;
  const uint32_t il = fast_div(k, a.hws_mul, a.hws_shift);
  return ((size_t)il * a.hr * a.ws + (k - il * hws)) * esz;
}

// Tile of a weight-gradient GEMM workgroup: the grid's (m block, n block,
// tap + taps * split) in that order of the linear workgroup index, each XCD
// taking a contiguous run of it (xcd_remap), so that the m blocks that read
// one Bt tile, and the taps that read one St tile, share an L2.
__device__ __forceinline__ void wgrad_block(int& bx, int& by, int& bz) {
  const int nx = gridDim.x, ny = gridDim.y;
  int b = xcd_remap(blockIdx.x + nx * (blockIdx.y + ny * blockIdx.z), nx * ny * gridDim.z);
  bx = b % nx;
  b /= nx;
  by = b % ny;
  bz = b / ny;
}

// The GEMM of all taps at once: column c = n * taps + tap of G is Bt's row
// (n, tap), so that G[m][c] is dw's element (m, n, tap) and a big tensor
// with few channels is not padded to a tile per tap.
// G[m][c] (+)= sum_k St[m][k] * Bt[c][k]: a 64 x 64 tile per
// workgroup of 4 waves (32 x 32 each), K in 128-byte stages through LDS,
// double buffered, the next stage's loads in registers while this one
// multiplies.  K order inside a stage is permuted identically for both
// operands (lane half h takes the stage's h-th half), as in the phase GEMM.
template <bool BF16>
__global__ __launch_bounds__(256) void wgrad_gemm_kernel(WgArgs a) {
  constexpr int ESZ = BF16 ? 2 : 4;
  constexpr int KB = 128, KC = KB / ESZ, ROWB = KB + 16;
  constexpr int STAGE_B = 2 * 64 * ROWB;
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE_B];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;
  const int taps = a.r * a.s;
  int bx, by, bz;
  wgrad_block(bx, by, bz);
  const int m0 = bx * 64, n0 = by * 64, tap = bz % taps;
  const int split = bz / taps;
  // this thread's two rows of each operand (rows past the end repeat the last)
  const int chunk = tid & 7, row = tid >> 3;  // 8 chunks of 16 bytes per row
  const char* const st = (const char*)(a.direct ? a.sm : a.st);
  const char* const bt = (const char*)a.bt;
  const size_t a0 = wgrad_a_row(a, min(m0 + row, a.ms - 1), ESZ) + chunk * 16;
  const size_t a1 = wgrad_a_row(a, min(m0 + row + 32, a.ms - 1), ESZ) + chunk * 16;
  const size_t b0 = wgrad_b_row(a, tap * a.nb + min(n0 + row, a.nb - 1), ESZ) + chunk * 16;
  const size_t b1 = wgrad_b_row(a, tap * a.nb + min(n0 + row + 32, a.nb - 1), ESZ) + chunk * 16;
  struct Regs {
    uint4 a0, a1, b0, b1;
  };
  auto load = [&](int ks) {
    const size_t off = wgrad_b_stage(a, ks, KC, ESZ), aoff = wgrad_a_stage(a, ks, KC, ESZ);
    Regs r;
    r.a0 = *(const uint4*)(st + a0 + aoff);
    r.a1 = *(const uint4*)(st + a1 + aoff);
    r.b0 = *(const uint4*)(bt + b0 + off);
    r.b1 = *(const uint4*)(bt + b1 + off);
    return r;
  };
  auto store = [&](int buf, const Regs& r) {
    char* as = smem + buf * STAGE_B;
    char* bs = as + 64 * ROWB;
    *(uint4*)(as + row * ROWB + chunk * 16) = r.a0;
    *(uint4*)(as + (row + 32) * ROWB + chunk * 16) = r.a1;
    *(uint4*)(bs + row * ROWB + chunk * 16) = r.b0;
    *(uint4*)(bs + (row + 32) * ROWB + chunk * 16) = r.b1;
  };
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
  auto compute = [&](int buf) {
    const char* as = smem + buf * STAGE_B + (wm * 32 + (lane & 31)) * ROWB + (lane >> 5) * (KB / 2);
    const char* bs = smem + buf * STAGE_B + (64 + wn * 32 + (lane & 31)) * ROWB + (lane >> 5) * (KB / 2);
    if constexpr (BF16) {
#pragma unroll
      for (int t = 0; t < KB / 32; ++t) {
        const bf16x8 va = __builtin_bit_cast(bf16x8, *(const uint4*)(as + 16 * t));
        const bf16x8 vb = __builtin_bit_cast(bf16x8, *(const uint4*)(bs + 16 * t));
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vb, va, acc, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int t4 = 0; t4 < KB / 32; ++t4) {
        const uint4 fa = *(const uint4*)(as + 16 * t4);
        const uint4 fb = *(const uint4*)(bs + 16 * t4);
        const uint32_t ea[4] = {fa.x, fa.y, fa.z, fa.w}, eb[4] = {fb.x, fb.y, fb.z, fb.w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(eb[e]), __uint_as_float(ea[e]), acc, 0, 0, 0);
      }
    }
  };
  // this split's K stages [k_lo, k_hi)
  const int nk_all = a.kp / KC;
  const int per = (nk_all + a.ksplit - 1) / a.ksplit;
  const int k_lo = min(split * per, nk_all), k_hi = min(k_lo + per, nk_all);
  if (k_hi > k_lo) {
    store(0, load(k_lo));
    __syncthreads();
    for (int ks = k_lo; ks < k_hi; ++ks) {
      // the next stage's loads (the first again past the end: unused)
      // overlap this stage's MFMAs
      const Regs nx = load(ks + 1 < k_hi ? ks + 1 : k_lo);
      compute((ks - k_lo) & 1);
      if (ks + 1 < k_hi) store((ks + 1 - k_lo) & 1, nx);
      __syncthreads();
    }
  }
  // acc: lane holds m = m0 + wm*32 + lane%32 (MFMA column: the St operand went
  // second) and n = n0 + wn*32 + 8*(r/4) + 4*(lane/32) + r%4 (rows)
  const int m = m0 + wm * 32 + (lane & 31);
  if (a.direct_out) {  // one K slice and one chunk: the gradient itself
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int n = n0 + wn * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      if (m >= a.ms || n >= a.nb) continue;
      const size_t d = (size_t)m * a.nb + n;
      if constexpr (BF16)
        ((uint16_t*)a.dw)[d] = f32_to_bf16_rne(acc[r]);
      else
        ((float*)a.dw)[d] = acc[r];
    }
    return;
  }
  float* gt = a.g + (((size_t)split * taps + tap) * a.ms + min(m, a.ms - 1)) * a.nb;
  const bool acc_in = a.accumulate != 0;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int n = n0 + wn * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
    const float v = acc[r];
    if (m < a.ms && n < a.nb) gt[n] = acc_in ? gt[n] + v : v;
  }
}

// The same product on 128 x 128 tiles: 4 waves of 64 x 64 (four
// accumulators each, so consecutive MFMAs do not wait for each other, and
// each fragment read from LDS feeds two MFMAs), two workgroups per compute
// unit.  The St fragments go first: a lane holds one output channel n of
// each 32 x 32 block, so the fp32 partial rows of G are written 128 bytes at
// a time.
template <bool BF16>
__global__ __launch_bounds__(256, 2) void wgrad_gemm2_kernel(WgArgs a) {
  constexpr int ESZ = BF16 ? 2 : 4;
  constexpr int KB = 128, KC = KB / ESZ, ROWB = KB + 16;
  constexpr int TM = 128, TN = 128;
  constexpr int STAGE_B = (TM + TN) * ROWB;
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE_B];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;
  const int taps = a.r * a.s;
  int bx, by, bz;
  wgrad_block(bx, by, bz);
  const int m0 = bx * TM, n0 = by * TN, tap = bz % taps;
  const int split = bz / taps;
  const int chunk = tid & 7, row = tid >> 3;  // 8 chunks of 16 bytes per row, 32 rows per pass
  const char* const st = (const char*)(a.direct ? a.sm : a.st);
  const char* const bt = (const char*)a.bt;
  // this thread's rows (rows past the end repeat the last: their products
  // are never stored)
  size_t ao[4], bo[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    ao[j] = wgrad_a_row(a, min(m0 + row + 32 * j, a.ms - 1), ESZ) + chunk * 16;
    bo[j] = wgrad_b_row(a, tap * a.nb + min(n0 + row + 32 * j, a.nb - 1), ESZ) + chunk * 16;
  }
  struct Regs {
    uint4 a[4], b[4];
  };
  auto load = [&](int ks, Regs& r) {
    const size_t off = wgrad_b_stage(a, ks, KC, ESZ), aoff = wgrad_a_stage(a, ks, KC, ESZ);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      r.a[j] = *(const uint4*)(st + ao[j] + aoff);
      r.b[j] = *(const uint4*)(bt + bo[j] + off);
    }
  };
  auto store = [&](int buf, const Regs& r) {
    char* as = smem + buf * STAGE_B;
    char* bs = as + TM * ROWB;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      *(uint4*)(as + (row + 32 * j) * ROWB + chunk * 16) = r.a[j];
      *(uint4*)(bs + (row + 32 * j) * ROWB + chunk * 16) = r.b[j];
    }
  };
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  auto compute = [&](int buf) {
    const char* as = smem + buf * STAGE_B + (wm * 64 + (lane & 31)) * ROWB + (lane >> 5) * (KB / 2);
    const char* bs =
        smem + buf * STAGE_B + (TM + wn * 64 + (lane & 31)) * ROWB + (lane >> 5) * (KB / 2);
#pragma unroll
    for (int t = 0; t < KB / 32; ++t) {
      uint4 fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        fa[i] = *(const uint4*)(as + 32 * i * ROWB + 16 * t);
        fb[i] = *(const uint4*)(bs + 32 * i * ROWB + 16 * t);
      }
      if constexpr (BF16) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                __builtin_bit_cast(bf16x8, fa[i]), __builtin_bit_cast(bf16x8, fb[j]), acc[i][j], 0, 0,
                0);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
              const uint32_t ea = e == 0 ? fa[i].x : e == 1 ? fa[i].y : e == 2 ? fa[i].z : fa[i].w;
              const uint32_t eb = e == 0 ? fb[j].x : e == 1 ? fb[j].y : e == 2 ? fb[j].z : fb[j].w;
              acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(ea), __uint_as_float(eb),
                                                               acc[i][j], 0, 0, 0);
            }
      }
    }
  };
  const int nk_all = a.kp / KC;
  const int per = (nk_all + a.ksplit - 1) / a.ksplit;
  const int k_lo = min(split * per, nk_all), k_hi = min(k_lo + per, nk_all);
  if (k_hi > k_lo) {
    // the split's stages from a start rotated by (column block, split):
    // the workgroups of one XCD do not stream the same power-of-two strided
    // rows at the same offsets in lockstep (the m blocks that share a Bt
    // tile keep the same order)
    const int nst = k_hi - k_lo, rot = ((bz * (int)gridDim.y + by) * 5) % nst;
    auto stage_of = [&](int i) {
      const int j = i + rot;
      return k_lo + (j >= nst ? j - nst : j);
    };
    Regs cur, nx;
    load(stage_of(0), cur);
    store(0, cur);
    __syncthreads();
    for (int i = 0; i < nst; ++i) {
      // the next stage's loads (the first again past the end: unused)
      // overlap this stage's MFMAs
      load(stage_of(i + 1 < nst ? i + 1 : 0), nx);
      compute(i & 1);
      if (i + 1 < nst) store((i + 1) & 1, nx);
      __syncthreads();
    }
  }
  // lane: n = n0 + wn*64 + 32 j + lane % 32; m = m0 + wm*64 + 32 i + 8 (r/4) + 4 (lane/32) + r%4
  const bool acc_in = a.accumulate != 0;
  const int n = n0 + wn * 64 + (lane & 31);
  if (a.direct_out) {  // one K slice and one chunk: the gradient itself
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * 64 + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (m >= a.ms) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          if (n + 32 * j >= a.nb) continue;
          const size_t d = (size_t)m * a.nb + n + 32 * j;
          if constexpr (BF16)
            ((uint16_t*)a.dw)[d] = f32_to_bf16_rne(acc[i][j][r]);
          else
            ((float*)a.dw)[d] = acc[i][j][r];
        }
      }
    return;
  }
  float* const gt = a.g + ((size_t)split * taps + tap) * a.ms * a.nb;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm * 64 + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
      if (m >= a.ms) continue;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        if (n + 32 * j >= a.nb) continue;
        float* gp = gt + (size_t)m * a.nb + n + 32 * j;
        *gp = acc_in ? *gp + acc[i][j][r] : acc[i][j][r];
      }
    }
}

// dw from the K slices of G (each in dw's layout), added in slice order and
// rounded to the dtype: a thread per element, reads and writes coalesced.
template <bool BF16>
__global__ __launch_bounds__(256) void wgrad_store_kernel(WgArgs a) {
  const uint32_t total = (uint32_t)a.ms * (uint32_t)a.nb * (uint32_t)(a.r * a.s);
  for (uint32_t e = blockIdx.x * blockDim.x + threadIdx.x; e < total; e += gridDim.x * blockDim.x) {
    float v = 0.f;
    for (int sp = 0; sp < a.ksplit; ++sp) v += a.g[(size_t)sp * total + e];
    if constexpr (BF16)
      ((uint16_t*)a.dw)[e] = f32_to_bf16_rne(v);
    else
      ((float*)a.dw)[e] = v;
  }
}

// The same for many K slices: a workgroup per 64 consecutive entries, wave w
// adding the slices w, w + 4, w + 8, ... in order (several loads in flight),
// then the four waves' sums added in wave order.
template <bool BF16>
__global__ __launch_bounds__(256) void wgrad_store_split_kernel(WgArgs a) {
  __shared__ float part[4][64];
  const uint32_t total = (uint32_t)a.ms * (uint32_t)a.nb * (uint32_t)(a.r * a.s);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t e = blockIdx.x * 64u + (uint32_t)lane;
  float v = 0.f;
  if (e < total) {
#pragma unroll 4
    for (int sp = wave; sp < a.ksplit; sp += 4) v += a.g[(size_t)sp * total + e];
  }
  part[wave][lane] = v;
  __syncthreads();
  if (wave != 0 || e >= total) return;
  const float sum = ((part[0][lane] + part[1][lane]) + part[2][lane]) + part[3][lane];
  if constexpr (BF16)
    ((uint16_t*)a.dw)[e] = f32_to_bf16_rne(sum);
  else
    ((float*)a.dw)[e] = sum;
}

static dim3 grid_for(long long total) {
  const long long want = (total + 255) / 256;
  return dim3((unsigned)(want < 65536 ? (want > 0 ? want : 1) : 65536));
}

// Bt through LDS (hs*ws a multiple of 8, a big-tensor plane within
// kWgGatherLds): workgroup (n, block of gather_ib images of the chunk) reads
// the block's planes big[img][n] whole and coalesced, then writes for every
// tap the block's run of row (n, tap), runs of 4 bytes of consecutive k per
// thread (coalesced across the lanes), the last block also the zero padding
// up to kp.  The strided gather then reads LDS, where
// the plain staging kernel's reads of the big tensor were scattered 2-byte
// loads across planes.
template <typename T>
__global__ __launch_bounds__(256) void wgrad_gather_kernel(WgArgs a) {
  extern __shared__ __attribute__((aligned(16))) char s_raw[];
  T* const s_pl = (T*)s_raw;
  const int n = (int)(blockIdx.x % (unsigned)a.nb);
  const int il0 = (int)(blockIdx.x / (unsigned)a.nb) * a.gather_ib;
  const int nim = min(a.gather_ib, a.nimg - il0);
  const int plane = a.hb * a.wb, hws = a.hs * a.ws;
  const T* bg = (const T*)a.bg;
  constexpr int VE = 16 / (int)sizeof(T);
  // the block's planes, all images in one loop (independent loads in flight)
  const T* src0 = bg + ((size_t)(a.img0 + il0) * a.nb + n) * plane;
  const size_t img_stride = (size_t)a.nb * plane;
  if (plane % VE == 0 && ((uintptr_t)bg & 15) == 0) {
    const int per = plane / VE;
#pragma unroll 4
    for (int e = threadIdx.x; e < nim * per; e += 256) {
      const int il = e / per, r = e - il * per;
      ((uint4*)s_pl)[e] = ((const uint4*)(src0 + il * img_stride))[r];
    }
  } else {
#pragma unroll 4
    for (int e = threadIdx.x; e < nim * plane; e += 256) {
      const int il = e / plane, r = e - il * plane;
      s_pl[e] = src0[il * img_stride + r];
    }
  }
  __syncthreads();
  // each thread takes 4-byte runs of k (EPT elements of one image: the run
  // starts at a multiple of 8), finds their pixels once, then writes them to
  // every tap's row: consecutive lanes hold consecutive k, so both the LDS
  // reads (stride-apart pixels of one row) and the row stores coalesce
  constexpr int EPT = 4 / (int)sizeof(T);
  if (a.bt_phase) {
    // phase planes: rows (n, ph * s + kw), each image hr rows of ws (the
    // block's images are a contiguous run of each row; ws is a multiple of 8)
    const int hrws = a.hr * a.ws, np = a.stride_h * a.s;
    const int kb0 = il0 * hrws, kb1 = (il0 + nim) * hrws;
    const size_t rowlen = (size_t)a.nimg * hrws;
    T* const bp0 = (T*)a.bt + (size_t)n * np * rowlen;
    for (int k0 = kb0 + EPT * (int)threadIdx.x; k0 < kb1; k0 += EPT * 256) {
      int base[EPT], rh[EPT], bw[EPT];
#pragma unroll
      for (int e = 0; e < EPT; ++e) {
        const int k = k0 + e;
        const int il = (int)fast_div((uint32_t)k, a.hrws_mul, a.hrws_shift), q = k - il * hrws;
        const int qh = (int)fast_div((uint32_t)q, a.ws_mul, a.ws_shift), qw = q - qh * a.ws;
        rh[e] = (qh + a.sh_min) * a.stride_h;
        bw[e] = qw * a.stride_w - a.pad_w;
        base[e] = (il - il0) * plane;
      }
      T* dst = bp0 + k0;
      for (int ph = 0; ph < a.stride_h; ++ph)
        for (int kw = 0; kw < a.s; ++kw, dst += rowlen) {
          T v[EPT];
#pragma unroll
          for (int e = 0; e < EPT; ++e) {
            const int ih = rh[e] + ph, iw = bw[e] + kw * a.dil_w;
            const bool in = (unsigned)ih < (unsigned)a.hb && (unsigned)iw < (unsigned)a.wb;
            v[e] = in ? s_pl[base[e] + ih * a.wb + iw] : T(0);
          }
          uint32_t u;
          __builtin_memcpy(&u, v, 4);
          *(uint32_t*)dst = u;
        }
    }
    return;
  }
  const int kbeg = il0 * hws, kreal = a.nimg * hws;
  const int kend = il0 + nim >= a.nimg ? a.kp : kbeg + nim * hws;
  const size_t row_stride = (size_t)a.kp;  // rows (n, tap): the taps of n in order
  T* const bt0 = (T*)a.bt + (size_t)n * (a.r * a.s) * a.kp;
  for (int k0 = kbeg + EPT * (int)threadIdx.x; k0 < kend; k0 += EPT * 256) {
    int base[EPT], bh[EPT], bw[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
      const int k = k0 + e;
      if (k < kreal) {
        const int il = k / hws, q = k - il * hws;
        const int qh = (int)(((uint64_t)(uint32_t)q * a.ws_mul) >> a.ws_shift), qw = q - qh * a.ws;
        bh[e] = qh * a.stride_h - a.pad_h;
        bw[e] = qw * a.stride_w - a.pad_w;
        base[e] = (il - il0) * plane;
      } else {
        bh[e] = -(1 << 29);  // no tap reaches the zero padding
        bw[e] = 0;
        base[e] = 0;
      }
    }
    T* dst = bt0 + k0;
    for (int kh = 0; kh < a.r; ++kh)
      for (int kw = 0; kw < a.s; ++kw, dst += row_stride) {
        T v[EPT];
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
          const int ih = bh[e] + kh * a.dil_h, iw = bw[e] + kw * a.dil_w;
          const bool in = (unsigned)ih < (unsigned)a.hb && (unsigned)iw < (unsigned)a.wb;
          v[e] = in ? s_pl[base[e] + ih * a.wb + iw] : T(0);
        }
        uint32_t u;
        __builtin_memcpy(&u, v, 4);
        *(uint32_t*)dst = u;
      }
  }
}

hipError_t launch_wgrad_stage(const WgArgs& a, int dtype, hipStream_t stream) {
  const long long bt = a.gather_ib > 0 ? 0 : (long long)a.r * a.s * a.nb * a.kp;
  const long long total = ((a.direct ? 0 : (long long)a.ms * a.kp) + bt) / 8;
  if (total > 0 && dtype == 1)
    hipLaunchKernelGGL(wgrad_stage_kernel<uint16_t>, grid_for(total), dim3(256), 0, stream, a);
  else if (total > 0)
    hipLaunchKernelGGL(wgrad_stage_kernel<uint32_t>, grid_for(total), dim3(256), 0, stream, a);
  if (a.gather_ib > 0) {
    const int blocks = (a.nimg + a.gather_ib - 1) / a.gather_ib;
    const size_t lds = (size_t)a.gather_ib * a.hb * a.wb * (dtype == 1 ? 2 : 4);
    const dim3 grid((unsigned)((long long)a.nb * blocks));
    if (dtype == 1)
      hipLaunchKernelGGL(wgrad_gather_kernel<uint16_t>, grid, dim3(256), lds, stream, a);
    else
      hipLaunchKernelGGL(wgrad_gather_kernel<uint32_t>, grid, dim3(256), lds, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_wgrad_gemm(const WgArgs& a0, int dtype, hipStream_t stream) {
  WgArgs a = a0;  // one GEMM of N = nb * taps (Bt's rows (n, tap) in order)
  a.g_taps = a.r * a.s;
  a.g_s = a.s;
  a.nb *= a.r * a.s;
  a.r = a.s = 1;
  const int t = wgrad_tile(a.ms, a.nb);
  const dim3 grid((a.ms + t - 1) / t, (a.nb + t - 1) / t, a.r * a.s * a.ksplit);
  if (t == 128 && dtype == 1)
    hipLaunchKernelGGL(wgrad_gemm2_kernel<true>, grid, dim3(256), 0, stream, a);
  else if (t == 128)
    hipLaunchKernelGGL(wgrad_gemm2_kernel<false>, grid, dim3(256), 0, stream, a);
  else if (dtype == 1)
    hipLaunchKernelGGL(wgrad_gemm_kernel<true>, grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(wgrad_gemm_kernel<false>, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_wgrad_store(const WgArgs& a, int dtype, hipStream_t stream) {
  const long long total = (long long)a.ms * a.nb * a.r * a.s;
  if (a.ksplit >= kWgSplitStore) {
    const dim3 grid((unsigned)((total + 63) / 64));
    if (dtype == 1)
      hipLaunchKernelGGL(wgrad_store_split_kernel<true>, grid, dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL(wgrad_store_split_kernel<false>, grid, dim3(256), 0, stream, a);
  } else if (dtype == 1) {
    hipLaunchKernelGGL(wgrad_store_kernel<true>, grid_for(total), dim3(256), 0, stream, a);
  } else {
    hipLaunchKernelGGL(wgrad_store_kernel<false>, grid_for(total), dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weight gradient of a grouped conv (groups > 1; groups = channels is the
// depthwise conv).  Weight plane (cs, bl) joins small-tensor channel cs to
// big-tensor channel cb = (cs / (ms/groups)) * (nb/groups) + bl, and
//   dw[cs][bl][m][q] = sum over images n and small pixels (i, j) of
//     small[n][cs][i][j] * big[n][cb][i*stride_h - pad_h + m*dil_h]
//                                    [j*stride_w - pad_w + q*dil_w]
// (out-of-range big pixels omitted): per plane the depthwise form of section
// 3.2.3, the outer product of two maps summed over the pixels.  No GEMM is
// left to tile (one channel on each side of a plane), so the sums run on the
// vector units in fp32: one workgroup per (plane, run of kWgGTaps taps), each
// thread summing a fixed stride of the pixels for every tap of the run, then
// the workgroup adds the threads' sums in a fixed tree order
// (deterministic) and rounds once to the dtype.
constexpr int kWgGTaps = 16;

template <typename T>
__global__ __launch_bounds__(256) void wgrad_grouped_kernel(WgArgs a) {
  __shared__ float red[kWgGTaps][257];
  const T* __restrict__ sm = (const T*)a.sm;
  const T* __restrict__ bg = (const T*)a.bg;
  const int tid = threadIdx.x;
  const int sgc = a.ms / a.groups, bgc = a.nb / a.groups;
  const int plane = blockIdx.x;
  const int cs = plane / bgc, bl = plane - cs * bgc;
  const int cb = (cs / sgc) * bgc + bl;
  const int taps = a.r * a.s, t0 = blockIdx.y * kWgGTaps;
  int dh[kWgGTaps], dwo[kWgGTaps];
#pragma unroll
  for (int u = 0; u < kWgGTaps; ++u) {
    const int t = min(t0 + u, taps - 1), m = t / a.s, q = t - m * a.s;
    dh[u] = m * a.dil_h - a.pad_h;
    dwo[u] = q * a.dil_w - a.pad_w;
  }
  float acc[kWgGTaps];
#pragma unroll
  for (int u = 0; u < kWgGTaps; ++u) acc[u] = 0.f;
  const int hws = a.hs * a.ws;
  for (int n = 0; n < a.nimg; ++n) {
    const T* sp = sm + ((size_t)n * a.ms + cs) * hws;
    const T* bp = bg + ((size_t)n * a.nb + cb) * ((size_t)a.hb * a.wb);
    for (int p = tid; p < hws; p += 256) {
      const int i = p / a.ws, j = p - i * a.ws;
      const float v = to_f32(sp[p]);
      const int bi = i * a.stride_h, bj = j * a.stride_w;
#pragma unroll
      for (int u = 0; u < kWgGTaps; ++u) {
        const int y = bi + dh[u], x = bj + dwo[u];
        if (t0 + u < taps && (unsigned)y < (unsigned)a.hb && (unsigned)x < (unsigned)a.wb)
          acc[u] = fmaf(v, to_f32(bp[(size_t)y * a.wb + x]), acc[u]);
      }
    }
  }
#pragma unroll
  for (int u = 0; u < kWgGTaps; ++u) red[u][tid] = acc[u];
  __syncthreads();
  for (int st = 128; st > 0; st >>= 1) {
    if (tid < st)
#pragma unroll
      for (int u = 0; u < kWgGTaps; ++u) red[u][tid] += red[u][tid + st];
    __syncthreads();
  }
  if (tid < kWgGTaps && t0 + tid < taps) {
    const float v = red[tid][0];
    const size_t o = (size_t)plane * taps + t0 + tid;
    if constexpr (std::is_same<T, uint16_t>::value)
      ((uint16_t*)a.dw)[o] = f32_to_bf16_rne(v);
    else
      ((float*)a.dw)[o] = v;
  }
}

hipError_t launch_wgrad_grouped(const WgArgs& a, int dtype, hipStream_t stream) {
  const long long planes = (long long)a.ms * (a.nb / a.groups);
  const int taps = a.r * a.s;
  if (planes <= 0 || planes >= (1ll << 31) || a.groups < 2) return hipErrorInvalidValue;
  const dim3 grid((unsigned)planes, (unsigned)((taps + kWgGTaps - 1) / kWgGTaps));
  if (dtype == 1)
    hipLaunchKernelGGL(wgrad_grouped_kernel<uint16_t>, grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(wgrad_grouped_kernel<uint32_t>, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Input staging: channel-contiguous pixels [n][h*w][c_stride], zero padded
// channels, for NCHW inputs and for NHWC inputs whose channel count is not a
// multiple of 16 bytes.

// NCHW source: a 64-channel x 64-pixel block per workgroup through LDS.
template <typename T>
__global__ __launch_bounds__(256) void stage_nchw_kernel(const T* __restrict__ x,
                                                         T* __restrict__ xs, int cin, int hw,
                                                         int cs) {
  __shared__ T tile[64][65];
  const int img = blockIdx.z, c0 = blockIdx.y * 64, p0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i, p = p0 + tx;
    tile[i][tx] = (c < cin && p < hw) ? x[((size_t)img * cin + c) * hw + p] : T(0);
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int p = p0 + i, c = c0 + tx;
    if (p < hw && c < cs) xs[((size_t)img * hw + p) * cs + c] = tile[tx][i];
  }
}

// NCHW source whose plane size is a multiple of 16 bytes: 64 channels x
// 128 bytes of pixels per workgroup, read and written in 16-byte pieces (a
// channel run of one pixel is gathered from an LDS column).
template <typename T>
__global__ __launch_bounds__(256) void stage_nchw_vec_kernel(const T* __restrict__ x,
                                                             T* __restrict__ xs, int cin, int hw,
                                                             int cs) {
  constexpr int VE = 16 / sizeof(T);  // elements per 16 bytes
  constexpr int PX = 8 * VE;          // pixels per tile (128 bytes per channel)
  constexpr int CC = 64 / VE;         // 16-byte channel chunks per pixel
  __shared__ __attribute__((aligned(16))) T tile[64][PX + VE];
  const int img = blockIdx.z, c0 = blockIdx.y * 64, p0 = blockIdx.x * PX;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int q = threadIdx.x + 256 * i;
    const int c = q >> 3, j = q & 7, p = p0 + j * VE;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (c0 + c < cin && p < hw)
      v = *(const uint4*)(x + ((size_t)img * cin + c0 + c) * hw + p);
    *(uint4*)&tile[c][j * VE] = v;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int q = threadIdx.x + 256 * i;
    const int cc = q % CC, px = q / CC;
    const int p = p0 + px, c = c0 + cc * VE;
    if (p >= hw || c >= cs) continue;
    uint32_t w[4];
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        w[e] = (uint32_t)tile[cc * VE + 2 * e][px] | ((uint32_t)tile[cc * VE + 2 * e + 1][px] << 16);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = (uint32_t)tile[cc * VE + e][px];
    }
    *(uint4*)(xs + ((size_t)img * hw + p) * cs + c) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// NHWC source with cin channels per pixel.
template <typename T>
__global__ void stage_nhwc_kernel(const T* __restrict__ x, T* __restrict__ xs, int cin, int cs,
                                  long long total) {
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(idx % cs);
    const long long p = idx / cs;
    xs[idx] = c < cin ? x[p * cin + c] : T(0);
  }
}

hipError_t launch_stage_input(const void* x, void* xs, int dtype, bool nchw, int n, int cin,
                              int hw, int c_stride, hipStream_t stream) {
  const int ve = dtype == 1 ? 8 : 4;
  if (nchw && hw % ve == 0) {
    dim3 grid((hw + 8 * ve - 1) / (8 * ve), (c_stride + 63) / 64, n), block(256);
    if (dtype == 1)
      hipLaunchKernelGGL(stage_nchw_vec_kernel<uint16_t>, grid, block, 0, stream,
                         (const uint16_t*)x, (uint16_t*)xs, cin, hw, c_stride);
    else
      hipLaunchKernelGGL(stage_nchw_vec_kernel<uint32_t>, grid, block, 0, stream,
                         (const uint32_t*)x, (uint32_t*)xs, cin, hw, c_stride);
  } else if (nchw) {
    dim3 grid((hw + 63) / 64, (c_stride + 63) / 64, n), block(256);
    if (dtype == 1)
      hipLaunchKernelGGL(stage_nchw_kernel<uint16_t>, grid, block, 0, stream,
                         (const uint16_t*)x, (uint16_t*)xs, cin, hw, c_stride);
    else
      hipLaunchKernelGGL(stage_nchw_kernel<uint32_t>, grid, block, 0, stream,
                         (const uint32_t*)x, (uint32_t*)xs, cin, hw, c_stride);
  } else {
    const long long total = (long long)n * hw * c_stride;
    const long long want = (total + 255) / 256;
    const int grid = (int)(want < 65536 ? want : 65536);
    if (dtype == 1)
      hipLaunchKernelGGL(stage_nhwc_kernel<uint16_t>, dim3(grid), dim3(256), 0, stream,
                         (const uint16_t*)x, (uint16_t*)xs, cin, c_stride, total);
    else
      hipLaunchKernelGGL(stage_nhwc_kernel<uint32_t>, dim3(grid), dim3(256), 0, stream,
                         (const uint32_t*)x, (uint32_t*)xs, cin, c_stride, total);
  }
  return hipGetLastError();
}

}  // namespace huge2
