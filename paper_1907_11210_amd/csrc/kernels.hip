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
#include "kernels.hpp"

namespace huge2 {

typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;

// Workgroups are dealt to the 8 XCDs round-robin (id mod 8).  Map them so
// that each XCD runs one contiguous run of the work list: neighbouring
// tiles share input rows and weight blocks, which then stay in that XCD's L2.
__device__ __forceinline__ int xcd_remap(int b, int g) {
  const int g8 = (g + 7) >> 3, r = g & 7, x = b & 7, y = b >> 3;
  if (r == 0 || x < r) return x * g8 + y;
  return r * g8 + (x - r) * (g8 - 1) + y;
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Decomposition of a segment pixel index into image, output and input coordinates.
struct PixelPos {
  int img, oh, ow, ih, iw;
};
__device__ __forceinline__ uint32_t fast_div(uint32_t v, uint32_t mul, uint32_t shift) {
  return (uint32_t)(((uint64_t)v * mul) >> shift);
}
__device__ __forceinline__ PixelPos pixel_pos(const SegDev& sg, int nimg, int m) {
  PixelPos p;
  uint32_t j = (uint32_t)m;
  uint32_t t = fast_div(j, sg.div_mul[0], sg.div_shift[0]);
  const int a_w = (int)(j - t * (uint32_t)sg.qn_w);
  j = t;
  t = fast_div(j, sg.div_mul[1], sg.div_shift[1]);
  const int a_h = (int)(j - t * (uint32_t)sg.qn_h);
  j = t;
  t = fast_div(j, sg.div_mul[2], sg.div_shift[2]);
  p.img = (int)(j - t * (uint32_t)nimg);
  const uint32_t iph = t;
  const uint32_t iph_h = fast_div(iph, sg.div_mul[3], sg.div_shift[3]);
  const int iph_w = (int)(iph - iph_h * (uint32_t)sg.nphase_w);
  const int qh = sg.q0_h + a_h, qw = sg.q0_w + a_w;
  p.oh = sg.phase0_h + (int)iph_h + sg.out_step_h * qh;
  p.ow = sg.phase0_w + iph_w + sg.out_step_w * qw;
  p.ih = sg.in0_h + sg.in_dphase_h * (int)iph_h + sg.in_step_h * qh;
  p.iw = sg.in0_w + sg.in_dphase_w * iph_w + sg.in_step_w * qw;
  return p;
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

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int work = xcd_remap(blockIdx.x, gridDim.x);
  const WorkDev wk = a.works[work];
  const SegDev sg = a.segs[wk.seg];
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.x, 0, a.x_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t wr =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.wp, 0, a.wp_bytes, 0x00020000);

  // This thread's A-tile rows (pixels) and its 16-byte chunk within a row.
  // Rows past the end of the segment repeat its last pixel: they compute
  // values the epilogue never stores.
  const int chunk = tid % CPR;
  int a_ih[A_LD], a_iw[A_LD];
  uint32_t a_base[A_LD];  // byte offset of (pixel, chunk) at tap offset (0, 0)
#pragma unroll
  for (int i = 0; i < A_LD; ++i) {
    const int m = min(wk.m0 + tid / CPR + (NT / CPR) * i, sg.m_total - 1);
    const PixelPos p = pixel_pos(sg, a.n, m);
    a_ih[i] = p.ih;
    a_iw[i] = p.iw;
    // unsigned (wrapping) arithmetic: the tap offset brings it back in range
    a_base[i] = (((uint32_t)p.img * (uint32_t)a.h + (uint32_t)p.ih) * (uint32_t)a.w +
                 (uint32_t)p.iw) * (uint32_t)a.cin * ESZ + (uint32_t)(chunk * VE * ESZ);
  }
  const int ntaps = sg.tap_count;
  const int cblocks = a.cin_pad / KC;
  const int nsteps = ntaps * cblocks;
  // channels of the last K block that exist (a partial block needs masking)
  const int tail_c = a.cin - (cblocks - 1) * KC;

  // The segment's taps in LDS: byte delta of the tapped pixel and byte
  // offset of the tap's weight block.
  __shared__ int4 s_taps[kMaxLdsTaps];
  const bool lds_taps = !sg.tap_ap && ntaps <= kMaxLdsTaps;
  if (lds_taps) {
    for (int t = tid; t < ntaps; t += NT) {
      const TapDev tp = a.taps[sg.tap_begin + t];
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
      __builtin_amdgcn_make_buffer_rsrc((void*)a.wp, 0, 0, 0x00020000);

  // K order: channel block outer, tap inner, so that the taps of one channel
  // block re-read the same input rows while they are still in cache.  A load
  // past the last stage goes through the empty resources instead of
  // branching around the loads: the load sequence stays the same on every
  // path, which lets the compiler wait only for the stage it stores.
  int ld_tap = 0, ld_cb = 0, ld_th = 0, ld_tw = 0;
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
        const TapDev tp = a.taps[sg.tap_begin + (valid ? ld_tap : 0)];
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
        compute(0);
        store_stage(1, r0);
        __syncthreads();
        load_step(r0, s + 3 < nsteps);
        compute(1);
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
        compute(1);
        store_stage(0, r0);
        __syncthreads();
      }
    }
  }

  // Epilogue: bias, rounding, and the scatter to the interleaved output.
  // 32x32 MFMA result layout: lane l holds column l%32 and rows
  // 8*(r/4) + 4*(l/32) + (r%4) for r = 0..15.
  const int hw_o = a.ho * a.wo;
  if constexpr (!NCHW_OUT) {
#pragma unroll
    for (int i = 0; i < TP; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = wk.m0 + wp_i * WP + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (m >= sg.m_total) continue;
        const PixelPos p = pixel_pos(sg, a.n, m);
        const int pix = (p.img * a.ho + p.oh) * a.wo + p.ow;
#pragma unroll
        for (int j = 0; j < TC; ++j) {
          const int ch = wk.n0 + wc_i * WC + 32 * j + (lane & 31);
          if (ch >= a.cout) continue;
          float v = acc[i][j][r];
          if (a.bias) v += a.bias[ch];
          const size_t off = (size_t)pix * a.cout + ch;
          if constexpr (BF16)
            ((uint16_t*)a.y)[off] = f32_to_bf16_rne(v);
          else
            ((float*)a.y)[off] = v;
        }
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < TP; ++i) {
      const int m = wk.m0 + wp_i * WP + 32 * i + (lane & 31);
      if (m >= sg.m_total) continue;
      const PixelPos p = pixel_pos(sg, a.n, m);
      const size_t base = (size_t)p.img * a.cout * hw_o + (size_t)p.oh * a.wo + p.ow;
#pragma unroll
      for (int j = 0; j < TC; ++j) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int ch = wk.n0 + wc_i * WC + 32 * j + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (ch >= a.cout) continue;
          float v = acc[i][j][r];
          if (a.bias) v += a.bias[ch];
          const size_t off = base + (size_t)ch * hw_o;
          if constexpr (BF16)
            ((uint16_t*)a.y)[off] = f32_to_bf16_rne(v);
          else
            ((float*)a.y)[off] = v;
        }
      }
    }
  }
}

template <bool BF16, bool NCHW_OUT, int CFG>
static void launch_one(const GemmArgs& a, hipStream_t stream) {
  constexpr TileShape t = kTiles[CFG];
  hipLaunchKernelGGL((phase_gemm_kernel<BF16, t.bm, t.bn, t.pw, t.cw, t.kb, t.depth, NCHW_OUT>),
                     dim3(a.n_works), dim3(t.pw * t.cw * 64), 0, stream, a);
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
// Weight packing: wp[slot][k][c] = w at kernel tap slot = (kh, kw).

template <typename T>
__global__ void pack_weights_kernel(const T* __restrict__ w, T* __restrict__ wp, bool transposed,
                                    int cin, int cout, int r, int s, int cin_pad, int cout_pad,
                                    long long total) {
  for (long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (long long)gridDim.x * blockDim.x) {
    const int c = (int)(idx % cin_pad);
    const long long t = idx / cin_pad;
    const int k = (int)(t % cout_pad);
    const int slot = (int)(t / cout_pad);
    const int kh = slot / s, kw = slot - kh * s;
    T v = T(0);
    if (c < cin && k < cout) {
      const long long src = transposed ? (((long long)c * cout + k) * r + kh) * s + kw
                                       : (((long long)k * cin + c) * r + kh) * s + kw;
      v = w[src];
    }
    wp[idx] = v;
  }
}

hipError_t launch_pack_weights(const void* w, void* wp, int dtype, bool transposed, int cin,
                               int cout, int r, int s, int cin_pad, int cout_pad,
                               hipStream_t stream) {
  const long long total = (long long)r * s * cout_pad * cin_pad;
  const int block = 256;
  const long long want = (total + block - 1) / block;
  const int grid = (int)(want < 65536 ? want : 65536);
  if (total == 0) return hipSuccess;
  if (dtype == 1)
    hipLaunchKernelGGL(pack_weights_kernel<uint16_t>, dim3(grid), dim3(block), 0, stream,
                       (const uint16_t*)w, (uint16_t*)wp, transposed, cin, cout, r, s, cin_pad,
                       cout_pad, total);
  else
    hipLaunchKernelGGL(pack_weights_kernel<uint32_t>, dim3(grid), dim3(block), 0, stream,
                       (const uint32_t*)w, (uint32_t*)wp, transposed, cin, cout, r, s, cin_pad,
                       cout_pad, total);
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
