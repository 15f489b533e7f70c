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
#include "kernels.hpp"

namespace huge2 {

typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;

int tile_bm(int cfg) {
  switch (cfg) {
    case TILE_256x32: return 256;
    case TILE_64x128: return 64;
    default: return 128;
  }
}
int tile_bn(int cfg) {
  switch (cfg) {
    case TILE_256x32: return 32;
    default: return 128;
  }
}

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
__device__ __forceinline__ PixelPos pixel_pos(const SegDev& sg, int nimg, int m) {
  PixelPos p;
  int j = m;
  const int a_w = j % sg.qn_w;
  j /= sg.qn_w;
  const int a_h = j % sg.qn_h;
  j /= sg.qn_h;
  p.img = j % nimg;
  const int iph = j / nimg;
  const int iph_h = iph / sg.nphase_w, iph_w = iph - iph_h * sg.nphase_w;
  const int qh = sg.q0_h + a_h, qw = sg.q0_w + a_w;
  p.oh = sg.phase0_h + iph_h + sg.out_step_h * qh;
  p.ow = sg.phase0_w + iph_w + sg.out_step_w * qw;
  p.ih = sg.in0_h + sg.in_dphase_h * iph_h + sg.in_step_h * qh;
  p.iw = sg.in0_w + sg.in_dphase_w * iph_w + sg.in_step_w * qw;
  return p;
}

// ---------------------------------------------------------------------------
// Phase GEMM.  A workgroup of 256 threads (4 waves) computes a BM x BN tile
// (BM pixels of one segment, BN output channels).  The K loop runs over the
// segment's taps and, per tap, over 64-byte blocks of input channels.  Each
// stage holds BM + BN rows of 64 bytes in LDS (row pitch 80 bytes, so that
// 16-byte accesses of 8 consecutive rows hit distinct banks), double
// buffered, with the next stage's global loads issued before the current
// stage's MFMAs.
//
// Input gather (IN_*): the tile row of a pixel at a tap is the 64-byte run of
// channels [cb*BK, cb*BK + BK) of input pixel (ih, iw) = pixel base + tap
// offset; rows that fall outside the input (or past cin) are zero.
//   IN_NHWC_VEC : 4 lanes per pixel, one 16-byte load each.
//   IN_NCHW     : lane j of a wave on pixel row j, one element load per
//                 channel (consecutive lanes read consecutive input columns),
//                 packed into 16-byte LDS writes.
//   IN_NHWC_ELEM: as IN_NCHW, for NHWC inputs whose channel count is not a
//                 multiple of 16 bytes.
//
// MFMA operands are K-contiguous per lane: lane l reads 32 bytes of its row
// at byte offset 32*(l/32).  The K order inside a stage is permuted
// identically for both operands, which leaves the contraction unchanged:
//   bf16: MFMA t (t = 0,1) uses row elements [16h + 8t, 16h + 8t + 8), h = l/32
//   fp32: MFMA t (t = 0..7) uses row element 8h + t.
// NHWC output puts pixels on MFMA rows (lanes hold consecutive channels, so
// the stores of a pixel's channels coalesce); NCHW output puts pixels on MFMA
// columns (lanes hold consecutive pixels).
template <bool BF16, int BM, int BN, int PWAVES, int CWAVES, int IN_MODE>
__global__ __launch_bounds__(256) void phase_gemm_kernel(GemmArgs a) {
  constexpr bool NHWC_OUT = IN_MODE != IN_NCHW;
  constexpr bool VEC_IN = IN_MODE == IN_NHWC_VEC;
  constexpr int ESZ = BF16 ? 2 : 4;
  constexpr int BK = kBlockK_bytes / ESZ;  // K elements per stage
  constexpr int VE = 16 / ESZ;             // elements per 16-byte chunk
  constexpr int ROWB = 80;
  constexpr int WP = BM / PWAVES, WC = BN / CWAVES;
  constexpr int TP = WP / 32, TC = WC / 32;
  constexpr int A_LD = BM * 4 / 256;
  constexpr int B_LD = (BN * 4 + 255) / 256;
  static_assert(BM % 64 == 0, "A-tile rows per thread");
  static_assert(PWAVES * CWAVES == 4, "4 waves");
  static_assert(TP >= 1 && TC >= 1 && WP % 32 == 0 && WC % 32 == 0, "32x32 MFMA blocks");
  constexpr int STAGE_B = (BM + BN) * ROWB;
  __shared__ __attribute__((aligned(16))) char smem[2 * STAGE_B];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int work = xcd_remap(blockIdx.x, gridDim.x);
  const WorkDev wk = a.works[work];
  const SegDev sg = a.segs[wk.seg];
  const char* xb = (const char*)a.x;
  const char* wb = (const char*)a.wp;

  // The A-tile units (row, 16-byte chunk) this thread loads, and their pixels'
  // input coordinates before the tap offset.
  int a_row[A_LD], a_chunk[A_LD], a_ih[A_LD], a_iw[A_LD], a_img[A_LD];
#pragma unroll
  for (int i = 0; i < A_LD; ++i) {
    const int u = tid + 256 * i;
    a_row[i] = VEC_IN ? (u >> 2) : (u % BM);
    a_chunk[i] = VEC_IN ? (u & 3) : (u / BM);
    const int m = wk.m0 + a_row[i];
    if (m < sg.m_total) {
      const PixelPos p = pixel_pos(sg, a.n, m);
      a_ih[i] = p.ih;
      a_iw[i] = p.iw;
      a_img[i] = p.img;
    } else {
      a_ih[i] = -(1 << 29);  // fails every bounds test
      a_iw[i] = 0;
      a_img[i] = 0;
    }
  }
  const int hw = a.h * a.w;

  const int cblocks = a.cin_pad / BK;
  const int nsteps = sg.tap_count * cblocks;
  uint4 ra[A_LD], rb[B_LD];

  auto load_step = [&](int s) {
    const int t = s / cblocks, cb = s - t * cblocks;
    const TapDev tp = a.taps[sg.tap_begin + t];
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      const int ih = a_ih[i] + tp.off_h, iw = a_iw[i] + tp.off_w;
      const bool in = (unsigned)ih < (unsigned)a.h && (unsigned)iw < (unsigned)a.w;
      const int c0 = cb * BK + a_chunk[i] * VE;
      if constexpr (VEC_IN) {
        if (in && c0 < a.cin) {
          const size_t off = ((size_t)a_img[i] * hw + ih * a.w + iw) * a.cin + c0;
          ra[i] = *(const uint4*)(xb + off * ESZ);
        } else {
          ra[i] = make_uint4(0, 0, 0, 0);
        }
      } else {
        uint32_t v[VE];
#pragma unroll
        for (int e = 0; e < VE; ++e) {
          const int c = c0 + e;
          v[e] = 0;
          if (in && c < a.cin) {
            const size_t off = IN_MODE == IN_NCHW
                                   ? ((size_t)a_img[i] * a.cin + c) * hw + ih * a.w + iw
                                   : ((size_t)a_img[i] * hw + ih * a.w + iw) * a.cin + c;
            if constexpr (BF16)
              v[e] = *(const uint16_t*)(xb + off * 2);
            else
              v[e] = *(const uint32_t*)(xb + off * 4);
          }
        }
        if constexpr (BF16)
          ra[i] = make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16),
                             v[6] | (v[7] << 16));
        else
          ra[i] = make_uint4(v[0], v[1], v[2], v[3]);
      }
    }
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int idx = tid + 256 * i;
      if (idx < BN * 4) {
        const int row = idx >> 2;
        const size_t off = ((size_t)tp.slot * a.cout_pad + wk.n0 + row) * a.cin_pad + cb * BK +
                           (idx & 3) * VE;
        rb[i] = *(const uint4*)(wb + off * ESZ);
      }
    }
  };
  auto store_stage = [&](int buf) {
    char* as = smem + buf * STAGE_B;
    char* bs = as + BM * ROWB;
#pragma unroll
    for (int i = 0; i < A_LD; ++i) *(uint4*)(as + a_row[i] * ROWB + a_chunk[i] * 16) = ra[i];
#pragma unroll
    for (int i = 0; i < B_LD; ++i) {
      const int idx = tid + 256 * i;
      if (idx < BN * 4) *(uint4*)(bs + (idx >> 2) * ROWB + (idx & 3) * 16) = rb[i];
    }
  };

  f32x16 acc[TP][TC];
#pragma unroll
  for (int i = 0; i < TP; ++i)
#pragma unroll
    for (int j = 0; j < TC; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int wp_i = wave % PWAVES, wc_i = wave / PWAVES;
  if (nsteps > 0) {
    load_step(0);
    store_stage(0);
    __syncthreads();
    for (int s = 0; s < nsteps; ++s) {
      const int cur = s & 1;
      if (s + 1 < nsteps) load_step(s + 1);
      const char* as = smem + cur * STAGE_B;
      const char* bs = as + BM * ROWB;
      uint4 fp[TP][2], fc[TC][2];
#pragma unroll
      for (int i = 0; i < TP; ++i) {
        const char* p = as + (wp_i * WP + 32 * i + (lane & 31)) * ROWB + (lane >> 5) * 32;
        fp[i][0] = *(const uint4*)p;
        fp[i][1] = *(const uint4*)(p + 16);
      }
#pragma unroll
      for (int j = 0; j < TC; ++j) {
        const char* p = bs + (wc_i * WC + 32 * j + (lane & 31)) * ROWB + (lane >> 5) * 32;
        fc[j][0] = *(const uint4*)p;
        fc[j][1] = *(const uint4*)(p + 16);
      }
      if constexpr (BF16) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int i = 0; i < TP; ++i)
#pragma unroll
            for (int j = 0; j < TC; ++j) {
              const bf16x8 vp = __builtin_bit_cast(bf16x8, fp[i][t]);
              const bf16x8 vc = __builtin_bit_cast(bf16x8, fc[j][t]);
              if constexpr (NHWC_OUT)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vp, vc, acc[i][j], 0, 0, 0);
              else
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vc, vp, acc[i][j], 0, 0, 0);
            }
      } else {
#pragma unroll
        for (int t = 0; t < 8; ++t)
#pragma unroll
          for (int i = 0; i < TP; ++i)
#pragma unroll
            for (int j = 0; j < TC; ++j) {
              const uint4 up = fp[i][t >> 2], uc = fc[j][t >> 2];
              const uint32_t bp = (t & 3) == 0 ? up.x : (t & 3) == 1 ? up.y : (t & 3) == 2 ? up.z : up.w;
              const uint32_t bc = (t & 3) == 0 ? uc.x : (t & 3) == 1 ? uc.y : (t & 3) == 2 ? uc.z : uc.w;
              const float vp = __uint_as_float(bp), vc = __uint_as_float(bc);
              if constexpr (NHWC_OUT)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(vp, vc, acc[i][j], 0, 0, 0);
              else
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(vc, vp, acc[i][j], 0, 0, 0);
            }
      }
      if (s + 1 < nsteps) store_stage(cur ^ 1);
      __syncthreads();
    }
  }

  // Epilogue: bias, rounding, and the scatter to the interleaved output.
  // 32x32 MFMA result layout: lane l holds column l%32 and rows
  // 8*(r/4) + 4*(l/32) + (r%4) for r = 0..15.
  const int hw_o = a.ho * a.wo;
  if constexpr (NHWC_OUT) {
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

template <bool BF16, int IN_MODE>
static hipError_t launch_cfg(const GemmArgs& a, int cfg, hipStream_t stream) {
  dim3 grid(a.n_works), block(256);
  switch (cfg) {
    case TILE_128x128:
      hipLaunchKernelGGL((phase_gemm_kernel<BF16, 128, 128, 2, 2, IN_MODE>), grid, block, 0,
                         stream, a);
      break;
    case TILE_256x32:
      hipLaunchKernelGGL((phase_gemm_kernel<BF16, 256, 32, 4, 1, IN_MODE>), grid, block, 0,
                         stream, a);
      break;
    case TILE_64x128:
      hipLaunchKernelGGL((phase_gemm_kernel<BF16, 64, 128, 1, 4, IN_MODE>), grid, block, 0,
                         stream, a);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <bool BF16>
static hipError_t launch_mode(const GemmArgs& a, int cfg, int in_mode, hipStream_t stream) {
  switch (in_mode) {
    case IN_NHWC_VEC: return launch_cfg<BF16, IN_NHWC_VEC>(a, cfg, stream);
    case IN_NCHW: return launch_cfg<BF16, IN_NCHW>(a, cfg, stream);
    case IN_NHWC_ELEM: return launch_cfg<BF16, IN_NHWC_ELEM>(a, cfg, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_phase_gemm(const GemmArgs& a, int dtype, int cfg, int in_mode,
                             hipStream_t stream) {
  if (a.n_works <= 0) return hipSuccess;
  return dtype == 1 ? launch_mode<true>(a, cfg, in_mode, stream)
                    : launch_mode<false>(a, cfg, in_mode, stream);
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

}  // namespace huge2
