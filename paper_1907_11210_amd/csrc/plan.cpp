// plan.cpp -- host-side phase decomposition (see plan.hpp).
#include "plan.hpp"

#include <algorithm>
#include <climits>

namespace huge2 {
namespace {

// floor(a / b) and ceil(a / b) for b > 0 and any sign of a.
int floor_div(int a, int b) { return a >= 0 ? a / b : -((-a + b - 1) / b); }
int ceil_div(int a, int b) { return -floor_div(-a, b); }

// q in [0, q_count) with 0 <= base + step*q < in_size, as [lo, hi).
void valid_range(int base, int step, int q_count, int in_size, int* lo, int* hi) {
  *lo = std::max(0, ceil_div(-base, step));
  *hi = std::min(q_count, floor_div(in_size - 1 - base, step) + 1);
  if (*hi < *lo) *hi = *lo;
}

bool same_taps(const std::vector<AxisTap>& a, const std::vector<AxisTap>& b) {
  if (a.size() != b.size()) return false;
  for (size_t i = 0; i < a.size(); ++i)
    if (a[i].k != b[i].k || a[i].off != b[i].off || a[i].lo != b[i].lo || a[i].hi != b[i].hi)
      return false;
  return true;
}

}  // namespace

bool decompose_axis(bool transposed, int in_size, int out_size, int ksize, int stride, int pad,
                    int dil, std::vector<AxisGroup>* groups) {
  groups->clear();
  if (in_size < 1 || out_size < 1 || ksize < 1 || stride < 1 || dil < 1 || pad < 0) return false;
  if (transposed) {
    // Output phase rho collects o = rho + stride*q.  Tap k lands there when
    // i*stride = o + pad - k*dil, i.e. (rho + pad - k*dil) divisible by the
    // stride, and then reads input i = q + (rho + pad - k*dil)/stride.
    for (int rho = 0; rho < std::min(stride, out_size); ++rho) {
      AxisGroup g;
      g.phase0 = rho;
      g.nphase = 1;
      g.out_step = stride;
      g.q_count = ceil_div(out_size - rho, stride);
      g.in0 = 0;
      g.in_dphase = 0;
      g.in_step = 1;
      for (int k = 0; k < ksize; ++k) {
        int num = rho + pad - k * dil;
        if (((num % stride) + stride) % stride != 0) continue;
        AxisTap t;
        t.k = k;
        t.off = num / stride;  // exact
        valid_range(t.off, 1, g.q_count, in_size, &t.lo, &t.hi);
        if (t.lo < t.hi) g.taps.push_back(t);
      }
      groups->push_back(g);
    }
    return true;
  }
  if (stride == 1) {
    // Phase views of a dilated conv (section 3.2.2): output o = phi + dil*q
    // reads input phi - pad + dil*(q + k), the phi-th sub-lattice shifted by k.
    int nphi = std::min(dil, out_size);
    for (int phi = 0; phi < nphi; ++phi) {
      AxisGroup g;
      g.phase0 = phi;
      g.nphase = 1;
      g.out_step = dil;
      g.q_count = ceil_div(out_size - phi, dil);
      g.in0 = phi - pad;
      g.in_dphase = 1;
      g.in_step = dil;
      for (int k = 0; k < ksize; ++k) {
        AxisTap t;
        t.k = k;
        t.off = k * dil;
        valid_range(g.in0 + t.off, dil, g.q_count, in_size, &t.lo, &t.hi);
        if (t.lo < t.hi) g.taps.push_back(t);
      }
      // consecutive phase views with the same shape share one group
      if (!groups->empty()) {
        AxisGroup& prev = groups->back();
        if (prev.q_count == g.q_count && same_taps(prev.taps, g.taps) &&
            prev.phase0 + prev.nphase == phi) {
          prev.nphase += 1;
          continue;
        }
      }
      groups->push_back(g);
    }
    return true;
  }
  // Strided (and possibly dilated) conv: a direct gather, one phase.
  AxisGroup g;
  g.phase0 = 0;
  g.nphase = 1;
  g.out_step = 1;
  g.q_count = out_size;
  g.in0 = -pad;
  g.in_dphase = 0;
  g.in_step = stride;
  for (int k = 0; k < ksize; ++k) {
    AxisTap t;
    t.k = k;
    t.off = k * dil;
    valid_range(g.in0 + t.off, stride, g.q_count, in_size, &t.lo, &t.hi);
    if (t.lo < t.hi) g.taps.push_back(t);
  }
  groups->push_back(g);
  return true;
}

std::vector<AxisPiece> axis_pieces(const AxisGroup& g, bool split) {
  std::vector<AxisPiece> out;
  if (!split) {
    AxisPiece p;
    p.q0 = 0;
    p.qn = g.q_count;
    for (int i = 0; i < (int)g.taps.size(); ++i) p.tap_idx.push_back(i);
    out.push_back(p);
    return out;
  }
  std::vector<int> cuts = {0, g.q_count};
  for (const AxisTap& t : g.taps) {
    cuts.push_back(t.lo);
    cuts.push_back(t.hi);
  }
  std::sort(cuts.begin(), cuts.end());
  cuts.erase(std::unique(cuts.begin(), cuts.end()), cuts.end());
  for (size_t c = 0; c + 1 < cuts.size(); ++c) {
    int a = cuts[c], b = cuts[c + 1];
    if (a < 0 || b > g.q_count || a >= b) continue;
    AxisPiece p;
    p.q0 = a;
    p.qn = b - a;
    for (int i = 0; i < (int)g.taps.size(); ++i)
      if (g.taps[i].lo <= a && b <= g.taps[i].hi) p.tap_idx.push_back(i);
    out.push_back(p);
  }
  return out;
}

bool output_dims(const huge2_conv_desc& d, bool transposed, int* ho, int* wo) {
  long long h, w;
  if (transposed) {
    h = (long long)(d.h - 1) * d.stride_h - 2LL * d.pad_h + (long long)d.dil_h * (d.r - 1) +
        d.out_pad_h + 1;
    w = (long long)(d.w - 1) * d.stride_w - 2LL * d.pad_w + (long long)d.dil_w * (d.s - 1) +
        d.out_pad_w + 1;
  } else {
    long long nh = (long long)d.h + 2LL * d.pad_h - (long long)d.dil_h * (d.r - 1) - 1;
    long long nw = (long long)d.w + 2LL * d.pad_w - (long long)d.dil_w * (d.s - 1) - 1;
    if (nh < 0 || nw < 0) return false;
    h = nh / d.stride_h + 1;
    w = nw / d.stride_w + 1;
  }
  if (h < 1 || w < 1 || h > INT_MAX || w > INT_MAX) return false;
  *ho = (int)h;
  *wo = (int)w;
  return true;
}

huge2_status validate_desc(const huge2_conv_desc* d, bool transposed) {
  if (!d) return HUGE2_ERR_INVALID_ARG;
  if (d->n < 1 || d->c_in < 1 || d->h < 1 || d->w < 1 || d->c_out < 1 || d->r < 1 || d->s < 1)
    return HUGE2_ERR_INVALID_ARG;
  if (d->stride_h < 1 || d->stride_w < 1 || d->dil_h < 1 || d->dil_w < 1)
    return HUGE2_ERR_INVALID_ARG;
  if (d->pad_h < 0 || d->pad_w < 0 || d->out_pad_h < 0 || d->out_pad_w < 0)
    return HUGE2_ERR_INVALID_ARG;
  if (d->layout != HUGE2_NCHW && d->layout != HUGE2_NHWC) return HUGE2_ERR_INVALID_ARG;
  if (d->dtype != HUGE2_F32 && d->dtype != HUGE2_BF16) return HUGE2_ERR_INVALID_ARG;
  if (d->activation != HUGE2_ACT_NONE && d->activation != HUGE2_ACT_RELU &&
      d->activation != HUGE2_ACT_TANH)
    return HUGE2_ERR_INVALID_ARG;
  if (d->groups < 0 || (d->groups > 1 && (d->c_in % d->groups != 0 || d->c_out % d->groups != 0)))
    return HUGE2_ERR_INVALID_ARG;
  if (transposed) {
    if (d->out_pad_h >= std::max(d->stride_h, d->dil_h) ||
        d->out_pad_w >= std::max(d->stride_w, d->dil_w))
      return HUGE2_ERR_INVALID_ARG;
  } else if (d->out_pad_h != 0 || d->out_pad_w != 0) {
    return HUGE2_ERR_INVALID_ARG;
  }
  int ho, wo;
  if (!output_dims(*d, transposed, &ho, &wo)) return HUGE2_ERR_INVALID_ARG;
  // The kernels address the input and the packed weights through buffer
  // resources with 32-bit byte offsets, and the output with 32-bit element
  // offsets: every extent (with channel padding) must stay below 2^31 bytes.
  const long long lim = INT_MAX;
  const long long esz = d->dtype == HUGE2_BF16 ? 2 : 4;
  long long cin_v = ((long long)d->c_in + 7) / 8 * 8;
  // the largest paddings any tile configuration applies
  long long cin_pad = ((long long)d->c_in + 127) / 128 * 128;
  long long cout_pad = ((long long)d->c_out + 255) / 256 * 256;
  long long nx = (long long)d->n * cin_v * d->h * d->w * esz;
  long long ny = (long long)d->n * d->c_out * ho * wo * esz;
  long long nw = cin_pad * cout_pad * d->r * d->s * esz;
  if (nx > lim || ny > lim || nw > lim) return HUGE2_ERR_UNSUPPORTED;
  return HUGE2_OK;
}

bool build_shape(const huge2_conv_desc& d, bool transposed, int class_split, int bm,
                 PlanShape* out) {
  int ho, wo;
  if (!output_dims(d, transposed, &ho, &wo)) return false;
  std::vector<AxisGroup> gh, gw;
  if (!decompose_axis(transposed, d.h, ho, d.r, d.stride_h, d.pad_h, d.dil_h, &gh)) return false;
  if (!decompose_axis(transposed, d.w, wo, d.s, d.stride_w, d.pad_w, d.dil_w, &gw)) return false;
  out->segs.clear();
  out->taps.clear();
  out->tile_taps = 0;

  long long vh = 0, vw = 0;
  for (const AxisGroup& g : gh)
    for (const AxisTap& t : g.taps) vh += (long long)g.nphase * (t.hi - t.lo);
  for (const AxisGroup& g : gw)
    for (const AxisTap& t : g.taps) vw += (long long)g.nphase * (t.hi - t.lo);
  out->nonzero_macs = (int64_t)d.n * d.c_in * d.c_out * vh * vw;

  if (bm < 1) bm = 1;
  auto tiles = [&](long long m) { return (m + bm - 1) / bm; };
  for (const AxisGroup& a : gh) {
    for (const AxisGroup& b : gw) {
      // choose border-class splitting per axis for this group pair
      int best_sh = 1, best_sw = 1;
      if (class_split != 1) {
        long long best = -1;
        for (int sh = 1; sh >= 0; --sh)
          for (int sw = 1; sw >= 0; --sw) {
            if (class_split == 0 && (sh || sw)) continue;
            long long cost = 0;
            for (const AxisPiece& ph : axis_pieces(a, sh))
              for (const AxisPiece& pw : axis_pieces(b, sw)) {
                long long m = (long long)d.n * a.nphase * b.nphase * ph.qn * pw.qn;
                cost += tiles(m) * (4LL * (long long)ph.tap_idx.size() * pw.tap_idx.size() + 1);
              }
            if (best < 0 || cost < best) {
              best = cost;
              best_sh = sh;
              best_sw = sw;
            }
          }
      }
      for (const AxisPiece& ph : axis_pieces(a, best_sh)) {
        for (const AxisPiece& pw : axis_pieces(b, best_sw)) {
          huge2_segment s;
          s.phase0_h = a.phase0;
          s.phase0_w = b.phase0;
          s.nphase_h = a.nphase;
          s.nphase_w = b.nphase;
          s.out_step_h = a.out_step;
          s.out_step_w = b.out_step;
          s.q0_h = ph.q0;
          s.q0_w = pw.q0;
          s.qn_h = ph.qn;
          s.qn_w = pw.qn;
          s.in0_h = a.in0;
          s.in0_w = b.in0;
          s.in_dphase_h = a.in_dphase;
          s.in_dphase_w = b.in_dphase;
          s.in_step_h = a.in_step;
          s.in_step_w = b.in_step;
          s.tap_begin = (int32_t)out->taps.size();
          for (int ih : ph.tap_idx)
            for (int iw : pw.tap_idx) {
              huge2_tap t;
              t.kh = a.taps[ih].k;
              t.kw = b.taps[iw].k;
              t.off_h = a.taps[ih].off;
              t.off_w = b.taps[iw].off;
              out->taps.push_back(t);
            }
          s.tap_count = (int32_t)out->taps.size() - s.tap_begin;
          long long m = (long long)d.n * a.nphase * b.nphase * ph.qn * pw.qn;
          out->tile_taps += tiles(m) * s.tap_count;
          out->segs.push_back(s);
        }
      }
    }
  }
  return true;
}

bool build_listed(const huge2_conv_desc& d, int bm, ListedShape* out) {
  if (d.stride_h != 1 || d.stride_w != 1 || (d.dil_h == 1 && d.dil_w == 1)) return false;
  if ((long long)d.r * d.s > 64 || bm < 1) return false;
  int ho, wo;
  if (!output_dims(d, false, &ho, &wo) || ho >= 65536 || wo >= 65536) return false;
  // per axis: the in-range taps of each output coordinate as a bit mask, and
  // the bands (maximal runs of equal masks)
  auto axis = [](int out_size, int in_size, int ksize, int pad, int dil, std::vector<uint64_t>* mask,
                 std::vector<int>* band_start) {
    mask->assign(out_size, 0);
    band_start->clear();
    for (int o = 0; o < out_size; ++o) {
      for (int k = 0; k < ksize; ++k) {
        const long long i = (long long)o - pad + (long long)k * dil;
        if (i >= 0 && i < in_size) (*mask)[o] |= 1ull << k;
      }
      if (o == 0 || (*mask)[o] != (*mask)[o - 1]) band_start->push_back(o);
    }
    band_start->push_back(out_size);
  };
  std::vector<uint64_t> mh, mw;
  std::vector<int> bh, bw;
  axis(ho, d.h, d.r, d.pad_h, d.dil_h, &mh, &bh);
  axis(wo, d.w, d.s, d.pad_w, d.dil_w, &mw, &bw);
  out->pix.clear();
  out->tile_taps.clear();
  out->pix.reserve((size_t)ho * wo);
  const int nbh = (int)bh.size() - 1, nbw = (int)bw.size() - 1;
  for (int a = 0; a < nbh; ++a) {
    for (int bi = 0; bi < nbw; ++bi) {
      const int b = (a % 2 == 0) ? bi : nbw - 1 - bi;  // snake order over the band grid
      // the cell's pixels by phase view, then by position in the view
      for (int ph = 0; ph < d.dil_h; ++ph)
        for (int pw = 0; pw < d.dil_w; ++pw)
          for (int oh = bh[a]; oh < bh[a + 1]; ++oh) {
            if (oh % d.dil_h != ph) continue;
            for (int ow = bw[b]; ow < bw[b + 1]; ++ow)
              if (ow % d.dil_w == pw) out->pix.push_back(((uint32_t)oh << 16) | (uint32_t)ow);
          }
    }
  }
  const int per_img = (int)out->pix.size();
  int64_t nz = 0;
  for (int o = 0; o < ho; ++o) nz += __builtin_popcountll(mh[o]);
  int64_t nzw = 0;
  for (int o = 0; o < wo; ++o) nzw += __builtin_popcountll(mw[o]);
  out->nonzero_macs = (int64_t)d.n * d.c_in * d.c_out * nz * nzw;
  out->issued_rows_taps = 0;
  for (int t0 = 0; t0 < per_img; t0 += bm) {
    std::vector<uint8_t> used((size_t)d.r * d.s, 0);
    for (int i = t0; i < std::min(per_img, t0 + bm); ++i) {
      const uint64_t h = mh[out->pix[i] >> 16], w = mw[out->pix[i] & 0xffff];
      for (int kh = 0; kh < d.r; ++kh)
        if (h >> kh & 1)
          for (int kw = 0; kw < d.s; ++kw)
            if (w >> kw & 1) used[(size_t)kh * d.s + kw] = 1;
    }
    std::vector<huge2_tap> taps;
    for (int kh = 0; kh < d.r; ++kh)
      for (int kw = 0; kw < d.s; ++kw)
        if (used[(size_t)kh * d.s + kw]) {
          huge2_tap t;
          t.kh = kh;
          t.kw = kw;
          t.off_h = kh * d.dil_h;
          t.off_w = kw * d.dil_w;
          taps.push_back(t);
        }
    out->issued_rows_taps += (int64_t)d.n * bm * (int64_t)taps.size();
    out->tile_taps.push_back(std::move(taps));
  }
  return true;
}

}  // namespace huge2
