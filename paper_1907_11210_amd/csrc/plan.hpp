// plan.hpp -- host-side phase decomposition for libhuge2 (no HIP calls).
//
// Section 3.1 of the paper (Eq. 1-4) splits a stride-s transposed kernel into
// s*s patterns: the output phase (o mod s) selects the kernel taps whose
// index has the matching residue, and each pattern is a dense convolution
// over the un-inflated input.  This file does that split per spatial axis,
// then refines each phase into border classes (maximal q-intervals on which
// the set of in-range taps is constant) so that the GEMM of a segment never
// multiplies a padding zero, and finally forms 2-D segments as products of
// per-axis pieces.
#pragma once

#include <cstdint>
#include <vector>

#include "huge2.h"

namespace huge2 {

// One kernel tap along one axis: kernel index k, input offset off (added to
// in0 + in_dphase * phase_index + in_step * q), and the q-interval [lo, hi)
// on which the read is in range.
struct AxisTap {
  int k, off, lo, hi;
};

// A run of consecutive phases along one axis that share Q and tap validity.
struct AxisGroup {
  int phase0, nphase, out_step;
  int q_count;                 // q in [0, q_count)
  int in0, in_dphase, in_step;
  std::vector<AxisTap> taps;   // taps valid somewhere in [0, q_count)
};

// One piece of an AxisGroup: a q-interval and the taps used on it.
struct AxisPiece {
  int q0, qn;
  std::vector<int> tap_idx;    // indices into AxisGroup::taps
};

// Decomposition of one axis.  Returns false if the axis is invalid.
//   transposed: o = i*stride - pad + k*dil
//   otherwise:  i = o*stride - pad + k*dil
bool decompose_axis(bool transposed, int in_size, int out_size, int ksize, int stride, int pad,
                    int dil, std::vector<AxisGroup>* groups);

// Border classes of one group: split=false -> one piece [0, Q) with every tap.
std::vector<AxisPiece> axis_pieces(const AxisGroup& g, bool split);

struct PlanShape {
  std::vector<huge2_segment> segs;
  std::vector<huge2_tap> taps;
  int64_t nonzero_macs = 0;  // structural products (closed form over the axes)
  int64_t tile_taps = 0;     // cost model: sum over segments of M-tiles x taps
};

// Output size, or false if the descriptor is invalid / the output is empty.
bool output_dims(const huge2_conv_desc& d, bool transposed, int* ho, int* wo);

// Validation shared by every entry point; returns HUGE2_OK or an error.
huge2_status validate_desc(const huge2_conv_desc* d, bool transposed);

// class_split: 0 = one piece per phase group, 1 = always split into border
// classes, 2 = choose per (group_h, group_w) by the tile cost model with
// M-tile height bm.
bool build_shape(const huge2_conv_desc& d, bool transposed, int class_split, int bm,
                 PlanShape* out);

// Listed form of a stride-1 dilated conv (section 3.2.2).  The output pixels
// of one image are listed in this order: the 2-D border cells (products of
// the per-axis bands on which the set of in-range taps is constant) in snake
// order over the grid of bands, and inside a cell by phase view (oh mod
// dil_h, ow mod dil_w), then by position in the view.  Every phase view's
// pixels with one tap set are thus one run of the list, and each tile of bm
// consecutive pixels uses the union of its pixels' tap sets (adjacent cells
// in snake order have nested tap sets for three bands per axis, so that union
// is the larger cell's set).  The same list serves every image.
struct ListedShape {
  std::vector<uint32_t> pix;                     // per image: (oh << 16) | ow
  std::vector<std::vector<huge2_tap>> tile_taps; // per tile of bm pixels of one image
  int64_t nonzero_macs = 0;
  int64_t issued_rows_taps = 0;  // sum over tiles (all images) of bm x taps
};
// False when the form does not apply (transposed, a stride above 1, dilation
// 1 on both axes, outputs of 65536 rows or columns, more than 64 taps).
bool build_listed(const huge2_conv_desc& d, int bm, ListedShape* out);

}  // namespace huge2
