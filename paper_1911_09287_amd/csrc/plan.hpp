// Internal plan structure shared by the host plan code and the launchers.
//
// Every problem is held in "row form": a 2-D layer is an Hi x Wi plane on an
// Lh x Lw grid; a 1-D layer is a single row (Hi = 1, Lh = 1) of length Wi on a
// grid of length Lw.  With Lh = 1 the kept-row set is {u = 0} and the 2-D
// kernels reduce to the 1-D transform, so one set of kernels serves both.
#pragma once

#include <cstddef>
#include <cstdint>
#include <vector>

#include "../../include/blconv.h"

// Tiling of the per-bin contraction [M x K] . [K x N] (complex) over `bins`
// bins: tile height (64 or 128 rows, 64 complex columns) and the number of
// k-splits: 64-row tiles when 128-row ones give fewer than ~512 work items
// (2 per CU of an MI355X), and k-splits while there are still fewer than ~512,
// each split keeping at least 64 complex k (the pass that sums the split
// partials only pays off when the splits are long).  Split partial tiles
// are summed in a fixed order by a separate pass (deterministic results).
struct BlContractTiling {
  int bm, splits;
};
inline BlContractTiling bl_contract_tiling(long M, long N, long K, long bins) {
  BlContractTiling t{M > 64 ? 128 : 64, 1};
  const long tiles = bins * ((M + t.bm - 1) / t.bm) * ((N + 63) / 64);
  if (tiles < 512 && t.bm == 128) {
    t.bm = 64;
  }
  const long tiles2 = bins * ((M + t.bm - 1) / t.bm) * ((N + 63) / 64);
  while (tiles2 * t.splits < 512 && K / (2 * t.splits) >= 64 && t.splits < 16) t.splits *= 2;
  return t;
}

struct bl_conv_plan_s {
  bl_conv_desc_t desc;
  int ndim;
  int N, Cin, Cout;
  // row form
  int Hi, Wi;          // input plane
  int Kh, Kw;          // filter support
  int pt, pb, pl, pr;  // zero padding
  int Hp, Wp;          // padded input
  int Ho, Wo;          // output plane
  int Lh, Lw;          // FFT grid
  int Wh;              // half-plane width Lw/2 + 1
  int t, r_h, r_w;     // peeled layers and radii of the kept band
  int R, V;            // kept rows and kept columns
  long kept, total;
  double c_eff;
  std::vector<uint8_t> mask;  // [Lh][Wh]
  // workspace layout (bytes)
  int wg_chunks;        // bin slices of the weight-gradient inverse DFT
  BlContractTiling ct[3];  // contraction tiling: forward, grad-input, grad-weight
  size_t off_X, off_W, off_DY, off_T, off_DW, off_Part, off_CPart, ws_bytes;
};

// FFT row index of the r-th kept row: the top-left corner (u = 0..r_h) first,
// then the bottom-left corner (u = Lh - r_h .. Lh - 1).
inline int bl_kept_row(int r, int r_h, int Lh, int R) { return r <= r_h ? r : r + (Lh - R); }

// Number of kept rows for radius r on an axis of length L.
inline int bl_rows_for_radius(int r, int L) {
  return (L % 2 == 0 && r == L / 2) ? L : 2 * r + 1;
}
