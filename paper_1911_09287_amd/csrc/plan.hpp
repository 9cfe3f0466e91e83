// Internal plan structure shared by the host plan code and the launchers.
//
// Every problem is held in "row form": a 2-D layer is an Hi x Wi plane on an
// Lh x Lw grid; a 1-D layer is a single row (Hi = 1, Lh = 1) of length Wi on a
// grid of length Lw.  With Lh = 1 the kept-row set is {u = 0} and the 2-D
// kernels reduce to the 1-D transform, so one set of kernels serves both.
#pragma once

#include <cmath>
#include <cstddef>
#include <cstdint>
#include <vector>

#include "../../include/blconv.h"

// Tiling of the per-bin contraction [M x K] . [K x N] (complex) over `bins`
// bins: tile height bm (64 or 128 rows), tile width bn (32 or 64 complex
// columns) and the number of k-splits.  Each candidate is priced by a model
// of a 256-CU part: a CU runs its share of the tiles one after another on its
// matrix cores (the busiest CU sets the time), every tile pays a fixed start
// (operand latency before the first MFMA), and k-splits add a pass that sums
// the partial tiles in a fixed order (deterministic results) at HBM speed.
// Dynamic LDS of one weight-gradient slice (its inverse-DFT weights): with
// the kernel's static LDS (at most 16 KB) a block stays within 64 KB.
constexpr long kWgradSliceLds = 48 * 1024;

struct BlContractTiling {
  int bm, bn, splits;
  int ks;  // groups of 4 waves per block splitting the tile's k range (fp32 tiles, 1 or 2)
};
inline BlContractTiling bl_contract_tiling(long M, long N, long K, long bins) {
  // constants fitted to measured launches of the tiles on an MI355X: the
  // matrix cores reach about 60% (1 or 4 MFMA chains per wave) or 50%
  // (2 chains) of their rate inside a tile
  const double kCUs = 256, kClock = 2.4e9, kStart = 0.3e-6, kHbm = 5.0e12, kPass = 4e-6;
  BlContractTiling best{64, 64, 1, 1};
  double best_t = 1e30;
  const int shapes[4][2] = {{128, 64}, {64, 64}, {128, 32}, {64, 32}};
  for (const auto& sh : shapes) {
    const int bm = sh[0], bn = sh[1];
    if (bm == 128 && M <= 64) continue;
    if (bn == 64 && N <= 32) continue;
    for (int splits = 1; splits <= 16; splits *= 2) {
      const long kper = ((K + splits - 1) / splits + 15) / 16 * 16;
      if (splits > 1 && kper < 64) break;
      const long tiles = bins * ((M + bm - 1) / bm) * ((N + bn - 1) / bn) * splits;
      const double per_cu = std::ceil(tiles / kCUs);
      // one wave per SIMD per tile: (bm/64)(bn/32) MFMAs of 64 cycles per complex k
      const int chains = (bm / 64) * (bn / 32);
      const double mfma = chains * 64.0 * kper / kClock / (chains == 2 ? 0.5 : 0.6);
      double t = per_cu * (mfma + kStart);
      if (splits > 1) t += kPass + 8.0 * bins * M * N * (splits + 1) / kHbm;
      if (t < best_t * 0.98) best_t = t, best = BlContractTiling{bm, bn, splits, 1};
    }
  }
  // no more tiles than compute units: one wave per SIMD would run each tile,
  // so two groups of four waves split its k range instead
  const long tiles = bins * ((M + best.bm - 1) / best.bm) * ((N + best.bn - 1) / best.bn) * best.splits;
  if (tiles <= (long)kCUs && best.bm == 64) best.ks = 2;
  return best;
}

struct bl_conv_plan_s {
  bl_conv_desc_t desc;
  int ndim;
  bool bf16;           // stored spectra X, W, DY as bfloat16 pairs (BL_DESC_BF16_SPECTRA)
  bool fused_fwd;      // forward through the fused small-map kernel where it applies
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
  int wg_bins;          // bins per slice (a multiple of 8)
  int wg_groups;        // groups of 256 threads per block summing parts of a slice (1, 2 or 4)
  BlContractTiling ct[3];  // contraction tiling: forward, grad-input, grad-weight
  // paired backward contraction (one launch for grad-input and grad-weight):
  // k-splits of the two passes (the longer split so that both have tiles of
  // equal k length; partial sums in the contraction-partials area, added by
  // the inverse transforms); 0 when the passes are not paired
  int bp_s1, bp_s2;
  int bp_bm, bp_bn;  // the paired launch's tile shape
  // forward contraction split along k into partial spectra that the 2-D
  // output inverse adds (1: not split), for launches of few tiles
  int fwd_split;
  size_t off_X, off_W, off_DY, off_T, off_DW, off_Part, off_CPart, ws_bytes;
  // small device tables (1-D chirps and filter spectra, weight-gradient
  // inverse-DFT weights), built on a plan's first call that needs them on
  // each device; freed with the plan
  mutable void* tables;
};

// Frees a plan's device tables (null is a no-op).
void bl_plan_tables_free(void* tables);

// Taps of the weight-gradient inverse DFT as its kernels are instantiated.
inline int wgrad_tmax(int T) { return T <= 9 ? T : T <= 16 ? 16 : T <= 32 ? 32 : 64; }

// FFT row index of the r-th kept row: the top-left corner (u = 0..r_h) first,
// then the bottom-left corner (u = Lh - r_h .. Lh - 1).
inline int bl_kept_row(int r, int r_h, int Lh, int R) { return r <= r_h ? r : r + (Lh - R); }

// Number of kept rows for radius r on an axis of length L.
inline int bl_rows_for_radius(int r, int L) {
  return (L % 2 == 0 && r == L / 2) ? L : 2 * r + 1;
}
