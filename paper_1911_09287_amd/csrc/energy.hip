// Energy-based (adaptive) compression, coarse-grained (Sec. 4.1 and the
// supplementary section "Compression Based on Preserved Energy"): the band is
// grown from the DC component in whole L-shaped layers until it holds a
// requested fraction of the energy of the layer's input.
//
//   k_bin_energy              per kept bin b: h_v * sum over the N C_in values of
//                             |X[b]|^2 in fp64 (h_v: Parseval on the half plane,
//                             1 in column 0 and in an even width's Nyquist
//                             column, else 2); one block per bin, a fixed-order
//                             tree sum, so results do not depend on scheduling;
//   bl_conv_rate_for_energy   host: per-layer sums, the most layers whose band
//                             still keeps the fraction, and the rate c that makes
//                             bl_conv_plan_create choose exactly that band.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <vector>

#include "common.hpp"

namespace blc {
namespace {

constexpr int kEnergyThreads = 1024;

// S: stored-spectrum element (float2 or bfloat16 pairs)
template <typename S>
__global__ __launch_bounds__(kEnergyThreads) void k_bin_energy(const S* __restrict__ X, double* __restrict__ e,
                                                               long P, int V, int nyq) {
  __shared__ double red[kEnergyThreads];
  const int b = blockIdx.x, tid = threadIdx.x;
  const S* row = X + (size_t)b * P;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  long i = tid;
  // four loads of a thread in flight together
  for (; i + 3 * kEnergyThreads < P; i += 4 * kEnergyThreads) {
    float2 z[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) z[k] = spec_get(row, i + k * kEnergyThreads);
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[k] += (double)z[k].x * z[k].x + (double)z[k].y * z[k].y;
  }
  for (int k = 0; i < P; i += kEnergyThreads, ++k) {
    const float2 z = spec_get(row, i);
    acc[k & 3] += (double)z.x * z.x + (double)z.y * z.y;
  }
  red[tid] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  __syncthreads();
  for (int h = kEnergyThreads / 2; h > 0; h >>= 1) {
    if (tid < h) red[tid] += red[tid + h];
    __syncthreads();
  }
  if (tid == 0) {
    const int v = b % V;
    e[b] = ((v == 0 || v == nyq) ? 1.0 : 2.0) * red[0];
  }
}

}  // namespace
}  // namespace blc

using namespace blc;

extern "C" bl_status_t bl_conv_input_energy(bl_conv_plan_t p, const float* x, void* ws, unsigned flags,
                                            double* energy, void* stream) {
  if (!p || !ws || !energy) return BL_ERR_INVALID_ARG;
  if (flags & ~BL_REUSE_X) return BL_ERR_INVALID_ARG;
  if (!(flags & BL_REUSE_X) && !x) return BL_ERR_INVALID_ARG;
  if (p->kept > 2147483647L) return BL_ERR_UNSUPPORTED;
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* X = static_cast<char*>(ws) + p->off_X;
  const long P = (long)p->N * p->Cin;
  if (!(flags & BL_REUSE_X)) {
    const bl_status_t st = launch_spec_fwd(p, x, X, P, p->Hi, p->Wi, p->pt, p->pl, s);
    if (st != BL_OK) return st;
  }
  const int nyq = (p->Lw % 2 == 0) ? p->Lw / 2 : -1;
  // one block per bin (splitting the bins of small grids over several blocks
  // and summing the slices in a second pass measured slower: the pass costs
  // more than the parallelism gains)
  const double bytes = (p->bf16 ? 4.0 : 8.0) * (double)p->kept * P + 8.0 * (double)p->kept;
  return timed_launch("input_energy", bytes, 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
    if (p->bf16)
      hipExtLaunchKernelGGL(k_bin_energy<unsigned>, dim3((unsigned)p->kept), dim3(kEnergyThreads), 0, s, e0, e1, 0,
                            static_cast<const unsigned*>(X), energy, P, p->V, nyq);
    else
      hipExtLaunchKernelGGL(k_bin_energy<float2>, dim3((unsigned)p->kept), dim3(kEnergyThreads), 0, s, e0, e1, 0,
                            static_cast<const float2*>(X), energy, P, p->V, nyq);
  });
}

namespace {
// The most layers that can be peeled with bin b of plan p still kept.
int bin_last_layer(const bl_conv_plan_s* p, long b) {
  const int r = (int)(b / p->V), v = (int)(b % p->V);
  int tb = p->Lw / 2 - v;
  if (p->ndim != 1) {
    const int u = bl_kept_row(r, p->r_h, p->Lh, p->R);
    const int su = u <= p->Lh / 2 ? u : u - p->Lh;
    tb = std::min(p->Lh / 2 - std::abs(su), tb);
  }
  return tb;
}
}  // namespace

extern "C" bl_status_t bl_conv_rate_for_energy(bl_conv_plan_t p, const double* energy, size_t n, double fraction,
                                               int* t_out, double* c_out, double* preserved_out) {
  if (!p || !energy || n != (size_t)p->kept) return BL_ERR_INVALID_ARG;
  if (!(fraction > 0.0 && fraction <= 1.0)) return BL_ERR_INVALID_ARG;  // also rejects NaN
  const bool one_d = p->ndim == 1;
  const int t_max = one_d ? p->Lw / 2 : std::min(p->Lh / 2, p->Lw / 2);
  // energy and count of the bins whose band ends at layer t (the most layers
  // that can be peeled with the bin still kept)
  std::vector<double> layer_e(t_max + 1, 0.0);
  std::vector<long> layer_n(t_max + 1, 0);
  for (long b = 0; b < p->kept; ++b) {
    const double eb = energy[b];
    if (!(eb >= 0.0) || std::isinf(eb)) return BL_ERR_INVALID_ARG;
    const int tb = bin_last_layer(p, b);
    if (tb < 0 || tb > t_max) return BL_ERR_INVALID_ARG;
    layer_e[tb] += eb;
    layer_n[tb] += 1;
  }
  // summed in the order of the scan below, so that the band of all the bins
  // (and any band that drops only bins without energy) keeps exactly 1
  double total = 0.0;
  for (int t = t_max; t >= 0; --t) total += layer_e[t];
  // the most layers whose band keeps at least the fraction (an input with no
  // energy keeps any fraction with any band)
  int best = p->t;
  double best_f = 1.0;
  double kept_e = 0.0;
  long kept_n = 0, best_n = p->kept;
  for (int t = t_max; t >= p->t; --t) {
    kept_e += layer_e[t];
    kept_n += layer_n[t];
    const double f = total > 0.0 ? kept_e / total : 1.0;
    if (f >= fraction) {
      best = t;
      best_f = f;
      best_n = kept_n;
      break;
    }
  }
  if (t_out) *t_out = best;
  if (preserved_out) *preserved_out = best_f;
  if (c_out) {
    // the plan's rule takes the fewest layers with kept <= (1 - c) total; half
    // a bin of slack keeps the choice away from rounding, and kept counts
    // fall strictly with t
    const double c = 1.0 - ((double)best_n + 0.5) / (double)p->total;
    *c_out = c > 0.0 ? c : 0.0;
  }
  return BL_OK;
}

extern "C" bl_status_t bl_conv_fine_band_for_energy(bl_conv_plan_t p, const double* energy, size_t n,
                                                    double fraction, int* t_out, double* c_out,
                                                    double* preserved_out, unsigned char* keep, size_t keep_cap,
                                                    size_t* keep_n) {
  int t = 0;
  double c = 0.0;
  const bl_status_t st = bl_conv_rate_for_energy(p, energy, n, fraction, &t, &c, nullptr);
  if (st != BL_OK) return st;
  const int t_max = p->ndim == 1 ? p->Lw / 2 : std::min(p->Lh / 2, p->Lw / 2);
  // bins of the coarse band t (plan order), with their layers
  std::vector<long> band;
  std::vector<double> layer_e(t_max + 1, 0.0);
  for (long b = 0; b < p->kept; ++b) {
    const int tb = bin_last_layer(p, b);
    layer_e[tb] += energy[b];
    if (tb >= t) band.push_back(b);
  }
  // the same sums, in the same order, as the coarse rule
  double total = 0.0;
  for (int l = t_max; l >= 0; --l) total += layer_e[l];
  double kept_e = 0.0;
  for (int l = t_max; l > t; --l) kept_e += layer_e[l];
  std::vector<unsigned char> k(band.size(), 1);
  if (t < t_max && total > 0.0) {
    // layer t's bins, largest energy first (equal energies in plan order),
    // added until the band keeps the fraction; the others are dropped
    std::vector<size_t> layer;
    for (size_t i = 0; i < band.size(); ++i)
      if (bin_last_layer(p, band[i]) == t) layer.push_back(i);
    std::stable_sort(layer.begin(), layer.end(),
                     [&](size_t a, size_t b) { return energy[band[a]] > energy[band[b]]; });
    for (size_t i : layer) k[i] = 0;
    for (size_t i : layer) {
      if (kept_e / total >= fraction) break;
      k[i] = 1;
      kept_e += energy[band[i]];
    }
  } else {
    kept_e = total;
  }
  if (keep_n) *keep_n = band.size();
  if (keep) {
    if (keep_cap < band.size()) return BL_ERR_INVALID_ARG;
    std::copy(k.begin(), k.end(), keep);
  }
  if (t_out) *t_out = t;
  if (c_out) *c_out = c;
  if (preserved_out) *preserved_out = total > 0.0 ? kept_e / total : 1.0;
  return BL_OK;
}

namespace blc {
namespace {
// rows of dropped bins set to zero: one block per (bin, slice of the row)
template <typename S>
__global__ __launch_bounds__(256) void k_zero_bins(S* __restrict__ spec, const unsigned char* __restrict__ keep,
                                                   long row) {
  const long b = blockIdx.y;
  if (keep[b]) return;
  S* r = spec + (size_t)b * row;
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < row; i += (long)gridDim.x * 256)
    spec_put(r, (size_t)i, make_float2(0.f, 0.f));
}
}  // namespace
}  // namespace blc

extern "C" bl_status_t bl_conv_zero_bins(bl_conv_plan_t p, void* ws, unsigned which, const unsigned char* keep,
                                         void* stream) {
  if (!p || !ws || !keep) return BL_ERR_INVALID_ARG;
  if (which != BL_SPEC_X && which != BL_SPEC_W) return BL_ERR_INVALID_ARG;
  if (p->kept > 65535) return BL_ERR_UNSUPPORTED;
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* spec = static_cast<char*>(ws) + (which == BL_SPEC_X ? p->off_X : p->off_W);
  const long row = which == BL_SPEC_X ? (long)p->N * p->Cin : (long)p->Cin * p->Cout;
  const long slices = std::max<long>(1, std::min<long>(64, (row + 4095) / 4096));
  const dim3 grid((unsigned)slices, (unsigned)p->kept);
  // traffic: the mask read; the dropped rows written (at most every row)
  const double bytes = (double)p->kept + (p->bf16 ? 4.0 : 8.0) * (double)row * (double)p->kept;
  return timed_launch("zero_bins", bytes, 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
    if (p->bf16)
      hipExtLaunchKernelGGL(k_zero_bins<unsigned>, grid, dim3(256), 0, s, e0, e1, 0, static_cast<unsigned*>(spec),
                            keep, row);
    else
      hipExtLaunchKernelGGL(k_zero_bins<float2>, grid, dim3(256), 0, s, e0, e1, 0, static_cast<float2*>(spec),
                            keep, row);
  });
}
