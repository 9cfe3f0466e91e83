// Weight-gradient inverse DFT onto the filter taps, sliced over bins: the block
// body shared by its own launch and the launch beside the 2-D inverse
// transform.
//
// dw[f][c][t] = sum over kept bins of Re(DW[b][c][f] E[b][t]),
// E[b][t] = h_v e^{+2 pi i (u a / Lh + v b' / Lw)} / (Lh Lw) (the c2r inverse
// restricted to the filter support; the projected weight gradient, Sec. 1).
#pragma once

#include "common.hpp"

namespace blc {

// Channel tile of the weight-gradient inverse DFT: TC input x 256 / TC output
// channels.  Rows wider than 256 output channels take 32-channel spans of 8
// input channels, so that the gradient rows dw[f][c0 .. c0 + 8][taps] are
// written 8 x taps floats at a time; otherwise a block spans whole rows of
// one input channel.
inline int chan_tile(int taps, int F) { return (taps <= 16 && F > 256) ? 8 : 1; }

struct WgradGeom {
  int F, C, Kh, Kw, T;
  int Lh, Lw, r_h, R, V;
  int bins_per_chunk, chunks;
  int tiles_f;  // 16-filter tiles along F (k_wgrad_tile)
  int nsplit;   // k_wgrad_idft: partial spectra of DW (their slices are more slices; 0 or 1: one)
  unsigned long long pstride;  // complex values between two partial spectra
};

// LDS of the transposed write (TC > 1), floats.
template <int TMAX, int TC>
constexpr int wgrad_res_floats() { return TC > 1 ? (kThreads / TC) * TC * TMAX : 1; }

// One block of the sliced inverse DFT: channel block bx, slice by (bin chunk
// by % chunks of partial spectrum by / chunks); `sliced`: more than one slice
// (partial sums to `part`, added later by k_wgrad_reduce).  E: the launch's
// dynamic LDS (bins_per_chunk x TMAX float2); res: wgrad_res_floats floats.
template <int TMAX, int TC>
__device__ __forceinline__ void wgrad_idft_block(const float2* __restrict__ DW, const float2* __restrict__ Et,
                                                 float* __restrict__ dw, float* __restrict__ part, const WgradGeom& g,
                                                 unsigned bx, unsigned by, bool sliced, float2* E, float* res) {
  constexpr int TF = kThreads / TC;
  const int B = g.R * g.V;
  const int sp = by / g.chunks;
  const int b0 = (by - sp * g.chunks) * g.bins_per_chunk;
  const int nb = min(g.bins_per_chunk, B - b0);
  DW += (size_t)sp * g.pstride;
  // copy this slice of the table, four loads of a thread in flight together
  const float2* Es = Et + (size_t)b0 * g.T;
  for (int e0 = threadIdx.x; e0 < nb * TMAX; e0 += 4 * kThreads) {
    float2 v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int e = e0 + k * kThreads, bb = e / TMAX, t = e - bb * TMAX;
      v[k] = (e < nb * TMAX && t < g.T) ? Es[bb * g.T + t] : make_float2(0.f, 0.f);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (e0 + k * kThreads < nb * TMAX) E[e0 + k * kThreads] = v[k];
  }
  __syncthreads();
  const long Q = (long)g.C * g.F;
  // TC == 1: 256 consecutive pairs q = c F + f per block; else a TC x TF tile
  const int tiles_f = (g.F + TF - 1) / TF;
  const int c0 = (bx / tiles_f) * TC, f0 = (bx % tiles_f) * TF;
  const int tc = threadIdx.x / TF, tf = threadIdx.x - (threadIdx.x / TF) * TF;
  const long q1 = (long)bx * kThreads + threadIdx.x;
  const int c = TC == 1 ? (int)(q1 / g.F) : c0 + tc, f = TC == 1 ? (int)(q1 % g.F) : f0 + tf;
  const bool valid = TC == 1 ? q1 < Q : (c < g.C && f < g.F);
  float acc[TMAX];
#pragma unroll
  for (int t = 0; t < TMAX; ++t) acc[t] = 0.f;
  const float2* src = DW + (size_t)b0 * Q + (valid ? (long)c * g.F + f : 0);
  // 8 bins' loads in flight at a time (indices clamped, surplus values zeroed)
  for (int bb = 0; bb < nb; bb += 8) {
    float2 d[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) d[j] = src[(size_t)min(bb + j, nb - 1) * Q];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const bool in = bb + j < nb;
      const float2 dj = in ? d[j] : make_float2(0.f, 0.f);
      const float2* Eb = E + min(bb + j, nb - 1) * TMAX;
#pragma unroll
      for (int t = 0; t < TMAX; ++t) acc[t] = fmaf(dj.x, Eb[t].x, fmaf(-dj.y, Eb[t].y, acc[t]));
    }
  }
  if (sliced) {
    if (valid) {
#pragma unroll
      for (int t = 0; t < TMAX; ++t)
        if (t < g.T) part[((size_t)by * g.T + t) * Q + (size_t)c * g.F + f] = acc[t];
    }
    return;
  }
  if (TC == 1) {
    if (valid) {
      float* o = dw + ((size_t)f * g.C + c) * g.T;
#pragma unroll
      for (int t = 0; t < TMAX; ++t)
        if (t < g.T) o[t] = acc[t];
    }
    return;
  }
  // transpose through LDS: res[tf][tc][t], then each output row f gets its
  // TC x T contiguous floats
#pragma unroll
  for (int t = 0; t < TMAX; ++t)
    if (t < g.T) res[(tf * TC + tc) * g.T + t] = acc[t];
  __syncthreads();
  const int seg = TC * g.T;
  for (int e = threadIdx.x; e < TF * seg; e += kThreads) {
    const int ef = e / seg, r = e - ef * seg;
    const int oc = c0 + r / g.T, of = f0 + ef;
    if (oc < g.C && of < g.F) dw[((size_t)of * g.C + c0) * g.T + r] = res[e];
  }
}

// Wide layers (many (c, f) pairs): one block per 64 consecutive pairs and all
// bins (of one spectrum, or with PARTS the sum of g.nsplit partial spectra
// g.pstride apart), its waves each reducing a share of the bins; the shares are
// added in a fixed order through LDS and written straight to dw, so no
// partial sums leave the block.  E comes from a table built once per plan.
// E: the launch's dynamic LDS ([kept][TMAX] float2, zero beyond T: the bin loop
// has no branches); red: NW * 64 * TMAX floats.  Block bx of 64 * NW threads.
template <int TMAX, int NW, bool PARTS = false>
__device__ __forceinline__ void wgrad_wide_block(const float2* __restrict__ DW, const float2* __restrict__ Et,
                                                 float* __restrict__ dw, const WgradGeom& g, unsigned bx, float2* E,
                                                 float* red) {
  const int B = g.R * g.V;
  for (int e = threadIdx.x; e < B * TMAX; e += blockDim.x) {
    const int bb = e / TMAX, t = e - bb * TMAX;
    E[e] = t < g.T ? Et[bb * g.T + t] : make_float2(0.f, 0.f);
  }
  __syncthreads();
  const unsigned Q = (unsigned)g.C * g.F;
  const int lane = threadIdx.x & 63, grp = threadIdx.x >> 6;
  const unsigned q = bx * 64u + lane;
  const bool valid = q < Q;
  const int bb0 = grp * B / NW, bb1 = (grp + 1) * B / NW;
  float acc[TMAX];
#pragma unroll
  for (int t = 0; t < TMAX; ++t) acc[t] = 0.f;
  const float2* src = DW + (valid ? q : 0u);
  // 8 bins' loads in flight at a time (indices clamped, surplus values zeroed);
  // with partial spectra (nsplit > 1) each bin is their sum, taken in order
  for (int bb = bb0; bb < bb1; bb += 8) {
    float2 d[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) d[j] = src[(size_t)min(bb + j, bb1 - 1) * Q];
    if constexpr (PARTS) {
      for (int sp = 1; sp < g.nsplit; ++sp) {
        const float2* ps = src + (size_t)sp * g.pstride;
        float2 e[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) e[j] = ps[(size_t)min(bb + j, bb1 - 1) * Q];
#pragma unroll
        for (int j = 0; j < 8; ++j) d[j] = make_float2(d[j].x + e[j].x, d[j].y + e[j].y);
      }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const bool in = bb + j < bb1;
      const float2 dj = in ? d[j] : make_float2(0.f, 0.f);
      const float2* Eb = E + min(bb + j, bb1 - 1) * TMAX;
#pragma unroll
      for (int t = 0; t < TMAX; ++t) acc[t] = fmaf(dj.x, Eb[t].x, fmaf(-dj.y, Eb[t].y, acc[t]));
    }
  }
#pragma unroll
  for (int t = 0; t < TMAX; ++t) red[(grp * 64 + lane) * TMAX + t] = acc[t];
  __syncthreads();
  if (grp == 0 && valid) {
    const int c = (int)(q / g.F), f = (int)(q % g.F);
    float* o = dw + ((size_t)f * g.C + c) * g.T;
#pragma unroll
    for (int t = 0; t < TMAX; ++t) {
      float sum = red[lane * TMAX + t];
#pragma unroll
      for (int w = 1; w < NW; ++w) sum += red[(w * 64 + lane) * TMAX + t];
      if (t < g.T) o[t] = sum;
    }
  }
}

// The one-pass wide path applies to a plan (see launch_wgrad_idft).
bool wgrad_wide(const bl_conv_plan_s* p);
// Its E table (E[bin][t], built once per plan).
bl_status_t wgrad_table(const bl_conv_plan_s* p, const float2** Et);

// Geometry of the sliced path for a plan (nsplit partial spectra of DW): the
// channel blocks, slices (nsplit x bin chunks), dynamic LDS bytes, channel
// tile and the E table; false when the plan's inverse DFT takes another path
// (channel tiles over all bins, or wide one-pass blocks) or the slices do not
// fit.
bool wgrad_sliced_setup(const bl_conv_plan_s* p, int nsplit, WgradGeom& g, long* xblocks, int* slices, size_t* lds,
                        int* tc, const float2** Et);
// Sum of a sliced launch's partial sums into dw (when it had more than one slice).
bl_status_t launch_wgrad_reduce(const bl_conv_plan_s* p, const float* part, float* dw, const WgradGeom& g,
                                hipStream_t s);

}  // namespace blc
