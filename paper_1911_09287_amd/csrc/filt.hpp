// Filter spectrum at the kept bins, shared by the filter-transform launch and
// the launch that runs it beside the 2-D input transform.
//
// W[b][c][f] = sum over taps (a, b') of w[f][c][a][b'] e^{-2 pi i (u a / Lh + v b' / Lw)}
// for each kept bin b = (u, v) (the padded filter's DFT restricted to the kept
// set, Sec. 3.2.1-3.2.2; the correlation takes its conjugate later).
#pragma once

#include "common.hpp"

namespace blc {

// e^{sign * 2 pi i k / L}, evaluated in double and rounded once to fp32.
__device__ inline float2 unit_root(int k, int L, double sign) {
  double s, c;
  sincospi(2.0 * (double)k / (double)L, &s, &c);
  return make_float2((float)c, (float)(sign * s));
}

__device__ inline void fill_roots(float2* tab, int L, double sign) {
  for (int k = threadIdx.x; k < L; k += blockDim.x) tab[k] = unit_root(k, L, sign);
}

struct FiltGeom {
  int F, C, Kh, Kw;
  int Lh, Lw, r_h, R, V;
  int bins_per_block;
  int xblocks;  // blocks of 256 (c, f) pairs
};

// Filter sizes with a compiled transform.
#define BL_FILT_CASES(X) \
  X(1, 1) X(1, 2) X(1, 3) X(1, 4) X(1, 5) X(1, 6) X(1, 7) X(1, 8) \
  X(2, 2) X(3, 3) X(4, 4) X(5, 5) X(6, 6) X(7, 7) X(8, 8)

// Geometry, roots-of-unity table (or null with use_table false: the blocks
// compute the roots), block count, dynamic LDS bytes and algorithmic bytes of
// the filter transform of a plan.  BL_ERR_UNSUPPORTED for a filter size
// outside BL_FILT_CASES or a grid too large.
bl_status_t filt_setup(const bl_conv_plan_s* p, bool use_table, FiltGeom& g, const float2** roots, long* blocks,
                       size_t* lds, double* bytes);

// One block (id of nb) of the filter transform: a chunk of kept bins for 256
// (c, f) pairs.  smem: at least (Lh + Lw) float2 of LDS.
template <int KH, int KW, typename S>
__device__ __forceinline__ void spec_filt_block(const float* __restrict__ w, const float2* __restrict__ roots,
                                                S* __restrict__ out, const FiltGeom& g, unsigned id, unsigned nb,
                                                float2* smem) {
  // roots: e^{-2 pi i k / Lh} (k < Lh) then e^{-2 pi i k / Lw} (k < Lw), from
  // a table built once per plan, or (roots == nullptr) computed here
  float2* twh = smem;
  float2* tww = twh + g.Lh;
  // logical block: consecutive ids on one XCD (the hardware deals blocks to
  // the 8 XCDs in turn); pair block = id % xblocks, bin chunk = id / xblocks
  if (nb % 8 == 0) id = (id % 8) * (nb / 8) + id / 8;
  const unsigned xblocks = (unsigned)g.xblocks;
  const unsigned bx = id % xblocks, by = id / xblocks;
  const long CF = (long)g.C * g.F;
  const long q = (long)bx * blockDim.x + threadIdx.x;  // q = c * F + f
  const bool live = q < CF;
  const int c = live ? (int)(q / g.F) : 0, f = live ? (int)(q % g.F) : 0;
  // the taps are loaded before the roots are staged, so both loads overlap
  float tap[KH][KW];
  const float* wp = w + ((size_t)f * g.C + c) * KH * KW;
#pragma unroll
  for (int a = 0; a < KH; ++a)
#pragma unroll
    for (int b = 0; b < KW; ++b) tap[a][b] = wp[a * KW + b];
  if (roots) {
    for (int k = threadIdx.x; k < g.Lh + g.Lw; k += blockDim.x) smem[k] = roots[k];
  } else {
    fill_roots(twh, g.Lh, -1.0);
    fill_roots(tww, g.Lw, -1.0);
  }
  __syncthreads();
  if (!live) return;
  const int B = g.R * g.V;
  const int b0 = (int)by * g.bins_per_block;
  const int b1 = min(B, b0 + g.bins_per_block);
  // twiddle indices (u a) mod Lh and (v b) mod Lw, advanced bin by bin
  int r = b0 / g.V, v = b0 - (b0 / g.V) * g.V;
  int ih[KH], iw[KW];
  auto row_start = [&]() {
    const int u = kept_row_d(r, g.r_h, g.Lh, g.R);
#pragma unroll
    for (int a = 0; a < KH; ++a) ih[a] = (int)(((long)u * a) % g.Lh);
  };
  row_start();
#pragma unroll
  for (int b = 0; b < KW; ++b) iw[b] = (int)(((long)v * b) % g.Lw);
  for (int bin = b0; bin < b1; ++bin) {
    float re = 0.f, im = 0.f;
#pragma unroll
    for (int a = 0; a < KH; ++a) {
      // row sum over columns: sum_b tap[a][b] e^{-2 pi i v b / Lw}
      float rr = 0.f, ri = 0.f;
#pragma unroll
      for (int b = 0; b < KW; ++b) {
        const float2 t = tww[iw[b]];
        rr = fmaf(tap[a][b], t.x, rr);
        ri = fmaf(tap[a][b], t.y, ri);
      }
      const float2 t = twh[ih[a]];
      re = fmaf(rr, t.x, fmaf(-ri, t.y, re));
      im = fmaf(rr, t.y, fmaf(ri, t.x, im));
    }
    spec_put(out, (size_t)bin * CF + q, make_float2(re, im));
    if (++v == g.V) {
      v = 0;
      ++r;
      row_start();
#pragma unroll
      for (int b = 0; b < KW; ++b) iw[b] = 0;
    } else {
#pragma unroll
      for (int b = 0; b < KW; ++b) {
        iw[b] += b;
        if (iw[b] >= g.Lw) iw[b] -= g.Lw;
      }
    }
  }
}

}  // namespace blc
