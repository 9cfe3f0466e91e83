// Fused forward pass for small maps: one kernel takes the input planes of a
// sample to its output planes for a group of output channels, with the
// transform, the per-bin channel contraction and the inverse transform in
// between held in LDS and registers instead of passing through HBM as stored
// spectra (the fused variant of Sec. 3.3's pipeline; the filter spectrum W is
// the plan's stored one, computed once per call by spec_filt or reused).
//
//   k_small_fwd  block = (sample n, FC output channels).  For each chunk of CC
//                input channels: the planes go to LDS, a pruned row DFT (kept
//                columns only) and column DFT (kept rows only) form X[b][c]
//                for the kept bins, and each thread accumulates its (bin,
//                output channel) pairs of Y = sum_c X conj(W) in registers.
//                Then Y goes to LDS, an inverse column DFT (output rows only)
//                and a real row DFT (output columns only, Hermitian weights)
//                write the output window.  The blocks of the first channel
//                group also store X in the workspace, so the map-reuse flags
//                of the backward passes keep their meaning.
//
// Every sum runs in a fixed order, so results do not depend on scheduling.
// The contraction runs on the vector ALUs, one (bin, output channel) pair per
// thread and input channel per step, and each block transforms its sample's
// planes again for every output-channel group.  Measured on the 4x4, 8x8 and
// 16x16 workload layers this costs 1.6-11x the unfused pipeline (whose
// contraction runs on the matrix cores), so the path is opt-in only.
#include <algorithm>
#include <cmath>

#include "common.hpp"

namespace blc {
namespace {

constexpr int kSmallThreads = 256;
constexpr int kSmallPairs = 4;  // (bin, output channel) accumulators per thread

struct SmallArgs {
  int N, Cin, Cout;
  int Hi, Wi, pt, pl;  // input plane and its placement in the grid
  int Ho, Wo;          // output window (at the grid origin)
  int Lh, Lw, r_h, R, V, kept;
  int FC, CC;          // output channels per block, input channels per chunk
  float scale;         // 1 / (Lh Lw)
  int store_x;         // write X[b][n][c] to the workspace
};

// e^{-2 pi i k / L}, evaluated in double and rounded once to fp32
__device__ inline float2 fwd_root(int k, int L) {
  double s, c;
  sincospi(2.0 * (double)k / (double)L, &s, &c);
  return make_float2((float)c, (float)(-s));
}

__global__ __launch_bounds__(kSmallThreads) void k_small_fwd(const float* __restrict__ x,
                                                            const float2* __restrict__ W, float* __restrict__ y,
                                                            float2* __restrict__ Xout, SmallArgs g) {
  extern __shared__ float2 sm[];
  float2* th = sm;              // Lh
  float2* tw = th + g.Lh;       // Lw
  float2* work = tw + g.Lw;
  float2* T1 = work;                                     // CC * Hi * V: row-pass results
  float2* Xs = T1 + g.CC * g.Hi * g.V;                   // kept * CC
  float* xs = reinterpret_cast<float*>(Xs + g.kept * g.CC);  // CC * Hi * Wi
  const int tid = threadIdx.x;
  const int n = blockIdx.x, f0 = blockIdx.y * g.FC;
  const int fc = min(g.FC, g.Cout - f0);
  const int npairs = g.kept * fc;

  for (int k = tid; k < g.Lh; k += kSmallThreads) th[k] = fwd_root(k, g.Lh);
  for (int k = tid; k < g.Lw; k += kSmallThreads) tw[k] = fwd_root(k, g.Lw);

  float2 acc[kSmallPairs];
#pragma unroll
  for (int s = 0; s < kSmallPairs; ++s) acc[s] = make_float2(0.f, 0.f);

  const int plane = g.Hi * g.Wi;
  for (int c0 = 0; c0 < g.Cin; c0 += g.CC) {
    const int cc = min(g.CC, g.Cin - c0);
    __syncthreads();  // the previous chunk's LDS is no longer read
    const float* src = x + ((size_t)n * g.Cin + c0) * plane;
    for (int e = tid; e < cc * plane; e += kSmallThreads) xs[e] = src[e];
    __syncthreads();
    // row pass: T1[c][i][v] = sum_j x[c][i][j] e^{-2 pi i v (j + pl) / Lw}
    for (int e = tid; e < cc * g.Hi * g.V; e += kSmallThreads) {
      const int v = e % g.V, ci = e / g.V;
      const float* xr = xs + ci * g.Wi;
      int idx = (v * g.pl) % g.Lw;
      float re = 0.f, im = 0.f;
      for (int j = 0; j < g.Wi; ++j) {
        const float2 w = tw[idx];
        re = fmaf(xr[j], w.x, re);
        im = fmaf(xr[j], w.y, im);
        idx += v;
        if (idx >= g.Lw) idx -= g.Lw;
      }
      T1[e] = make_float2(re, im);
    }
    __syncthreads();
    // column pass over kept rows: Xs[b][c] = sum_i T1[c][i][v] e^{-2 pi i u (i + pt) / Lh}
    for (int e = tid; e < g.kept * cc; e += kSmallThreads) {
      const int c = e % cc, b = e / cc;
      const int r = b / g.V, v = b - r * g.V;
      const int u = kept_row_d(r, g.r_h, g.Lh, g.R);
      int idx = (u * g.pt) % g.Lh;
      float re = 0.f, im = 0.f;
      const float2* tc = T1 + c * g.Hi * g.V + v;
      for (int i = 0; i < g.Hi; ++i) {
        const float2 a = tc[i * g.V];
        const float2 w = th[idx];
        re = fmaf(a.x, w.x, fmaf(-a.y, w.y, re));
        im = fmaf(a.x, w.y, fmaf(a.y, w.x, im));
        idx += u;
        if (idx >= g.Lh) idx -= g.Lh;
      }
      const float2 val = make_float2(re, im);
      Xs[b * g.CC + c] = val;
      if (g.store_x && blockIdx.y == 0) Xout[((size_t)b * g.N + n) * g.Cin + c0 + c] = val;
    }
    __syncthreads();
    // contraction: pair q = (bin q / fc, channel q % fc), Y += X conj(W) over the chunk
#pragma unroll
    for (int s = 0; s < kSmallPairs; ++s) {
      const int q = tid + kSmallThreads * s;
      if (q < npairs) {
        const int b = q / fc, f = q - b * fc;
        const float2* xp = Xs + b * g.CC;
        const float2* wp = W + ((size_t)b * g.Cin + c0) * g.Cout + f0 + f;
        float2 a = acc[s];
        for (int c = 0; c < cc; ++c) {
          const float2 xv = xp[c], wv = wp[(size_t)c * g.Cout];
          a.x = fmaf(xv.x, wv.x, fmaf(xv.y, wv.y, a.x));
          a.y = fmaf(xv.y, wv.x, fmaf(-xv.x, wv.y, a.y));
        }
        acc[s] = a;
      }
    }
  }
  __syncthreads();  // the last chunk's LDS is no longer read
  // inverse: Ys[b][f] in LDS, then the output window's rows and columns
  float2* Ys = work;                  // kept * fc
  float2* Z = Ys + g.kept * g.FC;     // fc * Ho * V
#pragma unroll
  for (int s = 0; s < kSmallPairs; ++s) {
    const int q = tid + kSmallThreads * s;
    if (q < npairs) Ys[q] = acc[s];
  }
  __syncthreads();
  // column pass: Z[f][i][v] = sum_r Y[(r, v)][f] e^{+2 pi i u_r i / Lh}
  for (int e = tid; e < fc * g.Ho * g.V; e += kSmallThreads) {
    const int v = e % g.V, t = e / g.V;
    const int i = t % g.Ho, f = t / g.Ho;
    float re = 0.f, im = 0.f;
    for (int r = 0; r < g.R; ++r) {
      const int u = kept_row_d(r, g.r_h, g.Lh, g.R);
      const float2 a = Ys[(r * g.V + v) * fc + f];
      const float2 w = cconj(th[(u * i) % g.Lh]);
      re = fmaf(a.x, w.x, fmaf(-a.y, w.y, re));
      im = fmaf(a.x, w.y, fmaf(a.y, w.x, im));
    }
    Z[e] = make_float2(re, im);
  }
  __syncthreads();
  // row pass (c2r): y = scale * sum_v h_v Re(Z[f][i][v] e^{+2 pi i v j / Lw}),
  // h_v = 1 in column 0 and an even width's Nyquist column, else 2
  const int nyq = (g.Lw % 2 == 0) ? g.Lw / 2 : -1;
  float* dst = y + ((size_t)n * g.Cout + f0) * g.Ho * g.Wo;
  for (int e = tid; e < fc * g.Ho * g.Wo; e += kSmallThreads) {
    const int j = e % g.Wo, t = e / g.Wo;
    const float2* zr = Z + t * g.V;  // t = f * Ho + i
    float a = 0.f;
    int idx = 0;
    for (int v = 0; v < g.V; ++v) {
      const float2 z = zr[v];
      const float2 w = cconj(tw[idx]);
      const float h = (v == 0 || v == nyq) ? 1.f : 2.f;
      a = fmaf(h, fmaf(z.x, w.x, -z.y * w.y), a);
      idx += j;
      if (idx >= g.Lw) idx -= g.Lw;
    }
    dst[e] = a * g.scale;
  }
}

// LDS bytes of a block for CC input channels and FC output channels
size_t small_lds(const SmallArgs& g) {
  const size_t fwd = (size_t)g.CC * g.Hi * g.V * 8 + (size_t)g.kept * g.CC * 8 + (size_t)g.CC * g.Hi * g.Wi * 4;
  const size_t inv = (size_t)g.kept * g.FC * 8 + (size_t)g.FC * g.Ho * g.V * 8;
  return (size_t)(g.Lh + g.Lw) * 8 + std::max(fwd, inv);
}

}  // namespace

bool small_fwd_eligible(const bl_conv_plan_s* p) {
  if (p->ndim != 2 || p->bf16) return false;
  if (p->kept > kSmallThreads * kSmallPairs) return false;  // at least one output channel per block
  if ((long)p->N * p->Cin * p->Hi * p->Wi >= 2147483647L || (long)p->kept * p->N * p->Cin >= 2147483647L)
    return false;
  SmallArgs g{};
  g.Hi = p->Hi; g.Wi = p->Wi; g.Ho = p->Ho; g.Wo = p->Wo;
  g.Lh = p->Lh; g.Lw = p->Lw; g.V = p->V; g.kept = (int)p->kept;
  g.CC = 1; g.FC = 1;
  return small_lds(g) <= kMaxLds;
}

bl_status_t launch_small_fwd(const bl_conv_plan_s* p, const float* x, const float2* Wf, float* y, float2* X,
                             hipStream_t s) {
  if (!small_fwd_eligible(p)) return BL_ERR_UNSUPPORTED;
  SmallArgs g{};
  g.N = p->N; g.Cin = p->Cin; g.Cout = p->Cout;
  g.Hi = p->Hi; g.Wi = p->Wi; g.pt = p->pt; g.pl = p->pl;
  g.Ho = p->Ho; g.Wo = p->Wo;
  g.Lh = p->Lh; g.Lw = p->Lw; g.r_h = p->r_h; g.R = p->R; g.V = p->V; g.kept = (int)p->kept;
  g.scale = 1.0f / ((float)p->Lh * (float)p->Lw);
  g.store_x = 1;
  // output channels per block: about 512 blocks, within the accumulators and LDS
  const int fmax = std::max(1, (kSmallThreads * kSmallPairs) / g.kept);
  const long want = ((long)p->N * p->Cout + 511) / 512;
  g.FC = (int)std::max<long>(1, std::min<long>({(long)fmax, want, (long)p->Cout}));
  g.CC = 1;
  while (g.FC > 1 && small_lds(g) > kMaxLds) --g.FC;
  // input channels per chunk: as many as LDS holds, at most 64
  g.CC = 1;
  while (g.CC < std::min(64, p->Cin)) {
    SmallArgs t = g;
    t.CC = g.CC * 2;
    if (small_lds(t) > kMaxLds) break;
    g.CC = t.CC;
  }
  g.CC = std::min(g.CC, p->Cin);
  const size_t lds = small_lds(g);
  const dim3 grid((unsigned)p->N, (unsigned)((p->Cout + g.FC - 1) / g.FC));
  if (grid.y > 65535) return BL_ERR_UNSUPPORTED;
  // compulsory traffic: x read, W read, y and X written
  const double bytes = 4.0 * p->N * p->Cin * p->Hi * p->Wi + 8.0 * p->kept * p->Cin * p->Cout +
                       4.0 * p->N * p->Cout * p->Ho * p->Wo + 8.0 * p->kept * p->N * p->Cin;
  const double flops = 8.0 * p->kept * p->N * p->Cin * p->Cout;
  return timed_launch("small_fwd", bytes, flops, s, [&](hipEvent_t e0, hipEvent_t e1) {
    hipExtLaunchKernelGGL(k_small_fwd, grid, dim3(kSmallThreads), lds, s, e0, e1, 0, x, Wf, y, X, g);
  });
}

}  // namespace blc
