// 2-D kept spectra on grids of size (2 MH) x (2 MW) with MH, MW odd (gfx950).
//
// Forward (real planes -> kept bins, Sec. 3.2.1 zero padding, Sec. 3.2.2 band):
//   row pass    one thread per input row: the real 2MW-point DFT of the padded
//               row is one MW-point complex DFT of z[q] = x[2q] + i x[2q+1],
//               split by conjugate symmetry; only columns v < V are kept.
//   column pass per (plane, kept column): the 2MH-point DFT over the padded
//               rows is two MH-point DFTs (even and odd rows) and one radix-2
//               butterfly, on one thread or split over a lane pair (one DFT
//               per thread, butterfly across the pair); only kept rows are
//               written, bin-major.
// Inverse (kept bins -> real window), the mirror image:
//   column pass per (plane, kept column): zero-filled 2MH-point inverse DFT
//               as two MH-point inverse DFTs (decimation in frequency), on one
//               thread or one per thread of a lane pair.
//   row pass    one thread per output row: the Hermitian (c2r) 2MW-point
//               inverse as one MW-point complex inverse DFT whose real and
//               imaginary parts are the even and odd samples; the imaginary
//               parts of the DC and Nyquist columns are dropped.
// Odd-length DFTs pair inputs j and M - j, so each output pair k, M - k costs
// (M - 1) complex x real products; all twiddles are compile-time constants.
// A block handles G planes; rows go through LDS once for the transpose.
#include <algorithm>
#include <cmath>

#include "common.hpp"
#include "filt.hpp"
#include "wgrad.hpp"

namespace blc {
namespace {

// ---- compile-time trigonometry (Taylor series after exact reduction) --------
constexpr double kPi = 3.141592653589793238462643383279502884;

constexpr double cx_sin_small(double x) {  // |x| <= pi / 2
  double term = x, sum = x;
  for (int n = 1; n < 16; ++n) {
    term *= -x * x / ((2.0 * n) * (2.0 * n + 1.0));
    sum += term;
  }
  return sum;
}
constexpr double cx_cos_small(double x) {
  double term = 1.0, sum = 1.0;
  for (int n = 1; n < 16; ++n) {
    term *= -x * x / ((2.0 * n - 1.0) * (2.0 * n));
    sum += term;
  }
  return sum;
}
// cos and sin of 2 pi k / n, k in [0, n): reduce to the first quadrant exactly.
constexpr double cx_cos2pi(int k, int n) {
  // angle = 2 pi k / n = (pi / 2) * (4k / n); quadrant q = floor(4k / n)
  const int q = (4 * k) / n;
  const double r = (kPi / 2.0) * ((4.0 * k - (double)q * n) / n);  // in [0, pi/2)
  switch (q & 3) {
    case 0: return cx_cos_small(r);
    case 1: return -cx_sin_small(r);
    case 2: return -cx_cos_small(r);
    default: return cx_sin_small(r);
  }
}
constexpr double cx_sin2pi(int k, int n) {
  const int q = (4 * k) / n;
  const double r = (kPi / 2.0) * ((4.0 * k - (double)q * n) / n);
  switch (q & 3) {
    case 0: return cx_sin_small(r);
    case 1: return cx_cos_small(r);
    case 2: return -cx_sin_small(r);
    default: return -cx_cos_small(r);
  }
}

// cos(2 pi k / N) and sin(2 pi k / N) for k < N.
template <int N>
struct Trig {
  float c[N], s[N];
  constexpr Trig() : c(), s() {
    for (int k = 0; k < N; ++k) {
      c[k] = (float)cx_cos2pi(k, N);
      s[k] = (float)cx_sin2pi(k, N);
    }
  }
};
template <int N>
__device__ constexpr Trig<N> kTrig{};

// M-point DFT (M odd) of z into Z; INV selects e^{+2 pi i jk / M}.
template <int M, bool INV>
__device__ __forceinline__ void dft_odd(const float2* z, float2* Z) {
  constexpr int H = (M - 1) / 2;
  float2 a[H + 1], b[H + 1];
  float2 s = z[0];
#pragma unroll
  for (int j = 1; j <= H; ++j) {
    a[j] = cadd(z[j], z[M - j]);
    b[j] = csub(z[j], z[M - j]);
    s = cadd(s, a[j]);
  }
  Z[0] = s;
#pragma unroll
  for (int k = 1; k <= H; ++k) {
    float2 P = z[0], Q = make_float2(0.f, 0.f);
#pragma unroll
    for (int j = 1; j <= H; ++j) {
      const float c = kTrig<M>.c[(j * k) % M], sn = kTrig<M>.s[(j * k) % M];
      P.x = fmaf(a[j].x, c, P.x);
      P.y = fmaf(a[j].y, c, P.y);
      Q.x = fmaf(b[j].x, sn, Q.x);
      Q.y = fmaf(b[j].y, sn, Q.y);
    }
    const float2 minus = make_float2(P.x + Q.y, P.y - Q.x);  // P - iQ
    const float2 plus = make_float2(P.x - Q.y, P.y + Q.x);   // P + iQ
    Z[k] = INV ? plus : minus;
    Z[M - k] = INV ? minus : plus;
  }
}

// e^{-2 pi i k / N} (or its conjugate) as a compile-time constant.
template <int N, bool INV>
__device__ __forceinline__ float2 root(int k) {
  const float c = kTrig<N>.c[k % N], s = kTrig<N>.s[k % N];
  return make_float2(c, INV ? s : -s);
}

// Value of the other lane of an even/odd lane pair (DPP quad permutation 1 0 3 2).
__device__ __forceinline__ float swap_pair(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));
}
__device__ __forceinline__ float2 swap_pair(float2 a) { return make_float2(swap_pair(a.x), swap_pair(a.y)); }

// Flag in Fft2Args::K of the inverse: the output window's rows are whole float4s.
constexpr unsigned kInvVec4 = 0x80000000u;

struct Fft2Args {
  int Hin, Win;    // forward: input plane; inverse: output window (OH, OW)
  int oi, oj;      // forward: placement offset; inverse: crop origin
  int r_h, R, V;   // kept band
  unsigned P;      // planes
  int G;           // planes per block
  int PS;          // LDS plane stride of the column-major spectra (complex)
  unsigned q4;     // Win / 4 (forward) or OW (inverse): divisor of the flat copy
  unsigned magic;  // ceil(2^32 / q4) for q4 > 1: e / q4 == umulhi(e, magic) for the block's e
  unsigned K;      // plane groups per 128-byte line of a bin row (plane_group)
  float scale;     // inverse: 1 / (Lh Lw)
  unsigned nsplit;               // inverse: partial spectra to add (0 or 1: one spectrum)
  unsigned long long pstride;    // inverse: complex values between two partial spectra
};

// A kept bin of the inverse's input: with PARTS the sum of its nsplit partial
// spectra in order, else one load (a separate instantiation, so that the
// common case keeps its code).
template <bool PARTS>
__device__ __forceinline__ float2 load_parts(const float2* q, const Fft2Args& g) {
  float2 v = q[0];
  if constexpr (PARTS)
    for (unsigned s = 1; s < g.nsplit; ++s) v = cadd(v, q[(size_t)s * g.pstride]);
  return v;
}

// Index of kept row u (or -1): the top-left corner rows 0..r_h, then the
// bottom-left corner rows Lh - (R - r_h - 1) .. Lh - 1.
__device__ __forceinline__ int row_slot(int u, int r_h, int R, int LH) {
  if (u <= r_h) return u;
  const int r = u - (LH - R);
  return r > r_h ? r : -1;
}

// Plane group of a block.  A block's planes form runs of G values in every bin
// row of the bin-major spectra; where a run is shorter than a 128-byte line,
// the K adjacent groups that fill one line are given to blocks of one XCD (the
// hardware deals consecutive blocks to the 8 XCDs in turn), so the line is
// fetched into that XCD's L2 once rather than by K XCDs.  Blocks in flight
// still cover one contiguous range of planes.  Trailing blocks short of a
// whole set of 8 K keep their own index.
__device__ inline unsigned plane_group(unsigned b, unsigned nb, unsigned K) {
  const unsigned set = 8u * K;
  if (K <= 1 || b >= nb / set * set) return b;
  const unsigned r = b % set;
  return b - r + (r % 8u) * K + r / 8u;
}

// LDS layout (complex spectra, column-major per plane): S[p * PS + v * (LH + 1) + i],
// so a column thread reads its LH rows at fixed offsets.
// S: stored-spectrum element of the output (float2 or bfloat16 pairs)
// One block (id of nb) of the forward transform; sm: the launch's LDS.
template <int MH, int MW, typename S, bool SPLIT>
__device__ __forceinline__ void fft2_fwd_block(const float* __restrict__ in, S* __restrict__ out, const Fft2Args& g,
                                               unsigned id, unsigned nb, float2* sm) {
  constexpr int LH = 2 * MH, LW = 2 * MW, LW1 = LW + 1, LH1 = LH + 1;
  float* xs = reinterpret_cast<float*>(sm);  // staging: G*Hin padded grid rows of LW1 floats
  float2* T = sm;                            // row spectra, column-major; aliases xs
  const int tid = threadIdx.x;
  const unsigned p0 = plane_group(id, nb, g.K) * (unsigned)g.G;
  const int np = (int)min((unsigned)g.G, g.P - p0);
  const int nrows = np * g.Hin;

  // each row thread zeroes the padding columns of its staging row
  if (tid < nrows) {
    float* xr = xs + tid * LW1;
    for (int j = 0; j < g.oj; ++j) xr[j] = 0.f;
    for (int j = g.oj + g.Win; j < LW; ++j) xr[j] = 0.f;
  }
  // coalesced copy of the block's rows into their grid columns: every load of
  // a thread is issued before the first is used (at most 256 rows of at most
  // LW floats, so NV4 float4 per thread), the last index repeated past the end
  const float4* src = reinterpret_cast<const float4*>(in + (size_t)p0 * g.Hin * g.Win);
  const unsigned n4 = (unsigned)nrows * g.q4;
  constexpr int NV4 = (LW + 3) / 4;
  float4 v4[NV4];
#pragma unroll
  for (int it = 0; it < NV4; ++it) v4[it] = src[min((unsigned)(tid + it * kThreads), n4 - 1)];
#pragma unroll
  for (int it = 0; it < NV4; ++it) {
    const unsigned e = (unsigned)(tid + it * kThreads);
    if (e < n4) {
      const unsigned row = g.q4 == 1 ? e : __umulhi(e, g.magic);
      const unsigned j4 = e - row * g.q4;
      float* xr = xs + row * LW1 + g.oj + 4 * j4;
      xr[0] = v4[it].x; xr[1] = v4[it].y; xr[2] = v4[it].z; xr[3] = v4[it].w;
    }
  }
  __syncthreads();

  // row pass: thread = (plane, input row)
  float2 X[MW + 1];
  int my_p = 0, my_i = 0;
  const bool has_row = tid < nrows;
  if (has_row) {
    my_p = tid / g.Hin;
    my_i = tid - my_p * g.Hin;
    const float* xr = xs + tid * LW1;
    float2 z[MW];
#pragma unroll
    for (int q = 0; q < MW; ++q) z[q] = make_float2(xr[2 * q], xr[2 * q + 1]);
    float2 Z[MW];
    dft_odd<MW, false>(z, Z);
#pragma unroll
    for (int v = 0; v <= MW; ++v) {
      const float2 zv = Z[v % MW];
      const float2 zc = cconj(Z[(MW - v) % MW]);
      const float2 E = cscale(cadd(zv, zc), 0.5f);
      const float2 d = csub(zv, zc);
      const float2 O = make_float2(0.5f * d.y, -0.5f * d.x);  // d / (2i)
      X[v] = cadd(E, cmul(root<LW, false>(v), O));
    }
  }
  __syncthreads();  // all rows read from the staging area before it is overwritten
  if (has_row) {
    float2* tr = T + my_p * g.PS + g.oi + my_i;
#pragma unroll
    for (int v = 0; v <= MW; ++v)
      if (v < g.V) tr[v * LH1] = X[v];
  }
  __syncthreads();

  if constexpr (SPLIT) {
    // column pass: two threads per (kept column, plane), planes fastest after
    // the pair: thread h of a pair takes the padded rows of parity h, the odd
    // half is twiddled, and the pair swaps halves to write rows k (h = 0) and
    // k + MH (h = 1).  A pair's lanes are active together (the count is even).
    const unsigned rs = (unsigned)g.V * g.P;
    for (int e = tid; e < 2 * np * g.V; e += kThreads) {
      const int h = e & 1, c = e >> 1;
      const int p = c % np, v = c / np;
      const float2* tc = T + p * g.PS + v * LH1;
      float2 z[MH];
#pragma unroll
      for (int q = 0; q < MH; ++q) {
        const int i = 2 * q + h;
        z[q] = (i >= g.oi && i < g.oi + g.Hin) ? tc[i] : make_float2(0.f, 0.f);
      }
      float2 D[MH];
      dft_odd<MH, false>(z, D);
      S* dst = out + (p0 + p) + (unsigned)v * g.P;
#pragma unroll
      for (int k = 0; k < MH; ++k) {
        const float2 mine = h ? cmul(root<LH, false>(k), D[k]) : D[k];
        const float2 other = swap_pair(mine);
        const int r = row_slot(k + h * MH, g.r_h, g.R, LH);
        if (r >= 0) spec_put(dst, (unsigned)r * rs, h ? csub(other, mine) : cadd(mine, other));
      }
    }
  } else {
    // column pass: thread = (kept column, plane), planes fastest
    for (int e = tid; e < np * g.V; e += kThreads) {
      const int p = e % np, v = e / np;
      float2* tc = T + p * g.PS + v * LH1;
      for (int i = 0; i < g.oi; ++i) tc[i] = make_float2(0.f, 0.f);
      for (int i = g.oi + g.Hin; i < LH; ++i) tc[i] = make_float2(0.f, 0.f);
      float2 ev[MH], od[MH];
#pragma unroll
      for (int q = 0; q < MH; ++q) {
        ev[q] = tc[2 * q];
        od[q] = tc[2 * q + 1];
      }
      float2 E[MH], O[MH];
      dft_odd<MH, false>(ev, E);
      dft_odd<MH, false>(od, O);
      S* dst = out + (p0 + p) + (unsigned)v * g.P;
      const unsigned rs = (unsigned)g.V * g.P;
#pragma unroll
      for (int k = 0; k < MH; ++k) {
        const float2 t = cmul(root<LH, false>(k), O[k]);
        const int r_lo = row_slot(k, g.r_h, g.R, LH);
        const int r_hi = row_slot(k + MH, g.r_h, g.R, LH);
        if (r_lo >= 0) spec_put(dst, (unsigned)r_lo * rs, cadd(E[k], t));
        if (r_hi >= 0) spec_put(dst, (unsigned)r_hi * rs, csub(E[k], t));
      }
    }
  }
}

template <int MH, int MW, typename S, bool SPLIT>
__global__ __launch_bounds__(kThreads) void k_fft2_fwd(const float* __restrict__ in, S* __restrict__ out,
                                                       Fft2Args g) {
  extern __shared__ float2 sm[];
  fft2_fwd_block<MH, MW, S, SPLIT>(in, out, g, blockIdx.x, gridDim.x, sm);
}

// The input transform and the filter transform of a forward pass in one
// launch (they are independent): blocks [0, nx) transform planes of x, the
// rest compute filter-spectrum chunks.  The filter transform is a short,
// latency-bound kernel; beside the input transform its blocks fill the CUs
// that the transform's last blocks leave idle, and one launch is saved.
template <int MH, int MW, typename S, bool SPLIT, int KH, int KW>
__global__ __launch_bounds__(kThreads) void k_fft2_fwd_filt(const float* __restrict__ in, S* __restrict__ out,
                                                            Fft2Args g, const float* __restrict__ w,
                                                            const float2* __restrict__ roots, S* __restrict__ wout,
                                                            FiltGeom fg, unsigned nx) {
  extern __shared__ float2 sm[];
  if (blockIdx.x < nx)
    fft2_fwd_block<MH, MW, S, SPLIT>(in, out, g, blockIdx.x, nx, sm);
  else
    spec_filt_block<KH, KW, S>(w, roots, wout, fg, blockIdx.x - nx, gridDim.x - nx, sm);
}

// One block (id of nb) of the inverse transform; sm: the launch's LDS.
template <int MH, int MW, bool SPLIT, bool PARTS>
__device__ __forceinline__ void fft2_inv_block(const float2* __restrict__ in, float* __restrict__ out,
                                               const Fft2Args& g, unsigned id, unsigned nb, float2* sm) {
  constexpr int LH = 2 * MH, LW = 2 * MW, LW1 = LW + 1, LH1 = LH + 1;
  float2* Zs = sm;                           // column results, column-major per plane
  float* ys = reinterpret_cast<float*>(sm);  // output staging: G*OH grid rows of LW1 floats; aliases Zs
  const int tid = threadIdx.x;
  const int OH = g.Hin, OW = g.Win;
  const unsigned p0 = plane_group(id, nb, g.K & ~kInvVec4) * (unsigned)g.G;
  const int np = (int)min((unsigned)g.G, g.P - p0);

  if constexpr (SPLIT) {
    // column pass: two threads per (kept column, plane), planes fastest after
    // the pair: thread h of a pair loads the kept rows k + h MH, the pair swaps
    // them, and thread h forms the even (h = 0) or twiddled odd (h = 1) half and
    // inverts it into the padded rows of parity h.  A pair's lanes are active
    // together (the count is even).
    for (int e = tid; e < 2 * np * g.V; e += kThreads) {
      const int h = e & 1, c = e >> 1;
      const int p = c % np, v = c / np;
      const float2* src = in + (p0 + p) + (unsigned)v * g.P;
      const unsigned rs = (unsigned)g.V * g.P;
      float2 mine[MH];
#pragma unroll
      for (int k = 0; k < MH; ++k) {
        const int r = row_slot(k + h * MH, g.r_h, g.R, LH);
        mine[k] = r >= 0 ? load_parts<PARTS>(src + (unsigned)r * rs, g) : make_float2(0.f, 0.f);
      }
      float2 z[MH];
#pragma unroll
      for (int k = 0; k < MH; ++k) {
        const float2 other = swap_pair(mine[k]);
        const float2 lo = h ? other : mine[k], hi = h ? mine[k] : other;
        z[k] = h ? cmul(root<LH, true>(k), csub(lo, hi)) : cadd(lo, hi);
      }
      float2 x[MH];
      dft_odd<MH, true>(z, x);
      float2* zc = Zs + p * g.PS + v * LH1;
#pragma unroll
      for (int q = 0; q < MH; ++q) zc[2 * q + h] = x[q];
    }
  } else {
    // column pass: thread = (kept column, plane), planes fastest
    for (int e = tid; e < np * g.V; e += kThreads) {
      const int p = e % np, v = e / np;
      const float2* src = in + (p0 + p) + (unsigned)v * g.P;
      const unsigned rs = (unsigned)g.V * g.P;
      float2 a[MH], b[MH];
#pragma unroll
      for (int k = 0; k < MH; ++k) {
        const int r0 = row_slot(k, g.r_h, g.R, LH);
        const int r1 = row_slot(k + MH, g.r_h, g.R, LH);
        const float2 lo = r0 >= 0 ? load_parts<PARTS>(src + r0 * rs, g) : make_float2(0.f, 0.f);
        const float2 hi = r1 >= 0 ? load_parts<PARTS>(src + r1 * rs, g) : make_float2(0.f, 0.f);
        a[k] = cadd(lo, hi);
        b[k] = cmul(root<LH, true>(k), csub(lo, hi));
      }
      float2 xe[MH], xo[MH];
      dft_odd<MH, true>(a, xe);
      dft_odd<MH, true>(b, xo);
      float2* zc = Zs + p * g.PS + v * LH1;
#pragma unroll
      for (int q = 0; q < MH; ++q) {
        zc[2 * q] = xe[q];
        zc[2 * q + 1] = xo[q];
      }
    }
  }
  __syncthreads();

  // row pass: thread = (plane, output row)
  const int nrows = np * OH;
  const bool has_row = tid < nrows;
  float yv[LW];
  if (has_row) {
    const int p = tid / OH, i = tid - (tid / OH) * OH;
    const float2* zr = Zs + p * g.PS + g.oi + i;
    float2 Zh[MW + 1];
#pragma unroll
    for (int v = 0; v <= MW; ++v) Zh[v] = v < g.V ? zr[v * LH1] : make_float2(0.f, 0.f);
    Zh[0].y = 0.f;   // c2r: imaginary parts of the DC and Nyquist columns are dropped
    Zh[MW].y = 0.f;
    float2 Q[MW];
#pragma unroll
    for (int k = 0; k < MW; ++k) {
      const float2 zk = Zh[k], zc = cconj(Zh[MW - k]);
      const float2 A = cadd(zk, zc);
      const float2 B = cmul(root<LW, true>(k), csub(zk, zc));
      Q[k] = make_float2(A.x - B.y, A.y + B.x);  // A + iB
    }
    float2 q[MW];
    dft_odd<MW, true>(Q, q);
#pragma unroll
    for (int n = 0; n < MW; ++n) {
      yv[2 * n] = q[n].x * g.scale;
      yv[2 * n + 1] = q[n].y * g.scale;
    }
  }
  __syncthreads();  // every row read from Zs before the staging overwrites it
  if (has_row) {
    float* yr = ys + tid * LW1;
#pragma unroll
    for (int j = 0; j < LW; ++j) yr[j] = yv[j];
  }
  __syncthreads();
  // coalesced copy of the cropped window (planes contiguous in HBM): 16-byte
  // stores when the window's rows are whole float4s (q4 = OW / 4), else floats
  // (q4 = OW)
  float* dst = out + (size_t)p0 * OH * OW;
  if (g.K & kInvVec4) {
    float4* dst4 = reinterpret_cast<float4*>(dst);
    const unsigned n4 = (unsigned)nrows * g.q4;
    for (unsigned e = tid; e < n4; e += blockDim.x) {
      const unsigned row = g.q4 == 1 ? e : __umulhi(e, g.magic);
      const float* yr = ys + row * LW1 + g.oj + 4 * (e - row * g.q4);
      dst4[e] = make_float4(yr[0], yr[1], yr[2], yr[3]);
    }
  } else {
    const unsigned n = (unsigned)nrows * OW;
    for (unsigned e = tid; e < n; e += blockDim.x) {
      const unsigned row = g.q4 == 1 ? e : __umulhi(e, g.magic);
      const unsigned j = e - row * g.q4;
      dst[e] = ys[row * LW1 + g.oj + j];
    }
  }
}

template <int MH, int MW, bool SPLIT, bool PARTS>
__global__ __launch_bounds__(kThreads) void k_fft2_inv(const float2* __restrict__ in, float* __restrict__ out,
                                                       Fft2Args g) {
  extern __shared__ float2 sm[];
  fft2_inv_block<MH, MW, SPLIT, PARTS>(in, out, g, blockIdx.x, gridDim.x, sm);
}

// The input-gradient inverse and the sliced weight-gradient inverse DFT of a
// backward pass in one launch (they are independent): blocks [0, nx) invert
// planes of DX, the rest are weight-gradient blocks (channel block j % wx,
// slice j / wx).  The weight-gradient launch is short and latency-bound;
// beside the transform its blocks fill the CUs that the transform's last
// blocks leave idle, and one launch is saved.
template <int MH, int MW, bool SPLIT, bool PARTS, int TMAX, int TC>
__global__ __launch_bounds__(kThreads) void k_fft2_inv_wgrad(const float2* __restrict__ in, float* __restrict__ out,
                                                             Fft2Args g, unsigned nx, const float2* __restrict__ DW,
                                                             const float2* __restrict__ Et, float* __restrict__ dw,
                                                             float* __restrict__ part, WgradGeom wg, unsigned wx,
                                                             unsigned wslices) {
  extern __shared__ float2 sm[];
  __shared__ float res[wgrad_res_floats<TMAX, TC>()];
  if (blockIdx.x < nx) {
    fft2_inv_block<MH, MW, SPLIT, PARTS>(in, out, g, blockIdx.x, nx, sm);
  } else {
    const unsigned j = blockIdx.x - nx;
    wgrad_idft_block<TMAX, TC>(DW, Et, dw, part, wg, j % wx, j / wx, wslices > 1, sm, res);
  }
}

// The same with the one-pass wide weight-gradient body (64 pairs and all bins
// per block, four waves each over a quarter of the bins); WPARTS: DW arrives
// as partial spectra, summed as they are loaded.
template <int MH, int MW, bool SPLIT, bool PARTS, int TMAX, bool WPARTS>
__global__ __launch_bounds__(kThreads) void k_fft2_inv_wgrad_wide(const float2* __restrict__ in,
                                                                  float* __restrict__ out, Fft2Args g, unsigned nx,
                                                                  const float2* __restrict__ DW,
                                                                  const float2* __restrict__ Et,
                                                                  float* __restrict__ dw, WgradGeom wg) {
  extern __shared__ float2 sm[];
  __shared__ float red[4 * 64 * TMAX];
  if (blockIdx.x < nx)
    fft2_inv_block<MH, MW, SPLIT, PARTS>(in, out, g, blockIdx.x, nx, sm);
  else
    wgrad_wide_block<TMAX, 4, WPARTS>(DW, Et, dw, wg, blockIdx.x - nx, sm, red);
}

// ceil(2^32 / d) for d > 1 (d = 1 is handled by the kernels directly).
unsigned magic_for(unsigned d) { return d > 1 ? (unsigned)((0x100000000ull + d - 1) / d) : 0u; }

// Column pass on lane pairs (one MH-point DFT per thread).  Always for the
// longest columns (MH >= 17), where two DFTs per thread hold too many registers
// for four waves per SIMD; for the forward on 18-point columns when the pairs
// of a block's G planes x V kept columns fit one pass of its threads.  On
// shorter columns, and for the inverse below 34 points, one thread per column
// measured faster.
bool column_split(bool fwd, int MH, int G, int V) {
  return MH >= 17 || (fwd && MH >= 9 && 2L * G * V <= kThreads);
}

// Plane groups whose runs of G elements of `elem` bytes fill a 128-byte line.
unsigned line_groups(int G, int elem) { return (unsigned)std::max(1, (128 + G * elem - 1) / (G * elem)); }

// Launch geometry of the forward transform.
struct FwdSetup {
  Fft2Args g;
  long blocks;
  size_t lds;
  double bytes, flops;
  bool split;
};

template <int MH, int MW>
bl_status_t fwd_setup(const bl_conv_plan_s* p, long P, int Hin, int Win, int oi, int oj, FwdSetup& f) {
  constexpr int LH = 2 * MH, LW = 2 * MW;
  if (Win % 4 != 0 || oj + Win > LW || oi + Hin > LH || (double)p->kept * P >= 2147483647.0 || P >= 2147483647L)
    return BL_ERR_UNSUPPORTED;
  Fft2Args g{Hin, Win, oi, oj, p->r_h, p->R, p->V, (unsigned)P, 0, 0, (unsigned)(Win / 4), 0, 1u, 1.0f};
  g.magic = magic_for(g.q4);
  g.PS = (p->V * (LH + 1)) | 1;
  // rows of a block must fit one pass of 256 threads; LDS for staging and spectra
  int G = std::max(1, kThreads / Hin);
  G = (int)std::min<long>(G, P);
  auto lds_for = [&](int gg) {
    const size_t stage = (size_t)gg * Hin * (LW + 1) * sizeof(float);
    const size_t spec = (size_t)gg * g.PS * sizeof(float2);
    return std::max(stage, spec);
  };
  while (G > 1 && lds_for(G) > kMaxLds) --G;
  if (Hin > kThreads || lds_for(G) > kMaxLds) return BL_ERR_UNSUPPORTED;
  g.G = G;
  // the forward writes its runs; sharing lines paid off for runs of 32 bytes
  // (1.2x) and cost time for runs of 64 bytes, so it is kept to the shorter runs
  const int run = G * (p->bf16 ? 4 : 8);
  g.K = run < 64 ? line_groups(G, p->bf16 ? 4 : 8) : 1u;
  f.g = g;
  f.blocks = (P + G - 1) / G;
  f.lds = lds_for(G);
  f.bytes = (double)P * Hin * Win * 4 + (double)P * p->kept * (p->bf16 ? 4 : 8);
  // conventional FFT counts: Hin real LW-point row FFTs (2.5 LW log2 LW) and V
  // complex LH-point column FFTs (5 LH log2 LH) per plane
  f.flops = (double)P * (Hin * 2.5 * LW * std::log2((double)LW) + p->V * 5.0 * LH * std::log2((double)LH));
  f.split = column_split(true, MH, G, p->V);
  return BL_OK;
}

template <int MH, int MW>
bl_status_t launch_fwd_t(const bl_conv_plan_s* p, const float* in, void* out, long P, int Hin, int Win, int oi,
                         int oj, hipStream_t s) {
  FwdSetup f;
  const bl_status_t fs = fwd_setup<MH, MW>(p, P, Hin, Win, oi, oj, f);
  if (fs != BL_OK) return fs;
  const Fft2Args g = f.g;
  const size_t lds = f.lds;
  return timed_launch("spec_fwd_2d", f.bytes, f.flops, s, [&](hipEvent_t e0, hipEvent_t e1) {
    const dim3 grid((unsigned)f.blocks), block(kThreads);
    if (p->bf16) {
      unsigned* o = static_cast<unsigned*>(out);
      if (f.split)
        hipExtLaunchKernelGGL((k_fft2_fwd<MH, MW, unsigned, true>), grid, block, lds, s, e0, e1, 0, in, o, g);
      else
        hipExtLaunchKernelGGL((k_fft2_fwd<MH, MW, unsigned, false>), grid, block, lds, s, e0, e1, 0, in, o, g);
    } else {
      float2* o = static_cast<float2*>(out);
      if (f.split)
        hipExtLaunchKernelGGL((k_fft2_fwd<MH, MW, float2, true>), grid, block, lds, s, e0, e1, 0, in, o, g);
      else
        hipExtLaunchKernelGGL((k_fft2_fwd<MH, MW, float2, false>), grid, block, lds, s, e0, e1, 0, in, o, g);
    }
  });
}

// Launch geometry of the inverse transform.
struct InvSetup {
  Fft2Args g;
  long blocks;
  size_t lds;
  double bytes, flops;
  bool split;
};

template <int MH, int MW>
bl_status_t inv_setup(const bl_conv_plan_s* p, long P, int OH, int OW, int ci, int cj, int nsplit, size_t pstride,
                      InvSetup& f) {
  constexpr int LH = 2 * MH, LW = 2 * MW;
  if ((double)p->kept * P >= 2147483647.0 || P >= 2147483647L) return BL_ERR_UNSUPPORTED;
  const bool vec4 = OW % 4 == 0;
  Fft2Args g{OH, OW, ci, cj, p->r_h, p->R, p->V, (unsigned)P, 0, 0, (unsigned)(vec4 ? OW / 4 : OW), 0, 1u,
             1.0f / ((float)p->Lh * (float)p->Lw)};
  g.magic = magic_for(g.q4);
  g.PS = (p->V * (LH + 1)) | 1;
  g.nsplit = (unsigned)std::max(1, nsplit);
  g.pstride = pstride;
  int G = std::max(1, kThreads / OH);
  G = (int)std::min<long>(G, P);
  auto lds_for = [&](int gg) {
    const size_t spec = (size_t)gg * g.PS * sizeof(float2);
    const size_t stage = (size_t)gg * OH * (LW + 1) * sizeof(float);
    return std::max(stage, spec);
  };
  while (G > 1 && lds_for(G) > kMaxLds) --G;
  if (OH > kThreads || lds_for(G) > kMaxLds) return BL_ERR_UNSUPPORTED;
  g.G = G;
  g.K = line_groups(G, 8) | (vec4 ? kInvVec4 : 0u);
  f.g = g;
  f.blocks = (P + G - 1) / G;
  f.lds = lds_for(G);
  f.bytes = (double)P * p->kept * 8 * g.nsplit + (double)P * OH * OW * 4;
  f.flops = (double)P * (p->V * 5.0 * LH * std::log2((double)LH) + OH * 2.5 * LW * std::log2((double)LW));
  f.split = column_split(false, MH, G, p->V);
  return BL_OK;
}

template <int MH, int MW>
bl_status_t launch_inv_t(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OH, int OW, int ci,
                         int cj, hipStream_t s, int nsplit, size_t pstride) {
  InvSetup f;
  const bl_status_t is = inv_setup<MH, MW>(p, P, OH, OW, ci, cj, nsplit, pstride, f);
  if (is != BL_OK) return is;
  const Fft2Args g = f.g;
  const size_t lds = f.lds;
  return timed_launch("spec_inv_2d", f.bytes, f.flops, s, [&](hipEvent_t e0, hipEvent_t e1) {
    const dim3 grid((unsigned)f.blocks), block(kThreads);
    if (g.nsplit > 1) {
      if (f.split)
        hipExtLaunchKernelGGL((k_fft2_inv<MH, MW, true, true>), grid, block, lds, s, e0, e1, 0, in, out, g);
      else
        hipExtLaunchKernelGGL((k_fft2_inv<MH, MW, false, true>), grid, block, lds, s, e0, e1, 0, in, out, g);
    } else if (f.split) {
      hipExtLaunchKernelGGL((k_fft2_inv<MH, MW, true, false>), grid, block, lds, s, e0, e1, 0, in, out, g);
    } else {
      hipExtLaunchKernelGGL((k_fft2_inv<MH, MW, false, false>), grid, block, lds, s, e0, e1, 0, in, out, g);
    }
  });
}

// The input-gradient inverse beside the sliced weight-gradient inverse DFT
// (3 x 3 filters), then the weight gradient's slice sum if it has slices.
template <int MH, int MW>
bl_status_t launch_inv_wgrad_t(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OH, int OW, int ci,
                               int cj, int nsplit, size_t pstride, const float2* DW, float* dw, float* part,
                               int wnsplit, hipStream_t s) {
  if (p->Kh != 3 || p->Kw != 3) return BL_ERR_UNSUPPORTED;
  InvSetup f;
  bl_status_t st = inv_setup<MH, MW>(p, P, OH, OW, ci, cj, nsplit, pstride, f);
  if (st != BL_OK) return st;
  WgradGeom wg;
  long wx;
  int slices, tc;
  size_t wlds;
  const float2* Et;
  if (!wgrad_sliced_setup(p, wnsplit, wg, &wx, &slices, &wlds, &tc, &Et)) {
    // the wide one-pass body (partial spectra summed as they are loaded)
    if (!wgrad_wide(p) || wgrad_table(p, &Et) != BL_OK) return BL_ERR_UNSUPPORTED;
    const long Q = (long)p->Cin * p->Cout;
    wg = WgradGeom{p->Cout, p->Cin, p->Kh, p->Kw, 9, p->Lh, p->Lw, p->r_h, p->R, p->V, 0, 0, 0,
                   std::max(1, wnsplit), (unsigned long long)p->kept * Q};
    const long wblocks = (Q + 63) / 64;
    const long total = f.blocks + wblocks;
    if (total >= 2147483647L) return BL_ERR_UNSUPPORTED;
    const size_t lds = std::max(f.lds, (size_t)p->kept * 9 * sizeof(float2));
    const Fft2Args g = f.g;
    const unsigned nx = (unsigned)f.blocks;
    const double wbytes = (double)Q * ((double)p->kept * 8 * wg.nsplit + 9 * 4);
    auto go = [&](auto kern) {
      // the dynamic part (at most 64 KB) plus the static reduction buffer can pass 64 KB
      const bl_status_t at = lds_opt_in(reinterpret_cast<const void*>(kern), 96 * 1024);
      if (at != BL_OK) return at;
      return timed_launch("spec_inv_wgrad_2d", f.bytes + wbytes, f.flops, s, [&](hipEvent_t e0, hipEvent_t e1) {
        hipExtLaunchKernelGGL(kern, dim3((unsigned)total), dim3(kThreads), lds, s, e0, e1, 0, in, out, g, nx, DW, Et,
                              dw, wg);
      });
    };
    if (g.nsplit > 1 && wg.nsplit > 1) return BL_ERR_UNSUPPORTED;  // the plan splits one pass at most
    if (g.nsplit > 1)
      return f.split ? go(k_fft2_inv_wgrad_wide<MH, MW, true, true, 9, false>)
                     : go(k_fft2_inv_wgrad_wide<MH, MW, false, true, 9, false>);
    if (wg.nsplit > 1)
      return f.split ? go(k_fft2_inv_wgrad_wide<MH, MW, true, false, 9, true>)
                     : go(k_fft2_inv_wgrad_wide<MH, MW, false, false, 9, true>);
    return f.split ? go(k_fft2_inv_wgrad_wide<MH, MW, true, false, 9, false>)
                   : go(k_fft2_inv_wgrad_wide<MH, MW, false, false, 9, false>);
  }
  const long total = f.blocks + wx * slices;
  if (total >= 2147483647L) return BL_ERR_UNSUPPORTED;
  const Fft2Args g = f.g;
  const size_t lds = std::max(f.lds, wlds);
  const unsigned nx = (unsigned)f.blocks, wxu = (unsigned)wx, ws = (unsigned)slices;
  const double wbytes = (double)p->Cin * p->Cout * ((double)p->kept * 8 * wg.nsplit + wg.T * 4);
  auto go = [&](auto kern) {
    return timed_launch("spec_inv_wgrad_2d", f.bytes + wbytes, f.flops, s, [&](hipEvent_t e0, hipEvent_t e1) {
      hipExtLaunchKernelGGL(kern, dim3((unsigned)total), dim3(kThreads), lds, s, e0, e1, 0, in, out, g, nx, DW, Et, dw,
                            part, wg, wxu, ws);
    });
  };
  if (g.nsplit > 1)
    st = f.split ? (tc == 8 ? go(k_fft2_inv_wgrad<MH, MW, true, true, 9, 8>) : go(k_fft2_inv_wgrad<MH, MW, true, true, 9, 1>))
                 : (tc == 8 ? go(k_fft2_inv_wgrad<MH, MW, false, true, 9, 8>)
                            : go(k_fft2_inv_wgrad<MH, MW, false, true, 9, 1>));
  else
    st = f.split ? (tc == 8 ? go(k_fft2_inv_wgrad<MH, MW, true, false, 9, 8>)
                            : go(k_fft2_inv_wgrad<MH, MW, true, false, 9, 1>))
                 : (tc == 8 ? go(k_fft2_inv_wgrad<MH, MW, false, false, 9, 8>)
                            : go(k_fft2_inv_wgrad<MH, MW, false, false, 9, 1>));
  if (st != BL_OK || slices == 1) return st;
  return launch_wgrad_reduce(p, part, dw, wg, s);
}

// The forward transform of x beside the filter transform (3 x 3 filters).
template <int MH, int MW>
bl_status_t launch_fwd_filt_t(const bl_conv_plan_s* p, const float* in, void* out, long P, int Hin, int Win, int oi,
                              int oj, const float* w, void* wout, hipStream_t s) {
  if (p->Kh != 3 || p->Kw != 3) return BL_ERR_UNSUPPORTED;
  FwdSetup f;
  bl_status_t st = fwd_setup<MH, MW>(p, P, Hin, Win, oi, oj, f);
  if (st != BL_OK) return st;
  FiltGeom fg;
  const float2* roots;
  long fblocks;
  size_t flds;
  double fbytes;
  st = filt_setup(p, true, fg, &roots, &fblocks, &flds, &fbytes);
  if (st != BL_OK) return st;
  if (f.blocks + fblocks >= 2147483647L) return BL_ERR_UNSUPPORTED;
  const dim3 grid((unsigned)(f.blocks + fblocks)), block(kThreads);
  const size_t lds = std::max(f.lds, flds);
  const unsigned nx = (unsigned)f.blocks;
  const Fft2Args g = f.g;
  return timed_launch("spec_fwd_filt_2d", f.bytes + fbytes, f.flops, s, [&](hipEvent_t e0, hipEvent_t e1) {
    if (p->bf16) {
      unsigned* o = static_cast<unsigned*>(out);
      unsigned* wo = static_cast<unsigned*>(wout);
      if (f.split)
        hipExtLaunchKernelGGL((k_fft2_fwd_filt<MH, MW, unsigned, true, 3, 3>), grid, block, lds, s, e0, e1, 0, in, o, g,
                              w, roots, wo, fg, nx);
      else
        hipExtLaunchKernelGGL((k_fft2_fwd_filt<MH, MW, unsigned, false, 3, 3>), grid, block, lds, s, e0, e1, 0, in, o,
                              g, w, roots, wo, fg, nx);
    } else {
      float2* o = static_cast<float2*>(out);
      float2* wo = static_cast<float2*>(wout);
      if (f.split)
        hipExtLaunchKernelGGL((k_fft2_fwd_filt<MH, MW, float2, true, 3, 3>), grid, block, lds, s, e0, e1, 0, in, o, g,
                              w, roots, wo, fg, nx);
      else
        hipExtLaunchKernelGGL((k_fft2_fwd_filt<MH, MW, float2, false, 3, 3>), grid, block, lds, s, e0, e1, 0, in, o,
                              g, w, roots, wo, fg, nx);
    }
  });
}

#define BL_FFT2_GRIDS(X) X(3, 3) X(5, 5) X(9, 9) X(17, 17) X(29, 29)

}  // namespace

bl_status_t launch_fft2_fwd(const bl_conv_plan_s* p, const float* in, void* out, long P, int Hin, int Win, int oi,
                            int oj, hipStream_t s) {
#define X(a, b) \
  if (p->Lh == 2 * a && p->Lw == 2 * b) return launch_fwd_t<a, b>(p, in, out, P, Hin, Win, oi, oj, s);
  BL_FFT2_GRIDS(X)
#undef X
  return BL_ERR_UNSUPPORTED;
}

bl_status_t launch_fft2_fwd_filt(const bl_conv_plan_s* p, const float* in, void* out, long P, int Hin, int Win,
                                 int oi, int oj, const float* w, void* wout, hipStream_t s) {
#define X(a, b)                         \
  if (p->Lh == 2 * a && p->Lw == 2 * b) \
    return launch_fwd_filt_t<a, b>(p, in, out, P, Hin, Win, oi, oj, w, wout, s);
  BL_FFT2_GRIDS(X)
#undef X
  return BL_ERR_UNSUPPORTED;
}

bl_status_t launch_fft2_inv_wgrad(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OH, int OW,
                                  int ci, int cj, int nsplit, size_t pstride, const float2* DW, float* dw, float* part,
                                  int wnsplit, hipStream_t s) {
#define X(a, b)                                                                                                   \
  if (p->Lh == 2 * a && p->Lw == 2 * b)                                                                           \
    return launch_inv_wgrad_t<a, b>(p, in, out, P, OH, OW, ci, cj, nsplit, pstride, DW, dw, part, wnsplit, s);
  BL_FFT2_GRIDS(X)
#undef X
  return BL_ERR_UNSUPPORTED;
}

bl_status_t launch_fft2_inv(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OH, int OW, int ci,
                            int cj, hipStream_t s, int nsplit, size_t pstride) {
#define X(a, b) \
  if (p->Lh == 2 * a && p->Lw == 2 * b) return launch_inv_t<a, b>(p, in, out, P, OH, OW, ci, cj, s, nsplit, pstride);
  BL_FFT2_GRIDS(X)
#undef X
  return BL_ERR_UNSUPPORTED;
}

}  // namespace blc
