// Direct (pruned DFT) transforms, filter spectrum, weight-gradient inverse
// DFT and the per-bin channel contraction on fp32 MFMA (gfx950).
//
//   spec_fwd_direct  zero-pad + real 2-D DFT + band mask of real planes (x or
//                    dy): a row pass that emits only kept columns v <= r_w, then
//                    a column pass over the nonzero input rows that emits only
//                    kept rows.  Discarded coefficients are never formed
//                    (Sec. 3.2.2, Fig. 2).  Any grid size.
//   spec_inv_direct  zero-fill + inverse real 2-D DFT + crop: only kept bins are
//                    read and only the cropped window is written.  Any grid.
//   spec_filt        filter spectrum at the kept bins, a K x K-tap DFT per bin.
//   wgrad_idft       inverse DFT of the kept weight-gradient bins onto the
//                    K x K taps (the projected weight gradient, Sec. 1).
//   contract         per kept bin, a complex matrix product over channels (the
//                    Hadamard product fused with the channel sum, Sec. 3.3).
#include <algorithm>
#include <cmath>

#include "common.hpp"
#include "filt.hpp"
#include "wgrad.hpp"

namespace blc {
namespace {


// ---------------------------------------------------------------------------
// spec_fwd: real planes [P][Hin][Win] placed at (oi, oj) of the Lh x Lw grid ->
// kept spectrum out[b * P + p].  TP planes per block.
// ---------------------------------------------------------------------------
struct FwdGeom {
  int Hin, Win, oi, oj;
  int Lh, Lw, r_h, R, V;
  long P;
  int TP;
};

// S: stored-spectrum element of the output (float2 or bfloat16 pairs)
template <typename S>
__global__ __launch_bounds__(kThreads) void k_spec_fwd(const float* __restrict__ in, S* __restrict__ out,
                                                       FwdGeom g) {
  extern __shared__ float2 smem[];
  float2* twh = smem;                       // Lh
  float2* tww = twh + g.Lh;                 // Lw
  const int Ts = g.Hin * g.V + 1;           // padded plane stride of the row-pass result
  float2* T = tww + g.Lw;                   // TP * Ts
  float* xs = reinterpret_cast<float*>(T + (size_t)g.TP * Ts);  // TP * Hin * Win

  const long p0 = (long)blockIdx.x * g.TP;
  const int np = (int)min((long)g.TP, g.P - p0);
  const int plane = g.Hin * g.Win;

  fill_roots(twh, g.Lh, -1.0);
  fill_roots(tww, g.Lw, -1.0);
  const float* src = in + p0 * plane;
  for (int e = threadIdx.x; e < np * plane; e += blockDim.x) xs[e] = src[e];
  __syncthreads();

  // Row pass: T[p][i][v] = sum_j x[p][i][j] e^{-2 pi i v (j + oj) / Lw}, v < V.
  for (int e = threadIdx.x; e < np * g.Hin * g.V; e += blockDim.x) {
    const int v = e % g.V;
    const int pi = e / g.V;  // p * Hin + i
    const int p = pi / g.Hin, i = pi % g.Hin;
    const float* xr = xs + (size_t)pi * g.Win;
    int idx = (int)(((long)v * g.oj) % g.Lw);
    float re = 0.f, im = 0.f;
    for (int j = 0; j < g.Win; ++j) {
      const float2 w = tww[idx];
      re = fmaf(xr[j], w.x, re);
      im = fmaf(xr[j], w.y, im);
      idx += v;
      if (idx >= g.Lw) idx -= g.Lw;
    }
    T[(size_t)p * Ts + i * g.V + v] = make_float2(re, im);
  }
  __syncthreads();

  // Column pass over kept rows u; store bin-major, planes fastest.
  const int B = g.R * g.V;
  for (int e = threadIdx.x; e < np * B; e += blockDim.x) {
    const int p = e % np;
    const int b = e / np;
    const int r = b / g.V, v = b % g.V;
    const int u = kept_row_d(r, g.r_h, g.Lh, g.R);
    int idx = (int)(((long)u * g.oi) % g.Lh);
    float re = 0.f, im = 0.f;
    const float2* tc = T + (size_t)p * Ts + v;
    for (int i = 0; i < g.Hin; ++i) {
      const float2 a = tc[i * g.V];
      const float2 w = twh[idx];
      re = fmaf(a.x, w.x, fmaf(-a.y, w.y, re));
      im = fmaf(a.x, w.y, fmaf(a.y, w.x, im));
      idx += u;
      if (idx >= g.Lh) idx -= g.Lh;
    }
    spec_put(out, (size_t)b * g.P + p0 + p, make_float2(re, im));
  }
}

// ---------------------------------------------------------------------------
// spec_inv: kept spectrum in[b * P + p] -> real planes [P][OH][OW] holding the
// grid window starting at (ci, cj), scaled by 1 / (Lh Lw).  Hermitian (c2r)
// convention: column v contributes with weight 2 except v = 0 and the Nyquist
// column of an even Lw, and only the real part of each term is kept.
// ---------------------------------------------------------------------------
struct InvGeom {
  int OH, OW, ci, cj;
  int Lh, Lw, r_h, R, V;
  long P;
  int TP;
  float scale;
};

__global__ __launch_bounds__(kThreads) void k_spec_inv(const float2* __restrict__ in, float* __restrict__ out,
                                                       InvGeom g) {
  extern __shared__ float2 smem[];
  float2* twh = smem;        // Lh, e^{+2 pi i k / Lh}
  float2* tww = twh + g.Lh;  // Lw
  const int B = g.R * g.V;
  const int Ss = B + 1;
  const int Zs = g.OH * g.V + 1;
  float2* S = tww + g.Lw;                 // TP * Ss
  float2* Z = S + (size_t)g.TP * Ss;      // TP * Zs

  const long p0 = (long)blockIdx.x * g.TP;
  const int np = (int)min((long)g.TP, g.P - p0);

  fill_roots(twh, g.Lh, 1.0);
  fill_roots(tww, g.Lw, 1.0);
  for (int e = threadIdx.x; e < np * B; e += blockDim.x) {
    const int p = e % np, b = e / np;
    S[(size_t)p * Ss + b] = in[(size_t)b * g.P + p0 + p];
  }
  __syncthreads();

  // Column pass: Z[p][i][v] = sum_r S[p][r][v] e^{+2 pi i u_r (ci + i) / Lh}.
  for (int e = threadIdx.x; e < np * g.OH * g.V; e += blockDim.x) {
    const int v = e % g.V;
    const int t2 = e / g.V;
    const int i = t2 % g.OH, p = t2 / g.OH;
    const int m = (g.ci + i) % g.Lh;
    float re = 0.f, im = 0.f;
    const float2* sc = S + (size_t)p * Ss + v;
    int idx = 0;  // (u * m) mod Lh, u = 0 first
    for (int r = 0; r < g.R; ++r) {
      if (r == g.r_h + 1) idx = (int)(((long)(r + g.Lh - g.R) * m) % g.Lh);
      const float2 a = sc[r * g.V];
      const float2 w = twh[idx];
      re = fmaf(a.x, w.x, fmaf(-a.y, w.y, re));
      im = fmaf(a.x, w.y, fmaf(a.y, w.x, im));
      idx += m;
      if (idx >= g.Lh) idx -= g.Lh;
    }
    Z[(size_t)p * Zs + i * g.V + v] = make_float2(re, im);
  }
  __syncthreads();

  // Row pass: y[p][i][j] = scale * sum_v h_v Re(Z[p][i][v] e^{+2 pi i v (cj + j) / Lw}).
  const int nyq = (g.Lw % 2 == 0) ? g.Lw / 2 : -1;
  float* dst = out + p0 * (long)g.OH * g.OW;
  for (int e = threadIdx.x; e < np * g.OH * g.OW; e += blockDim.x) {
    const int j = e % g.OW;
    const int t2 = e / g.OW;
    const int i = t2 % g.OH, p = t2 / g.OH;
    const int m = (g.cj + j) % g.Lw;
    const float2* zr = Z + (size_t)p * Zs + i * g.V;
    float acc = 0.f;
    int idx = 0;
    for (int v = 0; v < g.V; ++v) {
      const float2 a = zr[v];
      const float2 w = tww[idx];
      const float h = (v == 0 || v == nyq) ? 1.f : 2.f;
      acc = fmaf(h, fmaf(a.x, w.x, -a.y * w.y), acc);
      idx += m;
      if (idx >= g.Lw) idx -= g.Lw;
    }
    dst[e] = acc * g.scale;
  }
}

// ---------------------------------------------------------------------------
// spec_filt: w [F][C][Kh][Kw] -> W[b][c][f] at the kept bins (origin placement).
// One thread per (c, f) pair, consecutive threads on consecutive f (so the
// stores of a bin are contiguous); the grid is (pair blocks) x (bin chunks),
// numbered so that consecutive pair blocks run on one XCD: the taps of
// neighbouring channels c share cache lines, which are then fetched into one
// L2 rather than several.
// ---------------------------------------------------------------------------

template <int KH, int KW, typename S>
__global__ __launch_bounds__(kThreads) void k_spec_filt(const float* __restrict__ w, const float2* __restrict__ roots,
                                                        S* __restrict__ out, FiltGeom g) {
  extern __shared__ float2 smem[];
  spec_filt_block<KH, KW, S>(w, roots, out, g, blockIdx.x, gridDim.x, smem);
}

// ---------------------------------------------------------------------------
// wgrad_idft: DW[b][q] (q = c * F + f) -> dw[f][c][t], t = (a, b') < Kh x Kw:
//   dw = sum over kept bins (u, v) of Re(DW[u, v] * E[b][t]),
//   E[b][t] = h_v e^{+2 pi i (u a / Lh + v b' / Lw)} / (Lh Lw)
// (the c2r inverse restricted to the filter support), E tabulated once per
// plan.  Results do not depend on scheduling: every sum is taken in a fixed
// order.
// ---------------------------------------------------------------------------
template <int TMAX, int TC>
__global__ __launch_bounds__(kThreads) void k_wgrad_idft(const float2* __restrict__ DW, const float2* __restrict__ Et,
                                                         float* __restrict__ dw, float* __restrict__ part,
                                                         WgradGeom g) {
  extern __shared__ float2 E[];  // bins_per_chunk x TMAX, zero beyond T (no branches in the bin loop)
  __shared__ float res[wgrad_res_floats<TMAX, TC>()];
  wgrad_idft_block<TMAX, TC>(DW, Et, dw, part, g, blockIdx.x, blockIdx.y, gridDim.y > 1, E, res);
}

// One thread per (q, t): sums the slices in a fixed order (eight independent
// partial sums, combined pairwise at the end).
__global__ __launch_bounds__(kThreads) void k_wgrad_reduce(const float* __restrict__ part, float* __restrict__ dw,
                                                           WgradGeom g) {
  // four lanes per output value: lane j of a quad sums slices j, j + 4, ...
  // in order (all of its loads in flight together, eight at a time), and the
  // quad adds its four sums as (s0 + s1) + (s2 + s3); the order is fixed
  const long Q = (long)g.C * g.F;
  const long e = ((long)blockIdx.x * blockDim.x + threadIdx.x) >> 2;  // e = t * Q + q
  const int j = threadIdx.x & 3;
  const bool live = e < Q * g.T;
  const size_t stride = (size_t)g.T * Q;
  const float* src = part + (live ? e : 0);
  const int slices = g.chunks * max(1, g.nsplit);
  float acc = 0.f;
  for (int k0 = j; k0 < slices; k0 += 32) {
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int k = k0 + 4 * i;
      v[i] = k < slices ? src[(size_t)k * stride] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) acc += v[i];
  }
  acc += __shfl_xor(acc, 1);
  acc += __shfl_xor(acc, 2);
  if (!live || j != 0) return;
  const long q = e % Q;
  const int t = (int)(e / Q);
  const int c = (int)(q / g.F), f = (int)(q % g.F);
  dw[((size_t)f * g.C + c) * g.T + t] = acc;
}

template <int TMAX, int NW>
__global__ __launch_bounds__(64 * NW) void k_wgrad_wide(const float2* __restrict__ DW, const float2* __restrict__ Et,
                                                        float* __restrict__ dw, WgradGeom g) {
  extern __shared__ float2 E[];  // [kept][TMAX], zero beyond T: the bin loop has no branches
  __shared__ float red[NW * 64 * TMAX];
  wgrad_wide_block<TMAX, NW>(DW, Et, dw, g, blockIdx.x, E, red);
}

// Layers of 128 to 511 tiles of 16 x 16 channel pairs: a block
// takes a tile of 16 input channels x 16 filters and all kept bins; its NG
// groups of 256 threads (one pair (c, f) per thread) each sum a contiguous
// part of the bins, reading DW[bin][c][f] as runs of 16 filters (128 bytes)
// and E from LDS, 16 bins' loads in flight at a time.  The groups' sums are
// added in a fixed order through LDS and written transposed, so that each
// filter's row dw[f][c0 .. c0 + 16][:] is one contiguous run.
template <int TMAX, int NG>
__global__ __launch_bounds__(256 * NG) void k_wgrad_tile(const float2* __restrict__ DW, const float2* __restrict__ Et,
                                                         float* __restrict__ out, WgradGeom g) {
  extern __shared__ float2 smem2[];
  float2* E = smem2;                                                 // [bins_per_chunk][TMAX], zero beyond T
  float* red = reinterpret_cast<float*>(smem2 + (size_t)g.bins_per_chunk * TMAX);  // [NG][256][TMAX]
  const int B = g.R * g.V;
  const int b0 = blockIdx.y * g.bins_per_chunk;
  const int nb = min(g.bins_per_chunk, B - b0);
  const float2* Es = Et + (size_t)b0 * g.T;
  for (int e = threadIdx.x; e < nb * TMAX; e += blockDim.x) {
    const int bb = e / TMAX, t = e - bb * TMAX;
    E[e] = t < g.T ? Es[bb * g.T + t] : make_float2(0.f, 0.f);
  }
  __syncthreads();
  const size_t Q = (size_t)g.C * g.F;
  const int c0 = (blockIdx.x / g.tiles_f) * 16, f0 = (blockIdx.x % g.tiles_f) * 16;
  const int grp = threadIdx.x >> 8, pr = threadIdx.x & 255, cl = pr >> 4, fl = pr & 15;
  const int c = c0 + cl, f = f0 + fl;
  const bool valid = c < g.C && f < g.F;
  const int bb0 = grp * nb / NG, bb1 = (grp + 1) * nb / NG;
  float acc[TMAX];
#pragma unroll
  for (int t = 0; t < TMAX; ++t) acc[t] = 0.f;
  const float2* src = DW + (size_t)b0 * Q + (valid ? (size_t)c * g.F + f : 0);
  for (int bb = bb0; bb < bb1; bb += 16) {
    float2 d[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) d[j] = src[(size_t)min(bb + j, bb1 - 1) * Q];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const float2 dj = bb + j < bb1 ? d[j] : make_float2(0.f, 0.f);
      const float2* Eb = E + min(bb + j, bb1 - 1) * TMAX;
#pragma unroll
      for (int t = 0; t < TMAX; ++t) acc[t] = fmaf(dj.x, Eb[t].x, fmaf(-dj.y, Eb[t].y, acc[t]));
    }
  }
#pragma unroll
  for (int t = 0; t < TMAX; ++t) red[((size_t)grp * 256 + pr) * TMAX + t] = acc[t];
  __syncthreads();
  if (grp == 0) {
#pragma unroll
    for (int t = 0; t < TMAX; ++t) {
      float sum = red[pr * TMAX + t];
#pragma unroll
      for (int w = 1; w < NG; ++w) sum += red[((size_t)w * 256 + pr) * TMAX + t];
      acc[t] = sum;
    }
  }
  __syncthreads();
  // transposed: filter fl's 16 channels x T taps contiguous
  if (grp == 0) {
#pragma unroll
    for (int t = 0; t < TMAX; ++t)
      if (t < g.T) red[(fl * 16 + cl) * g.T + t] = acc[t];
  }
  __syncthreads();
  float* o = out;
  const int seg = 16 * g.T;
  for (int e = threadIdx.x; e < 16 * seg; e += blockDim.x) {
    const int ef = e / seg, r = e - ef * seg;
    const int oc = c0 + r / g.T, of = f0 + ef;
    if (oc < g.C && of < g.F) o[((size_t)of * g.C + c0) * g.T + r] = red[e];
  }
}

// Inverse-DFT weights E[bin][t] of the weight gradient, in double precision.
void host_wgrad_weights(const bl_conv_plan_s* p, std::vector<float2>& out) {
  const int T = p->Kh * p->Kw, B = (int)p->kept;
  const long LL = (long)p->Lh * p->Lw;
  const int nyq = (p->Lw % 2 == 0) ? p->Lw / 2 : -1;
  const double pi = 3.141592653589793238462643383279502884;
  out.assign((size_t)B * T, make_float2(0.f, 0.f));
  for (int bin = 0; bin < B; ++bin) {
    const int r = bin / p->V, v = bin % p->V;
    const int u = bl_kept_row(r, p->r_h, p->Lh, p->R);
    const double h = ((v == 0 || v == nyq) ? 1.0 : 2.0) / (double)LL;
    for (int t = 0; t < T; ++t) {
      const int ta = t / p->Kw, tb = t % p->Kw;
      const long idx = ((long)u * ta * p->Lw + (long)v * tb * p->Lh) % LL;
      const double ang = 2.0 * pi * (double)idx / (double)LL;
      out[(size_t)bin * T + t] = make_float2((float)(h * std::cos(ang)), (float)(h * std::sin(ang)));
    }
  }
}

// ---------------------------------------------------------------------------
// contract: per kept bin, O[m][n] = sum_k A[m][k] * op(B[k][n]) in complex64,
// op = conj or identity.  The complex product is embedded in a real GEMM:
// A is read as a real [M x 2K] matrix (interleaved re/im), B as the real
// [2K x 2N] matrix of 2x2 blocks [[br, -bi], [bi, br]] (conj) or
// [[br, bi], [-bi, br]] (identity), and the real output [M x 2N] is the
// interleaved complex O.  fp32 MFMA 32x32x2: each 2-deep real k step is one
// complex k.  Block tile: 64 rows x 32 complex columns, 16 complex k per stage;
// wave w owns rows 32*(w/2).. and complex columns 16*(w%2)...
// ---------------------------------------------------------------------------
struct ContractArgs {
  int M, N, K;
  long sAm, sAk, sBk, sBn, ldo;  // element strides (complex units)
  long bA, bB, bO;               // per-bin strides
  int tiles_n;
};

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int CBM = 64, CBN = 32, CBK = 16;

// S: stored-spectrum element of the operands (float2, or bfloat16 pairs whose
// products the fp32 MFMA forms exactly)
template <bool A_K_CONTIG, bool B_N_CONTIG, bool CONJ, typename S>
__global__ __launch_bounds__(kThreads) void k_contract(const S* __restrict__ A, const S* __restrict__ Bm,
                                                       float2* __restrict__ O, ContractArgs g) {
  __shared__ float As[2][CBK][CBM];
  __shared__ float Bs[2][CBK][CBN];
  const int bin = blockIdx.y;
  const int tm = blockIdx.x / g.tiles_n, tn = blockIdx.x % g.tiles_n;
  const int m0 = tm * CBM, n0 = tn * CBN;
  const S* Ab = A + (size_t)bin * g.bA;
  const S* Bb = Bm + (size_t)bin * g.bB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * 32, wn = (wave & 1) * 16;

  // B operand selection for lane: real column j = lane % 32 -> complex column
  // wn + j/2, part bcol = j & 1; real k row a = lane / 32.
  const int a_part = lane >> 5;
  const int jcol = lane & 31;
  const int bcol = jcol & 1;
  const int bn = wn + (jcol >> 1);
  const int b_src = (a_part == bcol) ? 0 : 1;  // take br on the diagonal, bi off it
  float b_sign = 1.f;
  if (CONJ && a_part == 0 && bcol == 1) b_sign = -1.f;
  if (!CONJ && a_part == 1 && bcol == 0) b_sign = -1.f;

  floatx16 acc;
#pragma unroll
  for (int i = 0; i < 16; ++i) acc[i] = 0.f;

  for (int k0 = 0; k0 < g.K; k0 += CBK) {
    // A tile: 64 rows x 16 complex k
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      int m, k;
      if (A_K_CONTIG) {
        const int e = tid * 4 + it;  // 0..1023
        m = e >> 4; k = e & 15;
      } else {
        const int e = tid * 4 + it;
        k = e >> 6; m = e & 63;
      }
      float2 v = make_float2(0.f, 0.f);
      if (m0 + m < g.M && k0 + k < g.K) v = spec_get(Ab, (size_t)(m0 + m) * g.sAm + (size_t)(k0 + k) * g.sAk);
      As[0][k][m] = v.x;
      As[1][k][m] = v.y;
    }
    // B tile: 16 complex k x 32 complex n
#pragma unroll
    for (int it = 0; it < 2; ++it) {
      int k, n;
      const int e = tid * 2 + it;  // 0..511
      if (B_N_CONTIG) { k = e >> 5; n = e & 31; }
      else { n = e >> 4; k = e & 15; }
      float2 v = make_float2(0.f, 0.f);
      if (n0 + n < g.N && k0 + k < g.K) v = spec_get(Bb, (size_t)(k0 + k) * g.sBk + (size_t)(n0 + n) * g.sBn);
      Bs[0][k][n] = v.x;
      Bs[1][k][n] = v.y;
    }
    __syncthreads();
#pragma unroll
    for (int s = 0; s < CBK; ++s) {
      const float av = As[a_part][s][wm + (lane & 31)];
      const float bv = b_sign * Bs[b_src][s][bn];
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc, 0, 0, 0);
    }
    __syncthreads();
  }

  // D[i][j]: VGPR v holds row 8*(v/4) + 4*(lane/32) + v%4, column lane%32.
  float* Of = reinterpret_cast<float*>(O + (size_t)bin * g.bO);
  const int n = n0 + bn;
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int i = 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
    const int m = m0 + wm + i;
    if (m < g.M && n < g.N) Of[((size_t)m * g.ldo + n) * 2 + bcol] = acc[v];
  }
}

int planes_per_block(size_t fixed_bytes, size_t per_plane_bytes, long P, int cap, size_t limit = kMaxLds) {
  int tp = (int)std::min<long>(cap, P);
  while (tp > 1 && fixed_bytes + tp * per_plane_bytes > limit) --tp;
  return std::max(tp, 1);
}

// A plane whose working set exceeds 64 KB (long 1-D series, wide maps) runs
// alone in a block with up to the CU's 160 KB of LDS, which the kernel must
// be allowed once per device.
constexpr size_t kMaxLdsLarge = 160 * 1024;
bool allow_large_lds(const void* kern) { return lds_opt_in(kern, (int)kMaxLdsLarge) == BL_OK; }

}  // namespace

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

// Real planes [P][Hin][Win] at offset (oi, oj) -> bin-major kept spectrum.
bl_status_t launch_spec_fwd_direct(const bl_conv_plan_s* p, const float* in, void* out, long P, int Hin, int Win, int oi,
                            int oj, hipStream_t s) {
  FwdGeom g{Hin, Win, oi, oj, p->Lh, p->Lw, p->r_h, p->R, p->V, P, 0};
  const size_t fixed = (size_t)(p->Lh + p->Lw) * sizeof(float2);
  const size_t per = (size_t)(Hin * p->V + 1) * sizeof(float2) + (size_t)Hin * Win * sizeof(float);
  const size_t limit = fixed + per > kMaxLds ? kMaxLdsLarge : kMaxLds;
  if (fixed + per > limit) return BL_ERR_UNSUPPORTED;
  g.TP = planes_per_block(fixed, per, P, 16, limit);
  const size_t lds = fixed + g.TP * per;
  if (lds > kMaxLds) {
    const void* kern = p->bf16 ? reinterpret_cast<const void*>(&k_spec_fwd<unsigned>)
                               : reinterpret_cast<const void*>(&k_spec_fwd<float2>);
    if (!allow_large_lds(kern)) return BL_ERR_HIP;
  }
  const long blocks = (P + g.TP - 1) / g.TP;
  const double bytes = (double)P * Hin * Win * 4 + (double)P * p->kept * (p->bf16 ? 4 : 8);
  return timed_launch("spec_fwd_direct", bytes, 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
    if (p->bf16)
      hipExtLaunchKernelGGL(k_spec_fwd<unsigned>, dim3((unsigned)blocks), dim3(kThreads), lds, s, e0, e1, 0, in,
                            static_cast<unsigned*>(out), g);
    else
      hipExtLaunchKernelGGL(k_spec_fwd<float2>, dim3((unsigned)blocks), dim3(kThreads), lds, s, e0, e1, 0, in,
                            static_cast<float2*>(out), g);
  });
}

bl_status_t launch_spec_inv_direct(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OH, int OW, int ci,
                            int cj, hipStream_t s) {
  InvGeom g{OH, OW, ci, cj, p->Lh, p->Lw, p->r_h, p->R, p->V, P, 0, 1.0f / ((float)p->Lh * (float)p->Lw)};
  const size_t fixed = (size_t)(p->Lh + p->Lw) * sizeof(float2);
  const size_t per = (size_t)(p->R * p->V + 1 + OH * p->V + 1) * sizeof(float2);
  const size_t limit = fixed + per > kMaxLds ? kMaxLdsLarge : kMaxLds;
  if (fixed + per > limit) return BL_ERR_UNSUPPORTED;
  g.TP = planes_per_block(fixed, per, P, 16, limit);
  const size_t lds = fixed + g.TP * per;
  if (lds > kMaxLds) {
    if (!allow_large_lds(reinterpret_cast<const void*>(&k_spec_inv))) return BL_ERR_HIP;
  }
  const long blocks = (P + g.TP - 1) / g.TP;
  const double bytes = (double)P * p->kept * 8 + (double)P * OH * OW * 4;
  return timed_launch("spec_inv_direct", bytes, 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
    hipExtLaunchKernelGGL(k_spec_inv, dim3((unsigned)blocks), dim3(kThreads), lds, s, e0, e1, 0, in, out, g);
  });
}


// e^{-2 pi i k / Lh} for k < Lh, then e^{-2 pi i k / Lw} for k < Lw, in double precision.
void host_filt_roots(const bl_conv_plan_s* p, std::vector<float2>& out) {
  const double pi = 3.141592653589793238462643383279502884;
  out.clear();
  for (int L : {p->Lh, p->Lw})
    for (int k = 0; k < L; ++k) {
      const double a = 2.0 * pi * (double)k / (double)L;
      out.push_back(make_float2((float)std::cos(a), (float)(-std::sin(a))));
    }
}

bl_status_t filt_setup(const bl_conv_plan_s* p, bool use_table, FiltGeom& g, const float2** roots, long* blocks,
                       size_t* lds, double* bytes) {
  g = FiltGeom{p->Cout, p->Cin, p->Kh, p->Kw, p->Lh, p->Lw, p->r_h, p->R, p->V, 0, 0};
  *roots = nullptr;
  bool known = false;
#define X(a, b) known = known || (p->Kh == a && p->Kw == b);
  BL_FILT_CASES(X)
#undef X
  if (!known) return BL_ERR_UNSUPPORTED;
  const long CF = (long)p->Cin * p->Cout;
  const int B = p->R * p->V;
  const long xblocks = (CF + kThreads - 1) / kThreads;
  // aim for about 1024 blocks in all
  int chunks = (int)std::max<long>(1, std::min<long>(B, (1024 + xblocks - 1) / xblocks));
  g.bins_per_block = (B + chunks - 1) / chunks;
  chunks = (B + g.bins_per_block - 1) / g.bins_per_block;
  g.xblocks = (int)xblocks;
  if ((double)xblocks * chunks >= 2147483647.0) return BL_ERR_UNSUPPORTED;
  *blocks = xblocks * chunks;
  *lds = (size_t)(p->Lh + p->Lw) * sizeof(float2);
  *bytes = (double)CF * p->Kh * p->Kw * 4 + (double)CF * B * (p->bf16 ? 4 : 8);
  if (use_table) {
    const std::vector<long> key{3, p->Lh, p->Lw};
    return plan_table(p, key, [&](std::vector<float2>& h) { host_filt_roots(p, h); }, roots);
  }
  return BL_OK;
}

bl_status_t launch_spec_filt(const bl_conv_plan_s* p, const float* w, void* out, hipStream_t s, bool use_table) {
  FiltGeom g;
  const float2* roots;
  long blocks;
  size_t lds;
  double bytes;
  const bl_status_t st = filt_setup(p, use_table, g, &roots, &blocks, &lds, &bytes);
  if (st != BL_OK) return st;
  const dim3 grid((unsigned)blocks);
#define X(a, b)                                                                                             \
  if (p->Kh == a && p->Kw == b)                                                                             \
    return timed_launch("spec_filt", bytes, 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {                    \
      if (p->bf16)                                                                                          \
        hipExtLaunchKernelGGL((k_spec_filt<a, b, unsigned>), grid, dim3(kThreads), lds, s, e0, e1, 0, w, roots, \
                              static_cast<unsigned*>(out), g);                                              \
      else                                                                                                  \
        hipExtLaunchKernelGGL((k_spec_filt<a, b, float2>), grid, dim3(kThreads), lds, s, e0, e1, 0, w, roots,   \
                              static_cast<float2*>(out), g);                                                \
    });
  BL_FILT_CASES(X)
#undef X
  return BL_ERR_UNSUPPORTED;
}

bool wgrad_wide(const bl_conv_plan_s* p) {
  const long Q = (long)p->Cin * p->Cout;
  const int B = (int)p->kept, T = p->Kh * p->Kw;
  const int tmax_w = T <= 9 ? T : 16;
  return (Q / 64 >= 256 || B <= 256) && p->Cout <= 256 && T <= 16 &&
         (long)(B * tmax_w * sizeof(float2)) <= kWgradSliceLds && Q < 2147483647L;
}

bl_status_t wgrad_table(const bl_conv_plan_s* p, const float2** Et) {
  const std::vector<long> key{2, p->Lh, p->Lw, p->r_h, p->R, p->V, p->Kh, p->Kw};
  return plan_table(p, key, [&](std::vector<float2>& h) { host_wgrad_weights(p, h); }, Et);
}

bool wgrad_sliced_setup(const bl_conv_plan_s* p, int nsplit, WgradGeom& g, long* xblocks, int* slices, size_t* lds,
                        int* tc, const float2** Et) {
  g = WgradGeom{p->Cout, p->Cin, p->Kh, p->Kw, p->Kh * p->Kw, p->Lh, p->Lw, p->r_h, p->R, p->V, 0, 0,
                (p->Cout + 15) / 16, 1, 0};
  if (g.T > 64 || p->wg_groups > 0 || wgrad_wide(p)) return false;
  const long Q = (long)p->Cin * p->Cout;
  if (nsplit > 1) {
    if (p->wg_chunks <= 1 || nsplit > std::max(1, p->bp_s2)) return false;  // partial-sum area sized for these
    g.nsplit = nsplit;
    g.pstride = (unsigned long long)p->kept * Q;
  }
  g.chunks = p->wg_chunks;  // the workspace holds partial sums for this many slices (per partial spectrum)
  g.bins_per_chunk = p->wg_bins;
  if ((long)g.chunks * g.nsplit > 65535) return false;
  const int tmax = g.T <= 9 ? g.T : g.T <= 16 ? 16 : g.T <= 32 ? 32 : 64;  // as instantiated
  *lds = (size_t)g.bins_per_chunk * tmax * sizeof(float2);
  if ((long)*lds > kWgradSliceLds) return false;
  const int TC = chan_tile(g.T, p->Cout), TF = kThreads / TC;
  *tc = TC;
  *xblocks = TC == 1 ? (Q + kThreads - 1) / kThreads : (long)((p->Cin + TC - 1) / TC) * ((p->Cout + TF - 1) / TF);
  *slices = g.chunks * g.nsplit;
  return wgrad_table(p, Et) == BL_OK;
}

bl_status_t launch_wgrad_reduce(const bl_conv_plan_s* p, const float* part, float* dw, const WgradGeom& g,
                                hipStream_t s) {
  const long Q = (long)p->Cin * p->Cout;
  const long rblocks = (4 * Q * g.T + kThreads - 1) / kThreads;  // four lanes per value
  return timed_launch("wgrad_reduce", (double)Q * g.T * 4 * (g.chunks * g.nsplit + 1), 0.0, s,
                      [&](hipEvent_t e0, hipEvent_t e1) {
    hipExtLaunchKernelGGL(k_wgrad_reduce, dim3((unsigned)rblocks), dim3(kThreads), 0, s, e0, e1, 0, part, dw, g);
  });
}

bl_status_t launch_wgrad_idft(const bl_conv_plan_s* p, const float2* DW, float* dw, float* part, hipStream_t s,
                              int nsplit, float2* tmp) {
  WgradGeom g{p->Cout, p->Cin, p->Kh, p->Kw, p->Kh * p->Kw, p->Lh, p->Lw, p->r_h, p->R, p->V, 0, 0,
              (p->Cout + 15) / 16, 1, 0};
  const long Q = (long)p->Cin * p->Cout;
  const int B = (int)p->kept;
  const int tmax_w = g.T <= 9 ? g.T : 16;
  const bool wide = wgrad_wide(p);
  if (nsplit > 1) {
    // partial spectra: more slices of the sliced path (whose partial-sum area
    // the plan sized for them), else summed into tmp first
    if (p->wg_groups == 0 && !wide && p->wg_chunks > 1 && nsplit <= std::max(1, p->bp_s2)) {
      g.nsplit = nsplit;
      g.pstride = (unsigned long long)B * Q;
    } else {
      if (!tmp) return BL_ERR_INVALID_ARG;
      const bl_status_t st = launch_split_reduce(DW, tmp, (unsigned long long)B * Q, nsplit, s);
      if (st != BL_OK) return st;
      DW = tmp;
    }
  }
  // one pass over all bins when there are at least 256 blocks of 64 pairs,
  // or few bins (at most 256: a sixteenth per wave), and taps and table fit
  // (rows of at most 256 output channels: wider rows write dw better from the
  // tiled kernel below); otherwise bin slices and a fixed-order sum
  if (g.T > 64) return BL_ERR_UNSUPPORTED;
  const float2* Et = nullptr;  // E[bin][t], built once per plan
  const bl_status_t ts = wgrad_table(p, &Et);
  if (ts != BL_OK) return ts;
  if (p->wg_groups > 0) {  // 16 x 16 channel tiles over all bins
    const int tmax = wgrad_tmax(g.T), NG = p->wg_groups;
    g.bins_per_chunk = B;
    g.chunks = 1;
    const size_t lds = (size_t)B * tmax * sizeof(float2) + (size_t)NG * 256 * tmax * sizeof(float);
    const long tiles = (long)((p->Cin + 15) / 16) * g.tiles_f;
    const double bytes = (double)Q * B * 8 + (double)Q * g.T * 4;
    bl_status_t st = BL_ERR_UNSUPPORTED;
    auto go = [&](auto kern, int ng) {
      if (lds > 64 * 1024) {
        const bl_status_t at = lds_opt_in(reinterpret_cast<const void*>(kern), 160 * 1024);
        if (at != BL_OK) return at;
      }
      return timed_launch("wgrad_idft", bytes, 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
        hipExtLaunchKernelGGL(kern, dim3((unsigned)tiles), dim3(256 * ng), lds, s, e0, e1, 0, DW, Et, dw, g);
      });
    };
#define BL_WG(TM)                                                                                            \
  case TM:                                                                                                   \
    st = NG == 4 ? go(k_wgrad_tile<TM, 4>, 4) : NG == 2 ? go(k_wgrad_tile<TM, 2>, 2) : go(k_wgrad_tile<TM, 1>, 1); \
    break;
    switch (tmax) {
      BL_WG(1) BL_WG(2) BL_WG(3) BL_WG(4) BL_WG(5) BL_WG(6) BL_WG(7) BL_WG(8) BL_WG(9) BL_WG(16)
      default: return BL_ERR_UNSUPPORTED;
    }
#undef BL_WG
    return st;
  }
  if (wide) {
    const size_t lds = (size_t)B * tmax_w * sizeof(float2);
    const long blocks = (Q + 63) / 64;
    // at most one block per CU: 16 waves per block, each over a sixteenth of
    // the bins, so that every SIMD still holds several waves (measured: with
    // 512 blocks, 4 waves per block are faster)
    const bool many = blocks <= 256;
    const double bytes = (double)Q * B * 8 + (double)Q * g.T * 4;
    auto go = [&](auto kern, int nw) {
      // the static reduction buffer plus up to kWgradSliceLds of weights can
      // pass 64 KB of LDS: allowed once per kernel instantiation and device
      const bl_status_t at = lds_opt_in(reinterpret_cast<const void*>(kern), (int)kWgradSliceLds);
      if (at != BL_OK) return at;
      return timed_launch("wgrad_idft", bytes, 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
        hipExtLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(64 * nw), lds, s, e0, e1, 0, DW, Et, dw, g);
      });
    };
#define BL_WIDE(t) \
  case t: return many ? go(k_wgrad_wide<t, 16>, 16) : go(k_wgrad_wide<t, 4>, 4);
    switch (g.T) {
      BL_WIDE(1) BL_WIDE(2) BL_WIDE(3) BL_WIDE(4) BL_WIDE(5) BL_WIDE(6) BL_WIDE(7) BL_WIDE(8) BL_WIDE(9)
      default: return many ? go(k_wgrad_wide<16, 16>, 16) : go(k_wgrad_wide<16, 4>, 4);
    }
#undef BL_WIDE
  }
  g.chunks = p->wg_chunks;  // the workspace holds partial sums for this many slices (per partial spectrum)
  g.bins_per_chunk = p->wg_bins;
  if ((long)g.chunks * g.nsplit > 65535) return BL_ERR_UNSUPPORTED;
  const int tmax = g.T <= 9 ? g.T : g.T <= 16 ? 16 : g.T <= 32 ? 32 : 64;  // as instantiated below
  const size_t lds = (size_t)g.bins_per_chunk * tmax * sizeof(float2);
  if ((long)lds > kWgradSliceLds) return BL_ERR_UNSUPPORTED;
  const int TC = chan_tile(g.T, p->Cout), TF = kThreads / TC;
  const long xblocks = TC == 1 ? (Q + kThreads - 1) / kThreads : (long)((p->Cin + TC - 1) / TC) * ((p->Cout + TF - 1) / TF);
  dim3 grid((unsigned)xblocks, (unsigned)(g.chunks * g.nsplit));
  const double bytes = (double)Q * B * 8 * g.nsplit + (double)Q * g.T * 4;
  bl_status_t st;
  auto go = [&](auto kern) {
    return timed_launch("wgrad_idft", bytes, 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
      hipExtLaunchKernelGGL(kern, grid, dim3(kThreads), lds, s, e0, e1, 0, DW, Et, dw, part, g);
    });
  };
  auto go2 = [&](auto k8, auto k1) { return TC == 8 ? go(k8) : go(k1); };
  switch (g.T) {
#define BL_WG_T(n) \
  case n: st = go2(k_wgrad_idft<n, 8>, k_wgrad_idft<n, 1>); break;
    BL_WG_T(1) BL_WG_T(2) BL_WG_T(3) BL_WG_T(4) BL_WG_T(5) BL_WG_T(6) BL_WG_T(7) BL_WG_T(8) BL_WG_T(9)
#undef BL_WG_T
    default:
      if (g.T <= 16) st = go2(k_wgrad_idft<16, 8>, k_wgrad_idft<16, 1>);
      else if (g.T <= 32) st = go(k_wgrad_idft<32, 1>);
      else st = go(k_wgrad_idft<64, 1>);
  }
  if (st != BL_OK || g.chunks * g.nsplit == 1) return st;
  return launch_wgrad_reduce(p, part, dw, g, s);
}

bl_status_t launch_contract_generic(const bl_conv_plan_s* p, Contract which, const void* A, const void* Bm, float2* O,
                            hipStream_t s) {
  ContractArgs g{};
  const long B = p->kept, N = p->N, Ci = p->Cin, Co = p->Cout;
  switch (which) {
    case Contract::Forward:  // Y[n][f] = sum_c X[n][c] conj(W[c][f])
      g.M = (int)N; g.N = (int)Co; g.K = (int)Ci;
      g.sAm = Ci; g.sAk = 1; g.sBk = Co; g.sBn = 1; g.ldo = Co;
      g.bA = N * Ci; g.bB = Ci * Co; g.bO = N * Co;
      break;
    case Contract::GradInput:  // DX[n][c] = sum_f DY[n][f] W[c][f]
      g.M = (int)N; g.N = (int)Ci; g.K = (int)Co;
      g.sAm = Co; g.sAk = 1; g.sBk = 1; g.sBn = Co; g.ldo = Ci;
      g.bA = N * Co; g.bB = Ci * Co; g.bO = N * Ci;
      break;
    case Contract::GradWeight:  // DW[c][f] = sum_n X[n][c] conj(DY[n][f])
      g.M = (int)Ci; g.N = (int)Co; g.K = (int)N;
      g.sAm = 1; g.sAk = Ci; g.sBk = Co; g.sBn = 1; g.ldo = Co;
      g.bA = N * Ci; g.bB = N * Co; g.bO = Ci * Co;
      break;
  }
  const int tiles_m = (g.M + CBM - 1) / CBM;
  g.tiles_n = (g.N + CBN - 1) / CBN;
  if (B > 65535) return BL_ERR_UNSUPPORTED;
  dim3 grid((unsigned)(tiles_m * g.tiles_n), (unsigned)B);
  // complex MAC = 8 real flops; compulsory traffic: both operands and the result once
  const double flops = 8.0 * B * g.M * g.N * g.K;
  const double ob = p->bf16 ? 4.0 : 8.0;  // bytes per stored operand element
  const double bytes = B * (ob * ((double)g.M * g.K + (double)g.K * g.N) + 8.0 * g.M * g.N);
  const char* name = which == Contract::Forward ? "contract_fwd"
                     : which == Contract::GradInput ? "contract_dgrad" : "contract_wgrad";
  auto go = [&](auto kern, auto* a, auto* b) {
    return timed_launch(name, bytes, flops, s, [&](hipEvent_t e0, hipEvent_t e1) {
      hipExtLaunchKernelGGL(kern, grid, dim3(kThreads), 0, s, e0, e1, 0, a, b, O, g);
    });
  };
  const unsigned* A16 = static_cast<const unsigned*>(A);
  const unsigned* B16 = static_cast<const unsigned*>(Bm);
  const float2* A32 = static_cast<const float2*>(A);
  const float2* B32 = static_cast<const float2*>(Bm);
  switch (which) {
    case Contract::Forward:
      return p->bf16 ? go(k_contract<true, true, true, unsigned>, A16, B16)
                     : go(k_contract<true, true, true, float2>, A32, B32);
    case Contract::GradInput:
      return p->bf16 ? go(k_contract<true, false, false, unsigned>, A16, B16)
                     : go(k_contract<true, false, false, float2>, A32, B32);
    case Contract::GradWeight:
      return p->bf16 ? go(k_contract<false, true, true, unsigned>, A16, B16)
                     : go(k_contract<false, true, true, float2>, A32, B32);
  }
  return BL_ERR_INVALID_ARG;
}

}  // namespace blc
