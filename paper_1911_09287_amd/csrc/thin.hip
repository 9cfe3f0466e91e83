// Per-kept-bin complex channel contraction when one of its sizes is small
// (at most 8): O[m][n] = sum_k A[m][k] op(B[k][n]), op = conj or identity, the
// Hadamard product of the spectra summed over a channel index (Sec. 3.3).
// Such a contraction moves far more bytes than it has products to compute
// (the first layer of a network, with one or three input channels, is the
// usual case), so it runs on the vector ALUs at memory speed instead of
// padding an MFMA tile that is mostly zeros:
//   k_thin_cols  (M <= 8 or K <= 8): lanes over 64 consecutive output columns n,
//                each lane accumulating MT rows; with K >= 64 the four waves
//                of a block split k and add their partial sums through LDS in
//                a fixed order;
//   k_thin_rows  (N <= 8): one output row per wave, lanes over k, each lane
//                accumulating the N columns, then a butterfly sum across the
//                wave (fixed order).
// Results do not depend on scheduling.
#include <algorithm>

#include "common.hpp"

namespace blc {
namespace {

struct ThinArgs {
  int M, N, K;
  long sAm, sAk, sBk, sBn, ldo;  // element strides (complex units)
  long bA, bB, bO;               // per-bin strides
  int items_n, items;            // (row group, 64-column group) items per bin
  int ks;                        // waves splitting k: 1 (a wave per item) or 4 (a block per item)
};

__device__ __forceinline__ float2 cmac(float2 acc, float2 a, float2 b) {
  return make_float2(fmaf(a.x, b.x, fmaf(-a.y, b.y, acc.x)), fmaf(a.x, b.y, fmaf(a.y, b.x, acc.y)));
}

// S: stored-spectrum element of the operands (float2 or bfloat16 pairs)
template <int MT, bool CONJ, typename S>
__global__ __launch_bounds__(256) void k_thin_cols(const S* __restrict__ A, const S* __restrict__ B,
                                                   float2* __restrict__ O, ThinArgs g) {
  __shared__ float2 red[3][MT][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int item = g.ks == 4 ? (int)blockIdx.x : (int)blockIdx.x * 4 + wave;
  const bool has = item < g.items;
  const int m0 = (item / g.items_n) * MT, n = (item % g.items_n) * 64 + lane;
  const bool live = has && n < g.N;
  int k0 = 0, k1 = g.K;
  if (g.ks == 4) {
    const int kc = (g.K + 3) / 4;
    k0 = min(g.K, wave * kc);
    k1 = min(g.K, k0 + kc);
  }
  const S* Ab = A + (size_t)blockIdx.y * g.bA;
  const S* Bb = B + (size_t)blockIdx.y * g.bB + (live ? (long)n * g.sBn : 0);
  float2 acc[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) acc[i] = make_float2(0.f, 0.f);
  if (live) {
    // rows past M repeat the last row (computed, never written)
    long arow[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) arow[i] = (long)min(m0 + i, g.M - 1) * g.sAm;
#pragma unroll 4
    for (int k = k0; k < k1; ++k) {
      float2 b = spec_get(Bb, (long)k * g.sBk);
      if (CONJ) b.y = -b.y;
#pragma unroll
      for (int i = 0; i < MT; ++i) acc[i] = cmac(acc[i], spec_get(Ab, arow[i] + (long)k * g.sAk), b);
    }
  }
  if (g.ks == 4) {
    if (wave > 0) {
#pragma unroll
      for (int i = 0; i < MT; ++i) red[wave - 1][i][lane] = acc[i];
    }
    __syncthreads();
    if (wave > 0) return;
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const float2 r1 = red[0][i][lane], r2 = red[1][i][lane], r3 = red[2][i][lane];
      acc[i] = make_float2(((acc[i].x + r1.x) + r2.x) + r3.x, ((acc[i].y + r1.y) + r2.y) + r3.y);
    }
  }
  if (!live) return;
  float2* Ob = O + (size_t)blockIdx.y * g.bO + n;
#pragma unroll
  for (int i = 0; i < MT; ++i)
    if (m0 + i < g.M) Ob[(long)(m0 + i) * g.ldo] = acc[i];
}

template <int NT, bool CONJ, typename S>
__global__ __launch_bounds__(256) void k_thin_rows(const S* __restrict__ A, const S* __restrict__ B,
                                                   float2* __restrict__ O, ThinArgs g) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int m = (int)blockIdx.x * 4 + wave;
  if (m >= g.M) return;  // whole waves leave together; no block barrier follows
  const S* Ab = A + (size_t)blockIdx.y * g.bA + (long)m * g.sAm;
  const S* Bb = B + (size_t)blockIdx.y * g.bB;
  float2 acc[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) acc[j] = make_float2(0.f, 0.f);
  for (int k = lane; k < g.K; k += 64) {
    const float2 a = spec_get(Ab, (long)k * g.sAk);
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      // columns past N repeat the last one (computed, never written)
      float2 b = spec_get(Bb, (long)k * g.sBk + (long)min(j, g.N - 1) * g.sBn);
      if (CONJ) b.y = -b.y;
      acc[j] = cmac(acc[j], a, b);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
#pragma unroll
    for (int j = 0; j < NT; ++j) {
      acc[j].x += __shfl_xor(acc[j].x, off, 64);
      acc[j].y += __shfl_xor(acc[j].y, off, 64);
    }
  }
  if (lane == 0) {
    float2* Ob = O + (size_t)blockIdx.y * g.bO + (long)m * g.ldo;
#pragma unroll
    for (int j = 0; j < NT; ++j)
      if (j < g.N) Ob[j] = acc[j];
  }
}

int pow2_at_least(int v) {
  int p = 1;
  while (p < v) p *= 2;
  return p;
}

}  // namespace

bool contract_is_thin(const bl_conv_plan_s* p, Contract which) {
  const long N = p->N, Ci = p->Cin, Co = p->Cout;
  long M = N, Nn = Co, K = Ci;
  if (which == Contract::GradInput) Nn = Ci, K = Co;
  if (which == Contract::GradWeight) M = Ci, K = N;
  return std::min({M, Nn, K}) <= 8;
}

bl_status_t launch_contract_thin(const bl_conv_plan_s* p, Contract which, const void* A, const void* Bm,
                                 float2* O, hipStream_t s) {
  ThinArgs g{};
  const long B = p->kept, N = p->N, Ci = p->Cin, Co = p->Cout;
  bool conj = true;
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
      conj = false;
      break;
    case Contract::GradWeight:  // DW[c][f] = sum_n X[n][c] conj(DY[n][f])
      g.M = (int)Ci; g.N = (int)Co; g.K = (int)N;
      g.sAm = 1; g.sAk = Ci; g.sBk = Co; g.sBn = 1; g.ldo = Co;
      g.bA = N * Ci; g.bB = N * Co; g.bO = Ci * Co;
      break;
  }
  if (B > 65535 || B < 1) return BL_ERR_UNSUPPORTED;
  const double flops = 8.0 * B * g.M * g.N * g.K;
  const double ob = p->bf16 ? 4.0 : 8.0;  // bytes per stored operand element
  const double bytes = B * (ob * ((double)g.M * g.K + (double)g.K * g.N) + 8.0 * g.M * g.N);
  const unsigned* A16 = static_cast<const unsigned*>(A);
  const unsigned* B16 = static_cast<const unsigned*>(Bm);
  const float2* A32 = static_cast<const float2*>(A);
  const float2* B32 = static_cast<const float2*>(Bm);
  const char* name = which == Contract::Forward ? "contract_fwd"
                     : which == Contract::GradInput ? "contract_dgrad" : "contract_wgrad";
  if (std::min(g.M, g.K) <= 8) {
    const int MT = g.M <= 8 ? pow2_at_least(g.M) : 8;
    g.items_n = (g.N + 63) / 64;
    const long items = (long)((g.M + MT - 1) / MT) * g.items_n;
    if (items > 2147483647L / 4) return BL_ERR_UNSUPPORTED;
    g.items = (int)items;
    g.ks = g.K >= 64 ? 4 : 1;
    const dim3 grid((unsigned)(g.ks == 4 ? items : (items + 3) / 4), (unsigned)B);
    auto go = [&](auto kern, auto* a, auto* b) {
      return timed_launch(name, bytes, flops, s, [&](hipEvent_t e0, hipEvent_t e1) {
        hipExtLaunchKernelGGL(kern, grid, dim3(256), 0, s, e0, e1, 0, a, b, O, g);
      });
    };
#define BL_THIN_C(mt)                                                                                        \
  if (MT == mt)                                                                                              \
    return p->bf16 ? (conj ? go(k_thin_cols<mt, true, unsigned>, A16, B16)                                   \
                           : go(k_thin_cols<mt, false, unsigned>, A16, B16))                                 \
                   : (conj ? go(k_thin_cols<mt, true, float2>, A32, B32) : go(k_thin_cols<mt, false, float2>, A32, B32));
    BL_THIN_C(1) BL_THIN_C(2) BL_THIN_C(4) BL_THIN_C(8)
#undef BL_THIN_C
    return BL_ERR_UNSUPPORTED;
  }
  if (g.N <= 8) {
    const int NT = pow2_at_least(g.N);
    const dim3 grid((unsigned)((g.M + 3) / 4), (unsigned)B);
    auto go = [&](auto kern, auto* a, auto* b) {
      return timed_launch(name, bytes, flops, s, [&](hipEvent_t e0, hipEvent_t e1) {
        hipExtLaunchKernelGGL(kern, grid, dim3(256), 0, s, e0, e1, 0, a, b, O, g);
      });
    };
#define BL_THIN_R(nt)                                                                                        \
  if (NT == nt)                                                                                              \
    return p->bf16 ? (conj ? go(k_thin_rows<nt, true, unsigned>, A16, B16)                                   \
                           : go(k_thin_rows<nt, false, unsigned>, A16, B16))                                 \
                   : (conj ? go(k_thin_rows<nt, true, float2>, A32, B32) : go(k_thin_rows<nt, false, float2>, A32, B32));
    BL_THIN_R(1) BL_THIN_R(2) BL_THIN_R(4) BL_THIN_R(8)
#undef BL_THIN_R
  }
  return BL_ERR_UNSUPPORTED;
}

}  // namespace blc
