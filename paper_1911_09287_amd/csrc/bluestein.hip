// 1-D kept spectra by Bluestein's chirp-z identity (gfx950).
//
// A length-L DFT evaluated only at n_out consecutive outputs from n_in
// consecutive inputs is a linear convolution with a chirp: with
// c[m] = exp(-i pi m^2 / L) and nk = (n^2 + k^2 - (k - n)^2) / 2,
//   sum_n a[n] exp(-2 pi i n k / L) = c[k] sum_n (a[n] c[n]) conj(c[k - n]).
// The convolution is done as a circular one over a power-of-two FFT of size
// M >= n_in + n_out - 1, so no wrap-around reaches the kept outputs.  This
// serves any sequence length (the FCN layers of the time-series experiments
// use 519 = 3 * 173, 516 and 514 = 2 * 257 points, where a mixed-radix FFT
// would need 173- and 257-point stages).
//
// Forward (real rows -> kept bins, Sec. 3.2.2: only v <= r_w is produced):
//   pre[j] = c[j + oj], filter[d] = conj(c[d - oj]), X[v] = c[v] * conv[v].
// Inverse (kept bins -> real rows, Hermitian weights h_v, crop offset cj):
//   pre[v] = h_v conj(c[v]), filter[d] = c[d + cj],
//   y[j] = Re(conj(c[j + cj]) * conv[j]) / L.
// Series are taken in groups of 16 consecutive ones (so each 128-byte line of
// the bin-major spectrum is written by one block); each wave runs its
// series' two M-point FFTs as radix-16/8/4 Stockham passes through its own
// LDS buffer, the first pass reading HBM directly and the last one writing
// HBM directly.  Blocks are persistent; the chirp filter's spectrum is
// computed once per block by all its threads.
#include <algorithm>
#include <cmath>
#include <mutex>
#include <new>
#include <vector>

#include "common.hpp"

namespace blc {
namespace {

// e^{-2 pi i k / 32}, k < 16.
constexpr float kW32c[16] = {1.0f, 0.98078528040323043f, 0.92387953251128674f, 0.83146961230254524f,
                             0.70710678118654757f, 0.55557023301960218f, 0.38268343236508984f, 0.19509032201612833f,
                             0.0f, -0.19509032201612819f, -0.38268343236508973f, -0.55557023301960196f,
                             -0.70710678118654746f, -0.83146961230254535f, -0.92387953251128674f,
                             -0.98078528040323043f};
constexpr float kW32s[16] = {0.0f, -0.19509032201612825f, -0.38268343236508978f, -0.55557023301960218f,
                             -0.70710678118654746f, -0.83146961230254524f, -0.92387953251128674f,
                             -0.98078528040323043f, -1.0f, -0.98078528040323043f, -0.92387953251128674f,
                             -0.83146961230254546f, -0.70710678118654757f, -0.55557023301960218f,
                             -0.38268343236508989f, -0.19509032201612861f};

// In-register R-point DFT (natural order in and out), radix-2 decimation in
// time, R <= 32.  A butterfly with a general twiddle w forms e + w o with four
// fused multiply-adds and takes the difference as 2 e - (e + w o), one more
// each (6 instructions instead of 4 for w o and 4 for the sum and difference).
template <int R>
struct RegFft {
  static __device__ __forceinline__ void run(float2* v) {
    float2 e[R / 2], o[R / 2];
#pragma unroll
    for (int k = 0; k < R / 2; ++k) {
      e[k] = v[2 * k];
      o[k] = v[2 * k + 1];
    }
    RegFft<R / 2>::run(e);
    RegFft<R / 2>::run(o);
#pragma unroll
    for (int k = 0; k < R / 2; ++k) {
      if (k == 0) {
        v[k] = cadd(e[k], o[k]);
        v[k + R / 2] = csub(e[k], o[k]);
      } else if (4 * k == R) {  // w = -i
        v[k] = make_float2(e[k].x + o[k].y, e[k].y - o[k].x);
        v[k + R / 2] = make_float2(e[k].x - o[k].y, e[k].y + o[k].x);
      } else {
        const float c = kW32c[k * (32 / R)], sn = kW32s[k * (32 / R)];
        const float2 x = make_float2(fmaf(o[k].x, c, fmaf(-o[k].y, sn, e[k].x)),
                                     fmaf(o[k].x, sn, fmaf(o[k].y, c, e[k].y)));
        v[k] = x;
        v[k + R / 2] = make_float2(fmaf(2.f, e[k].x, -x.x), fmaf(2.f, e[k].y, -x.y));
      }
    }
  }
};
template <>
struct RegFft<1> {
  static __device__ __forceinline__ void run(float2*) {}
};

// LDS index with one pad slot per 16 elements (spreads strided accesses over banks).
__device__ __forceinline__ int pidx(int n) { return n + (n >> 4); }
template <int M>
constexpr int padded() { return M + M / 16; }

// One Stockham autosort pass of radix R over M points, done by one wave (lane
// = 0..63) or by a whole block (NT threads; then it synchronises the block).
// load(i) returns element i of the input sequence and store(i, v) takes
// element i of the output sequence, so the first pass can read HBM and the
// last pass can write anywhere; in between the data stay in LDS.
// Twiddles: with `tw` set, tw[k * (R - 1) + r - 1] = w_{Ns R}^{r k} (a per-pass
// table whose rows are read with an odd stride, free of bank conflicts);
// otherwise roots[r k M / (Ns R)] of the M-point root table.
template <int M, int R, int NT, class LoadF, class StoreF>
__device__ __forceinline__ void stockham_pass(int Ns, int t, const float2* roots, const float2* tw, LoadF&& load,
                                              StoreF&& store) {
  constexpr int NB = M / R;
  constexpr int PER = NB >= NT ? NB / NT : 1;
  const bool active = NB >= NT || t < NB;
  float2 v[PER][R];
  if (active) {
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int j = t + q * NT;
#pragma unroll
      for (int r = 0; r < R; ++r) v[q][r] = load(j + r * NB);
    }
  }
  if constexpr (NT == 64) wave_sync(); else __syncthreads();
  if (active) {
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int j = t + q * NT;
      const int k = j & (Ns - 1);
      if (Ns > 1) {
        if (tw) {
#pragma unroll
          for (int r = 1; r < R; ++r) v[q][r] = cmul(v[q][r], tw[k * (R - 1) + r - 1]);
        } else {
          const int step = M / (Ns * R);
#pragma unroll
          for (int r = 1; r < R; ++r) v[q][r] = cmul(v[q][r], roots[r * k * step]);
        }
      }
      RegFft<R>::run(v[q]);
      const int base = (j - k) * R + k;
#pragma unroll
      for (int r = 0; r < R; ++r) store(base + r * Ns, v[q][r]);
    }
  }
  if constexpr (NT == 64) wave_sync(); else __syncthreads();
}

// Radix sequence of the per-wave FFTs: M = 512: 8, 8, 8; 256: 4, 4, 4, 4.
// Pass p has span Ns_p = product of the earlier radices.  (M = 1024 has a
// kernel of its own.)
template <int M>
struct WavePlan;
template <>
struct WavePlan<512> {
  static constexpr int n = 3;
  static constexpr int R[3] = {8, 8, 8};
};
template <>
struct WavePlan<256> {
  static constexpr int n = 4;
  static constexpr int R[4] = {4, 4, 4, 4};
};

// Offset of pass p's twiddle table inside the packed per-pass tables (passes
// with Ns > 1 only; sum of Ns (R - 1) over them is M - R_0 < M).
template <int M>
constexpr int tw_offset(int p) {
  int off = 0, Ns = 1;
  for (int i = 0; i < p; ++i) {
    if (Ns > 1) off += Ns * (WavePlan<M>::R[i] - 1);
    Ns *= WavePlan<M>::R[i];
  }
  return off;
}
template <int M>
constexpr int span(int p) {
  int Ns = 1;
  for (int i = 0; i < p; ++i) Ns *= WavePlan<M>::R[i];
  return Ns;
}

// Build the packed per-pass twiddle tables of the wave FFT into `tw`.
template <int M>
__device__ __forceinline__ void build_pass_twiddles(float2* tw, const float2* roots, int t, int nt) {
#pragma unroll
  for (int p = 1; p < WavePlan<M>::n; ++p) {
    const int R = WavePlan<M>::R[p], Ns = span<M>(p), off = tw_offset<M>(p);
    for (int e = t; e < Ns * (R - 1); e += nt) {
      const int k = e / (R - 1), r = e % (R - 1) + 1;
      tw[off + e] = roots[r * k * (M / (Ns * R))];
    }
  }
}

// Forward M-point FFT by one wave: the first pass reads through load0, the
// last pass writes through storeN, the passes in between use `buf` (padded).
template <int M, class L0, class SN>
__device__ __forceinline__ void wave_fft(float2* buf, int lane, const float2* tw, L0&& load0, SN&& storeN) {
  auto lb = [buf](int i) { return buf[pidx(i)]; };
  auto sb = [buf](int i, float2 v) { buf[pidx(i)] = v; };
  using WP = WavePlan<M>;
  if constexpr (WP::n == 3) {
    stockham_pass<M, WP::R[0], 64>(1, lane, nullptr, nullptr, load0, sb);
    stockham_pass<M, WP::R[1], 64>(span<M>(1), lane, nullptr, tw + tw_offset<M>(1), lb, sb);
    stockham_pass<M, WP::R[2], 64>(span<M>(2), lane, nullptr, tw + tw_offset<M>(2), lb, storeN);
  } else {
    stockham_pass<M, WP::R[0], 64>(1, lane, nullptr, nullptr, load0, sb);
    stockham_pass<M, WP::R[1], 64>(span<M>(1), lane, nullptr, tw + tw_offset<M>(1), lb, sb);
    stockham_pass<M, WP::R[2], 64>(span<M>(2), lane, nullptr, tw + tw_offset<M>(2), lb, sb);
    stockham_pass<M, WP::R[3], 64>(span<M>(3), lane, nullptr, tw + tw_offset<M>(3), lb, storeN);
  }
}

// Forward M-point FFT in place in `buf` by the whole block (NT threads).
template <int M, int NT>
__device__ __forceinline__ void block_fft(float2* buf, int t, const float2* roots) {
  auto lb = [buf](int i) { return buf[pidx(i)]; };
  auto sb = [buf](int i, float2 v) { buf[pidx(i)] = v; };
  int Ns = 1;
  for (; Ns * 4 <= M; Ns *= 4) stockham_pass<M, 4, NT>(Ns, t, roots, nullptr, lb, sb);
  if (Ns < M) stockham_pass<M, 2, NT>(Ns, t, roots, nullptr, lb, sb);
}

struct BlueGeom {
  int n_in, n_out;     // inputs and outputs of the chirp convolution per FFT
  int L;               // DFT length
  int V;               // kept bins per series
  int off_in, off_out; // DFT index of input 0 and of output 0
  int nyq;             // Nyquist bin (L even) or -1
  long P;              // number of series
  float out_scale;     // extra output scale (inverse: 1 / L)
  const float2* tab;   // 1024-point kernel: [pre n_in][post n_out][F 1024][TW 1024]
};
struct BlueArgs : BlueGeom {
  float2 root_hi[16], root_lo[64];    // e^{-2 pi i k / M} = hi[k >> 6] * lo[k & 63]
  float2 chirp_hi[64], chirp_lo[64];  // e^{-i pi q / L} = hi[q >> 6] * lo[q & 63], q < 2L
};

constexpr int kSeriesPerGroup = 16;
constexpr int kWaves = 4;

// c[m] = e^{-i pi m^2 / L} (m^2 reduced mod 2L exactly), conjugated for the inverse.
template <bool INV>
__device__ __forceinline__ float2 chirp(const BlueArgs& a, int m) {
  const unsigned mm = (unsigned)(m < 0 ? -m : m);
  const int q = (int)((mm * mm) % (2u * (unsigned)a.L));
  const float2 c = cmul(a.chirp_hi[q >> 6], a.chirp_lo[q & 63]);
  return INV ? cconj(c) : c;
}

// Modes: bit 0 = inverse (bins -> real rows), bit 1 = two series per FFT.
//   forward, single:  inputs x[0..Win), outputs X[0..V)
//   inverse, single:  inputs h_v Y[v], v < V; outputs y[0..OW)
//   forward, paired:  input x1 + i x2; outputs Z[k], k = -(V-1)..V-1, then
//                     X1 = (Z[k] + conj Z[-k]) / 2, X2 = (Z[k] - conj Z[-k]) / 2i
//                     (both spectra of real rows are conjugate-symmetric)
//   inverse, paired:  input the conjugate-symmetric extensions of Y1 and Y2
//                     over k = -(V-1)..V-1 as Y1 + i Y2 (real DC parts); the
//                     real and imaginary parts of the result are y1 and y2.
// S: stored-spectrum element of the forward modes' output (float2 or bfloat16 pairs)
template <int M, int MODE, typename S = float2>
__global__ __launch_bounds__(64 * kWaves) void k_bluestein(const void* __restrict__ in_, void* __restrict__ out_,
                                                           BlueArgs a) {
  constexpr bool INV = MODE & 1, PACK = MODE >= 2;
  extern __shared__ float2 sm[];
  constexpr int PM = padded<M>();
  float2* tw = sm;                // M: packed per-pass twiddle tables
  float2* F = tw + M;             // PM: spectrum of the chirp filter
  float2* pre = F + PM;           // n_in
  float2* post = pre + a.n_in;    // n_out
  float2* bufs = post + a.n_out;  // kWaves x PM: per-wave FFT buffers
  float2* roots = bufs;           // M: e^{-2 pi i k / M}, only while the tables are built
  const int tid = threadIdx.x;

  for (int k = tid; k < M; k += blockDim.x) roots[k] = cmul(a.root_hi[k >> 6], a.root_lo[k & 63]);
  for (int k = tid; k < a.n_in; k += blockDim.x) {
    float2 c = chirp<INV>(a, k + a.off_in);
    if (INV && !PACK && k != 0 && k != a.nyq) c = cscale(c, 2.f);
    pre[k] = c;
  }
  const float osc = a.out_scale / (float)M * (PACK && !INV ? 0.5f : 1.0f);
  for (int k = tid; k < a.n_out; k += blockDim.x) post[k] = cscale(chirp<INV>(a, k + a.off_out), osc);
  for (int m = tid; m < M; m += blockDim.x) {
    const int d = m < a.n_out ? m : m - M;
    float2 h = make_float2(0.f, 0.f);
    if (d >= -(a.n_in - 1)) h = cconj(chirp<INV>(a, d + a.off_out - a.off_in));
    F[pidx(m)] = h;
  }
  __syncthreads();
  build_pass_twiddles<M>(tw, roots, tid, blockDim.x);
  block_fft<M, 64 * kWaves>(F, tid, roots);  // ends with a block barrier: roots are free again

  const int wave = tid >> 6, lane = tid & 63;
  float2* buf = bufs + wave * PM;
  const float* xin = static_cast<const float*>(in_);
  const float2* yin = static_cast<const float2*>(in_);
  const long P = a.P;
  const long groups = (P + kSeriesPerGroup - 1) / kSeriesPerGroup;
  constexpr int SPF = PACK ? 2 : 1;  // series per FFT
  for (long g = blockIdx.x; g < groups; g += gridDim.x) {
    for (int sl = wave * SPF; sl < kSeriesPerGroup; sl += kWaves * SPF) {
      const long s1 = g * kSeriesPerGroup + sl;
      if (s1 >= P) break;
      const long s2 = s1 + 1;
      const bool two = PACK && s2 < P;
      // FFT of the pre-chirped input, straight from HBM; the last pass
      // multiplies by the filter spectrum and conjugates (inverse via conj).
      auto load_in = [&](int n) {
        float2 v = make_float2(0.f, 0.f);
        if (n < a.n_in) {
          if constexpr (MODE == 0) {
            v = make_float2(xin[(size_t)s1 * a.n_in + n], 0.f);
          } else if constexpr (MODE == 1) {
            v = yin[(size_t)n * P + s1];
          } else if constexpr (MODE == 2) {
            v = make_float2(xin[(size_t)s1 * a.n_in + n], two ? xin[(size_t)s2 * a.n_in + n] : 0.f);
          } else {
            const int k = n - (a.V - 1);
            const int kk = k < 0 ? -k : k;
            const float2 y1 = yin[(size_t)kk * P + s1];
            const float2 y2 = two ? yin[(size_t)kk * P + s2] : make_float2(0.f, 0.f);
            if (k > 0) v = make_float2(y1.x - y2.y, y1.y + y2.x);
            else if (k < 0) v = make_float2(y1.x + y2.y, y2.x - y1.y);
            else v = make_float2(y1.x, y2.x);
          }
          v = cmul(v, pre[n]);
        }
        return v;
      };
      auto store_prod = [&](int i, float2 v) { buf[pidx(i)] = cconj(cmul(v, F[pidx(i)])); };
      wave_fft<M>(buf, lane, tw, load_in, store_prod);
      // second FFT; its last pass writes the outputs with the post chirp
      auto load_buf = [&](int i) { return buf[pidx(i)]; };
      auto store_out = [&](int i, float2 v) {
        if (i < a.n_out) {
          const float2 r = cmul(post[i], cconj(v));
          if constexpr (MODE == 0) {
            spec_put(static_cast<S*>(out_), (size_t)i * P + s1, r);
          } else if constexpr (MODE == 1) {
            static_cast<float*>(out_)[(size_t)s1 * a.n_out + i] = r.x;
          } else if constexpr (MODE == 2) {
            buf[pidx(i)] = r;  // split below
          } else {
            static_cast<float*>(out_)[(size_t)s1 * a.n_out + i] = r.x;
            if (two) static_cast<float*>(out_)[(size_t)s2 * a.n_out + i] = r.y;
          }
        }
      };
      wave_fft<M>(buf, lane, tw, load_buf, store_out);
      if constexpr (MODE == 2) {
        // Z[k] sits at index k + V - 1
        S* X = static_cast<S*>(out_);
        for (int v = lane; v < a.V; v += 64) {
          const float2 zp = buf[pidx(a.V - 1 + v)];
          const float2 zm = cconj(buf[pidx(a.V - 1 - v)]);
          spec_put(X, (size_t)v * P + s1, cadd(zp, zm));
          if (two) {
            const float2 d = csub(zp, zm);
            spec_put(X, (size_t)v * P + s2, make_float2(d.y, -d.x));
          }
        }
        wave_sync();
      }
    }
  }
}

// ---------------------------------------------------------------------------
// M = 1024 as 32 x 32 per half-wave: with n = l + 32 j and k' = k + 32 m,
//   X[k + 32 m] = sum_l w32^{lm} [w1024^{lk} sum_j x[l + 32 j] w32^{jk}],
// lane l of a half-wave runs the inner 32-point FFT over j in registers, the
// twiddled results cross lanes once through LDS (a 32 x 33 transpose), and
// lane k runs the outer 32-point FFT over l, ending with X[k + 32 m] in its
// registers.  That is exactly the layout the second FFT's inner pass needs
// (lane k holding element k + 32 m), so the pointwise product with the filter
// spectrum needs no extra transpose: each Bluestein job costs one LDS
// transpose per FFT instead of a pass per radix stage.
//
// Every wave runs its own jobs, with no block barrier once the tables are in
// LDS: half-wave q of the wave with grid-wide index p takes job 2 p + q, then
// job 2 (p + W) + q for W waves in the grid, and so on.  A wave's jobs are two
// consecutive series (four in the paired modes), and the waves of a block
// hold consecutive jobs, so the rows of a bin-major spectrum are read and
// written in runs of consecutive series that meet in the L2.  A wave loads its
// inputs (the next round's while it transforms the current one, when they fit
// in 32 registers per lane), transforms and stores, and the waves of a CU fall
// into different phases, overlapping memory traffic with arithmetic.
// Inputs and outputs that run along the series (real samples) move straight
// between HBM and registers; bin-major spectra pass through the wave's slot
// buffers in LDS, where the conjugate-symmetric pairs of the paired modes are
// formed or split.
// ---------------------------------------------------------------------------
constexpr int kWaves1k = 8;
// Slot stride (complex): the 32 x 33 transpose tile plus 4 elements.
constexpr int kXS = 32 * 33 + 4;

// Rows of input one lane loads per round (NR, a compile-time bound; loads past
// the data are clamped to its last row and their values unused):
//   MODE 0, 2: rows j of the series, element h + 32 j;
//   MODE 1, 3: bins k = lane / 2 + 32 t, t < NR.
// Floats per row: 1 (MODE 0), 2 (MODE 1, 2), 4 (MODE 3).  The next round is
// prefetched when NR rows take at most 32 floats.
template <int MODE>
constexpr int floats_per_row() {
  return MODE == 0 ? 1 : MODE == 3 ? 4 : 2;
}

template <int MODE, int NR, typename S = float2>
__global__ __launch_bounds__(64 * kWaves1k) void k_bluestein1k(const void* __restrict__ in_, void* __restrict__ out_,
                                                               BlueGeom a, int wpb) {
  constexpr int M = 1024;
  constexpr bool PACK = MODE >= 2;
  constexpr int FPR = floats_per_row<MODE>();
  constexpr bool PREF = NR * FPR <= 32;
  extern __shared__ float2 sm[];
  float2* bufs = sm;                          // 16 slots x kXS
  float2* pre = bufs + 2 * kWaves1k * kXS;    // n_in
  float2* post = pre + a.n_in;                // n_out
  float2* F = post + a.n_out;                 // spectrum of the chirp filter (M)
  float2* TW = F + M;                         // TW[32 k + h] = w1024^{h k}
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q = lane >> 5, h = lane & 31;
  float2* xw = bufs + wave * 2 * kXS;  // the wave's two slot buffers
  float2* xb = xw + q * kXS;           // this half-wave's

  // the chirps, the filter's spectrum and the twiddles, built once per plan
  // in double precision on the host, are laid out in the table as in LDS
  // (all of a thread's table loads in flight together, and with the first
  // round's input loads: n_in + n_out <= M + 1)
  constexpr int NT = 64 * kWaves1k;
  constexpr int NTAB = (3 * M + 1 + NT - 1) / NT;
  const int ntab = a.n_in + a.n_out + 2 * M;
  float2 tv[NTAB];
#pragma unroll
  for (int u = 0; u < NTAB; ++u) tv[u] = a.tab[min(tid + NT * u, ntab - 1)];

  auto exchange = [&](float2* v) {
#pragma unroll
    for (int k = 0; k < 32; ++k) xb[k * 33 + h] = v[k];
    wave_sync();
#pragma unroll
    for (int l = 0; l < 32; ++l) v[l] = xb[h * 33 + l];
    wave_sync();
  };
  // inner FFT over j (input v[j] = element h + 32 j), twiddle, transpose, outer FFT:
  // leaves v[m] = element h + 32 m of the transform.
  auto fft1k = [&](float2* v) {
    RegFft<32>::run(v);
#pragma unroll
    for (int k = 1; k < 32; ++k) v[k] = cmul(v[k], TW[32 * k + h]);
    exchange(v);
    RegFft<32>::run(v);
  };

  // element indices fit in 32 bits (checked on the host)
  const float* xin = static_cast<const float*>(in_);
  const float2* yin = static_cast<const float2*>(in_);
  const unsigned P = (unsigned)a.P;
  const unsigned jobs = PACK ? (P + 1) / 2 : P;
  const unsigned pairs = (jobs + 1) / 2;  // rounds of the grid's waves: one job pair each
  // waves past the first wpb of a block only help with the tables
  const unsigned nw = gridDim.x * (unsigned)wpb;
  const unsigned p0 = wave < wpb ? blockIdx.x * (unsigned)wpb + wave : pairs;
  // series of the wave in round p: MODE 0/1: 2p + q; MODE 2/3: 4p .. 4p + 3
  float pf[PREF ? NR * FPR : 1];
  float2 v[32];
  auto load = [&](unsigned p, float* dst) {
    if constexpr (MODE == 0) {
      const unsigned s = min(2 * p + q, P - 1);
#pragma unroll
      for (int j = 0; j < NR; ++j) dst[j] = xin[s * (unsigned)a.n_in + min(h + 32 * j, a.n_in - 1)];
    } else if constexpr (MODE == 2) {
      const unsigned s1 = min(4 * p + 2 * q, P - 1), s2 = min(4 * p + 2 * q + 1, P - 1);
#pragma unroll
      for (int j = 0; j < NR; ++j) {
        const int n = min(h + 32 * j, a.n_in - 1);
        dst[2 * j] = xin[s1 * (unsigned)a.n_in + n];
        dst[2 * j + 1] = xin[s2 * (unsigned)a.n_in + n];
      }
    } else if constexpr (MODE == 1) {
      const unsigned s = min(2 * p + (lane & 1), P - 1);
#pragma unroll
      for (int t = 0; t < NR; ++t) {
        const float2 y = yin[(unsigned)min((lane >> 1) + 32 * t, a.V - 1) * P + s];
        dst[2 * t] = y.x;
        dst[2 * t + 1] = y.y;
      }
    } else {
      const unsigned s1 = min(4 * p + 2 * (lane & 1), P - 1), s2 = min(4 * p + 2 * (lane & 1) + 1, P - 1);
#pragma unroll
      for (int t = 0; t < NR; ++t) {
        const unsigned k = (unsigned)min((lane >> 1) + 32 * t, a.V - 1);
        const float2 y1 = yin[k * P + s1], y2 = yin[k * P + s2];
        dst[4 * t] = y1.x;
        dst[4 * t + 1] = y1.y;
        dst[4 * t + 2] = y2.x;
        dst[4 * t + 3] = y2.y;
      }
    }
  };
  // loaded rows -> v (element h + 32 j of this half-wave's job), times the pre-chirp
  auto stage = [&](unsigned p, const float* src) {
    if constexpr (MODE == 0 || MODE == 2) {
      const bool two = MODE == 2 && 4 * p + 2 * q + 1 < P;
      const int jfull = a.n_in >> 5;  // rows complete for every lane (uniform branch)
      const bool tail = h < (a.n_in & 31);
#pragma unroll
      for (int j = 0; j < 32; ++j) {
        v[j] = make_float2(0.f, 0.f);
        if (j < NR && (j < jfull || (j == jfull && tail))) {
          const float2 z = MODE == 0 ? make_float2(src[j], 0.f) : make_float2(src[2 * j], two ? src[2 * j + 1] : 0.f);
          v[j] = cmul(z, pre[h + 32 * j]);
        }
      }
    } else {
      float2* dst = xw + (lane & 1) * kXS;
#pragma unroll
      for (int t = 0; t < NR; ++t) {
        const int k = (lane >> 1) + 32 * t;
        if (k < a.V) {
          if constexpr (MODE == 1) {
            dst[k] = cmul(make_float2(src[2 * t], src[2 * t + 1]), pre[k]);
          } else {
            // two Hermitian spectra packed into one series: Z[k] = Y1[k] + i Y2[k]
            // at index k + V - 1 for |k| < V, with Y[-k] = conj(Y[k])
            const bool two = 4 * p + 2 * (lane & 1) + 1 < P;
            const float2 y1 = make_float2(src[4 * t], src[4 * t + 1]);
            const float2 y2 = two ? make_float2(src[4 * t + 2], src[4 * t + 3]) : make_float2(0.f, 0.f);
            const int ip = a.V - 1 + k, im = a.V - 1 - k;
            if (k == 0) {
              dst[ip] = cmul(make_float2(y1.x, y2.x), pre[ip]);
            } else {
              dst[ip] = cmul(make_float2(y1.x - y2.y, y1.y + y2.x), pre[ip]);
              dst[im] = cmul(make_float2(y1.x + y2.y, y2.x - y1.y), pre[im]);
            }
          }
        }
      }
      wave_sync();
#pragma unroll
      for (int j = 0; j < 32; ++j) {
        const int n = h + 32 * j;
        v[j] = n < a.n_in ? xb[n] : make_float2(0.f, 0.f);
      }
      wave_sync();
    }
  };

  if constexpr (PREF) load(min(p0, pairs - 1), pf);  // clamped: no branch between these loads and the table's
  // (indices past the table are clamped like the loads: those threads store
  // the last entry's own value again, so the stores need no branch)
#pragma unroll
  for (int u = 0; u < NTAB; ++u) pre[min(tid + NT * u, ntab - 1)] = tv[u];
  __syncthreads();  // tables in LDS; no block barrier follows

  for (unsigned p = p0; p < pairs; p += nw) {
    if constexpr (PREF) {
      stage(p, pf);
      load(p + nw < pairs ? p + nw : p, pf);  // the last round reloads its own rows (cache hits)
    } else {
      float ld[NR * FPR];
      load(p, ld);
      stage(p, ld);
    }
    fft1k(v);
    // inverse FFT of (A * F) as conj(FFT(conj(A * F)))
#pragma unroll
    for (int m = 0; m < 32; ++m) v[m] = cconj(cmul(v[m], F[h + 32 * m]));
    fft1k(v);
    // v[m] -> output element i = h + 32 m: post[i] conj(v[m])
    // rows m < nfull are complete for every lane (a uniform branch); row
    // nfull is partial
    const int nfull = a.n_out >> 5;
    const bool tail = h < (a.n_out & 31);
    if constexpr (MODE == 1) {
      const unsigned s = 2 * p + q;
      if (s < P) {
        float* dst = static_cast<float*>(out_) + s * (unsigned)a.n_out + h;
#pragma unroll
        for (int m = 0; m < 32; ++m) {
          if (m < nfull || (m == nfull && tail)) dst[32 * m] = cmul(post[h + 32 * m], cconj(v[m])).x;
        }
      }
    } else if constexpr (MODE == 3) {
      const unsigned s1 = 4 * p + 2 * q;
      const bool two = s1 + 1 < P;
      float* d1 = static_cast<float*>(out_) + s1 * (unsigned)a.n_out + h;
      float* d2 = d1 + a.n_out;
      if (two) {
#pragma unroll
        for (int m = 0; m < 32; ++m) {
          if (m < nfull || (m == nfull && tail)) {
            const float2 r = cmul(post[h + 32 * m], cconj(v[m]));
            d1[32 * m] = r.x;
            d2[32 * m] = r.y;
          }
        }
      } else if (s1 < P) {  // a lone last series
#pragma unroll
        for (int m = 0; m < 32; ++m) {
          if (m < nfull || (m == nfull && tail)) d1[32 * m] = cmul(post[h + 32 * m], cconj(v[m])).x;
        }
      }
    } else {
#pragma unroll
      for (int m = 0; m < 32; ++m) {
        if (m < nfull || (m == nfull && tail)) xb[h + 32 * m] = cmul(post[h + 32 * m], cconj(v[m]));
      }
      wave_sync();
      S* X = static_cast<S*>(out_);
      if constexpr (MODE == 0) {
        // bins i of the wave's two series, two consecutive series per bin row
        const unsigned s = 2 * p + (lane & 1);
        const float2* src = xw + (lane & 1) * kXS;
        if (s < P) {
          for (int i = lane >> 1; i < a.n_out; i += 32) spec_put(X, (unsigned)i * P + s, src[i]);
        }
      } else {
        // Z[k] sits at index k + V - 1; the two series of a job split by
        // conjugate symmetry; four consecutive series per bin row
        const unsigned s = 4 * p + (lane & 3);
        const float2* src = xw + ((lane >> 1) & 1) * kXS + (a.V - 1);
        if (s < P) {
          for (int k = lane >> 2; k < a.V; k += 16) {
            const float2 zp = src[k], zm = cconj(src[-k]);
            spec_put(X, (unsigned)k * P + s, (lane & 1) ? make_float2(zp.y - zm.y, zm.x - zp.x) : cadd(zp, zm));
          }
        }
      }
      wave_sync();  // slot buffers free for the next round's transposes
    }
  }
}

template <int M, int MODE, typename S>
bl_status_t launch_m(BlueArgs& a, const void* in, void* out, const char* name, double bytes, hipStream_t s) {
  // algorithmic arithmetic: two M-point complex FFTs (5 M log2 M flops each, the
  // conventional count) per series, or per pair of series when two share an FFT
  const double ffts = (MODE >= 2) ? (double)((a.P + 1) / 2) : (double)a.P;
  double lg = 0;
  for (int m = M; m > 1; m >>= 1) lg += 1;
  const double flops = ffts * 2.0 * 5.0 * M * lg;
  // host-side seeds of the root and chirp tables, in double precision
  for (int i = 0; i < M / 64; ++i) {
    const double t = -2.0 * M_PI * 64.0 * i / M;
    a.root_hi[i] = make_float2((float)std::cos(t), (float)std::sin(t));
  }
  for (int i = 0; i < 64; ++i) {
    const double t = -2.0 * M_PI * i / M;
    a.root_lo[i] = make_float2((float)std::cos(t), (float)std::sin(t));
  }
  for (int i = 0; i * 64 < 2 * a.L; ++i) {
    const double t = -M_PI * 64.0 * i / a.L;
    a.chirp_hi[i] = make_float2((float)std::cos(t), (float)std::sin(t));
  }
  for (int i = 0; i < 64; ++i) {
    const double t = -M_PI * i / a.L;
    a.chirp_lo[i] = make_float2((float)std::cos(t), (float)std::sin(t));
  }
  const size_t lds = (size_t)(M + (1 + kWaves) * padded<M>() + a.n_in + a.n_out) * sizeof(float2);
  if (lds > kMaxLds) return BL_ERR_UNSUPPORTED;
  const long groups = (a.P + kSeriesPerGroup - 1) / kSeriesPerGroup;
  const long blocks = std::min<long>(groups, 2L * device_cus());
  return timed_launch(name, bytes, flops, s, [&](hipEvent_t e0, hipEvent_t e1) {
    hipExtLaunchKernelGGL((k_bluestein<M, MODE, S>), dim3((unsigned)blocks), dim3(64 * kWaves), lds, s, e0, e1, 0, in, out, a);
  });
}

// ---- tables of the 1024-point kernel, built on the host in double precision ----
// For one transform geometry: pre[n] (n < n_in), post[k] (k < n_out), the
// spectrum F of the chirp filter, and the twiddles TW[32 k + h] = w^{h k}, in
// that order, as the kernel lays them out in LDS.
void host_tables_1k(const BlueGeom& a, int mode, std::vector<float2>& out) {
  constexpr int M = 1024;
  const bool inv = mode & 1, pack = mode >= 2;
  const double pi = 3.141592653589793238462643383279502884;
  auto chirp = [&](long m, double& re, double& im) {  // e^{-i pi m^2 / L}, conjugated for the inverse
    const long mm = m < 0 ? -m : m;
    const long q = (mm * mm) % (2L * a.L);
    re = std::cos(pi * (double)q / a.L);
    im = -std::sin(pi * (double)q / a.L);
    if (inv) im = -im;
  };
  out.assign((size_t)a.n_in + a.n_out + 2 * M, make_float2(0.f, 0.f));
  double re, im;
  for (int k = 0; k < a.n_in; ++k) {
    chirp(k + a.off_in, re, im);
    const double w = (inv && !pack && k != 0 && k != a.nyq) ? 2.0 : 1.0;
    out[k] = make_float2((float)(w * re), (float)(w * im));
  }
  const double osc = (double)a.out_scale / M * (pack && !inv ? 0.5 : 1.0);
  for (int k = 0; k < a.n_out; ++k) {
    chirp(k + a.off_out, re, im);
    out[a.n_in + k] = make_float2((float)(osc * re), (float)(osc * im));
  }
  // filter b[m] = conj(c[d + off_out - off_in]) for lags d in (-n_in, n_out),
  // d = m or m - M; its M-point DFT by iterative radix-2 in double
  std::vector<double> br(M, 0.0), bi(M, 0.0);
  for (int m = 0; m < M; ++m) {
    const int d = m < a.n_out ? m : m - M;
    if (d >= -(a.n_in - 1)) {
      chirp((long)d + a.off_out - a.off_in, re, im);
      br[m] = re;
      bi[m] = -im;
    }
  }
  for (int i = 1, j = 0; i < M; ++i) {  // bit reversal
    int bit = M >> 1;
    for (; j & bit; bit >>= 1) j ^= bit;
    j ^= bit;
    if (i < j) std::swap(br[i], br[j]), std::swap(bi[i], bi[j]);
  }
  for (int len = 2; len <= M; len <<= 1) {
    for (int i = 0; i < M; i += len) {
      for (int k = 0; k < len / 2; ++k) {
        const double t = -2.0 * pi * k / len, wr = std::cos(t), wi = std::sin(t);
        const int u = i + k, v = i + k + len / 2;
        const double xr = br[v] * wr - bi[v] * wi, xi = br[v] * wi + bi[v] * wr;
        br[v] = br[u] - xr; bi[v] = bi[u] - xi;
        br[u] += xr; bi[u] += xi;
      }
    }
  }
  float2* F = out.data() + a.n_in + a.n_out;
  for (int m = 0; m < M; ++m) F[m] = make_float2((float)br[m], (float)bi[m]);
  float2* TW = F + M;
  for (int i = 0; i < M; ++i) {
    const int e = ((i >> 5) * (i & 31)) & (M - 1);
    TW[i] = make_float2((float)std::cos(2.0 * pi * e / M), (float)-std::sin(2.0 * pi * e / M));
  }
}

// Device copy of the tables for this geometry (built and uploaded on first use).
bl_status_t blue_tables(const bl_conv_plan_s* p, const BlueGeom& a, int mode, const float2** out) {
  const std::vector<long> key{1, mode, a.n_in, a.n_out, a.off_in, a.off_out, a.L, a.nyq, float_key(a.out_scale)};
  return plan_table(p, key, [&](std::vector<float2>& host) { host_tables_1k(a, mode, host); }, out);
}

template <int MODE, int NR, typename S>
bl_status_t launch_1k_nr(const BlueGeom& a, const void* in, void* out, const char* name, double bytes,
                         hipStream_t s) {
  constexpr int M = 1024;
  const size_t lds = (size_t)(2 * kWaves1k * kXS + a.n_in + a.n_out + 2 * M) * sizeof(float2);
  if (lds > 160 * 1024) return BL_ERR_UNSUPPORTED;
  const bl_status_t at = lds_opt_in(reinterpret_cast<const void*>(&k_bluestein1k<MODE, NR, S>), 160 * 1024);
  if (at != BL_OK) return at;
  const long jobs = (MODE >= 2) ? (a.P + 1) / 2 : a.P;
  const long pairs = (jobs + 1) / 2;  // one job per half-wave
  // one block per CU at most; when there is less than a full block of work
  // per CU, fewer waves per block, so that the SIMDs are shared by fewer waves
  const long cus = device_cus();
  const int wpb = (int)std::min<long>(kWaves1k, (pairs + cus - 1) / cus);
  const long blocks = std::min<long>(cus, (pairs + wpb - 1) / wpb);
  const double flops = (double)jobs * 2.0 * 5.0 * M * 10.0;
  return timed_launch(name, bytes, flops, s, [&](hipEvent_t e0, hipEvent_t e1) {
    hipExtLaunchKernelGGL((k_bluestein1k<MODE, NR, S>), dim3((unsigned)blocks), dim3(64 * kWaves1k), lds, s, e0, e1, 0,
                          in, out, a, wpb);
  });
}

// NR: rows of input per lane as instantiated (the smallest that covers the
// data); the kernel prefetches the next round when they fit in 32 floats.
template <int MODE, typename S>
bl_status_t launch_1k(const bl_conv_plan_s* p, const BlueGeom& a0, const void* in, void* out, const char* name,
                      double bytes, hipStream_t s) {
  // the kernel indexes its input and output with 32-bit element offsets
  const long rows = std::max<long>({(long)a0.n_in, (long)a0.n_out, 2L * a0.V});
  if (a0.P < 1 || a0.P * rows >= 2147483647L || a0.P * rows < 0) return BL_ERR_UNSUPPORTED;
  BlueGeom a = a0;
  const bl_status_t ts = blue_tables(p, a, MODE, &a.tab);
  if (ts != BL_OK) return ts;
  if constexpr (MODE == 0 || MODE == 2) {
    const int nr = (a.n_in + 31) / 32;
    if (nr <= 16) return launch_1k_nr<MODE, 16, S>(a, in, out, name, bytes, s);
    return launch_1k_nr<MODE, 32, S>(a, in, out, name, bytes, s);
  } else {
    const int nr = (a.V + 31) / 32;
    if (nr <= 4) return launch_1k_nr<MODE, 4, S>(a, in, out, name, bytes, s);
    if (nr <= 8) return launch_1k_nr<MODE, 8, S>(a, in, out, name, bytes, s);
    if (nr <= 16) return launch_1k_nr<MODE, 16, S>(a, in, out, name, bytes, s);
    if constexpr (MODE == 1) return launch_1k_nr<MODE, 32, S>(a, in, out, name, bytes, s);
    return BL_ERR_UNSUPPORTED;
  }
}

int fft_size_for(int need) {
  int M = 256;
  while (M < need) M *= 2;
  return M;
}

// S: the stored-spectrum element the forward modes write (the inverse modes
// read complex64 contraction outputs and take float2)
template <int MODE, typename S = float2>
bl_status_t launch_mode(const bl_conv_plan_s* p, BlueArgs& a, int M, const void* in, void* out, const char* name,
                        double bytes, hipStream_t s) {
  if (M == 256) return launch_m<256, MODE, S>(a, in, out, name, bytes, s);
  if (M == 512) return launch_m<512, MODE, S>(a, in, out, name, bytes, s);
  if (M == 1024) return launch_1k<MODE, S>(p, a, in, out, name, bytes, s);
  return BL_ERR_UNSUPPORTED;
}

// Chooses between one series per FFT and two (when the conjugate-symmetric
// output or input range fits the same FFT size).
bl_status_t launch_any(const bl_conv_plan_s* p, BlueArgs& a, bool inv, int other, const void* in, void* out,
                       const char* name, double bytes, hipStream_t s) {
  if (2 * a.L > 64 * 64) return BL_ERR_UNSUPPORTED;
  if ((long)a.V * other < 2048) return BL_ERR_UNSUPPORTED;  // the direct DFT is as cheap
  const int M1 = fft_size_for(a.V + other - 1);
  const int M2 = fft_size_for(2 * a.V - 1 + other - 1);
  const bool pack = a.P >= 2 && 2 * (a.V - 1) < a.L && M2 <= M1 && M2 <= 1024;
  if (!pack && M1 > 1024) return BL_ERR_UNSUPPORTED;
  if (!inv) {
    a.n_in = other;
    if (pack) {
      a.n_out = 2 * a.V - 1;
      a.off_out = -(a.V - 1);
      return p->bf16 ? launch_mode<2, unsigned>(p, a, M2, in, out, name, bytes, s)
                     : launch_mode<2, float2>(p, a, M2, in, out, name, bytes, s);
    }
    a.n_out = a.V;
    a.off_out = 0;
    return p->bf16 ? launch_mode<0, unsigned>(p, a, M1, in, out, name, bytes, s)
                   : launch_mode<0, float2>(p, a, M1, in, out, name, bytes, s);
  }
  a.n_out = other;
  if (pack) {
    a.n_in = 2 * a.V - 1;
    a.off_in = -(a.V - 1);
    return launch_mode<3>(p, a, M2, in, out, name, bytes, s);
  }
  a.n_in = a.V;
  a.off_in = 0;
  return launch_mode<1>(p, a, M1, in, out, name, bytes, s);
}

}  // namespace

bl_status_t launch_bluestein_fwd(const bl_conv_plan_s* p, const float* in, void* out, long P, int Win, int oj,
                                 hipStream_t s) {
  BlueArgs a{};
  a.L = p->Lw;
  a.V = p->V;
  a.off_in = oj;
  a.nyq = (p->Lw % 2 == 0) ? p->Lw / 2 : -1;
  a.P = P;
  a.out_scale = 1.0f;
  const double bytes = (double)P * Win * 4 + (double)P * p->V * (p->bf16 ? 4 : 8);
  return launch_any(p, a, false, Win, in, out, "spec_fwd_1d", bytes, s);
}

bl_status_t launch_bluestein_inv(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OW, int cj,
                                 hipStream_t s) {
  BlueArgs a{};
  a.L = p->Lw;
  a.V = p->V;
  a.off_out = cj;
  a.nyq = (p->Lw % 2 == 0) ? p->Lw / 2 : -1;
  a.P = P;
  a.out_scale = 1.0f / (float)p->Lw;
  const double bytes = (double)P * p->V * 8 + (double)P * OW * 4;
  return launch_any(p, a, true, OW, in, out, "spec_inv_1d", bytes, s);
}

}  // namespace blc


