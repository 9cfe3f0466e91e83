// Fine-grained "top" compression (supplementary section "Error Incurred by 2D
// Convolution with Compression"): in a stored spectrum, the k coefficients of
// smallest magnitude of each group are set to zero and the tensor keeps its
// size.  A group is one sample's input spectrum (its C_in channels at every
// kept bin) or one output filter's spectrum (its C_in channels at every kept
// bin); coefficient i of a group is (bin i / C_in, channel i % C_in).
//
//   k_zero_smallest   one block per group (k_top_* below split few, large
//                     groups over several blocks): an exact radix select of the k-th
//                     smallest key |z|^2 (fp32 bit patterns of non-negative
//                     values order as unsigned integers) over three digits
//                     (11, 11 and 10 bits, one histogram pass each), then a
//                     pass that zeroes every key below the threshold and the
//                     first keys equal to it in index order, so that exactly k
//                     are zeroed and the result does not depend on scheduling.
#include <algorithm>
#include <type_traits>

#include "common.hpp"

namespace blc {
namespace {

constexpr int kTopThreads = 1024;
constexpr int kTopWaves = kTopThreads / 64;
constexpr int kDigitBins = 2048;  // largest digit: 11 bits

// Coefficient i of group g sits at (i / C) sB + (i % C) sC + g sG.
struct TopMap {
  unsigned C;
  unsigned long long sB, sC, sG;
};

struct TopArgs {
  unsigned n;     // coefficients per group
  unsigned k;     // how many to zero, 1 <= k
  TopMap src;     // where the keys are read (the spectrum, or a group-major copy)
  TopMap dst;     // where zeros are written (the stored spectrum)
};

// (i / C, i % C) advanced by a fixed step without a division per element
struct Walk {
  unsigned b, c, db, dc, C;
  __device__ Walk(unsigned i, unsigned step, unsigned C_) : b(i / C_), c(i % C_), db(step / C_), dc(step % C_), C(C_) {}
  __device__ void next() {
    b += db;
    c += dc;
    if (c >= C) {
      c -= C;
      ++b;
    }
  }
  __device__ size_t at(const TopMap& m, size_t base) const { return base + (size_t)b * m.sB + (size_t)c * m.sC; }
};

template <typename S>
__device__ __forceinline__ unsigned mag_key(const S* spec, size_t a) {
  const float2 v = spec_get(spec, a);
  return __float_as_uint(fmaf(v.x, v.x, v.y * v.y));
}

template <typename S>
__global__ __launch_bounds__(kTopThreads) void k_zero_smallest(S* __restrict__ spec, const S* __restrict__ keys,
                                                               TopArgs g) {
  __shared__ unsigned hist[kDigitBins];
  __shared__ unsigned wcount[kTopWaves];
  __shared__ unsigned sel[2];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const size_t sbase = (size_t)blockIdx.x * g.src.sG, dbase = (size_t)blockIdx.x * g.dst.sG;
  if (g.k >= g.n) {  // every coefficient of the group
    Walk d(tid, kTopThreads, g.dst.C);
    for (unsigned i = tid; i < g.n; i += kTopThreads, d.next()) spec_put(spec, d.at(g.dst, dbase), make_float2(0.f, 0.f));
    return;
  }
  // the keys matching `prefix` on the bits of `pmask` are the candidates; the
  // threshold is the krem-th smallest of them (1-based)
  unsigned prefix = 0, pmask = 0, krem = g.k;
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 21 : pass == 1 ? 10 : 0;
    const unsigned dmask = pass == 2 ? 0x3FFu : 0x7FFu;
    for (int j = tid; j < kDigitBins; j += kTopThreads) hist[j] = 0u;
    __syncthreads();
    // four keys in flight per thread
    Walk w0(tid, 4 * kTopThreads, g.src.C), w1(tid + kTopThreads, 4 * kTopThreads, g.src.C),
        w2(tid + 2 * kTopThreads, 4 * kTopThreads, g.src.C), w3(tid + 3 * kTopThreads, 4 * kTopThreads, g.src.C);
    unsigned i = tid;
    for (; i + 3 * kTopThreads < g.n; i += 4 * kTopThreads) {
      const unsigned k0 = mag_key(keys, w0.at(g.src, sbase)), k1 = mag_key(keys, w1.at(g.src, sbase));
      const unsigned k2 = mag_key(keys, w2.at(g.src, sbase)), k3 = mag_key(keys, w3.at(g.src, sbase));
      w0.next(); w1.next(); w2.next(); w3.next();
      if ((k0 & pmask) == prefix) atomicAdd(&hist[(k0 >> shift) & dmask], 1u);
      if ((k1 & pmask) == prefix) atomicAdd(&hist[(k1 >> shift) & dmask], 1u);
      if ((k2 & pmask) == prefix) atomicAdd(&hist[(k2 >> shift) & dmask], 1u);
      if ((k3 & pmask) == prefix) atomicAdd(&hist[(k3 >> shift) & dmask], 1u);
    }
    // at most three more elements per thread: i, i + 1024, i + 2048 (walkers 0-2)
    if (i < g.n) {
      const unsigned key = mag_key(keys, w0.at(g.src, sbase));
      if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & dmask], 1u);
    }
    if (i + kTopThreads < g.n) {
      const unsigned key = mag_key(keys, w1.at(g.src, sbase));
      if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & dmask], 1u);
    }
    if (i + 2 * kTopThreads < g.n) {
      const unsigned key = mag_key(keys, w2.at(g.src, sbase));
      if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & dmask], 1u);
    }
    __syncthreads();
    if (wave == 0) {
      // lane l holds the sum of bins 32 l .. 32 l + 31; the digit lies in the
      // first lane whose inclusive prefix reaches krem (one always does: the
      // candidates number at least krem)
      unsigned s = 0;
      for (int j = 0; j < 32; ++j) s += hist[lane * 32 + j];
      unsigned incl = s;
      for (int off = 1; off < 64; off <<= 1) {
        const unsigned t = __shfl_up(incl, off, 64);
        if (lane >= off) incl += t;
      }
      const unsigned long long hit = __ballot(incl >= krem);
      if (lane == __builtin_ctzll(hit)) {
        unsigned before = incl - s;
        int d = lane * 32;
        while (before + hist[d] < krem) before += hist[d++];
        sel[0] = (unsigned)d;
        sel[1] = krem - before;
      }
    }
    __syncthreads();
    prefix |= sel[0] << shift;
    pmask |= dmask << shift;
    krem = sel[1];
    __syncthreads();  // sel is written again by the next pass
  }
  // every key below the threshold, and the first krem keys equal to it
  const unsigned T = prefix;
  unsigned seen = 0;  // keys equal to T in earlier chunks
  Walk ws(tid, kTopThreads, g.src.C), wd(tid, kTopThreads, g.dst.C);
  for (unsigned start = 0; start < g.n; start += kTopThreads, ws.next(), wd.next()) {
    const bool in = start + tid < g.n;
    const unsigned key = in ? mag_key(keys, ws.at(g.src, sbase)) : 0xFFFFFFFFu;
    const bool eq = in && key == T;
    const unsigned long long bal = __ballot(eq);
    const unsigned below = (unsigned)__popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wcount[wave] = (unsigned)__popcll(bal);
    __syncthreads();
    unsigned rank = seen + below, total = 0;
    for (int w = 0; w < kTopWaves; ++w) {
      if (w < wave) rank += wcount[w];
      total += wcount[w];
    }
    if (in && (key < T || (eq && rank < krem))) spec_put(spec, wd.at(g.dst, dbase), make_float2(0.f, 0.f));
    seen += total;
    __syncthreads();  // wcount is written again by the next chunk
  }
}

// W [R][F] (R = kept C_in rows (bin, channel), F filters) -> Wt [F][R], 64 x 64
// tiles through LDS, so that each filter's coefficients lie contiguous
template <typename S>
__global__ __launch_bounds__(256) void k_transpose_filters(const S* __restrict__ W, S* __restrict__ Wt, unsigned R,
                                                           unsigned F) {
  __shared__ S tile[64][65];
  const unsigned r0 = blockIdx.x * 64, f0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int j = ty; j < 64; j += 4) {
    const unsigned r = r0 + j, f = f0 + tx;
    if (r < R && f < F) tile[j][tx] = W[(size_t)r * F + f];
  }
  __syncthreads();
  for (int j = ty; j < 64; j += 4) {
    const unsigned f = f0 + j, r = r0 + tx;
    if (r < R && f < F) Wt[(size_t)f * R + r] = tile[tx][j];
  }
}

// ---- several blocks per group (groups too few to fill the chip) ----------
// The same select, with each group's coefficients split into NB slices of
// `per` (one block of 256 each): per digit, every slice adds its LDS histogram
// into the group's histogram in global memory and one wave per group picks the
// digit; then each slice counts its keys equal to the threshold, and the
// zeroing pass ranks the equal keys of a slice after those of the slices
// before it, so the zeros are exactly those of the one-block select.
constexpr int kSliceThreads = 256;

struct TopState {
  unsigned prefix, pmask, krem, pad;
};

__global__ __launch_bounds__(256) void k_top_init(unsigned* __restrict__ hist, TopState* __restrict__ st,
                                                  unsigned k) {
  const unsigned g = blockIdx.x;
  for (int j = threadIdx.x; j < kDigitBins; j += 256) hist[(size_t)g * kDigitBins + j] = 0u;
  if (threadIdx.x == 0) st[g] = TopState{0u, 0u, k, 0u};
}

template <typename S>
__global__ __launch_bounds__(kSliceThreads) void k_top_hist(const S* __restrict__ keys, TopArgs g, unsigned per,
                                                            unsigned* __restrict__ hist,
                                                            const TopState* __restrict__ st, int pass) {
  __shared__ unsigned h[kDigitBins];
  const int tid = threadIdx.x;
  const unsigned grp = blockIdx.y, i0 = blockIdx.x * per, i1 = min(g.n, i0 + per);
  const size_t sbase = (size_t)grp * g.src.sG;
  const TopState cur = st[grp];
  const int shift = pass == 0 ? 21 : pass == 1 ? 10 : 0;
  const unsigned dmask = pass == 2 ? 0x3FFu : 0x7FFu;
  for (int j = tid; j < kDigitBins; j += kSliceThreads) h[j] = 0u;
  __syncthreads();
  Walk w(i0 + tid, kSliceThreads, g.src.C);
  for (unsigned i = i0 + tid; i < i1; i += kSliceThreads, w.next()) {
    const unsigned key = mag_key(keys, w.at(g.src, sbase));
    if ((key & cur.pmask) == cur.prefix) atomicAdd(&h[(key >> shift) & dmask], 1u);
  }
  __syncthreads();
  unsigned* gh = hist + (size_t)grp * kDigitBins;
  for (int j = tid; j < kDigitBins; j += kSliceThreads)
    if (h[j]) atomicAdd(&gh[j], h[j]);
}

// one wave per group: the digit holding the krem-th candidate; the histogram
// is cleared for the next digit
__global__ __launch_bounds__(64) void k_top_select(unsigned* __restrict__ hist, TopState* __restrict__ st,
                                                   int pass) {
  const int lane = threadIdx.x;
  const unsigned grp = blockIdx.x;
  unsigned* gh = hist + (size_t)grp * kDigitBins;
  const TopState cur = st[grp];
  const int shift = pass == 0 ? 21 : pass == 1 ? 10 : 0;
  const unsigned dmask = pass == 2 ? 0x3FFu : 0x7FFu;
  unsigned s = 0;
  for (int j = 0; j < 32; ++j) s += gh[lane * 32 + j];
  unsigned incl = s;
  for (int off = 1; off < 64; off <<= 1) {
    const unsigned t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  const unsigned long long hit = __ballot(incl >= cur.krem);
  if (lane == __builtin_ctzll(hit)) {
    unsigned before = incl - s;
    int d = lane * 32;
    while (before + gh[d] < cur.krem) before += gh[d++];
    st[grp] = TopState{cur.prefix | ((unsigned)d << shift), cur.pmask | (dmask << shift), cur.krem - before, 0u};
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  for (int j = lane; j < kDigitBins; j += 64) gh[j] = 0u;
}

template <typename S>
__global__ __launch_bounds__(kSliceThreads) void k_top_count(const S* __restrict__ keys, TopArgs g, unsigned per,
                                                             const TopState* __restrict__ st,
                                                             unsigned* __restrict__ cnt) {
  __shared__ unsigned wc[kSliceThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const unsigned grp = blockIdx.y, i0 = blockIdx.x * per, i1 = min(g.n, i0 + per);
  const size_t sbase = (size_t)grp * g.src.sG;
  const unsigned T = st[grp].prefix;
  unsigned c = 0;
  Walk w(i0 + tid, kSliceThreads, g.src.C);
  for (unsigned i = i0 + tid; i < i1; i += kSliceThreads, w.next()) c += mag_key(keys, w.at(g.src, sbase)) == T;
  for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off, 64);
  if (lane == 0) wc[wave] = c;
  __syncthreads();
  if (tid == 0) {
    unsigned t = 0;
    for (int q = 0; q < kSliceThreads / 64; ++q) t += wc[q];
    cnt[(size_t)grp * gridDim.x + blockIdx.x] = t;
  }
}

template <typename S>
__global__ __launch_bounds__(kSliceThreads) void k_top_zero(S* __restrict__ spec, const S* __restrict__ keys,
                                                            TopArgs g, unsigned per,
                                                            const TopState* __restrict__ st,
                                                            const unsigned* __restrict__ cnt) {
  __shared__ unsigned wc[kSliceThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const unsigned grp = blockIdx.y, i0 = blockIdx.x * per, i1 = min(g.n, i0 + per);
  const size_t sbase = (size_t)grp * g.src.sG, dbase = (size_t)grp * g.dst.sG;
  const TopState cur = st[grp];
  const unsigned T = cur.prefix;
  unsigned seen = 0;  // keys equal to T in earlier slices, then earlier chunks
  for (unsigned q = 0; q < blockIdx.x; ++q) seen += cnt[(size_t)grp * gridDim.x + q];
  Walk ws(i0 + tid, kSliceThreads, g.src.C), wd(i0 + tid, kSliceThreads, g.dst.C);
  for (unsigned start = i0; start < i1; start += kSliceThreads, ws.next(), wd.next()) {
    const bool in = start + tid < i1;
    const unsigned key = in ? mag_key(keys, ws.at(g.src, sbase)) : 0xFFFFFFFFu;
    const bool eq = in && key == T;
    const unsigned long long bal = __ballot(eq);
    const unsigned below = (unsigned)__popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wc[wave] = (unsigned)__popcll(bal);
    __syncthreads();
    unsigned rank = seen + below, total = 0;
    for (int q = 0; q < kSliceThreads / 64; ++q) {
      if (q < wave) rank += wc[q];
      total += wc[q];
    }
    if (in && (key < T || (eq && rank < cur.krem))) spec_put(spec, wd.at(g.dst, dbase), make_float2(0.f, 0.f));
    seen += total;
    __syncthreads();
  }
}

}  // namespace
}  // namespace blc

using namespace blc;

extern "C" bl_status_t bl_conv_zero_smallest(bl_conv_plan_t p, const float* src, void* ws, unsigned which,
                                             long long k, unsigned flags, void* stream) {
  if (!p || !ws || k < 0) return BL_ERR_INVALID_ARG;
  if (which != BL_SPEC_X && which != BL_SPEC_W) return BL_ERR_INVALID_ARG;
  const unsigned reuse = which == BL_SPEC_X ? BL_REUSE_X : BL_REUSE_W;
  if (flags & ~reuse) return BL_ERR_INVALID_ARG;
  if (!(flags & reuse) && !src) return BL_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* spec = static_cast<char*>(ws) + (which == BL_SPEC_X ? p->off_X : p->off_W);
  const long long n = (long long)p->kept * p->Cin;
  const long long groups = which == BL_SPEC_X ? p->N : p->Cout;
  if (n >= 2147483647LL || groups >= 2147483647LL) return BL_ERR_UNSUPPORTED;
  if (!(flags & reuse)) {
    const bl_status_t st = which == BL_SPEC_X
                               ? launch_spec_fwd(p, src, spec, (long)p->N * p->Cin, p->Hi, p->Wi, p->pt, p->pl, s)
                               : launch_spec_filt(p, src, spec, s);
    if (st != BL_OK) return st;
  }
  if (k == 0) return BL_OK;
  TopArgs g{};
  g.n = (unsigned)n;
  g.k = (unsigned)std::min<long long>(k, n);
  // the filters' coefficients are strided by C_out in W[b][c][f]: the keys are
  // read from a group-major copy in the weight-gradient region of ws (free
  // between calls), the zeros written to W
  void* keys = spec;
  if (which == BL_SPEC_X) {  // X[b][n][c]: group = sample n
    g.src = TopMap{(unsigned)p->Cin, (unsigned long long)p->N * p->Cin, 1ull, (unsigned long long)p->Cin};
    g.dst = g.src;
  } else {  // W[b][c][f]: group = filter f
    g.src = TopMap{(unsigned)n, 0ull, 1ull, (unsigned long long)n};
    g.dst = TopMap{(unsigned)p->Cin, (unsigned long long)p->Cin * p->Cout, (unsigned long long)p->Cout, 1ull};
    keys = static_cast<char*>(ws) + p->off_DW;
    const unsigned R = (unsigned)n, F = (unsigned)p->Cout;
    const dim3 tgrid((R + 63) / 64, (F + 63) / 64);
    if (tgrid.y > 65535) return BL_ERR_UNSUPPORTED;
    const double eb = p->bf16 ? 4.0 : 8.0;
    const bl_status_t st = timed_launch("zero_smallest_transpose", 2.0 * eb * R * F, 0.0, s,
                                        [&](hipEvent_t e0, hipEvent_t e1) {
      if (p->bf16)
        hipExtLaunchKernelGGL(k_transpose_filters<unsigned>, tgrid, dim3(256), 0, s, e0, e1, 0,
                              static_cast<const unsigned*>(spec), static_cast<unsigned*>(keys), R, F);
      else
        hipExtLaunchKernelGGL(k_transpose_filters<float2>, tgrid, dim3(256), 0, s, e0, e1, 0,
                              static_cast<const float2*>(spec), static_cast<float2*>(keys), R, F);
    });
    if (st != BL_OK) return st;
  }
  // compulsory traffic: the spectrum read once and the zeroed coefficients written
  const double eb = p->bf16 ? 4.0 : 8.0;
  const double bytes = eb * (double)groups * ((double)g.n + (double)g.k);
  // few, large groups: slices of at least 4096 coefficients, about 1024
  // blocks in all, at the price of nine launches instead of one (measured:
  // C5's 32 samples of 111 360 coefficients 143 -> 54 us; groups of 12 288 to
  // 39 168 coefficients are faster with one block each); scratch (histograms,
  // states, counts) in the contraction-output region of ws, which holds
  // nothing between calls
  if (g.k < g.n && groups <= 128 && g.n >= 65536) {
    const long want = std::max<long>(2, (1024 + groups - 1) / groups);
    const unsigned per = (unsigned)std::max<long>(4096, ((long)g.n + want - 1) / want);
    const unsigned nb = (g.n + per - 1) / per;
    char* scratch = static_cast<char*>(ws) + p->off_T;
    unsigned* hist = reinterpret_cast<unsigned*>(scratch);
    TopState* st = reinterpret_cast<TopState*>(hist + (size_t)groups * kDigitBins);
    unsigned* cnt = reinterpret_cast<unsigned*>(st + groups);
    const size_t need = (size_t)groups * (kDigitBins * 4 + sizeof(TopState) + (size_t)nb * 4);
    const size_t have = p->off_DW - p->off_T;
    if (need <= have && nb <= 65535) {
      const dim3 sg(nb, (unsigned)groups);
      auto run = [&](auto* sp, auto* kp) -> bl_status_t {
        using S = std::remove_const_t<std::remove_pointer_t<decltype(kp)>>;
        bl_status_t r = timed_launch("zero_smallest_init", (double)groups * kDigitBins * 4, 0.0, s,
                                     [&](hipEvent_t e0, hipEvent_t e1) {
          hipExtLaunchKernelGGL(k_top_init, dim3((unsigned)groups), dim3(256), 0, s, e0, e1, 0, hist, st, g.k);
        });
        for (int pass = 0; pass < 3 && r == BL_OK; ++pass) {
          r = timed_launch("zero_smallest_hist", eb * groups * (double)g.n, 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
            hipExtLaunchKernelGGL(k_top_hist<S>, sg, dim3(kSliceThreads), 0, s, e0, e1, 0, kp, g, per, hist, st,
                                  pass);
          });
          if (r != BL_OK) break;
          r = timed_launch("zero_smallest_select", (double)groups * kDigitBins * 8, 0.0, s,
                           [&](hipEvent_t e0, hipEvent_t e1) {
            hipExtLaunchKernelGGL(k_top_select, dim3((unsigned)groups), dim3(64), 0, s, e0, e1, 0, hist, st, pass);
          });
        }
        if (r != BL_OK) return r;
        r = timed_launch("zero_smallest_count", eb * groups * (double)g.n, 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
          hipExtLaunchKernelGGL(k_top_count<S>, sg, dim3(kSliceThreads), 0, s, e0, e1, 0, kp, g, per, st, cnt);
        });
        if (r != BL_OK) return r;
        return timed_launch("zero_smallest", bytes, 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
          hipExtLaunchKernelGGL(k_top_zero<S>, sg, dim3(kSliceThreads), 0, s, e0, e1, 0, sp, kp, g, per, st, cnt);
        });
      };
      if (p->bf16) return run(static_cast<unsigned*>(spec), static_cast<const unsigned*>(keys));
      return run(static_cast<float2*>(spec), static_cast<const float2*>(keys));
    }
  }
  return timed_launch("zero_smallest", bytes, 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
    if (p->bf16)
      hipExtLaunchKernelGGL(k_zero_smallest<unsigned>, dim3((unsigned)groups), dim3(kTopThreads), 0, s, e0, e1, 0,
                            static_cast<unsigned*>(spec), static_cast<const unsigned*>(keys), g);
    else
      hipExtLaunchKernelGGL(k_zero_smallest<float2>, dim3((unsigned)groups), dim3(kTopThreads), 0, s, e0, e1, 0,
                            static_cast<float2*>(spec), static_cast<const float2*>(keys), g);
  });
}
