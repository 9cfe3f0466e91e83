// Per-kept-bin complex channel contraction on fp32 MFMA (gfx950), tiled.
//
// For each kept bin, O[m][n] = sum_k A[m][k] op(B[k][n]) with op = conj or
// identity: the Hadamard product of the spectra fused with the sum over a
// channel index (Sec. 3.3).  The complex product is embedded in a real GEMM:
// A is read as the real [M x 2K] matrix of interleaved (re, im) pairs, B as the
// real [2K x 2N] matrix of 2x2 blocks [[br, -bi], [bi, br]] (conj) or
// [[br, bi], [-bi, br]] (identity), expanded on the fly from the complex values
// in LDS; the real [M x 2N] result is the interleaved complex O.  Each
// v_mfma_f32_32x32x2f32 step consumes one complex k.
//
// Block tile: BM rows x BN complex columns, 16 complex k per stage.  Global
// loads (16-byte vectors, two complex values each) run two stages ahead of
// the MFMAs through two register sets, and LDS is double buffered.  4 waves
// in a 2x2 grid; a wave owns BM/2 rows x BN/2 complex columns.  Operands are
// staged in LDS as separate real and imaginary planes (B also as its negated
// imaginary plane, so that each lane reads its block entry as is), k-major,
// with padded rows and planes offset by half or a quarter of the banks, so
// that the MFMA operand fetches (one 32-bit read per lane) are free of bank
// conflicts.  Blocks are numbered so that consecutive tiles (which share
// operand rows) run on the same XCD and its L2.
//
// With bfloat16 storage of the spectra the operands arrive as 32-bit (re, im)
// pairs (8-byte vectors, two values each) and run on v_mfma_f32_32x32x8_bf16,
// four complex k per instruction: A is staged as the pairs themselves, B as
// its two block columns per value, each a bf16 pair, with the signs applied to
// the bits.  Products of bfloat16 values are exact in the fp32 accumulators.
#include <algorithm>
#include <type_traits>

#include "common.hpp"

namespace blc {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

// Offsets inside one bin's matrices are 32-bit (a bin's matrices hold far
// fewer than 2^31 elements); the per-bin bases are 64-bit.
struct CgemmArgs {
  int M, N, K;                   // complex sizes
  unsigned sAm, sAk, sBk, sBn;   // element strides (complex units); one of each pair is 1
  unsigned ldo;
  unsigned long long bA, bB, bO;  // per-bin strides
  unsigned long long split_stride;  // complex elements between the partial outputs of two k-splits
  int tiles_n, tiles;               // tiles per bin along n, and per bin in all
  int kper;                         // complex k per split (multiple of the stage depth)
};

constexpr int kBK = 16;  // complex k per stage

// LDS plane of kBK rows of W floats: the smallest size of at least the rows
// that is 32 (mod 64) floats, so that consecutive planes sit half the banks apart.
template <int W>
constexpr int plane_floats() {
  return kBK * W + ((32 - kBK * W % 64) + 64) % 64;
}

typedef short shortx4 __attribute__((ext_vector_type(4)));

// BF16: operands stored as bfloat16 pairs (32-bit words, real part in the low
// half), multiplied on the bf16 matrix cores with fp32 accumulation; else
// complex64 on the fp32 ones.
// KS: groups of 4 waves sharing the tile (fp32 only): group q takes the
// k-stages q, q + KS, ... through its own LDS buffers, and the groups' sums are
// added through LDS in group order at the end.  Used when the launch has no
// more tiles than compute units, so that each SIMD runs KS waves instead of one.
// LDS layout of one tile's stage buffers (floats).
template <int BM, int BN, bool BF16, int KS>
struct CgemmLds {
  // rows padded by 2 floats: the 64 x 32 tile's buffers then take 30 KB, so
  // that five blocks fit one CU's LDS
  static constexpr int SA = BM + 2, SB = BN + 2;
  static constexpr int PA = plane_floats<SA>(), PB = plane_floats<SB>();
  static constexpr int ABUF = PA + kBK * SA, BBUF = 2 * PB + 16 + kBK * SB;  // floats per stage buffer
  // bf16 operands: A as packed (re, im) pairs [k][m]; B in two forms [form][k][n],
  // the (even, odd) real-k entries of the 2x2 block column the lane reads.
  // Row strides of 16 (mod 32) words put the two half-waves' rows (k and k + 2)
  // in disjoint banks; the form planes are 16 (mod 64) words apart.
  static constexpr int SA16 = BM + 16, SB16 = BN + 16;
  static constexpr int PB16 = ((kBK * SB16 + 63) / 64) * 64 + 16;
  static constexpr int floats = BF16 ? 2 * kBK * SA16 + 2 * 2 * PB16 : KS * 2 * (ABUF + BBUF);
};

// One output tile: tile id (bin-major over the launch's tiles) and k-split kz,
// with the stage buffers in smem (CgemmLds floats, 16-byte aligned).
template <int BM, int BN, bool A_KC, bool B_NC, bool CONJ, bool BF16, int KS>
__device__ __forceinline__ void cgemm_tile(const void* __restrict__ A_, const void* __restrict__ B_,
                                           float2* __restrict__ O, const CgemmArgs& g, unsigned id, int kz,
                                           float* smem) {
  static_assert(KS == 1 || !BF16, "the in-block k split is built for the fp32 operands");
  using S = std::conditional_t<BF16, unsigned, float2>;  // stored operand element
  using V = std::conditional_t<BF16, uint2, float4>;     // two consecutive elements
  const S* A = static_cast<const S*>(A_);
  const S* Bm = static_cast<const S*>(B_);
  constexpr int WM = BM / 2;   // rows per wave
  constexpr int WN = BN / 2;   // complex columns per wave
  constexpr int MI = WM / 32;  // 32-row MFMA blocks per wave
  constexpr int NJ = WN / 16;  // 16-complex-column MFMA blocks per wave
  constexpr int AV = BM / 32;  // 16-byte A loads per thread per stage
  constexpr int BV = BN / 32;  // 16-byte B loads per thread per stage
  using L = CgemmLds<BM, BN, BF16, KS>;
  constexpr int SA = L::SA, SB = L::SB, PA = L::PA, PB = L::PB, ABUF = L::ABUF, BBUF = L::BBUF;
  constexpr int SA16 = L::SA16, SB16 = L::SB16, PB16 = L::PB16;
  // fp32: A buffers [group][stage buffer] of ABUF floats, then B buffers of
  // BBUF; B planes: re at 0, im at PB (half the banks away), -im at 2 PB + 16
  // (a quarter of the banks away from both), so that no lane negates a value.
  // bf16: A buffers [2][kBK SA16] words, then B buffers [2][2 PB16].
  auto As = [&](int gq, int b) { return smem + (gq * 2 + b) * ABUF; };
  auto Bs = [&](int gq, int b) { return smem + KS * 2 * ABUF + (gq * 2 + b) * BBUF; };
  auto As16 = [&](int b) { return reinterpret_cast<unsigned*>(smem) + b * kBK * SA16; };
  auto Bs16 = [&](int b) { return reinterpret_cast<unsigned*>(smem) + 2 * kBK * SA16 + b * 2 * PB16; };

  const int bin = id / g.tiles;
  const int tile = id - bin * g.tiles;
  const int kbeg = kz * g.kper;
  const int kend = min(g.K, kbeg + g.kper);
  const int tm = tile / g.tiles_n, tn = tile - tm * g.tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const S* Ab = A + bin * g.bA;
  const S* Bb = Bm + bin * g.bB;
  const int tid = threadIdx.x & 255, grp = KS == 1 ? 0 : (int)(threadIdx.x >> 8), lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * WM, wn = (wave & 1) * WN;

  // B operand of this lane: real column jcol = lane % 32 of a 32-wide block is
  // complex column jcol / 2, part jcol % 2; real k row a_part = lane / 32.
  const int a_part = lane >> 5;
  const int jcol = lane & 31;
  const int bcol = jcol & 1;
  // br on the block diagonal, +bi or -bi off it
  const bool neg = CONJ ? (a_part == 0 && bcol == 1) : (a_part == 1 && bcol == 0);
  const int b_poff = (a_part == bcol) ? 0 : neg ? 2 * PB + 16 : PB;

  floatx16 acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const V zero4{};
  // Operand positions of this thread's two-element vectors in a stage, and whether
  // they lie inside the matrices.  Loads are unconditional (a vector outside
  // reads the bin's first one, which always exists) and the zero fill happens
  // when the registers are stored to LDS, so no branch separates a prefetch
  // from the loads after it and the loads stay in flight across the stage.
  auto a_pos = [&](int q, int& m, int& k) {
    const int e = tid + 256 * q;
    if (A_KC) { m = e >> 3; k = (e & 7) * 2; }
    else { k = e / (BM / 2); m = (e - k * (BM / 2)) * 2; }
  };
  auto b_pos = [&](int q, int& k, int& n) {
    const int e = tid + 256 * q;
    if (B_NC) { k = e / (BN / 2); n = (e - k * (BN / 2)) * 2; }
    else { n = e >> 3; k = (e & 7) * 2; }
  };
  // per-thread load geometry, fixed over the k loop: per stage each offset
  // is one add and one select (no branch)
  unsigned a_base[AV], b_base[BV];
  int a_kk[AV], b_kk[BV];
  bool a_in[AV], b_in[BV];
#pragma unroll
  for (int q = 0; q < AV; ++q) {
    int m, k;
    a_pos(q, m, k);
    a_in[q] = m0 + m < g.M;
    a_kk[q] = k;
    a_base[q] = (unsigned)(m0 + m) * g.sAm + (unsigned)k * g.sAk;
  }
#pragma unroll
  for (int q = 0; q < BV; ++q) {
    int k, n;
    b_pos(q, k, n);
    b_in[q] = n0 + n < g.N;
    b_kk[q] = k;
    b_base[q] = (unsigned)k * g.sBk + (unsigned)(n0 + n) * g.sBn;
  }
  auto load = [&](int k0, V* ra, V* rb) {
    const int lim = kend - k0;
    const unsigned ka = (unsigned)k0 * g.sAk, kb = (unsigned)k0 * g.sBk;
#pragma unroll
    for (int q = 0; q < AV; ++q) {
      const bool in = a_in[q] & (a_kk[q] < lim);
      ra[q] = *reinterpret_cast<const V*>(Ab + (in ? a_base[q] + ka : 0u));
    }
#pragma unroll
    for (int q = 0; q < BV; ++q) {
      const bool in = b_in[q] & (b_kk[q] < lim);
      rb[q] = *reinterpret_cast<const V*>(Bb + (in ? b_base[q] + kb : 0u));
    }
  };
  // the two forms of a stored value w = (br, bi): conj block [[br, -bi], [bi, br]],
  // identity block [[br, bi], [-bi, br]]; form f is column f of the block,
  // (even, odd) halves = (real-k rows 2k, 2k + 1); negation flips a sign bit
  auto form0 = [](unsigned w) { return CONJ ? w : w ^ 0x80000000u; };
  auto form1 = [](unsigned w) { return CONJ ? ((w >> 16) ^ 0x8000u) | (w << 16) : (w >> 16) | (w << 16); };
  // Column swizzle of the bf16 stages: row k stores column c at c ^ swz(k).
  // Threads that load along k store 8 columns x 8 even rows per wave, rows
  // that the padded strides alone would put on a few banks; the XOR spreads
  // them over all banks.  Rows 4q .. 4q + 3 share one value, and it only
  // permutes bits 3-4 of the column, so the MFMA operand reads (32 or 16
  // consecutive columns of rows 4q + {0, 1, 2, 3}) stay conflict-free.
  auto swz = [](int k) { return 8 * ((k >> 2) & 3); };
  auto store16 = [&](int buf, int k0, const V* ra, const V* rb) {
    unsigned* a16 = As16(buf);
#pragma unroll
    for (int q = 0; q < AV; ++q) {
      int m, k;
      a_pos(q, m, k);
      const V r = ((m0 + m < g.M) && (k0 + k < kend)) ? ra[q] : zero4;
      const int ms = m ^ swz(k);  // rows k and k + 1 share the swizzle (k even)
      if (A_KC) {
        a16[k * SA16 + ms] = r.x;
        a16[(k + 1) * SA16 + ms] = r.y;
      } else {
        a16[k * SA16 + ms] = r.x;
        a16[k * SA16 + ms + 1] = r.y;  // m even: (m + 1) ^ swz = ms + 1
      }
    }
    unsigned* b16 = Bs16(buf);
#pragma unroll
    for (int q = 0; q < BV; ++q) {
      int k, n;
      b_pos(q, k, n);
      const V r = ((n0 + n < g.N) && (k0 + k < kend)) ? rb[q] : zero4;
      // second value at (k, n + 1) when n runs along the vector, else (k + 1, n)
      const int i0 = k * SB16 + (n ^ swz(k)), i1 = B_NC ? i0 + 1 : i0 + SB16;
      b16[i0] = form0(r.x);
      b16[PB16 + i0] = form1(r.x);
      b16[i1] = form0(r.y);
      b16[PB16 + i1] = form1(r.y);
    }
  };
  auto store = [&](int buf, int k0, const V* ra, const V* rb) {
    if constexpr (BF16) {
      store16(buf, k0, ra, rb);
    } else {
      float* a0 = As(grp, buf);
      float* a1 = As(grp, buf) + PA;
#pragma unroll
      for (int q = 0; q < AV; ++q) {
        int m, k;
        a_pos(q, m, k);
        const float4 r = ((m0 + m < g.M) && (k0 + k < kend)) ? ra[q] : zero4;
        if (A_KC) {
          a0[k * SA + m] = r.x; a1[k * SA + m] = r.y;
          a0[(k + 1) * SA + m] = r.z; a1[(k + 1) * SA + m] = r.w;
        } else {
          *reinterpret_cast<float2*>(a0 + k * SA + m) = make_float2(r.x, r.z);
          *reinterpret_cast<float2*>(a1 + k * SA + m) = make_float2(r.y, r.w);
        }
      }
      float* b0 = Bs(grp, buf);
      float* b1 = Bs(grp, buf) + PB;
      float* b2 = Bs(grp, buf) + 2 * PB + 16;
#pragma unroll
      for (int q = 0; q < BV; ++q) {
        int k, n;
        b_pos(q, k, n);
        const float4 r = ((n0 + n < g.N) && (k0 + k < kend)) ? rb[q] : zero4;
        if (B_NC) {
          *reinterpret_cast<float2*>(b0 + k * SB + n) = make_float2(r.x, r.z);
          *reinterpret_cast<float2*>(b1 + k * SB + n) = make_float2(r.y, r.w);
          *reinterpret_cast<float2*>(b2 + k * SB + n) = make_float2(-r.y, -r.w);
        } else {
          b0[k * SB + n] = r.x; b1[k * SB + n] = r.y; b2[k * SB + n] = -r.y;
          b0[(k + 1) * SB + n] = r.z; b1[(k + 1) * SB + n] = r.w; b2[(k + 1) * SB + n] = -r.w;
        }
      }
    }
  };
  auto compute16 = [&](int buf) {
    // v_mfma_f32_32x32x8_bf16: lane l supplies real k = 4 (l / 32) .. + 3 of its
    // row (A) or column (B), i.e. complex k = 2 (l / 32) and 2 (l / 32) + 1 of
    // the four complex k an instruction consumes
    const unsigned* a16 = As16(buf);
    const unsigned* b16 = Bs16(buf) + bcol * PB16;
#pragma unroll
    for (int q = 0; q < kBK / 4; ++q) {
      const int kc = 4 * q + 2 * a_part;
      const int s = swz(4 * q);  // rows kc and kc + 1 lie in 4q .. 4q + 3
      shortx4 av[MI], bv[NJ];
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const int m = wm + 32 * i + (jcol ^ s);  // wm + 32 i has no bits below 5
        const unsigned lo = a16[kc * SA16 + m], hi = a16[(kc + 1) * SA16 + m];
        av[i] = shortx4{(short)(lo & 0xFFFF), (short)(lo >> 16), (short)(hi & 0xFFFF), (short)(hi >> 16)};
      }
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int n = (wn + 16 * j + (jcol >> 1)) ^ s;
        const unsigned lo = b16[kc * SB16 + n], hi = b16[(kc + 1) * SB16 + n];
        bv[j] = shortx4{(short)(lo & 0xFFFF), (short)(lo >> 16), (short)(hi & 0xFFFF), (short)(hi >> 16)};
      }
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
  };
  auto compute = [&](int buf) {
    if constexpr (BF16) {
      compute16(buf);
      return;
    }
    // all fragments of the stage first, so the LDS reads overlap the MFMAs
    const float* ap = As(grp, buf) + a_part * PA + wm + jcol;
    const float* bp = Bs(grp, buf) + b_poff + wn + (jcol >> 1);
    float av[kBK][MI], bv[kBK][NJ];
#pragma unroll
    for (int s = 0; s < kBK; ++s) {
#pragma unroll
      for (int i = 0; i < MI; ++i) av[s][i] = ap[s * SA + 32 * i];
#pragma unroll
      for (int j = 0; j < NJ; ++j) bv[s][j] = bp[s * SB + 16 * j];
    }
#pragma unroll
    for (int s = 0; s < kBK; ++s)
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[s][i], bv[s][j], acc[i][j], 0, 0, 0);
  };

  // stage st sits in LDS buffer st % 2; register set st % 2 receives stage
  // st + 2 while stage st + 1 (in the other set) waits to be stored.  The loop
  // body has no branch, so the compiler's wait before each store covers only
  // the loads of the stage being stored: a stage index past the last is
  // clamped for the load (a repeated, cached read) and zero-filled by the
  // store; with an odd number of stages the last pair's second stage is such
  // an all-zero stage (its MFMAs add nothing).
  // Group grp's local stage t is stage KS t + grp of the k range (the groups
  // loop the same number of times: a stage past the last is zero-filled).
  const int nst = (kend - kbeg + kBK - 1) / kBK;
  const int nst_l = (nst + KS - 1) / KS;
  auto kof = [&](int t) { return kbeg + min(KS * t + grp, nst - 1) * kBK; };
  auto k0of = [&](int t) { return kbeg + (KS * t + grp) * kBK; };
  V ra0[AV], rb0[BV], ra1[AV], rb1[BV];
  load(kof(0), ra0, rb0);
  load(kof(1), ra1, rb1);
  store(0, k0of(0), ra0, rb0);
  __syncthreads();
  for (int cs = 0; cs < nst_l; cs += 2) {
    load(kof(cs + 2), ra0, rb0);
    compute(0);
    store(1, k0of(cs + 1), ra1, rb1);
    __syncthreads();
    load(kof(cs + 3), ra1, rb1);
    compute(1);
    store(0, k0of(cs + 2), ra0, rb0);
    __syncthreads();
  }
  if constexpr (KS > 1) {
    // groups 1.. leave their sums in the (now idle) operand buffers; group 0
    // adds them in group order and stores the tile
    constexpr int kAcc = 256 * MI * NJ * 16;  // floats per group
    static_assert((KS - 1) * kAcc <= KS * 2 * ABUF, "reduction buffer");
    float* red = smem;
    if (grp > 0) {
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) red[(grp - 1) * kAcc + ((i * NJ + j) * 16 + v) * 256 + tid] = acc[i][j][v];
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll
      for (int q = 1; q < KS; ++q)
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
          for (int j = 0; j < NJ; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] += red[(q - 1) * kAcc + ((i * NJ + j) * 16 + v) * 256 + tid];
    }
    __syncthreads();  // the sums are read before the store staging below reuses the buffers
    if (grp > 0) return;
  }

  // D[i][j] of a 32x32 block: VGPR v holds row 8 (v / 4) + 4 (lane / 32) + v % 4, real column lane % 32.
  float* Of = reinterpret_cast<float*>(O + kz * g.split_stride + bin * g.bO);
  if constexpr (!BF16) {
    if (g.ldo % 2 == 0 && g.N % 2 == 0) {
      // through the idle operand buffers, 16 rows of a block at a time (rows
      // padded to 40 floats: the two half-waves' rows land on disjoint banks),
      // so that each lane stores 16 bytes: two complex columns of one row
      float* st = smem + wave * (16 * 40);
      static_assert(4 * 16 * 40 <= KS * 2 * ABUF, "store staging");
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j)
#pragma unroll
          for (int hv = 0; hv < 2; ++hv) {  // VGPRs 8 hv .. 8 hv + 7: rows 16 hv .. 16 hv + 15
#pragma unroll
            for (int v = 0; v < 8; ++v)
              st[(8 * (v >> 2) + 4 * (lane >> 5) + (v & 3)) * 40 + jcol] = acc[i][j][8 * hv + v];
            wave_sync();
#pragma unroll
            for (int it = 0; it < 2; ++it) {
              const int idx = it * 64 + lane, row = idx >> 3, c4 = idx & 7;
              const int m = m0 + wm + 32 * i + 16 * hv + row;
              const int n = n0 + wn + 16 * j + 2 * c4;
              const float4 val = *reinterpret_cast<const float4*>(st + row * 40 + 4 * c4);
              if (m < g.M && n < g.N) *reinterpret_cast<float4*>(Of + ((unsigned)m * g.ldo + n) * 2) = val;
            }
            wave_sync();
          }
      return;
    }
  }
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int n = n0 + wn + 16 * j + (jcol >> 1);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm + 32 * i + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        if (m < g.M && n < g.N) Of[((unsigned)m * g.ldo + n) * 2 + bcol] = acc[i][j][v];
      }
    }
}

// XCD-aware numbering of a launch's nb blocks: the hardware deals blocks to
// the 8 XCDs in turn, so consecutive logical ids (tiles of one bin, which
// share operand rows) land on one XCD and its L2.
__device__ __forceinline__ unsigned xcd_block_id(unsigned raw, unsigned nb) {
  return nb % 8 == 0 ? (raw % 8) * (nb / 8) + raw / 8 : raw;
}

template <int BM, int BN, bool A_KC, bool B_NC, bool CONJ, bool BF16, int KS>
__global__ __launch_bounds__(256 * KS, KS == 1 ? 2 : 1) void k_cgemm(const void* __restrict__ A_,
                                                                   const void* __restrict__ B_,
                                                                   float2* __restrict__ O, CgemmArgs g) {
  __shared__ __align__(16) float smem[CgemmLds<BM, BN, BF16, KS>::floats];
  const unsigned id = xcd_block_id(blockIdx.x + blockIdx.y * gridDim.x, gridDim.x * gridDim.y);
  cgemm_tile<BM, BN, A_KC, B_NC, CONJ, BF16, KS>(A_, B_, O, g, id, blockIdx.z, smem);
}

// The grad-input and grad-weight contractions of a layer in one launch (both
// need only the stored spectra): logical blocks [0, s1 t1) take grad-input
// tiles (DX = DY W), the rest grad-weight tiles (DW = X^T conj(DY)), one tile
// shape; t1, t2 = tiles x bins of a pass, s1, s2 its k ranges (a pass split
// along k writes partial sums, split_stride apart).  One launch instead of
// two, and the two passes' tiles, of equal k length, share the CUs.
template <int BM, int BN, bool BF16>
__global__ __launch_bounds__(256, 2) void k_cgemm_bwd(const void* __restrict__ A1, const void* __restrict__ B1,
                                                     float2* __restrict__ O1, CgemmArgs g1,
                                                     const void* __restrict__ A2, const void* __restrict__ B2,
                                                     float2* __restrict__ O2, CgemmArgs g2, unsigned t1, unsigned s1,
                                                     unsigned t2) {
  __shared__ __align__(16) float smem[CgemmLds<BM, BN, BF16, 1>::floats];
  const unsigned id = xcd_block_id(blockIdx.x, gridDim.x);
  if (id < t1 * s1) {
    cgemm_tile<BM, BN, true, false, false, BF16, 1>(A1, B1, O1, g1, id % t1, id / t1, smem);
  } else {
    const unsigned j = id - t1 * s1;
    cgemm_tile<BM, BN, false, true, true, BF16, 1>(A2, B2, O2, g2, j % t2, j / t2, smem);
  }
}

// out[i] = sum over k-splits of part[s][i], in split order.
__global__ __launch_bounds__(256) void k_split_reduce(const float4* __restrict__ part, float4* __restrict__ out,
                                                      unsigned long long n4, int splits) {
  const unsigned long long i = (unsigned long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n4) return;
  float4 acc = part[i];
  for (int s = 1; s < splits; ++s) {
    const float4 v = part[(unsigned long long)s * n4 + i];
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  out[i] = acc;
}

// Operand geometry of one pass for the tiled kernel; false when its 16-byte
// pairs do not align or a bin's matrices need 64-bit offsets.
bool tiled_args(const bl_conv_plan_s* p, Contract which, CgemmArgs& g) {
  g = CgemmArgs{};
  const unsigned long long B = p->kept, N = p->N, Ci = p->Cin, Co = p->Cout;
  bool a_kc = true, b_nc = true;
  switch (which) {
    case Contract::Forward:  // Y[n][f] = sum_c X[n][c] conj(W[c][f])
      g.M = (int)N; g.N = (int)Co; g.K = (int)Ci;
      g.sAm = (unsigned)Ci; g.sAk = 1; g.sBk = (unsigned)Co; g.sBn = 1; g.ldo = (unsigned)Co;
      g.bA = N * Ci; g.bB = Ci * Co; g.bO = N * Co;
      a_kc = true; b_nc = true;
      break;
    case Contract::GradInput:  // DX[n][c] = sum_f DY[n][f] W[c][f]
      g.M = (int)N; g.N = (int)Ci; g.K = (int)Co;
      g.sAm = (unsigned)Co; g.sAk = 1; g.sBk = 1; g.sBn = (unsigned)Co; g.ldo = (unsigned)Ci;
      g.bA = N * Co; g.bB = Ci * Co; g.bO = N * Ci;
      a_kc = true; b_nc = false;
      break;
    case Contract::GradWeight:  // DW[c][f] = sum_n X[n][c] conj(DY[n][f])
      g.M = (int)Ci; g.N = (int)Co; g.K = (int)N;
      g.sAm = 1; g.sAk = (unsigned)Ci; g.sBk = (unsigned)Co; g.sBn = 1; g.ldo = (unsigned)Co;
      g.bA = N * Ci; g.bB = N * Co; g.bO = Ci * Co;
      a_kc = false; b_nc = true;
      break;
  }
  // alignment of every 2-complex vector: even strides, even sizes along the vector
  const bool a_ok = (g.bA % 2 == 0) && (a_kc ? (g.sAm % 2 == 0 && g.K % 2 == 0) : (g.sAk % 2 == 0 && g.M % 2 == 0));
  const bool b_ok = (g.bB % 2 == 0) && (b_nc ? (g.sBk % 2 == 0 && g.N % 2 == 0) : (g.sBn % 2 == 0 && g.K % 2 == 0));
  if (!a_ok || !b_ok || B > 65535) return false;
  const long most = std::max<long>({(long)g.M * g.K, (long)g.K * g.N, (long)g.M * g.N});
  return 2 * most < 2147483647L;  // 32-bit offsets within a bin
}

double pass_bytes(const bl_conv_plan_s* p, const CgemmArgs& g) {
  const double ob = p->bf16 ? 4.0 : 8.0;  // bytes per stored operand element
  return (double)p->kept * (ob * ((double)g.M * g.K + (double)g.K * g.N) + 8.0 * g.M * g.N);
}

// Tile counts of a pass on BM x BN tiles and `splits` k ranges of whole
// stages (partial outputs split_stride = bins x M x N apart); returns the
// number of k ranges that hold stages.
int split_k_tiles(CgemmArgs& g, int BM, int BN, int splits, unsigned long long bins) {
  g.tiles_n = (g.N + BN - 1) / BN;
  g.tiles = ((g.M + BM - 1) / BM) * g.tiles_n;
  g.kper = ((g.K + splits - 1) / splits + kBK - 1) / kBK * kBK;
  g.split_stride = bins * (unsigned long long)g.M * g.N;
  return (g.K + g.kper - 1) / g.kper;
}

}  // namespace

// Tiled path: needs 16-byte aligned pairs of complex values along the
// contiguous dimension of each operand; returns BL_ERR_UNSUPPORTED otherwise.
bl_status_t launch_contract_tiled(const bl_conv_plan_s* p, Contract which, const void* A, const void* Bm,
                                  float2* O, float2* part, hipStream_t s, int parts) {
  CgemmArgs g;
  if (!tiled_args(p, which, g)) return BL_ERR_UNSUPPORTED;
  const unsigned long long B = p->kept;
  BlContractTiling t = p->ct[which == Contract::Forward ? 0 : which == Contract::GradInput ? 1 : 2];
  if (parts > 1) t.splits = parts, t.ks = 1;
  const int BM = t.bm, BN = t.bn;
  const int tiles_m = (g.M + BM - 1) / BM;
  g.tiles_n = (g.N + BN - 1) / BN;
  g.tiles = tiles_m * g.tiles_n;
  const unsigned long long total = B * (unsigned long long)g.M * g.N;  // complex outputs
  int splits = t.splits;
  g.kper = (g.K + splits - 1) / splits;
  g.kper = (g.kper + kBK - 1) / kBK * kBK;
  splits = (g.K + g.kper - 1) / g.kper;
  if (parts > 1 && splits != parts) return BL_ERR_UNSUPPORTED;
  if (parts <= 1 && total % 2 != 0) splits = 1, g.kper = g.K;  // the reduction works on pairs
  g.split_stride = total;
  float2* dst = splits > 1 ? part : O;
  // (tile, bin) pairs as a 2-D grid; the kernel renumbers them per XCD
  dim3 grid((unsigned)g.tiles, (unsigned)B, (unsigned)splits);
  const double flops = 8.0 * B * g.M * g.N * g.K;
  const double bytes = pass_bytes(p, g);
  const char* name = which == Contract::Forward ? "contract_fwd"
                     : which == Contract::GradInput ? "contract_dgrad" : "contract_wgrad";
  bl_status_t st = BL_ERR_UNSUPPORTED;
#define BL_GO(BMV, BNV, AK, BN_, CJ)                                                                        \
  st = timed_launch(name, bytes, flops, s, [&](hipEvent_t e0, hipEvent_t e1) {                               \
    if (p->bf16)                                                                                             \
      hipExtLaunchKernelGGL((k_cgemm<BMV, BNV, AK, BN_, CJ, true, 1>), grid, dim3(256), 0, s, e0, e1, 0, A, Bm, dst, g); \
    else if (t.ks == 2)                                                                                      \
      hipExtLaunchKernelGGL((k_cgemm<BMV, BNV, AK, BN_, CJ, false, 2>), grid, dim3(512), 0, s, e0, e1, 0, A, Bm, dst, g); \
    else                                                                                                     \
      hipExtLaunchKernelGGL((k_cgemm<BMV, BNV, AK, BN_, CJ, false, 1>), grid, dim3(256), 0, s, e0, e1, 0, A, Bm, dst, g); \
  })
#define BL_SHAPES(AK, BN_, CJ)                       \
  if (BM == 128 && BN == 64) BL_GO(128, 64, AK, BN_, CJ); \
  else if (BM == 64 && BN == 64) BL_GO(64, 64, AK, BN_, CJ); \
  else if (BM == 128 && BN == 32) BL_GO(128, 32, AK, BN_, CJ); \
  else if (BM == 64 && BN == 32) BL_GO(64, 32, AK, BN_, CJ);
  if (which == Contract::Forward) {
    BL_SHAPES(true, true, true)
  } else if (which == Contract::GradInput) {
    BL_SHAPES(true, false, false)
  } else {
    BL_SHAPES(false, true, true)
  }
#undef BL_SHAPES
#undef BL_GO
  if (st != BL_OK || splits == 1 || parts > 1) return st;
  const unsigned long long n4 = total / 2;
  const unsigned long long blocks = (n4 + 255) / 256;
  return timed_launch("contract_reduce", 8.0 * total * (splits + 1), 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
    hipExtLaunchKernelGGL(k_split_reduce, dim3((unsigned)blocks), dim3(256), 0, s, e0, e1, 0,
                       reinterpret_cast<const float4*>(part), reinterpret_cast<float4*>(O), n4, splits);
  });
}

bl_status_t launch_contract_bwd_pair(const bl_conv_plan_s* p, const void* DY, const void* W, float2* DX,
                                     const void* X, float2* DW, hipStream_t s) {
  if (p->bp_s1 < 1 || p->bp_s2 < 1) return BL_ERR_UNSUPPORTED;
  if (contract_is_thin(p, Contract::GradInput) || contract_is_thin(p, Contract::GradWeight)) return BL_ERR_UNSUPPORTED;
  CgemmArgs g1, g2;
  if (!tiled_args(p, Contract::GradInput, g1) || !tiled_args(p, Contract::GradWeight, g2)) return BL_ERR_UNSUPPORTED;
  // the plan split the pass with more k stages so that both passes' tiles take
  // about the same time: with unequal k lengths the long tiles end up sharing
  // CUs with short ones and finish last (a 4-fold ratio made the launch 70 %
  // slower than two launches; split 4 ways it is 17 % faster)
  const int BM = p->bp_bm, BN = p->bp_bn;
  const unsigned long long B = p->kept;
  if (split_k_tiles(g1, BM, BN, p->bp_s1, B) != p->bp_s1 || split_k_tiles(g2, BM, BN, p->bp_s2, B) != p->bp_s2)
    return BL_ERR_UNSUPPORTED;
  const unsigned long long n1 = (unsigned long long)g1.tiles * B, n2 = (unsigned long long)g2.tiles * B;
  if (n1 * p->bp_s1 + n2 * p->bp_s2 >= 2147483647ULL) return BL_ERR_UNSUPPORTED;
  const double flops = 8.0 * p->kept * ((double)g1.M * g1.N * g1.K + (double)g2.M * g2.N * g2.K);
  const double bytes = pass_bytes(p, g1) + pass_bytes(p, g2);
  const dim3 grid((unsigned)(n1 * p->bp_s1 + n2 * p->bp_s2));
  const unsigned t1 = (unsigned)n1, s1 = (unsigned)p->bp_s1, t2 = (unsigned)n2;
  bl_status_t st = BL_ERR_UNSUPPORTED;
#define BL_GO(BMV, BNV)                                                                                         \
  st = timed_launch("contract_bwd", bytes, flops, s, [&](hipEvent_t e0, hipEvent_t e1) {                       \
    if (p->bf16)                                                                                                \
      hipExtLaunchKernelGGL((k_cgemm_bwd<BMV, BNV, true>), grid, dim3(256), 0, s, e0, e1, 0, DY, W, DX, g1, X, DY, \
                            DW, g2, t1, s1, t2);                                                                \
    else                                                                                                        \
      hipExtLaunchKernelGGL((k_cgemm_bwd<BMV, BNV, false>), grid, dim3(256), 0, s, e0, e1, 0, DY, W, DX, g1, X,   \
                            DY, DW, g2, t1, s1, t2);                                                            \
  })
  if (BM == 128 && BN == 64) BL_GO(128, 64);
  else if (BM == 64 && BN == 64) BL_GO(64, 64);
  else if (BM == 128 && BN == 32) BL_GO(128, 32);
  else if (BM == 64 && BN == 32) BL_GO(64, 32);
#undef BL_GO
  return st;
}

bl_status_t launch_split_reduce(const float2* part, float2* out, unsigned long long n, int splits, hipStream_t s) {
  if (n % 2 != 0) return BL_ERR_UNSUPPORTED;  // summed as pairs of complex values
  const unsigned long long n4 = n / 2;
  const unsigned long long blocks = (n4 + 255) / 256;
  return timed_launch("contract_reduce", 8.0 * n * (splits + 1), 0.0, s, [&](hipEvent_t e0, hipEvent_t e1) {
    hipExtLaunchKernelGGL(k_split_reduce, dim3((unsigned)blocks), dim3(256), 0, s, e0, e1, 0,
                          reinterpret_cast<const float4*>(part), reinterpret_cast<float4*>(out), n4, splits);
  });
}

}  // namespace blc
