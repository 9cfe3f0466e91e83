// Internal declarations shared by the kernel files and the entry points.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <functional>
#include <vector>

#include "plan.hpp"

namespace blc {

constexpr int kThreads = 256;

// bfloat16 bit pattern of x (round to nearest, ties to even; finite inputs).
__device__ __forceinline__ unsigned bf16_bits(float x) {
  const unsigned u = __float_as_uint(x);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Stored spectra (X, W and DY in the workspace) hold complex64 values, or in
// plans with BL_DESC_BF16_SPECTRA bfloat16 pairs in 32-bit words (real
// part in the low half, imaginary part in the high half).  Kernels that
// produce or consume them are instantiated for both element types: float2
// and unsigned.
__device__ __forceinline__ void spec_put(float2* o, size_t i, float2 v) { o[i] = v; }
__device__ __forceinline__ void spec_put(unsigned* o, size_t i, float2 v) {
  o[i] = bf16_bits(v.x) | (bf16_bits(v.y) << 16);
}
__device__ __forceinline__ float2 spec_unpack(unsigned u) {
  return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xFFFF0000u));
}
__device__ __forceinline__ float2 spec_get(const float2* o, size_t i) { return o[i]; }
__device__ __forceinline__ float2 spec_get(const unsigned* o, size_t i) { return spec_unpack(o[i]); }
constexpr size_t kMaxLds = 64 * 1024;

// Orders the LDS accesses of one wave: everything a wave wrote before this
// point is seen by its later reads (LDS executes a wave's accesses in order;
// the fences keep the compiler from moving accesses across).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---- per-kernel timing (bl_profile_*) -------------------------------------
// Reserve a timing slot for one launch; -1 when profiling is off or full.
int prof_slot(const char* name, double bytes, double flops);
hipEvent_t prof_event(int slot, int end);

// Launch with optional event timing.  `bytes` and `flops` are the launch's
// algorithmic HBM traffic (compulsory reads + writes) and arithmetic, reported
// with the timing so that measurement tools can place it on a roofline.
// The launch takes a start and a stop event (null when not profiling), which
// hipExtLaunchKernelGGL stamps at the kernel's own start and end, so the
// timing is the kernel's execution time without the gaps around it.
template <typename Launch>
bl_status_t timed_launch(const char* name, double bytes, double flops, hipStream_t s, Launch&& launch) {
  const int slot = prof_slot(name, bytes, flops);
  (void)s;
  launch(slot >= 0 ? prof_event(slot, 0) : nullptr, slot >= 0 ? prof_event(slot, 1) : nullptr);
  if (hipGetLastError() != hipSuccess) return BL_ERR_HIP;
  return BL_OK;
}

// ---- device helpers ---------------------------------------------------------
__device__ inline float2 cmul(float2 a, float2 b) {
  return make_float2(fmaf(a.x, b.x, -a.y * b.y), fmaf(a.x, b.y, a.y * b.x));
}
__device__ inline float2 cconj(float2 a) { return make_float2(a.x, -a.y); }
__device__ inline float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ inline float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ inline float2 cscale(float2 a, float s) { return make_float2(a.x * s, a.y * s); }

// FFT row index of the r-th kept row.
__device__ inline int kept_row_d(int r, int r_h, int Lh, int R) { return r <= r_h ? r : r + (Lh - R); }

// ---- plan-owned device tables (tables.hip) ----------------------------------
// Returns the device copy, on the current device, of the table identified by
// `key`, building it with `build` (on the host) and uploading it on first use.
bl_status_t plan_table(const bl_conv_plan_s* p, const std::vector<long>& key,
                       const std::function<void(std::vector<float2>&)>& build, const float2** out);
long float_key(float x);  // bit pattern of x, for keys
// Allows kernel `kern` up to `bytes` of dynamic LDS on the current device
// (hipFuncAttributeMaxDynamicSharedMemorySize), once per kernel and device.
bl_status_t lds_opt_in(const void* kern, int bytes);
// Compute units of the current device (256 if the query fails).
int device_cus();

// ---- stage launchers --------------------------------------------------------
// Real planes [P][Hin][Win] placed at (oi, oj) of the grid -> kept spectrum
// out[b * P + p] (bin-major).
// `out` holds the plan's stored-spectrum type (complex64 or bfloat16 pairs).
bl_status_t launch_spec_fwd(const bl_conv_plan_s* p, const float* in, void* out, long P, int Hin, int Win,
                            int oi, int oj, hipStream_t s);
// Kept spectrum in[b * P + p] -> real planes [P][OH][OW] holding the grid
// window that starts at (ci, cj), scaled by 1 / (Lh Lw).  With nsplit > 1 the
// spectrum is the sum of nsplit partial spectra kept * P complex values apart
// (added in order while loading on the fast 2-D path, else first summed into
// tmp, which then holds the spectrum).
bl_status_t launch_spec_inv(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OH, int OW, int ci,
                            int cj, hipStream_t s, int nsplit = 1, float2* tmp = nullptr);
// Filter w [F][C][Kh][Kw] -> W[b][c][f] (stored-spectrum type).  The roots of
// unity come from the plan's device table (built on first use), or with
// use_table = false are computed by each block (no table, no allocation).
bl_status_t launch_spec_filt(const bl_conv_plan_s* p, const float* w, void* out, hipStream_t s,
                             bool use_table = true);
// The 2-D input transform of a forward pass (as launch_spec_fwd on the fast
// 2-D path) and the filter transform w -> wout (as launch_spec_filt) in one
// launch; BL_ERR_UNSUPPORTED (nothing enqueued) where either has no such path
// (only 3 x 3 filters are compiled for it).
bl_status_t launch_fft2_fwd_filt(const bl_conv_plan_s* p, const float* in, void* out, long P, int Hin, int Win,
                                 int oi, int oj, const float* w, void* wout, hipStream_t s);
// DW[b][c][f] -> dw [F][C][Kh][Kw]; `part` holds wg_chunks x Kh Kw x C F floats
// (times bp_s2 when the plan pairs the backward contractions).  With nsplit > 1
// DW is the sum of nsplit partial spectra kept * C * F complex values apart
// (their bin slices summed with the others on the sliced path, else first
// summed into tmp, which then holds the spectrum).
bl_status_t launch_wgrad_idft(const bl_conv_plan_s* p, const float2* DW, float* dw, float* part, hipStream_t s,
                              int nsplit = 1, float2* tmp = nullptr);

// Operands A and Bm are stored spectra (complex64 or bfloat16 pairs); the
// output O and the split-k partials are complex64.
enum class Contract { Forward, GradInput, GradWeight };
bl_status_t launch_contract(const bl_conv_plan_s* p, Contract which, const void* A, const void* Bm, float2* O,
                            float2* part, hipStream_t s);
// One of M, N, K at most 8: memory-bound, on the vector ALUs (thin.hip).
bool contract_is_thin(const bl_conv_plan_s* p, Contract which);
bl_status_t launch_contract_thin(const bl_conv_plan_s* p, Contract which, const void* A, const void* Bm,
                                 float2* O, hipStream_t s);
// Grad-input (DX = DY W) and grad-weight (DW = X^T conj(DY)) contractions in
// one launch where the plan pairs them (bp_s1, bp_s2 >= 1): a pass split
// s > 1 ways along k writes s partial spectra, kept * M * N complex values
// apart, to DX or DW, for the inverse transform to add; BL_ERR_UNSUPPORTED
// (nothing enqueued) otherwise.
bl_status_t launch_contract_bwd_pair(const bl_conv_plan_s* p, const void* DY, const void* W, float2* DX,
                                     const void* X, float2* DW, hipStream_t s);
// out[i] = sum over s < splits of part[s n + i] in order s = 0, 1, ... (n even).
bl_status_t launch_split_reduce(const float2* part, float2* out, unsigned long long n, int splits, hipStream_t s);
// Tiled, double-buffered fp32-MFMA contraction (aligned operands) and the
// generic one (any strides and sizes).
// parts > 1: split k into exactly that many ranges and leave the partial
// spectra in `part` (kept * M * N complex values apart) for the consumer to add.
bl_status_t launch_contract_tiled(const bl_conv_plan_s* p, Contract which, const void* A, const void* Bm,
                                  float2* O, float2* part, hipStream_t s, int parts = 0);
bl_status_t launch_contract_generic(const bl_conv_plan_s* p, Contract which, const void* A, const void* Bm,
                                    float2* O, hipStream_t s);

// Direct (pruned DFT) transforms: any grid; used where no fast path applies.
bl_status_t launch_spec_fwd_direct(const bl_conv_plan_s* p, const float* in, void* out, long P, int Hin, int Win,
                                   int oi, int oj, hipStream_t s);
bl_status_t launch_spec_inv_direct(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OH, int OW,
                                   int ci, int cj, hipStream_t s);

// 1-D transforms by Bluestein's chirp-z algorithm over a power-of-two FFT.
// Return BL_ERR_UNSUPPORTED when the shape is outside the fast path.
bl_status_t launch_bluestein_fwd(const bl_conv_plan_s* p, const float* in, void* out, long P, int Win, int oj,
                                 hipStream_t s);
bl_status_t launch_bluestein_inv(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OW, int cj,
                                 hipStream_t s);

// Fused small-map forward: x -> y in one kernel (W: the stored filter
// spectrum; X: where the input spectrum is stored for map reuse).
bool small_fwd_eligible(const bl_conv_plan_s* p);
bl_status_t launch_small_fwd(const bl_conv_plan_s* p, const float* x, const float2* Wf, float* y, float2* X,
                             hipStream_t s);

// 2-D transforms on (2 MH) x (2 MW) grids with MH, MW odd (mixed radix 2 x odd).
bl_status_t launch_fft2_fwd(const bl_conv_plan_s* p, const float* in, void* out, long P, int Hin, int Win, int oi,
                            int oj, hipStream_t s);
bl_status_t launch_fft2_inv(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OH, int OW, int ci,
                            int cj, hipStream_t s, int nsplit = 1, size_t pstride = 0);
// The input-gradient inverse (as launch_fft2_inv) and the weight-gradient
// inverse DFT (as launch_wgrad_idft on its sliced path, wnsplit partial
// spectra of DW) in one launch, then the slice sum; 3 x 3 filters;
// BL_ERR_UNSUPPORTED (nothing enqueued) where either has no such path.
bl_status_t launch_fft2_inv_wgrad(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OH, int OW,
                                  int ci, int cj, int nsplit, size_t pstride, const float2* DW, float* dw, float* part,
                                  int wnsplit, hipStream_t s);

}  // namespace blc
