// C ABI compute entry points, stage dispatch and per-kernel timing.
#include <mutex>
#include <utility>
#include <vector>

#include "common.hpp"

namespace blc {

// ---------------------------------------------------------------------------
// Per-kernel timing
// ---------------------------------------------------------------------------
namespace {
struct Profiler {
  std::mutex mu;
  bool on = false;
  int cap = 0, used = 0;
  std::vector<hipEvent_t> ev;
  std::vector<const char*> names;
  std::vector<double> bytes, flops;
} g_prof;
}  // namespace

int prof_slot(const char* name, double bytes, double flops) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (!g_prof.on || g_prof.used >= g_prof.cap) return -1;
  g_prof.names[g_prof.used] = name;
  g_prof.bytes[g_prof.used] = bytes;
  g_prof.flops[g_prof.used] = flops;
  return g_prof.used++;
}

hipEvent_t prof_event(int slot, int end) { return g_prof.ev[2 * slot + end]; }

// ---------------------------------------------------------------------------
// Stage dispatch: the fast transform for the shape when there is one, else
// the direct pruned DFT.
// ---------------------------------------------------------------------------
bl_status_t launch_spec_fwd(const bl_conv_plan_s* p, const float* in, void* out, long P, int Hin, int Win, int oi,
                            int oj, hipStream_t s) {
  if (p->Lh == 1) {
    bl_status_t st = launch_bluestein_fwd(p, in, out, P, Win, oj, s);
    if (st != BL_ERR_UNSUPPORTED) return st;
  } else {
    bl_status_t st = launch_fft2_fwd(p, in, out, P, Hin, Win, oi, oj, s);
    if (st != BL_ERR_UNSUPPORTED) return st;
  }
  return launch_spec_fwd_direct(p, in, out, P, Hin, Win, oi, oj, s);
}

bl_status_t launch_contract(const bl_conv_plan_s* p, Contract which, const void* A, const void* Bm, float2* O,
                            float2* part, hipStream_t s) {
  bl_status_t st = BL_ERR_UNSUPPORTED;
  if (contract_is_thin(p, which)) st = launch_contract_thin(p, which, A, Bm, O, s);
  if (st != BL_ERR_UNSUPPORTED) return st;
  st = launch_contract_tiled(p, which, A, Bm, O, part, s);
  if (st != BL_ERR_UNSUPPORTED) return st;
  return launch_contract_generic(p, which, A, Bm, O, s);
}

bl_status_t launch_spec_inv(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OH, int OW, int ci,
                            int cj, hipStream_t s, int nsplit, float2* tmp) {
  if (nsplit > 1) {
    const size_t n = (size_t)p->kept * P;
    if (p->Lh > 1) {
      const bl_status_t st = launch_fft2_inv(p, in, out, P, OH, OW, ci, cj, s, nsplit, n);
      if (st != BL_ERR_UNSUPPORTED) return st;
    }
    if (!tmp) return BL_ERR_INVALID_ARG;
    const bl_status_t st = launch_split_reduce(in, tmp, n, nsplit, s);
    if (st != BL_OK) return st;
    in = tmp;
  }
  if (p->Lh == 1) {
    bl_status_t st = launch_bluestein_inv(p, in, out, P, OW, cj, s);
    if (st != BL_ERR_UNSUPPORTED) return st;
  } else {
    bl_status_t st = launch_fft2_inv(p, in, out, P, OH, OW, ci, cj, s);
    if (st != BL_ERR_UNSUPPORTED) return st;
  }
  return launch_spec_inv_direct(p, in, out, P, OH, OW, ci, cj, s);
}

namespace {
inline float2* ws_at(void* ws, size_t off) { return reinterpret_cast<float2*>(static_cast<char*>(ws) + off); }
// a stored spectrum (complex64 or bfloat16 pairs, as the plan says)
inline void* spec_at(void* ws, size_t off) { return static_cast<char*>(ws) + off; }

#define BL_TRY(expr)                    \
  do {                                  \
    bl_status_t st_ = (expr);           \
    if (st_ != BL_OK) return st_;       \
  } while (0)


}  // namespace
}  // namespace blc

using namespace blc;

// ---------------------------------------------------------------------------
// C ABI compute entry points
// ---------------------------------------------------------------------------
extern "C" bl_status_t bl_conv_forward(bl_conv_plan_t p, const float* x, const float* w, float* y, void* ws,
                                       unsigned flags, void* stream) {
  if (!p || !y || !ws) return BL_ERR_INVALID_ARG;
  if (flags & ~(BL_REUSE_X | BL_REUSE_W)) return BL_ERR_INVALID_ARG;
  if ((!(flags & BL_REUSE_X) && !x) || (!(flags & BL_REUSE_W) && !w)) return BL_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* X = spec_at(ws, p->off_X);
  void* Wf = spec_at(ws, p->off_W);
  float2* T = ws_at(ws, p->off_T);
  float2* CP = ws_at(ws, p->off_CPart);
  // the contraction and the output inverse; a split contraction leaves
  // partial spectra that the 2-D inverse adds as it loads them
  auto contract_invert = [&]() -> bl_status_t {
    if (p->fwd_split > 1 && p->Lh > 1) {
      const bl_status_t st = launch_contract_tiled(p, Contract::Forward, X, Wf, T, CP, s, p->fwd_split);
      if (st == BL_OK) return launch_spec_inv(p, CP, y, (long)p->N * p->Cout, p->Ho, p->Wo, 0, 0, s, p->fwd_split, T);
      if (st != BL_ERR_UNSUPPORTED) return st;
    }
    BL_TRY(launch_contract(p, Contract::Forward, X, Wf, T, CP, s));
    return launch_spec_inv(p, T, y, (long)p->N * p->Cout, p->Ho, p->Wo, 0, 0, s);
  };
  const bool small = p->fused_fwd && small_fwd_eligible(p);
  if (!(flags & (BL_REUSE_W | BL_REUSE_X)) && !small && p->Lh > 1) {
    // input and filter transforms in one launch where the 2-D fast path has it
    const bl_status_t st = launch_fft2_fwd_filt(p, x, X, (long)p->N * p->Cin, p->Hi, p->Wi, p->pt, p->pl, w, Wf, s);
    if (st == BL_OK) return contract_invert();
    if (st != BL_ERR_UNSUPPORTED) return st;
  }
  if (!(flags & BL_REUSE_W)) BL_TRY(launch_spec_filt(p, w, Wf, s));
  if (small && !(flags & BL_REUSE_X)) {
    const bl_status_t st = launch_small_fwd(p, x, static_cast<const float2*>(Wf), y, static_cast<float2*>(X), s);
    if (st != BL_ERR_UNSUPPORTED) return st;
  }
  if (!(flags & BL_REUSE_X))
    BL_TRY(launch_spec_fwd(p, x, X, (long)p->N * p->Cin, p->Hi, p->Wi, p->pt, p->pl, s));
  return contract_invert();
}

extern "C" bl_status_t bl_conv_backward_input(bl_conv_plan_t p, const float* dy, const float* w, float* dx,
                                              void* ws, unsigned flags, void* stream) {
  if (!p || !dy || !dx || !ws) return BL_ERR_INVALID_ARG;
  if (flags & ~BL_REUSE_W) return BL_ERR_INVALID_ARG;
  if (!(flags & BL_REUSE_W) && !w) return BL_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* Wf = spec_at(ws, p->off_W);
  void* DY = spec_at(ws, p->off_DY);
  float2* T = ws_at(ws, p->off_T);
  BL_TRY(launch_spec_fwd(p, dy, DY, (long)p->N * p->Cout, p->Ho, p->Wo, 0, 0, s));
  if (!(flags & BL_REUSE_W)) BL_TRY(launch_spec_filt(p, w, Wf, s));
  BL_TRY(launch_contract(p, Contract::GradInput, DY, Wf, T, ws_at(ws, p->off_CPart), s));
  return launch_spec_inv(p, T, dx, (long)p->N * p->Cin, p->Hi, p->Wi, p->pt, p->pl, s);
}

extern "C" bl_status_t bl_conv_backward_weight(bl_conv_plan_t p, const float* x, const float* dy, float* dw,
                                               void* ws, unsigned flags, void* stream) {
  if (!p || !dw || !ws) return BL_ERR_INVALID_ARG;
  if (flags & ~(BL_REUSE_X | BL_REUSE_DY)) return BL_ERR_INVALID_ARG;
  if ((!(flags & BL_REUSE_X) && !x) || (!(flags & BL_REUSE_DY) && !dy)) return BL_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* X = spec_at(ws, p->off_X);
  void* DY = spec_at(ws, p->off_DY);
  float2* DW = ws_at(ws, p->off_DW);
  if (!(flags & BL_REUSE_X))
    BL_TRY(launch_spec_fwd(p, x, X, (long)p->N * p->Cin, p->Hi, p->Wi, p->pt, p->pl, s));
  if (!(flags & BL_REUSE_DY))
    BL_TRY(launch_spec_fwd(p, dy, DY, (long)p->N * p->Cout, p->Ho, p->Wo, 0, 0, s));
  BL_TRY(launch_contract(p, Contract::GradWeight, X, DY, DW, ws_at(ws, p->off_CPart), s));
  return launch_wgrad_idft(p, DW, dw, reinterpret_cast<float*>(ws_at(ws, p->off_Part)), s);
}

extern "C" bl_status_t bl_conv_backward(bl_conv_plan_t p, const float* dy, const float* w, const float* x,
                                        float* dx, float* dw, void* ws, unsigned flags, void* stream) {
  if (!p || !dx || !dw || !ws) return BL_ERR_INVALID_ARG;
  if (flags & ~(BL_REUSE_X | BL_REUSE_W | BL_REUSE_DY)) return BL_ERR_INVALID_ARG;
  if ((!(flags & BL_REUSE_DY) && !dy) || (!(flags & BL_REUSE_W) && !w) || (!(flags & BL_REUSE_X) && !x))
    return BL_ERR_INVALID_ARG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* X = spec_at(ws, p->off_X);
  void* Wf = spec_at(ws, p->off_W);
  void* DY = spec_at(ws, p->off_DY);
  float2* T = ws_at(ws, p->off_T);
  float2* DW = ws_at(ws, p->off_DW);
  if (!(flags & BL_REUSE_DY))
    BL_TRY(launch_spec_fwd(p, dy, DY, (long)p->N * p->Cout, p->Ho, p->Wo, 0, 0, s));
  if (!(flags & BL_REUSE_W)) BL_TRY(launch_spec_filt(p, w, Wf, s));
  if (!(flags & BL_REUSE_X))
    BL_TRY(launch_spec_fwd(p, x, X, (long)p->N * p->Cin, p->Hi, p->Wi, p->pt, p->pl, s));
  // the paired launch writes a pass that it splits along k as partial spectra
  // (contraction-partials area), which the inverse transform adds
  float2* CP = ws_at(ws, p->off_CPart);
  int s1 = p->bp_s1, s2 = p->bp_s2;
  const bl_status_t st = launch_contract_bwd_pair(p, DY, Wf, s1 > 1 ? CP : T, X, s2 > 1 ? CP : DW, s);
  if (st == BL_ERR_UNSUPPORTED) {
    s1 = s2 = 1;
    BL_TRY(launch_contract(p, Contract::GradInput, DY, Wf, T, CP, s));
    BL_TRY(launch_contract(p, Contract::GradWeight, X, DY, DW, CP, s));
  } else if (st != BL_OK) {
    return st;
  }
  float* part = reinterpret_cast<float*>(ws_at(ws, p->off_Part));
  const long P = (long)p->N * p->Cin;
  if (p->Lh > 1) {
    // both inverses in one launch where the 2-D fast path and the sliced
    // weight-gradient path allow it
    const bl_status_t si = launch_fft2_inv_wgrad(p, s1 > 1 ? CP : T, dx, P, p->Hi, p->Wi, p->pt, p->pl, s1,
                                                 (size_t)p->kept * P, s2 > 1 ? CP : DW, dw, part, s2, s);
    if (si != BL_ERR_UNSUPPORTED) return si;
  }
  BL_TRY(launch_spec_inv(p, s1 > 1 ? CP : T, dx, P, p->Hi, p->Wi, p->pt, p->pl, s, s1, T));
  return launch_wgrad_idft(p, s2 > 1 ? CP : DW, dw, part, s, s2, DW);
}

// ---------------------------------------------------------------------------
// Forward pass without any allocation: the spectra live in a fixed static
// device array instead of a caller workspace.
// ---------------------------------------------------------------------------
constexpr size_t kNoAllocBytes = (size_t)64 << 20;  // the array's size on each device
static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

namespace blc {
namespace {

// Address of `scratch` on the current device.  In host code the array's name
// is a host-side stand-in, not a device address: only the pointer
// hipGetSymbolAddress returns (looked up once per device, with that device
// current) is ever passed to kernels.
std::mutex g_scratch_mu;
std::vector<std::pair<int, void*>> g_scratch_at;

bl_status_t scratch_on_current_device(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return BL_ERR_HIP;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  for (const auto& e : g_scratch_at)
    if (e.first == dev) {
      *out = e.second;
      return BL_OK;
    }
  void* ptr = nullptr;
  if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return BL_ERR_HIP;
  g_scratch_at.emplace_back(dev, ptr);
  *out = ptr;
  return BL_OK;
}

inline size_t up256(size_t n) { return (n + 255) / 256 * 256; }

// The transforms that need no plan table: the 2-D mixed-radix kernels where
// the grid has them, else the direct DFT (whose blocks compute their roots of
// unity).  1-D plans take the direct DFT (the chirp-z kernels use tables).
bl_status_t spec_fwd_no_tables(const bl_conv_plan_s* p, const float* in, void* out, long P, int Hin, int Win,
                               int oi, int oj, hipStream_t s) {
  if (p->Lh != 1) {
    const bl_status_t st = launch_fft2_fwd(p, in, out, P, Hin, Win, oi, oj, s);
    if (st != BL_ERR_UNSUPPORTED) return st;
  }
  return launch_spec_fwd_direct(p, in, out, P, Hin, Win, oi, oj, s);
}

bl_status_t spec_inv_no_tables(const bl_conv_plan_s* p, const float2* in, float* out, long P, int OH, int OW,
                               int ci, int cj, hipStream_t s) {
  if (p->Lh != 1) {
    const bl_status_t st = launch_fft2_inv(p, in, out, P, OH, OW, ci, cj, s);
    if (st != BL_ERR_UNSUPPORTED) return st;
  }
  return launch_spec_inv_direct(p, in, out, P, OH, OW, ci, cj, s);
}

}  // namespace
}  // namespace blc

extern "C" bl_status_t bl_conv_forward_noalloc(bl_conv_plan_t p, const float* x, const float* w, float* y,
                                               void* stream) {
  if (!p || !x || !w || !y) return BL_ERR_INVALID_ARG;
  // layout inside the array: X, W, the output spectrum, the k-split partials
  const size_t sb = p->bf16 ? 4 : 8, B = (size_t)p->kept;
  const size_t nX = up256(B * p->N * p->Cin * sb), nW = up256(B * p->Cin * p->Cout * sb);
  const size_t nT = up256(B * p->N * p->Cout * 8);
  const size_t nP = p->ct[0].splits > 1 ? up256((size_t)p->ct[0].splits * B * p->N * p->Cout * 8) : 0;
  if (nX + nW + nT + nP > ::kNoAllocBytes) return BL_ERR_WORKSPACE_TOO_SMALL;
  void* base = nullptr;
  BL_TRY(scratch_on_current_device(&base));
  char* b = static_cast<char*>(base);
  void* X = b;
  void* Wf = b + nX;
  float2* T = reinterpret_cast<float2*>(b + nX + nW);
  float2* part = reinterpret_cast<float2*>(b + nX + nW + nT);
  hipStream_t s = static_cast<hipStream_t>(stream);
  BL_TRY(launch_spec_filt(p, w, Wf, s, /*use_table=*/false));
  if (p->fused_fwd && small_fwd_eligible(p)) {
    const bl_status_t st = launch_small_fwd(p, x, static_cast<const float2*>(Wf), y, static_cast<float2*>(X), s);
    if (st != BL_ERR_UNSUPPORTED) return st;
  }
  BL_TRY(spec_fwd_no_tables(p, x, X, (long)p->N * p->Cin, p->Hi, p->Wi, p->pt, p->pl, s));
  BL_TRY(launch_contract(p, Contract::Forward, X, Wf, T, part, s));
  return spec_inv_no_tables(p, T, y, (long)p->N * p->Cout, p->Ho, p->Wo, 0, 0, s);
}

// ---------------------------------------------------------------------------
// Profiling entry points
// ---------------------------------------------------------------------------
extern "C" bl_status_t bl_profile_begin(int capacity) {
  if (capacity <= 0) return BL_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if ((int)g_prof.ev.size() < 2 * capacity) {
    for (hipEvent_t e : g_prof.ev) (void)hipEventDestroy(e);
    g_prof.ev.assign(2 * capacity, nullptr);
    for (auto& e : g_prof.ev)
      if (hipEventCreate(&e) != hipSuccess) return BL_ERR_HIP;
  }
  g_prof.names.assign(capacity, nullptr);
  g_prof.bytes.assign(capacity, 0.0);
  g_prof.flops.assign(capacity, 0.0);
  g_prof.cap = capacity;
  g_prof.used = 0;
  g_prof.on = true;
  return BL_OK;
}

extern "C" bl_status_t bl_profile_end(void) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  g_prof.on = false;
  return BL_OK;
}

extern "C" int bl_profile_count(void) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  return g_prof.used;
}

extern "C" bl_status_t bl_profile_get(int i, const char** kernel, float* ms, double* bytes, double* flops) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (i < 0 || i >= g_prof.used) return BL_ERR_INVALID_ARG;
  if (kernel) *kernel = g_prof.names[i];
  if (bytes) *bytes = g_prof.bytes[i];
  if (flops) *flops = g_prof.flops[i];
  if (ms) {
    if (hipEventElapsedTime(ms, g_prof.ev[2 * i], g_prof.ev[2 * i + 1]) != hipSuccess) return BL_ERR_HIP;
  }
  return BL_OK;
}

extern "C" bl_status_t bl_profile_release(void) {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  for (hipEvent_t e : g_prof.ev) (void)hipEventDestroy(e);
  g_prof.ev.clear();
  g_prof.names.clear();
  g_prof.cap = g_prof.used = 0;
  g_prof.on = false;
  return BL_OK;
}
