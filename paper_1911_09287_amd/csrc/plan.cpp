// Host plan of the band-limited convolution: geometry, kept band, workspace.
// Pure host code; makes no HIP call, so plans can be built and inspected on a
// machine without a GPU.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>

#include "plan.hpp"

namespace {

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Kept count after peeling t L-shaped layers (Sec. 3.2.2, Fig. 2): rows with
// |s(u)| <= Lh/2 - t times columns v <= Lw/2 - t of the half plane.
long kept_after(int t, int Lh, int Lw, int ndim) {
  if (ndim == 1) return (long)(Lw / 2 + 1 - t);
  int r_h = Lh / 2 - t, r_w = Lw / 2 - t;
  return (long)bl_rows_for_radius(r_h, Lh) * (long)(r_w + 1);
}

}  // namespace

extern "C" bl_status_t bl_conv_plan_create(bl_conv_plan_t* out, const bl_conv_desc_t* d) {
  if (!out || !d) return BL_ERR_INVALID_ARG;
  *out = nullptr;
  if (d->ndim != 1 && d->ndim != 2) return BL_ERR_INVALID_ARG;
  if (d->N <= 0 || d->C_in <= 0 || d->C_out <= 0 || d->H <= 0 || d->K <= 0) return BL_ERR_INVALID_ARG;
  if (d->pad_lo[0] < 0 || d->pad_hi[0] < 0 || d->pad_lo[1] < 0 || d->pad_hi[1] < 0) return BL_ERR_INVALID_ARG;
  if (!(d->c >= 0.0 && d->c < 1.0)) return BL_ERR_INVALID_ARG;  // also rejects NaN
  if (d->fft_h < 0 || d->fft_w < 0) return BL_ERR_INVALID_ARG;
  if (d->flags & ~(BL_DESC_BF16_SPECTRA | BL_DESC_FUSED_FORWARD)) return BL_ERR_INVALID_ARG;
  if (d->ndim == 1 && (d->W != 1 || d->pad_lo[1] != 0 || d->pad_hi[1] != 0 || d->fft_w > 1))
    return BL_ERR_INVALID_ARG;
  if (d->ndim == 2 && d->W <= 0) return BL_ERR_INVALID_ARG;
  if (d->K > 8) return BL_ERR_UNSUPPORTED;

  bl_conv_plan_s* p = new (std::nothrow) bl_conv_plan_s();
  if (!p) return BL_ERR_OOM;
  p->desc = *d;
  p->ndim = d->ndim;
  p->bf16 = (d->flags & BL_DESC_BF16_SPECTRA) != 0;
  p->fused_fwd = (d->flags & BL_DESC_FUSED_FORWARD) != 0;
  p->N = d->N; p->Cin = d->C_in; p->Cout = d->C_out;
  if (d->ndim == 2) {
    p->Hi = d->H; p->Wi = d->W; p->Kh = d->K; p->Kw = d->K;
    p->pt = d->pad_lo[0]; p->pb = d->pad_hi[0]; p->pl = d->pad_lo[1]; p->pr = d->pad_hi[1];
  } else {
    p->Hi = 1; p->Wi = d->H; p->Kh = 1; p->Kw = d->K;
    p->pt = 0; p->pb = 0; p->pl = d->pad_lo[0]; p->pr = d->pad_hi[0];
  }
  p->Hp = p->Hi + p->pt + p->pb;
  p->Wp = p->Wi + p->pl + p->pr;
  p->Ho = p->Hp - p->Kh + 1;
  p->Wo = p->Wp - p->Kw + 1;
  if (p->Ho < 1 || p->Wo < 1) { delete p; return BL_ERR_INVALID_ARG; }
  if (d->ndim == 2) {
    p->Lh = d->fft_h ? d->fft_h : p->Hp;
    p->Lw = d->fft_w ? d->fft_w : p->Wp;
  } else {
    p->Lh = 1;
    p->Lw = d->fft_h ? d->fft_h : p->Wp;
  }
  if (p->Lh < p->Hp || p->Lw < p->Wp) { delete p; return BL_ERR_INVALID_ARG; }
  if (p->Lw > 4096 || p->Lh > 4096) { delete p; return BL_ERR_UNSUPPORTED; }
  p->Wh = p->Lw / 2 + 1;
  p->total = (long)p->Lh * (long)p->Wh;

  // Rate -> layers: the fewest t with kept(t) <= (1 - c) * total, in double.
  int t_max = (d->ndim == 1) ? p->Wh - 1 : std::min(p->Lh / 2, p->Lw / 2);
  const double budget = (1.0 - d->c) * (double)p->total;
  int t = t_max;
  for (int tt = 0; tt <= t_max; ++tt) {
    if ((double)kept_after(tt, p->Lh, p->Lw, d->ndim) <= budget) { t = tt; break; }
  }
  p->t = t;
  if (d->ndim == 1) {
    p->r_h = 0;
    p->r_w = p->Wh - 1 - t;
    p->R = 1;
  } else {
    p->r_h = p->Lh / 2 - t;
    p->r_w = p->Lw / 2 - t;
    p->R = bl_rows_for_radius(p->r_h, p->Lh);
  }
  p->V = p->r_w + 1;
  p->kept = (long)p->R * p->V;
  // every compute call must find a kernel for the shape, so that a call that
  // fails has enqueued nothing: the contraction takes at most 65535 kept bins,
  // and the direct transforms (the fallback of every faster one) hold a plane
  // in at most 160 KB of LDS
  {
    const size_t tw = (size_t)(p->Lh + p->Lw) * 8;
    const size_t fwd = tw + ((size_t)p->Hi * p->V + 1) * 8 + (size_t)p->Hi * p->Wi * 4;
    const size_t inv = tw + ((size_t)p->R * p->V + 1 + (size_t)p->Hi * p->V + 1) * 8;
    if (p->kept > 65535 || fwd > 160 * 1024 || inv > 160 * 1024) { delete p; return BL_ERR_UNSUPPORTED; }
  }
  p->c_eff = 1.0 - (double)p->kept / (double)p->total;

  p->mask.assign((size_t)p->total, 0);
  for (int r = 0; r < p->R; ++r) {
    int u = bl_kept_row(r, p->r_h, p->Lh, p->R);
    for (int v = 0; v < p->V; ++v) p->mask[(size_t)u * p->Wh + v] = 1;
  }

  const size_t cb = 8;                  // complex64
  const size_t sb = p->bf16 ? 4 : cb;  // a stored spectrum's element: complex64 or a bfloat16 pair
  const size_t B = (size_t)p->kept;
  size_t o = 0;
  p->off_X = o;  o = align_up(o + B * p->N * p->Cin * sb, 256);
  p->off_W = o;  o = align_up(o + B * p->Cin * p->Cout * sb, 256);
  p->off_DY = o; o = align_up(o + B * p->N * p->Cout * sb, 256);
  p->off_T = o;  o = align_up(o + B * p->N * (size_t)std::max(p->Cin, p->Cout) * cb, 256);
  p->off_DW = o; o = align_up(o + B * p->Cin * p->Cout * cb, 256);
  // contraction tiling of the three passes, and the paired backward launch:
  // one tile shape and no k split of their own; the pass with more k stages is
  // split (2 to 4 ways) to the other's length
  {
    const long Bk = p->kept, N = p->N, Ci = p->Cin, Co = p->Cout;
    p->ct[0] = bl_contract_tiling(N, Co, Ci, Bk);
    p->ct[1] = bl_contract_tiling(N, Ci, Co, Bk);
    p->ct[2] = bl_contract_tiling(Ci, Co, N, Bk);
    p->bp_s1 = p->bp_s2 = 0;
    const BlContractTiling &t1 = p->ct[1], &t2 = p->ct[2];
    // one shape for both passes: theirs if they agree, else the finest tile
    p->bp_bm = t1.bm == t2.bm && t1.bn == t2.bn ? t1.bm : 64;
    p->bp_bn = t1.bm == t2.bm && t1.bn == t2.bn ? t1.bn : 32;
    if (t1.splits == 1 && t2.splits == 1) {
      const long st1 = (Co + 15) / 16, st2 = (N + 15) / 16;  // k stages: grad-input sums C_out, grad-weight N
      if (st1 == st2) {
        p->bp_s1 = p->bp_s2 = 1;
      } else if (st1 > st2 && st1 % st2 == 0 && st1 / st2 <= 4) {
        p->bp_s1 = (int)(st1 / st2), p->bp_s2 = 1;
      } else if (st2 > st1 && st2 % st1 == 0 && st2 / st1 <= 4) {
        p->bp_s1 = 1, p->bp_s2 = (int)(st2 / st1);
      }
      // a split pays while the paired tiles run in about one or two rounds
      // of the CUs' resident blocks (measured on the 64-channel layer: 2208
      // tiles of 64 x 32, 5 per CU, 5 us faster; at 4896 tiles 5 us slower)
      const int bm = p->bp_bm, bn = p->bp_bn;
      const long tiles1 = Bk * ((N + bm - 1) / bm) * ((Ci + bn - 1) / bn);
      const long tiles2 = Bk * ((Ci + bm - 1) / bm) * ((Co + bn - 1) / bn);
      const int resident = bm == 64 && bn == 32 ? 5 : bm == 128 && bn == 64 ? 2 : 3;  // blocks per CU
      if ((p->bp_s1 > 1 || p->bp_s2 > 1) && tiles1 * p->bp_s1 + tiles2 * p->bp_s2 > 2L * resident * 256)
        p->bp_s1 = p->bp_s2 = 0;
    }
  }
  // a forward contraction with no more tiles than CUs (run with two wave
  // groups per tile) is split along k instead, into up to 4 ranges of at least
  // 8 stages and at most 768 tiles in all, when the 2-D inverse can add the
  // partial spectra as it loads them (the 512-channel layer at c = 0.5: 192
  // tiles of 32 stages become 768 of 8)
  p->fwd_split = 1;
  {
    const BlContractTiling& t0 = p->ct[0];
    const long tiles0 = (long)p->kept * ((p->N + t0.bm - 1) / t0.bm) * ((p->Cout + t0.bn - 1) / t0.bn);
    const long st0 = (p->Cin + 15) / 16;
    if (p->Lh > 1 && t0.splits == 1 && t0.ks == 2)
      while (p->fwd_split < 4 && st0 % (2 * p->fwd_split) == 0 && st0 / (2 * p->fwd_split) >= 8 &&
             tiles0 * 2 * p->fwd_split <= 768)
        p->fwd_split *= 2;
  }
  // partial sums of the weight-gradient inverse DFT over bin slices: enough
  // slices for ~1024 blocks of 256 (c, f) pairs, at least 16 bins per slice,
  // whole batches of 8 bins, and a slice's weights [bins][taps, padded as the
  // kernels are instantiated] within kWgradSliceLds
  {
    const long Q = (long)p->Cin * p->Cout;
    const int T = p->Kh * p->Kw;
    const long tmax = T <= 9 ? T : T <= 16 ? 16 : T <= 32 ? 32 : 64;
    const long xblocks = (Q + 255) / 256;
    const long want = (1024 + xblocks - 1) / xblocks;
    long per = std::max<long>(16, (p->kept + want - 1) / want);
    const long cap = std::max<long>(8, kWgradSliceLds / (tmax * 8) / 8 * 8);
    per = std::min((per + 7) / 8 * 8, cap);
    const long chunks = (p->kept + per - 1) / per;
    p->wg_bins = (int)per;
    p->wg_chunks = (int)chunks;
    // 128 to 511 tiles of 16 x 16 channel pairs: one pass over all bins with
    // 2 or 4 groups of 256 threads per tile (k_wgrad_tile), at least 2048
    // waves, the bins' weights and the groups' sums within 64 KB of LDS each.
    // With more tiles one group per tile would sum every bin in series; the
    // bin slices above split that work instead.
    {
      const long tiles = (long)((p->Cin + 15) / 16) * ((p->Cout + 15) / 16);
      int ng = 2;
      while (ng < 4 && tiles * ng * 4 < 2048) ng *= 2;
      const int tm = wgrad_tmax(T);
      p->wg_groups = (tiles < 512 && tiles * ng * 4 >= 2048 && T <= 16 && p->kept * tm * 8 <= 64 * 1024 &&
                      (long)ng * 256 * tm * 4 <= 64 * 1024) ? ng : 0;
    }
    p->off_Part = o;
    // (k-split partial spectra of a paired backward launch count as more slices)
    o = align_up(o + (chunks > 1 ? (size_t)std::max(1, p->bp_s2) * chunks * Q * p->Kh * p->Kw * sizeof(float) : 0),
                 256);
  }
  // split-k partial tiles of the contraction (largest of the three passes and
  // of the paired backward launch)
  {
    const long Bk = p->kept, N = p->N, Ci = p->Cin, Co = p->Cout;
    size_t need = 0;
    const long mn[3] = {N * Co, N * Ci, Ci * Co};
    for (int i = 0; i < 3; ++i)
      if (p->ct[i].splits > 1) need = std::max(need, (size_t)p->ct[i].splits * Bk * mn[i] * cb);
    if (p->fwd_split > 1) need = std::max(need, (size_t)p->fwd_split * Bk * mn[0] * cb);
    if (p->bp_s1 > 1) need = std::max(need, (size_t)p->bp_s1 * Bk * mn[1] * cb);
    if (p->bp_s2 > 1) need = std::max(need, (size_t)p->bp_s2 * Bk * mn[2] * cb);
    p->off_CPart = o;
    o = align_up(o + need, 256);
  }
  p->ws_bytes = o;
  *out = p;
  return BL_OK;
}

extern "C" bl_status_t bl_conv_plan_destroy(bl_conv_plan_t p) {
  if (!p) return BL_ERR_INVALID_ARG;
  bl_plan_tables_free(p->tables);
  delete p;
  return BL_OK;
}

extern "C" bl_status_t bl_conv_plan_info(bl_conv_plan_t p, int* fft_h, int* fft_w, int* r_h, int* r_w,
                                         long* kept, long* total, double* c_eff) {
  if (!p) return BL_ERR_INVALID_ARG;
  if (fft_h) *fft_h = p->ndim == 1 ? p->Lw : p->Lh;
  if (fft_w) *fft_w = p->ndim == 1 ? 1 : p->Lw;
  if (r_h) *r_h = p->r_h;
  if (r_w) *r_w = p->r_w;
  if (kept) *kept = p->kept;
  if (total) *total = p->total;
  if (c_eff) *c_eff = p->c_eff;
  return BL_OK;
}

extern "C" bl_status_t bl_conv_plan_get_mask(bl_conv_plan_t p, unsigned char* m, size_t n) {
  if (!p || !m || n != (size_t)p->total) return BL_ERR_INVALID_ARG;
  std::memcpy(m, p->mask.data(), n);
  return BL_OK;
}

extern "C" bl_status_t bl_conv_plan_get_bins(bl_conv_plan_t p, int* u, int* v, size_t n) {
  if (!p || !u || !v || n != (size_t)p->kept) return BL_ERR_INVALID_ARG;
  size_t b = 0;
  for (int r = 0; r < p->R; ++r)
    for (int vv = 0; vv < p->V; ++vv, ++b) {
      u[b] = bl_kept_row(r, p->r_h, p->Lh, p->R);
      v[b] = vv;
    }
  return BL_OK;
}

extern "C" bl_status_t bl_conv_workspace_size(bl_conv_plan_t p, size_t* bytes) {
  if (!p || !bytes) return BL_ERR_INVALID_ARG;
  *bytes = p->ws_bytes;
  return BL_OK;
}

extern "C" bl_status_t bl_conv_workspace_layout(bl_conv_plan_t p, size_t* off_x, size_t* off_w, size_t* off_dy) {
  if (!p) return BL_ERR_INVALID_ARG;
  if (off_x) *off_x = p->off_X;
  if (off_w) *off_w = p->off_W;
  if (off_dy) *off_dy = p->off_DY;
  return BL_OK;
}

extern "C" const char* bl_status_string(bl_status_t s) {
  switch (s) {
    case BL_OK: return "ok";
    case BL_ERR_INVALID_ARG: return "invalid argument";
    case BL_ERR_UNSUPPORTED: return "unsupported configuration";
    case BL_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case BL_ERR_HIP: return "HIP error";
    case BL_ERR_OOM: return "out of host memory";
  }
  return "unknown status";
}
