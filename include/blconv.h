/*
 * blconv.h -- band-limited FFT convolution layer for AMD Instinct MI355X (gfx950).
 *
 * The layer of Dziedzic et al., "Band-limited Training and Inference for
 * Convolutional Neural Networks" (ICML 2019):
 *
 *   Sec. 3, Eq. (1)/(2)  y = F^-1{ (F_x M_c) . conj(F_w M_c) }: the spectra of
 *                        input and filter are multiplied element-wise after a
 *                        0/1 low-pass mask M_c, summed over input channels and
 *                        transformed back.  The layer computes cross-correlation
 *                        (the filter spectrum enters conjugated), like a
 *                        deep-learning convolution layer.
 *   Sec. 3.2.1           input and filter are zero-padded so that the circular
 *                        correlation of the FFT equals the linear one.
 *   Sec. 3.2.2, Fig. 2   only the rfft half plane [L_h][L_w/2+1] is kept; the band
 *                        shrinks in L-shaped layers from the top-left and
 *                        bottom-left corners: bin (u, v) is kept iff
 *                        |s(u)| <= r_h and v <= r_w, with s(u) the signed row
 *                        frequency, r_h = L_h/2 - t, r_w = L_w/2 - t (integer
 *                        halves).  In 1-D the kept set is the prefix v <= L/2 - t.
 *   Sec. 3.1, Sec. 4.1   c is the fraction of half-spectrum coefficients
 *                        discarded.  The number of peeled layers t is the
 *                        smallest t with kept(t) <= (1 - c) * total, evaluated in
 *                        IEEE double ("discard at least c"); if no t qualifies,
 *                        the most layers that can be peeled.
 *   Abstract, Sec. 1     the band limit holds in forward and back-propagation:
 *                        grad-input and grad-weight apply the same mask, so the
 *                        weight gradient is projected onto the kept frequencies.
 *   Sec. 3.2.3           map reuse: the spectra of the input and the filter
 *                        computed by the forward pass are kept (here: in the
 *                        caller's workspace) and reused by the backward passes.
 *
 * FFT grid: by default the padded input size, L_h = H + pad_lo[0] + pad_hi[0]
 * and L_w = W + pad_lo[1] + pad_hi[1] (1-D: L = length + pad_lo[0] + pad_hi[0]);
 * this is the smallest grid on which none of the three passes wraps around.
 * A larger grid (e.g. the map-reuse size N + max(K-1, G-1) of Sec. 3.2.3) may
 * be requested with fft_h / fft_w; it changes results only when c > 0.
 *
 * Layouts (all contiguous, fp32, PyTorch order):
 *   2-D: x [N][C_in][H][W], w [C_out][C_in][K][K], y and dy [N][C_out][Ho][Wo],
 *        dx [N][C_in][H][W], dw [C_out][C_in][K][K];
 *   1-D: x [N][C_in][L],    w [C_out][C_in][K],    y and dy [N][C_out][Lo],
 *        dx [N][C_in][L],   dw [C_out][C_in][K];
 *   with Ho = H + pad_lo[0] + pad_hi[0] - K + 1 (and likewise Wo, Lo); stride 1,
 *   no dilation, no groups, no bias.
 *
 * Ownership: the caller owns every device buffer (x, w, y, dy, dx, dw and the
 * workspace ws).  Creating and querying a plan makes no HIP call.  The plan
 * also owns small device tables, built in double precision on the host: those
 * of its 1-D transforms (chirps, the chirp filter's spectrum and twiddles:
 * under 100 KB), the roots of unity of the filter DFT (8 (L_h + L_w) bytes)
 * and the inverse-DFT weights of the weight gradient (8 K^2 bytes per kept
 * bin, K^2 -> K in 1-D).  The first compute call of
 * the plan that needs a table on a device uploads it there; that call
 * allocates and copies synchronously, so make each kind of call once outside
 * stream capture before capturing it.  Every other compute call allocates nothing,
 * makes no host synchronisation and enqueues its kernels on `stream` (a
 * hipStream_t, passed as void*; NULL = the default stream).
 * bl_conv_plan_destroy frees the tables (no kernel of the plan may still be
 * running).
 *
 * Errors: every call returns a bl_status_t.  Arguments are validated on the host
 * before anything is enqueued; a call that returns an error has enqueued no
 * kernel, except BL_ERR_HIP, which reports a failed launch (work enqueued before
 * it by the same call may have run).
 *
 * Threading: a plan's geometry is immutable after creation (the device tables
 * are built under a lock); calls with distinct workspaces may run
 * concurrently from several threads and streams.
 */
#ifndef BLCONV_H
#define BLCONV_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BL_OK = 0,
  BL_ERR_INVALID_ARG = 1,         /* null pointer, non-positive size, c outside [0,1), grid too small */
  BL_ERR_UNSUPPORTED = 2,         /* valid but outside what this library implements (e.g. K > 8) */
  BL_ERR_WORKSPACE_TOO_SMALL = 3, /* bl_conv_forward_noalloc: the plan's spectra exceed its static array */
  BL_ERR_HIP = 4,                 /* a HIP launch or runtime call failed */
  BL_ERR_OOM = 5                  /* host or device allocation failed */
} bl_status_t;

typedef struct {
  int ndim;          /* 1 or 2 */
  int N, C_in, C_out;
  int H, W;          /* 2-D: input height and width.  1-D: H = sequence length, W = 1 */
  int K;             /* filter size: K x K (2-D) or K taps (1-D); 1 <= K <= 8 */
  int pad_lo[2];     /* leading zeros: [0] rows (1-D: the sequence), [1] columns (1-D: 0) */
  int pad_hi[2];     /* trailing zeros, same axes */
  double c;          /* compression rate, 0 <= c < 1 */
  int fft_h, fft_w;  /* 0 = padded size; else an FFT grid at least the padded size (1-D: fft_h) */
  unsigned flags;    /* 0, or BL_DESC_BF16_SPECTRA and/or BL_DESC_FUSED_FORWARD */
} bl_conv_desc_t;

/* Descriptor flag: reduced-precision spectra (the paper's reduced-precision
 * arithmetic combined with band-limiting: Sec. 4.3 and the supplementary
 * section "Reduced Precision and Bandlimited Training").  The forward
 * transforms round the kept spectra X, W and DY to bfloat16 (round to nearest
 * even on the fp32 transform results; bfloat16 keeps fp32's exponent range,
 * which sums over many samples need) and store them as 32-bit words holding a
 * bfloat16 pair, real part in the low 16 bits, imaginary part in the high 16
 * bits: half the workspace those saved maps take in fp32.  Every channel
 * contraction multiplies the stored values exactly and accumulates in fp32
 * (the tiled path on the bf16 matrix cores); its outputs, the transforms'
 * arithmetic and the layer's inputs and outputs stay fp32.  Expected deviation
 * from the fp32 path: about 2e-3 relative (8 significant bits per operand). */
#define BL_DESC_BF16_SPECTRA 0x1u

/* Descriptor flag: fused small-map forward.  bl_conv_forward runs the filter
 * transform (unless W is reused) and then one kernel that takes x to y: per
 * sample and group of output channels it transforms the input planes, forms
 * the per-bin channel sums and transforms them back in on-chip memory, so the
 * input and output spectra do not pass through HBM as separate stages (X is
 * still stored in ws for the reuse flags).  It applies to 2-D plans with
 * complex64 spectra and at most 1024 kept bins whose per-channel working set
 * fits in 64 KB of LDS, and to calls that do not reuse X; otherwise the flag
 * has no effect.  The channel sums run on the vector ALUs and each block
 * transforms its sample's planes again per output-channel group: measured on
 * the 4x4, 8x8 and 16x16 workload layers it takes 1.6-11x the time of the
 * unfused forward, whose contraction runs on the matrix cores, so it is not
 * chosen unless requested. */
#define BL_DESC_FUSED_FORWARD 0x2u

typedef struct bl_conv_plan_s* bl_conv_plan_t;

/* Flags of the compute calls (map reuse, Sec. 3.2.3).  Every compute call
 * leaves in the workspace the spectra it computed: forward the input spectrum
 * X and the filter spectrum W, backward_input the output-gradient spectrum DY
 * and W, backward_weight X and DY, backward all three.  A REUSE flag skips
 * recomputing that
 * spectrum and reads the copy in the workspace instead; the caller asserts that
 * the tensor it came from has not changed since, which the library cannot
 * check.  The tensor pointer may then be NULL. */
#define BL_REUSE_X  0x1u  /* forward, backward_weight, backward: reuse X */
#define BL_REUSE_W  0x2u  /* forward, backward_input, backward: reuse W */
#define BL_REUSE_DY 0x4u  /* backward_weight, backward: reuse DY */

/* Build a plan: geometry, the number of peeled layers t for rate c, the kept
 * bin set and the workspace layout.  Host only.  BL_ERR_UNSUPPORTED for
 * K > 8, a grid side above 4096, more than 65535 kept bins, or a plane whose
 * direct transform would need more than 160 KB of LDS (e.g. a 2-D grid
 * 8 x 4096), so that the compute calls of a plan never fail for its shape. */
bl_status_t bl_conv_plan_create(bl_conv_plan_t* out, const bl_conv_desc_t* desc);
bl_status_t bl_conv_plan_destroy(bl_conv_plan_t plan);

/* Grid, kept-set radii, counts and the effective rate c_eff = 1 - kept/total.
 * 1-D: fft_h = L, fft_w = 1, r_h = 0, r_w = r.  Any output pointer may be NULL. */
bl_status_t bl_conv_plan_info(bl_conv_plan_t plan, int* fft_h, int* fft_w, int* r_h, int* r_w,
                              long* kept, long* total, double* c_eff);

/* Copy the 0/1 half-plane mask to host memory: n must equal total;
 * row-major [fft_h][fft_w/2+1] (1-D: [L/2+1]). */
bl_status_t bl_conv_plan_get_mask(bl_conv_plan_t plan, unsigned char* host_mask, size_t n);

/* Kept bins in the order the stored spectra use (bin-major): rows in
 * increasing FFT index u, within a row increasing v.  n must equal kept;
 * u and v are host arrays (1-D: u = 0). */
bl_status_t bl_conv_plan_get_bins(bl_conv_plan_t plan, int* u, int* v, size_t n);

/* Workspace bytes needed by the compute calls of this plan. */
bl_status_t bl_conv_workspace_size(bl_conv_plan_t plan, size_t* bytes);

/* Byte offsets of the stored spectra inside the workspace (any pointer may be
 * NULL).  All are bin-major, interleaved complex64 (with BL_DESC_BF16_SPECTRA:
 * one 32-bit bfloat16 pair per value, as described there):
 *   X  [kept][N][C_in], W [kept][C_in][C_out], DY [kept][N][C_out]. */
bl_status_t bl_conv_workspace_layout(bl_conv_plan_t plan, size_t* off_x, size_t* off_w, size_t* off_dy);

/* y = band-limited correlation of x with w (Eq. 1).  Writes X and W to ws. */
bl_status_t bl_conv_forward(bl_conv_plan_t plan, const float* x, const float* w, float* y,
                            void* ws, unsigned flags, void* stream);

/* dx = gradient of <dy, y> with respect to x: the same mask on the spectrum of
 * dy times the (unconjugated) filter spectrum, summed over output channels,
 * inverse-transformed and cropped to the unpadded input window.  Writes DY and
 * W to ws. */
bl_status_t bl_conv_backward_input(bl_conv_plan_t plan, const float* dy, const float* w, float* dx,
                                   void* ws, unsigned flags, void* stream);

/* dw = gradient of <dy, y> with respect to w, projected onto the kept band:
 * sum over the batch of X times conj(DY) per kept bin, inverse-transformed and
 * cropped to the K x K filter support.  Writes X and DY to ws. */
bl_status_t bl_conv_backward_weight(bl_conv_plan_t plan, const float* x, const float* dy, float* dw,
                                    void* ws, unsigned flags, void* stream);

/* Both gradients of one layer (Sec. 3.2.3): dx as bl_conv_backward_input and
 * dw as bl_conv_backward_weight compute them, from one output-gradient
 * spectrum DY.  The two per-bin contractions run as one launch when both use
 * the tiled kernel with one tile shape, no k split and sums of the same length
 * (C_out = N: their tiles then share the GPU), else one after the other;
 * either way every output element is the same sum, in the same order, as in
 * the separate calls with the same tile shape.  Writes DY, W and X to ws; flags: any of BL_REUSE_X, BL_REUSE_W,
 * BL_REUSE_DY (the tensor may then be NULL).  dx, dw and ws may not be NULL;
 * errors as the other compute calls. */
bl_status_t bl_conv_backward(bl_conv_plan_t plan, const float* dy, const float* w, const float* x, float* dx,
                             float* dw, void* ws, unsigned flags, void* stream);

/* Forward pass that allocates nothing, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  It computes what bl_conv_forward computes (flags 0:
 * X and W are always computed from x and w) but keeps the input, filter and
 * output spectra (and the contraction's partial sums) in one static device
 * array of 64 MiB that the library holds on each GPU it runs on until the
 * process ends, instead of a caller workspace; it calls no hipMalloc or
 * hipFree and uses no plan table (the chirp-z 1-D transforms are replaced by
 * the direct DFT, and the filter transform computes its roots of unity), so
 * even a plan's first call allocates nothing.  The array is located once per
 * device (hipGetSymbolAddress), on the first call on that device.
 *
 * Limit: kept * (N * C_in + C_in * C_out) stored elements (8 bytes, 4 with
 * BL_DESC_BF16_SPECTRA) plus kept * N * C_out * 8 bytes of output spectrum
 * (plus the contraction's k-split partials where the plan's tiling splits k),
 * each rounded up to 256 bytes, must fit 64 MiB; larger plans return
 * BL_ERR_WORKSPACE_TOO_SMALL before anything is enqueued.  Every call on a GPU
 * shares that GPU's array and leaves its spectra there: calls that overlap on
 * one GPU (other streams, other threads) race and give wrong results, so
 * serialise them.  Nothing in the array needs to start at zero: each call
 * writes every part it reads.  Errors as bl_conv_forward; x, w, y may not be
 * NULL.  The spectra it leaves are not accessible to the caller. */
bl_status_t bl_conv_forward_noalloc(bl_conv_plan_t plan, const float* x, const float* w, float* y, void* stream);

/* Energy-based (adaptive) compression, coarse-grained (Sec. 4.1; supplementary
 * "Compression Based on Preserved Energy"): the band is grown from the DC
 * component in whole L-shaped layers until it holds a requested fraction of the
 * energy of the layer's input.
 *
 * bl_conv_input_energy writes, for every kept bin b of the plan (in the order of
 * bl_conv_plan_get_bins), energy[b] = h_v * sum over samples and input channels
 * of |X[b]|^2, in fp64, to the device array `energy` of `kept` doubles; h_v = 1 in
 * column 0 and in the Nyquist column of an even width, else 2 (Parseval on the
 * half plane), so with a plan of rate 0 the energies sum to L_h L_w times the
 * energy of x.  X, the input spectrum, is computed from x and left in ws
 * (BL_REUSE_X: read from ws; x may then be NULL); the sums are of X as stored
 * (rounded to bfloat16 in plans with BL_DESC_BF16_SPECTRA).  One kernel per call on
 * `stream`, summing in a fixed order (results do not depend on scheduling). */
bl_status_t bl_conv_input_energy(bl_conv_plan_t plan, const float* x, void* ws, unsigned flags,
                                 double* energy, void* stream);

/* Host only.  From bin energies in the plan's bin order (host memory, n = kept,
 * e.g. bl_conv_input_energy's output copied back), the band that keeps at least
 * `fraction` (0 < fraction <= 1) of their total: the most layers t that can be
 * peeled, counted from the full half plane (t >= the plan's own), with the bins
 * it keeps.  Outputs (any may be NULL): t; the rate c for which
 * bl_conv_plan_create chooses exactly that band; the fraction it preserves.
 * With a plan of rate 0 the fractions are of the input's whole energy.  Energies
 * that are all zero keep any fraction: the most layers are peeled.  Negative,
 * infinite or NaN energies are BL_ERR_INVALID_ARG. */
bl_status_t bl_conv_rate_for_energy(bl_conv_plan_t plan, const double* energy, size_t n, double fraction,
                                    int* t, double* c, double* preserved);

/* Fine-grained energy-based band (the same supplementary section, its
 * fine-grained variant): the coarse band of bl_conv_rate_for_energy (t layers
 * peeled) is cut inside its outermost layer.  Starting from the band with one
 * more layer peeled, that layer's bins are added back one at a time, largest
 * energy first (equal energies in bin order), until the band keeps at least
 * `fraction`; the layer's other bins are dropped.  (A 1-D layer is one bin, so
 * there the fine band is the coarse one.)
 *
 * bl_conv_fine_band_for_energy takes the same inputs as
 * bl_conv_rate_for_energy and returns the same t and c (the coarse band's; a
 * plan created with rate c has exactly that band), `preserved` = the fraction
 * the fine band keeps, and in keep[0 .. *keep_n) one byte per bin of the coarse
 * band in that plan's bin order: 1 kept, 0 dropped.  keep may be NULL to query
 * *keep_n; otherwise keep_cap must be at least *keep_n.  Host only; the same
 * errors as bl_conv_rate_for_energy, and BL_ERR_INVALID_ARG when keep_cap is
 * too small.
 *
 * bl_conv_zero_bins sets to zero, for every sample and channel, the stored
 * spectrum `which` (BL_SPEC_X or BL_SPEC_W) of ws at the bins with keep[b] == 0;
 * keep is a device array of `kept` bytes in the plan's bin order.  With X and W
 * so zeroed, bl_conv_forward (BL_REUSE_X | BL_REUSE_W) computes the layer on the
 * fine band, and grad-input (BL_REUSE_W) and grad-weight (BL_REUSE_X) project
 * onto it as well, since a zero coefficient of W or X contributes nothing to
 * them.  Errors: NULL arguments, another `which`: BL_ERR_INVALID_ARG; more than
 * 65535 kept bins: BL_ERR_UNSUPPORTED.  One kernel on `stream`. */
bl_status_t bl_conv_fine_band_for_energy(bl_conv_plan_t plan, const double* energy, size_t n, double fraction,
                                         int* t, double* c, double* preserved, unsigned char* keep,
                                         size_t keep_cap, size_t* keep_n);
bl_status_t bl_conv_zero_bins(bl_conv_plan_t plan, void* ws, unsigned which, const unsigned char* keep,
                              void* stream);

/* Fine-grained "top" compression (supplementary section "Error Incurred by 2D
 * Convolution with Compression"): the k coefficients of smallest magnitude of
 * a spectrum are set to zero, the tensors keeping their size.
 *
 * bl_conv_zero_smallest zeroes, in the stored spectrum `which` of ws, the k
 * coefficients of smallest |z| of every group: for BL_SPEC_X each sample's
 * input spectrum, for BL_SPEC_W each output filter's spectrum, each over its
 * C_in channels at every kept bin of the plan.  Coefficient i of a group is
 * (bin i / C_in in bl_conv_plan_get_bins order, channel i % C_in); among equal
 * magnitudes (|z|^2 in fp32) the lower i is zeroed first, so exactly
 * min(k, kept C_in) coefficients per group are zeroed and the result does not
 * depend on scheduling.  The spectrum is first computed from `src` (x
 * [N][C_in][H][W] for BL_SPEC_X, w [C_out][C_in][K][K] for BL_SPEC_W) unless
 * flags holds the reuse flag of that spectrum (BL_REUSE_X or BL_REUSE_W; src
 * may then be NULL).  A following bl_conv_forward with BL_REUSE_X | BL_REUSE_W
 * computes the layer on the zeroed spectra (the backward passes likewise with
 * their reuse flags).  k = 0 only computes the spectrum.  The call may use
 * the workspace outside X, W and DY as scratch (a group-major copy of W; the
 * histograms of groups split over several blocks), so what the compute calls
 * leave there is not kept.  Errors:
 * NULL plan or
 * ws, k < 0, another `which`, other flags, src NULL without the reuse flag:
 * BL_ERR_INVALID_ARG; a group of 2^31 or more coefficients:
 * BL_ERR_UNSUPPORTED.  One kernel (plus the transform) on `stream`. */
#define BL_SPEC_X 0u
#define BL_SPEC_W 1u
bl_status_t bl_conv_zero_smallest(bl_conv_plan_t plan, const float* src, void* ws, unsigned which, long long k,
                                  unsigned flags, void* stream);

const char* bl_status_string(bl_status_t status);

/* Per-kernel timing, for measurement tools.  While enabled, every kernel the
 * compute calls enqueue is bracketed by two HIP events on the same stream
 * (up to `capacity` launches; later launches are not timed).  bl_profile_begin
 * creates the events (it is the only call that allocates) and must not be
 * called while work from a previous profile is in flight.  After the stream
 * has been synchronised, bl_profile_count / bl_profile_get return each
 * launch's kernel name (a static string), its duration in milliseconds and
 * its algorithmic cost: the compulsory HBM bytes (every input read once, every
 * output written once) and the arithmetic: for the channel contraction the
 * real flops of the complex products (8 per complex multiply-add), for the
 * transforms the conventional FFT count (5 N log2 N per complex N-point FFT,
 * 2.5 N log2 N per real one) of the FFTs the kernel performs.  Output pointers
 * may be NULL.  bl_profile_end stops recording; bl_profile_release frees the events. */
bl_status_t bl_profile_begin(int capacity);
bl_status_t bl_profile_end(void);
int bl_profile_count(void);
bl_status_t bl_profile_get(int i, const char** kernel, float* ms, double* bytes, double* flops);
bl_status_t bl_profile_release(void);

#ifdef __cplusplus
}
#endif

#endif /* BLCONV_H */
