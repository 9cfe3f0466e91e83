"""fp64 CPU oracle of the band-limited FFT convolution layer.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import or call
this module: only the tests, the package's smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code with the HIP library.

What it computes (Dziedzic et al., "Band-limited Training and Inference for
Convolutional Neural Networks", ICML 2019):

* Sec. 3, Eq. (1)/(2): the band-limited convolution  x *_c y  is the inverse
  FFT of the product of the two spectra, each multiplied by a 0/1 mask M_c
  that keeps a low-frequency band.
* Sec. 3.2.1: input and filter are zero-padded so that the FFT's circular
  correlation equals the linear one (no wrapped-around filter data).
* Sec. 3.2.2 and Fig. 2: only the half-plane rfft spectrum is stored
  (conjugate symmetry); the band is shrunk layer by layer in L-shaped layers
  taken from the top-left and bottom-left corners of that half plane.
* Sec. 3.1 / Sec. 4.1: the compression rate c is the fraction of the
  half-spectrum coefficients that are discarded.
* Abstract, Sec. 1: the band limit holds in forward and back-propagation;
  the weight gradient is projected onto the kept frequencies.

Readings taken where the paper is silent or ambiguous (each one is a
decision, listed with its reason in the design notes of the repository):

* R1 FFT grid: (L_h, L_w) = (H + p_top + p_bottom, W + p_left + p_right),
  the padded input size; an explicit grid override (e.g. the map-reuse size
  N + max(K-1, G-1) of Sec. 3.2.3) is accepted.
* R2 band shape: keep bin (u, v) of the half plane iff |s(u)| <= r_h and
  v <= r_w, where s(u) is the signed row frequency; r_h = floor(L_h/2) - t,
  r_w = floor(L_w/2) - t after peeling t L-shaped layers.  In 1-D keep the
  prefix v <= floor(L/2) - t.
* R3 rate -> layers: the fewest layers t with kept(t) <= (1 - c) * total,
  evaluated in IEEE fp64 ("discard at least c"); if none qualifies, the most
  layers that can be peeled.
* R4 the layer computes cross-correlation (as a deep-learning conv layer),
  i.e. the filter spectrum enters conjugated.
* R5 the mask is applied in all three passes (forward, grad-input,
  grad-weight), which makes the backward passes exact adjoints.

Parity status: every function here is pinned by tests against brute-force
direct correlation, direct-sum DFTs, Parseval, the adjoint identity, central
finite differences and the worked example of the supplementary section
"Error Incurred by 2D Convolution with Compression" (a 59x30 half spectrum
losing one layer keeps 57x29).  The rate->layers rounding (R3) is not fixed
by the paper: parity of that rule is unpinned beyond the worked example.
"""
from __future__ import annotations

import numpy as np

# ----------------------------------------------------------------------------
# Geometry and the compression mask (Sec. 3.1, Sec. 3.2.2, Fig. 2)
# ----------------------------------------------------------------------------


def signed_freq(u: int, L: int) -> int:
    """Signed frequency of FFT index u on a length-L axis (DC at 0)."""
    return u if u <= L // 2 else u - L


def band_2d(Lh: int, Lw: int, t: int) -> np.ndarray:
    """Half-plane 0/1 mask [Lh][Lw//2+1] after peeling t L-shaped layers."""
    r_h = Lh // 2 - t
    r_w = Lw // 2 - t
    m = np.zeros((Lh, Lw // 2 + 1), dtype=np.uint8)
    for u in range(Lh):
        if abs(signed_freq(u, Lh)) > r_h:
            continue
        for v in range(Lw // 2 + 1):
            if v <= r_w:
                m[u, v] = 1
    return m


def band_1d(L: int, t: int) -> np.ndarray:
    """Half-spectrum 0/1 mask [L//2+1] after discarding the t highest bins."""
    B = L // 2 + 1
    m = np.zeros(B, dtype=np.uint8)
    m[: B - t] = 1
    return m


def layers_for_rate(c: float, total: int, kept_of_t, t_max: int) -> int:
    """Reading R3: the fewest layers t whose kept count is <= (1 - c) * total."""
    budget = (1.0 - c) * total
    for t in range(t_max + 1):
        if kept_of_t(t) <= budget:
            return t
    return t_max


def mask_2d(Lh: int, Lw: int, c: float):
    """(mask [Lh][Lw//2+1] uint8, t, r_h, r_w) for compression rate c."""
    t_max = min(Lh // 2, Lw // 2)
    total = Lh * (Lw // 2 + 1)
    t = layers_for_rate(c, total, lambda tt: int(band_2d(Lh, Lw, tt).sum()), t_max)
    return band_2d(Lh, Lw, t), t, Lh // 2 - t, Lw // 2 - t


def mask_1d(L: int, c: float):
    """(mask [L//2+1] uint8, t, r) for compression rate c."""
    B = L // 2 + 1
    t = layers_for_rate(c, B, lambda tt: int(band_1d(L, tt).sum()), B - 1)
    return band_1d(L, t), t, L // 2 - t


def kept_bins_2d(mask: np.ndarray):
    """Kept (u, v) pairs in the bin-major order used for stored spectra:
    rows in increasing FFT index u (top-left corner, then bottom-left
    corner), and within a row increasing v."""
    return [(u, v) for u in range(mask.shape[0]) for v in range(mask.shape[1]) if mask[u, v]]


def geometry_2d(H, W, K, pad, fft=None):
    pt, pb, pl, pr = pad
    Hp, Wp = H + pt + pb, W + pl + pr
    Ho, Wo = Hp - K + 1, Wp - K + 1
    if Ho < 1 or Wo < 1:
        raise ValueError("filter larger than the padded input")
    Lh, Lw = (Hp, Wp) if fft is None else fft
    if Lh < Hp or Lw < Wp:
        raise ValueError("FFT grid smaller than the padded input would wrap around")
    return dict(Hp=Hp, Wp=Wp, Ho=Ho, Wo=Wo, Lh=Lh, Lw=Lw)


def geometry_1d(L, K, pad, fft=None):
    lo, hi = pad
    Lp = L + lo + hi
    Lo = Lp - K + 1
    if Lo < 1:
        raise ValueError("filter longer than the padded input")
    Lf = Lp if fft is None else fft
    if Lf < Lp:
        raise ValueError("FFT length smaller than the padded input would wrap around")
    return dict(Lp=Lp, Lo=Lo, L=Lf)


# ----------------------------------------------------------------------------
# 2-D passes (Eq. 1 with zero padding, Sec. 3.2.1; half-plane spectra, Sec. 3.2.2)
# ----------------------------------------------------------------------------


def _embed(a, Lh, Lw, oi, oj):
    """Zero array of spatial size Lh x Lw holding a at offset (oi, oj)."""
    out = np.zeros(a.shape[:-2] + (Lh, Lw), dtype=np.float64)
    out[..., oi:oi + a.shape[-2], oj:oj + a.shape[-1]] = a
    return out


def _rfft2(a):
    return np.fft.rfft2(a, axes=(-2, -1))


def _irfft2(A, Lh, Lw):
    return np.fft.irfft2(A, s=(Lh, Lw), axes=(-2, -1))


def _channel_contract(A, B, conj_b: bool, rounding=None):
    """Per-frequency complex product summed over a shared channel index.

    A: [P, Q, h, w] complex, B: [R, Q, h, w] complex -> [P, R, h, w] with
    out[p, r] = sum_q A[p, q] * (conj(B[r, q]) if conj_b else B[r, q]).
    Written as one complex matrix product per frequency bin.  With
    `rounding` (a function of real arrays), the real and imaginary parts of
    both operands are rounded first and the products are exact: the reduced
    precision operands of the contraction (reduced-precision arithmetic
    combined with band-limiting), accumulated in fp64.
    """
    if rounding is not None:
        A = rounding(A.real) + 1j * rounding(A.imag)
        B = rounding(B.real) + 1j * rounding(B.imag)
    Bq = np.conj(B) if conj_b else B
    a = np.moveaxis(A, (0, 1), (-2, -1))  # [h, w, P, Q]
    b = np.moveaxis(Bq, (0, 1), (-1, -2))  # [h, w, Q, R]
    return np.moveaxis(a @ b, (-2, -1), (0, 1))


def spectra_2d(x, w, pad, c, fft=None):
    """Masked half-plane spectra (X*M, W*M, M) of the embedded input and filter."""
    N, C, H, W = x.shape
    K = w.shape[-1]
    g = geometry_2d(H, W, K, pad, fft)
    M = mask_2d(g["Lh"], g["Lw"], c)[0]
    X = _rfft2(_embed(np.asarray(x, np.float64), g["Lh"], g["Lw"], pad[0], pad[2])) * M
    Wf = _rfft2(_embed(np.asarray(w, np.float64), g["Lh"], g["Lw"], 0, 0)) * M
    return X, Wf, M, g


def forward_2d(x, w, pad, c, fft=None, rounding=None):
    """y[n,f] = crop_{Ho x Wo} irfft2( sum_c (X[n,c] M) conj(W[f,c] M) )."""
    X, Wf, M, g = spectra_2d(x, w, pad, c, fft)
    Y = _channel_contract(X, Wf, conj_b=True, rounding=rounding)
    return _irfft2(Y, g["Lh"], g["Lw"])[..., : g["Ho"], : g["Wo"]]


def backward_input_2d(dy, w, x_hw, pad, c, fft=None, rounding=None):
    """dx[n,c] = crop_{pad window} irfft2( sum_f (DY[n,f] M) (W[f,c] M) )."""
    H, W = x_hw
    K = w.shape[-1]
    g = geometry_2d(H, W, K, pad, fft)
    M = mask_2d(g["Lh"], g["Lw"], c)[0]
    DY = _rfft2(_embed(np.asarray(dy, np.float64), g["Lh"], g["Lw"], 0, 0)) * M
    Wf = _rfft2(_embed(np.asarray(w, np.float64), g["Lh"], g["Lw"], 0, 0)) * M
    # sum over f of DY[n,f] * W[f,c]: contract DY [n,f] with W^T [c,f]
    DX = _channel_contract(DY, np.swapaxes(Wf, 0, 1), conj_b=False, rounding=rounding)
    full = _irfft2(DX, g["Lh"], g["Lw"])
    return full[..., pad[0]:pad[0] + H, pad[2]:pad[2] + W]


def backward_weight_2d(x, dy, K, pad, c, fft=None, rounding=None):
    """dw[f,c] = crop_{K x K} irfft2( sum_n (X[n,c] M) conj(DY[n,f] M) )."""
    N, C, H, W = x.shape
    g = geometry_2d(H, W, K, pad, fft)
    M = mask_2d(g["Lh"], g["Lw"], c)[0]
    X = _rfft2(_embed(np.asarray(x, np.float64), g["Lh"], g["Lw"], pad[0], pad[2])) * M
    DY = _rfft2(_embed(np.asarray(dy, np.float64), g["Lh"], g["Lw"], 0, 0)) * M
    # DW[f,c] = sum_n DY*[n,f] X[n,c]: contract over n
    DW = _channel_contract(np.swapaxes(X, 0, 1), np.swapaxes(DY, 0, 1), conj_b=True, rounding=rounding)  # [c, f]
    return np.swapaxes(_irfft2(DW, g["Lh"], g["Lw"])[..., :K, :K], 0, 1)


def kept_spectrum_2d(a, offset, Lh, Lw, c):
    """Bin-major kept spectrum [B][planes] of real planes a[..., h, w] placed at
    offset (oi, oj) in the Lh x Lw grid (what the library stores for x and dy)."""
    M = mask_2d(Lh, Lw, c)[0]
    A = _rfft2(_embed(np.asarray(a, np.float64), Lh, Lw, offset[0], offset[1]))
    bins = kept_bins_2d(M)
    flat = A.reshape((-1,) + A.shape[-2:])
    return np.stack([flat[:, u, v] for (u, v) in bins], axis=0)


def kept_filter_spectrum_2d(w, Lh, Lw, c):
    """Bin-major kept filter spectrum [B][C_in][C_out] (the library's layout)."""
    M = mask_2d(Lh, Lw, c)[0]
    Wf = _rfft2(_embed(np.asarray(w, np.float64), Lh, Lw, 0, 0))  # [F, C, h, w]
    bins = kept_bins_2d(M)
    return np.stack([Wf[:, :, u, v].T for (u, v) in bins], axis=0)


# ----------------------------------------------------------------------------
# 1-D passes (the time-series variant of Sec. 3.2.2: keep the low prefix)
# ----------------------------------------------------------------------------


def _embed1(a, L, o):
    out = np.zeros(a.shape[:-1] + (L,), dtype=np.float64)
    out[..., o:o + a.shape[-1]] = a
    return out


def forward_1d(x, w, pad, c, fft=None, rounding=None):
    N, C, Lx = x.shape
    K = w.shape[-1]
    g = geometry_1d(Lx, K, pad, fft)
    M = mask_1d(g["L"], c)[0]
    X = np.fft.rfft(_embed1(np.asarray(x, np.float64), g["L"], pad[0])) * M
    Wf = np.fft.rfft(_embed1(np.asarray(w, np.float64), g["L"], 0)) * M
    Y = _channel_contract(X[..., None, :], Wf[..., None, :], conj_b=True, rounding=rounding)[..., 0, :]
    return np.fft.irfft(Y, n=g["L"])[..., : g["Lo"]]


def backward_input_1d(dy, w, Lx, pad, c, fft=None, rounding=None):
    K = w.shape[-1]
    g = geometry_1d(Lx, K, pad, fft)
    M = mask_1d(g["L"], c)[0]
    DY = np.fft.rfft(_embed1(np.asarray(dy, np.float64), g["L"], 0)) * M
    Wf = np.fft.rfft(_embed1(np.asarray(w, np.float64), g["L"], 0)) * M
    DX = _channel_contract(DY[..., None, :], np.swapaxes(Wf, 0, 1)[..., None, :], conj_b=False,
                           rounding=rounding)[..., 0, :]
    return np.fft.irfft(DX, n=g["L"])[..., pad[0]:pad[0] + Lx]


def backward_weight_1d(x, dy, K, pad, c, fft=None, rounding=None):
    N, C, Lx = x.shape
    g = geometry_1d(Lx, K, pad, fft)
    M = mask_1d(g["L"], c)[0]
    X = np.fft.rfft(_embed1(np.asarray(x, np.float64), g["L"], pad[0])) * M
    DY = np.fft.rfft(_embed1(np.asarray(dy, np.float64), g["L"], 0)) * M
    DW = _channel_contract(np.swapaxes(X, 0, 1)[..., None, :], np.swapaxes(DY, 0, 1)[..., None, :],
                           conj_b=True, rounding=rounding)[..., 0, :]
    return np.swapaxes(np.fft.irfft(DW, n=g["L"])[..., :K], 0, 1)


def kept_spectrum_1d(a, offset, L, c):
    M = mask_1d(L, c)[0]
    A = np.fft.rfft(_embed1(np.asarray(a, np.float64), L, offset))
    flat = A.reshape(-1, A.shape[-1])
    return np.ascontiguousarray(flat[:, M.astype(bool)].T)


def kept_filter_spectrum_1d(w, L, c):
    M = mask_1d(L, c)[0]
    Wf = np.fft.rfft(_embed1(np.asarray(w, np.float64), L, 0))  # [F, C, B]
    return np.ascontiguousarray(np.transpose(Wf[:, :, M.astype(bool)], (2, 1, 0)))


# ----------------------------------------------------------------------------
# Dimension-generic front door used by tests and the benchmark's CPU leg
# ----------------------------------------------------------------------------


def forward(x, w, pad, c, fft=None, rounding=None):
    f = forward_1d if x.ndim == 3 else forward_2d
    return f(x, w, pad, c, fft, rounding)


def backward_input(dy, w, x_spatial, pad, c, fft=None, rounding=None):
    if dy.ndim == 3:
        return backward_input_1d(dy, w, x_spatial[0], pad, c, fft, rounding)
    return backward_input_2d(dy, w, x_spatial, pad, c, fft, rounding)


def backward_weight(x, dy, K, pad, c, fft=None, rounding=None):
    f = backward_weight_1d if x.ndim == 3 else backward_weight_2d
    return f(x, dy, K, pad, c, fft, rounding)


def mask(ndim, L, c):
    """Mask for a grid: ndim=1 -> L is an int; ndim=2 -> L is (Lh, Lw)."""
    return mask_1d(L, c)[0] if ndim == 1 else mask_2d(L[0], L[1], c)[0]


def plan_info(ndim, L, c):
    """(r_h, r_w, kept, total, c_eff) of the mask rule, for comparison with the
    library's plan report (1-D: r_h = 0, r_w = r)."""
    if ndim == 1:
        m, t, r = mask_1d(L, c)
        kept, total = int(m.sum()), m.size
        return 0, r, kept, total, 1.0 - kept / total
    m, t, r_h, r_w = mask_2d(L[0], L[1], c)
    kept, total = int(m.sum()), m.size
    return r_h, r_w, kept, total, 1.0 - kept / total


# ----------------------------------------------------------------------------
# Energy-based (adaptive) compression, coarse-grained (Sec. 4.1 and the
# supplementary section "Compression Based on Preserved Energy")
# ----------------------------------------------------------------------------
#
# The paper's second compression scheme chooses how much of the band to keep
# from the energy the band preserves, instead of from a fixed rate: starting
# at the DC component, whole L-shaped layers of rows and columns are added
# until the kept coefficients hold the requested fraction of the energy.  The
# energy is that of the layer's input (Sec. 4.1 defines it for an input tensor
# x through Parseval's theorem).  Readings taken here (listed in the design
# notes): E1 the energy of a half-plane bin counts twice unless the bin is its
# own conjugate partner (column 0, and the Nyquist column of an even width):
# Parseval on the half plane (reading R7); E2 the band kept is the smallest
# L-shaped band (the most peeled layers t) whose energy is at least the
# requested fraction of the total ("preserve at least E"); E3 an input with no
# energy preserves any fraction with any band: the most layers are peeled.
# Parity: pinned by Parseval, by the band energy evaluated in the signal
# domain with direct-sum DFTs, and by single-frequency and constant inputs.


def parseval_weights(Lw: int) -> np.ndarray:
    """h_v over the half-plane columns v = 0 .. Lw//2 (reading E1 / R7)."""
    h = np.full(Lw // 2 + 1, 2.0)
    h[0] = 1.0
    if Lw % 2 == 0:
        h[-1] = 1.0
    return h


def bin_energy_2d(x, pad, fft=None) -> np.ndarray:
    """[Lh][Lw//2+1]: h_v * sum over samples and channels of |X[n,c,u,v]|^2,
    X the spectrum of the input placed at (pad top, pad left) of the grid."""
    N, C, H, W = x.shape
    Lh, Lw = (H + pad[0] + pad[1], W + pad[2] + pad[3]) if fft is None else fft
    X = _rfft2(_embed(np.asarray(x, np.float64), Lh, Lw, pad[0], pad[2]))
    return parseval_weights(Lw)[None, :] * (np.abs(X) ** 2).sum(axis=(0, 1))


def bin_energy_1d(x, pad, fft=None) -> np.ndarray:
    """[L//2+1]: h_v * sum over series of |X[n,c,v]|^2."""
    N, C, Lx = x.shape
    L = Lx + pad[0] + pad[1] if fft is None else fft
    X = np.fft.rfft(_embed1(np.asarray(x, np.float64), L, pad[0]))
    return parseval_weights(L) * (np.abs(X) ** 2).sum(axis=(0, 1))


def last_layer_kept(ndim, L) -> np.ndarray:
    """For every half-plane bin, the most layers t that can be peeled with the
    bin still kept (from the band definition, t by t)."""
    if ndim == 1:
        t_max = L // 2
        out = np.full(L // 2 + 1, -1, dtype=np.int64)
        for t in range(t_max + 1):
            out[band_1d(L, t).astype(bool)] = t
        return out
    Lh, Lw = L
    t_max = min(Lh // 2, Lw // 2)
    out = np.full((Lh, Lw // 2 + 1), -1, dtype=np.int64)
    for t in range(t_max + 1):
        out[band_2d(Lh, Lw, t).astype(bool)] = t
    return out


def preserved_fractions(E: np.ndarray, last: np.ndarray) -> np.ndarray:
    """f[t] = energy of the bins kept after peeling t layers / total energy
    (1 for every t when the total is zero, reading E3)."""
    t_max = int(last.max())
    total = float(E.sum())
    kept = np.array([float(E[last >= t].sum()) for t in range(t_max + 1)])
    return np.ones(t_max + 1) if total == 0.0 else kept / total


def layers_for_energy(fraction: float, f: np.ndarray) -> int:
    """Reading E2: the most layers t whose band keeps at least `fraction`."""
    return max(t for t in range(len(f)) if f[t] >= fraction)


def energy_rate(x, pad, fraction, fft=None):
    """Band chosen for input x so that at least `fraction` of its energy is
    kept: dict(t, kept, total, c_eff, preserved, fractions)."""
    if x.ndim == 3:
        L = x.shape[-1] + pad[0] + pad[1] if fft is None else fft
        E, last = bin_energy_1d(x, pad, fft), last_layer_kept(1, L)
    else:
        Lh, Lw = (x.shape[-2] + pad[0] + pad[1], x.shape[-1] + pad[2] + pad[3]) if fft is None else fft
        E, last = bin_energy_2d(x, pad, fft), last_layer_kept(2, (Lh, Lw))
    f = preserved_fractions(E, last)
    t = layers_for_energy(fraction, f)
    kept, total = int((last >= t).sum()), last.size
    return dict(t=t, kept=kept, total=total, c_eff=1.0 - kept / total, preserved=float(f[t]), fractions=f)


# Fine-grained energy-based band (the same supplementary section, its
# fine-grained variant): within the outermost layer that the energy target
# needs, coefficients are added one at a time, and the layer's others are zeroed
# in both the activation map's and the filter's spectrum.
#
# Readings:
# * F1 the coarse band is E2's: the most layers t_c whose band keeps at least
#   the fraction.  The fine-grained band starts from the band with one more
#   layer peeled (t_c + 1, which keeps less) and adds back bins of layer t_c
#   (the bins with last_layer_kept == t_c), largest energy first (equal
#   energies in stored bin order), until it keeps at least the fraction.  With
#   t_c the deepest band, or an input without energy, it is the coarse band.
# * F2 it is computed with the coarse band's plan and the dropped bins' stored
#   coefficients zeroed for every sample and channel, in the input spectrum and
#   the filter spectrum; that also projects grad-input and grad-weight onto the
#   fine band (a zero coefficient of W or X contributes nothing to them).
def fine_energy_band(E, last, fraction):
    """(t_c, keep): E and last over the same bins in stored order; keep is a
    boolean over the bins of band t_c (those with last >= t_c), in that order,
    False for the bins the fine-grained band drops."""
    E = np.asarray(E, dtype=np.float64).ravel()
    last = np.asarray(last).ravel()
    f = preserved_fractions(E, last)
    t = layers_for_energy(fraction, f)
    band = last >= t
    keep = np.ones(int(band.sum()), dtype=bool)
    total = float(E.sum())
    if t == len(f) - 1 or total == 0.0:
        return t, keep
    Eb, lb = E[band], last[band]
    layer = np.nonzero(lb == t)[0]
    keep[layer] = False
    kept_e = float(Eb[lb > t].sum())
    for i in layer[np.argsort(-Eb[layer], kind="stable")]:
        if kept_e / total >= fraction:
            break
        keep[i] = True
        kept_e += float(Eb[i])
    return t, keep


# ----------------------------------------------------------------------------
# Reduced-precision contraction operands: the paper compares band-limiting
# with reduced-precision arithmetic (Sec. 4.3) and combines the two in the
# supplementary section "Reduced Precision and Bandlimited Training".  Here
# the operands of the channel contraction are rounded to bfloat16 (reading
# P1: the exponent range of fp32, which sums of many samples need; the
# paper's runs used fp16) and the products are accumulated exactly.
# ----------------------------------------------------------------------------


def round_bf16(a) -> np.ndarray:
    """Values rounded to bfloat16 (8 significant bits, the exponent range of
    fp32), round to nearest, ties to even: first to fp32 (how the spectra are
    held), then the 16 low bits of the fp32 pattern are rounded away.
    Returned as float64."""
    f = np.asarray(a, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


# ----------------------------------------------------------------------------
# Fine-grained "top" compression (supplementary section "Error Incurred by 2D
# Convolution with Compression"): the k coefficients of smallest magnitude in a
# spectrum are zeroed; the tensors keep their size.
#
# Readings (the paper works with one image and one filter):
# * T1 "the whole tensor" is, for the input, one sample's spectrum over its
#   channels and the plan's kept half-plane bins, and for the filter one output
#   filter's spectrum over its input channels and the kept bins; each is ranked
#   on its own.
# * T2 among coefficients of equal magnitude the one earlier in (bin, channel)
#   order, bins in the stored bin-major order, goes first (any order is a valid
#   reading; this one is deterministic).
# * T3 a zeroed coefficient loses its real and imaginary parts; column 0 (and
#   an even width's Nyquist column) keep the inverse transform's real-part
#   convention, so zeroing one of a conjugate pair halves that frequency.
# ----------------------------------------------------------------------------


def zero_smallest(S: np.ndarray, k: int) -> np.ndarray:
    """Rows of S (complex, [segments, m]) with the k entries of smallest |S|
    set to zero (all of them when k >= m); equal magnitudes in row order."""
    if k < 0:
        raise ValueError("k must be non-negative")
    S = np.array(S, dtype=np.complex128, copy=True)
    if k == 0:
        return S
    order = np.argsort(np.abs(S), axis=1, kind="stable")[:, :k]
    np.put_along_axis(S, order, 0.0, axis=1)
    return S


def _kept_index(M: np.ndarray):
    """Index arrays of the kept bins of a 2-D (or 1-D) mask in stored order."""
    if M.ndim == 1:
        return (np.nonzero(M)[0],)
    bins = kept_bins_2d(M)
    return (np.array([u for u, _ in bins], dtype=np.int64), np.array([v for _, v in bins], dtype=np.int64))


def _zero_smallest_per_plane_group(A: np.ndarray, idx, k: int) -> np.ndarray:
    """A: [G, C, *grid] masked spectra; rank the kept coefficients of each
    group g over (bin, channel) in that order, zero the k smallest."""
    A = A.copy()
    Ak = A[(slice(None), slice(None)) + idx]  # [G, C, B]
    G, C, B = Ak.shape
    seg = np.swapaxes(Ak, 1, 2).reshape(G, B * C)  # index b * C + c
    z = zero_smallest(seg, k).reshape(G, B, C)
    A[(slice(None), slice(None)) + idx] = np.swapaxes(z, 1, 2)
    return A


def forward_top(x, w, pad, c, k_x, k_w, fft=None):
    """Forward pass (Eq. 1) with the k_x smallest-magnitude coefficients of
    each sample's input spectrum and the k_w smallest of each filter's
    spectrum zeroed (readings T1-T3), on the band of rate c."""
    if x.ndim == 4:
        X, Wf, M, g = spectra_2d(x, w, pad, c, fft)
        idx = _kept_index(M)
        X = _zero_smallest_per_plane_group(X, idx, k_x)
        Wf = _zero_smallest_per_plane_group(Wf, idx, k_w)
        Y = _channel_contract(X, Wf, conj_b=True)
        return _irfft2(Y, g["Lh"], g["Lw"])[..., : g["Ho"], : g["Wo"]]
    N, C, Lx = x.shape
    K = w.shape[-1]
    g = geometry_1d(Lx, K, pad, fft)
    M = mask_1d(g["L"], c)[0]
    X = np.fft.rfft(_embed1(np.asarray(x, np.float64), g["L"], pad[0])) * M
    Wf = np.fft.rfft(_embed1(np.asarray(w, np.float64), g["L"], 0)) * M
    idx = _kept_index(M)
    X = _zero_smallest_per_plane_group(X, idx, k_x)
    Wf = _zero_smallest_per_plane_group(Wf, idx, k_w)
    Y = _channel_contract(X[..., None, :], Wf[..., None, :], conj_b=True)[..., 0, :]
    return np.fft.irfft(Y, n=g["L"])[..., : g["Lo"]]


def top_zeroed(S_kept: np.ndarray, k: int, per_last: bool) -> np.ndarray:
    """Boolean mask of the entries zero_smallest ranks among the k smallest,
    for a stored kept spectrum laid out bin-major as the library stores it:
    [B][G][C] for inputs (per_last False: group G = sample, ranked over
    (b, c)) or [B][C][G] for filters (per_last True: group = output filter)."""
    S = np.asarray(S_kept)
    if per_last:
        S = np.swapaxes(S, 1, 2)  # [B][G][C]
    B, G, C = S.shape
    seg = np.swapaxes(S, 0, 1).reshape(G, B * C)
    z = np.zeros(seg.shape, dtype=bool)
    if k > 0:
        np.put_along_axis(z, np.argsort(np.abs(seg), axis=1, kind="stable")[:, :k], True, axis=1)
    z = np.swapaxes(z.reshape(G, B, C), 0, 1)
    return np.swapaxes(z, 1, 2) if per_last else z


def forward_zeroed(x, w, pad, c, zero_x, zero_w, fft=None):
    """Forward pass (Eq. 1) with chosen kept coefficients zeroed: zero_x is a
    boolean [B][N][C_in] over the stored input spectrum, zero_w [B][C_in][C_out]
    over the stored filter spectrum (bins in stored order).  With the masks of
    top_zeroed it is forward_top; with none set, the band-limited forward."""
    if x.ndim == 4:
        X, Wf, M, g = spectra_2d(x, w, pad, c, fft)
    else:
        g = geometry_1d(x.shape[-1], w.shape[-1], pad, fft)
        M = mask_1d(g["L"], c)[0]
        X = np.fft.rfft(_embed1(np.asarray(x, np.float64), g["L"], pad[0])) * M
        Wf = np.fft.rfft(_embed1(np.asarray(w, np.float64), g["L"], 0)) * M
    idx = _kept_index(M)
    sel = (slice(None), slice(None)) + idx
    Xk = X[sel]  # [N, C, B]
    Xk[np.transpose(np.asarray(zero_x, bool), (1, 2, 0))] = 0.0
    X[sel] = Xk
    Wk = Wf[sel]  # [F, C, B]
    Wk[np.transpose(np.asarray(zero_w, bool), (2, 1, 0))] = 0.0
    Wf[sel] = Wk
    if x.ndim == 4:
        Y = _channel_contract(X, Wf, conj_b=True)
        return _irfft2(Y, g["Lh"], g["Lw"])[..., : g["Ho"], : g["Wo"]]
    Y = _channel_contract(X[..., None, :], Wf[..., None, :], conj_b=True)[..., 0, :]
    return np.fft.irfft(Y, n=g["L"])[..., : g["Lo"]]
