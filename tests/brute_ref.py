"""Brute-force references that pin the oracle (test code only).

Nothing here uses an FFT library.  Linear correlations are written as
explicit sums over filter taps, the DFT as an explicit sum of complex
exponentials, and circular correlation as an explicit sum over shifts.
They are slow and meant for tiny shapes.
"""
from __future__ import annotations

import numpy as np


def pad2(x, pad):
    pt, pb, pl, pr = pad
    return np.pad(np.asarray(x, np.float64), ((0, 0), (0, 0), (pt, pb), (pl, pr)))


def direct_corr_2d(x, w, pad):
    """y[n,f,i,j] = sum_{c,a,b} xpad[n,c,i+a,j+b] * w[f,c,a,b] (stride 1)."""
    xp = pad2(x, pad)
    N, C, Hp, Wp = xp.shape
    F, _, K, _ = w.shape
    Ho, Wo = Hp - K + 1, Wp - K + 1
    y = np.zeros((N, F, Ho, Wo))
    for a in range(K):
        for b in range(K):
            patch = xp[:, :, a:a + Ho, b:b + Wo]  # [N, C, Ho, Wo]
            for f in range(F):
                for c in range(C):
                    y[:, f] += patch[:, c] * float(w[f, c, a, b])
    return y


def direct_grad_input_2d(dy, w, x_hw, pad):
    """dx = d/dx <dy, direct_corr_2d(x, w)> by scattering every tap."""
    H, W = x_hw
    pt, pb, pl, pr = pad
    N, F, Ho, Wo = dy.shape
    _, C, K, _ = w.shape
    dxp = np.zeros((N, C, H + pt + pb, W + pl + pr))
    for a in range(K):
        for b in range(K):
            for f in range(F):
                for c in range(C):
                    dxp[:, c, a:a + Ho, b:b + Wo] += np.asarray(dy[:, f], np.float64) * float(w[f, c, a, b])
    return dxp[:, :, pt:pt + H, pl:pl + W]


def direct_grad_weight_2d(x, dy, K, pad):
    """dw[f,c,a,b] = sum_{n,i,j} dy[n,f,i,j] * xpad[n,c,i+a,j+b]."""
    xp = pad2(x, pad)
    N, C, Hp, Wp = xp.shape
    F = dy.shape[1]
    Ho, Wo = Hp - K + 1, Wp - K + 1
    dw = np.zeros((F, C, K, K))
    dy = np.asarray(dy, np.float64)
    for f in range(F):
        for c in range(C):
            for a in range(K):
                for b in range(K):
                    dw[f, c, a, b] = np.sum(dy[:, f] * xp[:, c, a:a + Ho, b:b + Wo])
    return dw


def direct_corr_1d(x, w, pad):
    lo, hi = pad
    xp = np.pad(np.asarray(x, np.float64), ((0, 0), (0, 0), (lo, hi)))
    N, C, Lp = xp.shape
    F, _, K = w.shape
    Lo = Lp - K + 1
    y = np.zeros((N, F, Lo))
    for a in range(K):
        for f in range(F):
            for c in range(C):
                y[:, f] += xp[:, c, a:a + Lo] * float(w[f, c, a])
    return y


def direct_grad_input_1d(dy, w, Lx, pad):
    lo, hi = pad
    N, F, Lo = dy.shape
    _, C, K = w.shape
    dxp = np.zeros((N, C, Lx + lo + hi))
    for a in range(K):
        for f in range(F):
            for c in range(C):
                dxp[:, c, a:a + Lo] += np.asarray(dy[:, f], np.float64) * float(w[f, c, a])
    return dxp[:, :, lo:lo + Lx]


def direct_grad_weight_1d(x, dy, K, pad):
    lo, hi = pad
    xp = np.pad(np.asarray(x, np.float64), ((0, 0), (0, 0), (lo, hi)))
    N, C, Lp = xp.shape
    F = dy.shape[1]
    Lo = Lp - K + 1
    dw = np.zeros((F, C, K))
    for f in range(F):
        for c in range(C):
            for a in range(K):
                dw[f, c, a] = np.sum(np.asarray(dy[:, f], np.float64) * xp[:, c, a:a + Lo])
    return dw


# --------------------------------------------------------------------------
# Direct-sum DFT and an independent, full-plane statement of the band
# --------------------------------------------------------------------------


def dft_matrix(L, sign=-1):
    k = np.arange(L)
    return np.exp(sign * 2j * np.pi * np.outer(k, k) / L)


def full_band_2d(Lh, Lw, t):
    """Full-plane band: |signed u| <= Lh//2 - t and |signed v| <= Lw//2 - t.

    Written independently of the half-plane mask: a coefficient and its
    conjugate partner are kept or dropped together."""
    def sf(k, L):
        k = np.arange(L)
        return np.where(k <= L // 2, k, k - L)
    su = np.abs(sf(None, Lh))[:, None]
    sv = np.abs(sf(None, Lw))[None, :]
    return ((su <= Lh // 2 - t) & (sv <= Lw // 2 - t)).astype(np.float64)


def lowpass_2d(z, band):
    """Real part of IDFT(band * DFT(z)) over the last two axes, direct sums."""
    Lh, Lw = z.shape[-2:]
    Fh, Fw = dft_matrix(Lh), dft_matrix(Lw)
    Z = np.einsum("ui,...ij,vj->...uv", Fh, z, Fw)
    Z = Z * band
    Ih, Iw = dft_matrix(Lh, +1), dft_matrix(Lw, +1)
    back = np.einsum("iu,...uv,jv->...ij", Ih, Z, Iw) / (Lh * Lw)
    return back.real, np.abs(back.imag).max()


def lowpass_1d(z, keep_lowest):
    """Keep signed frequencies |s| <= keep_lowest (a symmetric set), direct sums."""
    L = z.shape[-1]
    k = np.arange(L)
    s = np.abs(np.where(k <= L // 2, k, k - L))
    band = (s <= keep_lowest).astype(np.float64)
    F = dft_matrix(L)
    Z = (z @ F.T) * band
    back = (Z @ dft_matrix(L, +1).T) / L
    return back.real, np.abs(back.imag).max()


def circ_corr_2d(a, b):
    """z[k1,k2] = sum_{m1,m2} a[(m1+k1)%Lh, (m2+k2)%Lw] * b[m1, m2] (explicit shifts)."""
    Lh, Lw = a.shape[-2:]
    z = np.zeros(np.broadcast_shapes(a.shape, b.shape))
    for m1 in range(Lh):
        for m2 in range(Lw):
            z += np.roll(a, shift=(-m1, -m2), axis=(-2, -1)) * b[..., m1:m1 + 1, m2:m2 + 1]
    return z


def circ_corr_1d(a, b):
    L = a.shape[-1]
    z = np.zeros(np.broadcast_shapes(a.shape, b.shape))
    for m in range(L):
        z += np.roll(a, shift=-m, axis=-1) * b[..., m:m + 1]
    return z


def circ_conv_2d(a, b):
    """z[k1,k2] = sum_{m1,m2} a[(k1-m1)%Lh, (k2-m2)%Lw] * b[m1, m2]."""
    Lh, Lw = a.shape[-2:]
    z = np.zeros(np.broadcast_shapes(a.shape, b.shape))
    for m1 in range(Lh):
        for m2 in range(Lw):
            z += np.roll(a, shift=(m1, m2), axis=(-2, -1)) * b[..., m1:m1 + 1, m2:m2 + 1]
    return z


def circ_conv_1d(a, b):
    L = a.shape[-1]
    z = np.zeros(np.broadcast_shapes(a.shape, b.shape))
    for m in range(L):
        z += np.roll(a, shift=m, axis=-1) * b[..., m:m + 1]
    return z
