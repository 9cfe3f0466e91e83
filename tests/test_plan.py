"""Host plan of the C-ABI library against the oracle (CPU only, no GPU calls).

The library's kept mask must equal the oracle's byte for byte; its counts,
radii and c_eff must agree; its bin order must be the documented one; and
invalid descriptors must be rejected with the documented status codes.
"""
import ctypes
import math
import os
import re

import numpy as np
import pytest

from oracle import bl_oracle as bo
from paper_1911_09287_amd import blconv, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.skipif(not os.path.exists(blconv.LIB_PATH), reason="libblconv.so not built")


def test_library_exports_every_declared_symbol():
    header = open(os.path.join(ROOT, "include", "blconv.h")).read()
    declared = set(re.findall(r"\b(bl_[a-z_]+)\s*\(", header))
    lib = blconv.load()
    for name in declared:
        assert hasattr(lib, name), name
    assert declared == set(blconv.EXPORTED)


def _grid(layer):
    if layer.ndim == 1:
        return layer.H + layer.pad[0] + layer.pad[1]
    return (layer.H + layer.pad[0] + layer.pad[1], layer.W + layer.pad[2] + layer.pad[3])


@pytest.mark.parametrize("cfg", sorted(synth.WORKLOADS))
def test_config_masks_match_oracle(cfg):
    for layer in synth.WORKLOADS[cfg].layers:
        for c in (0.0, 0.25, 0.5, 0.75) + synth.WORKLOADS[cfg].rates:
            plan = blconv.plan_for_layer(layer, c)
            L = _grid(layer)
            assert (plan.mask() == bo.mask(layer.ndim, L, c)).all()
            r_h, r_w, kept, total, ceff = bo.plan_info(layer.ndim, L, c)
            assert (plan.r_h, plan.r_w, plan.kept, plan.total) == (r_h, r_w, kept, total)
            assert plan.c_eff == ceff
            assert plan.c_eff >= c - 1e-15 or plan.kept == 1


def test_random_grids_and_rates_match_oracle():
    rng = np.random.default_rng(7)
    for _ in range(300):
        if rng.random() < 0.5:
            L = int(rng.integers(1, 1100))
            c = float(rng.random())
            layer = synth.Layer("r", 1, 1, 1, 1, L, 1, 1, (0, 0), "walk")
            plan = blconv.plan_for_layer(layer, c)
            assert (plan.mask() == bo.mask(1, L, c)).all()
        else:
            Lh, Lw = int(rng.integers(1, 70)), int(rng.integers(1, 70))
            c = float(rng.choice([rng.random(), 0.25, 0.5, 0.75, 0.0]))
            layer = synth.Layer("r", 2, 1, 1, 1, Lh, Lw, 1, (0, 0, 0, 0), "blur")
            plan = blconv.plan_for_layer(layer, c)
            assert (plan.mask() == bo.mask(2, (Lh, Lw), c)).all(), (Lh, Lw, c)


def test_grid_override_worked_example():
    # 3x32x32 input, 5x5 filter, grid 59 (the map-reuse size): one layer -> 57 x 29
    plan = blconv.Plan(2, 1, 3, 1, (32, 32), 5, (0, 0, 0, 0), 0.066, fft=(59, 59))
    assert plan.fft == (59, 59) and plan.total == 59 * 30
    assert plan.kept == 57 * 29
    assert round(100 * plan.c_eff, 2) == 6.61


def test_bins_order_is_documented_order():
    for (Lh, Lw, c) in ((34, 34, 0.5), (9, 7, 0.3), (6, 6, 0.75), (1, 519, 0.25)):
        if Lh == 1:
            layer = synth.Layer("r", 1, 1, 1, 1, Lw, 1, 1, (0, 0), "walk")
            m = bo.mask(1, Lw, c)
            expect = [(0, v) for v in range(m.size) if m[v]]
        else:
            layer = synth.Layer("r", 2, 1, 1, 1, Lh, Lw, 1, (0, 0, 0, 0), "blur")
            expect = bo.kept_bins_2d(bo.mask(2, (Lh, Lw), c))
        u, v = blconv.plan_for_layer(layer, c).bins()
        assert list(zip(u.tolist(), v.tolist())) == expect


def test_workspace_layout_is_disjoint_and_large_enough():
    for cfg in sorted(synth.WORKLOADS):
        for layer in synth.WORKLOADS[cfg].layers:
            p = blconv.plan_for_layer(layer, 0.0)
            sizes = {"X": p.kept * p.N * p.C_in * 8, "W": p.kept * p.C_in * p.C_out * 8,
                     "DY": p.kept * p.N * p.C_out * 8}
            spans = sorted((p.offsets[k], p.offsets[k] + sizes[k]) for k in sizes)
            for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
                assert a1 <= b0
            assert spans[-1][1] <= p.workspace_bytes
            assert all(o % 256 == 0 for o in p.offsets.values())


def _create(**kw):
    lib = blconv.load()
    d = blconv.Desc()
    base = dict(ndim=2, N=1, C_in=1, C_out=1, H=8, W=8, K=3, c=0.0)
    base.update({k: v for k, v in kw.items() if k not in ("pad_lo", "pad_hi")})
    for k, v in base.items():
        setattr(d, k, v)
    for k in ("pad_lo", "pad_hi"):
        if k in kw:
            getattr(d, k)[0], getattr(d, k)[1] = kw[k]
    h = ctypes.c_void_p()
    code = lib.bl_conv_plan_create(ctypes.byref(h), ctypes.byref(d))
    if code == 0:
        lib.bl_conv_plan_destroy(h)
    return code


@pytest.mark.parametrize("kw,code", [
    (dict(), 0),
    (dict(ndim=3), 1), (dict(N=0), 1), (dict(C_in=-1), 1), (dict(C_out=0), 1), (dict(H=0), 1),
    (dict(W=0), 1), (dict(K=0), 1), (dict(K=9), 2), (dict(K=9, H=20, W=20), 2),
    (dict(c=1.0), 1), (dict(c=-0.1), 1), (dict(c=float("nan")), 1), (dict(c=0.999), 0),
    (dict(pad_lo=(-1, 0)), 1), (dict(fft_h=9, fft_w=8), 0), (dict(fft_h=9, fft_w=7), 1), (dict(fft_h=7), 1), (dict(fft_h=12, fft_w=10), 0),
    (dict(flags=1), 0), (dict(flags=2), 0), (dict(flags=3), 0), (dict(flags=4), 1), (dict(flags=0x80000000), 1), (dict(H=2, W=2, K=3), 1), (dict(H=2, W=2, K=3, pad_lo=(1, 1)), 0),
    (dict(ndim=1, W=1, H=10), 0), (dict(ndim=1, W=2, H=10), 1), (dict(ndim=1, W=1, H=10, pad_lo=(0, 1)), 1),
    (dict(ndim=1, W=1, H=10, fft_w=4), 1), (dict(ndim=1, W=1, H=10, fft_h=9), 1),
    # the largest grid side is 4096 points
    (dict(ndim=1, W=1, H=4096), 0), (dict(ndim=1, W=1, H=4097), 2), (dict(H=3, W=4096), 0), (dict(H=4097, W=8), 2),
    (dict(ndim=1, W=1, H=10, fft_h=4097), 2),
    # shapes no kernel path holds: a plane over 160 KB of LDS, more than 65535 kept bins
    (dict(H=8, W=4096), 2), (dict(H=400, W=400), 2), (dict(H=128, W=128, c=0.5), 0),
])
def test_plan_create_validation(kw, code):
    assert _create(**kw) == code


def test_bf16_flag_keeps_the_band_and_halves_the_stored_spectra():
    """Reduced precision changes the stored spectra and the arithmetic of the
    channel sums only: the band and the grid are those of the fp32 plan, and
    X, W and DY take 4 bytes per complex value instead of 8."""
    def up(v):
        return (v + 255) // 256 * 256

    for args in [(2, 3, 16, 24, (20, 20), 3, (1, 1, 1, 1), 0.5), (1, 5, 3, 7, (90,), 5, (2, 2), 0.3)]:
        a = blconv.Plan(*args)
        b = blconv.Plan(*args, desc_flags=blconv.BL_DESC_BF16_SPECTRA)
        assert (a.fft, a.r_h, a.r_w, a.kept, a.total, a.c_eff) == (b.fft, b.r_h, b.r_w, b.kept, b.total, b.c_eff)
        assert np.array_equal(a.mask(), b.mask())
        _, N, Ci, Co = args[:4]
        for plan, eb in ((a, 8), (b, 4)):
            o = plan.offsets
            assert o["X"] == 0
            assert o["W"] == up(plan.kept * N * Ci * eb)
            assert o["DY"] == o["W"] + up(plan.kept * Ci * Co * eb)
        saved = (up(a.kept * N * Ci * 8) - up(a.kept * N * Ci * 4) + up(a.kept * Ci * Co * 8)
                 - up(a.kept * Ci * Co * 4) + up(a.kept * N * Co * 8) - up(a.kept * N * Co * 4))
        assert a.workspace_bytes - b.workspace_bytes == saved


def test_null_arguments_are_rejected_without_gpu():
    lib = blconv.load()
    assert lib.bl_conv_plan_create(None, None) == 1
    assert lib.bl_conv_plan_destroy(None) == 1
    assert lib.bl_conv_plan_info(None, None, None, None, None, None, None, None) == 1
    assert lib.bl_conv_workspace_size(None, None) == 1
    # compute calls validate on the host before touching the GPU
    assert lib.bl_conv_forward(None, None, None, None, None, 0, None) == 1
    assert lib.bl_conv_backward_input(None, None, None, None, None, 0, None) == 1
    assert lib.bl_conv_backward_weight(None, None, None, None, None, 0, None) == 1
    assert lib.bl_conv_backward(None, None, None, None, None, None, None, 0, None) == 1
    p = blconv.Plan(2, 1, 1, 1, (8, 8), 3, (1, 1, 1, 1), 0.5)
    h = p._h
    assert lib.bl_conv_forward(h, None, None, None, None, 0, None) == 1
    # bad flags
    assert lib.bl_conv_forward(h, 8, 8, 8, 8, 0x4, None) == 1
    assert lib.bl_conv_backward_input(h, 8, 8, 8, 8, 0x1, None) == 1
    assert lib.bl_conv_backward_weight(h, 8, 8, 8, 8, 0x2, None) == 1
    assert lib.bl_conv_backward(h, 8, 8, 8, 8, 8, 8, 0x8, None) == 1
    # a tensor missing without its reuse flag
    assert lib.bl_conv_backward(h, None, 8, 8, 8, 8, 8, 0x3, None) == 1
    assert lib.bl_conv_backward(h, 8, None, 8, 8, 8, 8, 0x5, None) == 1
    assert lib.bl_conv_backward(h, 8, 8, None, 8, 8, 8, 0x6, None) == 1
    assert lib.bl_conv_backward(h, 8, 8, 8, None, 8, 8, 0x7, None) == 1
    # fine-grained top compression: argument checks happen before any HIP call
    ws8 = ctypes.c_void_p(8)
    assert lib.bl_conv_zero_smallest(None, None, ws8, 0, 1, 0, None) == 1
    assert lib.bl_conv_zero_smallest(h, None, None, 0, 1, 1, None) == 1
    assert lib.bl_conv_zero_smallest(h, None, ws8, 0, -1, 1, None) == 1
    assert lib.bl_conv_zero_smallest(h, None, ws8, 2, 1, 1, None) == 1
    assert lib.bl_conv_zero_smallest(h, None, ws8, 0, 1, 0x2, None) == 1  # BL_REUSE_W with BL_SPEC_X
    assert lib.bl_conv_zero_smallest(h, None, ws8, 1, 1, 0x1, None) == 1  # BL_REUSE_X with BL_SPEC_W
    assert lib.bl_conv_zero_smallest(h, None, ws8, 0, 1, 0, None) == 1    # no source, no reuse
    # wrong sizes for host copies
    m = np.zeros(p.total + 1, np.uint8)
    assert lib.bl_conv_plan_get_mask(h, m.ctypes.data, m.size) == 1
    assert lib.bl_status_string(3) == b"workspace too small"


# ------------------------------------------- energy-based rate (host rule) --


def _plan_t(plan, layer):
    L = _grid(layer)
    return (L // 2 - plan.r_w) if layer.ndim == 1 else (L[0] // 2 - plan.r_h)


def _energies_in_bin_order(plan, layer, E):
    u, v = plan.bins()
    return E[v] if layer.ndim == 1 else E[u, v]


def test_rate_for_energy_matches_oracle():
    """The library's host rule, fed the oracle's bin energies in the plan's bin
    order, picks the oracle's band, reports its preserved fraction, and returns a
    rate for which a new plan peels exactly that many layers."""
    rng = np.random.default_rng(11)
    checked = 0
    for i in range(60):
        layer = synth.random_layer(rng, 1 if i % 2 else 2)
        x = synth.random_inputs(layer, 50 + i)[0].astype(np.float64)
        if layer.ndim == 1:
            E, last = bo.bin_energy_1d(x, layer.pad), bo.last_layer_kept(1, _grid(layer))
        else:
            E, last = bo.bin_energy_2d(x, layer.pad), bo.last_layer_kept(2, _grid(layer))
        f = bo.preserved_fractions(E, last)
        plan = blconv.plan_for_layer(layer, 0.0)
        e = _energies_in_bin_order(plan, layer, E)
        for fraction in (0.3, 0.6, 0.9, 0.99):
            want = bo.layers_for_energy(fraction, f)
            if np.min(np.abs(f - fraction)) < 1e-9:
                continue  # a tie within rounding: either side is correct
            t, c, kept_f = plan.rate_for_energy(e, fraction)
            assert t == want, (layer, fraction, t, want)
            assert abs(kept_f - f[want]) < 1e-12
            assert _plan_t(blconv.plan_for_layer(layer, c), layer) == want
            checked += 1
    assert checked > 150


def test_rate_for_energy_on_a_compressed_plan():
    """With a plan that already peels t0 layers the fractions are of the energy
    of its own bins, and the band chosen peels at least t0 layers."""
    layer = synth.Layer("e2d", 2, 2, 3, 4, 14, 14, 3, (1, 1, 1, 1), "blur")
    x = synth.random_inputs(layer, 3)[0].astype(np.float64)
    E, last = bo.bin_energy_2d(x, layer.pad), bo.last_layer_kept(2, _grid(layer))
    plan = blconv.plan_for_layer(layer, 0.5)
    t0 = _plan_t(plan, layer)
    e = _energies_in_bin_order(plan, layer, E)
    own = E[last >= t0].sum()
    for fraction in (0.5, 0.8, 0.95, 1.0):
        t, c, kept_f = plan.rate_for_energy(e, fraction)
        assert t >= t0
        assert E[last >= t].sum() / own >= fraction - 1e-12
        assert t == last.max() or E[last >= t + 1].sum() / own < fraction


def test_rate_for_energy_edge_cases():
    layer = synth.Layer("e1d", 1, 1, 1, 1, 20, 1, 3, (1, 1), "walk")
    plan = blconv.plan_for_layer(layer, 0.0)
    zero = np.zeros(plan.kept)
    t, c, f = plan.rate_for_energy(zero, 0.9)
    assert t == 22 // 2 and f == 1.0 and _plan_t(blconv.plan_for_layer(layer, c), layer) == t
    dc = zero.copy()
    dc[0] = 5.0
    assert plan.rate_for_energy(dc, 1.0)[0] == 11
    top = zero.copy()
    top[-1] = 1.0
    t, c, f = plan.rate_for_energy(top, 1.0)
    assert t == 0 and c == 0.0
    for bad in (0.0, -0.1, 1.5, float("nan")):
        with pytest.raises(blconv.BlError) as e:
            plan.rate_for_energy(dc, bad)
        assert e.value.code == 1
    neg = dc.copy()
    neg[3] = -1.0
    with pytest.raises(blconv.BlError):
        plan.rate_for_energy(neg, 0.5)
    with pytest.raises(blconv.BlError):
        plan.rate_for_energy(dc[:-1], 0.5)


def test_fine_band_for_energy_matches_oracle():
    """The library's fine-grained band, fed the oracle's bin energies in the
    plan's bin order, keeps the same bins as the oracle's (compared in the
    coarse plan's bin order), away from ties of the fraction; 1-D bands are the
    coarse ones; a too-small keep buffer is an error."""
    rng = np.random.default_rng(12)
    cut = checked = 0
    for i in range(40):
        layer = synth.random_layer(rng, 1 if i % 4 == 3 else 2)
        x = synth.random_inputs(layer, 80 + i)[0].astype(np.float64)
        if layer.ndim == 1:
            E, last = bo.bin_energy_1d(x, layer.pad), bo.last_layer_kept(1, _grid(layer))
        else:
            E, last = bo.bin_energy_2d(x, layer.pad), bo.last_layer_kept(2, _grid(layer))
        f = bo.preserved_fractions(E, last)
        plan = blconv.plan_for_layer(layer, 0.0)
        e = _energies_in_bin_order(plan, layer, E)
        for fraction in (0.5, 0.8, 0.9, 0.97):
            if np.min(np.abs(f - fraction)) < 1e-9:
                continue
            t_o, keep_o = bo.fine_energy_band(E, last, fraction)
            # the oracle's kept fraction must not sit on the threshold either
            band = last.ravel() >= t_o
            Eb = E.ravel()[band]
            if abs(Eb[keep_o].sum() / E.sum() - fraction) < 1e-9:
                continue
            t, c, kept_f, keep = plan.fine_band_for_energy(e, fraction)
            assert t == t_o
            coarse = blconv.plan_for_layer(layer, c)
            assert coarse.kept == keep.size == keep_o.size
            # the oracle's bins are in row-major (u, v) order, the same order the plans use
            assert np.array_equal(keep.astype(bool), keep_o), (layer, fraction)
            assert abs(kept_f - Eb[keep_o].sum() / E.sum()) < 1e-12
            cut += int(not keep.all())
            checked += 1
            if layer.ndim == 1:
                assert keep.all()
    assert checked > 60 and cut > 10
    lib = blconv.load()
    plan = blconv.plan_for_layer(synth.Layer("e", 2, 1, 1, 1, 6, 6, 3, (1, 1, 1, 1), "blur"), 0.0)
    e = np.ones(plan.kept)
    n = ctypes.c_size_t()
    t, c, pr = ctypes.c_int(), ctypes.c_double(), ctypes.c_double()
    buf = np.zeros(1, np.uint8)
    assert lib.bl_conv_fine_band_for_energy(plan._h, e.ctypes.data, e.size, 0.5, ctypes.byref(t), ctypes.byref(c),
                                            ctypes.byref(pr), buf.ctypes.data, 0, ctypes.byref(n)) == 1
    assert lib.bl_conv_zero_bins(None, None, 0, None, None) == 1
    assert lib.bl_conv_zero_bins(plan._h, ctypes.c_void_p(8), 2, ctypes.c_void_p(8), None) == 1
