"""GPU parity: the HIP library against the fp64 oracle on identical inputs.

Bar: for each of y, dx and dw (fp32 path vs fp64 oracle) both the relative
Frobenius error and the largest element error max|g - o| / max|o| are at most
1e-4, so an error confined to a few elements of a large output is not diluted
by the norm; stored spectra <= 1e-5 at unit level; masks byte-equal (CPU
test).  Every compute call goes through the C ABI (ctypes binding).
"""
import numpy as np
import pytest

from oracle import bl_oracle as bo
from paper_1911_09287_amd import blconv, synth

pytestmark = pytest.mark.gpu

TOL = 1e-4
SPEC_TOL = 1e-5


def rel(a, b):
    return float(np.linalg.norm(np.ravel(a - b)) / max(np.linalg.norm(np.ravel(b)), 1e-30))


def elem(a, b):
    """Largest element error relative to the largest reference element."""
    d = np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))
    return float(d.max() / max(float(np.abs(b).max()), 1e-30)) if d.size else 0.0


def err(a, b):
    """The fp32 parity measure: the larger of the norm-wise and element-wise errors."""
    return max(rel(a, b), elem(a, b))


@pytest.fixture(scope="module")
def torch():
    import torch as _torch
    if not _torch.cuda.is_available():
        pytest.skip("no GPU")
    blconv.load()
    return _torch


def say(*a):
    print(*a, flush=True)


def gpu_passes(torch, layer, c, x, w, dy, reuse=True, poison=True, fft=None, desc_flags=0):
    plan = blconv.plan_for_layer(layer, c, fft, desc_flags)
    dev = torch.device("cuda:0")
    ws = plan.workspace(dev)
    if poison:
        ws.fill_(0xFF)  # every float32 word of the workspace is a NaN
    xt, wt, dyt = (torch.from_numpy(a).to(dev) for a in (x, w, dy))
    nan = float("nan")
    y = torch.full(plan.y_shape(), nan, device=dev) if poison else torch.empty(plan.y_shape(), device=dev)
    dx = torch.full(plan.x_shape(), nan, device=dev) if poison else torch.empty(plan.x_shape(), device=dev)
    dw = torch.full(plan.w_shape(), nan, device=dev) if poison else torch.empty(plan.w_shape(), device=dev)
    plan.forward(xt, wt, y, ws)
    plan.backward_input(dyt, wt, dx, ws, flags=blconv.BL_REUSE_W if reuse else 0)
    plan.backward_weight(xt, dyt, dw, ws, flags=(blconv.BL_REUSE_X | blconv.BL_REUSE_DY) if reuse else 0)
    torch.cuda.synchronize()
    return y.cpu().numpy(), dx.cpu().numpy(), dw.cpu().numpy(), plan, ws


def oracle_passes(layer, c, x, w, dy, fft=None, rounding=None):
    spatial = (layer.H,) if layer.ndim == 1 else (layer.H, layer.W)
    return (bo.forward(x, w, layer.pad, c, fft, rounding),
            bo.backward_input(dy, w, spatial, layer.pad, c, fft, rounding),
            bo.backward_weight(x, dy, layer.K, layer.pad, c, fft, rounding))


CASES = [(cfg, li, c) for cfg in sorted(synth.WORKLOADS) for li in range(len(synth.WORKLOADS[cfg].layers))
         for c in synth.WORKLOADS[cfg].rates]


@pytest.mark.parametrize("cfg,li,c", CASES, ids=[f"C{a}-L{b}-c{c}" for a, b, c in CASES])
def test_config_parity(torch, cfg, li, c):
    layer = synth.WORKLOADS[cfg].layers[li]
    say(f"[parity] config {cfg} layer {layer.name} c={c}")
    x, w, dy = synth.layer_inputs(cfg, li)
    y, dx, dw, plan, ws = gpu_passes(torch, layer, c, x, w, dy)
    ry, rdx, rdw = oracle_passes(layer, c, x, w, dy)
    errs = (err(y, ry), err(dx, rdx), err(dw, rdw))
    say(f"    rel err y={errs[0]:.2e} dx={errs[1]:.2e} dw={errs[2]:.2e} kept={plan.kept}/{plan.total}")
    assert all(np.isfinite(a).all() for a in (y, dx, dw))
    assert max(errs) <= TOL, errs


def test_stored_spectra_match_oracle(torch):
    """Unit level: X, W and DY left in the workspace vs the oracle's kept spectra."""
    for cfg, li, c in ((1, 0, 0.5), (3, 0, 0.25), (2, 1, 0.5), (5, 0, 0.75), (3, 3, 0.0)):
        layer = synth.WORKLOADS[cfg].layers[li]
        say(f"[spectra] config {cfg} layer {layer.name} c={c}")
        x, w, dy = synth.layer_inputs(cfg, li)
        _, _, _, plan, ws = gpu_passes(torch, layer, c, x, w, dy)
        if layer.ndim == 2:
            Lh, Lw = plan.fft
            X = bo.kept_spectrum_2d(x, (layer.pad[0], layer.pad[2]), Lh, Lw, c)
            DY = bo.kept_spectrum_2d(dy, (0, 0), Lh, Lw, c)
            Wf = bo.kept_filter_spectrum_2d(w, Lh, Lw, c)
        else:
            L = plan.fft[0]
            X = bo.kept_spectrum_1d(x, layer.pad[0], L, c)
            DY = bo.kept_spectrum_1d(dy, 0, L, c)
            Wf = bo.kept_filter_spectrum_1d(w, L, c)
        gX = plan.spectrum(ws, "X").cpu().numpy().reshape(X.shape)
        gW = plan.spectrum(ws, "W").cpu().numpy().reshape(Wf.shape)
        gDY = plan.spectrum(ws, "DY").cpu().numpy().reshape(DY.shape)
        assert err(gX, X) <= SPEC_TOL and err(gW, Wf) <= SPEC_TOL and err(gDY, DY) <= SPEC_TOL


@pytest.mark.parametrize("ndim", [1, 2])
def test_random_small_layers(torch, ndim):
    """Odd and even sizes, asymmetric padding, larger grids, ragged tiles."""
    rng = np.random.default_rng(40 + ndim)
    for i in range(24):
        layer = synth.random_layer(rng, ndim, max_hw=20, max_c=70, max_n=5, max_k=8 if ndim == 1 else 6)
        if ndim == 2 and layer.K > 8:
            continue
        c = float(rng.choice([0.0, 0.1, 0.5, 0.9]))
        fft = None
        if rng.random() < 0.3:
            if ndim == 1:
                fft = layer.H + layer.pad[0] + layer.pad[1] + int(rng.integers(0, 5))
            else:
                fft = (layer.H + layer.pad[0] + layer.pad[1] + int(rng.integers(0, 4)),
                       layer.W + layer.pad[2] + layer.pad[3] + int(rng.integers(0, 4)))
        say(f"[random] ndim={ndim} #{i} {layer} c={c} fft={fft}")
        x, w, dy = synth.random_inputs(layer, 500 + i)
        y, dx, dw, plan, _ = gpu_passes(torch, layer, c, x, w, dy, fft=fft)
        ry, rdx, rdw = oracle_passes(layer, c, x, w, dy, fft)
        assert max(err(y, ry), err(dx, rdx), err(dw, rdw)) <= TOL


def test_reuse_flags_give_identical_results(torch):
    for cfg, li, c in ((1, 0, 0.5), (2, 0, 0.25), (4, 1, 0.75)):
        layer = synth.WORKLOADS[cfg].layers[li]
        say(f"[reuse] config {cfg} layer {layer.name} c={c}")
        x, w, dy = synth.layer_inputs(cfg, li)
        a = gpu_passes(torch, layer, c, x, w, dy, reuse=True)
        b = gpu_passes(torch, layer, c, x, w, dy, reuse=False)
        for u, v in zip(a[:3], b[:3]):
            assert np.array_equal(u, v)


def test_adjoint_identity_fp32(torch):
    """<dy, y> = <dx, x> = <dw, w> on the GPU path: the three passes are adjoint."""
    for cfg, li, c in ((1, 0, 0.5), (3, 1, 0.25), (2, 2, 0.75), (5, 0, 0.5)):
        layer = synth.WORKLOADS[cfg].layers[li]
        say(f"[adjoint] config {cfg} layer {layer.name} c={c}")
        x, w, dy = synth.layer_inputs(cfg, li)
        y, dx, dw, _, _ = gpu_passes(torch, layer, c, x, w, dy)
        a = float((dy.astype(np.float64) * y).sum())
        b = float((dx.astype(np.float64) * x).sum())
        d = float((dw.astype(np.float64) * w).sum())
        scale = float(np.abs(dy).astype(np.float64).ravel() @ np.abs(y).astype(np.float64).ravel())
        assert abs(a - b) <= 1e-5 * scale and abs(a - d) <= 1e-5 * scale


def test_edge_cases(torch):
    """Degenerate shapes: 1x1 maps, K = 1, a filter as large as the padded input,
    a single channel and sample, the highest rate (DC only)."""
    cases = [
        synth.Layer("one_pixel", 2, 1, 1, 1, 1, 1, 1, (0, 0, 0, 0), "blur"),
        synth.Layer("k_eq_input", 2, 2, 3, 2, 5, 5, 5, (0, 0, 0, 0), "blur"),
        synth.Layer("k1", 2, 3, 5, 7, 6, 9, 1, (0, 0, 0, 0), "blur"),
        synth.Layer("pad_only", 2, 1, 2, 2, 1, 1, 3, (1, 1, 1, 1), "blur"),
        synth.Layer("len1", 1, 2, 2, 2, 1, 1, 1, (0, 0), "walk"),
        synth.Layer("k8_1d", 1, 3, 2, 3, 8, 1, 8, (0, 0), "walk"),
        synth.Layer("wide", 2, 1, 1, 1, 2, 40, 3, (1, 1, 1, 1), "blur"),
    ]
    for layer in cases:
        for c in (0.0, 0.5, 0.999):
            say(f"[edge] {layer.name} c={c}")
            x, w, dy = synth.random_inputs(layer, 11)
            y, dx, dw, plan, _ = gpu_passes(torch, layer, c, x, w, dy)
            ry, rdx, rdw = oracle_passes(layer, c, x, w, dy)
            assert max(err(y, ry), err(dx, rdx), err(dw, rdw)) <= TOL, (layer.name, c)


def test_largest_grids(torch):
    """Grid sides at the 4096-point limit (1-D length 4096), a 2-D map 2048
    wide, and a large 2-D grid outside the fast transforms (66 x 66), through
    the direct DFT path (a plane per block with up to 160 KB of LDS where 64 KB
    does not hold it), at rates 0 and 0.5."""
    cases = [synth.Layer("max1d", 1, 2, 2, 3, 4090, 1, 7, (3, 3), "walk"),
             synth.Layer("wide2d", 2, 1, 2, 2, 3, 2046, 3, (1, 1, 1, 1), "blur"),
             synth.Layer("grid66", 2, 2, 3, 4, 64, 64, 3, (1, 1, 1, 1), "blur")]
    for i, layer in enumerate(cases):
        for c in (0.0, 0.5):
            say(f"[max] {layer.name} c={c}")
            x, w, dy = synth.random_inputs(layer, 2700 + i)
            y, dx, dw, plan, _ = gpu_passes(torch, layer, c, x, w, dy)
            ry, rdx, rdw = oracle_passes(layer, c, x, w, dy)
            errs = (err(y, ry), err(dx, rdx), err(dw, rdw))
            say(f"    grid {plan.fft} kept {plan.kept}/{plan.total}; rel err {errs}")
            assert max(errs) <= TOL, errs


def test_1d_long_sequences(torch):
    """1-D lengths that take the chirp-z (Bluestein) path with FFT sizes 256,
    512 and 1024, odd and even grids, offsets, grid overrides, and lengths
    beyond it (direct DFT path)."""
    rng = np.random.default_rng(77)
    for i in range(16):
        L = int(rng.integers(60, 700))
        K = int(rng.integers(1, 9))
        lo, hi = int(rng.integers(0, K)), int(rng.integers(0, K))
        layer = synth.Layer("long1d", 1, int(rng.integers(1, 4)), int(rng.integers(1, 20)),
                            int(rng.integers(1, 20)), L, 1, K, (lo, hi), "walk")
        c = float(rng.choice([0.0, 0.25, 0.5, 0.75, 0.9]))
        fft = None if rng.random() < 0.6 else L + lo + hi + int(rng.integers(0, 40))
        say(f"[long1d] #{i} L={L} K={K} pad=({lo},{hi}) c={c} fft={fft}")
        x, w, dy = synth.random_inputs(layer, 900 + i)
        y, dx, dw, plan, _ = gpu_passes(torch, layer, c, x, w, dy, fft=fft)
        ry, rdx, rdw = oracle_passes(layer, c, x, w, dy, fft)
        errs = (err(y, ry), err(dx, rdx), err(dw, rdw))
        say(f"    rel err {errs}")
        assert max(errs) <= TOL


def test_1d_many_series(torch):
    """1-D layers with thousands of series, so that waves of the chirp-z kernel
    run more than one round: inputs longer than 512 (each round loaded when it
    starts) and shorter ones (the next round loaded during the current one),
    forward and inverse, paired and single series."""
    cases = [
        (synth.Layer("rounds_long", 1, 64, 160, 4, 600, 1, 3, (1, 1), "walk"), 0.5),
        (synth.Layer("rounds_short", 1, 64, 160, 4, 300, 1, 5, (2, 2), "walk"), 0.5),
        (synth.Layer("rounds_single", 1, 40, 130, 3, 510, 1, 3, (1, 1), "walk"), 0.0),
    ]
    for i, (layer, c) in enumerate(cases):
        say(f"[many series] {layer.name} c={c}")
        x, w, dy = synth.random_inputs(layer, 1300 + i)
        y, dx, dw, plan, _ = gpu_passes(torch, layer, c, x, w, dy)
        ry, rdx, rdw = oracle_passes(layer, c, x, w, dy)
        errs = (err(y, ry), err(dx, rdx), err(dw, rdw))
        say(f"    rel err {errs}")
        assert max(errs) <= TOL


def test_2d_fast_grids(torch):
    """Grids 6, 10, 18, 34, 58 (2 x odd: the mixed-radix 2-D path) reached with
    other filter sizes, asymmetric padding, non-square inputs and grid
    overrides, at several rates."""
    rng = np.random.default_rng(123)
    cases = []
    for L in (6, 10, 18, 34, 58):
        for _ in range(3):
            K = int(rng.integers(1, min(L, 8) + 1))
            pt, pb, pl, pr = (int(rng.integers(0, K)) for _ in range(4))
            H, W = L - pt - pb, L - pl - pr
            if H < 1 or W < 1 or H + pt + pb < K or W + pl + pr < K:
                continue
            cases.append((synth.Layer("fast2d", 2, int(rng.integers(1, 4)), int(rng.integers(1, 24)),
                                      int(rng.integers(1, 24)), H, W, K, (pt, pb, pl, pr), "blur"), None))
        # an input smaller than the grid, reached through the grid override
        cases.append((synth.Layer("fast2d_ovr", 2, 2, 5, 7, L - 5, L - 4, 3, (1, 1, 0, 2), "blur"), (L, L)))
    for layer, fft in cases:
        for c in (0.0, 0.3, 0.6, 0.9):
            say(f"[fast2d] {layer} c={c} fft={fft}")
            x, w, dy = synth.random_inputs(layer, 77)
            y, dx, dw, plan, _ = gpu_passes(torch, layer, c, x, w, dy, fft=fft)
            ry, rdx, rdw = oracle_passes(layer, c, x, w, dy, fft)
            errs = (err(y, ry), err(dx, rdx), err(dw, rdw))
            assert max(errs) <= TOL, errs


def test_wgrad_paths(torch):
    """Each route of the weight-gradient inverse DFT: one pass over all bins
    for wide layers (taps padded to 16 or exact), bin slices whose weights fill
    the LDS cap (8 x 8 taps), channel-tiled slices for more than 256 output
    channels, a single slice written without partial sums, and 16 x 16
    channel tiles over all bins (2 and 4 groups per tile, ragged tiles)."""
    cases = [
        synth.Layer("wg_wide_k3", 2, 2, 128, 128, 8, 8, 3, (1, 1, 1, 1), "blur"),
        synth.Layer("wg_wide_k4", 2, 2, 128, 128, 8, 8, 4, (2, 1, 2, 1), "blur"),
        synth.Layer("wg_lds_cap_k8", 2, 1, 256, 256, 32, 32, 8, (0, 0, 0, 0), "blur"),
        synth.Layer("wg_tiled_f384", 2, 2, 16, 384, 12, 12, 3, (1, 1, 1, 1), "blur"),
        synth.Layer("wg_single_slice", 1, 2, 4, 300, 20, 1, 3, (1, 1), "walk"),
        synth.Layer("wg_tile_ng2", 2, 2, 256, 256, 8, 8, 3, (1, 1, 1, 1), "blur"),
        synth.Layer("wg_tile_ng4_ragged", 2, 2, 200, 260, 6, 6, 4, (2, 1, 2, 1), "blur"),
    ]
    for i, layer in enumerate(cases):
        for c in (0.0, 0.5):
            say(f"[wgrad] {layer.name} c={c}")
            x, w, dy = synth.random_inputs(layer, 1500 + i)
            y, dx, dw, plan, _ = gpu_passes(torch, layer, c, x, w, dy)
            # the oracle's forward of the 65536-filter case takes a minute: dw only there
            rdw = bo.backward_weight(x, dy, layer.K, layer.pad, c, None)
            errs = [err(dw, rdw)]
            if layer.C_in * layer.C_out < 65536:
                ry, rdx, _ = oracle_passes(layer, c, x, w, dy)
                errs += [err(y, ry), err(dx, rdx)]
            say(f"    rel err {errs}")
            assert max(errs) <= TOL, errs


def test_contraction_shapes(torch):
    """The tiled contraction at edge shapes: ragged tiles in m, n and k; a
    single bin with 2048 input channels (k split over many partial tiles,
    summed in a fixed order); few bins with long k; an odd channel count (the
    operands' 16-byte pairs do not align: the generic path); a 1-D layer.
    Each twice in a row on one workspace: results equal run to run."""
    cases = [
        (synth.Layer("ragged", 2, 70, 66, 130, 6, 6, 3, (1, 1, 1, 1), "blur"), 0.0),
        (synth.Layer("one_bin", 2, 64, 2048, 256, 1, 1, 1, (0, 0, 0, 0), "blur"), 0.0),
        (synth.Layer("long_k", 2, 96, 640, 640, 2, 2, 1, (0, 0, 0, 0), "blur"), 0.0),
        (synth.Layer("odd_k", 2, 64, 65, 64, 4, 4, 3, (1, 1, 1, 1), "blur"), 0.5),
        (synth.Layer("one_d", 1, 64, 96, 192, 60, 1, 3, (1, 1), "walk"), 0.5),
    ]
    for i, (layer, c) in enumerate(cases):
        say(f"[contraction] {layer.name} c={c}")
        x, w, dy = synth.random_inputs(layer, 1900 + i)
        plan = blconv.plan_for_layer(layer, c)
        dev = torch.device("cuda:0")
        ws = plan.workspace(dev)
        ws.fill_(0xFF)
        xt, wt, dyt = (torch.from_numpy(a).to(dev) for a in (x, w, dy))
        outs = []
        for rep in range(2):
            y = torch.full(plan.y_shape(), float("nan"), device=dev)
            dx = torch.full(plan.x_shape(), float("nan"), device=dev)
            dw = torch.full(plan.w_shape(), float("nan"), device=dev)
            plan.forward(xt, wt, y, ws)
            plan.backward_input(dyt, wt, dx, ws, flags=blconv.BL_REUSE_W)
            plan.backward_weight(xt, dyt, dw, ws, flags=blconv.BL_REUSE_X | blconv.BL_REUSE_DY)
            torch.cuda.synchronize()
            outs.append([t.cpu().numpy() for t in (y, dx, dw)])
        for a, b in zip(*outs):
            assert np.array_equal(a, b)
        ry, rdx, rdw = oracle_passes(layer, c, x, w, dy)
        errs = (err(outs[0][0], ry), err(outs[0][1], rdx), err(outs[0][2], rdw))
        say(f"    err {errs}")
        assert max(errs) <= TOL, errs


def test_combined_backward(torch):
    """bl_conv_backward (both gradients from one DY spectrum; the two
    contractions in one launch where they share a tile shape, the pass with
    the longer sum split along k into partial spectra that the inverse
    transforms add) against the oracle, equal run to run and with or without
    reuse flags, and within rounding of the separate backward calls.  The
    ResNet stack at c = 0.5 covers the 64-channel layer (grad-weight split in
    two, its partials added as more bin slices), the 128-channel layer (no
    split), the 256-channel layer (different tiles: two launches) and the
    512-channel layer (grad-input split in four, added by the 2-D inverse as
    it loads); the 64-channel layer at c = 0 and 0.75 (grad-weight partials
    summed by the one-pass inverse DFT as it loads them); then a ragged layer,
    a 1-D layer (grad-input partials summed before the chirp-z inverse), a
    layer whose grad-weight partials the one-pass inverse DFT sums beside the
    2-D inverse, and a bfloat16 plan."""
    # (layer, rate, plan flags, workload (config, layer) or None for random inputs)
    cases = [(synth.WORKLOADS[3].layers[i], 0.5, 0, (3, i)) for i in range(4)]
    cases += [(synth.WORKLOADS[3].layers[0], c, 0, (3, 0)) for c in (0.0, 0.75)]
    cases += [(synth.Layer("ragged", 2, 70, 66, 130, 6, 6, 3, (1, 1, 1, 1), "blur"), 0.0, 0, None),
              (synth.WORKLOADS[2].layers[1], 0.5, 0, (2, 1)),
              (synth.Layer("split_wide", 2, 128, 32, 32, 8, 8, 3, (1, 1, 1, 1), "blur"), 0.0, 0, None),
              (synth.Layer("bf_pair", 2, 64, 32, 64, 12, 12, 3, (1, 1, 1, 1), "blur"), 0.5,
               blconv.BL_DESC_BF16_SPECTRA, None)]
    dev = torch.device("cuda:0")
    for i, (layer, c, flags, src) in enumerate(cases):
        say(f"[backward] {layer.name} c={c} desc_flags={flags}")
        x, w, dy = synth.layer_inputs(*src) if src else synth.random_inputs(layer, 2100 + i)
        plan = blconv.plan_for_layer(layer, c, None, flags)
        ws = plan.workspace(dev)
        ws.fill_(0xFF)
        xt, wt, dyt = (torch.from_numpy(a).to(dev) for a in (x, w, dy))
        outs = []
        for reuse in (False, True, True):
            dx = torch.full(plan.x_shape(), float("nan"), device=dev)
            dw = torch.full(plan.w_shape(), float("nan"), device=dev)
            if reuse:
                plan.backward(None, None, None, dx, dw, ws,
                              flags=blconv.BL_REUSE_X | blconv.BL_REUSE_W | blconv.BL_REUSE_DY)
            else:
                plan.backward(dyt, wt, xt, dx, dw, ws)
            torch.cuda.synchronize()
            outs.append((dx.cpu().numpy(), dw.cpu().numpy()))
        for a, b in zip(outs[0], outs[1]):
            assert np.array_equal(a, b)
        for a, b in zip(outs[1], outs[2]):
            assert np.array_equal(a, b)
        sdx = torch.full(plan.x_shape(), float("nan"), device=dev)
        sdw = torch.full(plan.w_shape(), float("nan"), device=dev)
        plan.backward_input(dyt, wt, sdx, ws)
        plan.backward_weight(xt, dyt, sdw, ws)
        torch.cuda.synchronize()
        sep = (sdx.cpu().numpy(), sdw.cpu().numpy())
        rounding = bo.round_bf16 if flags else None
        spatial = (layer.H,) if layer.ndim == 1 else (layer.H, layer.W)
        ref = (bo.backward_input(dy, w, spatial, layer.pad, c, None, rounding),
               bo.backward_weight(x, dy, layer.K, layer.pad, c, None, rounding))
        errs = [err(a, b) for a, b in zip(outs[0], ref)]
        gaps = [rel(a, b) for a, b in zip(outs[0], sep)]
        say(f"    err vs oracle dx={errs[0]:.2e} dw={errs[1]:.2e}; vs separate calls {gaps}")
        assert all(np.isfinite(a).all() for a in outs[0])
        assert max(errs) <= (BF16_TOL if flags else TOL), errs
        assert max(gaps) <= 1e-5, gaps


def test_combined_backward_random_medium(torch):
    """Forward and bl_conv_backward on random medium layers whose channel and
    batch counts reach the tiled contractions (multiples of the tile sizes and
    ragged counts, up to about 600 channels), so that the plan's choices of
    tile shape, pairing of the two backward contractions and k splits (partial
    spectra added by the inverses or the weight-gradient slices) vary from case
    to case; 2-D and 1-D, against the oracle and the separate backward calls."""
    rng = np.random.default_rng(3100)
    chans = [16, 32, 48, 64, 96, 128, 160, 192, 256, 320, 384, 512, 17, 33, 70, 130, 200, 260, 513, 600]
    dev = torch.device("cuda:0")
    done = 0
    while done < 14:
        ndim = 2 if done < 10 else 1
        N = int(rng.choice([1, 2, 8, 32, 64, 100, 128, 160]))
        ci, co = int(rng.choice(chans)), int(rng.choice(chans))
        K = int(rng.choice([3, 3, 3, 1, 5]))
        if ndim == 2:
            H = int(rng.choice([4, 6, 8, 12, 16, 20]))
            layer = synth.Layer("rand_med2d", 2, N, ci, co, H, H, K, (K // 2,) * 4, "blur")
            size = N * ci * co * H * H
        else:
            H = int(rng.integers(100, 600))
            layer = synth.Layer("rand_med1d", 1, N, ci, co, H, 1, K, (K // 2, K // 2), "walk")
            size = N * ci * co * H
        if size > 4e8:
            continue
        c = float(rng.choice([0.0, 0.25, 0.5, 0.75]))
        say(f"[backward-rand] {layer} c={c}")
        x, w, dy = synth.random_inputs(layer, 3200 + done)
        done += 1
        plan = blconv.plan_for_layer(layer, c)
        ws = plan.workspace(dev)
        ws.fill_(0xFF)
        xt, wt, dyt = (torch.from_numpy(a).to(dev) for a in (x, w, dy))
        y = torch.full(plan.y_shape(), float("nan"), device=dev)
        dx = torch.full(plan.x_shape(), float("nan"), device=dev)
        dw = torch.full(plan.w_shape(), float("nan"), device=dev)
        plan.forward(xt, wt, y, ws)
        plan.backward(dyt, None, None, dx, dw, ws, flags=blconv.BL_REUSE_W | blconv.BL_REUSE_X)
        sdx = torch.full(plan.x_shape(), float("nan"), device=dev)
        sdw = torch.full(plan.w_shape(), float("nan"), device=dev)
        plan.backward_input(dyt, wt, sdx, ws)
        plan.backward_weight(xt, dyt, sdw, ws)
        torch.cuda.synchronize()
        got = (y.cpu().numpy(), dx.cpu().numpy(), dw.cpu().numpy())
        ref = oracle_passes(layer, c, x, w, dy)
        errs = [err(a, b) for a, b in zip(got, ref)]
        gaps = [rel(a, b.cpu().numpy()) for a, b in zip(got[1:], (sdx, sdw))]
        say(f"    err y={errs[0]:.2e} dx={errs[1]:.2e} dw={errs[2]:.2e}; vs separate calls {gaps}")
        assert all(np.isfinite(a).all() for a in got)
        assert max(errs) <= TOL, errs
        assert max(gaps) <= 1e-5, gaps


def test_thin_contractions(torch):
    """Layers where a contraction size (batch, input or output channels) is at
    most 8, which run the memory-bound vector-ALU contraction: lanes over
    output columns with k split over a block's waves or not, strided and
    contiguous operands, and one output row per wave with a cross-lane sum."""
    cases = [
        synth.Layer("thin_c1_1d", 1, 64, 1, 128, 200, 1, 8, (3, 4), "walk"),
        synth.Layer("thin_c3_2d", 2, 4, 3, 64, 12, 12, 3, (1, 1, 1, 1), "blur"),
        synth.Layer("thin_f2_2d", 2, 16, 64, 2, 10, 10, 3, (1, 1, 1, 1), "blur"),
        synth.Layer("thin_n1_2d", 2, 1, 96, 80, 9, 9, 3, (1, 1, 1, 1), "blur"),
        synth.Layer("thin_f5_1d", 1, 70, 100, 5, 90, 1, 5, (2, 2), "walk"),
    ]
    for i, layer in enumerate(cases):
        for c in (0.0, 0.5):
            say(f"[thin] {layer.name} c={c}")
            x, w, dy = synth.random_inputs(layer, 1700 + i)
            y, dx, dw, plan, _ = gpu_passes(torch, layer, c, x, w, dy)
            ry, rdx, rdw = oracle_passes(layer, c, x, w, dy)
            errs = (err(y, ry), err(dx, rdx), err(dw, rdw))
            say(f"    rel err {errs}")
            assert max(errs) <= TOL, errs


# bfloat16 operands: a spectrum value that the fp32 transforms leave within
# their rounding error of a bfloat16 tie can round the other way than in the
# fp64 oracle (an error of one bfloat16 ulp, 2^-8 relative, in that value); at
# fp32 transform errors of ~1e-6 this happens to a few values in ten thousand
# and gives relative errors ~1e-4.  Rounding itself moves the result by ~2e-3,
# so the tolerance still tells a rounded contraction from an unrounded one.
BF16_TOL = 5e-4
BF16_EXACT_TOL = 1e-2


def test_bf16_contraction_parity(torch):
    """Plans with BL_DESC_BF16_SPECTRA against the oracle whose channel
    contraction rounds both operands to bfloat16 (round to nearest even) and
    sums exactly: the MFMA tiles (with and without split k), the thin
    vector-ALU contraction and the generic one, 1-D and 2-D."""
    cases = [
        synth.Layer("bf_tiled_2d", 2, 16, 32, 48, 12, 12, 3, (1, 1, 1, 1), "blur"),
        synth.Layer("bf_tiled_1d", 1, 32, 16, 24, 200, 1, 8, (3, 4), "walk"),
        synth.Layer("bf_split_2d", 2, 256, 16, 32, 8, 8, 3, (1, 1, 1, 1), "blur"),
        synth.Layer("bf_thin_2d", 2, 4, 3, 64, 12, 12, 3, (1, 1, 1, 1), "blur"),
        synth.Layer("bf_thin_1d", 1, 70, 100, 5, 90, 1, 5, (2, 2), "walk"),
        synth.Layer("bf_generic_2d", 2, 10, 17, 33, 9, 9, 3, (1, 1, 1, 1), "blur"),
    ]
    for i, layer in enumerate(cases):
        for c in (0.0, 0.5):
            say(f"[bf16] {layer.name} c={c}")
            x, w, dy = synth.random_inputs(layer, 1900 + i)
            got = gpu_passes(torch, layer, c, x, w, dy, desc_flags=blconv.BL_DESC_BF16_SPECTRA)[:3]
            ref = oracle_passes(layer, c, x, w, dy, rounding=bo.round_bf16)
            exact = oracle_passes(layer, c, x, w, dy)
            errs = [rel(a, b) for a, b in zip(got, ref)]
            errs_exact = [rel(a, b) for a, b in zip(got, exact)]
            gaps = [rel(a, b) for a, b in zip(ref, exact)]
            say(f"    rel err vs bf16 oracle {errs}; vs exact {errs_exact}; oracle gap {gaps}")
            assert all(np.isfinite(a).all() for a in got)
            assert max(errs) <= BF16_TOL, errs
            assert max(errs_exact) <= BF16_EXACT_TOL, errs_exact
            assert min(gaps) > 2 * BF16_TOL, gaps  # the tolerance separates rounded from exact


def _decode_bf16_pairs(words):
    u = np.ascontiguousarray(words).view(np.uint32)
    return (u << np.uint32(16)).view(np.float32), (u & np.uint32(0xFFFF0000)).view(np.float32)


def _check_bf16_words(words, ref):
    """Stored bfloat16 pairs against the oracle's spectrum rounded to bfloat16:
    equal, except parts whose fp32 value lay within its rounding error of a
    tie, which may sit one bfloat16 ulp away, and parts that are zero or tiny
    in exact arithmetic (imaginary parts of real bins), which keep the fp32
    transform's absolute error (1e-5 of the spectrum's RMS bounds it)."""
    re, im = _decode_bf16_pairs(words)
    got = np.concatenate([re.ravel(), im.ravel()]).astype(np.float64)
    r = np.asarray(ref).ravel()
    want = np.concatenate([bo.round_bf16(r.real), bo.round_bf16(r.imag)])
    diff = got != want
    frac = float(diff.mean())
    rms = float(np.sqrt(np.mean(np.abs(r) ** 2)))
    bound = 2.0 ** -7 * np.maximum(np.abs(got), np.abs(want)) + 1e-5 * rms
    excess = float(np.max((np.abs(got - want) - bound)[diff], initial=-1.0))
    assert excess <= 0, f"a stored value is more than one bfloat16 ulp off (by {excess:.3e}, rms {rms:.3e})"
    return frac


def test_bf16_stored_spectra_and_energy(torch):
    """With BL_DESC_BF16_SPECTRA the spectra X, W and DY are stored as
    bfloat16 pairs: every forward-transform path (2-D radix 2 x odd grids,
    1-D chirp-z over 1024 points with one or two series per transform and over
    256/512 points, the direct DFT on odd grids, the filter transform) against
    the oracle's spectra rounded to bfloat16, and the per-bin input energies of
    the stored spectrum against the oracle's energies of the rounded one."""
    dev = torch.device("cuda:0")
    cases = [(synth.WORKLOADS[3].layers[0], 0.25, synth.layer_inputs(3, 0)),
             (synth.WORKLOADS[5].layers[0], 0.5, synth.layer_inputs(5, 0)),
             (synth.WORKLOADS[2].layers[1], 0.0, synth.layer_inputs(2, 1)),
             (synth.WORKLOADS[2].layers[2], 0.5, synth.layer_inputs(2, 2))]
    small = [synth.Layer("bf_blue512_1d", 1, 24, 3, 5, 200, 1, 8, (3, 4), "walk"),
             synth.Layer("bf_direct_2d", 2, 6, 5, 7, 9, 9, 3, (1, 1, 1, 1), "blur")]
    for i, layer in enumerate(small):
        for c in (0.0, 0.5):
            cases.append((layer, c, synth.random_inputs(layer, 2300 + i)))
    for layer, c, (x, w, dy) in cases:
        say(f"[bf16 spectra] {layer.name} c={c}")
        _, _, _, plan, ws = gpu_passes(torch, layer, c, x, w, dy, desc_flags=blconv.BL_DESC_BF16_SPECTRA)
        if layer.ndim == 2:
            Lh, Lw = plan.fft
            X = bo.kept_spectrum_2d(x, (layer.pad[0], layer.pad[2]), Lh, Lw, c)
            DY = bo.kept_spectrum_2d(dy, (0, 0), Lh, Lw, c)
            Wf = bo.kept_filter_spectrum_2d(w, Lh, Lw, c)
        else:
            Lw = plan.fft[0]
            X = bo.kept_spectrum_1d(x, layer.pad[0], Lw, c)
            DY = bo.kept_spectrum_1d(dy, 0, Lw, c)
            Wf = bo.kept_filter_spectrum_1d(w, Lw, c)
        fr = [_check_bf16_words(plan.spectrum(ws, k).cpu().numpy(), ref) for k, ref in (("X", X), ("W", Wf), ("DY", DY))]
        say(f"    parts one ulp off: X {fr[0]:.1e} W {fr[1]:.1e} DY {fr[2]:.1e}")
        assert max(fr) <= 5e-2, fr  # systematic mis-rounding (truncation) would put about half off
        # energies of the stored (rounded) input spectrum, reusing it
        e = plan.input_energy(None, ws, flags=blconv.BL_REUSE_X).cpu().numpy()
        Xr = bo.round_bf16(X.real) + 1j * bo.round_bf16(X.imag)
        _, v = plan.bins()
        h = np.where((v == 0) | ((Lw % 2 == 0) & (v == Lw // 2)), 1.0, 2.0)
        want = h * np.sum(np.abs(Xr.reshape(plan.kept, -1)) ** 2, axis=1)
        err = rel(e, want)
        say(f"    energy rel err {err:.2e}")
        assert err <= 1e-4, err


def _stored_complex(plan, ws, which):
    """A stored spectrum as complex128 [kept][rows][cols], decoding bfloat16 pairs."""
    a = plan.spectrum(ws, which).cpu().numpy()
    if a.dtype == np.int32:
        re, im = _decode_bf16_pairs(a)
        return re.astype(np.float64) + 1j * im.astype(np.float64)
    return a.astype(np.complex128)


def _groups(S, which):
    """[groups][B * C] views (coefficient i = (bin i / C, channel i % C)) of a
    stored X [B][N][C] (groups = samples) or W [B][C][F] (groups = filters)."""
    if which == "X":
        return np.transpose(S, (1, 0, 2)).reshape(S.shape[1], -1)
    return np.transpose(S, (2, 0, 1)).reshape(S.shape[2], -1)


def _check_zeroed(before, after, ref, k, which, tie_tol):
    """Exactly the k smallest of each group zeroed (counted with the zeros it
    already had), the rest untouched bit for bit, the choice valid in the
    GPU's own values, and equal to the oracle's ranking except among
    coefficients within tie_tol of the oracle's k-th magnitude.  Returns the
    zero mask in the stored layout."""
    gb, ga, gr = _groups(before, which), _groups(after, which), _groups(ref, which)
    n = gb.shape[1]
    kk = min(k, n)
    za = ga == 0
    assert np.array_equal(ga[~za], gb[~za]), "a coefficient that was kept changed"
    counts = za.sum(axis=1)
    assert np.all(counts == np.maximum(kk, (gb == 0).sum(axis=1))), (counts[:4], kk)
    if 0 < kk < n:
        mb = np.abs(gb)
        hi = np.where(za, mb, -np.inf).max(axis=1)
        lo = np.where(~za, mb, np.inf).min(axis=1)
        assert np.all(hi <= lo * (1 + 1e-6)), "a zeroed coefficient is larger than a kept one"
        mr = np.abs(gr)
        thr = np.sort(mr, axis=1)[:, kk - 1:kk]
        zo = np.zeros_like(za)
        np.put_along_axis(zo, np.argsort(mr, axis=1, kind="stable")[:, :kk], True, axis=1)
        diff = za != zo
        rms = np.sqrt(np.mean(mr ** 2))
        assert np.all(np.abs(mr - thr)[diff] <= tie_tol * thr.repeat(n, axis=1)[diff] + 1e-6 * rms), \
            "the GPU's choice differs from the oracle's away from a tie"
    # back to the stored layout
    if which == "X":
        return np.transpose(za.reshape(before.shape[1], before.shape[0], before.shape[2]), (1, 0, 2))
    return np.transpose(za.reshape(before.shape[2], before.shape[0], before.shape[1]), (1, 2, 0))


def test_zero_smallest_parity(torch):
    """Fine-grained top compression on the GPU: per sample and per filter the
    k smallest-magnitude stored coefficients are zeroed (k = 1, a third, all
    but one, all, more than all), checked against the oracle's ranking and by
    the forward pass on the zeroed spectra against the oracle's forward with the
    same coefficients zeroed (and against forward_top where the choices agree);
    a 2-D workload layer, the 1-D stack's widest layer, small odd shapes, groups
    large enough to be split over several blocks, and bfloat16 spectra."""
    dev = torch.device("cuda:0")
    cases = [(synth.WORKLOADS[3].layers[0], 0.5, 0, synth.layer_inputs(3, 0)),
             (synth.WORKLOADS[2].layers[1], 0.5, 0, synth.layer_inputs(2, 1))]
    # the last: few groups of more than 65 536 coefficients, selected over
    # several blocks each (the others one block per group)
    small = [synth.Layer("top_2d_odd", 2, 3, 5, 7, 9, 11, 3, (1, 1, 1, 1), "blur"),
             synth.Layer("top_1d", 1, 4, 3, 6, 90, 1, 5, (2, 2), "walk"),
             synth.Layer("top_2d_wide", 2, 2, 80, 3, 40, 40, 3, (1, 1, 1, 1), "blur")]
    for i, layer in enumerate(small):
        cases.append((layer, 0.0, 0, synth.random_inputs(layer, 2400 + i)))
        cases.append((layer, 0.3, blconv.BL_DESC_BF16_SPECTRA, synth.random_inputs(layer, 2400 + i)))
    for layer, c, fl, (x, w, dy) in cases:
        plan = blconv.plan_for_layer(layer, c, None, fl)
        n = plan.kept * layer.C_in
        xt, wt = (torch.from_numpy(a).to(dev) for a in (x, w))
        if layer.ndim == 2:
            Lh, Lw = plan.fft
            Xo = bo.kept_spectrum_2d(x, (layer.pad[0], layer.pad[2]), Lh, Lw, c)
            Wo = bo.kept_filter_spectrum_2d(w, Lh, Lw, c)
        else:
            Xo = bo.kept_spectrum_1d(x, layer.pad[0], plan.fft[0], c)
            Wo = bo.kept_filter_spectrum_1d(w, plan.fft[0], c)
        Xo = Xo.reshape(plan.kept, layer.N, layer.C_in)
        tie = 1e-2 if fl else 1e-5
        for kx, kw in ((1, n // 3), (n // 3, 1), (n - 1, n), (n, n - 1), (n + 7, 0)):
            say(f"[top] {layer.name} c={c} flags={fl} kx={kx} kw={kw} of {n}")
            ws = plan.workspace(dev)
            ws.fill_(0xFF)
            y = torch.full(plan.y_shape(), float("nan"), device=dev)
            plan.forward(xt, wt, y, ws)
            Xb, Wb = _stored_complex(plan, ws, "X"), _stored_complex(plan, ws, "W")
            plan.zero_smallest(None, ws, "X", kx, flags=blconv.BL_REUSE_X)
            plan.zero_smallest(wt, ws, "W", kw)  # recomputes W first
            Xa, Wa = _stored_complex(plan, ws, "X"), _stored_complex(plan, ws, "W")
            zx = _check_zeroed(Xb, Xa, Xo, kx, "X", tie)
            zw = _check_zeroed(Wb, Wa, Wo, kw, "W", tie)
            plan.forward(None, None, y, ws, flags=blconv.BL_REUSE_X | blconv.BL_REUSE_W)
            torch.cuda.synchronize()
            got = y.cpu().numpy()
            want = bo.forward_zeroed(x, w, layer.pad, c, zx, zw)
            err = rel(got, want) if np.abs(want).max() > 0 else float(np.abs(got).max())
            agree = np.array_equal(zx, bo.top_zeroed(Xo, kx, False)) and np.array_equal(zw, bo.top_zeroed(Wo, kw, True))
            say(f"    forward rel err {err:.2e}; choice equal to the oracle's: {agree}")
            assert np.isfinite(got).all()
            assert err <= (BF16_EXACT_TOL if fl else TOL), err
            if agree and not fl:
                assert rel(got, bo.forward_top(x, w, layer.pad, c, kx, kw)) <= TOL


def test_fused_small_forward(torch):
    """BL_DESC_FUSED_FORWARD: the forward pass as one kernel after the filter
    transform, on small maps (4x4 and 8x8 workload layers, odd and even grids,
    1x1 maps, three input channels, output-channel groups that do not divide
    C_out), against the oracle; the input spectrum it stores serves the
    backward passes' reuse flags, and the fused kernel is the one that ran."""
    cases = [(synth.WORKLOADS[4].layers[2], c, synth.layer_inputs(4, 2)) for c in (0.0, 0.5)]
    cases += [(synth.WORKLOADS[3].layers[3], 0.25, synth.layer_inputs(3, 3)),
              (synth.WORKLOADS[3].layers[2], 0.75, synth.layer_inputs(3, 2))]
    small = [synth.Layer("fz_odd", 2, 5, 3, 7, 7, 9, 3, (1, 1, 1, 1), "blur"),
             synth.Layer("fz_1x1", 2, 3, 4, 5, 1, 1, 1, (0, 0, 0, 0), "blur"),
             synth.Layer("fz_pad2", 2, 2, 6, 37, 6, 6, 5, (2, 2, 2, 2), "blur")]
    for i, layer in enumerate(small):
        for c in (0.0, 0.4):
            cases.append((layer, c, synth.random_inputs(layer, 2500 + i)))
    for layer, c, (x, w, dy) in cases:
        say(f"[fused] {layer.name} c={c}")
        prof = blconv.Profile(capacity=256)
        with prof:
            y, dx, dw, plan, ws = gpu_passes(torch, layer, c, x, w, dy, desc_flags=blconv.BL_DESC_FUSED_FORWARD)
        names = [r[0] for r in prof.records()]
        ry, rdx, rdw = oracle_passes(layer, c, x, w, dy)
        errs = (err(y, ry), err(dx, rdx), err(dw, rdw))
        say(f"    rel err {errs}; kernels {sorted(set(names))}")
        assert "small_fwd" in names and "contract_fwd" not in names
        assert all(np.isfinite(a).all() for a in (y, dx, dw))
        assert max(errs) <= TOL, errs


def test_fine_band_forward(torch):
    """Fine-grained energy-based band on the GPU: energies of the input on a
    rate-0 plan, the fine band from them, a plan at the coarse rate, X and W
    computed and zeroed at the dropped bins, and the forward pass on them,
    against the oracle's forward with the same bins zeroed (2-D workload layers
    and odd shapes, fp32 and bf16 spectra); the backward passes then run on the
    same zeroed spectra and are checked against the adjoint identity."""
    dev = torch.device("cuda:0")
    cases = [(synth.WORKLOADS[3].layers[0], 0, synth.layer_inputs(3, 0)),
             (synth.WORKLOADS[5].layers[0], 0, synth.layer_inputs(5, 0)),
             (synth.WORKLOADS[4].layers[2], blconv.BL_DESC_BF16_SPECTRA, synth.layer_inputs(4, 2))]
    layer = synth.Layer("fine_odd", 2, 3, 4, 5, 11, 9, 3, (1, 1, 1, 1), "blur")
    cases.append((layer, 0, synth.random_inputs(layer, 2600)))
    cut = 0
    for layer, fl, (x, w, dy) in cases:
        xt, wt, dyt = (torch.from_numpy(a).to(dev) for a in (x, w, dy))
        p0 = blconv.plan_for_layer(layer, 0.0)
        ws0 = p0.workspace(dev)
        e = p0.input_energy(xt, ws0).cpu().numpy()
        for fraction in (0.9, 0.99):
            t, c, kept_f, keep = p0.fine_band_for_energy(e, fraction)
            say(f"[fine] {layer.name} flags={fl} fraction={fraction}: t={t} c={c:.4f} kept {int(keep.sum())}/{keep.size}")
            cut += int(not keep.all())
            plan = blconv.plan_for_layer(layer, c, None, fl)
            assert plan.kept == keep.size
            ws = plan.workspace(dev)
            ws.fill_(0xFF)
            kt = torch.from_numpy(keep).to(dev)
            plan.zero_smallest(xt, ws, "X", 0)  # computes X only
            plan.zero_smallest(wt, ws, "W", 0)  # computes W only
            plan.zero_bins(ws, "X", kt)
            plan.zero_bins(ws, "W", kt)
            y = torch.full(plan.y_shape(), float("nan"), device=dev)
            dx = torch.full(plan.x_shape(), float("nan"), device=dev)
            dw = torch.full(plan.w_shape(), float("nan"), device=dev)
            R = blconv.BL_REUSE_X | blconv.BL_REUSE_W
            plan.forward(None, None, y, ws, flags=R)
            plan.backward_input(dyt, None, dx, ws, flags=blconv.BL_REUSE_W)
            plan.backward_weight(None, dyt, dw, ws, flags=blconv.BL_REUSE_X)
            torch.cuda.synchronize()
            drop = keep == 0
            zx = np.broadcast_to(drop[:, None, None], (keep.size, layer.N, layer.C_in))
            zw = np.broadcast_to(drop[:, None, None], (keep.size, layer.C_in, layer.C_out))
            want = bo.forward_zeroed(x, w, layer.pad, c, zx, zw)
            got = y.cpu().numpy()
            err = rel(got, want)
            # adjoint identity of the fine-band layer: <dy, y(x)> = <dx, x> = <dw, w>
            gx, gw = dx.cpu().numpy().astype(np.float64), dw.cpu().numpy().astype(np.float64)
            a0 = float(np.sum(dy.astype(np.float64) * got))
            a1, a2 = float(np.sum(gx * x)), float(np.sum(gw * w))
            say(f"    forward rel err {err:.2e}; adjoint {a0:.6e} {a1:.6e} {a2:.6e}")
            assert err <= (BF16_EXACT_TOL if fl else TOL), err
            tol = 1e-2 if fl else 1e-4
            assert abs(a1 - a0) <= tol * abs(a0) and abs(a2 - a0) <= tol * abs(a0)
    assert cut > 0


def test_graph_replays_match_eager(torch):
    """A layer's three passes captured in a HIP graph and replayed several times,
    with other eager library work, a poisoned workspace and outputs, and
    synchronisations between the replays: every replay's outputs are
    bit-identical to the eager calls' (1-D chirp-z, 2-D, thin and tiled
    contractions, bfloat16 spectra, the fused small-map forward)."""
    dev = torch.device("cuda:0")
    cases = [
        (synth.Layer("graph_1d", 1, 16, 24, 40, 300, 1, 5, (2, 2), "walk"), 0.5, 0),
        (synth.Layer("graph_2d", 2, 4, 16, 32, 16, 16, 3, (1, 1, 1, 1), "blur"), 0.25, 0),
        (synth.Layer("graph_thin", 1, 8, 1, 64, 200, 1, 8, (3, 4), "walk"), 0.0, 0),
        (synth.Layer("graph_bf16", 2, 16, 32, 48, 12, 12, 3, (1, 1, 1, 1), "blur"), 0.25, blconv.BL_DESC_BF16_SPECTRA),
        (synth.Layer("graph_fused", 2, 4, 8, 6, 8, 8, 3, (1, 1, 1, 1), "blur"), 0.0, blconv.BL_DESC_FUSED_FORWARD),
    ]
    other = synth.Layer("graph_other", 2, 2, 8, 8, 10, 10, 3, (1, 1, 1, 1), "blur")
    ox, ow, ody = synth.random_inputs(other, 5)
    for i, (layer, c, fl) in enumerate(cases):
        say(f"[graph] {layer.name} c={c} flags={fl}")
        x, w, dy = (torch.from_numpy(a).to(dev) for a in synth.random_inputs(layer, 1900 + i))
        plan = blconv.plan_for_layer(layer, c, None, fl)
        ws = plan.workspace(dev)
        y = torch.empty(plan.y_shape(), device=dev)
        dx = torch.empty(plan.x_shape(), device=dev)
        dw = torch.empty(plan.w_shape(), device=dev)
        dx2 = torch.empty(plan.x_shape(), device=dev)
        dw2 = torch.empty(plan.w_shape(), device=dev)

        def step():
            plan.forward(x, w, y, ws)
            plan.backward_input(dy, w, dx, ws, flags=blconv.BL_REUSE_W)
            plan.backward_weight(x, dy, dw, ws, flags=blconv.BL_REUSE_X | blconv.BL_REUSE_DY)
            plan.backward(dy, None, None, dx2, dw2, ws, flags=blconv.BL_REUSE_W | blconv.BL_REUSE_X)

        step()
        torch.cuda.synchronize()
        outs = (y, dx, dw, dx2, dw2)
        ref = tuple(t.clone() for t in outs)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        torch.cuda.synchronize()
        for r in range(3):
            for t in outs:
                t.fill_(float("nan"))
            ws.fill_(0xFF)
            g.replay()
            oy, odx, odw, _, _ = gpu_passes(torch, other, 0.5, ox, ow, ody, poison=False)
            torch.cuda.synchronize()
            for name, got, want in zip(("y", "dx", "dw", "dx (backward)", "dw (backward)"), outs, ref):
                assert torch.equal(got, want), (layer.name, r, name)


def _oracle_bin_energy(layer, x):
    if layer.ndim == 1:
        L = layer.H + layer.pad[0] + layer.pad[1]
        return bo.bin_energy_1d(x, layer.pad), bo.last_layer_kept(1, L)
    L = (layer.H + layer.pad[0] + layer.pad[1], layer.W + layer.pad[2] + layer.pad[3])
    return bo.bin_energy_2d(x, layer.pad), bo.last_layer_kept(2, L)


def test_input_energy_parity(torch):
    """Energy-based compression on the GPU: per-bin input energies (fp64 sums
    of the fp32 spectrum) against the oracle's, the band chosen from them
    against the oracle's band, for full-size workload layers (2-D grids 34 and
    58, the 1-D stack), random odd shapes, a plan that already compresses, and
    the energies of a spectrum stored by the forward pass (reuse flag)."""
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(2100)
    cases = [(synth.WORKLOADS[3].layers[0], 0.0, synth.layer_inputs(3, 0)[0]),
             (synth.WORKLOADS[5].layers[0], 0.0, synth.layer_inputs(5, 0)[0]),
             (synth.WORKLOADS[2].layers[1], 0.0, synth.layer_inputs(2, 1)[0]),
             (synth.WORKLOADS[4].layers[1], 0.5, synth.layer_inputs(4, 1)[0])]
    for i in range(6):
        layer = synth.random_layer(rng, 1 + i % 2)
        cases.append((layer, float(rng.choice([0.0, 0.0, 0.3])), synth.random_inputs(layer, 2200 + i)[0]))
    decided = 0
    for layer, c, x in cases:
        say(f"[energy] {layer} c={c}")
        plan = blconv.plan_for_layer(layer, c)
        ws = plan.workspace(dev)
        ws.fill_(0xFF)
        xt = torch.from_numpy(x).to(dev)
        e = plan.input_energy(xt, ws).cpu().numpy()
        E, last = _oracle_bin_energy(layer, x.astype(np.float64))
        u, v = plan.bins()
        want = E[v] if layer.ndim == 1 else E[u, v]
        err = rel(e, want)
        say(f"    rel err {err:.2e}")
        assert err <= 1e-5
        assert np.all(np.abs(e - want) <= 1e-4 * want + 1e-7 * want.sum() / want.size)
        # the band chosen from the GPU's energies is the oracle's
        own = want.sum()
        tb = last[v] if layer.ndim == 1 else last[u, v]
        for fraction in (0.5, 0.9, 0.99):
            f = np.array([want[tb >= t].sum() / own for t in range(int(tb.min()), int(tb.max()) + 1)])
            if np.min(np.abs(f - fraction)) < 1e-4:
                continue  # closer to a tie than the fp32 spectrum resolves
            expect = int(tb.min()) + max(k for k in range(len(f)) if f[k] >= fraction)
            t, cc, kept_f = plan.rate_for_energy(e, fraction)
            assert t == expect, (layer, fraction, t, expect)
            decided += 1
        # reuse: the spectrum the forward pass stored gives the same energies
        w = torch.from_numpy(synth.random_inputs(layer, 7)[1]).to(dev)
        y = torch.empty(plan.y_shape(), device=dev)
        plan.forward(xt, w, y, ws)
        e2 = plan.input_energy(None, ws, flags=blconv.BL_REUSE_X).cpu().numpy()
        assert np.array_equal(e, e2)
    assert decided >= 10
