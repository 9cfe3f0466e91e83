"""The forward pass that allocates nothing (bl_conv_forward_noalloc) against
bl_conv_forward, through the C ABI: two calls in a row, the second on a
smaller layer, each within the fp32 parity bar of the workspace path (and of
the fp64 oracle); a plan too large for the static array is refused."""
import numpy as np
import pytest

from oracle import bl_oracle as bo
from paper_1911_09287_amd import blconv, synth

pytestmark = pytest.mark.gpu

TOL = 1e-4


def err(a, b):
    a64, b64 = np.asarray(a, np.float64), np.asarray(b, np.float64)
    rel = np.linalg.norm(a64 - b64) / max(np.linalg.norm(b64), 1e-30)
    return max(float(rel), float(np.abs(a64 - b64).max() / max(np.abs(b64).max(), 1e-30)))


@pytest.fixture(scope="module")
def torch():
    import torch as _torch
    if not _torch.cuda.is_available():
        pytest.skip("no GPU")
    blconv.load()
    return _torch


def _both(torch, layer, c, x, w, desc_flags=0):
    dev = torch.device("cuda:0")
    plan = blconv.plan_for_layer(layer, c, None, desc_flags)
    xt, wt = torch.from_numpy(x).to(dev), torch.from_numpy(w).to(dev)
    y_ws = torch.full(plan.y_shape(), float("nan"), device=dev)
    y_na = torch.full(plan.y_shape(), float("nan"), device=dev)
    plan.forward(xt, wt, y_ws, plan.workspace(dev))
    plan.forward_noalloc(xt, wt, y_na)
    torch.cuda.synchronize()
    return y_ws.cpu().numpy(), y_na.cpu().numpy()


@pytest.mark.parametrize("first,second", [
    ((4, 1, 0.5), (1, 0, 0.0)),   # 2-D: DenseNet 128->32 @16x16, then the tiny 3->16 @32x32 layer
    ((3, 2, 0.5), (4, 2, 0.75)),  # 2-D: ResNet 256->256 @8x8, then DenseNet 128->32 @8x8
    ((2, 1, 0.75), (2, 0, 0.5)),  # 1-D: FCN 128->256 (direct DFT path), then 1->128
])
def test_noalloc_forward_matches_workspace_forward(torch, first, second):
    sizes = []
    for cfg, li, c in (first, second):
        layer = synth.WORKLOADS[cfg].layers[li]
        x, w, _ = synth.layer_inputs(cfg, li)
        print(f"[noalloc] config {cfg} layer {layer.name} c={c}", flush=True)
        y_ws, y_na = _both(torch, layer, c, x, w)
        ref = bo.forward(x, w, layer.pad, c)
        e_ws, e_orc = err(y_na, y_ws), err(y_na, ref)
        print(f"    vs workspace forward {e_ws:.2e}, vs oracle {e_orc:.2e}", flush=True)
        assert np.isfinite(y_na).all()
        assert e_ws <= TOL and e_orc <= TOL
        sizes.append(x.size)
    assert sizes[1] < sizes[0]


def test_noalloc_bf16_and_random_shapes(torch):
    """bfloat16 spectra (same rounding as the workspace path), and odd shapes
    through the direct DFT, twice in a row with shrinking sizes."""
    layer = synth.WORKLOADS[4].layers[1]
    x, w, _ = synth.layer_inputs(4, 1)
    y_ws, y_na = _both(torch, layer, 0.25, x, w, blconv.BL_DESC_BF16_SPECTRA)
    assert err(y_na, y_ws) <= TOL
    rng = np.random.default_rng(9)
    for i, hw in enumerate((19, 7)):
        L = synth.Layer("odd", 2, 3, 5, 6, hw, hw + 2, 3, (1, 0, 2, 1), "blur", 1.0)
        x, w, _ = synth.random_inputs(L, 3100 + i)
        c = float(rng.choice([0.0, 0.4]))
        y_ws, y_na = _both(torch, L, c, x, w)
        assert err(y_na, y_ws) <= TOL and err(y_na, bo.forward(x, w, L.pad, c)) <= TOL


def test_noalloc_refuses_plans_beyond_the_array(torch):
    """ResNet 64->64 @32x32 at c = 0 needs about 100 MB of spectra: refused on
    the host with BL_ERR_WORKSPACE_TOO_SMALL, y untouched."""
    layer = synth.WORKLOADS[3].layers[0]
    plan = blconv.plan_for_layer(layer, 0.0)
    dev = torch.device("cuda:0")
    x = torch.zeros(plan.x_shape(), device=dev)
    w = torch.zeros(plan.w_shape(), device=dev)
    y = torch.full(plan.y_shape(), 7.0, device=dev)
    with pytest.raises(blconv.BlError) as e:
        plan.forward_noalloc(x, w, y)
    assert e.value.code == 3
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())
