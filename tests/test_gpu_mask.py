"""GPU mask building (onexn_build_mask_dev) against the host library's
onexn_build_mask and the oracle: perm, mask and t bit for bit on every
workload layer and on a fuzz of shapes, value kinds (ties everywhere, bf16)
and pruning rates."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2105_14713_amd as onexn
import workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    onexn.load_library()


def _check(w, N, p, rearrange, with_oracle=False):
    perm_d, mask_d, t_d = onexn.build_mask_dev(w.cuda(), N, p, rearrange)
    torch.cuda.synchronize()
    perm_h, mask_h, t_h = onexn.build_mask(w, N, p, rearrange)
    assert t_d == t_h
    np.testing.assert_array_equal(perm_d.cpu().numpy(), perm_h.numpy())
    np.testing.assert_array_equal(mask_d.cpu().numpy(), mask_h.numpy())
    if with_oracle:
        pr = oracle.prune(w.double().numpy(), N, p, rearrange)
        np.testing.assert_array_equal(perm_d.cpu().numpy(), pr.perm)
        np.testing.assert_array_equal(mask_d.cpu().numpy(), pr.T)
        assert t_d == pr.t


@pytest.mark.parametrize("wl", [workloads.config0(), workloads.config1(), workloads.config4()],
                         ids=lambda w: w.name)
def test_single_layer_workloads(wl):
    layer = wl.layers[0]
    w, _ = workloads.gen_layer(layer, 1, wl.dtype)
    _check(w, layer.N, layer.p, layer.rearrange, with_oracle=True)


def test_resnet50_layers_with_and_without_rearrangement():
    for layer in workloads.resnet50_convs():
        w, _ = workloads.gen_layer(layer, 1)
        _check(w, layer.N, layer.p, False)
        _check(w, layer.N, layer.p, True)


@pytest.mark.parametrize("N", [4, 8, 16, 32])
def test_mobilenet_v2_layers(N):
    for p in (0.3, 0.5, 0.7):
        for layer in workloads.mobilenet_v2_pointwise(N, p):
            w, _ = workloads.gen_layer(layer, 1)
            _check(w, N, p, True)


def test_fuzz():
    rng = np.random.default_rng(4321)
    for trial in range(160):
        n, m = int(rng.integers(1, 130)), int(rng.integers(1, 130))
        k = int(rng.choice([1, 3, 7]))
        N = int(rng.choice([1, 2, 4, 8, 16, 32]))
        p = float(rng.choice([0.0, 0.3, 0.5, 0.7, 0.99, 1.0]))
        kind = trial % 4
        if kind == 0:
            w = torch.from_numpy(rng.standard_normal((n, m, k, k)).astype(np.float32))
        elif kind == 1:      # integer-valued: many equal scores and norms
            w = torch.from_numpy(rng.integers(-2, 3, (n, m, k, k)).astype(np.float32))
        elif kind == 2:      # all equal: every score ties
            w = torch.full((n, m, k, k), 0.25)
        else:                # bf16 weights
            w = torch.from_numpy(rng.standard_normal((n, m, k, k)).astype(np.float32)).bfloat16()
        _check(w, N, p, bool(rng.integers(0, 2)), with_oracle=trial < 40)


def test_long_filters_and_many_blocks():
    """Filters longer than a wave's 64-element pass with a ragged tail, and more
    blocks than the selection workgroup has threads (several per thread)."""
    gen = torch.Generator().manual_seed(3)
    _check(torch.randn(96, 700, 3, 3, generator=gen), 32, 0.5, True)
    _check(torch.randn(2048, 2048, 1, 1, generator=gen).bfloat16(), 32, 0.7, False)
    _check(torch.randn(300, 4099, 1, 1, generator=gen), 1, 0.6, True)


def test_nan_weights_still_give_a_valid_mask():
    w = torch.randn(40, 16, 3, 3)
    w[3, 5, 1, 1] = float("nan")
    perm, mask, t = onexn.build_mask_dev(w.cuda(), 8, 0.5, True)
    torch.cuda.synchronize()
    assert sorted(perm.cpu().tolist()) == list(range(40))
    assert int(mask.sum()) == t


def test_workspace_errors():
    lib = onexn.load_library()
    w = torch.randn(32, 16, 3, 3, device="cuda")
    perm = torch.empty(32, dtype=torch.int32, device="cuda")
    mask = torch.empty(16 * 4, dtype=torch.uint8, device="cuda")
    need = onexn.mask_workspace_bytes(32, 16, 8)
    ws = torch.empty(need + 16, dtype=torch.uint8, device="cuda")
    t = ctypes.c_int64(-1)
    args = [w.data_ptr(), 0, 32, 16, 3, 3, 8, 0.5, 1, perm.data_ptr(), mask.data_ptr(),
            ctypes.addressof(t)]
    assert lib.onexn_build_mask_dev(*args, ws.data_ptr(), need - 8, None) == 6    # BUFSIZE
    assert lib.onexn_build_mask_dev(*args, ws.data_ptr() + 4, need, None) == 2    # ARG: alignment
    assert lib.onexn_build_mask_dev(*args, None, need, None) == 1                 # NULL
    assert t.value == -1
    assert lib.onexn_build_mask_dev(*args, ws.data_ptr(), need, None) == 0
    torch.cuda.synchronize()
    assert t.value == 16 * 4 // 2
