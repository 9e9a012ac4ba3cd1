"""GPU parity of the fully connected entry point (Sec. 3.1: the kh = kw = 1
case on [batch][m] inputs) against the oracle's convolution of the same
layer on [batch][m][1][1], in both layouts."""
import numpy as np
import pytest
import torch

import oracle
import paper_2105_14713_amd as onexn
import workloads
from gpu_helpers import rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    onexn.load_library()


def _fc(w, x, N, p, layout, out_dtype=None, **ep):
    """(GPU y as [B][n] fp64, oracle y as [B][n], packed layer)."""
    layer = onexn.prepare_layer(w.reshape(w.shape[0], w.shape[1], 1, 1), N, p, True)
    xd = x.cuda() if layout == "rows" else x.t().contiguous().cuda()
    ep = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in ep.items()}
    y = onexn.fc_fwd(layer.P, layer.I, layer.D, w.shape[0], xd, layout, out_dtype, **ep)
    torch.cuda.synchronize()
    y = y if layout == "rows" else y.t()
    pr = oracle.prune(w.double().numpy()[:, :, None, None], N, p, True)
    assert layer.t == pr.t
    ref = oracle.conv2d(x.double().numpy()[:, :, None, None], pr.wbar)[:, :, 0, 0]
    return y.double().cpu().numpy(), ref, layer


@pytest.mark.parametrize("layout", ["rows", "cols"])
@pytest.mark.parametrize("B", [1, 64, 256])
@pytest.mark.parametrize("N", [2, 4, 16, 32])
def test_fc_integer_exact(N, B, layout):
    print(f"fc N={N} B={B} {layout}", flush=True)
    gen = torch.Generator().manual_seed(N * 1000 + B)
    n, m = 100, 300                     # n = 100: a ragged last col-group for N = 16, 32
    w = torch.randint(-3, 4, (n, m), generator=gen).float()
    x = torch.randint(0, 4, (B, m), generator=gen).float()
    y, ref, _ = _fc(w, x, N, 0.5, layout)
    np.testing.assert_array_equal(y, ref)


@pytest.mark.parametrize("layout", ["rows", "cols"])
@pytest.mark.parametrize("N", [4, 32])
def test_fc_fp32_resnet50_classifier(N, layout):
    """The ResNet-50 classifier shape (2048 -> 1000) at batch 256, random fp32."""
    gen = torch.Generator().manual_seed(N)
    w = workloads.gen_weight(gen, 1000, 2048, 1).reshape(1000, 2048)
    x = workloads.gen_activation(gen, (256, 2048))
    y, ref, _ = _fc(w, x, N, 0.5, layout)
    assert rel_err(y, ref) <= 1e-5


@pytest.mark.parametrize("out_dtype", [torch.bfloat16, torch.float32], ids=["ybf16", "yf32"])
@pytest.mark.parametrize("layout", ["rows", "cols"])
def test_fc_bf16(layout, out_dtype):
    gen = torch.Generator().manual_seed(5)
    w = workloads.gen_weight(gen, 96, 512, 1).reshape(96, 512).bfloat16()
    x = workloads.gen_activation(gen, (64, 512)).bfloat16()
    y, ref, _ = _fc(w, x, 32, 0.7, layout, out_dtype)
    assert rel_err(y, ref) <= (2e-2 if out_dtype == torch.bfloat16 else 1e-5)


def test_fc_epilogue_and_batch_zero():
    gen = torch.Generator().manual_seed(6)
    w = torch.randint(-2, 3, (40, 64), generator=gen).float()
    x = torch.randint(0, 3, (9, 64), generator=gen).float()
    layer = onexn.prepare_layer(w.reshape(40, 64, 1, 1), 8, 0.5, True)
    bias = torch.randint(-5, 6, (40,), generator=gen).float()
    bp = bias[layer.perm.long()]
    y, ref, _ = _fc(w, x, 8, 0.5, "rows", bias=bp, act="relu")
    np.testing.assert_array_equal(y, np.maximum(ref + bp.double().numpy()[None, :], 0.0))
    empty = torch.zeros((0, 64), device="cuda")
    out = onexn.fc_fwd(layer.P, layer.I, layer.D, 40, empty, "rows")
    assert out.shape == (0, 40)
