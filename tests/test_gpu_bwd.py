"""GPU parity of the backward kernels (input gradient through Omega-bar, and
the kept blocks' weight gradient in D's layout) against the oracle's
backward of Eq. 7 on the same inputs."""
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


def _bwd(w, x, dy, N, p, s, pd, dx_dtype=None):
    """(GPU dX, GPU dD, oracle dX, oracle dD) as fp64 numpy; w, x, dy on the host.
    Both outputs start as NaN, so an entry a kernel leaves unwritten fails."""
    n, m, k, _ = w.shape
    B, H, W = x.shape[0], x.shape[2], x.shape[3]
    layer = onexn.prepare_layer(w, N, p, True)
    dxo = torch.full((B, m, H, W), float("nan"), dtype=dx_dtype or dy.dtype, device="cuda")
    dDo = torch.full((layer.t, N, k, k), float("nan"), dtype=torch.float32, device="cuda")
    dx = onexn.conv2d_bwd_data(layer.P, layer.I, layer.D, n, m, dy.cuda(), (H, W), s, pd, dx_dtype, out=dxo)
    dD = onexn.conv2d_bwd_weight(layer.P, layer.I, n, N, (k, k), x.cuda(), dy.cuda(), s, pd, out=dDo)
    torch.cuda.synchronize()
    pr = oracle.prune(w.double().numpy(), N, p, True)
    assert layer.t == pr.t
    ref_dx = oracle.conv2d_bwd_data(dy.double().numpy(), pr.wbar, (H, W), (s, s), (pd, pd))
    dw = oracle.conv2d_bwd_weight(x.double().numpy(), dy.double().numpy(), pr.T, N, (k, k), (s, s),
                                  (pd, pd))
    _, _, ref_dD = oracle.pack(dw, pr.T, N)
    return dx.double().cpu().numpy(), dD.double().cpu().numpy(), ref_dx, ref_dD


CASES = [  # (n, m, k, stride, pad, B, H, W, N)
    (72, 13, 3, 1, 1, 2, 11, 9, 32),    # ragged last col-group
    (40, 9, 3, 2, 1, 2, 12, 11, 16),
    (18, 24, 1, 1, 0, 3, 7, 7, 4),
    (28, 17, 1, 2, 0, 2, 9, 10, 8),
    (9, 6, 7, 2, 3, 1, 15, 13, 2),
    (7, 20, 5, 3, 2, 2, 13, 12, 1),
    (64, 3, 7, 2, 3, 1, 20, 20, 32),    # stem-like
    # 1x1 stride 1 at N = 16 / 32: the matrix-core input gradient
    (80, 45, 1, 1, 0, 3, 7, 9, 32),     # ragged last col-group, pixels not a multiple of 32
    (40, 70, 1, 1, 0, 2, 10, 10, 16),   # three channel tiles, the last partial
    (96, 300, 1, 1, 0, 1, 9, 9, 32),    # col-groups of up to 300 blocks (narrowing rounds)
    (48, 1100, 1, 1, 0, 1, 5, 4, 16),   # col-groups longer than 1024 blocks
    (72, 40, 1, 1, 0, 3, 8, 6, 32),     # 48-pixel images: the weight gradient staged in pixel quads
    (40, 33, 1, 1, 0, 2, 4, 5, 16),
    # 1x1 strided at N = 16 / 32: the matrix-core kernel, zeros off the stride grid
    (80, 45, 1, 2, 0, 2, 9, 11, 32),    # odd map: the last block row/column clipped
    (40, 70, 1, 3, 0, 1, 10, 8, 16),
    # 3x3 at N = 16 / 32 (stride 1 and 2, padding 0-2): the matrix-core tap kernel
    (64, 100, 3, 1, 1, 1, 8, 8, 32),    # four channel tiles, the last partial
    (48, 40, 3, 1, 0, 2, 9, 10, 32),
    (36, 33, 3, 2, 2, 1, 11, 12, 16),   # ragged last col-group
    (300, 40, 3, 2, 1, 1, 9, 9, 32),    # ten col-groups, the last ragged
    (32, 20, 3, 1, 2, 3, 5, 4, 16),     # padding wider than the map's margin
    # 3x3 at N = 8: the matrix-core input gradient (stride 1, and stride 2 by parity class)
    (48, 40, 3, 1, 1, 2, 9, 10, 8),
    (36, 33, 3, 2, 1, 1, 11, 12, 8),
    # at most four input channels: the one-lane-per-pixel input gradient
    (20, 4, 3, 1, 1, 2, 9, 7, 4),
    (33, 1, 5, 3, 2, 1, 11, 13, 8),     # stride 3, output channels not a multiple of 8
    (64, 2, 1, 2, 0, 2, 9, 9, 16),
    (16, 3, 7, 2, 3, 1, 9, 150, 16),    # stem-like, two 64-column chunks per residue class
]


@pytest.mark.parametrize("p", [0.0, 0.5, 0.9])
@pytest.mark.parametrize("case", CASES, ids=lambda c: "n%d_m%d_k%d_s%d_p%d_N%d" % (c[:5] + (c[8],)))
def test_bwd_integer_exact(case, p):
    n, m, k, s, pd, B, H, W, N = case
    print(f"bwd {case} p={p}", flush=True)
    w, x = workloads.gen_integer_layer(seed=n + m + k, cout=n, cin=m, k=k, batch=B, H=H, W=W,
                                       wmax=2, xmax=2)
    Ho, Wo = (H + 2 * pd - k) // s + 1, (W + 2 * pd - k) // s + 1
    gen = torch.Generator().manual_seed(n * k)
    dy = torch.randint(-2, 3, (B, n, Ho, Wo), generator=gen).float()
    dx, dD, ref_dx, ref_dD = _bwd(w, x, dy, N, p, s, pd)
    np.testing.assert_array_equal(dx, ref_dx)
    np.testing.assert_array_equal(dD, ref_dD)


@pytest.mark.parametrize("case", CASES[:4], ids=lambda c: "n%d_m%d_k%d" % c[:3])
def test_bwd_fp32_random(case):
    n, m, k, s, pd, B, H, W, N = case
    gen = torch.Generator().manual_seed(5 * n + m)
    w = workloads.gen_weight(gen, n, m, k)
    x = workloads.gen_activation(gen, (B, m, H, W))
    Ho, Wo = (H + 2 * pd - k) // s + 1, (W + 2 * pd - k) // s + 1
    dy = torch.randn((B, n, Ho, Wo), generator=gen)
    dx, dD, ref_dx, ref_dD = _bwd(w, x, dy, N, 0.5, s, pd)
    assert rel_err(dx, ref_dx) <= 1e-5
    assert rel_err(dD, ref_dD) <= 1e-5


@pytest.mark.parametrize("dx_dtype", [torch.float32, torch.bfloat16], ids=["dxf32", "dxbf16"])
def test_bwd_bf16(dx_dtype):
    """bf16 weights, activations and output gradient; fp32 accumulation.  The
    oracle sees the same bf16 values; the bf16 dX has one final rounding."""
    gen = torch.Generator().manual_seed(17)
    w = workloads.gen_weight(gen, 64, 40, 3).bfloat16()
    x = workloads.gen_activation(gen, (2, 40, 10, 10)).bfloat16()
    dy = torch.randn((2, 64, 10, 10), generator=gen).bfloat16()
    dx, dD, ref_dx, ref_dD = _bwd(w, x, dy, 32, 0.5, 1, 1, dx_dtype)
    assert rel_err(dx, ref_dx) <= (2e-2 if dx_dtype == torch.bfloat16 else 1e-5)
    assert rel_err(dD, ref_dD) <= 1e-5


def test_bwd_resnet50_layer_shape_and_reproducibility():
    """A ResNet-50 3x3 layer (256 -> 256 at 14x14, N = 32, p = 0.5) at batch 4:
    fp32 random within 1e-5 of the oracle, and two runs bit-identical."""
    layer = [l for l in workloads.resnet50_convs() if l.name == "s3b2_3x3"][0]
    w, x = workloads.gen_layer(layer, 4)
    gen = torch.Generator().manual_seed(99)
    dy = torch.randn((4, 256, 14, 14), generator=gen)
    dx, dD, ref_dx, ref_dD = _bwd(w, x, dy, 32, 0.5, 1, 1)
    assert rel_err(dx, ref_dx) <= 1e-5
    assert rel_err(dD, ref_dD) <= 1e-5
    dx2, dD2, _, _ = _bwd(w, x, dy, 32, 0.5, 1, 1)
    np.testing.assert_array_equal(dx, dx2)
    np.testing.assert_array_equal(dD, dD2)


@pytest.mark.parametrize("name", ["s2b1_3x3", "s2b1_down", "s3b2_1x1a", "s1b1_1x1b"])
def test_bwd_resnet50_full_batch(name):
    """ResNet-50 layers at the backward benchmark's size and launch
    configuration (batch 64, fp32, N = 32, p = 0.5): the stride-2 3x3 input
    gradient's parity-class launches and the pair-tiled weight gradient; the
    strided 1x1 input gradient with its zeroed positions; the 1x1 input
    gradient with 1024 input channels; the 64 -> 256 layer's quad-staged
    weight gradient.  Every dX and dD entry against the oracle, within 1e-5
    of the largest."""
    layer = [l for l in workloads.resnet50_convs() if l.name == name][0]
    print(f"bwd full batch {name}", flush=True)
    w, x = workloads.gen_layer(layer, 64)
    gen = torch.Generator().manual_seed(layer.seed + 7)
    dy = torch.randn((64, layer.cout, layer.Ho, layer.Ho), generator=gen)
    dx, dD, ref_dx, ref_dD = _bwd(w, x, dy, layer.N, layer.p, layer.stride, layer.pad)
    assert rel_err(dx, ref_dx) <= 1e-5
    assert rel_err(dD, ref_dD) <= 1e-5


@pytest.mark.parametrize("kernel", ["matrix", "matrix_split3", "no_quads", "no_quads_split3", "general"])
@pytest.mark.parametrize("N", [16, 32])
def test_bwd_1x1_kernels_agree_with_oracle(kernel, N, tune):
    """The 1x1 gradients through the matrix-core kernels (the weight gradient
    with one pixel range per tile, and with three whose sums are added; staged
    in pixel quads where the 132-pixel images allow, and one pixel per access
    with bwd_kernel = 3) and through the general ones (bwd_kernel = 1): fp32
    random, 300 -> 256, and integer data exactly."""
    if kernel == "general":
        tune("bwd_kernel", 1)
    if kernel.startswith("no_quads"):
        tune("bwd_kernel", 3)
    if kernel.endswith("split3"):
        tune("bwd_split", 3)
    gen = torch.Generator().manual_seed(23 + N)
    w = workloads.gen_weight(gen, 256, 300, 1)
    x = workloads.gen_activation(gen, (2, 300, 12, 11))
    dy = torch.randn((2, 256, 12, 11), generator=gen)
    dx, dD, ref_dx, ref_dD = _bwd(w, x, dy, N, 0.5, 1, 0)
    assert rel_err(dx, ref_dx) <= 1e-5
    assert rel_err(dD, ref_dD) <= 1e-5
    wi, xi = workloads.gen_integer_layer(seed=N, cout=72, cin=50, k=1, batch=3, H=9, W=12, wmax=2, xmax=2)
    dyi = torch.randint(-2, 3, (3, 72, 9, 12), generator=gen).float()
    dx, dD, ref_dx, ref_dD = _bwd(wi, xi, dyi, N, 0.5, 1, 0)
    np.testing.assert_array_equal(dx, ref_dx)
    np.testing.assert_array_equal(dD, ref_dD)


@pytest.mark.parametrize("kernel", ["matrix", "matrix_split3", "general", "nine_taps"])
@pytest.mark.parametrize("geom", [(3, 1, 1), (3, 2, 1), (3, 2, 0), (7, 2, 3)], ids=["3x3s1", "3x3s2", "3x3s2p0", "7x7s2"])
@pytest.mark.parametrize("N", [8, 16, 32])
def test_bwd_kxk_kernels_agree_with_oracle(kernel, geom, N, tune):
    """The k x k gradients through the matrix-core kernels (weight gradient
    over (block, tap) pair tiles with one pixel range per tile and with three;
    stride-2 3x3 input gradient by parity class, and with all nine taps per
    pixel: bwd_kernel = 2) and through the general ones: fp32 random 72 -> 40
    at 13x11 within 1e-5, and integer data exactly."""
    k, s, pd = geom
    if kernel == "general":
        tune("bwd_kernel", 1)
    if kernel == "nine_taps":
        tune("bwd_kernel", 2)
    if kernel == "matrix_split3":
        tune("bwd_split", 3)
    gen = torch.Generator().manual_seed(31 + N + k)
    H, W = 13, 11
    Ho, Wo = (H + 2 * pd - k) // s + 1, (W + 2 * pd - k) // s + 1
    w = workloads.gen_weight(gen, 72, 40, k)
    x = workloads.gen_activation(gen, (2, 40, H, W))
    dy = torch.randn((2, 72, Ho, Wo), generator=gen)
    dx, dD, ref_dx, ref_dD = _bwd(w, x, dy, N, 0.5, s, pd)
    assert rel_err(dx, ref_dx) <= 1e-5
    assert rel_err(dD, ref_dD) <= 1e-5
    wi, xi = workloads.gen_integer_layer(seed=N + k, cout=48, cin=21, k=k, batch=2, H=H, W=W,
                                         wmax=2, xmax=2)
    dyi = torch.randint(-2, 3, (2, 48, Ho, Wo), generator=gen).float()
    dx, dD, ref_dx, ref_dD = _bwd(wi, xi, dyi, N, 0.5, s, pd)
    np.testing.assert_array_equal(dx, ref_dx)
    np.testing.assert_array_equal(dD, ref_dD)


@pytest.mark.parametrize("split", ["default", "3"])
@pytest.mark.parametrize("hw", [(8, 8), (7, 5)], ids=["quads", "no_quads"])
@pytest.mark.parametrize("N", [2, 4, 8])
def test_bwd_1x1_small_n(N, hw, split, tune):
    """1x1 layers at N = 2 / 4 / 8 on the matrix cores: the input gradient with
    256/N col-groups per stage, the weight gradient as the dense product of
    32-channel tiles stored at the kept blocks (staged in pixel quads where
    the images allow, one pixel per access otherwise; one pixel range per
    tile and three added with atomics).  fp32 random 70 -> 100 (three channel
    tiles, ragged col-group tiles) within 1e-5, and integer data exactly."""
    if split != "default":
        tune("bwd_split", int(split))
    H, W = hw
    gen = torch.Generator().manual_seed(41 + N + H)
    w = workloads.gen_weight(gen, 100, 70, 1)
    x = workloads.gen_activation(gen, (2, 70, H, W))
    dy = torch.randn((2, 100, H, W), generator=gen)
    dx, dD, ref_dx, ref_dD = _bwd(w, x, dy, N, 0.5, 1, 0)
    assert rel_err(dx, ref_dx) <= 1e-5
    assert rel_err(dD, ref_dD) <= 1e-5
    wi, xi = workloads.gen_integer_layer(seed=N + W, cout=66, cin=40, k=1, batch=3, H=H, W=W, wmax=2, xmax=2)
    dyi = torch.randint(-2, 3, (3, 66, H, W), generator=gen).float()
    dx, dD, ref_dx, ref_dD = _bwd(wi, xi, dyi, N, 0.5, 1, 0)
    np.testing.assert_array_equal(dx, ref_dx)
    np.testing.assert_array_equal(dD, ref_dD)


def _fuzz_cases(count, seed):
    """Seeded random small layers spanning the backward dispatch: N, kernel
    size, stride, padding, channel counts (ragged col-groups and channel
    tiles), map sizes (pixel quads or not), batch and p."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < count:
        N = int(rng.choice([1, 2, 4, 8, 16, 32]))
        k = int(rng.choice([1, 1, 3, 3, 5, 7]))
        s = int(rng.choice([1, 1, 2, 3]))
        pd = int(rng.integers(0, (k + 1) // 2 + 1))
        H, W = int(rng.integers(k, 15)), int(rng.integers(k, 15))
        if (H + 2 * pd - k) // s + 1 < 1 or (W + 2 * pd - k) // s + 1 < 1:
            continue
        n = int(rng.integers(1, 3 * N + 40))
        m = int(rng.integers(1, 90))
        B = int(rng.integers(1, 4))
        p = float(rng.choice([0.0, 0.5, 0.9]))
        cases.append((n, m, k, s, pd, B, H, W, N, p))
    return cases


@pytest.mark.parametrize("case", _fuzz_cases(200, 2024),
                         ids=lambda c: "n%d_m%d_k%d_s%d_p%d_B%d_%dx%d_N%d_p%g" % c)
def test_bwd_fuzz_integer_exact(case):
    """Both gradients integer-exact against the oracle on 200 seeded random
    small layers (outputs pre-filled with NaN)."""
    n, m, k, s, pd, B, H, W, N, p = case
    print(f"bwd fuzz {case}", flush=True)
    w, x = workloads.gen_integer_layer(seed=n * 7 + m + k, cout=n, cin=m, k=k, batch=B, H=H, W=W,
                                       wmax=2, xmax=2)
    Ho, Wo = (H + 2 * pd - k) // s + 1, (W + 2 * pd - k) // s + 1
    gen = torch.Generator().manual_seed(n + 13 * m)
    dy = torch.randint(-2, 3, (B, n, Ho, Wo), generator=gen).float()
    dx, dD, ref_dx, ref_dD = _bwd(w, x, dy, N, p, s, pd)
    np.testing.assert_array_equal(dx, ref_dx)
    np.testing.assert_array_equal(dD, ref_dD)


@pytest.mark.parametrize("k,N", [(3, 16), (1, 32)])
def test_bwd_everything_pruned(k, N):
    w, x = workloads.gen_integer_layer(seed=1, cout=32, cin=5, k=k, batch=1, H=6)
    layer = onexn.prepare_layer(w, N, 1.0, False)
    dy = torch.ones((1, 32, 6, 6), device="cuda")
    dx = onexn.conv2d_bwd_data(layer.P, layer.I, layer.D, 32, 5, dy, (6, 6), 1, k // 2)
    dD = onexn.conv2d_bwd_weight(layer.P, layer.I, 32, N, (k, k), x.cuda(), dy, 1, k // 2)
    torch.cuda.synchronize()
    assert layer.t == 0 and dD.numel() == 0
    assert torch.all(dx == 0)
