"""GPU parity: the HIP path (through the C ABI) against the oracle.

Bars: integer-valued inputs are bit-exact in fp32; fp32 inputs within
max|y - ref| / max|ref| <= 1e-5; bf16 inputs (fp32 accumulation) within 2e-2
for bf16 output (and 1e-5 for fp32 output, where only accumulation rounds),
the oracle seeing the same bf16-rounded values.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2105_14713_amd as onexn
import workloads
from gpu_helpers import gpu_conv, oracle_conv, rel_err, sample_indices

pytestmark = pytest.mark.gpu

SHAPES = [  # (k, stride, pad)
    (1, 1, 0), (1, 2, 0), (3, 1, 1), (3, 2, 1), (7, 2, 3), (3, 1, 0),
]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib = onexn.load_library()
    assert os.path.samefile(lib._name, onexn.LIB_PATH)


def _n_for(N):
    # several col-groups with a ragged last one (none for N = 1)
    return {1: 7, 2: 9, 4: 18, 8: 28, 16: 40, 32: 72}[N]


@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
@pytest.mark.parametrize("kshape", SHAPES, ids=lambda s: f"k{s[0]}s{s[1]}p{s[2]}")
@pytest.mark.parametrize("N", [1, 2, 4, 8, 16, 32])
def test_integer_exact(N, kshape, layout):
    k, s, pd = kshape
    n = _n_for(N)
    print(f"case N={N} k={k} s={s} pad={pd} layout={layout}", flush=True)
    w, x = workloads.gen_integer_layer(seed=10 * N + k, cout=n, cin=13, k=k, batch=3, H=19, W=17)
    y, layer = gpu_conv(w, x, N, 0.5, True, s, pd, layout)
    ref, pr = oracle_conv(w, x, N, 0.5, True, s, pd)
    assert layer.t == pr.t
    np.testing.assert_array_equal(y, ref)


@pytest.mark.parametrize("kshape", SHAPES, ids=lambda s: f"k{s[0]}s{s[1]}p{s[2]}")
@pytest.mark.parametrize("N", [4, 8, 16, 32])
def test_float_fp32(N, kshape):
    k, s, pd = kshape
    gen = torch.Generator().manual_seed(N * 100 + k)
    n, m = _n_for(N), 37
    w = workloads.gen_weight(gen, n, m, k)
    x = workloads.gen_activation(gen, (2, m, 23, 21))
    y, _ = gpu_conv(w, x, N, 0.3, False, s, pd)
    ref, _ = oracle_conv(w, x, N, 0.3, False, s, pd)
    assert rel_err(y, ref) <= 1e-5


@pytest.mark.parametrize("out_dtype", [torch.bfloat16, torch.float32], ids=["ybf16", "yf32"])
@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
@pytest.mark.parametrize("kshape", [(1, 1, 0), (3, 1, 1), (3, 2, 1)], ids=lambda s: f"k{s[0]}s{s[1]}")
@pytest.mark.parametrize("N", [4, 8, 16, 32])
def test_bf16(N, kshape, layout, out_dtype):
    k, s, pd = kshape
    gen = torch.Generator().manual_seed(N + k)
    n, m = _n_for(N), 45
    w = workloads.gen_weight(gen, n, m, k).bfloat16()
    x = workloads.gen_activation(gen, (2, m, 20, 19)).bfloat16()
    y, _ = gpu_conv(w, x, N, 0.7, True, s, pd, layout, out_dtype)
    ref, _ = oracle_conv(w, x, N, 0.7, True, s, pd)
    err = rel_err(y, ref)
    if out_dtype == torch.bfloat16:
        assert err <= 2e-2
        assert err <= 2.0 ** -8          # one bf16 rounding of the output
    else:
        assert err <= 1e-5


def test_fma_split_contraction_bf16_nhwc():
    """The N <= 8 generic kernel with its contraction split over waves, on bf16
    NHWC input (small integers: exact in bf16 and in fp32 accumulation)."""
    w, x = workloads.gen_integer_layer(seed=77, cout=18, cin=64, k=3, batch=1, H=12, wmax=2, xmax=2)
    y, _ = gpu_conv(w.bfloat16(), x.bfloat16(), 4, 0.5, True, 1, 1, "nhwc", torch.float32)
    ref, _ = oracle_conv(w, x, 4, 0.5, True, 1, 1)
    np.testing.assert_array_equal(y, ref)


def test_bf16_integer_exact():
    """Small integers are exact in bf16, so bf16 -> fp32 output must be bit-exact."""
    for N in (8, 16, 32):
        w, x = workloads.gen_integer_layer(seed=N, cout=_n_for(N), cin=40, k=3, batch=2, H=14)
        y, _ = gpu_conv(w.bfloat16(), x.bfloat16(), N, 0.5, False, 1, 1, "nchw", torch.float32)
        ref, _ = oracle_conv(w, x, N, 0.5, False, 1, 1)
        np.testing.assert_array_equal(y, ref)


# ---------------------------------------------------------------------------
# Edge cases.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("N", [4, 16, 32])
def test_all_pruned_writes_zeros(N):
    w, x = workloads.gen_integer_layer(seed=1, cout=40, cin=9, k=3, batch=2, H=10)
    y, layer = gpu_conv(w, x, N, 1.0, True, 1, 1)      # output prefilled with NaN
    assert layer.t == 0
    assert np.all(y == 0.0)


@pytest.mark.parametrize("N", [4, 8, 16, 32])
def test_dense_p0_equals_library_conv(N):
    gen = torch.Generator().manual_seed(3)
    w = workloads.gen_weight(gen, 64, 24, 3)
    x = workloads.gen_activation(gen, (2, 24, 15, 15))
    y, layer = gpu_conv(w, x, N, 0.0, False, 1, 1)
    ref = torch.nn.functional.conv2d(x.double(), w.double(), padding=1).numpy()
    assert layer.t == 24 * (64 // N)
    assert rel_err(y, ref) <= 1e-5


def test_batch_zero_is_noop():
    w, _ = workloads.gen_integer_layer(seed=2, cout=32, cin=8, k=1, batch=1, H=4)
    layer = onexn.prepare_layer(w, 16, 0.5, False)
    x = torch.zeros((0, 8, 4, 4), device="cuda")
    y = layer.forward(x)
    assert y.shape == (0, 32, 4, 4)


@pytest.mark.parametrize("case", [
    dict(n=32, m=5, k=1, N=32, B=1, H=1, s=1, pd=0),     # one col-group, one pixel
    dict(n=16, m=3, k=1, N=16, B=1, H=3, s=2, pd=0),     # stride larger than the kernel
    dict(n=8, m=2, k=3, N=4, B=1, H=2, s=1, pd=2),       # padding larger than the input
    dict(n=33, m=600, k=3, N=32, B=1, H=6, s=1, pd=1),   # long contraction, 1-row last group
    dict(n=100, m=17, k=1, N=4, B=5, H=13, s=1, pd=0),   # many groups, ragged pixel tail
    dict(n=48, m=7, k=5, N=16, B=2, H=9, s=3, pd=2),     # 5x5, stride 3
    dict(n=8, m=3, k=16, N=8, B=1, H=20, s=8, pd=15),    # largest kernel, stride and pad
    dict(n=20, m=2, k=16, N=16, B=2, H=17, s=8, pd=15),  # the same on the MFMA kernel
    dict(n=18, m=64, k=3, N=4, B=1, H=12, s=1, pd=1),    # few pixels, long col-groups: split contraction
    dict(n=20, m=40, k=3, N=8, B=1, H=9, s=2, pd=1),     # the same at N = 8, stride 2
    dict(n=7, m=70, k=3, N=1, B=1, H=6, s=1, pd=0),      # and at N = 1
])
def test_edge_shapes_integer_exact(case):
    c = case
    print(f"edge case {c}", flush=True)
    w, x = workloads.gen_integer_layer(seed=c["n"] + c["m"], cout=c["n"], cin=c["m"], k=c["k"],
                                       batch=c["B"], H=c["H"], wmax=2, xmax=2)
    y, _ = gpu_conv(w, x, c["N"], 0.5, True, c["s"], c["pd"])
    ref, _ = oracle_conv(w, x, c["N"], 0.5, True, c["s"], c["pd"])
    np.testing.assert_array_equal(y, ref)


@pytest.mark.parametrize("k,N,dt", [(1, 16, "f32"), (1, 32, "f32"), (3, 16, "f32"), (1, 4, "f32"),
                                    (3, 4, "f32"), (1, 32, "bf16"), (1, 32, "bf16s"), (1, 32, "nhwc"),
                                    (1, 16, "nhwc_long")])
def test_out_of_range_channels_are_skipped(k, N, dt, tune):
    """Entries of I outside [0, m) contribute nothing (kept ascending, so the
    rest of the col-group is unaffected); P is clamped to [0, t]."""
    print(f"skip case k={k} N={N} {dt}", flush=True)
    H = 10 if dt.startswith("bf16") else 9   # bf16 1x1 N=32 with H*W % 4 == 0: the bf16 pointwise kernels
    tune("pwb_kernel", 2 if dt == "bf16s" else 1)
    # (nhwc_long: col-groups longer than the NHWC kernel keeps in registers)
    w, x = workloads.gen_integer_layer(seed=4, cout=4 * N, cin=300 if dt == "nhwc_long" else 70, k=k,
                                       batch=2, H=H)
    if dt.startswith("bf16"):
        w, x = w.bfloat16(), x.bfloat16()
    nhwc = dt.startswith("nhwc")
    xin = (x.permute(0, 2, 3, 1).contiguous() if nhwc else x).cuda()
    lay = "nhwc" if nhwc else "nchw"
    back = (lambda t: t.permute(0, 3, 1, 2)) if nhwc else (lambda t: t)
    layer = onexn.prepare_layer(w, N, 0.5, False)
    P, I, D = layer.P.cpu(), layer.I.cpu().clone(), layer.D.cpu().clone()
    hi, lo = int(P[1]) - 1, int(P[1])          # last entry of group 0, first of group 1
    I[hi], I[lo] = 1 << 20, -5
    y = back(onexn.conv2d_fwd(layer.P, I.cuda(), layer.D, 4 * N, xin, 1, k // 2, lay,
                              out_dtype=torch.float32))
    # Expected: the same arrays with those two entries' weights zeroed.
    D0 = D.clone()
    D0[hi] = 0
    D0[lo] = 0
    I0 = I.clone()
    I0[hi], I0[lo] = 0, 0
    ref = oracle.decode(x.double().numpy(), P.numpy(), I0.numpy(), D0.double().numpy(), 4 * N,
                        (1, 1), (k // 2, k // 2))
    np.testing.assert_array_equal(y.double().cpu().numpy(), ref)
    Pbad = layer.P.clone()
    Pbad[-1] = 1 << 30
    y2 = onexn.conv2d_fwd(Pbad, layer.I, layer.D, 4 * N, xin, 1, k // 2, lay)
    torch.cuda.synchronize()
    assert torch.isfinite(y2).all()


def test_runs_on_a_side_stream():
    w, x = workloads.gen_integer_layer(seed=5, cout=32, cin=6, k=3, batch=2, H=8)
    layer = onexn.prepare_layer(w, 16, 0.5, False)
    s = torch.cuda.Stream()
    xd = x.cuda()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        y = layer.forward(xd, 1, 1)
    s.synchronize()
    ref, _ = oracle_conv(w, x, 16, 0.5, False, 1, 1)
    np.testing.assert_array_equal(y.double().cpu().numpy(), ref)


# ---------------------------------------------------------------------------
# The benchmark workloads at full size (same entry point and launch
# configuration as the benchmark), checked on sampled outputs.
# ---------------------------------------------------------------------------

def _check_sampled(layer, batch, dtype, out_dtype, y, pr, x_cpu, count=10000, seed=0):
    idx = sample_indices(tuple(y.shape), count, seed, layer.N)
    got = y.float().reshape(-1)[torch.from_numpy(idx).cuda()].double().cpu().numpy()
    ref = oracle.conv2d_at(x_cpu.double().numpy(), pr.wbar, idx, (layer.stride,) * 2,
                           (layer.pad,) * 2)
    err = rel_err(got, ref)
    bar = 2e-2 if out_dtype == "bf16" else 1e-5
    assert err <= bar, f"{layer.name}: rel err {err:.3g} > {bar}"
    return err


def _run_layer(layer, batch, dtype="f32", out_dtype="f32"):
    w, x = workloads.gen_layer(layer, batch, dtype)
    packed = onexn.prepare_layer(w, layer.N, layer.p, layer.rearrange)
    odt = torch.bfloat16 if out_dtype == "bf16" else torch.float32
    y = packed.forward(x.cuda(), layer.stride, layer.pad, "nchw", odt)
    torch.cuda.synchronize()
    pr = oracle.prune(w.double().numpy(), layer.N, layer.p, layer.rearrange)
    assert packed.t == pr.t
    return y, pr, x


def test_config0_full():
    wl = workloads.config0()
    layer = wl.layers[0]
    y, pr, x = _run_layer(layer, wl.batch)
    ref = oracle.conv2d(x.double().numpy(), pr.wbar, (1, 1), (1, 1))
    assert rel_err(y.double().cpu().numpy(), ref) <= 1e-5


def test_config1_full_size_sampled():
    wl = workloads.config1()
    y, pr, x = _run_layer(wl.layers[0], wl.batch)
    _check_sampled(wl.layers[0], wl.batch, "f32", "f32", y, pr, x)


@pytest.mark.parametrize("kernel", ["gathered", "staged"])
@pytest.mark.parametrize("out_dtype", ["bf16", "f32"])
def test_config4_full_size_sampled(out_dtype, kernel, tune):
    tune("pwb_kernel", 1 if kernel == "gathered" else 2)
    wl = workloads.config4(out_dtype)
    y, pr, x = _run_layer(wl.layers[0], wl.batch, "bf16", out_dtype)
    _check_sampled(wl.layers[0], wl.batch, "bf16", out_dtype, y, pr, x)


_R50 = workloads.resnet50_convs()


@pytest.mark.parametrize("li", range(len(_R50)), ids=[l.name for l in _R50])
def test_config2_resnet50_layer_sampled(li):
    layer = _R50[li]
    print(f"resnet50 layer {layer.name}", flush=True)
    y, pr, x = _run_layer(layer, 64)
    _check_sampled(layer, 64, "f32", "f32", y, pr, x, seed=li)


_MB = workloads.mobilenet_v2_pointwise(4, 0.5)


@pytest.mark.parametrize("li", range(len(_MB)), ids=[l.name for l in _MB])
def test_config3_mobilenet_v2_layer_sampled(li):
    """All twelve (N, p) sub-configurations on one layer's input (the input
    depends only on the layer, not on N or p)."""
    base = _MB[li]
    print(f"mobilenet-v2 layer {base.name}", flush=True)
    w, x = workloads.gen_layer(base, 128)
    xd = x.cuda()
    x64 = x.double().numpy()
    for N in (4, 8, 16, 32):
        for p in (0.3, 0.5, 0.7):
            packed = onexn.prepare_layer(w, N, p, False)
            y = packed.forward(xd)
            torch.cuda.synchronize()
            pr = oracle.prune(w.double().numpy(), N, p, False)
            assert packed.t == pr.t
            idx = sample_indices(tuple(y.shape), 10000, li * 31 + N, N)
            got = y.reshape(-1)[torch.from_numpy(idx).cuda()].double().cpu().numpy()
            ref = oracle.conv2d_at(x64, pr.wbar, idx)
            assert rel_err(got, ref) <= 1e-5, (base.name, N, p)


@pytest.mark.parametrize("li", range(len(_MB)), ids=[l.name for l in _MB])
def test_config3_mobilenet_v2_layer_sampled_nhwc(li):
    """The MobileNet-V2 layers with NHWC activations at full size (batch 128),
    N = 16 and 32 at p = 0.5: the NHWC 1x1 kernel in the launch configuration
    the benchmark times, on >= 10^4 sampled outputs (one in every (block,
    col-group) cell among them)."""
    base = _MB[li]
    print(f"mobilenet-v2 nhwc layer {base.name}", flush=True)
    w, x = workloads.gen_layer(base, 128)
    xh = x.permute(0, 2, 3, 1).contiguous().cuda()
    x64 = x.double().numpy()
    for N in (16, 32):
        packed = onexn.prepare_layer(w, N, 0.5, False)
        y = packed.forward(xh, 1, 0, "nhwc").permute(0, 3, 1, 2).contiguous()
        torch.cuda.synchronize()
        pr = oracle.prune(w.double().numpy(), N, 0.5, False)
        assert packed.t == pr.t
        idx = sample_indices(tuple(y.shape), 10000, li * 37 + N, N)
        got = y.reshape(-1)[torch.from_numpy(idx).cuda()].double().cpu().numpy()
        ref = oracle.conv2d_at(x64, pr.wbar, idx)
        assert rel_err(got, ref) <= 1e-5, (base.name, N)


def test_config1_full_size_sampled_nhwc():
    wl = workloads.config1()
    layer = wl.layers[0]
    w, x = workloads.gen_layer(layer, wl.batch)
    packed = onexn.prepare_layer(w, layer.N, layer.p, layer.rearrange)
    y = packed.forward(x.permute(0, 2, 3, 1).contiguous().cuda(), 1, 0, "nhwc").permute(0, 3, 1, 2).contiguous()
    torch.cuda.synchronize()
    pr = oracle.prune(w.double().numpy(), layer.N, layer.p, layer.rearrange)
    _check_sampled(layer, wl.batch, "f32", "f32", y, pr, x)


@pytest.mark.parametrize("wgs", ["1", "5", "default"])
@pytest.mark.parametrize("hw", [(12, 12), (7, 7)], ids=["hw%4=0", "hw%4!=0"])
@pytest.mark.parametrize("N,groups,m", [
    (16, 10, 200),   # 64-pixel slices
    (16, 10, 400),   # 32-pixel slices
    (16, 10, 900),   # 16-pixel slices
    (16, 2, 200),    # 16-pixel slices, 4 slices per tile
    (32, 10, 200),   # 64-pixel slices
    (32, 10, 400),   # 32-pixel slices
    (32, 8, 120),    # 64-pixel slices, exactly 8 units per tile
    (32, 4, 120),    # 64-pixel slices, 2 slices per tile
], ids=lambda v: str(v))
def test_pw_tile_variants_integer_exact(N, groups, m, hw, wgs, tune):
    """The resident-tile pointwise kernel at each slice width, with one and
    several slices per tile, a ragged last col-group and ragged pixel tail,
    pixel rows that do and do not allow 16-byte copies, and workgroup counts
    that cut the cost ranges inside tiles (1, 5 and the default).  Every case
    is a shape the kernel takes (forcing it on one it does not fit is an
    error, not a skip)."""
    tune("pw_kernel", 1)
    if wgs != "default":
        tune("pw_wgs", wgs)
    n = (groups - 1) * N + N // 2
    w, x = workloads.gen_integer_layer(seed=N + m, cout=n, cin=m, k=1, batch=2, H=hw[0], W=hw[1],
                                       wmax=1, xmax=2)
    print(f"pw tile N={N} n={n} m={m} hw={hw} wgs={wgs}", flush=True)
    for p in (0.0, 0.5, 0.95):
        y, _ = gpu_conv(w, x, N, p, True, 1, 0)
        ref, _ = oracle_conv(w, x, N, p, True, 1, 0)
        np.testing.assert_array_equal(y, ref)


@pytest.mark.parametrize("variant", ["g4rp2", "g4rp4", "g4rp6", "g8rp1", "g8rp2", "staged",
                                     "staged_w1", "staged_w3"])
@pytest.mark.parametrize("shape", [
    dict(m=300, B=3, H=14, W=14),    # 5 channel chunks (ragged last), partial last granule per image
    dict(m=64, B=2, H=12, W=12),     # one chunk, whole granules, tiles across images
    dict(m=45, B=1, H=4, W=3),       # fewer pixels than one tile
    dict(m=700, B=1, H=8, W=6),      # long contraction: several pipeline periods and a tail
    dict(m=2100, B=1, H=4, W=4),     # more input channels than the register kernel stages
], ids=["m300", "m64", "m45", "m700", "m2100"])
def test_pw_bf16_integer_exact(shape, variant, tune):
    """The bf16 pointwise kernel (1x1, N = 32, pixels per image a multiple of
    4): the register-gathered kernel with 4-pixel granules at pipeline depths
    2, 4, 6 and with 8-pixel granules at depths 1, 2 (images of 12 and 196
    pixels end in a half-duplicate granule), where more input channels than
    it stages (m = 2100) take the generic kernel; and the LDS-staged kernel
    (any m; images of 12 and 196 pixels end in a half-filled granule) on its
    default grid and on grids of 1 and 3 workgroups, which walk several work
    items each (the chunk ring runs on across items, and the next item's
    first windows are loaded before the stores).  At p = 0.97 a window of 16
    kept blocks spans more than two 128-channel chunks and is multiplied in
    several passes.  Small integers are exact in bf16 and in fp32
    accumulation, so fp32 output is bit-exact and bf16 output equals the
    oracle rounded to bf16.  Covers ragged col-groups, a partial last set of
    col-groups (n = 304: 8 per set gathered, 15 per set staged) and dense to
    nearly empty col-groups (p = 0, 0.5, 0.97)."""
    if variant.startswith("staged"):
        tune("pwb_kernel", 2)
        if "_w" in variant:
            tune("pwb_wgs", variant.split("_w")[1])
    else:
        tune("pwb_kernel", 1)
        tune("pwb_gp", variant[1])
        tune("pwb_rp", variant[4:])
    c = shape
    n = 9 * 32 + 16
    w, x = workloads.gen_integer_layer(seed=c["m"] + int(c["B"]), cout=n, cin=c["m"], k=1,
                                       batch=c["B"], H=c["H"], W=c["W"], wmax=3, xmax=3)
    print(f"pw bf16 {c} {variant}", flush=True)
    for p in (0.0, 0.5, 0.97):
        ref, _ = oracle_conv(w, x, 32, p, False, 1, 0)
        y, _ = gpu_conv(w.bfloat16(), x.bfloat16(), 32, p, False, 1, 0, "nchw", torch.float32)
        np.testing.assert_array_equal(y, ref)
        yb, _ = gpu_conv(w.bfloat16(), x.bfloat16(), 32, p, False, 1, 0, "nchw", torch.bfloat16)
        refb = torch.from_numpy(ref).to(torch.bfloat16).double().numpy()
        np.testing.assert_array_equal(yb, refb)


@pytest.mark.parametrize("split", ["1", "4"])
@pytest.mark.parametrize("case", [
    dict(N=4, m=64, n=64, B=1, H=56, W=56, s=1, pd=1),    # the 3x3 N = 4 batch-1 workload's shape
    dict(N=1, m=13, n=5, B=3, H=19, W=17, s=1, pd=1),     # odd sizes, pixel blocks across images
    dict(N=2, m=30, n=9, B=2, H=15, W=13, s=2, pd=1),     # stride 2
    dict(N=8, m=21, n=28, B=2, H=12, W=11, s=1, pd=0),    # no padding, ragged last col-group
    dict(N=8, m=300, n=16, B=1, H=7, W=7, s=1, pd=1),     # long contraction, few pixels
    dict(N=4, m=7, n=12, B=4, H=9, W=10, s=3, pd=2),      # stride 3, padding 2
], ids=lambda c: f"N{c['N']}_m{c['m']}_n{c['n']}_B{c['B']}_{c['H']}x{c['W']}_s{c['s']}p{c['pd']}")
def test_kxk_fma_integer_exact(case, split, tune):
    """The 3x3 FMA kernel (N <= 8) with four col-groups per workgroup and with
    the contraction split over the four waves, p from dense to nearly empty
    (odd and single kept blocks at the end of a share)."""
    tune("kxkf_split", split)
    c = case
    w, x = workloads.gen_integer_layer(seed=c["m"] * 3 + c["N"], cout=c["n"], cin=c["m"], k=3,
                                       batch=c["B"], H=c["H"], W=c["W"], wmax=2, xmax=2)
    print(f"kxk fma {c} split={split}", flush=True)
    for p in (0.0, 0.5, 0.95):
        y, _ = gpu_conv(w, x, c["N"], p, True, c["s"], c["pd"])
        ref, _ = oracle_conv(w, x, c["N"], p, True, c["s"], c["pd"])
        np.testing.assert_array_equal(y, ref)


@pytest.mark.parametrize("tile", [None, "3", "16"])
@pytest.mark.parametrize("case", [
    dict(N=32, m=64, n=80, B=2, H=12, W=12, s=1, pd=0),     # 3 col-groups, 2 waves each; ragged last col-group
    dict(N=16, m=13, n=40, B=3, H=9, W=7, s=1, pd=0),       # rows not a multiple of 4, tiles across images
    dict(N=32, m=300, n=300, B=2, H=14, W=14, s=2, pd=0),   # stride 2, 10 col-groups (sets of 8 and 2)
    dict(N=16, m=150, n=64, B=1, H=10, W=11, s=2, pd=1),    # padding: input pixels outside the image
    dict(N=32, m=400, n=64, B=1, H=7, W=7, s=1, pd=0),      # longest rows, several index windows
    dict(N=16, m=390, n=48, B=2, H=5, W=6, s=1, pd=0),      # long rows not a multiple of 4
    dict(N=32, m=45, n=33, B=4, H=3, W=5, s=1, pd=0),       # n not a multiple of 4 (scalar stores)
    dict(N=16, m=32, n=16, B=2, H=19, W=21, s=1, pd=0),     # one col-group shared by 8 waves
], ids=lambda c: f"N{c['N']}_m{c['m']}_n{c['n']}_B{c['B']}_{c['H']}x{c['W']}_s{c['s']}p{c['pd']}")
def test_pw_nhwc_integer_exact(case, tile, tune):
    """The NHWC 1x1 kernel (input rows of a pixel tile staged in LDS, shared by
    up to eight col-groups) at several tile sizes: strides, padding, ragged
    col-groups and tiles, col-groups held in registers and streamed (p from
    dense to nearly empty), rows longer than one index window."""
    if tile is not None:
        tune("nhwc_tile", tile)
    c = case
    w, x = workloads.gen_integer_layer(seed=c["m"] + c["N"] + c["s"], cout=c["n"], cin=c["m"], k=1,
                                       batch=c["B"], H=c["H"], W=c["W"], wmax=2, xmax=2)
    print(f"pw nhwc {c} tile={tile}", flush=True)
    for p in (0.0, 0.5, 0.95):
        y, _ = gpu_conv(w, x, c["N"], p, True, c["s"], c["pd"], "nhwc")
        ref, _ = oracle_conv(w, x, c["N"], p, True, c["s"], c["pd"])
        np.testing.assert_array_equal(y, ref)


@pytest.mark.parametrize("tp", ["128", "256"])
@pytest.mark.parametrize("case", [
    dict(k=3, s=1, pd=1, B=2, H=56, W=56, m=20, N=32),   # 4 whole rows per tile
    dict(k=3, s=1, pd=1, B=5, H=14, W=14, m=37, N=32),   # tiles span images
    dict(k=3, s=2, pd=1, B=3, H=28, W=28, m=19, N=32),   # stride 2: rows straddle images
    dict(k=3, s=1, pd=1, B=9, H=7, W=7, m=70, N=16),     # many images per tile
    dict(k=3, s=1, pd=0, B=2, H=11, W=13, m=9, N=16),    # no padding, non-square
    dict(k=1, s=2, pd=0, B=3, H=28, W=28, m=45, N=32),   # strided 1x1 (downsample)
    dict(k=1, s=2, pd=0, B=2, H=15, W=9, m=40, N=16),
    dict(k=7, s=2, pd=3, B=2, H=40, W=40, m=3, N=32),    # stem-like: 3 channels
    dict(k=7, s=2, pd=3, B=2, H=33, W=30, m=5, N=32),    # odd kept count after whole chunks
    dict(k=7, s=2, pd=3, B=2, H=33, W=30, m=5, N=16),
], ids=lambda c: f"k{c['k']}s{c['s']}p{c['pd']}_B{c['B']}_{c['H']}x{c['W']}_m{c['m']}_N{c['N']}")
def test_kxk_integer_exact(case, tp, tune):
    """The LDS-staged k x k kernel at both tile sizes: tiles of whole output
    rows that span images, padding and stride, ragged last col-group, and p
    from dense to nearly empty (chunks with fewer kept blocks than a step)."""
    tune("kxk_tp", tp)
    c = case
    n = 2 * c["N"] + c["N"] // 2
    w, x = workloads.gen_integer_layer(seed=c["m"] * 7 + c["k"], cout=n, cin=c["m"], k=c["k"],
                                       batch=c["B"], H=c["H"], W=c["W"], wmax=2, xmax=3)
    print(f"kxk {c} tp={tp}", flush=True)
    for p in (0.0, 0.5, 0.9):
        y, _ = gpu_conv(w, x, c["N"], p, True, c["s"], c["pd"])
        ref, _ = oracle_conv(w, x, c["N"], p, True, c["s"], c["pd"])
        np.testing.assert_array_equal(y, ref)


@pytest.mark.parametrize("split", ["0", "1", "4"])
@pytest.mark.parametrize("case", [
    dict(k=3, s=1, pd=1, B=2, H=56, W=56, m=20, N=32),
    dict(k=3, s=1, pd=1, B=5, H=14, W=14, m=37, N=32),
    dict(k=3, s=2, pd=1, B=3, H=28, W=28, m=19, N=32),
    dict(k=3, s=1, pd=1, B=9, H=7, W=7, m=70, N=16),
    dict(k=7, s=2, pd=3, B=2, H=33, W=30, m=5, N=32),
    dict(k=7, s=2, pd=3, B=2, H=33, W=30, m=5, N=16),
], ids=lambda c: f"k{c['k']}s{c['s']}p{c['pd']}_B{c['B']}_{c['H']}x{c['W']}_m{c['m']}_N{c['N']}")
def test_kxk_balanced_split_integer_exact(case, split, tune):
    """The k x k kernel with the (tile, col-group, chunk) sequence cut into
    equal ranges per workgroup: blocks cut into up to eight parts that add
    into a zeroed output, col-groups with no kept block, and ranges that end
    inside the last chunk of a col-group."""
    tune("kxk_split", split)
    c = case
    n = 2 * c["N"] + c["N"] // 2
    w, x = workloads.gen_integer_layer(seed=c["m"] * 5 + c["k"], cout=n, cin=c["m"], k=c["k"],
                                       batch=c["B"], H=c["H"], W=c["W"], wmax=2, xmax=3)
    print(f"kxk split {c} split={split}", flush=True)
    for p in (0.0, 0.5, 0.9, 1.0):
        y, _ = gpu_conv(w, x, c["N"], p, True, c["s"], c["pd"])
        ref, _ = oracle_conv(w, x, c["N"], p, True, c["s"], c["pd"])
        np.testing.assert_array_equal(y, ref)


@pytest.mark.parametrize("split", ["1", "4"])
def test_kxk_balanced_split_random_fp32(split, tune):
    """Random fp32 data with blocks much longer than the split's ranges (cut
    into up to eight parts that add into the output in arrival order):
    every launch is within 1e-5 of the oracle, and repeated launches agree to
    the order-of-summation error."""
    tune("kxk_split", split)
    tune("kxk_tp", 128)
    gen = torch.Generator().manual_seed(23)
    w = workloads.gen_weight(gen, 80, 256, 3)
    x = workloads.gen_activation(gen, (2, 256, 14, 14))
    layer = onexn.prepare_layer(w, 32, 0.5, False)
    xd = x.cuda()
    ys = [layer.forward(xd, 1, 1).double().cpu().numpy() for _ in range(5)]
    ref, _ = oracle_conv(w, x, 32, 0.5, False, 1, 1)
    for y in ys:
        assert rel_err(y, ref) <= 1e-5
        assert rel_err(y, ys[0]) <= 1e-6


def test_kxk_matches_generic_on_random_fp32():
    """Random-valued fp32 3x3 layer: the staged kernel and the oracle agree to
    1e-5 of max |y| over a contraction of 288 * 9 entries."""
    gen = torch.Generator().manual_seed(11)
    w = workloads.gen_weight(gen, 96, 288, 3)
    x = workloads.gen_activation(gen, (3, 288, 14, 14))
    y, _ = gpu_conv(w, x, 32, 0.5, True, 1, 1)
    ref, _ = oracle_conv(w, x, 32, 0.5, True, 1, 1)
    assert rel_err(y, ref) <= 1e-5


@pytest.mark.parametrize("kind", ["kxk", "tile", "bf16", "bf16s", "generic", "fma", "fma5", "pwfma", "direct",
                                  "nhwc16", "nhwc32"])
def test_reads_stay_inside_I_and_D(kind, tune):
    """I and D are views at the start of larger buffers whose tails hold a
    valid channel index (0) and NaN weights: a kernel that used any entry past
    t would put NaN into the output."""
    k, N, m, dt, H = {"kxk": (3, 32, 40, torch.float32, 12), "tile": (1, 16, 200, torch.float32, 12),
                      "bf16": (1, 32, 96, torch.bfloat16, 12), "bf16s": (1, 32, 300, torch.bfloat16, 12),
                      "generic": (5, 16, 30, torch.float32, 12), "fma": (3, 4, 30, torch.float32, 12),
                      "fma5": (5, 4, 30, torch.float32, 12),
                      "pwfma": (1, 4, 30, torch.float32, 12), "direct": (1, 32, 90, torch.float32, 12),
                      "nhwc16": (1, 16, 90, torch.float32, 12), "nhwc32": (1, 32, 90, torch.float32, 12)}[kind]
    if kind in ("tile", "direct"):
        tune("pw_kernel", {"tile": 1, "direct": 3}[kind])
    if kind in ("bf16", "bf16s"):
        tune("pwb_kernel", 1 if kind == "bf16" else 2)
    n = 3 * N + N // 2
    w, x = workloads.gen_integer_layer(seed=7, cout=n, cin=m, k=k, batch=2, H=H, wmax=2, xmax=2)
    w, x = w.to(dt), x.to(dt)
    layer = onexn.prepare_layer(w, N, 0.5, False)
    t = layer.t
    extra = 4096
    I_big = torch.zeros(t + extra, dtype=torch.int32, device="cuda")
    I_big[:t] = layer.I
    D_big = torch.full((t + extra, N, k, k), float("nan"), dtype=dt, device="cuda")
    D_big[:t] = layer.D
    pd = k // 2
    if kind.startswith("nhwc"):
        y = onexn.conv2d_fwd(layer.P, I_big[:t], D_big[:t], n, x.permute(0, 2, 3, 1).contiguous().cuda(),
                             1, pd, "nhwc", out_dtype=torch.float32).permute(0, 3, 1, 2)
    else:
        y = onexn.conv2d_fwd(layer.P, I_big[:t], D_big[:t], n, x.cuda(), 1, pd, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref, _ = oracle_conv(w.float(), x.float(), N, 0.5, False, 1, pd)
    np.testing.assert_array_equal(y.double().cpu().numpy(), ref)


@pytest.mark.parametrize("tile", ["1", "2", "3", "4", "5"])
@pytest.mark.parametrize("case", [
    dict(N=4, m=24, n=98, B=3, H=9, W=7),        # odd pixels per image, ragged last col-group
    dict(N=8, m=1100, n=44, B=2, H=5, W=5),      # contractions longer than one staged window
    dict(N=1, m=37, n=5, B=2, H=13, W=11),
    dict(N=2, m=64, n=17, B=1, H=16, W=16),
    dict(N=4, m=20, n=50, B=3, H=12, W=10),      # pixels per image a multiple of 4 (16-byte path)
    dict(N=8, m=16, n=72, B=5, H=28, W=28),
], ids=lambda c: f"N{c['N']}_m{c['m']}_n{c['n']}_B{c['B']}_{c['H']}x{c['W']}")
def test_pw_fma_integer_exact(case, tile, tune):
    """The 1x1 FMA kernel at every tile shape (pixels per lane, col-groups per
    workgroup, waves splitting a contraction), with a partial last set of
    col-groups and p from dense to nearly empty."""
    tune("fma_tile", tile)
    c = case
    w, x = workloads.gen_integer_layer(seed=c["m"] + c["N"], cout=c["n"], cin=c["m"], k=1,
                                       batch=c["B"], H=c["H"], W=c["W"], wmax=1, xmax=2)
    print(f"pw fma {c} tile={tile}", flush=True)
    for p in (0.0, 0.5, 0.95):
        y, _ = gpu_conv(w, x, c["N"], p, True, 1, 0)
        ref, _ = oracle_conv(w, x, c["N"], p, True, 1, 0)
        np.testing.assert_array_equal(y, ref)


@pytest.mark.parametrize("kdb", ["2", "8"])
@pytest.mark.parametrize("tile", ["1", "2", "3", "4"])
@pytest.mark.parametrize("case", [
    dict(N=32, m=45, n=80, B=3, H=28, W=28, s=2, pd=0),   # strided 1x1 (downsample)
    dict(N=16, m=300, n=56, B=2, H=15, W=9, s=2, pd=1),   # stride and padding
    dict(N=32, m=700, n=40, B=2, H=7, W=7, s=1, pd=0),    # long contraction, few pixels
    dict(N=16, m=33, n=20, B=1, H=10, W=13, s=3, pd=2),
], ids=lambda c: f"N{c['N']}_m{c['m']}_n{c['n']}_{c['H']}x{c['W']}_s{c['s']}p{c['pd']}")
def test_pw_direct_integer_exact(case, tile, kdb, tune):
    """The 1x1 kernel with register-loaded operands at every tile shape
    (column blocks per unit, waves splitting the contraction) and both batch
    sizes (2 and 8 MFMA steps; odd batch counts run a batch of zeros):
    strides, padding, ragged col-groups and pixel tails, p from dense to
    nearly empty."""
    tune("direct_tile", tile)
    tune("direct_kdb", kdb)
    tune("pw_kernel", 3)
    c = case
    w, x = workloads.gen_integer_layer(seed=c["m"] + c["n"], cout=c["n"], cin=c["m"], k=1,
                                       batch=c["B"], H=c["H"], W=c["W"], wmax=1, xmax=2)
    print(f"pw direct {c} tile={tile} kdb={kdb}", flush=True)
    for p in (0.0, 0.5, 0.95):
        y, _ = gpu_conv(w, x, c["N"], p, True, c["s"], c["pd"])
        ref, _ = oracle_conv(w, x, c["N"], p, True, c["s"], c["pd"])
        np.testing.assert_array_equal(y, ref)


def _fwd_fuzz_cases(count, seed):
    """Seeded random small layers spanning the forward dispatch: N, kernel
    size, stride, padding, NCHW / NHWC, fp32 / bf16 inputs, channel counts
    (ragged col-groups), map sizes, batch, p and the rearrangement."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < count:
        N = int(rng.choice([1, 2, 4, 8, 16, 32]))
        k = int(rng.choice([1, 1, 1, 3, 3, 5, 7]))
        s = int(rng.choice([1, 1, 2, 3]))
        pd = int(rng.integers(0, (k + 1) // 2 + 1))
        H, W = int(rng.integers(k, 17)), int(rng.integers(k, 17))
        if (H + 2 * pd - k) // s + 1 < 1 or (W + 2 * pd - k) // s + 1 < 1:
            continue
        n = int(rng.integers(1, 3 * N + 40))
        m = int(rng.integers(1, 120))
        B = int(rng.integers(1, 4))
        p = float(rng.choice([0.0, 0.5, 0.9]))
        layout = str(rng.choice(["nchw", "nchw", "nhwc"]))
        dt = str(rng.choice(["f32", "f32", "bf16"]))
        re = bool(rng.integers(0, 2))
        cases.append((n, m, k, s, pd, B, H, W, N, p, layout, dt, re))
    return cases


@pytest.mark.parametrize("case", _fwd_fuzz_cases(300, 7),
                         ids=lambda c: "n%d_m%d_k%d_s%d_p%d_B%d_%dx%d_N%d_p%g_%s_%s_re%d" % c)
def test_conv_fuzz_integer_exact(case):
    """The forward integer-exact against the oracle on 300 seeded random small
    layers (outputs pre-filled with NaN; bf16 inputs write fp32 outputs, so
    the integer sums stay exact)."""
    n, m, k, s, pd, B, H, W, N, p, layout, dt, re = case
    print(f"conv fuzz {case}", flush=True)
    w, x = workloads.gen_integer_layer(seed=n * 3 + m + k, cout=n, cin=m, k=k, batch=B, H=H, W=W,
                                       wmax=2, xmax=2)
    if dt == "bf16":
        w, x = w.bfloat16(), x.bfloat16()
    y, _ = gpu_conv(w, x, N, p, re, s, pd, layout, out_dtype=torch.float32)
    ref, _ = oracle_conv(w.float(), x.float(), N, p, re, s, pd)
    np.testing.assert_array_equal(y, ref)
