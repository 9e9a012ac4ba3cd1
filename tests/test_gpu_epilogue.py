"""GPU parity of the fused epilogue (per-channel scale/bias, ReLU/ReLU6, output
cast) in every kernel family, and of a two-layer chain that consumes the
rearranged layer's output with the next layer's input channels permuted
(Sec. 3.3), against the oracle's network in the original channel order."""

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


# kind -> (k, stride, pad, N, m, dtype, H, tuning overrides)
KINDS = {
    "kxk": (3, 1, 1, 32, 40, torch.float32, 14, {}),
    "kxk_split_requested": (3, 1, 1, 32, 40, torch.float32, 14, {"kxk_split": 4, "kxk_tp": 128}),
    "kxk_split_7x7": (3, 1, 1, 32, 40, torch.float32, 7, {"kxk_split": 4, "kxk_tp": 128}),
    "kxk_stem": (7, 2, 3, 32, 3, torch.float32, 30, {}),
    "tile": (1, 1, 0, 16, 200, torch.float32, 12, {"pw_kernel": 1}),
    "direct": (1, 2, 0, 32, 90, torch.float32, 12, {"pw_kernel": 3}),
    "bf16r": (1, 1, 0, 32, 96, torch.bfloat16, 12, {"pwb_kernel": 1}),
    "bf16s": (1, 1, 0, 32, 300, torch.bfloat16, 14, {"pwb_kernel": 2}),
    "generic_mfma": (5, 1, 2, 16, 30, torch.float32, 12, {}),
    "kxk_fma": (3, 1, 1, 4, 30, torch.float32, 12, {}),
    "kxk_fma_split": (3, 1, 1, 8, 30, torch.float32, 12, {"kxkf_split": 4}),
    "generic_fma": (5, 1, 2, 4, 30, torch.float32, 12, {}),
    "pw_fma": (1, 1, 0, 8, 30, torch.float32, 12, {}),
    "bf16_kxk": (3, 1, 1, 16, 24, torch.bfloat16, 10, {}),
}


def _params(n, seed):
    gen = torch.Generator().manual_seed(seed)
    scale = torch.randint(-2, 3, (n,), generator=gen).float()
    bias = torch.randint(-9, 10, (n,), generator=gen).float()
    return scale, bias


@pytest.mark.parametrize("act", ["none", "relu", "relu6"])
@pytest.mark.parametrize("kind", sorted(KINDS))
def test_epilogue_integer_exact(kind, act, tune):
    """Small integers: conv, affine map and clamps are exact in fp32 (and the
    results exact in bf16), so the output equals the oracle's bit for bit.
    Channels are in rearranged order and so are the parameters."""
    k, s, pd, N, m, dt, H, knobs = KINDS[kind]
    for name, v in knobs.items():
        tune(name, v)
    n = 3 * N + N // 2
    print(f"epilogue {kind} act={act}", flush=True)
    w, x = workloads.gen_integer_layer(seed=k * 11 + N, cout=n, cin=m, k=k, batch=2, H=H,
                                       wmax=2, xmax=2)
    scale, bias = _params(n, N + m)
    layer = onexn.prepare_layer(w.to(dt), N, 0.5, True)
    pr = oracle.prune(w.double().numpy(), N, 0.5, True)
    sp, bp = scale[layer.perm.long()], bias[layer.perm.long()]
    ref = oracle.epilogue(oracle.conv2d(x.double().numpy(), pr.wbar, (s, s), (pd, pd)),
                          sp.double().numpy(), bp.double().numpy(), act)
    for odt in ([torch.float32, torch.bfloat16] if dt == torch.bfloat16 else [torch.float32]):
        y = layer.forward(x.to(dt).cuda(), s, pd, "nchw", odt, scale=sp.cuda(), bias=bp.cuda(),
                          act=act)
        torch.cuda.synchronize()
        want = torch.from_numpy(ref).to(odt).double().numpy()   # exact: small integers
        np.testing.assert_array_equal(y.double().cpu().numpy(), want)


@pytest.mark.parametrize("k,N", [(3, 16), (1, 16), (1, 32)])
def test_epilogue_nhwc_and_partial_parameters(k, N):
    """NHWC layout (3x3: the generic kernel; 1x1: the NHWC kernel); scale
    alone, bias alone."""
    w, x = workloads.gen_integer_layer(seed=3, cout=40, cin=17, k=k, batch=2, H=9, wmax=2, xmax=2)
    scale, bias = _params(40, 5)
    layer = onexn.prepare_layer(w, N, 0.5, True)
    pr = oracle.prune(w.double().numpy(), N, 0.5, True)
    pd = k // 2
    conv = oracle.conv2d(x.double().numpy(), pr.wbar, (1, 1), (pd, pd))
    xh = x.permute(0, 2, 3, 1).contiguous().cuda()
    sp, bp = scale[layer.perm.long()], bias[layer.perm.long()]
    for sc, bi in ((sp, None), (None, bp), (sp, bp)):
        y = layer.forward(xh, 1, pd, "nhwc", scale=None if sc is None else sc.cuda(),
                          bias=None if bi is None else bi.cuda(), act="relu")
        torch.cuda.synchronize()
        ref = oracle.epilogue(conv, None if sc is None else sc.double().numpy(),
                              None if bi is None else bi.double().numpy(), "relu")
        np.testing.assert_array_equal(y.permute(0, 3, 1, 2).double().cpu().numpy(), ref)


def test_fused_without_epilogue_equals_plain_call():
    """onexn_conv2d_fwd_fused with no scale, no bias and no activation is the
    plain convolution, bit for bit (3x3 and 1x1; integer-valued data, since a
    k x k layer whose blocks are split over workgroups adds their parts in
    arrival order)."""
    lib = onexn.load_library()
    for k, N in ((3, 32), (1, 16), (1, 4)):
        w, x = workloads.gen_integer_layer(seed=k + N, cout=80, cin=48, k=k, batch=2, H=14)
        x = x.cuda()
        layer = onexn.prepare_layer(w, N, 0.5, False)
        y0 = layer.forward(x, 1, k // 2)
        y1 = torch.full_like(y0, float("nan"))
        stream = torch.cuda.current_stream().cuda_stream
        st = lib.onexn_conv2d_fwd_fused(layer.P.data_ptr(), layer.I.data_ptr(), layer.D.data_ptr(),
                                        0, 80, 48, k, k, N, layer.t, x.data_ptr(), 0, 0, 2, 14, 14,
                                        1, 1, k // 2, k // 2, y1.data_ptr(), 0, None, None, 0, stream)
        assert st == 0
        torch.cuda.synchronize()
        assert torch.equal(y0, y1)


def _chain(dtype, integer, N1, N2, seed):
    """conv 3x3 (rearranged, pruned) -> folded BN -> ReLU -> conv 1x1 (pruned,
    input channels permuted by layer 1's perm) -> bias -> ReLU6, on the GPU
    through the C ABI; and the same network in the original channel order in
    the oracle."""
    B, m, H, n1, n2 = 3, 24, 14, 72, 40
    gen = torch.Generator().manual_seed(seed)
    if integer:
        w1, x = workloads.gen_integer_layer(seed=seed, cout=n1, cin=m, k=3, batch=B, H=H,
                                            wmax=2, xmax=2)
        w2 = torch.randint(-2, 3, (n2, n1, 1, 1), generator=gen).float()
        s1, b1 = _params(n1, seed + 1)
        s1 = s1.abs() + 1
        _, b2 = _params(n2, seed + 2)
    else:
        w1 = workloads.gen_weight(gen, n1, m, 3)
        x = workloads.gen_activation(gen, (B, m, H, H))
        w2 = workloads.gen_weight(gen, n2, n1, 1)
        s1 = torch.rand(n1, generator=gen) + 0.5
        b1 = torch.randn(n1, generator=gen) * 0.1
        b2 = torch.randn(n2, generator=gen) * 0.1
    w1, w2, x = w1.to(dtype), w2.to(dtype), x.to(dtype)

    # GPU: layer 1 rearranged; its BN parameters and layer 2's input channels follow perm.
    l1 = onexn.prepare_layer(w1, N1, 0.5, True)
    perm = l1.perm.long()
    l2 = onexn.prepare_layer(w2[:, perm].contiguous(), N2, 0.5, False)
    h = l1.forward(x.cuda(), 1, 1, scale=s1[perm].cuda(), bias=b1[perm].cuda(), act="relu")
    y = l2.forward(h, 1, 0, out_dtype=torch.float32, bias=b2.cuda(), act="relu6")
    torch.cuda.synchronize()

    # Oracle: the network in the original order (layer 1's pruned filters put back).
    pr1 = oracle.prune(w1.double().numpy(), N1, 0.5, True)
    assert np.array_equal(pr1.perm, l1.perm.numpy())
    pr2 = oracle.prune(w2[:, perm].double().numpy(), N2, 0.5, False)
    w1o = np.empty_like(pr1.wbar)
    w1o[pr1.perm] = pr1.wbar
    w2o = np.empty_like(pr2.wbar)
    w2o[:, pr1.perm] = pr2.wbar
    h_ref = oracle.epilogue(oracle.conv2d(x.double().numpy(), w1o, (1, 1), (1, 1)),
                            s1.double().numpy(), b1.double().numpy(), "relu")
    if dtype == torch.bfloat16:     # the GPU's intermediate is bf16: round the oracle's the same way
        h_ref = torch.from_numpy(h_ref).to(torch.bfloat16).double().numpy()
    y_ref = oracle.epilogue(oracle.conv2d(h_ref, w2o), None, b2.double().numpy(), "relu6")
    return y.double().cpu().numpy(), y_ref


@pytest.mark.parametrize("N1,N2", [(32, 16), (16, 32), (4, 8), (8, 4)])
def test_two_layer_chain_integer_exact(N1, N2):
    print(f"chain N1={N1} N2={N2}", flush=True)
    y, ref = _chain(torch.float32, True, N1, N2, seed=N1 + N2)
    np.testing.assert_array_equal(y, ref)


@pytest.mark.parametrize("N1,N2", [(32, 16), (4, 32)])
def test_two_layer_chain_fp32(N1, N2):
    y, ref = _chain(torch.float32, False, N1, N2, seed=7 * N1 + N2)
    assert rel_err(y, ref) <= 1e-5


def test_two_layer_chain_bf16():
    """bf16 weights and activations, bf16 intermediate (fused cast), fp32 final
    output.  The GPU rounds layer 1's fp32 accumulator to bf16 and the oracle
    its fp64 value, so an intermediate can differ by one bf16 step: the bf16
    bar applies."""
    y, ref = _chain(torch.bfloat16, False, 32, 32, seed=41)
    assert rel_err(y, ref) <= 2e-2


def test_unknown_activation_is_rejected():
    lib = onexn.load_library()
    w, x = workloads.gen_integer_layer(seed=1, cout=32, cin=8, k=1, batch=1, H=4)
    layer = onexn.prepare_layer(w, 16, 0.5, False)
    xd = x.cuda()
    y = torch.empty((1, 32, 4, 4), device="cuda")
    st = lib.onexn_conv2d_fwd_fused(layer.P.data_ptr(), layer.I.data_ptr(), layer.D.data_ptr(), 0,
                                    32, 8, 1, 1, 16, layer.t, xd.data_ptr(), 0, 0, 1, 4, 4, 1, 1, 0,
                                    0, y.data_ptr(), 0, None, None, 3, None)
    assert st == 2   # ONEXN_ERR_ARG
    assert "activation" in onexn.last_error()
