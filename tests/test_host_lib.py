"""Host side of libonexn.so on the CPU: exports, bit-exact mask/pack vs the
oracle, and error paths.  No GPU work is launched by any test here."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import paper_2105_14713_amd as onexn
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(onexn.LIB_PATH):
        pytest.fail("libonexn.so is not built (run `python -m paper_2105_14713_amd.build`)")
    return onexn.load_library()


def test_exports_every_declared_symbol(lib):
    with open(os.path.join(ROOT, "include", "onexn.h")) as f:
        header = f.read()
    declared = set(re.findall(r"\b(onexn_[a-z0-9_]+)\s*\(", header))
    assert declared == set(onexn.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name
    for s in range(8):
        assert onexn.status_string(s) == onexn._STATUS_NAMES[s]
    assert onexn.status_string(99) == "ONEXN_UNKNOWN"


def _compare_with_oracle(oracle_lib, w: torch.Tensor, N: int, p: float, rearrange: bool):
    perm, mask, t = onexn.build_mask(w, N, p, rearrange)
    P, I, D = onexn.pack(w, N, perm, mask, t)
    ref = oracle_lib.prune(w.double().numpy(), N, p, rearrange)
    np.testing.assert_array_equal(perm.numpy(), ref.perm)
    np.testing.assert_array_equal(mask.numpy(), ref.T)
    assert t == ref.t
    np.testing.assert_array_equal(P.numpy(), ref.P)
    np.testing.assert_array_equal(I.numpy(), ref.I)
    # D is a bit copy of weights in w's dtype; the oracle holds the same values in fp64.
    np.testing.assert_array_equal(D.double().numpy(), ref.D)
    return t


@pytest.mark.parametrize("wl", [workloads.config0(), workloads.config1(), workloads.config4()],
                         ids=lambda w: w.name)
def test_mask_pack_bit_exact_single_layer_configs(oracle_lib, wl):
    layer = wl.layers[0]
    w, _ = workloads.gen_layer(layer, 1, wl.dtype)
    t = _compare_with_oracle(oracle_lib, w, layer.N, layer.p, layer.rearrange)
    K = layer.cin * -(-layer.cout // layer.N)
    assert t == K - int(np.floor(layer.p * K + 0.5))


def test_mask_pack_bit_exact_resnet50(oracle_lib):
    for layer in workloads.resnet50_convs():
        w, _ = workloads.gen_layer(layer, 1)
        _compare_with_oracle(oracle_lib, w, layer.N, layer.p, layer.rearrange)


@pytest.mark.parametrize("N", [4, 8, 16, 32])
def test_mask_pack_bit_exact_mobilenet_v2(oracle_lib, N):
    for p in (0.3, 0.5, 0.7):
        for layer in workloads.mobilenet_v2_pointwise(N, p):
            w, _ = workloads.gen_layer(layer, 1)
            _compare_with_oracle(oracle_lib, w, layer.N, layer.p, layer.rearrange)


def test_mask_pack_fuzz(oracle_lib):
    rng = np.random.default_rng(1234)
    for trial in range(120):
        n, m = int(rng.integers(1, 97)), int(rng.integers(1, 97))
        k = int(rng.choice([1, 3, 7]))
        N = int(rng.choice([1, 2, 4, 8, 16, 32]))
        p = float(rng.choice([0.0, 0.3, 0.5, 0.7, 1.0]))
        kind = trial % 4
        if kind == 0:
            w = torch.from_numpy(rng.standard_normal((n, m, k, k)).astype(np.float32))
        elif kind == 1:      # integer-valued: many equal scores
            w = torch.from_numpy(rng.integers(-2, 3, (n, m, k, k)).astype(np.float32))
        elif kind == 2:      # all equal: every score ties
            w = torch.full((n, m, k, k), 0.25)
        else:                # bf16 weights
            w = torch.from_numpy(rng.standard_normal((n, m, k, k)).astype(np.float32)).bfloat16()
        _compare_with_oracle(oracle_lib, w, N, p, bool(rng.integers(0, 2)))


def test_pack_accepts_any_mask_and_perm(oracle_lib):
    rng = np.random.default_rng(5)
    w = torch.from_numpy(rng.standard_normal((20, 9, 3, 3)).astype(np.float32))
    N, G = 8, 3
    perm = torch.from_numpy(rng.permutation(20).astype(np.int32))
    mask = torch.from_numpy(rng.integers(0, 2, (9, G)).astype(np.uint8))
    t = int(mask.sum())
    P, I, D = onexn.pack(w, N, perm, mask, t)
    wt = oracle_lib.apply_perm(w.double().numpy(), perm.numpy())
    rP, rI, rD = oracle_lib.pack(wt, mask.numpy(), N)
    np.testing.assert_array_equal(P.numpy(), rP)
    np.testing.assert_array_equal(I.numpy(), rI)
    np.testing.assert_array_equal(D.double().numpy(), rD)


# ---------------------------------------------------------------------------
# Error paths.
# ---------------------------------------------------------------------------

ERR = {name: i for i, name in enumerate(onexn._STATUS_NAMES)}


def test_build_mask_errors(lib):
    w = torch.randn(8, 4, 3, 3)
    perm = torch.empty(8, dtype=torch.int32)
    mask = torch.empty(4 * 2, dtype=torch.uint8)
    t = ctypes.c_int64(0)
    good = [w.data_ptr(), onexn.F32, 8, 4, 3, 3, 4, 0.5, 1, perm.data_ptr(), mask.data_ptr(),
            ctypes.addressof(t)]
    assert lib.onexn_build_mask(*good) == 0

    def call(i, v):
        args = list(good)
        args[i] = v
        return lib.onexn_build_mask(*args)

    assert call(0, None) == ERR["ONEXN_ERR_NULL"]
    assert call(9, None) == ERR["ONEXN_ERR_NULL"]
    assert call(11, None) == ERR["ONEXN_ERR_NULL"]
    assert call(1, 7) == ERR["ONEXN_ERR_DTYPE"]
    assert call(2, 0) == ERR["ONEXN_ERR_ARG"]
    assert call(6, 0) == ERR["ONEXN_ERR_ARG"]
    assert call(6, -4) == ERR["ONEXN_ERR_ARG"]
    assert call(7, -0.1) == ERR["ONEXN_ERR_ARG"]
    assert call(7, 1.5) == ERR["ONEXN_ERR_ARG"]
    assert call(7, float("nan")) == ERR["ONEXN_ERR_ARG"]
    assert "p must lie" in onexn.last_error()
    wn = w.clone()
    wn[3, 1, 0, 0] = float("nan")
    assert call(0, wn.data_ptr()) == ERR["ONEXN_ERR_ARG"]
    args = list(good)
    args[2], args[3] = 1 << 16, 1 << 16      # n*m*kh*kw >= 2^31: rejected before any access
    assert lib.onexn_build_mask(*args) == ERR["ONEXN_ERR_BUFSIZE"]
    with pytest.raises(onexn.OnexnError):
        onexn.build_mask(w, 0, 0.5, True)


def test_pack_errors(lib):
    w = torch.randn(8, 4, 1, 1)
    perm, mask, t = onexn.build_mask(w, 4, 0.5, False)
    P = torch.empty(3, dtype=torch.int32)
    I = torch.empty(max(t, 1), dtype=torch.int32)
    D = torch.empty((max(t, 1), 4, 1, 1))
    good = [w.data_ptr(), onexn.F32, 8, 4, 1, 1, 4, perm.data_ptr(), mask.data_ptr(), t,
            P.data_ptr(), I.data_ptr(), D.data_ptr()]
    assert lib.onexn_pack(*good) == 0

    def call(i, v):
        args = list(good)
        args[i] = v
        return lib.onexn_pack(*args)

    assert call(0, None) == ERR["ONEXN_ERR_NULL"]
    assert call(10, None) == ERR["ONEXN_ERR_NULL"]
    assert call(11, None) == ERR["ONEXN_ERR_NULL"]
    assert call(1, 3) == ERR["ONEXN_ERR_DTYPE"]
    assert call(9, t + 1) == ERR["ONEXN_ERR_ARG"]
    assert call(9, -1) == ERR["ONEXN_ERR_ARG"]
    bad_perm = perm.clone()
    bad_perm[0] = bad_perm[1]
    assert call(7, bad_perm.data_ptr()) == ERR["ONEXN_ERR_ARG"]
    out_of_range = perm.clone()
    out_of_range[2] = 8
    assert call(7, out_of_range.data_ptr()) == ERR["ONEXN_ERR_ARG"]
    bad_mask = mask.clone()
    bad_mask[0, 0] = 2
    assert call(8, bad_mask.data_ptr()) == ERR["ONEXN_ERR_ARG"]


def test_conv_argument_errors_launch_nothing(lib):
    """Every case below differs from a batch == 0 call (which is a no-op) in one
    argument, so even a validation bug could not start a kernel."""
    fake = 4096   # never dereferenced: all cases fail validation or have batch == 0
    #      P     I     D   wdt n  m  kh kw N  t   x    xdt lay  B  H  W  sh sw ph pw y    ydt stream
    good = [fake, fake, fake, 0, 8, 4, 3, 3, 4, 4, fake, 0, 0, 0, 9, 9, 1, 1, 1, 1, fake, 0, None]
    assert lib.onexn_conv2d_fwd(*good) == 0

    def call(**kw):
        names = ["P", "I", "D", "wdt", "n", "m", "kh", "kw", "N", "t", "x", "xdt", "layout", "B",
                 "H", "W", "sh", "sw", "ph", "pw", "y", "ydt", "stream"]
        args = list(good)
        for k, v in kw.items():
            args[names.index(k)] = v
        return lib.onexn_conv2d_fwd(*args)

    assert call(P=None) == ERR["ONEXN_ERR_NULL"]
    assert call(x=None, y=None) == 0                         # empty batch: nothing is touched
    assert call(I=None) == ERR["ONEXN_ERR_NULL"]
    assert call(I=None, D=None, t=0) == 0
    assert call(wdt=5) == ERR["ONEXN_ERR_DTYPE"]
    assert call(wdt=1) == ERR["ONEXN_ERR_DTYPE"]            # w and x differ
    assert call(ydt=1) == ERR["ONEXN_ERR_DTYPE"]            # f32 in, bf16 out
    assert call(wdt=1, xdt=1, ydt=0) == 0                   # bf16 in, f32 out is allowed
    assert call(layout=3) == ERR["ONEXN_ERR_ARG"]
    assert call(B=-1) == ERR["ONEXN_ERR_ARG"]
    assert call(n=0) == ERR["ONEXN_ERR_ARG"]
    assert call(sh=0) == ERR["ONEXN_ERR_ARG"]
    assert call(ph=-1) == ERR["ONEXN_ERR_ARG"]
    assert call(t=-1) == ERR["ONEXN_ERR_ARG"]
    assert call(N=3) == ERR["ONEXN_ERR_UNSUPPORTED"]
    assert call(N=64) == ERR["ONEXN_ERR_UNSUPPORTED"]
    assert call(kh=17) == ERR["ONEXN_ERR_UNSUPPORTED"]
    assert call(sh=9) == ERR["ONEXN_ERR_UNSUPPORTED"]
    assert call(H=1, ph=0) == ERR["ONEXN_ERR_SHAPE"]        # 3x3 kernel on a 1-row input
    assert call(t=9) == ERR["ONEXN_ERR_UNSUPPORTED"]        # more kept blocks than m*G = 8
    assert call(m=1 << 16, H=1 << 8, W=1 << 8) == ERR["ONEXN_ERR_UNSUPPORTED"]


@pytest.mark.skipif(torch.cuda.is_available(), reason="CPU-only check: the NULL checks are the "
                    "only thing between these fake pointers and a launch")
def test_conv_null_io_with_nonzero_batch(lib):
    fake = 4096
    args = [fake, fake, fake, 0, 8, 4, 3, 3, 4, 4, fake, 0, 0, 1, 9, 9, 1, 1, 1, 1, fake, 0, None]
    for pos in (10, 20):          # x, y
        bad = list(args)
        bad[pos] = None
        assert lib.onexn_conv2d_fwd(*bad) == ERR["ONEXN_ERR_NULL"]


def test_binding_refuses_host_tensors():
    P = torch.zeros(2, dtype=torch.int32)
    I = torch.zeros(1, dtype=torch.int32)
    D = torch.zeros(1, 4, 1, 1)
    x = torch.zeros(1, 1, 2, 2)
    with pytest.raises(ValueError, match="device tensor"):
        onexn.conv2d_fwd(P, I, D, 4, x)


def test_set_tuning_errors(lib):
    assert lib.onexn_set_tuning(b"pw_kernel", -1) == 0
    assert lib.onexn_set_tuning(b"no_such_knob", 1) == 2        # ONEXN_ERR_ARG
    assert "no_such_knob" in onexn.last_error()
    assert lib.onexn_set_tuning(b"pw_wpg", 1) == 2              # the streamed kernel's knob is gone
    assert lib.onexn_set_tuning(None, 1) == 1                    # ONEXN_ERR_NULL
    assert lib.onexn_set_tuning(b"kxk_split", -2) == 2
    for name in ("kernel", "pw_kernel", "pw_wgs", "pwb_gp", "pwb_rp", "direct_kdb", "direct_tile",
                 "fma_tpw", "fma_no_v4", "fma_tile", "kxk_split", "kxk_tp", "pwb_kernel", "pwb_wgs",
                 "kxkf_split", "nhwc_tile", "bwd_kernel", "bwd_split"):
        assert lib.onexn_set_tuning(name.encode(), -1) == 0, name


def test_fused_conv_rejects_unknown_activation_before_any_launch(lib):
    """The argument checks run on the host before anything is enqueued (batch 0:
    nothing would be launched anyway), so this runs without a GPU."""
    dummy = ctypes.c_int32(0)
    p = ctypes.addressof(dummy)
    st = lib.onexn_conv2d_fwd_fused(p, p, p, 0, 32, 8, 1, 1, 16, 1, None, 0, 0, 0, 4, 4, 1, 1, 0, 0,
                                    None, 0, None, None, 3, None)
    assert st == 2 and "activation" in onexn.last_error()
    st = lib.onexn_conv2d_fwd_fused(p, p, p, 0, 32, 8, 1, 1, 16, 1, None, 0, 0, 0, 4, 4, 1, 1, 0, 0,
                                    None, 0, None, None, 2, None)
    assert st == 0   # batch 0 with a valid activation: a no-op



def test_build_mask_dev_checks_arguments_on_the_host(lib):
    """onexn_build_mask_dev validates before enqueuing anything, so its errors
    show without a GPU; the workspace size grows with n and m * G."""
    assert lib.onexn_mask_workspace_bytes(32, 16, 8) >= 8 * (32 + 16 * 4)
    assert lib.onexn_mask_workspace_bytes(0, 16, 8) == 0
    dummy = ctypes.c_int64(0)
    p = ctypes.addressof(dummy)
    t = ctypes.c_int64(-1)
    base = [p, 0, 32, 16, 3, 3, 8, 0.5, 1, p, p, ctypes.addressof(t)]

    def call(i, v, ws=p, wsb=1 << 20):
        args = list(base)
        args[i] = v
        return lib.onexn_build_mask_dev(*args, ws, wsb, None)
    assert call(0, None) == ERR["ONEXN_ERR_NULL"]
    assert call(1, 7) == ERR["ONEXN_ERR_DTYPE"]
    assert call(2, 0) == ERR["ONEXN_ERR_ARG"]
    assert call(6, 0) == ERR["ONEXN_ERR_ARG"]
    assert call(7, 1.5) == ERR["ONEXN_ERR_ARG"]
    assert call(7, 0.5, None) == ERR["ONEXN_ERR_NULL"]
    assert call(7, 0.5, p, 8) == ERR["ONEXN_ERR_BUFSIZE"]
    assert t.value == -1
