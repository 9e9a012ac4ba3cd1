"""The no-allocation mask entry point (onexn_build_mask_dev_noalloc), called
through the C ABI, against the workspace entry point (onexn_build_mask_dev):
perm, mask and t bit for bit on two calls in a row, the second on a smaller
layer (the library's scratch array keeps the first call's contents), and the
size limit."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2105_14713_amd as onexn

pytestmark = pytest.mark.gpu


def _noalloc(lib, w, N, p, rearrange):
    n, m, kh, kw = w.shape
    G = -(-n // N)
    perm = torch.full((n,), -1, dtype=torch.int32, device="cuda")
    mask = torch.full((m, G), 7, dtype=torch.uint8, device="cuda")
    t = ctypes.c_int64(-1)
    st = lib.onexn_build_mask_dev_noalloc(w.data_ptr(), onexn._dtype_code(w.dtype), n, m, kh, kw, N,
                                          float(p), int(rearrange), perm.data_ptr(), mask.data_ptr(),
                                          ctypes.addressof(t), torch.cuda.current_stream().cuda_stream)
    return st, perm, mask, t.value


def test_noalloc_matches_workspace_entry_point_on_two_calls():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib = onexn.load_library()
    gen = torch.Generator().manual_seed(11)
    layers = [(torch.randn(512, 256, 3, 3, generator=gen), 32, 0.5, True),    # 1 call: 4096 blocks
              (torch.randn(40, 16, 1, 1, generator=gen).bfloat16(), 8, 0.7, False)]   # smaller
    for w, N, p, re in layers:
        wd = w.cuda()
        st, perm, mask, t = _noalloc(lib, wd, N, p, re)
        assert st == 0, onexn.last_error()
        perm_ref, mask_ref, t_ref = onexn.build_mask_dev(wd, N, p, re)
        torch.cuda.synchronize()
        assert t == t_ref
        assert torch.equal(perm, perm_ref)
        assert torch.equal(mask, mask_ref)
        perm_h, mask_h, t_h = onexn.build_mask(w, N, p, re)
        np.testing.assert_array_equal(mask.cpu().numpy(), mask_h.numpy())
        np.testing.assert_array_equal(perm.cpu().numpy(), perm_h.numpy())


def test_noalloc_rejects_layers_beyond_its_scratch():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib = onexn.load_library()
    n, m, N = 4096, 4096, 1          # 4096 * 4096 scores of 8 bytes: 128 MiB
    assert onexn.mask_workspace_bytes(n, m, N) > (8 << 20)
    w = torch.zeros((1,), device="cuda")   # never read: the size check comes first
    perm = torch.empty(1, dtype=torch.int32, device="cuda")
    mask = torch.empty(1, dtype=torch.uint8, device="cuda")
    t = ctypes.c_int64(-1)
    st = lib.onexn_build_mask_dev_noalloc(w.data_ptr(), 0, n, m, 1, 1, N, 0.5, 1, perm.data_ptr(),
                                          mask.data_ptr(), ctypes.addressof(t), None)
    assert st == 6                   # ONEXN_ERR_BUFSIZE
    assert "scratch" in onexn.last_error()
    assert t.value == -1
