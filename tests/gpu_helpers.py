"""Shared helpers of the GPU parity tests: run one layer through the HIP path and
through the oracle on the same seeded inputs."""
import numpy as np
import torch

import oracle
import paper_2105_14713_amd as onexn
import workloads


def rel_err(y, ref):
    """max |y - ref| / max |ref| (0 when both are all zero)."""
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.abs(ref).max() if ref.size else 0.0
    num = np.abs(y - ref).max() if ref.size else 0.0
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return float(num / den)


def gpu_conv(w, x_nchw, N, p, rearrange, stride, pad, layout="nchw", out_dtype=None, fill_nan=True):
    """HIP path: mask + pack on the host library, conv on the GPU.  Returns
    (y as NCHW CPU float64 numpy, packed layer)."""
    layer = onexn.prepare_layer(w, N, p, rearrange)
    x = x_nchw if layout == "nchw" else x_nchw.permute(0, 2, 3, 1).contiguous()
    xd = x.cuda()
    B = x_nchw.shape[0]
    Ho, Wo = onexn.out_hw(x_nchw.shape[2], x_nchw.shape[3], w.shape[2], w.shape[3],
                          (stride, stride), (pad, pad))
    odt = x.dtype if out_dtype is None else out_dtype
    shape = (B, w.shape[0], Ho, Wo) if layout == "nchw" else (B, Ho, Wo, w.shape[0])
    out = torch.full(shape, float("nan") if fill_nan else 0.0, dtype=odt, device="cuda")
    y = layer.forward(xd, stride, pad, layout, odt, out=out)
    torch.cuda.synchronize()
    y = y.float().cpu()
    if layout == "nhwc":
        y = y.permute(0, 3, 1, 2).contiguous()
    return y.double().numpy(), layer


def oracle_conv(w, x_nchw, N, p, rearrange, stride, pad):
    pr = oracle.prune(w.double().numpy(), N, p, rearrange)
    return oracle.conv2d(x_nchw.double().numpy(), pr.wbar, (stride, stride), (pad, pad)), pr


def sample_indices(shape, count, seed, N):
    """Flat NCHW output indices for a sampled check: ``count`` random ones, one in
    every (pixel tile, col-group) cell, the corners and the last col-group's rows
    (``workloads.sample_outputs``)."""
    return workloads.sample_outputs(shape, N, count, seed)
