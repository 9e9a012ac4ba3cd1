"""onexn: 1xN-pruned convolution on AMD Instinct MI355X (gfx950).

Thin ctypes binding of ``libonexn.so`` (C ABI in ``include/onexn.h``).  The
functions here only marshal arguments: mask building and packing run in the
library's host C++, the convolution runs in its HIP kernels.  torch is used
for host/device memory and for the current HIP stream.  There is no fallback:
if the library is missing every call raises.

    perm, mask, t = build_mask(w, N, p, rearrange)        # Sec. 3.2-3.3, Eq. 1/5
    P, I, D = pack(w, N, perm, mask, t)                     # Sec. 3.4, Fig. 3
    y = conv2d_fwd(P, I, D, n, x, N, stride, pad)           # Eq. 8 on the GPU
"""
import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libonexn.so")

ONEXN_OK = 0
_STATUS_NAMES = ["ONEXN_OK", "ONEXN_ERR_NULL", "ONEXN_ERR_ARG", "ONEXN_ERR_SHAPE",
                 "ONEXN_ERR_DTYPE", "ONEXN_ERR_UNSUPPORTED", "ONEXN_ERR_BUFSIZE", "ONEXN_ERR_HIP"]
F32, BF16 = 0, 1
NCHW, NHWC = 0, 1

EXPORTED = ("onexn_build_mask", "onexn_mask_workspace_bytes", "onexn_build_mask_dev",
            "onexn_build_mask_dev_noalloc", "onexn_pack", "onexn_conv2d_fwd", "onexn_conv2d_fwd_fused",
            "onexn_conv2d_bwd_data", "onexn_conv2d_bwd_weight", "onexn_fc_fwd", "onexn_set_tuning", "onexn_status_string", "onexn_last_error")
ACTS = {"none": 0, "relu": 1, "relu6": 2}

_lib = None


class OnexnError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        self.status = status
        name = _STATUS_NAMES[status] if 0 <= status < len(_STATUS_NAMES) else str(status)
        super().__init__(f"{where}: {name}: {message}")


def load_library():
    """Loads libonexn.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2105_14713_amd.build` (no CPU fallback exists)")
    lib = ctypes.CDLL(LIB_PATH)
    c_i32, c_i64, c_vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
    lib.onexn_build_mask.argtypes = [c_vp, ctypes.c_int, c_i32, c_i32, c_i32, c_i32, c_i32,
                                     ctypes.c_double, c_i32, c_vp, c_vp, c_vp]
    lib.onexn_build_mask.restype = ctypes.c_int
    lib.onexn_mask_workspace_bytes.argtypes = [c_i32, c_i32, c_i32]
    lib.onexn_mask_workspace_bytes.restype = ctypes.c_size_t
    lib.onexn_build_mask_dev.argtypes = [c_vp, ctypes.c_int, c_i32, c_i32, c_i32, c_i32, c_i32,
                                         ctypes.c_double, c_i32, c_vp, c_vp, c_vp, c_vp,
                                         ctypes.c_size_t, c_vp]
    lib.onexn_build_mask_dev.restype = ctypes.c_int
    lib.onexn_build_mask_dev_noalloc.argtypes = [c_vp, ctypes.c_int, c_i32, c_i32, c_i32, c_i32, c_i32,
                                                 ctypes.c_double, c_i32, c_vp, c_vp, c_vp, c_vp]
    lib.onexn_build_mask_dev_noalloc.restype = ctypes.c_int
    lib.onexn_pack.argtypes = [c_vp, ctypes.c_int, c_i32, c_i32, c_i32, c_i32, c_i32, c_vp, c_vp,
                               c_i64, c_vp, c_vp, c_vp]
    lib.onexn_pack.restype = ctypes.c_int
    lib.onexn_conv2d_fwd.argtypes = ([c_vp, c_vp, c_vp, ctypes.c_int] + [c_i32] * 5 + [c_i64] +
                                     [c_vp, ctypes.c_int, ctypes.c_int] + [c_i32] * 7 +
                                     [c_vp, ctypes.c_int, c_vp])
    lib.onexn_conv2d_fwd.restype = ctypes.c_int
    lib.onexn_conv2d_fwd_fused.argtypes = ([c_vp, c_vp, c_vp, ctypes.c_int] + [c_i32] * 5 + [c_i64] +
                                           [c_vp, ctypes.c_int, ctypes.c_int] + [c_i32] * 7 +
                                           [c_vp, ctypes.c_int, c_vp, c_vp, ctypes.c_int, c_vp])
    lib.onexn_conv2d_fwd_fused.restype = ctypes.c_int
    lib.onexn_conv2d_bwd_data.argtypes = ([c_vp, c_vp, c_vp, ctypes.c_int] + [c_i32] * 5 + [c_i64] +
                                          [c_vp, ctypes.c_int] + [c_i32] * 7 + [c_vp, ctypes.c_int, c_vp])
    lib.onexn_conv2d_bwd_data.restype = ctypes.c_int
    lib.onexn_conv2d_bwd_weight.argtypes = ([c_vp, c_vp] + [c_i32] * 5 + [c_i64] + [c_vp, ctypes.c_int, c_vp] +
                                            [c_i32] * 7 + [c_vp, c_vp])
    lib.onexn_conv2d_bwd_weight.restype = ctypes.c_int
    lib.onexn_fc_fwd.argtypes = ([c_vp, c_vp, c_vp, ctypes.c_int, c_i32, c_i32, c_i32, c_i64, c_vp,
                                  ctypes.c_int, ctypes.c_int, c_i32, c_vp, ctypes.c_int, c_vp, c_vp,
                                  ctypes.c_int, c_vp])
    lib.onexn_fc_fwd.restype = ctypes.c_int
    lib.onexn_set_tuning.argtypes = [ctypes.c_char_p, c_i32]
    lib.onexn_set_tuning.restype = ctypes.c_int
    lib.onexn_status_string.argtypes = [ctypes.c_int]
    lib.onexn_status_string.restype = ctypes.c_char_p
    lib.onexn_last_error.argtypes = []
    lib.onexn_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().onexn_status_string(int(status)).decode()


def last_error() -> str:
    return load_library().onexn_last_error().decode()


def set_tuning(name: str, value: int) -> None:
    """``onexn_set_tuning``: force a kernel variant or launch shape (-1 restores
    the automatic choice).  For tests and A/B timing."""
    _check(load_library().onexn_set_tuning(name.encode(), int(value)), "onexn_set_tuning")


def _check(status: int, where: str):
    if status != ONEXN_OK:
        raise OnexnError(status, where, last_error())


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.float32:
        return F32
    if dt == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {dt}; expected float32 or bfloat16")


def _host_weight(w: torch.Tensor) -> torch.Tensor:
    if w.dim() != 4:
        raise ValueError("weight must be [n][m][kh][kw]")
    if w.device.type != "cpu":
        raise ValueError("mask building and packing take a host (CPU) weight tensor")
    return w.contiguous()


def build_mask(w: torch.Tensor, N: int, p: float, rearrange: bool) -> Tuple[torch.Tensor, torch.Tensor, int]:
    """``onexn_build_mask``: returns (perm int32[n], mask uint8[m][G], t)."""
    w = _host_weight(w)
    n, m, kh, kw = w.shape
    G = -(-n // int(N)) if N > 0 else 1
    perm = torch.empty(n, dtype=torch.int32)
    mask = torch.empty((m, G), dtype=torch.uint8)
    t = ctypes.c_int64(0)
    st = load_library().onexn_build_mask(w.data_ptr(), _dtype_code(w.dtype), n, m, kh, kw, int(N),
                                         float(p), int(bool(rearrange)), perm.data_ptr(),
                                         mask.data_ptr(), ctypes.addressof(t))
    _check(st, "onexn_build_mask")
    return perm, mask, int(t.value)


def mask_workspace_bytes(n: int, m: int, N: int) -> int:
    """``onexn_mask_workspace_bytes``: device scratch that build_mask_dev needs."""
    return int(load_library().onexn_mask_workspace_bytes(int(n), int(m), int(N)))


def build_mask_dev(w: torch.Tensor, N: int, p: float, rearrange: bool,
                   workspace: Optional[torch.Tensor] = None, stream: Optional[int] = None):
    """``onexn_build_mask_dev`` on a device weight: returns (perm int32[n],
    mask uint8[m][G], both on the device, and t).  Enqueued on ``stream``
    (default: torch's current stream); ``workspace`` (a device uint8 tensor of
    at least mask_workspace_bytes bytes) is allocated here when not given."""
    if w.dim() != 4 or w.device.type != "cuda" or not w.is_contiguous():
        raise ValueError("w must be a contiguous device tensor [n][m][kh][kw]")
    n, m, kh, kw = w.shape
    G = -(-n // int(N)) if N > 0 else 1
    need = mask_workspace_bytes(n, m, N)
    if workspace is None:
        workspace = torch.empty(max(need, 8), dtype=torch.uint8, device=w.device)
    elif workspace.device.type != "cuda" or workspace.dtype != torch.uint8 or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous device uint8 tensor")
    perm = torch.empty(n, dtype=torch.int32, device=w.device)
    mask = torch.empty((m, G), dtype=torch.uint8, device=w.device)
    t = ctypes.c_int64(0)
    if stream is None:
        stream = torch.cuda.current_stream(w.device).cuda_stream
    st = load_library().onexn_build_mask_dev(w.data_ptr(), _dtype_code(w.dtype), n, m, kh, kw, int(N),
                                             float(p), int(bool(rearrange)), perm.data_ptr(),
                                             mask.data_ptr(), ctypes.addressof(t), workspace.data_ptr(),
                                             workspace.numel(), stream)
    _check(st, "onexn_build_mask_dev")
    return perm, mask, int(t.value)


def pack(w: torch.Tensor, N: int, perm: torch.Tensor, mask: torch.Tensor, t: int):
    """``onexn_pack``: returns host (P int32[G+1], I int32[t], D [t][N][kh][kw] in w's dtype)."""
    w = _host_weight(w)
    n, m, kh, kw = w.shape
    G = -(-n // int(N))
    perm = perm.to(torch.int32).contiguous()
    mask = mask.to(torch.uint8).contiguous()
    if perm.numel() != n or mask.numel() != m * G:
        raise ValueError("perm/mask sizes do not match the weight and N")
    P = torch.empty(G + 1, dtype=torch.int32)
    I = torch.empty(max(int(t), 1), dtype=torch.int32)
    D = torch.empty((max(int(t), 1), int(N), kh, kw), dtype=w.dtype)
    st = load_library().onexn_pack(w.data_ptr(), _dtype_code(w.dtype), n, m, kh, kw, int(N),
                                   perm.data_ptr(), mask.data_ptr(), int(t), P.data_ptr(),
                                   I.data_ptr(), D.data_ptr())
    _check(st, "onexn_pack")
    return P, I[:int(t)], D[:int(t)]


def out_hw(H: int, W: int, kh: int, kw: int, stride, pad) -> Tuple[int, int]:
    return (H + 2 * pad[0] - kh) // stride[0] + 1, (W + 2 * pad[1] - kw) // stride[1] + 1


def _pair(v):
    return (int(v), int(v)) if isinstance(v, int) else (int(v[0]), int(v[1]))


def _epilogue_args(n, scale, bias, act):
    """(scale ptr, bias ptr, act code, fused?) for the fused entry point."""
    if act not in ACTS:
        raise ValueError(f"act must be one of {sorted(ACTS)}")
    for name, v in (("scale", scale), ("bias", bias)):
        if v is not None and (v.device.type != "cuda" or v.dtype != torch.float32 or
                              not v.is_contiguous() or v.numel() != n):
            raise ValueError(f"{name} must be a contiguous float32 device tensor of {n} entries")
    fused = scale is not None or bias is not None or act != "none"
    return (scale.data_ptr() if scale is not None else 0, bias.data_ptr() if bias is not None else 0,
            ACTS[act], fused)


def _conv_call(P, I, D, n, x, stride, pad, layout, out_dtype, out, stream, scale, bias, act):
    """Validates a conv2d_fwd call and marshals its arguments: returns (library
    function, argument tuple, out).  Nothing is launched."""
    for name, tns in (("P", P), ("I", I), ("D", D), ("x", x)):
        if tns.device.type != "cuda":
            raise ValueError(f"{name} must be a device tensor (the convolution only runs on the GPU)")
        if not tns.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if D.dim() != 4:
        raise ValueError("D must be [t][N][kh][kw]")
    t, N, kh, kw = D.shape
    if t != I.numel():
        raise ValueError("D and I disagree on t")
    lay = {"nchw": NCHW, "nhwc": NHWC}[layout]
    if lay == NCHW:
        B, m, H, W = x.shape
    else:
        B, H, W, m = x.shape
    stride, pad = _pair(stride), _pair(pad)
    Ho, Wo = out_hw(H, W, kh, kw, stride, pad)
    odt = x.dtype if out_dtype is None else out_dtype
    shape = (B, n, Ho, Wo) if lay == NCHW else (B, Ho, Wo, n)
    if out is None:
        out = torch.empty(shape, dtype=odt, device=x.device)
    elif tuple(out.shape) != shape or out.dtype != odt or not out.is_contiguous():
        raise ValueError("out has the wrong shape, dtype or layout")
    if stream is None:
        stream = torch.cuda.current_stream(x.device).cuda_stream
    sp, bp, ac, fused = _epilogue_args(int(n), scale, bias, act)
    args = (P.data_ptr(), I.data_ptr() if t else 0, D.data_ptr() if t else 0, _dtype_code(D.dtype),
            int(n), m, kh, kw, N, t, x.data_ptr(), _dtype_code(x.dtype), lay, B, H, W, stride[0],
            stride[1], pad[0], pad[1], out.data_ptr(), _dtype_code(odt))
    lib = load_library()
    if fused:
        return lib.onexn_conv2d_fwd_fused, args + (sp, bp, ac, stream), out
    return lib.onexn_conv2d_fwd, args + (stream,), out


def conv2d_fwd(P: torch.Tensor, I: torch.Tensor, D: torch.Tensor, n: int, x: torch.Tensor,
               stride=1, pad=0, layout: str = "nchw", out_dtype: Optional[torch.dtype] = None,
               out: Optional[torch.Tensor] = None, stream: Optional[int] = None,
               scale: Optional[torch.Tensor] = None, bias: Optional[torch.Tensor] = None,
               act: str = "none") -> torch.Tensor:
    """``onexn_conv2d_fwd`` on device tensors; enqueued on ``stream`` (default:
    torch's current stream), no synchronisation.  Returns y (rearranged channel order).
    With ``scale``, ``bias`` (fp32 [n], rearranged channel order) or ``act``
    ("relu", "relu6") it calls ``onexn_conv2d_fwd_fused``: y = act(scale * acc + bias)."""
    fn, args, out = _conv_call(P, I, D, n, x, stride, pad, layout, out_dtype, out, stream, scale,
                               bias, act)
    _check(fn(*args), fn.__name__)
    return out


def _dev_contig(**tensors):
    for name, tns in tensors.items():
        if tns.device.type != "cuda" or not tns.is_contiguous():
            raise ValueError(f"{name} must be a contiguous device tensor")


def conv2d_bwd_data(P, I, D, n: int, m: int, dy: torch.Tensor, input_hw, stride=1, pad=0,
                    out_dtype: Optional[torch.dtype] = None, out: Optional[torch.Tensor] = None,
                    stream: Optional[int] = None) -> torch.Tensor:
    """``onexn_conv2d_bwd_data``: dX [B][m][H][W] of the 1xN conv from dY
    [B][n][Ho][Wo] (NCHW, rearranged output channels)."""
    _dev_contig(P=P, I=I, D=D, dy=dy)
    t, N, kh, kw = D.shape
    B = dy.shape[0]
    H, W = input_hw
    stride, pad = _pair(stride), _pair(pad)
    if tuple(dy.shape) != (B, n) + out_hw(H, W, kh, kw, stride, pad):
        raise ValueError("dy does not have the layer's output shape")
    odt = dy.dtype if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty((B, m, H, W), dtype=odt, device=dy.device)
    elif tuple(out.shape) != (B, m, H, W) or out.dtype != odt or not out.is_contiguous():
        raise ValueError("out has the wrong shape, dtype or layout")
    if stream is None:
        stream = torch.cuda.current_stream(dy.device).cuda_stream
    st = load_library().onexn_conv2d_bwd_data(
        P.data_ptr(), I.data_ptr() if t else 0, D.data_ptr() if t else 0, _dtype_code(D.dtype), int(n),
        int(m), kh, kw, N, t, dy.data_ptr(), _dtype_code(dy.dtype), B, H, W, stride[0], stride[1],
        pad[0], pad[1], out.data_ptr(), _dtype_code(odt), stream)
    _check(st, "onexn_conv2d_bwd_data")
    return out


def conv2d_bwd_weight(P, I, n: int, N: int, kernel_hw, x: torch.Tensor, dy: torch.Tensor, stride=1,
                      pad=0, out: Optional[torch.Tensor] = None,
                      stream: Optional[int] = None) -> torch.Tensor:
    """``onexn_conv2d_bwd_weight``: the fp32 gradient dD [t][N][kh][kw] of the
    kept blocks from X [B][m][H][W] and dY [B][n][Ho][Wo] (NCHW)."""
    _dev_contig(P=P, I=I, x=x, dy=dy)
    t = I.numel()
    kh, kw = kernel_hw
    B, m, H, W = x.shape
    stride, pad = _pair(stride), _pair(pad)
    if tuple(dy.shape) != (B, n) + out_hw(H, W, kh, kw, stride, pad) or dy.dtype != x.dtype:
        raise ValueError("dy does not have the layer's output shape or x's dtype")
    if out is None:
        out = torch.empty((t, N, kh, kw), dtype=torch.float32, device=x.device)
    elif tuple(out.shape) != (t, N, kh, kw) or out.dtype != torch.float32 or not out.is_contiguous():
        raise ValueError("out must be a contiguous fp32 tensor [t][N][kh][kw]")
    if stream is None:
        stream = torch.cuda.current_stream(x.device).cuda_stream
    st = load_library().onexn_conv2d_bwd_weight(
        P.data_ptr(), I.data_ptr() if t else 0, int(n), m, kh, kw, int(N), t, x.data_ptr(),
        _dtype_code(x.dtype), dy.data_ptr(), B, H, W, stride[0], stride[1], pad[0], pad[1],
        out.data_ptr() if t else 0, stream)
    _check(st, "onexn_conv2d_bwd_weight")
    return out


def fc_fwd(P: torch.Tensor, I: torch.Tensor, D: torch.Tensor, n: int, x: torch.Tensor,
           layout: str = "rows", out_dtype: Optional[torch.dtype] = None,
           out: Optional[torch.Tensor] = None, stream: Optional[int] = None,
           scale: Optional[torch.Tensor] = None, bias: Optional[torch.Tensor] = None,
           act: str = "none") -> torch.Tensor:
    """``onexn_fc_fwd``: x is [B][m] ("rows", one row per sample) or [m][B]
    ("cols", one row per feature); returns y [B][n] or [n][B] (rearranged
    feature order).  D is [t][N] or [t][N][1][1]."""
    for name, tns in (("P", P), ("I", I), ("D", D), ("x", x)):
        if tns.device.type != "cuda":
            raise ValueError(f"{name} must be a device tensor")
        if not tns.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if x.dim() != 2 or D.dim() not in (2, 4) or (D.dim() == 4 and tuple(D.shape[2:]) != (1, 1)):
        raise ValueError("x must be 2-D and D [t][N] (or [t][N][1][1])")
    t, N = int(D.shape[0]), int(D.shape[1])
    if t != I.numel():
        raise ValueError("D and I disagree on t")
    lay = {"rows": NHWC, "cols": NCHW}[layout]
    B, m = (x.shape[0], x.shape[1]) if layout == "rows" else (x.shape[1], x.shape[0])
    odt = x.dtype if out_dtype is None else out_dtype
    shape = (B, n) if layout == "rows" else (n, B)
    if out is None:
        out = torch.empty(shape, dtype=odt, device=x.device)
    elif tuple(out.shape) != shape or out.dtype != odt or not out.is_contiguous():
        raise ValueError("out has the wrong shape, dtype or layout")
    if stream is None:
        stream = torch.cuda.current_stream(x.device).cuda_stream
    sp, bp, ac, _ = _epilogue_args(int(n), scale, bias, act)
    st = load_library().onexn_fc_fwd(P.data_ptr(), I.data_ptr() if t else 0, D.data_ptr() if t else 0,
                                     _dtype_code(D.dtype), int(n), int(m), N, t, x.data_ptr(),
                                     _dtype_code(x.dtype), lay, int(B), out.data_ptr(),
                                     _dtype_code(odt), sp, bp, ac, stream)
    _check(st, "onexn_fc_fwd")
    return out


class BoundConv:
    """A conv2d_fwd call with its arguments validated and marshalled once;
    calling it issues the launch (same tensors, same stream).  The tensors must
    stay alive and unmoved while this object is used."""

    def __init__(self, P, I, D, n, x, out, stride=1, pad=0, layout="nchw", stream=None,
                 scale=None, bias=None, act="none"):
        self._fn, self._args, _ = _conv_call(P, I, D, n, x, stride, pad, layout, out.dtype, out,
                                             stream, scale, bias, act)
        self._keep = (P, I, D, x, out, scale, bias)

    def __call__(self):
        st = self._fn(*self._args)
        if st != ONEXN_OK:
            _check(st, self._fn.__name__)


@dataclass
class PackedLayer:
    """A pruned layer's BSR arrays resident on the device plus its metadata."""
    n: int
    m: int
    kh: int
    kw: int
    N: int
    t: int
    perm: torch.Tensor   # host int32[n]
    mask: torch.Tensor   # host uint8[m][G]
    P: torch.Tensor      # device int32[G+1]
    I: torch.Tensor      # device int32[t]
    D: torch.Tensor      # device [t][N][kh][kw]

    def forward(self, x, stride=1, pad=0, layout="nchw", out_dtype=None, out=None, stream=None,
                scale=None, bias=None, act="none"):
        return conv2d_fwd(self.P, self.I, self.D, self.n, x, stride, pad, layout, out_dtype, out,
                          stream, scale, bias, act)


def prepare_layer(w: torch.Tensor, N: int, p: float, rearrange: bool,
                  device="cuda") -> PackedLayer:
    """Offline steps (mask, pack) on the host, then one copy of P, I, D to the device."""
    perm, mask, t = build_mask(w, N, p, rearrange)
    P, I, D = pack(w, N, perm, mask, t)
    n, m, kh, kw = w.shape
    dev = torch.device(device)
    if t == 0:   # keep valid device allocations even with nothing kept
        I = torch.zeros(1, dtype=torch.int32)[:0]
        D = torch.zeros((0, N, kh, kw), dtype=w.dtype)
    return PackedLayer(n, m, kh, kw, int(N), t, perm, mask, P.to(dev), I.to(dev), D.to(dev))


__all__ = ["ACTS", "BF16", "BoundConv", "EXPORTED", "F32", "build_mask_dev", "conv2d_bwd_data",
           "conv2d_bwd_weight", "fc_fwd",
           "mask_workspace_bytes", "LIB_PATH", "NCHW", "NHWC", "OnexnError", "PackedLayer",
           "build_mask", "conv2d_fwd", "last_error", "load_library", "out_hw", "pack",
           "prepare_layer", "set_tuning", "status_string"]
