"""Tiled symmetric InfoNCE (CLIP) loss on AMD MI355X: Python binding of libinfcl.so.

This module only marshals arguments: every step of the loss runs in the HIP
kernels behind the C ABI declared in ``include/infcl.h``.  PyTorch provides
device memory and the stream.  There is no fallback: if the library is not
built, or no GPU is present, calls raise.

Entry points with the C ABI's names (tensors in, status checked):
    infcl_workspace_size(b, d, dtype) -> int
    infcl_fwd(img, txt, scale, loss, loss64, lse_r, lse_c, aux, workspace)
    infcl_fwd_noalloc(img, txt, scale, loss, loss64, lse_r, lse_c, aux)
    infcl_bwd(img, txt, scale, lse_r, lse_c, aux, dloss, dimg, dtxt, dscale, workspace)
        (the gradient type passed to the C call is dimg's dtype)
Convenience wrappers that allocate outputs with torch:
    clip_loss_fwd(img, txt, scale) -> dict
    clip_loss_bwd(img, txt, scale, fwd, dloss=None, grad_dtype=None) -> (dimg, dtxt, dscale)
    clip_loss(img, txt, scale) -> loss   (torch.autograd.Function)
"""

from __future__ import annotations

import ctypes
import os
import re

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libinfcl.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "infcl.h")
ABLATION_HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "infcl_ablation.h")

INFCL_OK, INFCL_ERR_INVALID, INFCL_ERR_UNSUPPORTED, INFCL_ERR_WORKSPACE, INFCL_ERR_HIP = range(5)
INFCL_BF16, INFCL_F32, INFCL_F16 = 0, 1, 2

_lib = None


class InfclError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_str(status)} (status {status})")
        self.status = status


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libinfcl.so (built by ``python -m paper_2410_17243_amd.build``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2410_17243_amd.build`")
    # torch ships its own HIP runtime under another file name; it must be the
    # one loaded when this library's kernels register, or the process ends up
    # with two runtimes and launches on torch's streams fail
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    i64, sz, vp, ip = ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int
    lib.infcl_workspace_size.argtypes = [i64, i64, ip, ctypes.POINTER(sz)]
    lib.infcl_workspace_size.restype = ip
    lib.infcl_fwd.argtypes = [vp, vp, i64, i64, ip, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.infcl_fwd.restype = ip
    lib.infcl_fwd_noalloc.argtypes = [vp, vp, i64, i64, ip, vp, vp, vp, vp, vp, vp, vp]
    lib.infcl_fwd_noalloc.restype = ip
    lib.infcl_bwd.argtypes = [vp, vp, i64, i64, ip, vp, vp, vp, vp, vp, vp, vp, ip, vp, vp, sz, vp]
    lib.infcl_bwd.restype = ip
    lib.infcl_fwd_shard.argtypes = [vp, vp, i64, i64, ip, i64, i64, vp, vp, vp, sz, vp]
    lib.infcl_fwd_shard.restype = ip
    lib.infcl_fwd_shard_finish.argtypes = [i64, i64, ip, i64, i64, i64, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.infcl_fwd_shard_finish.restype = ip
    lib.infcl_bwd_shard.argtypes = [vp, vp, i64, i64, ip, i64, i64, vp, vp, vp, vp, vp, vp, vp, ip, vp, vp, sz, vp]
    lib.infcl_bwd_shard.restype = ip
    lib.infcl_ablation_bwd_single.argtypes = [vp, vp, i64, i64, ip, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.infcl_ablation_bwd_single.restype = ip
    lib.infcl_status_str.argtypes = [ip]
    lib.infcl_status_str.restype = ctypes.c_char_p
    _lib = lib
    return lib


def header_functions(path: str = HEADER_PATH):
    """Names of the functions that include/infcl.h declares."""
    text = open(path).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(infcl_\w+)\s*\(", text)))


def status_str(status: int) -> str:
    return load_library().infcl_status_str(int(status)).decode()


def _check(status: int, where: str):
    if status != INFCL_OK:
        raise InfclError(status, where)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dtype_code(t) -> int:
    import torch

    if t.dtype == torch.bfloat16:
        return INFCL_BF16
    if t.dtype == torch.float16:
        return INFCL_F16
    if t.dtype == torch.float32:
        return INFCL_F32
    raise TypeError(f"embeddings must be bfloat16, float16 or float32, got {t.dtype}")


def _stream(t):
    import torch

    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


# ------------------------------------------------------------------ C ABI names

def infcl_workspace_size(b: int, d: int, dtype: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().infcl_workspace_size(int(b), int(d), int(dtype), ctypes.byref(out)), "infcl_workspace_size")
    return out.value


def infcl_fwd(img, txt, scale, loss, loss64, lse_r, lse_c, aux, workspace):
    b, d = img.shape
    _check(load_library().infcl_fwd(_ptr(img), _ptr(txt), b, d, _dtype_code(img), _ptr(scale), _ptr(loss),
                                     _ptr(loss64), _ptr(lse_r), _ptr(lse_c), _ptr(aux), _ptr(workspace),
                                     workspace.numel() * workspace.element_size(), _stream(img)), "infcl_fwd")


def infcl_fwd_noalloc(img, txt, scale, loss, loss64, lse_r, lse_c, aux):
    b, d = img.shape
    _check(load_library().infcl_fwd_noalloc(_ptr(img), _ptr(txt), b, d, _dtype_code(img), _ptr(scale), _ptr(loss),
                                             _ptr(loss64), _ptr(lse_r), _ptr(lse_c), _ptr(aux), _stream(img)),
           "infcl_fwd_noalloc")


def infcl_bwd(img, txt, scale, lse_r, lse_c, aux, dloss, dimg, dtxt, dscale, workspace):
    b, d = img.shape
    _check(load_library().infcl_bwd(_ptr(img), _ptr(txt), b, d, _dtype_code(img), _ptr(scale), _ptr(lse_r),
                                     _ptr(lse_c), _ptr(aux), _ptr(dloss), _ptr(dimg), _ptr(dtxt), _dtype_code(dimg),
                                     _ptr(dscale), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                     _stream(img)), "infcl_bwd")


def infcl_fwd_shard(img, txt, scale, r0, bs, colpair, workspace):
    b, d = img.shape
    _check(load_library().infcl_fwd_shard(_ptr(img), _ptr(txt), b, d, _dtype_code(img), int(r0), int(bs), _ptr(scale),
                                           _ptr(colpair), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                           _stream(img)), "infcl_fwd_shard")


def infcl_fwd_shard_finish(b, d, dtype, r0, bs, colpairs, scale, lse_r, lse_c, aux, loss_part, workspace):
    nparts = colpairs.shape[0]
    _check(load_library().infcl_fwd_shard_finish(int(b), int(d), int(dtype), int(r0), int(bs), int(nparts),
                                                  _ptr(colpairs), _ptr(scale), _ptr(lse_r), _ptr(lse_c), _ptr(aux),
                                                  _ptr(loss_part), _ptr(workspace),
                                                  workspace.numel() * workspace.element_size(), _stream(scale)),
           "infcl_fwd_shard_finish")


def infcl_bwd_shard(img, txt, scale, r0, bs, lse_r, lse_c, aux, dloss, dimg, dtxt, dscale_part, workspace):
    b, d = img.shape
    _check(load_library().infcl_bwd_shard(_ptr(img), _ptr(txt), b, d, _dtype_code(img), int(r0), int(bs), _ptr(scale),
                                           _ptr(lse_r), _ptr(lse_c), _ptr(aux), _ptr(dloss), _ptr(dimg), _ptr(dtxt),
                                           _dtype_code(dimg), _ptr(dscale_part), _ptr(workspace),
                                           workspace.numel() * workspace.element_size(), _stream(img)),
           "infcl_bwd_shard")


def infcl_ablation_bwd_single(img, txt, scale, lse_r, lse_c, aux, dloss, dimg, dtxt, dscale, workspace):
    """The single-launch backward with atomic text-gradient updates (include/infcl_ablation.h)."""
    b, d = img.shape
    _check(load_library().infcl_ablation_bwd_single(
        _ptr(img), _ptr(txt), b, d, _dtype_code(img), _ptr(scale), _ptr(lse_r), _ptr(lse_c), _ptr(aux), _ptr(dloss),
        _ptr(dimg), _ptr(dtxt), _ptr(dscale), _ptr(workspace), workspace.numel() * workspace.element_size(),
        _stream(img)), "infcl_ablation_bwd_single")


# ------------------------------------------------------------- torch wrappers

def _validate(img, txt, scale):
    import torch

    if not (img.is_cuda and txt.is_cuda and scale.is_cuda):
        raise ValueError("img, txt and scale must be device tensors")
    if not (img.device == txt.device == scale.device):
        raise ValueError(f"img, txt and scale must be on one device, got {img.device}, {txt.device}, {scale.device}")
    if img.shape != txt.shape or img.dim() != 2 or img.dtype != txt.dtype:
        raise ValueError(f"img and txt must be [b, d] of one dtype, got {tuple(img.shape)}, {tuple(txt.shape)}")
    if not (img.is_contiguous() and txt.is_contiguous()):
        raise ValueError("img and txt must be contiguous")
    if scale.numel() != 1 or scale.dtype != torch.float32:
        raise ValueError("scale must be a float32 tensor with one element")


def _check_vec(t, n: int, name: str, dev):
    """t must be a contiguous float32 device tensor of n elements on dev."""
    import torch

    if t.device != dev or t.dtype != torch.float32 or t.numel() != n or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous float32 tensor of {n} elements on {dev}, "
                         f"got {t.dtype} {tuple(t.shape)} on {t.device}")


def _check_workspace(ws, dev):
    import torch

    if ws.device != dev or ws.dtype != torch.uint8 or not ws.is_contiguous():
        raise ValueError(f"workspace must be a contiguous uint8 tensor on {dev}, got {ws.dtype} on {ws.device}")


def workspace_for(img):
    import torch

    b, d = img.shape
    n = infcl_workspace_size(b, d, _dtype_code(img))
    return torch.empty(max(n, 256), dtype=torch.uint8, device=img.device)


def clip_loss_fwd(img, txt, scale, workspace=None) -> dict:
    import torch

    _validate(img, txt, scale)
    b, _ = img.shape
    dev = img.device
    out = {
        "loss": torch.empty((), dtype=torch.float32, device=dev),
        "loss64": torch.empty((), dtype=torch.float64, device=dev),
        "lse_r": torch.empty(b, dtype=torch.float32, device=dev),
        "lse_c": torch.empty(b, dtype=torch.float32, device=dev),
        "aux": torch.empty(3 * b, dtype=torch.float32, device=dev),
    }
    ws = workspace if workspace is not None else workspace_for(img)
    _check_workspace(ws, dev)
    infcl_fwd(img, txt, scale.reshape(()), out["loss"], out["loss64"], out["lse_r"], out["lse_c"], out["aux"], ws)
    out["workspace"] = ws
    return out


def clip_loss_bwd(img, txt, scale, fwd: dict, dloss=None, workspace=None, grad_dtype=None):
    """dimg, dtxt and dscale.  grad_dtype: torch.float32 (default), or the
    inputs' own 16-bit dtype (rounded once from the fp32 accumulators)."""
    import torch

    _validate(img, txt, scale)
    b, d = img.shape
    dev = img.device
    _check_vec(fwd["lse_r"], b, "lse_r", dev)
    _check_vec(fwd["lse_c"], b, "lse_c", dev)
    _check_vec(fwd["aux"], 3 * b, "aux", dev)
    gdt = torch.float32 if grad_dtype is None else grad_dtype
    if gdt not in (torch.float32, img.dtype):
        raise TypeError(f"grad_dtype must be float32 or the inputs' dtype {img.dtype}, got {gdt}")
    dimg = torch.empty((b, d), dtype=gdt, device=img.device)
    dtxt = torch.empty((b, d), dtype=gdt, device=img.device)
    dscale = torch.empty((), dtype=torch.float32, device=img.device)
    ws = workspace if workspace is not None else fwd.get("workspace")
    if ws is None:
        ws = workspace_for(img)
    _check_workspace(ws, dev)
    if dloss is not None:
        if dloss.device != dev or dloss.numel() != 1:
            raise ValueError(f"dloss must be one element on {dev}, got {tuple(dloss.shape)} on {dloss.device}")
        dloss = dloss.reshape(()).to(torch.float32).contiguous()
    infcl_bwd(img, txt, scale.reshape(()), fwd["lse_r"], fwd["lse_c"], fwd["aux"], dloss, dimg, dtxt, dscale, ws)
    return dimg, dtxt, dscale


def _make_function():
    import torch

    class ClipLoss(torch.autograd.Function):
        @staticmethod
        def forward(ctx, img, txt, scale):
            f = clip_loss_fwd(img, txt, scale)
            ctx.save_for_backward(img, txt, scale, f["lse_r"], f["lse_c"], f["aux"])
            ctx.ws = f["workspace"]
            return f["loss"]

        @staticmethod
        def backward(ctx, dloss):
            img, txt, scale, lse_r, lse_c, aux = ctx.saved_tensors
            fwd = {"lse_r": lse_r, "lse_c": lse_c, "aux": aux}
            # gradients in the inputs' dtype straight from the kernels (one
            # rounding of the fp32 accumulators, as a cast would do)
            dimg, dtxt, dscale = clip_loss_bwd(img, txt, scale, fwd, dloss=dloss, workspace=ctx.ws,
                                               grad_dtype=img.dtype)
            return dimg, dtxt, dscale.reshape(scale.shape)

    return ClipLoss


_ClipLoss = None


def clip_loss(img, txt, scale):
    """Symmetric InfoNCE loss of img/txt [b, d] with logit scale `scale` (float32, 1 element)."""
    global _ClipLoss
    if _ClipLoss is None:
        _ClipLoss = _make_function()
    return _ClipLoss.apply(img, txt, scale)
