"""Thin Python binding of libot's C ABI (include/ot.h).

Argument marshalling only: torch tensors in, device pointers and the current
HIP stream out to the library; every computation runs in libot's kernels.
The names match the C entry points.  Outputs are caller-allocated, as in C.

The library is loaded on first use: ``libot.so`` next to this file, or the
build named by the environment variable OT_LIBRARY (e.g. a sanitizer build).
If it has not been built the first call raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import re

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("OT_LIBRARY") or os.path.join(HERE, "libot.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "ot.h")

OT_OK, OT_EINVAL, OT_ESHAPE, OT_ERANGE, OT_ENONFINITE, OT_EHIP, OT_ENOSCRATCH = range(7)

_lib = None


class OTError(RuntimeError):
    """A nonzero ot_status from libot."""

    def __init__(self, code: int, where: str):
        self.code = int(code)
        super().__init__(f"{where}: {ot_strerror(code)} (status {code})")


def lib() -> ctypes.CDLL:
    """The loaded libot (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i64, c_int = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        L.ot_strerror.restype = ctypes.c_char_p
        L.ot_strerror.argtypes = [c_int]
        L.ot_abi_version.restype = c_int
        L.ot_abi_version.argtypes = []
        L.ot_build_info.restype = ctypes.c_char_p
        L.ot_build_info.argtypes = []
        L.ot_calibrate.restype = c_int
        L.ot_calibrate.argtypes = [vp, i64, i64, c_int, c_int, vp, vp, vp, vp, vp]
        L.ot_fold_weights.restype = c_int
        L.ot_fold_weights.argtypes = [vp, vp, i64, i64, c_int, vp, vp, vp, vp, vp, vp]
        L.ot_quantize_act.restype = c_int
        L.ot_quantize_act.argtypes = [vp, i64, i64, c_int, vp, vp, vp, vp]
        L.ot_ln_quantize_act.restype = c_int
        L.ot_ln_quantize_act.argtypes = [vp, i64, i64, vp, vp, ctypes.c_float, c_int, vp, vp, vp,
                                         vp]
        L.ot_quantize_act_per_token.restype = c_int
        L.ot_quantize_act_per_token.argtypes = [vp, i64, i64, c_int, vp, vp, vp]
        L.ot_fold_weights_per_token.restype = c_int
        L.ot_fold_weights_per_token.argtypes = [vp, vp, vp, i64, i64, c_int, vp, vp, vp, vp]
        L.ot_qlinear_per_token.restype = c_int
        L.ot_qlinear_per_token.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, c_int, c_int, vp, vp,
                                           vp, vp]
        L.ot_scales_from_minmax.restype = c_int
        L.ot_scales_from_minmax.argtypes = [vp, i64, c_int, c_int, vp, vp, vp, vp]
        L.ot_fold_weights_asym.restype = c_int
        L.ot_fold_weights_asym.argtypes = [vp, vp, i64, i64, c_int, vp, vp, vp, vp, vp, vp, vp]
        L.ot_qlinear_asym.restype = c_int
        L.ot_qlinear_asym.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, c_int, c_int, vp, vp, vp,
                                      vp]
        L.ot_qlinear.restype = c_int
        L.ot_qlinear.argtypes = [vp, vp, vp, vp, i64, i64, i64, c_int, c_int, vp, vp, vp, vp]
        L.ot_qlinear_noalloc.restype = c_int
        L.ot_qlinear_noalloc.argtypes = [vp, vp, vp, vp, i64, i64, i64, c_int, c_int, vp, vp, vp]
        L.ot_qlinear_workspace_size.restype = ctypes.c_size_t
        L.ot_qlinear_workspace_size.argtypes = [i64, i64, i64]
        L.ot_qlinear_plan.restype = c_int
        L.ot_qlinear_plan.argtypes = [i64, i64, i64, c_int, c_int, ctypes.c_char_p, ctypes.c_size_t]
        L.ot_packed_weights_size.restype = ctypes.c_size_t
        L.ot_packed_weights_size.argtypes = [i64, i64]
        L.ot_pack_weights.restype = c_int
        L.ot_pack_weights.argtypes = [vp, i64, i64, vp, vp]
        L.ot_qlinear_packed.restype = c_int
        L.ot_qlinear_packed.argtypes = [vp, vp, vp, vp, i64, i64, i64, c_int, c_int, vp, vp, vp, vp]
        _lib = L
    return _lib


def declared_symbols() -> list:
    """Entry points declared in include/ot.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(ot_\w+)\s*\(", text, re.M)))


def ot_strerror(code: int) -> str:
    return lib().ot_strerror(int(code)).decode()


def ot_abi_version() -> int:
    return int(lib().ot_abi_version())


def ot_build_info() -> str:
    return lib().ot_build_info().decode()


def build_info() -> dict:
    """ot_build_info()'s fields, the loaded library's path, and whether its
    sources_sha256 is that of the sources in this tree now (False means the
    library was built from other sources: rebuild it)."""
    from . import build_lib
    info = dict(f.split("=", 1) for f in ot_build_info().split(";") if "=" in f)
    info["library"] = os.path.relpath(LIB_PATH, os.path.dirname(HERE))
    info["matches_sources"] = info.get("sources_sha256") == build_lib.source_digest()
    return info


def _check(rc: int, where: str) -> None:
    if rc != OT_OK:
        raise OTError(rc, where)


def _dev(t, dtype, name, shape=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t.data_ptr()


def _dev_ws(workspace, M, N, K):
    """Device pointer of an optional workspace, checked against the bytes the
    library asks for at these sizes (the C ABI cannot see its size)."""
    if workspace is None:
        return None
    ptr = _dev(workspace, torch.uint8, "workspace")
    need = ot_qlinear_workspace_size(M, N, K)
    if workspace.numel() < need:
        raise ValueError(f"workspace holds {workspace.numel()} bytes, the call needs {need}")
    return ptr


# The current device's current stream as a raw handle: torch's C accessors
# take ~0.2 us against ~2.7 us for building a torch.cuda.Stream object per
# call (measured on MI355X); the public call remains the fallback.
_raw_current_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_current_device = getattr(torch._C, "_cuda_getDevice", None)


def _stream(stream):
    if stream is None:
        if _raw_current_stream is not None and _current_device is not None:
            return _raw_current_stream(_current_device())
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def ot_calibrate(x, a_bits, first, minmax, z, s, inv_s, stream=None):
    """Folds the calibration batch x [rows, K] fp16 into minmax [2K] and
    rewrites z, s, inv_s [K] (fp32).  Synchronous."""
    rows, K = x.shape
    rc = lib().ot_calibrate(_dev(x, torch.float16, "x"), rows, K, int(a_bits), int(bool(first)),
                            _dev(minmax, torch.float32, "minmax", (2 * K,)),
                            _dev(z, torch.float32, "z", (K,)), _dev(s, torch.float32, "s", (K,)),
                            _dev(inv_s, torch.float32, "inv_s", (K,)), _stream(stream))
    _check(rc, "ot_calibrate")


def ot_fold_weights(W, b, w_bits, z, s, Wq, sW, bprime, stream=None):
    """W [N, K] fp16, b [N] fp16 or None -> Wq [N, K] int8, sW, bprime [N]
    fp32.  Synchronous."""
    N, K = W.shape
    rc = lib().ot_fold_weights(_dev(W, torch.float16, "W"), _dev(b, torch.float16, "b", (N,)),
                               N, K, int(w_bits), _dev(z, torch.float32, "z", (K,)),
                               _dev(s, torch.float32, "s", (K,)),
                               _dev(Wq, torch.int8, "Wq", (N, K)),
                               _dev(sW, torch.float32, "sW", (N,)),
                               _dev(bprime, torch.float32, "bprime", (N,)), _stream(stream))
    _check(rc, "ot_fold_weights")


def ot_quantize_act(x, a_bits, z, inv_s, Xq, stream=None):
    """x [M, K] fp16 -> Xq [M, K] int8.  Asynchronous."""
    M, K = x.shape
    rc = lib().ot_quantize_act(_dev(x, torch.float16, "x"), M, K, int(a_bits),
                               _dev(z, torch.float32, "z", (K,)),
                               _dev(inv_s, torch.float32, "inv_s", (K,)),
                               _dev(Xq, torch.int8, "Xq", (M, K)), _stream(stream))
    _check(rc, "ot_quantize_act")


def ot_ln_quantize_act(h, gamma, beta, eps, a_bits, z, inv_s, Xq, stream=None):
    """h [M, K] fp16 LayerNorm input -> Xq [M, K] int8 codes of the symmetrized
    LayerNorm output.  Asynchronous."""
    M, K = h.shape
    rc = lib().ot_ln_quantize_act(_dev(h, torch.float16, "h"), M, K,
                                  _dev(gamma, torch.float16, "gamma", (K,)),
                                  _dev(beta, torch.float16, "beta", (K,)), float(eps), int(a_bits),
                                  _dev(z, torch.float32, "z", (K,)),
                                  _dev(inv_s, torch.float32, "inv_s", (K,)),
                                  _dev(Xq, torch.int8, "Xq", (M, K)), _stream(stream))
    _check(rc, "ot_ln_quantize_act")


def ot_qlinear(Xq, Wq, sW, bprime, a_bits, w_bits, Y, acc_out=None, workspace=None, stream=None):
    """Xq [M, K] int8, Wq [N, K] int8 -> Y [M, N] fp16 (and acc_out [M, N]
    int32 if given).  Asynchronous."""
    M, K = Xq.shape
    N = Wq.shape[0]
    if Wq.shape[1] != K:
        raise ValueError("Xq and Wq disagree on K")
    ws = _dev_ws(workspace, M, N, K)
    rc = lib().ot_qlinear(_dev(Xq, torch.int8, "Xq"), _dev(Wq, torch.int8, "Wq"),
                          _dev(sW, torch.float32, "sW", (N,)),
                          _dev(bprime, torch.float32, "bprime", (N,)), M, N, K, int(a_bits),
                          int(w_bits), _dev(Y, torch.float16, "Y", (M, N)),
                          _dev(acc_out, torch.int32, "acc_out", (M, N)), ws, _stream(stream))
    _check(rc, "ot_qlinear")


def ot_qlinear_noalloc(Xq, Wq, sW, bprime, a_bits, w_bits, Y, acc_out=None, stream=None):
    """ot_qlinear with the split-K scratch in the library's fixed device
    array (no workspace, no allocation).  Asynchronous."""
    M, K = Xq.shape
    N = Wq.shape[0]
    if Wq.shape[1] != K:
        raise ValueError("Xq and Wq disagree on K")
    rc = lib().ot_qlinear_noalloc(_dev(Xq, torch.int8, "Xq"), _dev(Wq, torch.int8, "Wq"),
                                  _dev(sW, torch.float32, "sW", (N,)),
                                  _dev(bprime, torch.float32, "bprime", (N,)), M, N, K,
                                  int(a_bits), int(w_bits), _dev(Y, torch.float16, "Y", (M, N)),
                                  _dev(acc_out, torch.int32, "acc_out", (M, N)), _stream(stream))
    _check(rc, "ot_qlinear_noalloc")


def ot_qlinear_workspace_size(M: int, N: int, K: int) -> int:
    return int(lib().ot_qlinear_workspace_size(M, N, K))


def ot_qlinear_plan(M: int, N: int, K: int, packed=False, with_workspace=False) -> str:
    """The kernel configuration the quantized-linear calls launch for these
    sizes on the current device (text; no device work)."""
    buf = ctypes.create_string_buffer(96)
    _check(lib().ot_qlinear_plan(M, N, K, int(bool(packed)), int(bool(with_workspace)), buf,
                                 len(buf)), "ot_qlinear_plan")
    return buf.value.decode()


def ot_packed_weights_size(N: int, K: int) -> int:
    return int(lib().ot_packed_weights_size(N, K))


def ot_pack_weights(Wq, Wp, stream=None):
    """Wq [N, K] int8 -> Wp (ot_packed_weights_size(N, K) bytes, int8), the
    decode micro-tile layout.  Asynchronous."""
    N, K = Wq.shape
    rc = lib().ot_pack_weights(_dev(Wq, torch.int8, "Wq"), N, K,
                               _dev(Wp, torch.int8, "Wp", (ot_packed_weights_size(N, K),)),
                               _stream(stream))
    _check(rc, "ot_pack_weights")


def ot_qlinear_packed(Xq, Wp, N, sW, bprime, a_bits, w_bits, Y, acc_out=None, workspace=None,
                      stream=None):
    """ot_qlinear for M <= 64 with packed weights Wp (of N output channels)
    from ot_pack_weights.  Asynchronous."""
    M, K = Xq.shape
    rc = lib().ot_qlinear_packed(_dev(Xq, torch.int8, "Xq"),
                                 _dev(Wp, torch.int8, "Wp", (ot_packed_weights_size(N, K),)),
                                 _dev(sW, torch.float32, "sW", (N,)),
                                 _dev(bprime, torch.float32, "bprime", (N,)), M, N, K,
                                 int(a_bits), int(w_bits), _dev(Y, torch.float16, "Y", (M, N)),
                                 _dev(acc_out, torch.int32, "acc_out", (M, N)),
                                 _dev_ws(workspace, M, N, K), _stream(stream))
    _check(rc, "ot_qlinear_packed")


# ---------------------------------------------------------------------------
# Conveniences that allocate outputs with torch and call the entry points.
# ---------------------------------------------------------------------------
def ot_scales_from_minmax(minmax, a_bits, symmetrize, z, s, inv_s, stream=None):
    """minmax [2K] fp32 -> z, s, inv_s [K] fp32 for a_bits, with or without
    symmetrization.  Asynchronous."""
    K = minmax.shape[0] // 2
    rc = lib().ot_scales_from_minmax(_dev(minmax, torch.float32, "minmax", (2 * K,)), K,
                                     int(a_bits), 1 if symmetrize else 0,
                                     _dev(z, torch.float32, "z", (K,)),
                                     _dev(s, torch.float32, "s", (K,)),
                                     _dev(inv_s, torch.float32, "inv_s", (K,)), _stream(stream))
    _check(rc, "ot_scales_from_minmax")


def scales_from_minmax(minmax, a_bits, symmetrize=True):
    K = minmax.shape[0] // 2
    z, s, inv_s = (torch.empty(K, dtype=torch.float32, device=minmax.device) for _ in range(3))
    ot_scales_from_minmax(minmax, a_bits, symmetrize, z, s, inv_s)
    return z, s, inv_s


def ot_quantize_act_per_token(x, a_bits, Xq, sX, stream=None):
    """x [M, K] fp16 -> Xq [M, K] int8 and per-token scales sX [M] fp32
    (Eq. (c)).  Asynchronous."""
    M, K = x.shape
    rc = lib().ot_quantize_act_per_token(_dev(x, torch.float16, "x"), M, K, int(a_bits),
                                         _dev(Xq, torch.int8, "Xq", (M, K)),
                                         _dev(sX, torch.float32, "sX", (M,)), _stream(stream))
    _check(rc, "ot_quantize_act_per_token")


def ot_fold_weights_per_token(W, b, zres, w_bits, Wq, sW, bprime, stream=None):
    """W [N, K] fp16, b [N] fp16 or None, zres [N] fp32 or None -> Wq, sW and
    bprime = b + zres (Eq. (h)).  Synchronous."""
    N, K = W.shape
    rc = lib().ot_fold_weights_per_token(_dev(W, torch.float16, "W"),
                                         _dev(b, torch.float16, "b", (N,)),
                                         _dev(zres, torch.float32, "zres", (N,)), N, K,
                                         int(w_bits), _dev(Wq, torch.int8, "Wq", (N, K)),
                                         _dev(sW, torch.float32, "sW", (N,)),
                                         _dev(bprime, torch.float32, "bprime", (N,)),
                                         _stream(stream))
    _check(rc, "ot_fold_weights_per_token")


def ot_qlinear_per_token(Xq, Wq, sX, sW, bprime, a_bits, w_bits, Y, acc_out=None, workspace=None,
                         stream=None):
    """Eq. (c): Xq [M, K], Wq [N, K] int8, sX [M], sW [N], bprime [N] fp32 ->
    Y [M, N] fp16 (and acc_out [M, N] int32 if given).  Asynchronous."""
    M, K = Xq.shape
    N = Wq.shape[0]
    if Wq.shape[1] != K:
        raise ValueError("Xq and Wq disagree on K")
    rc = lib().ot_qlinear_per_token(_dev(Xq, torch.int8, "Xq"), _dev(Wq, torch.int8, "Wq"),
                                    _dev(sX, torch.float32, "sX", (M,)),
                                    _dev(sW, torch.float32, "sW", (N,)),
                                    _dev(bprime, torch.float32, "bprime", (N,)), M, N, K,
                                    int(a_bits), int(w_bits),
                                    _dev(Y, torch.float16, "Y", (M, N)),
                                    _dev(acc_out, torch.int32, "acc_out", (M, N)),
                                    _dev_ws(workspace, M, N, K), _stream(stream))
    _check(rc, "ot_qlinear_per_token")


def ot_fold_weights_asym(W, b, w_bits, z, s, Wq, sW, zW, bprime, stream=None):
    """Asymmetric ("Int8") weights: W [N, K] fp16, b [N] fp16 or None ->
    shifted codes Wq [N, K] int8, sW [N] fp32, shifted zero points zW [N]
    int32, bprime [N] fp32.  Synchronous."""
    N, K = W.shape
    rc = lib().ot_fold_weights_asym(_dev(W, torch.float16, "W"), _dev(b, torch.float16, "b", (N,)),
                                    N, K, int(w_bits), _dev(z, torch.float32, "z", (K,)),
                                    _dev(s, torch.float32, "s", (K,)),
                                    _dev(Wq, torch.int8, "Wq", (N, K)),
                                    _dev(sW, torch.float32, "sW", (N,)),
                                    _dev(zW, torch.int32, "zW", (N,)),
                                    _dev(bprime, torch.float32, "bprime", (N,)), _stream(stream))
    _check(rc, "ot_fold_weights_asym")


def ot_qlinear_asym(Xq, Wq, sW, zW, bprime, a_bits, w_bits, Y, acc_out=None, workspace=None,
                    stream=None):
    """Quantized linear with asymmetric weights: acc = Xq (Wq - zW)^T, then
    the per-channel epilogue.  Asynchronous."""
    M, K = Xq.shape
    N = Wq.shape[0]
    if Wq.shape[1] != K:
        raise ValueError("Xq and Wq disagree on K")
    rc = lib().ot_qlinear_asym(_dev(Xq, torch.int8, "Xq"), _dev(Wq, torch.int8, "Wq"),
                               _dev(sW, torch.float32, "sW", (N,)),
                               _dev(zW, torch.int32, "zW", (N,)),
                               _dev(bprime, torch.float32, "bprime", (N,)), M, N, K, int(a_bits),
                               int(w_bits), _dev(Y, torch.float16, "Y", (M, N)),
                               _dev(acc_out, torch.int32, "acc_out", (M, N)),
                               _dev_ws(workspace, M, N, K), _stream(stream))
    _check(rc, "ot_qlinear_asym")


def calibrate(batches, a_bits, device="cuda"):
    """Runs ot_calibrate over an iterable of fp16 [rows, K] batches (host
    numpy or device tensors).  Returns (minmax, z, s, inv_s) on the GPU."""
    minmax = z = s = inv_s = None
    first = True
    for x in batches:
        if not isinstance(x, torch.Tensor):
            x = torch.from_numpy(x)
        x = x.to(device)
        K = x.shape[1]
        if minmax is None:
            minmax = torch.empty(2 * K, dtype=torch.float32, device=device)
            z, s, inv_s = (torch.empty(K, dtype=torch.float32, device=device) for _ in range(3))
        ot_calibrate(x, a_bits, first, minmax, z, s, inv_s)
        first = False
    if minmax is None:
        raise ValueError("no calibration batches")
    return minmax, z, s, inv_s


def fold_weights(W, b, w_bits, z, s):
    """Allocating wrapper of ot_fold_weights; returns (Wq, sW, bprime)."""
    N, K = W.shape
    Wq = torch.empty((N, K), dtype=torch.int8, device=W.device)
    sW = torch.empty(N, dtype=torch.float32, device=W.device)
    bprime = torch.empty(N, dtype=torch.float32, device=W.device)
    ot_fold_weights(W, b, w_bits, z, s, Wq, sW, bprime)
    return Wq, sW, bprime


def quantize_act(x, a_bits, z, inv_s):
    Xq = torch.empty(x.shape, dtype=torch.int8, device=x.device)
    ot_quantize_act(x, a_bits, z, inv_s, Xq)
    return Xq


def ln_quantize_act(h, gamma, beta, eps, a_bits, z, inv_s):
    Xq = torch.empty(h.shape, dtype=torch.int8, device=h.device)
    ot_ln_quantize_act(h, gamma, beta, eps, a_bits, z, inv_s, Xq)
    return Xq


def workspace_for(M: int, N: int, K: int, device=None):
    """A scratch buffer of ot_qlinear_workspace_size(M, N, K) bytes for the
    quantized-linear calls, or None when they use none at these sizes."""
    n = ot_qlinear_workspace_size(M, N, K)
    return torch.empty(n, dtype=torch.uint8, device=device or "cuda") if n else None


def _ws(workspace, Xq, Wq):
    """workspace=True allocates one for the call's sizes; a tensor is used as given."""
    if workspace is True:
        return workspace_for(Xq.shape[0], Wq.shape[0], Xq.shape[1], Xq.device)
    return None if workspace is None or workspace is False else workspace


def qlinear(Xq, Wq, sW, bprime, a_bits, w_bits, want_acc=False, workspace=None):
    M, N = Xq.shape[0], Wq.shape[0]
    Y = torch.empty((M, N), dtype=torch.float16, device=Xq.device)
    acc = torch.empty((M, N), dtype=torch.int32, device=Xq.device) if want_acc else None
    ot_qlinear(Xq, Wq, sW, bprime, a_bits, w_bits, Y, acc, _ws(workspace, Xq, Wq))
    return (Y, acc) if want_acc else Y


def pack_weights(Wq):
    N, K = Wq.shape
    Wp = torch.empty(ot_packed_weights_size(N, K), dtype=torch.int8, device=Wq.device)
    ot_pack_weights(Wq, Wp)
    return Wp


def qlinear_packed(Xq, Wp, N, sW, bprime, a_bits, w_bits, want_acc=False, workspace=None):
    M, K = Xq.shape
    Y = torch.empty((M, N), dtype=torch.float16, device=Xq.device)
    acc = torch.empty((M, N), dtype=torch.int32, device=Xq.device) if want_acc else None
    ws = workspace_for(M, N, K, Xq.device) if workspace is True else (
        None if workspace is None or workspace is False else workspace)
    ot_qlinear_packed(Xq, Wp, N, sW, bprime, a_bits, w_bits, Y, acc, ws)
    return (Y, acc) if want_acc else Y


def quantize_act_per_token(x, a_bits):
    M = x.shape[0]
    Xq = torch.empty(x.shape, dtype=torch.int8, device=x.device)
    sX = torch.empty(M, dtype=torch.float32, device=x.device)
    ot_quantize_act_per_token(x, a_bits, Xq, sX)
    return Xq, sX


def fold_weights_per_token(W, b, zres, w_bits):
    N, K = W.shape
    Wq = torch.empty((N, K), dtype=torch.int8, device=W.device)
    sW = torch.empty(N, dtype=torch.float32, device=W.device)
    bprime = torch.empty(N, dtype=torch.float32, device=W.device)
    ot_fold_weights_per_token(W, b, zres, w_bits, Wq, sW, bprime)
    return Wq, sW, bprime


def qlinear_per_token(Xq, Wq, sX, sW, bprime, a_bits, w_bits, want_acc=False, workspace=None):
    M, N = Xq.shape[0], Wq.shape[0]
    Y = torch.empty((M, N), dtype=torch.float16, device=Xq.device)
    acc = torch.empty((M, N), dtype=torch.int32, device=Xq.device) if want_acc else None
    ot_qlinear_per_token(Xq, Wq, sX, sW, bprime, a_bits, w_bits, Y, acc, _ws(workspace, Xq, Wq))
    return (Y, acc) if want_acc else Y


def fold_weights_asym(W, b, w_bits, z, s):
    N, K = W.shape
    Wq = torch.empty((N, K), dtype=torch.int8, device=W.device)
    sW = torch.empty(N, dtype=torch.float32, device=W.device)
    zW = torch.empty(N, dtype=torch.int32, device=W.device)
    bprime = torch.empty(N, dtype=torch.float32, device=W.device)
    ot_fold_weights_asym(W, b, w_bits, z, s, Wq, sW, zW, bprime)
    return Wq, sW, zW, bprime


def qlinear_asym(Xq, Wq, sW, zW, bprime, a_bits, w_bits, want_acc=False, workspace=None):
    M, N = Xq.shape[0], Wq.shape[0]
    Y = torch.empty((M, N), dtype=torch.float16, device=Xq.device)
    acc = torch.empty((M, N), dtype=torch.int32, device=Xq.device) if want_acc else None
    ot_qlinear_asym(Xq, Wq, sW, zW, bprime, a_bits, w_bits, Y, acc, _ws(workspace, Xq, Wq))
    return (Y, acc) if want_acc else Y
