"""ctypes binding of libquasar.so (the C ABI in include/quasar.h).

Argument marshalling only: every step of the reconstruction runs in the HIP
kernels behind ``quasar_reconstruct``.  Tensors are torch tensors on the GPU
(torch supplies device memory and the current stream); there is no CPU path,
and a missing library raises instead of falling back.

The functions named ``quasar_*`` (``EXPORTS``) mirror the C entry points one
to one; ``reconstruct``, ``reconstruct_batch``, ``adamw_reconstruct``,
``adamw_reconstruct_batch`` and ``absmax_batch`` are convenience wrappers that
allocate the outputs and call them.
"""
from __future__ import annotations

import ctypes as C
import os
import threading

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libquasar.so")

OK, ERR_ARG, ERR_SHAPE, ERR_ALIGN, ERR_FORMAT, ERR_WORKSPACE, ERR_DEVICE = 0, -1, -2, -3, -4, -5, -6
F32, BF16, F16 = 0, 1, 2
INT, NVFP4, RUBIN_INT3, INT_SYM = 0, 1, 2, 3
WEIGHT_H, WEIGHT_H2, WEIGHT_NONE = 0, 1, 2
WEIGHTINGS = {"h": WEIGHT_H, "h2": WEIGHT_H2, "none": WEIGHT_NONE}
PARAM_DTYPES = {"fp32": F32, "fp16": F16, "bf16": BF16}
MAX_CLIPS = 16

EXPORTS = ("quasar_reconstruct", "quasar_reconstruct_noalloc", "quasar_absmax", "quasar_check", "quasar_adamw_reconstruct", "quasar_adamw_check",
           "quasar_reconstruct_batch", "quasar_batch_check", "quasar_absmax_batch", "quasar_absmax_batch_check",
           "quasar_adamw_reconstruct_batch", "quasar_adamw_batch_check",
           "quasar_num_groups", "quasar_int_path", "quasar_codes_bytes",
           "quasar_workspace_bytes", "quasar_status_string", "quasar_version")
MAX_BATCH = 16


class QuasarError(RuntimeError):
    def __init__(self, status: int, where: str = "quasar_reconstruct"):
        self.status = status
        super().__init__(f"{where}: status {status} ({quasar_status_string(status)})")


class Desc(C.Structure):
    _fields_ = [("rows", C.c_int64), ("cols", C.c_int64), ("w_dtype", C.c_int32), ("format", C.c_int32),
                ("bits", C.c_int32), ("group", C.c_int32), ("clip_ratios", C.POINTER(C.c_float)),
                ("n_clips", C.c_int32), ("g_dtype", C.c_int32), ("beta2", C.c_float),
                ("weighting", C.c_int32), ("param_dtype", C.c_int32)]


class Matrix(C.Structure):
    """quasar_matrix: one matrix of a batched call."""
    _fields_ = [("rows", C.c_int64), ("cols", C.c_int64), ("W", C.c_void_p), ("v", C.c_void_p), ("g", C.c_void_p),
                ("codes", C.c_void_p), ("scales", C.c_void_p), ("zeros", C.c_void_p), ("r", C.c_void_p),
                ("best_clip", C.c_void_p), ("err", C.c_void_p), ("tensor_scale", C.c_void_p),
                ("tensor_amax", C.c_void_p)]


class AdamWMatrix(C.Structure):
    """quasar_adamw_matrix: one matrix of a batched fused AdamW call."""
    _fields_ = [("rows", C.c_int64), ("cols", C.c_int64), ("W", C.c_void_p), ("m", C.c_void_p), ("v", C.c_void_p),
                ("g", C.c_void_p), ("codes", C.c_void_p), ("scales", C.c_void_p), ("zeros", C.c_void_p),
                ("r", C.c_void_p), ("best_clip", C.c_void_p), ("err", C.c_void_p), ("tensor_scale", C.c_void_p),
                ("tensor_amax", C.c_void_p), ("amax_out", C.c_void_p)]


class AdamW(C.Structure):
    """quasar_adamw: the hyper-parameters of one AdamW step."""
    _fields_ = [("lr", C.c_float), ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float),
                ("weight_decay", C.c_float), ("step", C.c_int64)]


_lib = None
_lock = threading.Lock()


def lib():
    """Open libquasar.so (built in-tree by ``paper_2608_13966_amd.build``)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_13966_amd.build` "
                                   "(there is no fallback path)")
            L = C.CDLL(LIB_PATH)
            vp, dp = C.c_void_p, C.POINTER(Desc)
            L.quasar_reconstruct.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, C.c_size_t, vp]
            L.quasar_reconstruct.restype = C.c_int
            L.quasar_reconstruct_noalloc.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
            L.quasar_reconstruct_noalloc.restype = C.c_int
            L.quasar_absmax.argtypes = [dp, vp, vp, vp]
            L.quasar_absmax.restype = C.c_int
            L.quasar_check.argtypes = [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, C.c_size_t]
            L.quasar_check.restype = C.c_int
            ap = C.POINTER(AdamW)
            L.quasar_adamw_reconstruct.argtypes = [dp, ap, vp, vp, vp, vp, vp, vp, vp, vp, C.c_int, vp, vp, vp, vp,
                                                   vp, vp]
            L.quasar_adamw_reconstruct.restype = C.c_int
            L.quasar_adamw_check.argtypes = [dp, ap, vp, vp, vp, vp, vp, vp, vp, vp, C.c_int, vp, vp, vp, vp, vp]
            L.quasar_adamw_check.restype = C.c_int
            mp = C.POINTER(Matrix)
            L.quasar_reconstruct_batch.argtypes = [dp, mp, C.c_int, vp]
            L.quasar_reconstruct_batch.restype = C.c_int
            L.quasar_batch_check.argtypes = [dp, mp, C.c_int]
            L.quasar_batch_check.restype = C.c_int
            amp = C.POINTER(AdamWMatrix)
            L.quasar_adamw_reconstruct_batch.argtypes = [dp, ap, amp, C.c_int, C.c_int, vp]
            L.quasar_adamw_reconstruct_batch.restype = C.c_int
            L.quasar_adamw_batch_check.argtypes = [dp, ap, amp, C.c_int, C.c_int]
            L.quasar_adamw_batch_check.restype = C.c_int
            pp = C.POINTER(vp)
            L.quasar_absmax_batch.argtypes = [dp, mp, C.c_int, pp, vp]
            L.quasar_absmax_batch.restype = C.c_int
            L.quasar_absmax_batch_check.argtypes = [dp, mp, C.c_int, pp]
            L.quasar_absmax_batch_check.restype = C.c_int
            L.quasar_num_groups.argtypes = [dp]
            L.quasar_num_groups.restype = C.c_int64
            L.quasar_int_path.argtypes = [dp]
            L.quasar_int_path.restype = C.c_int
            L.quasar_codes_bytes.argtypes = [dp]
            L.quasar_codes_bytes.restype = C.c_size_t
            L.quasar_workspace_bytes.argtypes = [dp, C.c_int]
            L.quasar_workspace_bytes.restype = C.c_size_t
            L.quasar_status_string.argtypes = [C.c_int]
            L.quasar_status_string.restype = C.c_char_p
            L.quasar_version.argtypes = []
            L.quasar_version.restype = C.c_char_p
            _lib = L
    return _lib


class Descriptor:
    """A quasar_desc plus the host clip array it points to (kept alive here)."""

    def __init__(self, rows, cols, *, fmt="int", bits=4, group=128, clips=(1.0,), w_dtype=BF16,
                 g_dtype=BF16, beta2=0.999, weighting="h", param_dtype="fp32"):
        self.clips = np.ascontiguousarray(np.asarray(clips, dtype=np.float32))
        nv = fmt == "nvfp4"
        wt = WEIGHTINGS[weighting] if isinstance(weighting, str) else int(weighting)
        pd = PARAM_DTYPES[param_dtype] if isinstance(param_dtype, str) else int(param_dtype)
        if fmt == "rubin":
            form, bits, group = RUBIN_INT3, 3, 512
        elif fmt == "int_sym":
            form, bits, group = INT_SYM, int(bits), int(group)
        else:
            form, bits, group = (NVFP4, 4, 16) if nv else (INT, int(bits), int(group))
        self.desc = Desc(int(rows), int(cols), int(w_dtype), form, bits, group,
                         self.clips.ctypes.data_as(C.POINTER(C.c_float)), int(self.clips.size), int(g_dtype),
                         float(beta2), wt, pd)

    @property
    def ref(self):
        return C.byref(self.desc)


def _p(x):
    """Device pointer of a tensor (or raw int / None)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def quasar_reconstruct(d: Descriptor, W, v, g, codes, scales, zeros, r, best_clip, err, tensor_scale,
                       tensor_amax, workspace, workspace_bytes: int, stream) -> int:
    return lib().quasar_reconstruct(d.ref, _p(W), _p(v), _p(g), _p(codes), _p(scales), _p(zeros), _p(r),
                                    _p(best_clip), _p(err), _p(tensor_scale), _p(tensor_amax), _p(workspace),
                                    int(workspace_bytes), stream)


def quasar_reconstruct_noalloc(d: Descriptor, W, v, g, codes, scales, zeros, r, best_clip, err, tensor_scale,
                               tensor_amax, stream) -> int:
    return lib().quasar_reconstruct_noalloc(d.ref, _p(W), _p(v), _p(g), _p(codes), _p(scales), _p(zeros), _p(r),
                                            _p(best_clip), _p(err), _p(tensor_scale), _p(tensor_amax), stream)


def quasar_absmax(d: Descriptor, W, amax_out, stream) -> int:
    return lib().quasar_absmax(d.ref, _p(W), _p(amax_out), stream)


def quasar_check(d: Descriptor, W, v, g, codes, scales, zeros, r, best_clip, err, tensor_scale, tensor_amax,
                 workspace, workspace_bytes: int) -> int:
    return lib().quasar_check(d.ref, _p(W), _p(v), _p(g), _p(codes), _p(scales), _p(zeros), _p(r),
                              _p(best_clip), _p(err), _p(tensor_scale), _p(tensor_amax), _p(workspace),
                              int(workspace_bytes))


def quasar_adamw_reconstruct(d: Descriptor, opt: AdamW, W, m, v, g, codes, scales, zeros, r, r_dtype: int,
                             best_clip, err, tensor_scale, tensor_amax, amax_out, stream) -> int:
    return lib().quasar_adamw_reconstruct(d.ref, C.byref(opt), _p(W), _p(m), _p(v), _p(g), _p(codes), _p(scales),
                                          _p(zeros), _p(r), int(r_dtype), _p(best_clip), _p(err),
                                          _p(tensor_scale), _p(tensor_amax), _p(amax_out), stream)


def quasar_adamw_check(d: Descriptor, opt: AdamW, W, m, v, g, codes, scales, zeros, r, r_dtype: int, best_clip,
                       err, tensor_scale, tensor_amax, amax_out) -> int:
    return lib().quasar_adamw_check(d.ref, None if opt is None else C.byref(opt), _p(W), _p(m), _p(v), _p(g),
                                    _p(codes), _p(scales), _p(zeros), _p(r), int(r_dtype), _p(best_clip), _p(err),
                                    _p(tensor_scale), _p(tensor_amax), _p(amax_out))


def quasar_adamw_reconstruct_batch(d: Descriptor, opt: AdamW, mats, r_dtype: int, stream) -> int:
    arr = (AdamWMatrix * len(mats))(*mats)
    return lib().quasar_adamw_reconstruct_batch(d.ref, C.byref(opt), arr, len(mats), int(r_dtype), stream)


def quasar_adamw_batch_check(d: Descriptor, opt: AdamW, mats, r_dtype: int) -> int:
    arr = (AdamWMatrix * max(1, len(mats)))(*mats)
    return lib().quasar_adamw_batch_check(d.ref, None if opt is None else C.byref(opt), arr, len(mats),
                                          int(r_dtype))


def matrix(W, v, g, out, tensor_amax=None) -> Matrix:
    """A quasar_matrix for tensors W, v, g (or None) and an alloc_outputs dict."""
    return Matrix(W.shape[0], W.shape[1], _p(W), _p(v), _p(g), _p(out["codes"]), _p(out["scales"]),
                  _p(out["zeros"]), _p(out["r"]), _p(out["best_clip"]), _p(out["err"]), _p(out["tensor_scale"]),
                  _p(tensor_amax))


def quasar_reconstruct_batch(d: Descriptor, mats, stream) -> int:
    arr = (Matrix * len(mats))(*mats)
    return lib().quasar_reconstruct_batch(d.ref, arr, len(mats), stream)


def quasar_batch_check(d: Descriptor, mats) -> int:
    arr = (Matrix * max(1, len(mats)))(*mats)
    return lib().quasar_batch_check(d.ref, arr, len(mats))


def _ptr_array(ts):
    return (C.c_void_p * max(1, len(ts)))(*[_p(t) for t in ts])


def quasar_absmax_batch(d: Descriptor, mats, amax_out, stream) -> int:
    """amax_out: one device fp32 tensor (or None) per matrix."""
    arr = (Matrix * max(1, len(mats)))(*mats)
    return lib().quasar_absmax_batch(d.ref, arr, len(mats), _ptr_array(amax_out), stream)


def quasar_absmax_batch_check(d: Descriptor, mats, amax_out) -> int:
    arr = (Matrix * max(1, len(mats)))(*mats)
    return lib().quasar_absmax_batch_check(d.ref, arr, len(mats), _ptr_array(amax_out))


def quasar_num_groups(d: Descriptor) -> int:
    return int(lib().quasar_num_groups(d.ref))


def quasar_int_path(d: Descriptor) -> int:
    return int(lib().quasar_int_path(d.ref))


def quasar_codes_bytes(d: Descriptor) -> int:
    return int(lib().quasar_codes_bytes(d.ref))


def quasar_workspace_bytes(d: Descriptor, has_tensor_amax: bool) -> int:
    return int(lib().quasar_workspace_bytes(d.ref, int(bool(has_tensor_amax))))


def quasar_status_string(status: int) -> str:
    return lib().quasar_status_string(int(status)).decode()


def quasar_version() -> str:
    return lib().quasar_version().decode()


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _check_same(items, *, slots, what):
    """Argument checks of the batched wrappers, before anything is allocated
    or launched: the C side applies one descriptor (W's dtype, g's dtype and
    whether there is a g) to every matrix and reads each buffer with its
    matrix's shape, so a mismatch would read or write out of bounds.
    ``slots`` names the tensor positions of an item: "W", "v", "m" (fp32,
    W's shape), "g" (W's shape, the first item's dtype, present in all or
    none)."""
    import torch
    if not items:
        raise ValueError(f"{what}: no matrices")
    if len(items) > MAX_BATCH:
        raise ValueError(f"{what}: at most {MAX_BATCH} matrices per call")
    first = dict(zip(slots, items[0]))
    W0, g0 = first["W"], first.get("g")
    for i, it in enumerate(items):
        t = dict(zip(slots, it))
        W = t["W"]
        if W.dim() != 2 or W.dtype != W0.dtype or W.device != W0.device:
            raise ValueError(f"{what}: matrix {i}: W must be 2-D with the first matrix's dtype "
                             f"({W0.dtype}) and device")
        for k in ("v", "m"):
            if k in t and (t[k].dtype != torch.float32 or t[k].shape != W.shape or t[k].device != W.device):
                raise ValueError(f"{what}: matrix {i}: {k} must be fp32 with W's shape and device")
        if "g" in t:
            g = t["g"]
            if (g is None) != (g0 is None):
                raise ValueError(f"{what}: either every matrix has a gradient or none has")
            if g is not None and (g.dtype != g0.dtype or g.shape != W.shape or g.device != W.device):
                raise ValueError(f"{what}: matrix {i}: g must have W's shape and the first gradient's dtype "
                                 f"({g0.dtype})")
        for k in slots:
            x = t.get(k)
            if x is not None and not x.is_contiguous():
                raise ValueError(f"{what}: matrix {i}: {k} must be contiguous")


def alloc_outputs(d: Descriptor, W, *, want_r=True, want_diag=True, has_amax=False):
    """Allocate the output buffers of one call (torch, on W's device)."""
    import torch
    dev = W.device
    ng = quasar_num_groups(d)
    nv = d.desc.format == NVFP4
    out = {"codes": torch.empty(quasar_codes_bytes(d), dtype=torch.uint8, device=dev)}
    if d.desc.format == RUBIN_INT3:   # the codebook: 8 E4M3 bytes per block
        out["scales"] = torch.empty(ng * 8, dtype=torch.uint8, device=dev)
        out["zeros"] = None
        out["tensor_scale"] = None
    elif nv:
        out["scales"] = torch.empty(ng, dtype=torch.uint8, device=dev)
        out["zeros"] = None
        out["tensor_scale"] = torch.empty(4, dtype=torch.float32, device=dev)
    else:
        out["scales"] = torch.empty(ng, dtype=torch.float32, device=dev)
        out["zeros"] = torch.empty(ng, dtype=torch.float32, device=dev)
        out["tensor_scale"] = None
    out["r"] = torch.empty_like(W) if want_r else None
    out["best_clip"] = torch.empty(ng, dtype=torch.uint8, device=dev) if want_diag else None
    out["err"] = torch.empty(ng, dtype=torch.float32, device=dev) if want_diag else None
    wsb = quasar_workspace_bytes(d, has_amax)
    out["workspace"] = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev) if wsb else None
    out["workspace_bytes"] = wsb
    return out


def reconstruct(W, v, g=None, *, fmt="int", bits=4, group=128, clips=(1.0,), beta2=0.999, tensor_amax=None,
                want_r=True, want_diag=True, out=None, stream=None, weighting="h", param_dtype="fp32"):
    """Reconstruct W (torch tensor [rows, cols], fp32 or bf16, on the GPU).

    ``fmt``: "int" (bits, group), "int_sym" (symmetric, bits, group), "nvfp4"
    or "rubin" (Rubin INT3 LUT, blocks
    of 8 rows x 64 columns; ``scales`` is then the 8-byte E4M3 codebook per
    block).

    ``weighting`` ("h", "h2", "none") and ``param_dtype`` ("fp32", "fp16",
    "bf16") select the variants documented at quasar_desc in quasar.h.

    ``v`` (fp32, same shape) is overwritten with the EMA when ``g`` is given.
    Returns the dict of output tensors (see ``alloc_outputs``).  The call is
    asynchronous on ``stream`` (default: torch's current stream).
    """
    import torch
    if W.dim() != 2 or v.shape != W.shape or v.dtype != torch.float32:
        raise ValueError("W must be 2-D and v an fp32 tensor of the same shape")
    for t in (W, v, g):
        if t is not None and not t.is_contiguous():
            raise ValueError("tensors must be contiguous")
    d = Descriptor(W.shape[0], W.shape[1], fmt=fmt, bits=bits, group=group, clips=clips, w_dtype=_dtype_code(W),
                   g_dtype=_dtype_code(g) if g is not None else BF16, beta2=beta2, weighting=weighting,
                   param_dtype=param_dtype)
    if out is None:
        out = alloc_outputs(d, W, want_r=want_r, want_diag=want_diag, has_amax=tensor_amax is not None)
    if stream is None:
        stream = torch.cuda.current_stream(W.device).cuda_stream
    s = quasar_reconstruct(d, W, v, g, out["codes"], out["scales"], out["zeros"], out["r"], out["best_clip"],
                           out["err"], out["tensor_scale"], tensor_amax, out["workspace"], out["workspace_bytes"],
                           stream)
    if s != OK:
        raise QuasarError(s)
    out["desc"] = d
    return out


def adamw_reconstruct(W, m, v, g, *, lr, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, step=1, fmt="int",
                      bits=4, group=128, clips=(1.0,), tensor_amax=None, r_dtype=None, want_r=True, want_diag=True,
                      want_amax_out=False, out=None, stream=None, weighting="h", param_dtype="fp32"):
    """One fused AdamW step + reconstruction (quasar_adamw_reconstruct).

    W (fp32 or bf16), m and v (fp32) are updated in place; g is the gradient
    (fp32 or bf16).  r is bf16 unless r_dtype="fp32" (fp32 W only).  NVFP4
    needs ``tensor_amax`` (device fp32 tensor); ``want_amax_out`` adds
    ``amax_out`` = max |W'| to the returned dict.
    """
    import torch
    for t in (W, m, v, g):
        if not t.is_contiguous() or t.shape != W.shape:
            raise ValueError("W, m, v, g must be contiguous tensors of one shape")
    if m.dtype != torch.float32 or v.dtype != torch.float32:
        raise ValueError("m and v must be fp32")
    d = Descriptor(W.shape[0], W.shape[1], fmt=fmt, bits=bits, group=group, clips=clips, w_dtype=_dtype_code(W),
                   g_dtype=_dtype_code(g), beta2=beta2, weighting=weighting, param_dtype=param_dtype)
    rd = BF16 if r_dtype in (None, "bf16") else F32
    if out is None:
        out = alloc_outputs(d, W, want_r=False, want_diag=want_diag, has_amax=True)
        if want_r:
            out["r"] = torch.empty(W.shape, dtype=torch.bfloat16 if rd == BF16 else torch.float32, device=W.device)
        out["amax_out"] = (torch.empty(4, dtype=torch.float32, device=W.device)
                           if (want_amax_out and fmt == "nvfp4") else None)
    if stream is None:
        stream = torch.cuda.current_stream(W.device).cuda_stream
    opt = AdamW(lr, beta1, beta2, eps, weight_decay, int(step))
    s = quasar_adamw_reconstruct(d, opt, W, m, v, g, out["codes"], out["scales"], out["zeros"], out.get("r"), rd,
                                 out["best_clip"], out["err"], out["tensor_scale"], tensor_amax,
                                 out.get("amax_out"), stream)
    if s != OK:
        raise QuasarError(s, "quasar_adamw_reconstruct")
    out["desc"] = d
    return out


def adamw_reconstruct_batch(items, *, lr, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, step=1,
                            fmt="int", bits=4, group=128, clips=(1.0,), r_dtype=None, want_r=True, want_diag=True,
                            want_amax_out=False, stream=None, weighting="h", param_dtype="fp32"):
    """One batched fused AdamW step + reconstruction
    (quasar_adamw_reconstruct_batch) over ``items``: a list of (W, m, v, g)
    or, for NVFP4, (W, m, v, g, tensor_amax), with one W dtype and one g
    dtype.  W, m, v are updated in place.  Returns one output dict per matrix,
    as adamw_reconstruct()."""
    import torch
    _check_same(items, slots=("W", "m", "v", "g"), what="adamw_reconstruct_batch")
    if items[0][3] is None:
        raise ValueError("adamw_reconstruct_batch: the optimiser step needs a gradient")
    W0, g0 = items[0][0], items[0][3]
    d = Descriptor(W0.shape[0], W0.shape[1], fmt=fmt, bits=bits, group=group, clips=clips,
                   w_dtype=_dtype_code(W0), g_dtype=_dtype_code(g0), beta2=beta2, weighting=weighting,
                   param_dtype=param_dtype)
    rd = BF16 if r_dtype in (None, "bf16") else F32
    outs, mats = [], []
    for it in items:
        W, m, v, g = it[:4]
        amax = it[4] if len(it) > 4 else None
        dd = Descriptor(W.shape[0], W.shape[1], fmt=fmt, bits=bits, group=group, clips=clips,
                        w_dtype=_dtype_code(W), g_dtype=_dtype_code(g), beta2=beta2, weighting=weighting,
                        param_dtype=param_dtype)
        o = alloc_outputs(dd, W, want_r=False, want_diag=want_diag, has_amax=True)
        if want_r:
            o["r"] = torch.empty(W.shape, dtype=torch.bfloat16 if rd == BF16 else torch.float32, device=W.device)
        o["amax_out"] = (torch.empty(4, dtype=torch.float32, device=W.device)
                         if (want_amax_out and fmt == "nvfp4") else None)
        o["desc"] = dd
        outs.append(o)
        mats.append(AdamWMatrix(W.shape[0], W.shape[1], _p(W), _p(m), _p(v), _p(g), _p(o["codes"]),
                                _p(o["scales"]), _p(o["zeros"]), _p(o.get("r")), _p(o["best_clip"]), _p(o["err"]),
                                _p(o["tensor_scale"]), _p(amax), _p(o["amax_out"])))
    if stream is None:
        stream = torch.cuda.current_stream(W0.device).cuda_stream
    opt = AdamW(lr, beta1, beta2, eps, weight_decay, int(step))
    s = quasar_adamw_reconstruct_batch(d, opt, mats, rd, stream)
    if s != OK:
        raise QuasarError(s, "quasar_adamw_reconstruct_batch")
    return outs


def absmax_batch(Ws, *, stream=None):
    """max |W| of each NVFP4 matrix in ``Ws`` (one dtype) in one batched pass
    (quasar_absmax_batch); returns one device fp32 tensor [4] per matrix,
    the value in element 0."""
    import torch
    _check_same([(W,) for W in Ws], slots=("W",), what="absmax_batch")
    W0 = Ws[0]
    d = Descriptor(W0.shape[0], W0.shape[1], fmt="nvfp4", w_dtype=_dtype_code(W0))
    outs = [torch.zeros(4, dtype=torch.float32, device=W0.device) for _ in Ws]
    mats = [Matrix(W.shape[0], W.shape[1], _p(W)) for W in Ws]
    if stream is None:
        stream = torch.cuda.current_stream(W0.device).cuda_stream
    s = quasar_absmax_batch(d, mats, outs, stream)
    if s != OK:
        raise QuasarError(s, "quasar_absmax_batch")
    return outs


def reconstruct_batch(items, *, fmt="int", bits=4, group=128, clips=(1.0,), beta2=0.999, want_r=True,
                      want_diag=True, stream=None, weighting="h", param_dtype="fp32"):
    """One batched call (quasar_reconstruct_batch) over ``items``: a list of
    (W, v, g) or (W, v, g, tensor_amax) with one W dtype and one g dtype (or
    every g None).  NVFP4 items without a tensor_amax get theirs from one
    batched absmax pass first.  Returns one output dict per matrix, as
    reconstruct()."""
    import torch
    _check_same([tuple(it[:3]) for it in items], slots=("W", "v", "g"), what="reconstruct_batch")
    for i, it in enumerate(items):
        a = it[3] if len(it) > 3 else None
        if a is not None and (a.dtype != torch.float32 or a.device != it[0].device):
            raise ValueError(f"reconstruct_batch: matrix {i}: tensor_amax must be an fp32 tensor on W's device")
    W0, g0 = items[0][0], items[0][2]
    d = Descriptor(W0.shape[0], W0.shape[1], fmt=fmt, bits=bits, group=group, clips=clips,
                   w_dtype=_dtype_code(W0), g_dtype=_dtype_code(g0) if g0 is not None else BF16, beta2=beta2,
                   weighting=weighting, param_dtype=param_dtype)
    if fmt == "nvfp4" and any(len(it) < 4 or it[3] is None for it in items):
        need = [i for i, it in enumerate(items) if len(it) < 4 or it[3] is None]
        am = absmax_batch([items[i][0] for i in need], stream=stream)
        items = list(items)
        for i, a in zip(need, am):
            items[i] = (items[i][0], items[i][1], items[i][2], a)
    outs, mats = [], []
    for it in items:
        W, v, g = it[0], it[1], it[2]
        amax = it[3] if len(it) > 3 else None
        dd = Descriptor(W.shape[0], W.shape[1], fmt=fmt, bits=bits, group=group, clips=clips,
                        w_dtype=_dtype_code(W), g_dtype=_dtype_code(g) if g is not None else BF16, beta2=beta2,
                        weighting=weighting, param_dtype=param_dtype)
        o = alloc_outputs(dd, W, want_r=want_r, want_diag=want_diag, has_amax=True)
        o["desc"] = dd
        outs.append(o)
        mats.append(matrix(W, v, g, o, amax))
    if stream is None:
        stream = torch.cuda.current_stream(W0.device).cuda_stream
    s = quasar_reconstruct_batch(d, mats, stream)
    if s != OK:
        raise QuasarError(s, "quasar_reconstruct_batch")
    return outs
