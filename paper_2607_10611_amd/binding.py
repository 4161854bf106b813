"""Thin ctypes binding of ``libmadd.so`` (declared in ``include/madd.h``).

Argument marshalling only: every step of the update runs in the library's HIP
kernels.  Tensors are torch tensors on the GPU (PyTorch provides device memory
and streams); the functions pass their data pointers and the current HIP
stream to the C ABI and raise ``MaddError`` on any non-OK status.  There is no
CPU fallback: if the library is missing, ``lib()`` raises.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmadd.so")

# enum values of madd.h
W_BF16, W_FP8_E4M3, W_FP8_E5M2, W_FP32, W_MXFP4, W_NVFP4, W_NVFP4_CURRENT = 0, 1, 2, 3, 4, 5, 6
G_FP32, G_BF16 = 0, 1
ROUND_RNE, ROUND_SR = 0, 1
WFMT = {"bf16": W_BF16, "e4m3": W_FP8_E4M3, "e5m2": W_FP8_E5M2, "fp32": W_FP32,
        "mxfp4": W_MXFP4, "nvfp4": W_NVFP4, "nvfp4_current": W_NVFP4_CURRENT}
MX_BLOCK = 32  # elements per MXFP4 block (one E8M0 scale byte)
NV_BLOCK = 16  # elements per NVFP4 block (one E4M3 scale byte after the fp32 tensor scale)
_WFMT_NAME = {v: k for k, v in WFMT.items()}
GFMT = {"fp32": G_FP32, "bf16": G_BF16}
S_FP32, S_BF16, S_BF16_SR = 0, 1, 2
SFMT = {"fp32": S_FP32, "bf16": S_BF16, "bf16_sr": S_BF16_SR}
ROUND = {"rne": ROUND_RNE, "sr": ROUND_SR}

STATUS = {0: "MADD_OK", -1: "MADD_EINVAL", -2: "MADD_EALIGN", -3: "MADD_EUNSUPPORTED",
          -4: "MADD_EDEVICE", -5: "MADD_ENOMEM", -6: "MADD_ECAPTURE", -7: "MADD_ESCRATCH"}

EXPORTS = ("madd_init_state", "madd_encode_weights", "madd_step", "madd_multi_tensor_step",
           "madd_plain_step", "madd_status_string", "madd_scalars_bytes", "madd_prepare_scalars",
           "madd_multi_tensor_step_dev", "madd_multi_tensor_step_noalloc", "madd_toy_gradient")


class MaddError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        msg = _lib.madd_status_string(status).decode() if _lib is not None else STATUS.get(status)
        super().__init__(f"{fn} failed: {msg} ({status})")


class madd_hparams(ctypes.Structure):
    _fields_ = [
        ("lr_add", ctypes.c_double), ("lr_mul", ctypes.c_double),
        ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
        ("eps", ctypes.c_double), ("tau", ctypes.c_double),
        ("r_max", ctypes.c_double), ("eps0", ctypes.c_double),
        ("g_max", ctypes.c_double), ("d_mult_max", ctypes.c_double),
        ("w_max", ctypes.c_double),
        ("bias_correction", ctypes.c_int32), ("rounding", ctypes.c_int32),
        ("seed", ctypes.c_uint64), ("step", ctypes.c_int64),
    ]


@dataclass
class HParams:
    """Hyper-parameters of one step (field meanings in include/madd.h)."""
    lr_add: float = 1e-3
    lr_mul: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    tau: float = 1e-8
    r_max: float = 0.75
    eps0: float = 0.0
    g_max: float = math.inf
    d_mult_max: float = math.inf
    w_max: float = math.inf
    bias_correction: int = 1
    rounding: str = "rne"
    seed: int = 0
    step: int = 1

    @classmethod
    def from_dict(cls, d: dict) -> "HParams":
        return cls(**{k: d[k] for k in cls.__dataclass_fields__ if k in d})

    def to_c(self) -> madd_hparams:
        return madd_hparams(float(self.lr_add), float(self.lr_mul), float(self.beta1),
                            float(self.beta2), float(self.eps), float(self.tau), float(self.r_max),
                            float(self.eps0), float(self.g_max), float(self.d_mult_max),
                            float(self.w_max), int(self.bias_correction),
                            ROUND[self.rounding] if isinstance(self.rounding, str)
                            else int(self.rounding),
                            int(self.seed) & (2**64 - 1), int(self.step))


_lib = None


def lib():
    """Load libmadd.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it first "
                              "(python -c 'import __graft_entry__ as g; g.build()')")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        HP = ctypes.POINTER(madd_hparams)
        L.madd_init_state.argtypes = [P, P, P, I32, I64, P]
        L.madd_init_state.restype = I32
        L.madd_encode_weights.argtypes = [P, P, I32, P, I64, P]
        L.madd_encode_weights.restype = I32
        L.madd_step.argtypes = [P, I32, P, P, P, I32, P, P, P, I32, I64, I64, HP, P]
        L.madd_step.restype = I32
        PP = ctypes.POINTER(ctypes.c_void_p)
        L.madd_multi_tensor_step.argtypes = [I32, PP, ctypes.POINTER(I32), PP, PP, PP, I32, PP, PP,
                                             PP, I32, ctypes.POINTER(I64), I64, HP, P]
        L.madd_multi_tensor_step.restype = I32
        L.madd_multi_tensor_step_noalloc.argtypes = L.madd_multi_tensor_step.argtypes
        L.madd_multi_tensor_step_noalloc.restype = I32
        L.madd_toy_gradient.argtypes = [P, I32, P, P, P, I64, I64, P, P, P]
        L.madd_toy_gradient.restype = I32
        L.madd_plain_step.argtypes = [P, I32, P, I32, I64, I64, HP, P]
        L.madd_plain_step.restype = I32
        L.madd_status_string.argtypes = [I32]
        L.madd_status_string.restype = ctypes.c_char_p
        L.madd_scalars_bytes.argtypes = []
        L.madd_scalars_bytes.restype = I64
        L.madd_prepare_scalars.argtypes = [HP, P]
        L.madd_prepare_scalars.restype = I32
        L.madd_multi_tensor_step_dev.argtypes = [I32, PP, ctypes.POINTER(I32), PP, PP, PP, I32,
                                                 PP, PP, PP, I32, ctypes.POINTER(I64), I64, HP,
                                                 P, P]
        L.madd_multi_tensor_step_dev.restype = I32
        _lib = L
    return _lib


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# Bytes per element of each storage, for the size checks below (the C ABI
# receives bare pointers and cannot check them).
CODE_BYTES = {"bf16": 2, "e4m3": 1, "e5m2": 1, "fp32": 4, "mxfp4": 0.5, "nvfp4": 0.5,
              "nvfp4_current": 0.5}
GRAD_BYTES = {"fp32": 4, "bf16": 2}
STATE_BYTES = {"fp32": 4, "bf16": 2, "bf16_sr": 2}


def scale_bytes(wfmt: str, n: int) -> int:
    """Bytes of the block-scale array of n elements: FP16 per 128 (block FP8),
    E8M0 per 32 (MXFP4), the fp32 tensor scale then E4M3 per 16 (NVFP4), and
    for NVFP4 with current scaling the amax word between them."""
    if wfmt == "mxfp4":
        return n // MX_BLOCK
    if wfmt == "nvfp4":
        return 4 + n // NV_BLOCK
    if wfmt == "nvfp4_current":
        return 8 + n // NV_BLOCK
    return (n // 128) * 2


def torch_dtype(name: str):
    import torch
    return getattr(torch, name)


def _need(what: str, t, nbytes: int):
    """A tensor argument must be a contiguous GPU tensor of at least `nbytes`
    bytes (a raw int pointer is the caller's responsibility)."""
    if t is None or isinstance(t, int):
        return
    if not t.is_cuda:
        raise ValueError(f"{what} must be a GPU tensor (got one on {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{what} holds {have} bytes; the call reads or writes {nbytes}")


def _need_tensor(fn: str, wfmt: str, n: int, w, m, v, ve, sfmt: str, scales=None, copy=None):
    _need(f"{fn}: w", w, math.ceil(n * CODE_BYTES[wfmt]))
    for name, t in (("m", m), ("v", v), ("ve", ve)):
        _need(f"{fn}: {name}", t, n * STATE_BYTES[sfmt])
    if scales is not None:
        _need(f"{fn}: scales", scales, scale_bytes(wfmt, n))
    if copy is not None:
        _need(f"{fn}: copy", copy, 2 * n)


def _check(fn: str, rc: int):
    if rc != 0:
        raise MaddError(fn, rc)


def _hp(hp) -> madd_hparams:
    if isinstance(hp, madd_hparams):
        return hp
    if isinstance(hp, dict):
        hp = HParams.from_dict(hp)
    return hp.to_c()


def state_format(t) -> str:
    """Moment storage of a torch tensor: float32 -> "fp32"; bfloat16 (or its
    16-bit integer view) -> "bf16" (pass sfmt="bf16_sr" explicitly for
    stochastically rounded bf16 moments)."""
    import torch
    if t.dtype == torch.float32:
        return "fp32"
    if t.dtype in (torch.bfloat16, torch.int16):
        return "bf16"
    raise TypeError(f"unsupported moment dtype {t.dtype}")


def madd_init_state(m, v, ve, sfmt: str | None = None, stream=None):
    n = m.numel()
    sfmt = sfmt or state_format(m)
    for name, t in (("m", m), ("v", v), ("ve", ve)):
        _need(f"madd_init_state: {name}", t, n * STATE_BYTES[sfmt])
    _check("madd_init_state", lib().madd_init_state(_ptr(m), _ptr(v), _ptr(ve), SFMT[sfmt], n,
                                                    _stream(stream)))


def madd_encode_weights(x, w, wfmt: str, scales=None, stream=None):
    """Round fp32 ``x`` into the storage ``w`` (and its block ``scales``)."""
    n = x.numel()
    _need("madd_encode_weights: x", x, 4 * n)
    _need("madd_encode_weights: w", w, math.ceil(n * CODE_BYTES[wfmt]))
    if scales is not None:
        _need("madd_encode_weights: scales", scales, scale_bytes(wfmt, n))
    _check("madd_encode_weights",
           lib().madd_encode_weights(_ptr(x), _ptr(w), WFMT[wfmt], _ptr(scales), x.numel(),
                                     _stream(stream)))


def madd_step(w, wfmt: str, g, m, v, ve, hp, gfmt: str = "fp32", scales=None, index_base: int = 0,
              n: int | None = None, sfmt: str | None = None, copy=None, stream=None):
    """One step on one tensor.  ``w`` holds the weight codes (uint16 / uint8 /
    int32 storage for bf16 / fp8 / fp32; n/2 packed bytes for mxfp4, whose
    ``scales`` are n/32 uint8 E8M0 codes, and for nvfp4, whose ``scales`` are
    4 + n/16 bytes, 4-byte aligned: the fp32 tensor scale, then E4M3 codes;
    for nvfp4_current 8 + n/16 bytes, the tensor scale derived anew each step
    and ``g`` (fp32) overwritten with the updated weights);
    the moments' storage follows their dtype unless ``sfmt`` is given; ``copy`` (16-bit tensor) receives the
    bf16 compute copy of the new weights."""
    h = _hp(hp)
    n = m.numel() if n is None else n
    sfmt = sfmt or state_format(m)
    _need_tensor("madd_step", wfmt, n, w, m, v, ve, sfmt, scales, copy)
    _need("madd_step: g", g, n * GRAD_BYTES[gfmt])
    _check("madd_step",
           lib().madd_step(_ptr(w), WFMT[wfmt], _ptr(scales), _ptr(copy), _ptr(g), GFMT[gfmt],
                           _ptr(m), _ptr(v), _ptr(ve), SFMT[sfmt], int(n), int(index_base),
                           ctypes.byref(h), _stream(stream)))


def madd_plain_step(w, wfmt: str, g, hp, gfmt: str = "fp32", index_base: int = 0, stream=None):
    """One step of Appendix B's moment-free rules (additive: lr_mul = 0,
    multiplicative: lr_add = 0, combined: both) on one tensor."""
    h = _hp(hp)
    _need("madd_plain_step: g", g, w.numel() * GRAD_BYTES[gfmt])
    _check("madd_plain_step",
           lib().madd_plain_step(_ptr(w), WFMT[wfmt], _ptr(g), GFMT[gfmt], w.numel(),
                                 int(index_base), ctypes.byref(h), _stream(stream)))


def madd_toy_gradient(w, wfmt: str, target, c, idx, counts, g, stream=None):
    """Gradient of Appendix B's sampled quartic loss into g (fp32); idx holds
    the sampled entries (int64), counts is an int32 workspace of w's size."""
    n = w.numel()
    if idx.dtype != torch_dtype("int64") or counts.element_size() != 4:
        raise ValueError("madd_toy_gradient: idx must be int64 and counts a 4-byte integer array")
    for name, t, nb in (("target", target, 4 * n), ("c", c, 4 * n), ("counts", counts, 4 * n),
                        ("g", g, 4 * n), ("idx", idx, 8 * idx.numel())):
        _need(f"madd_toy_gradient: {name}", t, nb)
    _check("madd_toy_gradient",
           lib().madd_toy_gradient(_ptr(w), WFMT[wfmt], _ptr(target), _ptr(c), _ptr(idx),
                                   idx.numel(), n, _ptr(counts), _ptr(g), _stream(stream)))


class TensorList:
    """Marshalled pointer arrays of a tensor list, built once and reused.  It
    holds references to every tensor it points into, so the memory stays
    allocated for as long as the list can be stepped."""

    def __init__(self, ws, wfmts, gs, ms, vs, ves, scales=None, sfmt: str | None = None,
                 copies=None):
        k = len(ws)
        self._tensors = [list(ws), list(gs), list(ms), list(vs), list(ves),
                         list(scales) if scales is not None else [],
                         list(copies) if copies is not None else []]
        self.sfmt = sfmt or (state_format(ms[0]) if k else "fp32")
        assert all(len(x) == k for x in (wfmts, gs, ms, vs, ves))
        self.n = k
        Arr = ctypes.c_void_p * k
        self.w = Arr(*[_ptr(t) for t in ws])
        self.g = Arr(*[_ptr(t) for t in gs])
        self.m = Arr(*[_ptr(t) for t in ms])
        self.v = Arr(*[_ptr(t) for t in vs])
        self.ve = Arr(*[_ptr(t) for t in ves])
        self.scales = Arr(*[_ptr(t) for t in scales]) if scales is not None else None
        self.copy = Arr(*[_ptr(t) for t in copies]) if copies is not None else None
        self.wfmt = (ctypes.c_int32 * k)(*[WFMT[f] if isinstance(f, str) else int(f)
                                           for f in wfmts])
        self.numel = (ctypes.c_int64 * k)(*[t.numel() for t in ms])
        self.total = sum(t.numel() for t in ms)
        for i in range(k):
            f = wfmts[i] if isinstance(wfmts[i], str) else _WFMT_NAME[int(wfmts[i])]
            _need_tensor(f"TensorList[{i}]", f, ms[i].numel(), ws[i], ms[i], vs[i], ves[i],
                         self.sfmt, scales[i] if scales is not None else None,
                         copies[i] if copies is not None else None)
        self._grads_ok = set()  # gradient formats the current gradients were checked for

    def set_grads(self, gs):
        gs = list(gs)
        assert len(gs) == self.n
        for i, t in enumerate(gs):
            self.g[i] = _ptr(t)
        self._tensors[1] = gs
        self._grads_ok = set()

    def check_grads(self, gfmt: str):
        if gfmt in self._grads_ok:
            return
        for i, t in enumerate(self._tensors[1]):
            _need(f"TensorList[{i}]: g", t, self.numel[i] * GRAD_BYTES[gfmt])
        self._grads_ok.add(gfmt)


def madd_multi_tensor_step(tl: TensorList, hp, gfmt: str = "fp32", index_base: int = 0,
                           stream=None):
    """One step over a TensorList (one launch per weight format)."""
    h = _hp(hp)
    tl.check_grads(gfmt)
    PP = ctypes.POINTER(ctypes.c_void_p)
    cast = lambda a: ctypes.cast(a, PP) if a is not None else None  # noqa: E731
    _check("madd_multi_tensor_step",
           lib().madd_multi_tensor_step(tl.n, cast(tl.w), tl.wfmt, cast(tl.scales), cast(tl.copy),
                                        cast(tl.g), GFMT[gfmt], cast(tl.m), cast(tl.v), cast(tl.ve),
                                        SFMT[tl.sfmt], tl.numel, int(index_base),
                                        ctypes.byref(h), _stream(stream)))


def madd_multi_tensor_step_noalloc(tl: TensorList, hp, gfmt: str = "fp32", index_base: int = 0,
                                   stream=None):
    """madd_multi_tensor_step without device allocation: the descriptor
    tables go to the library's fixed per-GPU array (at most 4096 tensors)."""
    h = _hp(hp)
    tl.check_grads(gfmt)
    PP = ctypes.POINTER(ctypes.c_void_p)
    cast = lambda a: ctypes.cast(a, PP) if a is not None else None  # noqa: E731
    _check("madd_multi_tensor_step_noalloc",
           lib().madd_multi_tensor_step_noalloc(tl.n, cast(tl.w), tl.wfmt, cast(tl.scales),
                                                cast(tl.copy), cast(tl.g), GFMT[gfmt],
                                                cast(tl.m), cast(tl.v), cast(tl.ve),
                                                SFMT[tl.sfmt], tl.numel, int(index_base),
                                                ctypes.byref(h), _stream(stream)))


def prepare_scalars(hp) -> bytes:
    """The step's hyper-parameter scalars for hp, as the bytes that
    madd_multi_tensor_step_dev reads from device memory."""
    h = _hp(hp)
    buf = ctypes.create_string_buffer(int(lib().madd_scalars_bytes()))
    _check("madd_prepare_scalars", lib().madd_prepare_scalars(ctypes.byref(h), buf))
    return buf.raw


def madd_multi_tensor_step_dev(tl: TensorList, hp, dev_scalars, gfmt: str = "fp32",
                               index_base: int = 0, stream=None):
    """madd_multi_tensor_step with the scalars read at run time from
    ``dev_scalars`` (a GPU tensor holding prepare_scalars' bytes); ``hp``
    selects the kernels (rounding mode, clamps)."""
    h = _hp(hp)
    tl.check_grads(gfmt)
    _need("madd_multi_tensor_step_dev: dev_scalars", dev_scalars, int(lib().madd_scalars_bytes()))
    PP = ctypes.POINTER(ctypes.c_void_p)
    cast = lambda a: ctypes.cast(a, PP) if a is not None else None  # noqa: E731
    _check("madd_multi_tensor_step_dev",
           lib().madd_multi_tensor_step_dev(tl.n, cast(tl.w), tl.wfmt, cast(tl.scales),
                                            cast(tl.copy), cast(tl.g), GFMT[gfmt], cast(tl.m),
                                            cast(tl.v), cast(tl.ve), SFMT[tl.sfmt], tl.numel,
                                            int(index_base), ctypes.byref(h), _ptr(dev_scalars),
                                            _stream(stream)))
