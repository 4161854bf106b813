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
W_BF16, W_FP8_E4M3, W_FP8_E5M2, W_FP32, W_MXFP4, W_NVFP4 = 0, 1, 2, 3, 4, 5
G_FP32, G_BF16 = 0, 1
ROUND_RNE, ROUND_SR = 0, 1
WFMT = {"bf16": W_BF16, "e4m3": W_FP8_E4M3, "e5m2": W_FP8_E5M2, "fp32": W_FP32,
        "mxfp4": W_MXFP4, "nvfp4": W_NVFP4}
MX_BLOCK = 32  # elements per MXFP4 block (one E8M0 scale byte)
NV_BLOCK = 16  # elements per NVFP4 block (one E4M3 scale byte after the fp32 tensor scale)
GFMT = {"fp32": G_FP32, "bf16": G_BF16}
S_FP32, S_BF16, S_BF16_SR = 0, 1, 2
SFMT = {"fp32": S_FP32, "bf16": S_BF16, "bf16_sr": S_BF16_SR}
ROUND = {"rne": ROUND_RNE, "sr": ROUND_SR}

STATUS = {0: "MADD_OK", -1: "MADD_EINVAL", -2: "MADD_EALIGN", -3: "MADD_EUNSUPPORTED",
          -4: "MADD_EDEVICE", -5: "MADD_ENOMEM"}

EXPORTS = ("madd_init_state", "madd_encode_weights", "madd_step", "madd_multi_tensor_step",
           "madd_plain_step", "madd_status_string")


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
        L.madd_plain_step.argtypes = [P, I32, P, I32, I64, I64, HP, P]
        L.madd_plain_step.restype = I32
        L.madd_status_string.argtypes = [I32]
        L.madd_status_string.restype = ctypes.c_char_p
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
    _check("madd_init_state", lib().madd_init_state(_ptr(m), _ptr(v), _ptr(ve), SFMT[sfmt], n,
                                                    _stream(stream)))


def madd_encode_weights(x, w, wfmt: str, scales=None, stream=None):
    """Round fp32 ``x`` into the storage ``w`` (and its block ``scales``)."""
    _check("madd_encode_weights",
           lib().madd_encode_weights(_ptr(x), _ptr(w), WFMT[wfmt], _ptr(scales), x.numel(),
                                     _stream(stream)))


def madd_step(w, wfmt: str, g, m, v, ve, hp, gfmt: str = "fp32", scales=None, index_base: int = 0,
              n: int | None = None, sfmt: str | None = None, copy=None, stream=None):
    """One step on one tensor.  ``w`` holds the weight codes (uint16 / uint8 /
    int32 storage for bf16 / fp8 / fp32; n/2 packed bytes for mxfp4, whose
    ``scales`` are n/32 uint8 E8M0 codes, and for nvfp4, whose ``scales`` are
    4 + n/16 bytes, 4-byte aligned: the fp32 tensor scale, then E4M3 codes);
    the moments' storage follows their dtype unless ``sfmt`` is given; ``copy`` (16-bit tensor) receives the
    bf16 compute copy of the new weights."""
    h = _hp(hp)
    n = m.numel() if n is None else n
    sfmt = sfmt or state_format(m)
    _check("madd_step",
           lib().madd_step(_ptr(w), WFMT[wfmt], _ptr(scales), _ptr(copy), _ptr(g), GFMT[gfmt],
                           _ptr(m), _ptr(v), _ptr(ve), SFMT[sfmt], int(n), int(index_base),
                           ctypes.byref(h), _stream(stream)))


def madd_plain_step(w, wfmt: str, g, hp, gfmt: str = "fp32", index_base: int = 0, stream=None):
    """One step of Appendix B's moment-free rules (additive: lr_mul = 0,
    multiplicative: lr_add = 0, combined: both) on one tensor."""
    h = _hp(hp)
    _check("madd_plain_step",
           lib().madd_plain_step(_ptr(w), WFMT[wfmt], _ptr(g), GFMT[gfmt], w.numel(),
                                 int(index_base), ctypes.byref(h), _stream(stream)))


class TensorList:
    """Marshalled pointer arrays of a tensor list, built once and reused."""

    def __init__(self, ws, wfmts, gs, ms, vs, ves, scales=None, sfmt: str | None = None,
                 copies=None):
        k = len(ws)
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

    def set_grads(self, gs):
        for i, t in enumerate(gs):
            self.g[i] = _ptr(t)


def madd_multi_tensor_step(tl: TensorList, hp, gfmt: str = "fp32", index_base: int = 0,
                           stream=None):
    """One step over a TensorList (one launch per weight format)."""
    h = _hp(hp)
    PP = ctypes.POINTER(ctypes.c_void_p)
    cast = lambda a: ctypes.cast(a, PP) if a is not None else None  # noqa: E731
    _check("madd_multi_tensor_step",
           lib().madd_multi_tensor_step(tl.n, cast(tl.w), tl.wfmt, cast(tl.scales), cast(tl.copy),
                                        cast(tl.g), GFMT[gfmt], cast(tl.m), cast(tl.v), cast(tl.ve),
                                        SFMT[tl.sfmt], tl.numel, int(index_base),
                                        ctypes.byref(h), _stream(stream)))
