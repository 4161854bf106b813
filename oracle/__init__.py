"""CPU oracle for the M+Adam optimizer step -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding in ``paper_2607_10611_amd``) never imports, links or runs it, and
the two share no code.

The arithmetic lives in ``madd_oracle.c`` (plain scalar C, FP32 step in one
fixed operation order, codecs by grid search).  This module compiles it with
gcc (``build()``) and exposes it through ctypes with numpy arrays.

What each function follows in the paper:
  * ``step``        -- Algorithm 1 (additive and multiplicative branches,
                       combine), the optional clamps of Algorithm 2
                       (Appendix A), rounded into the storage format as in the
                       FP32-step / BF16-storage round trip of Appendix B.
  * ``step_block``  -- the same step on FP8 payloads with FP16 block scales
                       (Section 4.2, FP8 master-weight setting).
  * ``step_nv``     -- the same step on NVFP4 storage (E2M1 payloads, one E4M3
                       scale per 16 elements, one fp32 scale per tensor; the
                       format of the 4-bit master weights of Section 4.2).
  * ``step_nv_current`` -- the NVFP4 step with its per-tensor scale derived
                       anew from the updated tensor, as a dequantize / FP32
                       step / quantize round trip does.
  * ``step_mx``     -- the same step on MXFP4 storage (E2M1 payloads, one
                       E8M0 scale per 32 elements; OCP's 4-bit block format).
  * ``toy_gradient`` -- the gradient of Appendix B's sampled quartic loss
                       (the diagnostic's workload, not the optimizer step).
  * ``encode`` / ``decode`` / ``encode_array`` / ``encode_block`` -- the
                       storage formats' value grids.
  * ``philox`` / ``draw16`` -- the counter-based generator that keys
                       stochastic rounding (not defined by the paper).

Parity pins live in ``tests/test_oracle_*.py``.  Function-level status:
``philox`` is pinned to published known-answer vectors and to rocRAND's
implementation; everything else is pinned by closed forms, limits,
invariants, library conversions and brute force (see the tests).  Parity
unpinned against the paper (the paper does not fix them): the exact fp32
operation order, the block-scaled FP8 block length and scale rule, the 4-bit
formats (``step_mx`` and ``step_nv``: pinned to the OCP MX specification and
to NVFP4's published definition instead; when NVFP4's tensor scale is
refreshed is a choice, and both are built: at encoding only (``step_nv``) or
at every step (``step_nv_current``)) and the stochastic-rounding rule with its
generator.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "madd_oracle.c")
_LIB = os.path.join(_HERE, "libmadd_oracle.so")

# format / rounding numbering of the oracle's C interface
FMT = {"bf16": 0, "e4m3": 1, "e5m2": 2, "fp32": 3, "fp16": 4, "e2m1": 5, "e8m0": 6}
GFMT = {"fp32": 0, "bf16": 1}
SFMT = {"fp32": 0, "bf16": 1, "bf16_sr": 2}
ROUND = {"rne": 0, "sr": 1}

_CODE_DTYPE = {"bf16": np.uint16, "e4m3": np.uint8, "e5m2": np.uint8, "fp32": np.uint32,
               "fp16": np.uint16}


def build() -> str:
    """Compile the oracle with gcc (no fast-math, no FP contraction)."""
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
           "-Wall", "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("MADD_ORACLE_LIB")  # a deliberately mutated copy (mutation tests)
        if path is None:
            path = _LIB
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build()
        L = ctypes.CDLL(path)
        P = ctypes.c_void_p
        D = ctypes.c_double
        I = ctypes.c_int
        I64 = ctypes.c_int64
        U64 = ctypes.c_uint64
        U32 = ctypes.c_uint32
        hp_args = [D] * 11 + [I, I, U64, I64]
        L.oracle_step.argtypes = [I, P, P, I, P, I, P, P, P, I64, P, I64] + hp_args
        L.oracle_step.restype = I
        L.oracle_step_block.argtypes = [I, P, P, P, I, P, I, P, P, P, I64, P, I64] + hp_args
        L.oracle_step_block.restype = I
        L.oracle_plain_step.argtypes = [I, P, I, P, I64, P, I64] + [D] * 7 + [I, U64, I64]
        L.oracle_plain_step.restype = I
        L.oracle_encode_array.argtypes = [I, P, P, I64]
        L.oracle_encode_array.restype = I
        L.oracle_encode_block.argtypes = [I, P, P, P, I64]
        L.oracle_encode_block.restype = I
        L.oracle_step_mx.argtypes = [P, P, P, I, P, I, P, P, P, I64, P, I64] + hp_args
        L.oracle_step_mx.restype = I
        L.oracle_encode_mx.argtypes = [P, P, P, I64]
        L.oracle_encode_mx.restype = I
        L.oracle_step_nv.argtypes = [P, P, P, I, P, I, P, P, P, I64, P, I64] + hp_args
        L.oracle_step_nv.restype = I
        L.oracle_step_nv_current.argtypes = [P, P, P, P, P, I, P, P, P, I64, P, I64, P] + hp_args
        L.oracle_step_nv_current.restype = I
        L.oracle_encode_nv.argtypes = [P, P, P, I64]
        L.oracle_encode_nv.restype = I
        L.oracle_decode.argtypes = [I, U32]
        L.oracle_decode.restype = D
        L.oracle_encode.argtypes = [I, ctypes.c_float, I, U32]
        L.oracle_encode.restype = U32
        L.oracle_philox4x32_10.argtypes = [P, P, P]
        L.oracle_philox4x32_10.restype = None
        L.oracle_draw16.argtypes = [U64, I64, U32, I64]
        L.oracle_draw16.restype = U32
        L.oracle_scalars.argtypes = [D] * 11 + [I, I64, P]
        L.oracle_scalars.restype = I
        _lib = L
    return _lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _hp_args(hp: dict):
    return [float(hp["lr_add"]), float(hp["lr_mul"]), float(hp["beta1"]), float(hp["beta2"]),
            float(hp["eps"]), float(hp["tau"]), float(hp["r_max"]), float(hp["eps0"]),
            float(hp["g_max"]), float(hp["d_mult_max"]), float(hp["w_max"]),
            int(hp["bias_correction"]), ROUND[hp["rounding"]], int(hp["seed"]) & (2**64 - 1),
            int(hp["step"])]


class OracleError(RuntimeError):
    pass


def _check_state(n, g, m, v, ve, gfmt, sfmt):
    gd = np.float32 if gfmt == "fp32" else np.uint16
    sd = np.float32 if sfmt == "fp32" else np.uint16
    for name, a, dt in (("g", g, gd), ("m", m, sd), ("v", v, sd), ("ve", ve, sd)):
        if a.dtype != dt or a.size != n:
            raise OracleError(f"{name}: expected {n} x {np.dtype(dt)}, got {a.size} x {a.dtype}")


def _check_copy(copy, n):
    if copy is not None and (copy.dtype != np.uint16 or copy.size != n):
        raise OracleError("copy must hold one uint16 bf16 code per element")


def step(wfmt: str, w: np.ndarray, g: np.ndarray, m: np.ndarray, v: np.ndarray, ve: np.ndarray,
         hp: dict, gfmt: str = "fp32", index_base: int = 0, gidx: np.ndarray | None = None,
         sfmt: str = "fp32", copy: np.ndarray | None = None):
    """One M+Adam step in place on host arrays (w codes, g, m, v, ve).

    ``sfmt`` is the storage of the moments: "fp32" (float32 arrays) or
    "bf16" (uint16 codes).  ``copy`` (uint16, optional) receives the bf16
    compute copy of the new stored weights.

    ``gidx`` (int64, one per element) gives each element's global index for the
    stochastic-rounding draw; without it element i has index ``index_base + i``.
    """
    n = w.size
    if w.dtype != _CODE_DTYPE[wfmt]:
        raise OracleError(f"w: expected {np.dtype(_CODE_DTYPE[wfmt])} codes, got {w.dtype}")
    _check_state(n, g, m, v, ve, gfmt, sfmt)
    if gidx is not None:
        gidx = np.ascontiguousarray(gidx, dtype=np.int64)
        assert gidx.size == n
    _check_copy(copy, n)
    rc = lib().oracle_step(FMT[wfmt], _ptr(w), _ptr(copy), GFMT[gfmt], _ptr(g), SFMT[sfmt],
                           _ptr(m), _ptr(v), _ptr(ve), n, _ptr(gidx), int(index_base),
                           *_hp_args(hp))
    if rc != 0:
        raise OracleError(f"oracle_step returned {rc}")


def step_block(wfmt: str, q: np.ndarray, scales: np.ndarray, g: np.ndarray, m: np.ndarray,
               v: np.ndarray, ve: np.ndarray, hp: dict, gfmt: str = "fp32", index_base: int = 0,
               gidx: np.ndarray | None = None, sfmt: str = "fp32",
               copy: np.ndarray | None = None):
    """Block-scaled FP8 step (blocks of 128 contiguous elements, FP16 scales)."""
    n = q.size
    if q.dtype != np.uint8 or scales.dtype != np.uint16 or scales.size * 128 != n:
        raise OracleError("q must be uint8 codes and scales uint16, one per 128 elements")
    _check_state(n, g, m, v, ve, gfmt, sfmt)
    if gidx is not None:
        gidx = np.ascontiguousarray(gidx, dtype=np.int64)
        assert gidx.size == n
    _check_copy(copy, n)
    rc = lib().oracle_step_block(FMT[wfmt], _ptr(q), _ptr(scales), _ptr(copy), GFMT[gfmt],
                                 _ptr(g), SFMT[sfmt], _ptr(m), _ptr(v), _ptr(ve), n, _ptr(gidx),
                                 int(index_base), *_hp_args(hp))
    if rc != 0:
        raise OracleError(f"oracle_step_block returned {rc}")


def step_mx(q: np.ndarray, scales: np.ndarray, g: np.ndarray, m: np.ndarray, v: np.ndarray,
            ve: np.ndarray, hp: dict, gfmt: str = "fp32", index_base: int = 0,
            gidx: np.ndarray | None = None, sfmt: str = "fp32", copy: np.ndarray | None = None):
    """MXFP4 step: ``q`` holds n/2 bytes (element 2k in the low nibble),
    ``scales`` one E8M0 code per 32 elements."""
    n = 2 * q.size
    if q.dtype != np.uint8 or scales.dtype != np.uint8 or scales.size * 32 != n:
        raise OracleError("q must be n/2 packed bytes and scales uint8, one per 32 elements")
    _check_state(n, g, m, v, ve, gfmt, sfmt)
    if gidx is not None:
        gidx = np.ascontiguousarray(gidx, dtype=np.int64)
        assert gidx.size == n
    _check_copy(copy, n)
    rc = lib().oracle_step_mx(_ptr(q), _ptr(scales), _ptr(copy), GFMT[gfmt], _ptr(g), SFMT[sfmt],
                              _ptr(m), _ptr(v), _ptr(ve), n, _ptr(gidx), int(index_base),
                              *_hp_args(hp))
    if rc != 0:
        raise OracleError(f"oracle_step_mx returned {rc}")


def encode_mx(x: np.ndarray):
    """MXFP4 encoding (nearest-even): packed payload bytes and E8M0 scales."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    q = np.zeros(x.size // 2, dtype=np.uint8)
    s = np.zeros(x.size // 32, dtype=np.uint8)
    if lib().oracle_encode_mx(_ptr(x), _ptr(q), _ptr(s), x.size) != 0:
        raise OracleError("oracle_encode_mx failed")
    return q, s


def step_nv(q: np.ndarray, scales: np.ndarray, g: np.ndarray, m: np.ndarray, v: np.ndarray,
            ve: np.ndarray, hp: dict, gfmt: str = "fp32", index_base: int = 0,
            gidx: np.ndarray | None = None, sfmt: str = "fp32", copy: np.ndarray | None = None):
    """NVFP4 step: ``q`` holds n/2 bytes, ``scales`` 4 + n/16 bytes (the fp32
    per-tensor scale, then one E4M3 code per 16 elements)."""
    n = 2 * q.size
    if q.dtype != np.uint8 or scales.dtype != np.uint8 or scales.size != 4 + n // 16:
        raise OracleError("q must be n/2 packed bytes and scales 4 + n/16 bytes")
    _check_state(n, g, m, v, ve, gfmt, sfmt)
    if gidx is not None:
        gidx = np.ascontiguousarray(gidx, dtype=np.int64)
        assert gidx.size == n
    _check_copy(copy, n)
    rc = lib().oracle_step_nv(_ptr(q), _ptr(scales), _ptr(copy), GFMT[gfmt], _ptr(g), SFMT[sfmt],
                              _ptr(m), _ptr(v), _ptr(ve), n, _ptr(gidx), int(index_base),
                              *_hp_args(hp))
    if rc != 0:
        raise OracleError(f"oracle_step_nv returned {rc}")


def step_nv_current(q: np.ndarray, scales: np.ndarray, g: np.ndarray, m: np.ndarray,
                    v: np.ndarray, ve: np.ndarray, hp: dict, index_base: int = 0,
                    gidx: np.ndarray | None = None, sfmt: str = "fp32",
                    copy: np.ndarray | None = None) -> np.ndarray:
    """NVFP4 step with current scaling: the per-tensor scale is derived anew
    from the updated tensor.  ``q`` and ``scales`` are NVFP4 storage as
    ``encode_nv`` lays it out (4 + n/16 scale bytes: the fp32 per-tensor
    scale, then the E4M3 block codes), updated in place; ``g`` (fp32) is only
    read.  Returns the FP32 step's updated weights w' (before re-quantization)."""
    n = 2 * q.size
    if q.dtype != np.uint8 or scales.dtype != np.uint8 or scales.size != 4 + n // 16:
        raise OracleError("q must be n/2 packed bytes and scales 4 + n/16 bytes")
    if g.dtype != np.float32:
        raise OracleError("current scaling takes fp32 gradients")
    _check_state(n, g, m, v, ve, "fp32", sfmt)
    if gidx is not None:
        gidx = np.ascontiguousarray(gidx, dtype=np.int64)
        assert gidx.size == n
    _check_copy(copy, n)
    assert scales.flags.c_contiguous
    wn = np.empty(n, np.float32)
    codes = ctypes.c_void_p(scales.ctypes.data + 4)
    rc = lib().oracle_step_nv_current(_ptr(q), _ptr(scales), codes, _ptr(copy), _ptr(g),
                                      SFMT[sfmt], _ptr(m), _ptr(v), _ptr(ve), n, _ptr(gidx),
                                      int(index_base), _ptr(wn), *_hp_args(hp))
    if rc != 0:
        raise OracleError(f"oracle_step_nv_current returned {rc}")
    return wn


def encode_nv(x: np.ndarray):
    """NVFP4 encoding (nearest-even): packed payload bytes and the scale array
    (fp32 per-tensor scale in bytes 0-3, then the E4M3 block codes)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    q = np.zeros(x.size // 2, dtype=np.uint8)
    s = np.zeros(4 + x.size // 16, dtype=np.uint8)
    if lib().oracle_encode_nv(_ptr(x), _ptr(q), _ptr(s), x.size) != 0:
        raise OracleError("oracle_encode_nv failed")
    return q, s


def nv_values(q: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """Stored NVFP4 weights as the fp32 values the step reads."""
    st = np.frombuffer(scales[:4].tobytes(), np.float32)[0]
    den = (decode_array("e4m3", scales[4:]).astype(np.float32) * st).astype(np.float32)
    el = decode_array("e2m1", unpack_e2m1(q)).astype(np.float32)
    return (el.reshape(-1, 16) * den[:, None]).astype(np.float32).ravel()


def unpack_e2m1(q: np.ndarray) -> np.ndarray:
    """Element codes (one per element) of packed MXFP4 payload bytes."""
    q = np.ascontiguousarray(q, dtype=np.uint8)
    out = np.empty(2 * q.size, dtype=np.uint8)
    out[0::2] = q & 0xF
    out[1::2] = q >> 4
    return out


def mx_values(q: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """Stored MXFP4 weights as float64 (payload x scale)."""
    el = decode_array("e2m1", unpack_e2m1(q))
    sc = decode_array("e8m0", scales)
    return (el.reshape(-1, 32) * sc[:, None]).ravel()


def toy_gradient(w: np.ndarray, target: np.ndarray, c: np.ndarray, idx: np.ndarray,
                 batch: int) -> np.ndarray:
    """Gradient of Appendix B's diagnostic loss on sampled entries,
    (1/B) sum_k c_i (w_i - w*_i)^4 over the B sampled entries idx (with
    replacement): g_i = (4/B) cnt_i c_i (w_i - w*_i)^3, cnt_i the number of
    samples equal to i, in fp32 in the order ((s d) d) d with d = w - w* and
    s = (fp32(4/B) cnt) c.  Plain numpy; pinned by its fp64 derivative and a
    finite difference of the loss (tests/test_oracle_toy.py)."""
    w = np.asarray(w, np.float32)
    n = w.size
    idx = np.asarray(idx, np.int64)
    cnt = np.bincount(idx[(idx >= 0) & (idx < n)], minlength=n).astype(np.float32)
    d = (w - np.asarray(target, np.float32)).astype(np.float32)
    s = ((np.float32(4.0 / batch) * cnt).astype(np.float32) * np.asarray(c, np.float32)).astype(np.float32)
    return (((s * d).astype(np.float32) * d).astype(np.float32) * d).astype(np.float32)


def plain_step(wfmt: str, w: np.ndarray, g: np.ndarray, hp: dict, gfmt: str = "fp32",
               index_base: int = 0, gidx: np.ndarray | None = None):
    """Appendix B's moment-free rules in place on host weight codes: additive
    (lr_mul = 0), multiplicative (lr_add = 0) or combined."""
    n = w.size
    if w.dtype != _CODE_DTYPE[wfmt]:
        raise OracleError("w: wrong code dtype")
    gd = np.float32 if gfmt == "fp32" else np.uint16
    if g.dtype != gd or g.size != n:
        raise OracleError("g: wrong dtype or size")
    if gidx is not None:
        gidx = np.ascontiguousarray(gidx, dtype=np.int64)
    rc = lib().oracle_plain_step(FMT[wfmt], _ptr(w), GFMT[gfmt], _ptr(g), n, _ptr(gidx),
                                 int(index_base), float(hp["lr_add"]), float(hp["lr_mul"]),
                                 float(hp["tau"]), float(hp["r_max"]), float(hp["eps0"]),
                                 float(hp["d_mult_max"]), float(hp["w_max"]),
                                 ROUND[hp["rounding"]], int(hp["seed"]) & (2**64 - 1),
                                 int(hp["step"]))
    if rc != 0:
        raise OracleError(f"oracle_plain_step returned {rc}")


def encode_array(fmt: str, x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.size, dtype=_CODE_DTYPE[fmt])
    if lib().oracle_encode_array(FMT[fmt], _ptr(x), _ptr(out), x.size) != 0:
        raise OracleError("oracle_encode_array failed")
    return out


def encode_block(fmt: str, x: np.ndarray):
    x = np.ascontiguousarray(x, dtype=np.float32)
    q = np.empty(x.size, dtype=np.uint8)
    s = np.empty(x.size // 128, dtype=np.uint16)
    if lib().oracle_encode_block(FMT[fmt], _ptr(x), _ptr(q), _ptr(s), x.size) != 0:
        raise OracleError("oracle_encode_block failed")
    return q, s


def decode(fmt: str, code: int) -> float:
    return lib().oracle_decode(FMT[fmt], int(code))


def decode_array(fmt: str, codes: np.ndarray) -> np.ndarray:
    return np.array([decode(fmt, int(c)) for c in codes.ravel()], dtype=np.float64)


def encode(fmt: str, x: float, rounding: str = "rne", r16: int = 0) -> int:
    return int(lib().oracle_encode(FMT[fmt], float(np.float32(x)), ROUND[rounding], int(r16)))


def philox(ctr, key):
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def draw16(seed: int, step_: int, stream: int, idx: int) -> int:
    return int(lib().oracle_draw16(int(seed) & (2**64 - 1), int(step_), int(stream), int(idx)))


def scalars(hp: dict) -> dict:
    out = np.zeros(13, dtype=np.float32)
    a = _hp_args(hp)
    rc = lib().oracle_scalars(*a[:11], a[11], a[14], _ptr(out))
    if rc != 0:
        raise OracleError("oracle_scalars failed")
    names = ["B1", "B2", "OMB1", "OMB2", "SA", "IBC2", "LRM", "EPS", "TAU", "GMAX", "ULO", "UHI",
             "WMAX"]
    return dict(zip(names, out.tolist()))
