"""The C-ABI library loads, exports every entry point of include/madd.h, and
rejects invalid arguments before any device work (CPU: no kernel runs)."""
import ctypes
import math
import os
import re

import pytest

from paper_2607_10611_amd import binding as B


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:  # noqa: BLE001
        return False


# Tests that pass made-up device addresses: each call must fail validation
# before any launch; where a GPU is visible they are skipped, so that a
# broken check could never launch a kernel on those addresses.
fake_addresses = pytest.mark.skipif(_gpu_visible(), reason="made-up device addresses; CPU only")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "madd.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(madd_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(B.EXPORTS)


def test_every_header_symbol_is_exported_by_its_library():
    """include/ holds the boundary only (madd.h); the measurement probes'
    header sits beside their source in bench_probes/."""
    from paper_2607_10611_amd import _build
    headers = sorted(os.listdir(os.path.join(ROOT, "include")))
    assert [h for h in headers if h.endswith(".h")] == ["madd.h"]
    libs = {HEADER: _build.LIB, _build.PROBE_HDR: _build.PROBE_LIB}
    for h, so in libs.items():
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names = set(re.findall(r"\b(madd_\w+)\s*\(", text))
        assert names, h
        nm = os.popen(f"nm -D --defined-only {so}").read()
        for name in names:
            assert re.search(rf"\bT {name}\b", nm), (h, name)


@fake_addresses
def test_ceiling_probe_rejects_bad_arguments():
    from paper_2607_10611_amd import _build
    L = ctypes.CDLL(_build.PROBE_LIB)
    f = L.madd_ceiling_stream
    f.argtypes = [ctypes.c_void_p] * 5 + [ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p]
    f.restype = ctypes.c_int32
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 4, -1, None) == -1
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, 3, 64, None) == -1
    assert f(None, FAKE, FAKE, FAKE, FAKE, 4, 64, None) == -1
    assert f(FAKE, FAKE + 4, FAKE, FAKE, FAKE, 4, 64, None) == -2
    assert f(None, None, None, None, None, 2, 0, None) == 0
    sm = L.madd_stream_modes
    sm.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                   ctypes.c_void_p]
    sm.restype = ctypes.c_int32
    assert sm(3, FAKE, FAKE, 8192, None) == -1           # no such mode
    assert sm(2, FAKE, FAKE, 4096, None) == -1           # not a multiple of 8192
    assert sm(2, FAKE, FAKE, 0, None) == -1
    assert sm(0, None, FAKE, 8192, None) == -1           # read needs a
    assert sm(1, FAKE, None, 8192, None) == -1           # every mode needs b
    assert sm(2, FAKE + 8, FAKE, 8192, None) == -2       # unaligned
    L.madd_probe_bf16_rounding.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    L.madd_probe_bf16_rounding.restype = ctypes.c_int32
    assert L.madd_probe_bf16_rounding(None, None) == -1
    L.madd_probe_delay.argtypes = [ctypes.c_int32, ctypes.c_void_p]
    L.madd_probe_delay.restype = ctypes.c_int32
    assert L.madd_probe_delay(-1, None) == -1
    assert L.madd_probe_delay((1 << 20) + 1, None) == -1


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name
    nm = os.popen(f"nm -D --defined-only {B.LIB_PATH}").read()
    for name in declared_functions():
        assert re.search(rf"\bT {name}\b", nm), name


def test_status_strings():
    lib = B.lib()
    for code, name in B.STATUS.items():
        assert lib.madd_status_string(code).decode().startswith(name)
    assert lib.madd_status_string(12345) == b"unknown madd status"


def _hp(**kw):
    h = B.HParams(**kw).to_c()
    return ctypes.byref(h), h


FAKE = 0x10000  # never dereferenced: every call below fails validation first
# distinct fake device addresses (1 MiB apart) for the buffers of one call,
# so that a rejection comes from the rule under test, not from overlap
W_, S_, C_, G_, M_, V_, E_ = (0x100000 * (k + 1) for k in range(7))


@fake_addresses
@pytest.mark.parametrize("kw", [dict(beta1=1.0), dict(beta2=-0.5), dict(eps=-1.0), dict(tau=0.0),
                                dict(r_max=0.0), dict(r_max=1.0), dict(eps0=0.75),
                                dict(g_max=0.0), dict(d_mult_max=-1.0), dict(w_max=0.0),
                                dict(step=0), dict(step=2 ** 32), dict(bias_correction=2),
                                dict(rounding=7), dict(lr_add=math.nan)])
def test_step_rejects_bad_hparams(kw):
    lib = B.lib()
    ref, _h = _hp(**kw)
    rc = lib.madd_step(W_, B.W_BF16, None, None, G_, B.G_FP32, M_, V_, E_, 0, 1024, 0, ref, None)
    assert rc == -1


@fake_addresses
def test_step_rejects_bad_arguments():
    lib = B.lib()
    ref, _h = _hp()
    call = lambda w, wf, sc, *a: lib.madd_step(w, wf, sc, None, *a, ref, None)  # noqa: E731
    assert lib.madd_step(W_, 0, None, None, G_, 0, M_, V_, E_, 0, 8, 0, None, None) == -1
    assert lib.madd_step(W_, 1, S_, C_ + 8, G_, 0, M_, V_, E_, 0, 128, 0, ref,
                         None) == -2  # block-scaled with an unaligned copy
    assert call(W_, 0, None, G_, 0, M_, V_, E_, 0, -1, 0) == -1          # n < 0
    assert call(None, 0, None, G_, 0, M_, V_, E_, 0, 8, 0) == -1         # null w
    assert call(W_, 0, None, G_, 0, M_, None, E_, 0, 8, 0) == -1         # null v
    assert call(W_, 9, None, G_, 0, M_, V_, E_, 0, 8, 0) == -1           # bad wfmt
    assert call(W_, 0, None, G_, 5, M_, V_, E_, 0, 8, 0) == -1           # bad gfmt
    assert call(W_, 0, None, G_, 0, M_, V_, E_, 3, 8, 0) == -1           # bad sfmt
    assert call(W_, 0, None, G_, 0, M_, V_, E_, 0, 8, -3) == -1          # base < 0
    assert call(W_, 0, S_, G_, 0, M_, V_, E_, 0, 128, 0) == -1           # scales + bf16
    assert call(W_, 1, S_, G_, 0, M_, V_, E_, 0, 100, 0) == -1           # n % 128
    assert call(W_ + 4, 1, S_, G_, 0, M_, V_, E_, 0, 128, 0) == -2       # unaligned
    assert call(None, 0, None, None, 0, None, None, None, 0, 0, 0) == 0  # empty: no-op
    assert call(W_, 0, None, G_, 0, M_, V_, E_, 0, 2 ** 62, 2 ** 62) == -1  # index overflow


@fake_addresses
def test_step_rejects_overlapping_buffers():
    """The byte ranges of one tensor's buffers, sized from the formats, must
    be pairwise disjoint: identical, partly overlapping or nested ranges are
    rejected before any device work."""
    lib = B.lib()
    ref, _h = _hp()
    n = 256
    step = lambda w, wf, sc, cp, g, gf, m, v, ve, sf=0: lib.madd_step(  # noqa: E731
        w, wf, sc, cp, g, gf, m, v, ve, sf, n, 0, ref, None)
    assert step(W_, 0, None, None, G_, 0, M_, M_, E_) == -1               # v is m
    assert step(W_, 0, None, None, G_, 0, M_, M_ + 4 * n - 16, E_) == -1  # v starts inside m
    assert step(W_, 0, None, None, G_, 0, M_, V_, V_ + 2 * n - 2, 1) == -1  # bf16 v, ve share 2 bytes
    assert step(W_, 0, None, None, M_ + 64, 0, M_, V_, E_) == -1          # g inside m
    assert step(G_ + 4 * n - 2, 0, None, None, G_, 0, M_, V_, E_) == -1   # w's first code in g
    assert step(W_, 1, W_ + 128, None, G_, 0, M_, V_, E_) == -1           # FP8 scales in the codes
    assert step(W_, B.W_NVFP4, W_ + 112, None, G_, 0, M_, V_, E_) == -1   # NVFP4 scales in the codes
    assert step(W_, 0, None, G_ + 16, G_, 0, M_, V_, E_) == -1            # compute copy in g
    PP = ctypes.POINTER(ctypes.c_void_p)
    arr = lambda *x: ctypes.cast((ctypes.c_void_p * len(x))(*x), PP)  # noqa: E731
    fm = (ctypes.c_int32 * 2)(0, 0)
    ne = (ctypes.c_int64 * 2)(n, n)
    w, g, m, v = (arr(p, p + 0x80000) for p in (W_, G_, M_, V_))
    ve = arr(E_, V_ + 0x80000 + 4 * n - 4)  # second tensor's ve overlaps its v
    assert lib.madd_multi_tensor_step(2, w, fm, None, None, g, 0, m, v, ve, 0, ne, 0, ref,
                                      None) == -1
    assert lib.madd_plain_step(W_, 0, W_ + 2 * n - 2, 0, n, 0, ref, None) == -1  # g in w
    assert lib.madd_init_state(M_, V_, M_ + 4 * n - 4, 0, n, None) == -1          # ve in m
    assert lib.madd_init_state(M_, V_, M_ + 2 * n - 2, 1, n, None) == -1          # bf16 ve in m
    assert lib.madd_encode_weights(G_, G_ + 4 * n - 2, 0, None, n, None) == -1    # w in x
    assert lib.madd_encode_weights(G_, W_, B.W_MXFP4, W_ + n // 2 - 1, n, None) == -1  # scales


@fake_addresses
def test_mxfp4_argument_rules():
    lib = B.lib()
    ref, _h = _hp()
    call = lambda w, sc, n, cp=None: lib.madd_step(w, B.W_MXFP4, sc, cp, G_, 0, M_, V_,  # noqa: E731
                                                   E_, 0, n, 0, ref, None)
    assert call(W_, None, 64) == -1            # MXFP4 needs its scales
    assert call(W_, S_, 48) == -1            # n % 32
    assert call(W_ + 2, S_, 64) == -2        # unaligned payload bytes
    assert call(W_, S_, 64, C_ + 4) == -2  # unaligned compute copy
    assert lib.madd_plain_step(W_, B.W_MXFP4, G_, 0, 64, 0, ref, None) == -1
    assert lib.madd_encode_weights(G_, W_, B.W_MXFP4, None, 64, None) == -1
    assert lib.madd_encode_weights(G_, W_, B.W_MXFP4, S_, 40, None) == -1
    assert lib.madd_encode_weights(G_, W_, 7, S_, 64, None) == -1   # no such format


@fake_addresses
def test_nvfp4_argument_rules():
    lib = B.lib()
    ref, _h = _hp()
    call = lambda w, sc, n, cp=None: lib.madd_step(w, B.W_NVFP4, sc, cp, G_, 0, M_, V_,  # noqa: E731
                                                   E_, 0, n, 0, ref, None)
    assert call(W_, None, 64) == -1            # NVFP4 needs its scales
    assert call(W_, S_, 40) == -1            # n % 16
    assert call(W_, S_ + 2, 64) == -2        # tensor scale not 4-byte aligned
    assert call(W_ + 2, S_, 64) == -2        # unaligned payload bytes
    assert call(W_, S_, 64, C_ + 4) == -2  # unaligned compute copy
    assert lib.madd_plain_step(W_, B.W_NVFP4, G_, 0, 64, 0, ref, None) == -1
    assert lib.madd_encode_weights(G_, W_, B.W_NVFP4, None, 64, None) == -1
    assert lib.madd_encode_weights(G_, W_, B.W_NVFP4, S_, 40, None) == -1
    assert lib.madd_encode_weights(G_, W_, B.W_NVFP4, S_ + 2, 64, None) == -2


@fake_addresses
def test_nvfp4_current_argument_rules():
    lib = B.lib()
    ref, _h = _hp()
    W = B.W_NVFP4_CURRENT
    call = lambda w, sc, n, gfmt=0, cp=None: lib.madd_step(w, W, sc, cp, G_, gfmt, M_, V_,  # noqa: E731
                                                           E_, 0, n, 0, ref, None)
    assert call(W_, None, 64) == -1            # scales required
    assert call(W_, S_, 40) == -1            # n % 16
    assert call(W_, S_ + 2, 64) == -2        # scale array not 4-byte aligned
    assert call(W_, S_, 64, gfmt=1) == -1    # w' is written over the gradient: fp32 only
    assert lib.madd_plain_step(W_, W, G_, 0, 64, 0, ref, None) == -1
    assert lib.madd_encode_weights(G_, W_, W, None, 64, None) == -1
    assert lib.madd_encode_weights(G_, W_, W, S_, 40, None) == -1
    PP = ctypes.POINTER(ctypes.c_void_p)
    arr = lambda *x: ctypes.cast((ctypes.c_void_p * len(x))(*x), PP)  # noqa: E731
    n = (ctypes.c_int64 * 1)(64)
    wf = (ctypes.c_int32 * 1)(W)
    assert lib.madd_multi_tensor_step(1, arr(W_), wf, arr(S_), None, arr(G_), 1, arr(M_),
                                      arr(V_), arr(E_), 0, n, 0, ref, None) == -1


@fake_addresses
def test_multi_tensor_rejects_bad_arguments():
    lib = B.lib()
    ref, _h = _hp()
    PP = ctypes.POINTER(ctypes.c_void_p)
    arr = lambda *x: ctypes.cast((ctypes.c_void_p * len(x))(*x), PP)  # noqa: E731
    fm = (ctypes.c_int32 * 2)(0, 0)
    ne = (ctypes.c_int64 * 2)(128, 256)
    w, g, m, v, ve = (arr(p, p + 0x80000) for p in (W_, G_, M_, V_, E_))
    mt = lib.madd_multi_tensor_step
    assert mt(0, None, None, None, None, None, 0, None, None, None, 0, None, 0, ref, None) == 0
    assert mt(-1, w, fm, None, None, g, 0, m, v, ve, 0, ne, 0, ref, None) == -1
    assert mt(2, w, fm, None, None, g, 0, m, v, ve, 0, ne, 0, None, None) == -1
    assert mt(2, w, fm, None, None, g, 0, m, v, ve, 3, ne, 0, ref, None) == -1      # bad sfmt
    bad = arr(V_, None)
    assert mt(2, w, fm, None, None, g, 0, m, bad, ve, 0, ne, 0, ref, None) == -1
    fm_bad = (ctypes.c_int32 * 2)(0, 11)
    assert mt(2, w, fm_bad, None, None, g, 0, m, v, ve, 0, ne, 0, ref, None) == -1
    ne_bad = (ctypes.c_int64 * 2)(128, -5)
    assert mt(2, w, fm, None, None, g, 0, m, v, ve, 0, ne_bad, 0, ref, None) == -1
    sc = arr(None, S_)  # second tensor block-scaled but bf16
    assert mt(2, w, fm, sc, None, g, 0, m, v, ve, 0, ne, 0, ref, None) == -1
    fm_mx = (ctypes.c_int32 * 2)(4, 4)
    sc_one = arr(S_, None)  # second MXFP4 tensor without scales
    assert mt(2, w, fm_mx, sc_one, None, g, 0, m, v, ve, 0, ne, 0, ref, None) == -1


@fake_addresses
def test_plain_step_rejects_bad_arguments():
    lib = B.lib()
    ref, _h = _hp()
    assert lib.madd_plain_step(W_, 0, G_, 0, 8, 0, None, None) == -1        # no hparams
    assert lib.madd_plain_step(W_, 6, G_, 0, 8, 0, ref, None) == -1         # bad wfmt
    assert lib.madd_plain_step(W_, 0, G_, 3, 8, 0, ref, None) == -1         # bad gfmt
    assert lib.madd_plain_step(W_, 0, None, 0, 8, 0, ref, None) == -1         # null g
    assert lib.madd_plain_step(W_, 0, G_, 0, -2, 0, ref, None) == -1        # n < 0
    assert lib.madd_plain_step(None, 0, None, 0, 0, 0, ref, None) == 0          # empty
    bad, _h2 = _hp(r_max=1.5)
    assert lib.madd_plain_step(W_, 0, G_, 0, 8, 0, bad, None) == -1


@fake_addresses
def test_toy_gradient_rejects_bad_arguments():
    lib = B.lib()
    f = lib.madd_toy_gradient
    n = 64
    W_, T_, C_, I_, K_, G_ = (FAKE + k * (1 << 20) for k in range(6))
    assert f(W_, 0, T_, C_, I_, 10, -1, K_, G_, None) == -1           # n < 0
    assert f(W_, 0, T_, C_, I_, -1, n, K_, G_, None) == -1            # batch < 0
    assert f(W_, B.W_MXFP4, T_, C_, I_, 10, n, K_, G_, None) == -1    # 4-bit storage
    assert f(W_, 9, T_, C_, I_, 10, n, K_, G_, None) == -1            # unknown format
    assert f(W_, 0, None, C_, I_, 10, n, K_, G_, None) == -1          # null target
    assert f(W_, 0, T_, C_, None, 10, n, K_, G_, None) == -1          # samples, no idx
    assert f(W_, 0, T_, C_, I_, 10, n, T_ + 8, G_, None) == -1        # counts inside target
    assert f(W_, 0, T_, C_, I_, 10, n, K_, W_ + 64, None) == -1       # g overlaps w
    assert f(None, 0, None, None, None, 0, 0, None, None, None) == 0  # empty


@fake_addresses
def test_init_and_encode_reject_bad_arguments():
    lib = B.lib()
    assert lib.madd_init_state(M_, V_, E_, 0, -1, None) == -1
    assert lib.madd_init_state(None, V_, E_, 0, 5, None) == -1
    assert lib.madd_init_state(M_, V_, E_, 4, 5, None) == -1   # bad sfmt
    assert lib.madd_init_state(None, None, None, 1, 0, None) == 0
    assert lib.madd_encode_weights(G_, W_, 7, None, 8, None) == -1
    assert lib.madd_encode_weights(G_, W_, 0, S_, 128, None) == -1   # scales + bf16
    assert lib.madd_encode_weights(G_, W_, 1, S_, 130, None) == -1   # n % 128
    assert lib.madd_encode_weights(None, W_, 1, None, 8, None) == -1


def test_binding_has_no_cpu_fallback(monkeypatch, tmp_path):
    monkeypatch.setattr(B, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(B, "_lib", None)
    with pytest.raises(ImportError):
        B.lib()


def test_binding_rejects_host_tensors_before_any_call():
    import torch
    t16 = torch.zeros(64, dtype=torch.int16)
    t32 = torch.zeros(64)
    with pytest.raises(ValueError, match="GPU tensor"):
        B.madd_step(t16, "bf16", t32, t32, t32, t32, _hp()[1])
    with pytest.raises(ValueError, match="GPU tensor"):
        B.madd_init_state(t32, t32, t32)
    with pytest.raises(ValueError, match="GPU tensor"):
        B.madd_encode_weights(t32, t16, "bf16")


def test_scale_bytes():
    assert B.scale_bytes("e4m3", 1024) == 16
    assert B.scale_bytes("mxfp4", 1024) == 32
    assert B.scale_bytes("nvfp4", 1024) == 68
    assert B.scale_bytes("nvfp4_current", 1024) == 72


def test_prepared_scalars():
    lib = B.lib()
    assert lib.madd_scalars_bytes() == 64
    ref, _h = _hp(step=5, seed=2 ** 40 + 7)
    buf = ctypes.create_string_buffer(64)
    assert lib.madd_prepare_scalars(ref, buf) == 0
    import struct
    *_f, key0, key1, t = struct.unpack("13f3I", buf.raw)
    assert (key0, key1, t) == (7, 2 ** 8, 5)
    assert lib.madd_prepare_scalars(ref, None) == -1
    bad, _h2 = _hp(beta1=1.0)
    assert lib.madd_prepare_scalars(bad, buf) == -1
    assert lib.madd_prepare_scalars(None, buf) == -1


@fake_addresses
def test_device_scalars_step_rejects_bad_arguments():
    lib = B.lib()
    ref, _h = _hp()
    PP = ctypes.POINTER(ctypes.c_void_p)
    arr = lambda *x: ctypes.cast((ctypes.c_void_p * len(x))(*x), PP)  # noqa: E731
    fm = (ctypes.c_int32 * 1)(0)
    ne = (ctypes.c_int64 * 1)(256)
    w, g, m, v, ve = (arr(p) for p in (W_, G_, M_, V_, E_))
    mt = lib.madd_multi_tensor_step_dev
    assert mt(1, w, fm, None, None, g, 0, m, v, ve, 0, ne, 0, ref, None, None) == -1  # no scalars
    assert mt(1, w, fm, None, None, g, 0, m, v, ve, 0, ne, 0, ref, S_ + 2, None) == -2  # unaligned
    assert mt(1, w, fm, None, None, g, 0, m, v, ve, 3, ne, 0, ref, S_, None) == -1     # bad sfmt
    assert mt(1, w, fm, None, None, g, 0, m, v, ve, 0, ne, 0, None, S_, None) == -1    # no hp


@pytest.mark.parametrize("kw", [dict(step=1), dict(step=37, lr_add=3e-4, lr_mul=2e-3),
                                dict(step=5, bias_correction=0, eps0=0.05, d_mult_max=0.25,
                                     g_max=2.0, w_max=8.0, beta1=0.8, beta2=0.95)])
def test_prepared_scalars_follow_algorithm_2(kw):
    """The fp32 coefficients the kernels use (Section 3.1 / Algorithm 2,
    derived in double and rounded once), restated here from the update rule:
    bias-corrected eta_a and 1/(1 - beta2^t), the u_m clip bounds narrowed by
    the exponent cap 2^+-d, the Philox key and counter."""
    import struct
    import numpy as np
    h = B.HParams(**kw)
    got = struct.unpack("13f3I", B.prepare_scalars(h))
    t = h.step
    bc = h.bias_correction
    sa = h.lr_add / (1 - h.beta1 ** t) if bc else h.lr_add
    ibc2 = 1 / (1 - h.beta2 ** t) if bc else 1.0
    lo, hi = -(h.r_max - h.eps0), h.r_max
    if math.isfinite(h.d_mult_max):
        lo, hi = max(lo, 2.0 ** -h.d_mult_max - 1), min(hi, 2.0 ** h.d_mult_max - 1)
    want = [h.beta1, h.beta2, 1 - h.beta1, 1 - h.beta2, sa, ibc2, h.lr_mul, h.eps, h.tau,
            h.g_max, lo, hi, h.w_max]
    assert [float(np.float32(x)) for x in want] == list(got[:13])
    assert got[13:] == (h.seed & 0xFFFFFFFF, h.seed >> 32, t)
