"""Helpers shared by the GPU parity tests: moving codes and states between
numpy (oracle side) and torch device tensors (HIP side), and comparisons."""
import gc

import numpy as np
import torch

import oracle
from paper_2607_10611_amd import binding as B

CODE_NP = {"bf16": np.uint16, "e4m3": np.uint8, "e5m2": np.uint8, "fp32": np.uint32,
           "mxfp4": np.uint8, "nvfp4": np.uint8,  # 4-bit: packed bytes, two elements each
           "nvfp4_current": np.uint8}
CODE_T = {"bf16": torch.int16, "e4m3": torch.uint8, "e5m2": torch.uint8, "fp32": torch.int32,
          "mxfp4": torch.uint8, "nvfp4": torch.uint8, "nvfp4_current": torch.uint8}
SIGNED_NP = {np.uint16: np.int16, np.uint32: np.int32, np.uint8: np.uint8}


def to_dev(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype in (np.uint16, np.uint32):
        a = a.view(SIGNED_NP[a.dtype.type])
    return torch.from_numpy(a.copy()).cuda()


def to_host(t: torch.Tensor, np_dtype=None) -> np.ndarray:
    a = t.detach().cpu().numpy()
    if np_dtype is not None:
        a = a.view(np_dtype)
    return a


def ulp_dist(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Distance in units in the last place between fp32 arrays (NaN pairs: 0)."""
    ia = a.astype(np.float32).view(np.int32).astype(np.int64)
    ib = b.astype(np.float32).view(np.int32).astype(np.int64)
    ia = np.where(ia < 0, -(ia & 0x7FFFFFFF), ia)
    ib = np.where(ib < 0, -(ib & 0x7FFFFFFF), ib)
    d = np.abs(ia - ib)
    both_nan = np.isnan(a) & np.isnan(b)
    return np.where(both_nan, 0, d)


def assert_state_equal(tag, w_gpu, w_ref, m_gpu, m_ref, v_gpu, v_ref, ve_gpu, ve_ref,
                       max_ulp=2):
    """Weight codes bit-exact; fp32 moments within max_ulp (NaN where NaN);
    bf16 moment codes bit-exact."""
    bad = np.nonzero(w_gpu != w_ref)[0]
    assert bad.size == 0, (f"{tag}: {bad.size} weight codes differ, first at {bad[:5]}: "
                           f"gpu {w_gpu[bad[:5]]} oracle {w_ref[bad[:5]]}")
    for name, a, b in (("m", m_gpu, m_ref), ("v", v_gpu, v_ref), ("ve", ve_gpu, ve_ref)):
        if a.dtype == np.uint16:
            nb = np.nonzero(a != b)[0]
            assert nb.size == 0, f"{tag}: {name}: {nb.size} bf16 codes differ, first at {nb[:5]}"
            continue
        assert (np.isnan(a) == np.isnan(b)).all(), f"{tag}: {name} NaN pattern differs"
        d = ulp_dist(a, b)
        assert d.max() <= max_ulp, f"{tag}: {name} max ulp {d.max()} at {np.argmax(d)}"


STATE_T = {"fp32": torch.float32, "bf16": torch.int16, "bf16_sr": torch.int16}
STATE_NP = {"fp32": np.float32, "bf16": np.uint16, "bf16_sr": np.uint16}


class DevState:
    """Device copies of one tensor's weight codes and moments."""

    def __init__(self, wfmt, codes, n, scales=None, sfmt="fp32", copy=False):
        self.wfmt = wfmt
        self.sfmt = sfmt
        self.w = to_dev(codes)
        self.copy = torch.full((n,), 0x1234, dtype=torch.int16, device="cuda") if copy else None
        self.m = torch.zeros(n, dtype=STATE_T[sfmt], device="cuda")
        self.v = torch.zeros(n, dtype=STATE_T[sfmt], device="cuda")
        self.ve = torch.zeros(n, dtype=STATE_T[sfmt], device="cuda")
        self.scales = to_dev(scales) if scales is not None else None

    def host(self):
        sn = STATE_NP[self.sfmt]
        return (to_host(self.w, CODE_NP[self.wfmt]), to_host(self.m, sn), to_host(self.v, sn),
                to_host(self.ve, sn))


class HostState:
    """Oracle copies of one tensor's weight codes and moments."""

    def __init__(self, codes, n, scales=None, sfmt="fp32", copy=False):
        self.sfmt = sfmt
        self.w = codes.copy()
        self.copy = np.full(n, 0x1234, np.uint16) if copy else None
        self.m = np.zeros(n, STATE_NP[sfmt])
        self.v = np.zeros(n, STATE_NP[sfmt])
        self.ve = np.zeros(n, STATE_NP[sfmt])
        self.scales = scales.copy() if scales is not None else None


# NVFP4 with current scaling, device layout: the kernels' scale array holds
# the fp32 tensor scale, a 4-byte word in which pass 1 gathers the largest
# finite |w'| of the tensor, then the E4M3 block codes; pass 1 also writes w'
# over the fp32 gradient buffer.  The oracle keeps NVFP4 storage as the
# format defines it (tensor scale, block codes) and returns w'; these helpers
# map one onto the other on the test side.

def nvcs_device_scales(s_nv: np.ndarray, amax_bits: int = 0) -> np.ndarray:
    """Device scale array from NVFP4 storage (4 + n/16 bytes) and an amax word."""
    word = np.array([amax_bits], np.uint32).view(np.uint8)
    return np.concatenate([s_nv[:4], word, s_nv[4:]])


def nvcs_storage_scales(s_dev: np.ndarray) -> np.ndarray:
    """NVFP4 storage (tensor scale, block codes) from a device scale array."""
    return np.concatenate([s_dev[:4], s_dev[8:]])


def encode_nv_current(x: np.ndarray):
    """The oracle's NVFP4 encoding in the device layout (amax word zero)."""
    q, s = oracle.encode_nv(x)
    return q, nvcs_device_scales(s)


def finite_amax_bits(wn: np.ndarray) -> int:
    """Bits of the largest finite |w'| (0 when there is none)."""
    fin = np.abs(wn[np.isfinite(wn)]).astype(np.float32)
    return int(fin.max().view(np.uint32)) if fin.size else 0


def oracle_step(wfmt, hs: HostState, g, hp, gfmt="fp32", index_base=0, gidx=None):
    """One oracle step on hs.  For nvfp4_current hs.scales is in the device
    layout: the oracle steps the storage part, and the test side writes the
    amax word of the returned w' and, as the device's pass 1 does, w' over
    g (fp32)."""
    if wfmt == "nvfp4_current":
        assert gfmt == "fp32"
        s_nv = nvcs_storage_scales(hs.scales)
        wn = oracle.step_nv_current(hs.w, s_nv, g, hs.m, hs.v, hs.ve, hp, index_base=index_base,
                                    gidx=gidx, sfmt=hs.sfmt, copy=hs.copy)
        hs.scales = nvcs_device_scales(s_nv, finite_amax_bits(wn))
        g[:] = wn
    elif wfmt == "mxfp4":
        oracle.step_mx(hs.w, hs.scales, g, hs.m, hs.v, hs.ve, hp, gfmt=gfmt,
                       index_base=index_base, gidx=gidx, sfmt=hs.sfmt, copy=hs.copy)
    elif wfmt == "nvfp4":
        oracle.step_nv(hs.w, hs.scales, g, hs.m, hs.v, hs.ve, hp, gfmt=gfmt,
                       index_base=index_base, gidx=gidx, sfmt=hs.sfmt, copy=hs.copy)
    elif hs.scales is not None:
        oracle.step_block(wfmt, hs.w, hs.scales, g, hs.m, hs.v, hs.ve, hp, gfmt=gfmt,
                          index_base=index_base, gidx=gidx, sfmt=hs.sfmt, copy=hs.copy)
    else:
        oracle.step(wfmt, hs.w, g, hs.m, hs.v, hs.ve, hp, gfmt=gfmt, index_base=index_base,
                    gidx=gidx, sfmt=hs.sfmt, copy=hs.copy)


def gpu_step(ds: DevState, g_dev, hp, gfmt="fp32", index_base=0):
    B.madd_step(ds.w, ds.wfmt, g_dev, ds.m, ds.v, ds.ve, hp, gfmt=gfmt, scales=ds.scales,
                index_base=index_base, sfmt=ds.sfmt, copy=ds.copy)


def assert_copy_equal(tag, ds: DevState, hs: HostState):
    if hs.copy is None:
        return
    got = to_host(ds.copy, np.uint16)
    bad = np.nonzero(got != hs.copy)[0]
    assert bad.size == 0, f"{tag}: {bad.size} compute-copy codes differ, first at {bad[:5]}"


def free_device_bytes() -> int:
    """Device memory free for a large test: blocks that earlier tests left in
    torch's caching allocator are returned to the driver first."""
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return torch.cuda.mem_get_info()[0]
