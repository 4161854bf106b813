"""Sharding by global index range and the streaming-ceiling probe (GPU).

The step is elementwise and its random draws are keyed by global index, so
splitting the index space into contiguous shards, each stepped with its own
index base (one GPU's share under optimizer-state sharding), must give the
same bits as one call over the whole list.  Checked on the 1.1B-parameter
list in the benchmark's flat per-role layout, on full buffers, plus oracle
parity on elements around every shard boundary.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from paper_2607_10611_amd import _build
from paper_2607_10611_amd import binding as B
from paper_2607_10611_amd import workloads as W
from gpu_parity_util import HostState, assert_state_equal, oracle_step, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


def flat_list(cfg):
    specs = W.specs(cfg)
    n = W.total_params(cfg)
    w = torch.empty(n, dtype=torch.int16, device="cuda")
    off = 0
    for i, s in enumerate(specs):
        x = W.init_fp32_device(cfg, i)
        B.madd_encode_weights(x, w[off:off + s.numel], "bf16")
        off += s.numel
    return specs, n, w


def grads(cfg, specs, n, t):
    g = torch.empty(n, device="cuda")
    off = 0
    for i, s in enumerate(specs):
        W.grad_fp32_device_(cfg, i, t, g[off:off + s.numel])
        off += s.numel
    return g


def test_eight_shards_equal_one_call_llama_1b():
    cfg = "c3"
    specs, n, w = flat_list(cfg)
    w8 = w.clone()
    m, v, ve = (torch.zeros(n, device="cuda") for _ in range(3))
    m8, v8, ve8 = (torch.zeros(n, device="cuda") for _ in range(3))
    views = []
    off = 0
    for s in specs:
        views.append(slice(off, off + s.numel))
        off += s.numel
    tl = B.TensorList([w[sl] for sl in views], ["bf16"] * len(views), [None] * len(views),
                      [m[sl] for sl in views], [v[sl] for sl in views], [ve[sl] for sl in views])
    per = (n // 8) // 128 * 128
    bounds = [k * per for k in range(8)] + [n]
    # oracle samples: 256 elements on each side of every inner boundary
    idx = np.unique(np.concatenate([np.arange(b - 256, b + 256) for b in bounds[1:-1]]))
    idx_t = torch.from_numpy(idx).cuda()
    hs = HostState(to_host(w[idx_t], np.uint16), idx.size)
    for t in range(1, 4):
        g = grads(cfg, specs, n, t)
        tl.set_grads([g[sl] for sl in views])
        h = W.hparams(cfg, step=t)
        B.madd_multi_tensor_step(tl, h)
        for k in range(8):
            lo, hi = bounds[k], bounds[k + 1]
            B.madd_step(w8[lo:hi], "bf16", g[lo:hi], m8[lo:hi], v8[lo:hi], ve8[lo:hi], h,
                        index_base=lo)
        oracle_step("bf16", hs, to_host(g[idx_t]), h, gidx=idx)
        torch.cuda.synchronize()
        for a, b, name in ((w, w8, "w"), (m, m8, "m"), (v, v8, "v"), (ve, ve8, "ve")):
            assert torch.equal(a.view(torch.int16) if a.dtype == torch.float32 else a,
                               b.view(torch.int16) if b.dtype == torch.float32 else b), (name, t)
        assert_state_equal(f"shard boundaries t={t}", to_host(w8[idx_t], np.uint16), hs.w,
                           to_host(m8[idx_t]), hs.m, to_host(v8[idx_t]), hs.v,
                           to_host(ve8[idx_t]), hs.ve)
        del g


def _ceiling():
    L = ctypes.CDLL(_build.PROBE_LIB)
    f = L.madd_ceiling_stream
    f.argtypes = [ctypes.c_void_p] * 5 + [ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p]
    f.restype = ctypes.c_int32
    return f


@pytest.mark.parametrize("state_bytes,n", [(4, 2048 * 37 + 1000), (2, 2048 * 5 + 3), (4, 17)])
def test_ceiling_probe_writes_back_what_it_read(state_bytes, n):
    gen = torch.Generator(device="cuda")
    gen.manual_seed(n)
    sdt = torch.int32 if state_bytes == 4 else torch.int16
    hi = 2**31 - 1 if state_bytes == 4 else 2**15 - 1
    w = torch.randint(-2**15, 2**15 - 1, (n,), dtype=torch.int16, device="cuda", generator=gen)
    g = torch.randn(n, device="cuda", generator=gen)
    st = [torch.randint(-hi, hi, (n,), dtype=sdt, device="cuda", generator=gen) for _ in range(3)]
    before = [t.clone() for t in (w, *st)]
    rc = _ceiling()(w.data_ptr(), g.data_ptr(), st[0].data_ptr(), st[1].data_ptr(),
                    st[2].data_ptr(), state_bytes, n, torch.cuda.current_stream().cuda_stream)
    assert rc == 0
    torch.cuda.synchronize()
    for a, b in zip(before, (w, *st)):
        assert torch.equal(a, b)


def test_stream_modes_move_exactly_their_bytes():
    L = ctypes.CDLL(_build.PROBE_LIB)
    f = L.madd_stream_modes
    f.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                  ctypes.c_void_p]
    f.restype = ctypes.c_int32
    nbytes = 8192 * 37
    gen = torch.Generator(device="cuda")
    gen.manual_seed(5)
    a = torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), dtype=torch.int32, device="cuda",
                      generator=gen)
    b = torch.zeros_like(a)
    st = torch.cuda.current_stream().cuda_stream
    assert f(2, a.data_ptr(), b.data_ptr(), nbytes, st) == 0          # copy
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert f(1, None, b.data_ptr(), nbytes, st) == 0                  # write: word k of 16 B
    torch.cuda.synchronize()
    want = torch.arange(nbytes // 16, device="cuda", dtype=torch.int64).to(torch.int32)
    assert torch.equal(b.view(-1, 4), want[:, None].expand(-1, 4))
    z = torch.zeros_like(a)                                           # XOR 0 never meets the key
    before = b.clone()
    assert f(0, z.data_ptr(), b.data_ptr(), nbytes, st) == 0          # read
    torch.cuda.synchronize()
    assert torch.equal(b, before)
