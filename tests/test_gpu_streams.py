"""Asynchronous use of the C ABI (GPU): two tensor lists stepped on two HIP
streams at once, and from two host threads at once, give the same bits as
stepping them one after the other on one stream (every call only enqueues
work on its stream; the descriptor-table cache is shared under a lock)."""
import threading

import numpy as np
import pytest
import torch

import oracle
from paper_2607_10611_amd import binding as B
from paper_2607_10611_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()
    yield
    torch.cuda.synchronize()


def make_list(seed, sizes, fmts):
    rng = np.random.default_rng(seed)
    ws, ss, cs, ms, vs, ves = [], [], [], [], [], []
    for n, f in zip(sizes, fmts):
        x = rng.normal(0, 0.02, n).astype(np.float32)
        if f == "bf16":
            ws.append(torch.from_numpy(oracle.encode_array("bf16", x).view(np.int16)).cuda())
            ss.append(None)
            cs.append(None)
        else:
            q, s = oracle.encode_nv(x) if f == "nvfp4" else oracle.encode_mx(x)
            ws.append(torch.from_numpy(q).cuda())
            ss.append(torch.from_numpy(s).cuda())
            cs.append(torch.zeros(n, dtype=torch.int16, device="cuda"))
        for lst in (ms, vs, ves):
            lst.append(torch.zeros(n, device="cuda"))
    return dict(w=ws, s=ss, c=cs, m=ms, v=vs, ve=ves, fmts=fmts, sizes=sizes)


def clone(L):
    c = lambda xs: [x.clone() if x is not None else None for x in xs]  # noqa: E731
    return dict(w=c(L["w"]), s=c(L["s"]), c=c(L["c"]), m=c(L["m"]), v=c(L["v"]), ve=c(L["ve"]),
                fmts=L["fmts"], sizes=L["sizes"])


def grads(seed, sizes, steps):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return [[torch.randn(n, device="cuda", generator=g) * 1e-3 for n in sizes]
            for _ in range(steps)]


def tlist(L, gs):
    return B.TensorList(L["w"], L["fmts"], gs, L["m"], L["v"], L["ve"], scales=L["s"], copies=L["c"])


def same(A, Bl):
    for k in ("w", "s", "c", "m", "v", "ve"):
        for a, b in zip(A[k], Bl[k]):
            if a is not None:
                assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), k


SIZES = ([8192 * 9 + 48, 4096, 2048 * 33], [4096 * 5 + 32, 1024 * 3, 16 * 999])
FMTS = (["nvfp4", "bf16", "mxfp4"], ["mxfp4", "bf16", "nvfp4"])
STEPS = 4


def test_two_streams_at_once_equal_one_stream_in_turn():
    lists = [make_list(5 + k, SIZES[k], FMTS[k]) for k in range(2)]
    refs = [clone(L) for L in lists]
    gs = [grads(100 + k, SIZES[k], STEPS) for k in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for t in range(1, STEPS + 1):
        for k in range(2):
            h = W.hparams("c2", step=t)
            B.madd_multi_tensor_step(tlist(lists[k], gs[k][t - 1]), h, stream=streams[k],
                                     index_base=1000 * k)
    torch.cuda.synchronize()
    for k in range(2):
        for t in range(1, STEPS + 1):
            B.madd_multi_tensor_step(tlist(refs[k], gs[k][t - 1]), W.hparams("c2", step=t),
                                     index_base=1000 * k)
    torch.cuda.synchronize()
    for k in range(2):
        same(lists[k], refs[k])


def test_two_host_threads_at_once_equal_one_thread_in_turn():
    lists = [make_list(7 + k, SIZES[k], FMTS[k]) for k in range(2)]
    refs = [clone(L) for L in lists]
    gs = [grads(200 + k, SIZES[k], STEPS) for k in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    errors = []

    def run(k):
        try:
            for t in range(1, STEPS + 1):
                B.madd_multi_tensor_step(tlist(lists[k], gs[k][t - 1]), W.hparams("c2", step=t),
                                         stream=streams[k], index_base=1000 * k)
        except Exception as e:  # reported below
            errors.append(e)

    threads = [threading.Thread(target=run, args=(k,)) for k in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for k in range(2):
        for t in range(1, STEPS + 1):
            B.madd_multi_tensor_step(tlist(refs[k], gs[k][t - 1]), W.hparams("c2", step=t),
                                     index_base=1000 * k)
    torch.cuda.synchronize()
    for k in range(2):
        same(lists[k], refs[k])
