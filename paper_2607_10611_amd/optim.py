"""``torch.optim`` front end of the M+Adam step (Section 3, Algorithm 2).

A parameter's own storage is its weight storage: a bfloat16 parameter holds
bf16 codes, a float32 one fp32 codes, float8_e4m3fn / float8_e5m2 ones E4M3 /
E5M2 codes.  Each step rounds w' back into that format (to nearest, or
stochastically with draws keyed by seed, step and each element's global
index) and keeps m, v and v_e in the optimizer state, as fp32 or bf16.  Every
update runs in the HIP kernels of libmadd.so: one madd_multi_tensor_step call
per run of consecutive parameters that share a gradient dtype and a step
count, on the current stream; nothing falls back to the CPU.

Global indices: the optimizer's k-th parameter (counting over all groups in
order) starts at the total size of the parameters before it, fixed when it
is added, so its draws do not depend on which other parameters have
gradients in a step, and a rebuilt optimizer over the same parameters draws
the same bits.
"""
from __future__ import annotations

import math
from collections import OrderedDict

import torch

from . import binding as B

# weight dtype -> (storage format, integer view of the codes)
_WEIGHTS = {torch.bfloat16: ("bf16", torch.int16), torch.float32: ("fp32", torch.int32)}
for _name, _fmt in (("float8_e4m3fn", "e4m3"), ("float8_e5m2", "e5m2")):
    if hasattr(torch, _name):
        _WEIGHTS[getattr(torch, _name)] = (_fmt, torch.uint8)
_GRADS = {torch.float32: "fp32", torch.bfloat16: "bf16"}
_STATES = {"fp32": torch.float32, "bf16": torch.int16, "bf16_sr": torch.int16}
# block-scaled master formats -> elements per block
_MASTERS = {"e4m3": 128, "e5m2": 128, "mxfp4": B.MX_BLOCK, "nvfp4": B.NV_BLOCK,
            "nvfp4_current": B.NV_BLOCK}
_SAVED = ("m", "v", "ve", "q", "scales")  # state tensors whose dtype and bits are kept
_HP_KEYS = ("lr_add", "lr_mul", "eps", "tau", "r_max", "eps0", "g_max", "d_mult_max", "w_max",
            "rounding", "seed")


class MAdam(torch.optim.Optimizer):
    """M+Adam with its weights kept in the parameters' low-precision storage.

    lr_add, lr_mul: the additive and multiplicative learning rates (eta_a,
    eta_m); betas: (beta1, beta2); eps; tau: the floor of |w| in the relative
    multiplicative update; r_max, eps0: its clip (-(r_max - eps0), r_max);
    g_max: clip of the normalized exponent gradient; d_mult_max: cap on the
    exponent change (2^+-d); w_max: final clamp of w'; bias_correction;
    rounding: "sr" or "rne"; seed: the stochastic-rounding key; state_format:
    "fp32", "bf16" or "bf16_sr" (bf16 moments rounded to nearest or
    stochastically).

    master_format (per group; default None): keep the master weights of the
    group's bfloat16 parameters in the optimizer state in a block-scaled
    format -- "e4m3" / "e5m2" (blocks of 128, FP16 scales), "mxfp4", "nvfp4"
    (its tensor scale kept) or "nvfp4_current" (derived anew every step,
    which overwrites the fp32 gradient with w') -- encoded from the
    parameters when the state is made (Section 4.2's FP8-master setting and
    its 4-bit analogues).  Each step then writes the bf16 compute copy of the
    new master weights into the parameter (until the first step the
    parameter keeps its own values).  Such parameters need a size that
    is a multiple of the block and 16-byte-aligned storage.

    capturable: the kernels read each group's hyper-parameters from a small
    device buffer, so that a step captured in a graph can be replayed for
    the steps that follow.  Take at least one eager step first (it makes
    the state and caches the launch tables), keep the gradient tensors in
    place (write new gradients into them), and call prepare_replay() before
    each replay: it advances the step counters and writes the next step's
    hyper-parameters.  Every parameter of a group then needs a gradient at
    every step, of one dtype."""

    def __init__(self, params, lr_add: float = 1e-3, lr_mul: float = 1e-3,
                 betas=(0.9, 0.999), eps: float = 1e-8, tau: float = 1e-8, r_max: float = 0.75,
                 eps0: float = 0.0, g_max: float = math.inf, d_mult_max: float = math.inf,
                 w_max: float = math.inf, bias_correction: bool = True, rounding: str = "sr",
                 seed: int = 0, state_format: str = "fp32", master_format: str | None = None,
                 capturable: bool = False):
        if rounding not in B.ROUND:
            raise ValueError(f"rounding must be one of {sorted(B.ROUND)}, not {rounding!r}")
        if state_format not in _STATES:
            raise ValueError(f"state_format must be one of {sorted(_STATES)}, "
                             f"not {state_format!r}")
        if len(tuple(betas)) != 2:
            raise ValueError("betas must be (beta1, beta2)")
        self._check_master(master_format)
        defaults = dict(lr_add=lr_add, lr_mul=lr_mul, betas=tuple(betas), eps=eps, tau=tau,
                        r_max=r_max, eps0=eps0, g_max=g_max, d_mult_max=d_mult_max,
                        w_max=w_max, bias_correction=bool(bias_correction), rounding=rounding,
                        seed=int(seed), state_format=state_format, master_format=master_format)
        self._base = {}          # parameter -> global index of its first element
        self._next_base = 0
        self._lists = OrderedDict()  # marshalled lists of recent runs (LRU)
        self._capturable = bool(capturable)
        self._scalars = {}       # group index -> device buffer of its prepared scalars
        super().__init__(params, defaults)

    @staticmethod
    def _check_master(fmt):
        if fmt is not None and fmt not in _MASTERS:
            raise ValueError(f"master_format must be None or one of {sorted(_MASTERS)}, "
                             f"not {fmt!r}")

    def add_param_group(self, param_group):
        self._check_master(param_group.get("master_format"))
        super().add_param_group(param_group)
        for p in self.param_groups[-1]["params"]:
            if p not in self._base:
                self._base[p] = self._next_base
                self._next_base += p.numel()

    def load_state_dict(self, state_dict):
        """As torch.optim.Optimizer's, except that the moments and any master
        codes and scales keep the dtype and bits they were saved with (the
        base class casts every state tensor to its parameter's dtype)."""
        from itertools import chain
        saved = state_dict["state"]
        super().load_state_dict(state_dict)
        ids = chain.from_iterable(g["params"] for g in state_dict["param_groups"])
        params = chain.from_iterable(g["params"] for g in self.param_groups)
        for pid, p in zip(ids, params):
            for k in _SAVED:
                if pid in saved and k in saved[pid]:
                    self.state[p][k] = saved[pid][k].to(device=p.device, copy=True)
        self._lists.clear()

    @staticmethod
    def _check_param(p, master):
        if master is not None:
            if p.dtype != torch.bfloat16:
                raise TypeError(f"MAdam: parameters with a {master} master hold its bf16 "
                                f"compute copy and must be bfloat16 (got {p.dtype})")
            if p.numel() % _MASTERS[master] != 0:
                raise ValueError(f"MAdam: a {master} master needs a multiple of "
                                 f"{_MASTERS[master]} elements (got {p.numel()})")
            for what, t in (("parameter", p), ("gradient", p.grad)):
                if t.data_ptr() % 16 != 0:
                    raise ValueError(f"MAdam: a block-scaled master needs a 16-byte-aligned "
                                     f"{what}")
            if master == "nvfp4_current" and p.grad.dtype != torch.float32:
                raise TypeError("MAdam: nvfp4_current writes w' over the gradient, which "
                                "must be float32")
        if p.dtype not in _WEIGHTS:
            raise TypeError(f"MAdam: parameters of dtype {p.dtype} have no storage format "
                            f"(supported: {sorted(str(d) for d in _WEIGHTS)})")
        g = p.grad
        if g.is_sparse:
            raise TypeError("MAdam: sparse gradients are not supported")
        if g.dtype not in _GRADS:
            raise TypeError(f"MAdam: gradients of dtype {g.dtype} are not supported "
                            "(float32 or bfloat16)")
        for what, t in (("parameter", p), ("gradient", g)):
            if not t.is_cuda:
                raise ValueError(f"MAdam: every {what} must be a GPU tensor (got {t.device})")
            if not t.is_contiguous():
                raise ValueError(f"MAdam: every {what} must be contiguous")
        if g.shape != p.shape:
            raise ValueError("MAdam: gradient and parameter shapes differ")

    def _state_of(self, p, sfmt: str, master):
        st = self.state[p]
        if not st:
            dt = _STATES[sfmt]
            st["step"] = 0
            st["m"], st["v"], st["ve"] = (torch.empty(p.numel(), dtype=dt, device=p.device)
                                          for _ in range(3))
            B.madd_init_state(st["m"], st["v"], st["ve"], sfmt=sfmt)
            if master is not None:
                n = p.numel()
                st["q"] = torch.empty(math.ceil(n * B.CODE_BYTES[master]), dtype=torch.uint8,
                                      device=p.device)
                st["scales"] = torch.empty(B.scale_bytes(master, n), dtype=torch.uint8,
                                           device=p.device)
                x = p.detach().float().reshape(-1).contiguous()
                B.madd_encode_weights(x, st["q"], master, scales=st["scales"])
        if (master is not None) != ("q" in st):
            raise ValueError("MAdam: a parameter's state does not match its group's "
                             "master_format")
        if st["m"].dtype != _STATES[sfmt] or st["m"].numel() != p.numel():
            raise ValueError(f"MAdam: the state of a parameter does not hold {sfmt} moments of "
                             f"{p.numel()} elements")
        return st

    def _marshal(self, run, sfmt: str, master):
        key = (sfmt, master) + tuple(
            (p.data_ptr(), p.numel(), p.dtype) +
            tuple(t.data_ptr() for k, t in self.state[p].items() if k in _SAVED) for p in run)
        tl = self._lists.get(key)
        gs = [p.grad for p in run]
        if tl is None:
            st = [self.state[p] for p in run]
            ms, vs, ves = ([s[k] for s in st] for k in ("m", "v", "ve"))
            if master is None:
                ws = [p.detach().view(_WEIGHTS[p.dtype][1]).view(-1) for p in run]
                tl = B.TensorList(ws, [_WEIGHTS[p.dtype][0] for p in run], gs, ms, vs, ves,
                                  sfmt=sfmt)
            else:
                copies = [p.detach().view(torch.int16).view(-1) for p in run]
                tl = B.TensorList([s["q"] for s in st], [master] * len(run), gs, ms, vs, ves,
                                  scales=[s["scales"] for s in st], sfmt=sfmt, copies=copies)
            self._lists[key] = tl
            while len(self._lists) > 16:
                self._lists.popitem(last=False)
        else:
            self._lists.move_to_end(key)
            tl.set_grads(gs)
        return tl

    @staticmethod
    def _hparams(group, t):
        hp = {k: group[k] for k in _HP_KEYS}
        b1, b2 = group["betas"]
        hp.update(beta1=b1, beta2=b2, bias_correction=int(group["bias_correction"]), step=t)
        return hp

    def _write_scalars(self, gi, group, t):
        """The group's hyper-parameters for step t into its device buffer
        (ordered on the current stream)."""
        buf = self._scalars.get(gi)
        dev = group["params"][0].device
        if buf is None:
            buf = self._scalars[gi] = torch.empty(int(B.lib().madd_scalars_bytes()),
                                                  dtype=torch.uint8, device=dev)
        raw = torch.frombuffer(bytearray(B.prepare_scalars(self._hparams(group, t))),
                               dtype=torch.uint8)
        buf.copy_(raw)
        return buf

    def _runs(self, group, capturing):
        sfmt = group["state_format"]
        master = group.get("master_format")
        runs, cur, cur_key, end = [], None, None, None
        for p in group["params"]:
            if p.grad is None:
                if self._capturable:
                    raise ValueError("MAdam(capturable=True): every parameter of a group "
                                     "needs a gradient at every step")
                cur = None
                continue
            self._check_param(p, master)
            if capturing and not self.state[p]:
                raise RuntimeError("MAdam: take an eager step before capturing one")
            st = self._state_of(p, sfmt, master)
            key = (_GRADS[p.grad.dtype], st["step"])
            if cur is None or key != cur_key or self._base[p] != end:
                cur, cur_key = [], key
                runs.append((key, cur))
            cur.append(p)
            end = self._base[p] + p.numel()
        if self._capturable and len(runs) > 1:
            raise ValueError("MAdam(capturable=True): the parameters of a group need one "
                             "gradient dtype and one step count")
        return runs

    @torch.no_grad()
    def step(self, closure=None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        capturing = torch.cuda.is_available() and torch.cuda.is_current_stream_capturing()
        if capturing and not self._capturable:
            raise RuntimeError("MAdam: capturing a step needs MAdam(capturable=True)")
        for gi, group in enumerate(self.param_groups):
            sfmt = group["state_format"]
            master = group.get("master_format")
            for (gfmt, t), run in self._runs(group, capturing):
                hp = self._hparams(group, t + 1)
                tl = self._marshal(run, sfmt, master)
                base = self._base[run[0]]
                if self._capturable:
                    # captured: the replays read what prepare_replay() writes
                    buf = self._scalars[gi] if capturing else self._write_scalars(gi, group, t + 1)
                    B.madd_multi_tensor_step_dev(tl, hp, buf, gfmt=gfmt, index_base=base)
                else:
                    B.madd_multi_tensor_step(tl, hp, gfmt=gfmt, index_base=base)
                # the launch is ordered on the current stream: the gradients
                # need no reference past it
                tl.set_grads([None] * tl.n)
                if not capturing:
                    for p in run:
                        self.state[p]["step"] = t + 1
        return loss

    @torch.no_grad()
    def prepare_replay(self):
        """Before replaying a captured step: advance every step counter and
        write the next step's hyper-parameters (capturable optimizers)."""
        if not self._capturable:
            raise RuntimeError("prepare_replay() is for MAdam(capturable=True)")
        for gi, group in enumerate(self.param_groups):
            steps = {self.state[p]["step"] for p in group["params"] if self.state[p]}
            if not steps:
                continue
            if len(steps) > 1 or gi not in self._scalars:
                raise RuntimeError("MAdam: prepare_replay() needs every group stepped together "
                                   "at least once")
            t = steps.pop() + 1
            self._write_scalars(gi, group, t)
            for p in group["params"]:
                self.state[p]["step"] = t
