"""Appendix B's BF16-stored matrix-fitting diagnostic on the GPU.

Minimises the sampled quartic loss of one regime (workloads.toy_regime):
each step draws B entries uniformly with replacement and takes the gradient
of (1/B) sum_k c_i (w_i - w*_i)^4 over the drawn entries,
g_i = (4/B) cnt_i c_i (w_i - w*_i)^3 (madd_toy_gradient), then applies one
of the moment-free update rules (madd_plain_step) with round-to-nearest
BF16 storage.  Both run as the library's HIP kernels; torch draws the
sampled entries and holds the buffers.

The paper writes the loss as c ||W - W*||_F^4 evaluated on sampled entries,
with per-entry c in the mixed regime; the entrywise sampled reading above is
the one consistent with per-entry scales.
"""
from __future__ import annotations

import math

import numpy as np

from . import binding as B
from . import workloads as W

RULES = ("additive", "multiplicative", "combined")


def rule_hparams(rule: str, lr: float, step: int) -> dict:
    hp = dict(W.DEFAULT_HPARAMS, rounding="rne", step=step)
    hp["lr_add"] = lr if rule in ("additive", "combined") else 0.0
    hp["lr_mul"] = lr if rule in ("multiplicative", "combined") else 0.0
    return hp


def run(regime: str, rule: str, lr: float, steps: int = 200, batch: int = W.TOY_N,
        seed: int = 0, device="cuda") -> dict:
    """Run one regime with one rule; returns final weights and summary metrics."""
    import torch

    ws, w0, c = W.toy_regime(regime, seed)
    n = ws.size
    dev = torch.device(device)
    codes = torch.empty(n, dtype=torch.int16, device=dev)
    B.madd_encode_weights(torch.from_numpy(w0).to(dev), codes, "bf16")
    target = torch.from_numpy(ws).to(dev)
    cc = torch.from_numpy(c).to(dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(W.torch_seed(6, 1, seed))
    g = torch.empty(n, dtype=torch.float32, device=dev)
    counts = torch.empty(n, dtype=torch.int32, device=dev)
    for t in range(1, steps + 1):
        idx = torch.randint(0, n, (batch,), generator=gen, device=dev)
        B.madd_toy_gradient(codes, "bf16", target, cc, idx, counts, g)
        B.madd_plain_step(codes, "bf16", g, rule_hparams(rule, lr, t))
    w = codes.view(torch.bfloat16).float().cpu().numpy().astype(np.float64)
    return dict(w=w, target=ws.astype(np.float64), w0=w0.astype(np.float64),
                rel_err=float(np.linalg.norm(w - ws) / np.linalg.norm(ws)),
                sign_agree=float(np.mean(np.sign(w) == np.sign(ws))),
                unchanged=float(np.mean(w == w0)),
                loss=float(np.mean(c * (w - ws) ** 4)),
                loss0=float(np.mean(c * (w0.astype(np.float64) - ws) ** 4)))


def figure3(lr: float = 10.0, steps: int = 200) -> dict:
    """Every regime x rule at one shared learning rate."""
    return {(r, rule): run(r, rule, lr, steps) for r in W.TOY_REGIMES for rule in RULES}


if __name__ == "__main__":
    res = figure3()
    for (r, rule), m in res.items():
        print(f"{r:13s} {rule:15s} rel_err {m['rel_err']:.3f} sign {m['sign_agree']:.2f} "
              f"unchanged {m['unchanged']:.2f} loss/loss0 "
              f"{m['loss'] / m['loss0'] if m['loss0'] else math.nan:.3e}")
