"""Adapter distillation (section "Training Objective").

The adapter of layer l predicts the next layer's routing from the router
input of layer l: pi_hat^{l+1} = softmax(B^l A^l x^l).  It is trained to match
the frozen native router of layer l+1, pi^{l+1} = softmax(z^{l+1}), by
minimising the mean over tokens of KL(pi^{l+1} || pi_hat^{l+1}); only A^l and
B^l change.

This is the offline step before the decode path: the traces (router inputs x
and native router logits z of every layer) come from the device path itself
(moe_layer_forward with prediction off, spp_get_last_router_input,
spp_get_last_logits), and the adapters it returns are bound like any other.
The optimiser follows the paper's implementation details: AdamW with
betas (0.9, 0.999), eps 1e-8, a linear warm-up over the first 3% of steps
then cosine decay, gradient clipping at 0.5.  Learning rate and step count
are set for the size of the synthetic traces.  The arithmetic runs on the
host in fp32 with PyTorch.
"""
from __future__ import annotations

import math
from typing import List, Tuple

import numpy as np


def collect_traces(stack, h_tokens: np.ndarray) -> Tuple[List[np.ndarray], List[np.ndarray]]:
    """Run ``h_tokens`` [T, B, D] (storage) through every layer with prediction
    off; returns per layer the router inputs x [T*B, D] and logits z [T*B, n]."""
    from . import spp
    cfg = stack.cfg
    B = h_tokens.shape[1]
    X: List[list] = [[] for _ in range(cfg.L)]
    Z: List[list] = [[] for _ in range(cfg.L)]
    stack.reset()
    for t in range(h_tokens.shape[0]):
        stack.upload_hidden(h_tokens[t], 0)
        src = 0
        for l in range(cfg.L):
            stack.layer(l, src, 1 - src, -1, B)
            X[l].append(spp.spp_get_last_router_input(stack.ctx, B, cfg.D))
            Z[l].append(spp.spp_get_last_logits(stack.ctx, B, cfg.n))
            src = 1 - src
    return [np.concatenate(x) for x in X], [np.concatenate(z) for z in Z]


def kl_loss(A, Bm, X, P, logP):
    """Mean over rows of KL(P || softmax(X A^T B^T)) (torch tensors)."""
    import torch
    logq = torch.log_softmax((X @ A.T) @ Bm.T, dim=-1)
    return (P * (logP - logq)).sum(dim=-1).mean()


def distill_adapter(X: np.ndarray, Z_next: np.ndarray, A0: np.ndarray, B0: np.ndarray, steps: int = 1500,
                    lr: float = 2e-3, batch: int = 256, seed: int = 0, val_frac: float = 0.1, eval_every: int = 50):
    """Train one adapter (A [r,D], B [n,r], starting from A0, B0) on pairs
    (x^l, z^{l+1}); a fraction val_frac of the pairs is held out and the
    parameters with the lowest held-out KL are kept (the start included).
    Returns (A, B, (held-out KL at the start, held-out KL kept))."""
    import torch
    g = torch.Generator().manual_seed(seed)
    Xa = torch.tensor(np.asarray(X, dtype=np.float32))
    Za = torch.tensor(np.asarray(Z_next, dtype=np.float32))
    perm = torch.randperm(Xa.shape[0], generator=g)
    nv = int(val_frac * Xa.shape[0]) if val_frac > 0 else 0
    vi, ti = perm[:nv], perm[nv:]
    Xt, Zt = Xa[ti], Za[ti]
    logP = torch.log_softmax(Zt, dim=-1)
    P = logP.exp()
    Xv = Xa[vi] if nv else Xt
    logPv = torch.log_softmax(Za[vi], dim=-1) if nv else logP
    Pv = logPv.exp()
    A = torch.nn.Parameter(torch.tensor(np.asarray(A0, dtype=np.float32)))
    Bm = torch.nn.Parameter(torch.tensor(np.asarray(B0, dtype=np.float32)))
    opt = torch.optim.AdamW([A, Bm], lr=lr, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.0)
    warm = max(1, int(0.03 * steps))

    def factor(step):
        if step < warm:
            return (step + 1) / warm
        return 0.5 * (1.0 + math.cos(math.pi * (step - warm) / max(1, steps - warm)))
    sched = torch.optim.lr_scheduler.LambdaLR(opt, factor)
    with torch.no_grad():
        start = float(kl_loss(A, Bm, Xv, Pv, logPv))
    best = (start, A.detach().clone(), Bm.detach().clone())
    n = Xt.shape[0]
    for step in range(steps):
        idx = torch.randint(0, n, (min(batch, n),), generator=g)
        loss = kl_loss(A, Bm, Xt[idx], P[idx], logP[idx])
        opt.zero_grad()
        loss.backward()
        torch.nn.utils.clip_grad_norm_([A, Bm], 0.5)
        opt.step()
        sched.step()
        if (step + 1) % eval_every == 0 or step + 1 == steps:
            with torch.no_grad():
                v = float(kl_loss(A, Bm, Xv, Pv, logPv))
            if v < best[0]:
                best = (v, A.detach().clone(), Bm.detach().clone())
    return best[1].numpy(), best[2].numpy(), (start, best[0])


def expert_recall(A: np.ndarray, Bm: np.ndarray, X: np.ndarray, Z_next: np.ndarray, K: int, M: int) -> float:
    """Mean over rows of |Top_K(z^{l+1}) cap Top_M(B A x^l)| / K (ExpertRecall@M
    at batch 1, where the priority order equals the order of B A x)."""
    zh = (np.asarray(X, dtype=np.float64) @ np.asarray(A, dtype=np.float64).T) @ np.asarray(Bm, dtype=np.float64).T
    tgt = np.argsort(-np.asarray(Z_next, dtype=np.float64), axis=1, kind="stable")[:, :K]
    pred = np.argsort(-zh, axis=1, kind="stable")[:, :M]
    hit = [len(set(tgt[i].tolist()) & set(pred[i].tolist())) for i in range(tgt.shape[0])]
    return float(np.mean(hit)) / K
