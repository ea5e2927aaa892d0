"""Adapter distillation (section "Training Objective").

The training loss and its autograd gradient equal the oracle's pinned
KL(pi || pi_hat) and closed-form gradient; on a synthetic teacher whose
next-layer logits are an exact rank-r map of the router input the optimum is
known: KL 0 and perfect recall."""
import numpy as np
import pytest

import oracle as o
from paper_2607_24787_amd import distill


def _torch_case(seed, N=33, D=12, r=4, n=9):
    import torch
    rng = np.random.default_rng(seed)
    X = rng.normal(size=(N, D))
    A, B = 0.6 * rng.normal(size=(r, D)), 0.6 * rng.normal(size=(n, r))
    Z = 2.0 * rng.normal(size=(N, n))
    return X, A, B, Z, torch


@pytest.mark.parametrize("seed", range(3))
def test_kl_loss_and_its_gradient_match_the_oracle(seed):
    X, A, B, Z, torch = _torch_case(seed)
    At = torch.tensor(A, requires_grad=True)
    Bt = torch.tensor(B, requires_grad=True)
    logP = torch.log_softmax(torch.tensor(Z), dim=-1)
    loss = distill.kl_loss(At, Bt, torch.tensor(X), logP.exp(), logP)
    loss.backward()
    assert abs(float(loss.detach()) - o.distill_pair_loss(A, B, X, Z)) < 1e-12
    dA, dB = o.distill_pair_grad(A, B, X, Z)
    np.testing.assert_allclose(At.grad.numpy(), dA, rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(Bt.grad.numpy(), dB, rtol=1e-10, atol=1e-13)


def test_kl_loss_on_the_hand_pair():
    """z_hat = (ln 9, 0) against target logits (0, 0): KL(pi || pi_hat) = ln(5/3)
    (the reverse direction would give 0.368)."""
    import math
    import torch
    A = torch.tensor([[1.0]], dtype=torch.float64)
    B = torch.tensor([[math.log(9.0)], [0.0]], dtype=torch.float64)
    logP = torch.log_softmax(torch.zeros(1, 2, dtype=torch.float64), dim=-1)
    v = float(distill.kl_loss(A, B, torch.ones(1, 1, dtype=torch.float64), logP.exp(), logP))
    assert abs(v - math.log(5.0 / 3.0)) < 1e-15


def test_held_out_loss_reported_by_training_is_the_oracles():
    """distill_adapter's reported held-out KL at the start is the oracle's loss
    of the starting adapter on the same held-out rows (fp32 arithmetic)."""
    import torch
    X, A, B, Z, _ = _torch_case(7, N=200)
    _, _, (start, end) = distill.distill_adapter(X, Z, A, B, steps=20, lr=1e-3, batch=64, seed=3, val_frac=0.25)
    perm = torch.randperm(200, generator=torch.Generator().manual_seed(3))
    vi = perm[:50].numpy()
    want = o.distill_pair_loss(A.astype(np.float32), B.astype(np.float32), X[vi].astype(np.float32),
                               Z[vi].astype(np.float32))
    assert abs(start - want) < 1e-5 * max(1.0, want)
    assert end <= start


def _teacher(seed=0, N=1536, D=32, n=16, r=4, scale=3.0):
    rng = np.random.default_rng(seed)
    U, _ = np.linalg.qr(rng.normal(size=(n, r)))
    V, _ = np.linalg.qr(rng.normal(size=(D, r)))
    sig = np.array([4.0, 3.0, 2.0, 1.5])[:r]
    W = scale * (U * sig) @ V.T                       # [n, D], rank r
    X = rng.normal(size=(N, D)).astype(np.float32)
    return X, (X @ W.T).astype(np.float32), U, sig * scale, V


def test_exact_low_rank_adapter_has_zero_loss():
    X, Z, U, sig, V = _teacher()
    A = (np.sqrt(sig)[:, None] * V.T).astype(np.float32)
    B = (U * np.sqrt(sig)[None, :]).astype(np.float32)
    _, _, (start, end) = distill.distill_adapter(X, Z, A, B, steps=5, lr=1e-6, val_frac=0.0)
    assert start < 1e-6
    assert distill.expert_recall(A, B, X, Z, K=2, M=2) == 1.0


def test_distillation_recovers_the_teacher_from_a_random_start():
    X, Z, U, sig, V = _teacher(seed=1)
    rng = np.random.default_rng(5)
    A0 = (0.1 * rng.normal(size=(4, X.shape[1]))).astype(np.float32)
    B0 = (0.1 * rng.normal(size=(Z.shape[1], 4))).astype(np.float32)
    tr, ho = slice(0, 1280), slice(1280, None)
    before = distill.expert_recall(A0, B0, X[ho], Z[ho], K=2, M=2)
    A, B, (start, end) = distill.distill_adapter(X[tr], Z[tr], A0, B0, steps=1500, lr=2e-2, batch=256)
    assert end < 0.05 * start                        # the KL objective falls by more than 20x
    after = distill.expert_recall(A, B, X[ho], Z[ho], K=2, M=2)
    assert after > 0.9 and after > before + 0.3      # held-out ExpertRecall@K
    assert distill.expert_recall(A, B, X[ho], Z[ho], K=2, M=16) == 1.0   # M = n covers everything


def test_expert_recall_brute_force():
    rng = np.random.default_rng(2)
    X = rng.normal(size=(40, 6))
    A, B = rng.normal(size=(3, 6)), rng.normal(size=(5, 3))
    Z = rng.normal(size=(40, 5))
    for K, M in ((1, 1), (2, 3), (3, 5)):
        want = 0.0
        for i in range(40):
            zh = B @ (A @ X[i])
            top = set(sorted(range(5), key=lambda e: (-Z[i, e], e))[:K])
            pred = set(sorted(range(5), key=lambda e: (-zh[e], e))[:M])
            want += len(top & pred) / K
        assert abs(distill.expert_recall(A, B, X, Z, K, M) - want / 40) < 1e-12
