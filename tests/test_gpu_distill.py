"""Adapter distillation (section "Training Objective") on the device path.

The traces the distillation trains on (router inputs x^l and native router
logits z^{l+1}) are read back from the device and match the oracle's; adapters
distilled on the oracle's traces, bound to the device, keep the lock-step
parity with the oracle given the same stored adapter values (selections,
priorities, prefetch sets and slot tables exact; outputs within tolerance).
"""
import sys

import numpy as np
import pytest

import oracle as o
import workload as w
from workload import gen

pytestmark = pytest.mark.gpu


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _oracle_traces(cfg, W, h0, tokens):
    """Per layer: router inputs x [tokens*B, D] and logits z [tokens*B, n] of an OFF decode."""
    ref = o.run_decode(cfg, W, h0, M_max=-1, tokens=tokens, keep_x=True)
    X = [[] for _ in range(cfg.L)]
    Z = [[] for _ in range(cfg.L)]
    for st in ref.steps:
        X[st.l].append(st.x)
        Z[st.l].append(st.z)
    return [np.concatenate(x) for x in X], [np.concatenate(z) for z in Z]


def test_collect_traces_match_the_oracle(torch_cuda):
    """fp32 stack, free running: the device's trace equals the oracle's."""
    from paper_2607_24787_amd import distill
    from paper_2607_24787_amd.model import OffloadedMoEStack
    cfg = w.get("c0").with_(tokens=8)
    h0 = gen.hidden_states(cfg)
    Xo, Zo = _oracle_traces(cfg, o.OracleWeights(cfg), h0, cfg.tokens)
    st = OffloadedMoEStack(cfg)
    try:
        _log("[distill traces] c0, 8 tokens")
        X, Z = distill.collect_traces(st, h0)
    finally:
        st.close()
    for l in range(cfg.L):
        assert X[l].shape == Xo[l].shape and Z[l].shape == Zo[l].shape
        assert np.max(np.abs(X[l] - Xo[l])) <= 1e-5 * np.max(np.abs(Xo[l]))
        assert np.max(np.abs(Z[l] - Zo[l])) <= 1e-5 * np.max(np.abs(Zo[l]))


def test_lockstep_parity_with_distilled_adapters(torch_cuda):
    """Recall-calibrated DeepSeek-shaped layers: distill both adapters on the
    oracle's traces of 48 tokens, bind them, and run the lock-step."""
    from lockstep import run_lockstep
    from paper_2607_24787_amd import distill
    from paper_2607_24787_amd.model import OffloadedMoEStack
    from workload.gen import f32_to_bf16_bits
    cfg = w.get("c3p").with_(L=3)
    W = o.OracleWeights(cfg)
    h_train = gen.hidden_states(cfg.with_(seed=cfg.seed + 100), tokens=48)
    _log("[distill lockstep] oracle traces, 48 tokens")
    X, Z = _oracle_traces(cfg, W, h_train, 48)
    stored = {}
    for l in range(cfg.L - 1):
        A0, B0 = (np.asarray(m, np.float32) for m in W.adapter(l))
        A, B, (k0, k1) = distill.distill_adapter(X[l], Z[l + 1], A0, B0, steps=150, lr=2e-3, batch=32, seed=l)
        _log(f"[distill lockstep] layer {l}: held-out KL {k0:.5f} -> {k1:.5f}")
        assert k1 <= k0
        stored[l] = (f32_to_bf16_bits(A), f32_to_bf16_bits(B))
        assert not np.array_equal(stored[l][0], f32_to_bf16_bits(A0))   # the adapter did change
    values = lambda l: tuple(o.decode(m, "bf16") for m in stored[l])  # noqa: E731
    st = OffloadedMoEStack(cfg, adapter_values=values)
    try:
        rep = run_lockstep(st, cfg, 4, 2, adapter_override=values)
    finally:
        st.close()
    _log(f"[distill lockstep] layers={rep.layers} exempt={len(rep.exempt)} max_rel_h={rep.max_rel_h:.3g} "
         f"max_ulp_h={rep.max_ulp_h:.3g} s={rep.max_err_s:.3g}")
    assert rep.max_ulp_h <= 1.0 + 1e-9
    assert rep.max_err_g <= 1e-5
    assert len(rep.exempt) <= 1
    assert rep.prefetched > 0
