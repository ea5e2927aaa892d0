"""Pins of the CPU oracle to things other than itself (no GPU needed).

Each test checks an oracle function against brute force, a closed form, an
independent library routine (torch / scipy), an invariant the paper states, or
a hand-worked trace, so that a plausible slip in the oracle (a dropped term, a
wrong sign or index, a transposed operand, a wrong tie rule) fails here.
"""
import itertools
import math

import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F

import oracle as o
import workload as w
from workload import gen


# ---------------------------------------------------------------- top-k ----

def _brute_top_k(v, k):
    """Definition by pairwise comparison: a beats b iff v[a] > v[b] or (equal and a < b)."""
    n = len(v)
    beats = lambda a, b: v[a] > v[b] or (v[a] == v[b] and a < b)
    best = None
    for combo in itertools.permutations(range(n), k):
        ok = all(beats(combo[i], combo[i + 1]) for i in range(k - 1))
        rest = [e for e in range(n) if e not in combo]
        ok = ok and all(beats(combo[-1], e) for e in rest) if k else ok
        if ok:
            assert best is None
            best = list(combo)
    return best


@pytest.mark.parametrize("seed", range(40))
def test_top_k_matches_brute_force_with_ties(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 7))
    v = rng.integers(-2, 3, size=n).astype(np.float32)     # many ties
    for k in range(0, n + 1):
        assert o.top_k(v, k).tolist() == _brute_top_k(v, k)


def test_top_k_lowest_index_wins_tie():
    assert o.top_k(np.array([1.0, 3.0, 3.0, 2.0, 3.0]), 2).tolist() == [1, 2]


# --------------------------------------------------- elementary functions --

def test_softmax_against_scipy_and_shift_invariance():
    rng = np.random.default_rng(1)
    v = rng.normal(size=(4, 17)) * 3
    np.testing.assert_allclose(o.softmax(v), scipy.special.softmax(v, axis=-1), rtol=1e-13, atol=0)
    np.testing.assert_allclose(o.softmax(v + 123.0), o.softmax(v), rtol=1e-12, atol=0)
    np.testing.assert_allclose(o.softmax(v).sum(-1), 1.0, rtol=1e-14)


def test_silu_against_torch():
    v = np.linspace(-20, 20, 401)
    np.testing.assert_allclose(o.silu(v), F.silu(torch.tensor(v, dtype=torch.float64)).numpy(), rtol=1e-14, atol=1e-300)


def test_rms_normalize_closed_form():
    rng = np.random.default_rng(2)
    u = rng.normal(size=(3, 64)) * 5
    eps = 1e-6
    x = o.rms_normalize(u, eps)
    m = np.mean(u * u, axis=-1)
    np.testing.assert_allclose(np.mean(x * x, axis=-1), m / (m + eps), rtol=1e-13)
    np.testing.assert_allclose(x / u, (1 / np.sqrt(m + eps))[:, None] * np.ones_like(u), rtol=1e-13)


def test_bf16_encode_hand_ties_and_torch():
    # hand-worked ties: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7 -> even (1.0);
    # 1 + 3*2^-8 lies halfway between 1 + 2^-7 and 1 + 2^-6 -> even (1 + 2^-6).
    vals = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 0.0, 2.0 ** -20])
    expect = [0x3F80, 0x3F82, 0xBF80, 0x0000, 0x3580]
    assert o.encode(vals, "bf16").tolist() == expect
    rng = np.random.default_rng(3)
    v = rng.normal(size=5000).astype(np.float32).astype(np.float64)   # fp32-exact: no double rounding
    ours = o.encode(v, "bf16")
    ref = torch.tensor(v, dtype=torch.float32).to(torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)
    assert np.array_equal(ours, ref)
    np.testing.assert_array_equal(o.decode(ours, "bf16"),
                                  torch.tensor(v, dtype=torch.float32).to(torch.bfloat16).double().numpy())


# ------------------------------------------------------ routing + adapter --

def _torch_layer(u, Wr, K, experts, shared, eps, proj=None):
    """Textbook MoE block built from torch library routines (no oracle code)."""
    u = torch.tensor(u, dtype=torch.float64)
    if proj is not None:
        u = u + F.linear(u * torch.rsqrt(u.pow(2).mean(-1, keepdim=True) + eps), torch.tensor(proj))
    x = u * torch.rsqrt(u.pow(2).mean(-1, keepdim=True) + eps)
    logits = F.linear(x, torch.tensor(Wr)).float().double()
    top = torch.topk(logits, K, dim=-1, sorted=True)
    p = torch.softmax(logits, dim=-1)
    gsel = torch.gather(p, 1, top.indices)
    gsel = (gsel / gsel.sum(-1, keepdim=True)).float().double()
    y = torch.zeros_like(u)
    for b in range(u.shape[0]):
        for k in range(K):
            Wg, Wu, Wd = (torch.tensor(m, dtype=torch.float64) for m in experts[int(top.indices[b, k])])
            y[b] += gsel[b, k] * F.linear(F.silu(F.linear(x[b], Wg)) * F.linear(x[b], Wu), Wd)
        for (Wg, Wu, Wd) in shared:
            Wg, Wu, Wd = (torch.tensor(m, dtype=torch.float64) for m in (Wg, Wu, Wd))
            y[b] += F.linear(F.silu(F.linear(x[b], Wg)) * F.linear(x[b], Wu), Wd)
    return top.indices.numpy(), gsel.numpy(), (u + y).numpy(), x.numpy()


@pytest.mark.parametrize("has_proj,n_shared", [(False, 0), (True, 0), (False, 2)])
def test_layer_against_torch_textbook_block(has_proj, n_shared):
    cfg = w.MoEConfig(name="t", L=2, D=96, n=12, K=3, I=40, r=8, S=12, windows=(1,), tokens=3,
                      batch=3, dtype="f32", has_proj=has_proj, n_shared=n_shared, seed=7)
    W = o.OracleWeights(cfg)
    h = o.decode(gen.hidden_states(cfg)[0], "f32") * 1.7
    cache = o.SlotCache(cfg.S, cfg.n, list(range(cfg.n)))
    u, x = o.layer_prologue(cfg, W, 0, h)
    T, g, z = o.route(W.router(0), x, cfg.K)
    assert cache.on_demand(o.batch_demand(T), 1) == []           # all resident: nothing to load
    out = o.moe_output(cfg, W, 0, cache, u, x, T, g)
    experts = [W.expert(0, e) for e in range(cfg.n)]
    shared = [W.shared(0, j) for j in range(cfg.n_shared)]
    tT, tg, tout, tx = _torch_layer(h, W.router(0), cfg.K, experts, shared, cfg.rms_eps,
                                    W.proj(0) if has_proj else None)
    np.testing.assert_allclose(x, tx, rtol=1e-13, atol=1e-15)
    assert np.array_equal(T, tT)
    np.testing.assert_allclose(g, tg, rtol=1e-7)
    np.testing.assert_allclose(out, tout, rtol=1e-11, atol=1e-12)


def test_expert_ffn_against_torch():
    rng = np.random.default_rng(4)
    Wg, Wu = rng.normal(size=(30, 20)), rng.normal(size=(30, 20))
    Wd = rng.normal(size=(20, 30))
    x = rng.normal(size=20)
    ref = F.linear(F.silu(F.linear(torch.tensor(x), torch.tensor(Wg))) * F.linear(torch.tensor(x), torch.tensor(Wu)),
                   torch.tensor(Wd)).numpy()
    np.testing.assert_allclose(o.expert_ffn(Wg, Wu, Wd, x), ref, rtol=1e-12)
    # a gate row orthogonal to x switches its unit off exactly: silu(0) = 0
    Wg2 = Wg.copy()
    Wg2[5] -= (Wg2[5] @ x) / (x @ x) * x
    Wd2 = np.zeros_like(Wd)
    Wd2[:, 5] = 1.0
    assert abs(o.expert_ffn(Wg2, Wu, Wd2, x)).max() < 1e-12


def test_expert_ffn_rows_are_the_one_token_values():
    """The row form (tokens routed to one expert at once) against torch's
    batched F.linear and against the one-token form, row by row."""
    rng = np.random.default_rng(7)
    Wg, Wu = rng.normal(size=(30, 20)), rng.normal(size=(30, 20))
    Wd = rng.normal(size=(20, 30))
    X = rng.normal(size=(5, 20))
    got = o.expert_ffn(Wg, Wu, Wd, X)
    Xt = torch.tensor(X)
    ref = F.linear(F.silu(F.linear(Xt, torch.tensor(Wg))) * F.linear(Xt, torch.tensor(Wu)), torch.tensor(Wd)).numpy()
    assert got.shape == (5, 20)
    np.testing.assert_allclose(got, ref, rtol=1e-12)
    for i in range(5):
        np.testing.assert_allclose(got[i], o.expert_ffn(Wg, Wu, Wd, X[i]), rtol=1e-12)


def test_route_gates_and_adapter_scores_invariants():
    rng = np.random.default_rng(5)
    B, D, n, r, K = 5, 32, 10, 4, 3
    Wr, A, Bm = rng.normal(size=(n, D)), rng.normal(size=(r, D)), rng.normal(size=(n, r))
    x = rng.normal(size=(B, D))
    T, g, z = o.route(Wr, x, K)
    np.testing.assert_allclose(g.sum(-1), 1.0, rtol=1e-6)
    assert np.all(np.diff(g, axis=1) <= 0)             # descending logits -> descending gates
    assert np.array_equal(z, z.astype(np.float32).astype(np.float64))
    zhat, pi, s = o.adapter_scores(A, Bm, x)
    np.testing.assert_allclose(pi.sum(-1), 1.0, rtol=1e-14)
    np.testing.assert_allclose(s.sum(), B, rtol=1e-6)     # sum_e s_e = |Omega|
    ref = torch.softmax(torch.tensor(zhat), -1).sum(0).float().double().numpy()
    np.testing.assert_allclose(s, ref, rtol=1e-7)
    # z_hat = B (A x): against a single fused product (B A) x
    np.testing.assert_allclose(zhat, x @ (Bm @ A).T, rtol=1e-6, atol=1e-6)


def test_adapter_param_count_matches_generated_arrays():
    for name in ("c0", "c1", "c3"):
        cfg = w.get(name)
        count = 0
        for l in range(cfg.L - 1) if cfg.L <= 2 else range(1):
            A, B = gen.adapter_weights(cfg, l)
            count += A.size + B.size
        per_pair = cfg.r * (cfg.D + cfg.n)
        assert count == per_pair * (min(cfg.L - 1, 1) if cfg.L > 2 else cfg.L - 1)
        assert o.adapter_param_count(cfg.L, cfg.r, cfg.D, cfg.n) == (cfg.L - 1) * per_pair
    # 48-layer Qwen-shaped stack at r = 64: 47 * 64 * 2176
    assert o.adapter_param_count(48, 64, 2048, 128) == 6_545_408


# --------------------------------------------------------------- budget ----

def test_prefetch_budget_rule():
    assert o.prefetch_budget(300.0, 150.0, 128) == 2
    assert o.prefetch_budget(299.9, 150.0, 128) == 1
    assert o.prefetch_budget(0.0, 150.0, 128) == 0
    assert o.prefetch_budget(-5.0, 150.0, 128) == 0
    assert o.prefetch_budget(1e9, 1.0, 128) == 128
    for bad in [(1.0, 0.0), (1.0, -1.0), (float("nan"), 1.0), (1.0, float("inf")), (float("inf"), 1.0)]:
        with pytest.raises(o.BudgetError):
            o.prefetch_budget(bad[0], bad[1], 8)
    rng = np.random.default_rng(6)
    for _ in range(200):
        W_, c = rng.uniform(0, 1000), rng.uniform(1, 300)
        m = o.prefetch_budget(W_, c, 64)
        assert m * c <= W_ + 1e-9 and ((m + 1) * c > W_ or m == 64)
        assert o.prefetch_budget(W_ + 50, c, 64) >= m          # monotone in the window
        assert o.prefetch_budget(W_, c + 10, 64) <= m          # antitone in the cost


@pytest.mark.parametrize("seed", range(30))
def test_select_prefetch_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 8))
    s = rng.integers(0, 4, size=n).astype(np.float64) / 4      # ties
    occ = rng.random(n) < 0.4
    for M in range(0, n + 2):
        P = o.select_prefetch(s, occ, M)
        elig = [e for e in range(n) if not occ[e]]
        assert len(P) == min(max(M, 0), len(elig))
        assert not any(occ[e] for e in P)
        beats = lambda a, b: s[a] > s[b] or (s[a] == s[b] and a < b)
        assert all(beats(P[i], P[i + 1]) for i in range(len(P) - 1))
        assert all(beats(P[-1], e) for e in elig if e not in P) if P else True


# ---------------------------------------------------------- slot cache -----

def test_slot_cache_hand_worked_trace():
    """Expected tables derived by hand from the replacement rules in SlotCache's docstring."""
    c = o.SlotCache(3, 6, [0, 1, 2])                      # table [0,1,2], stamps [0,0,0]
    # tau=1, need {1,4}: miss 4; victims exclude needed {1,4}: slots 0 (st 0), 2 (st 0) -> slot 0
    assert c.on_demand([4, 1], 1) == [(4, 0, 0)]
    assert c.expert.tolist() == [4, 1, 2] and c.stamp.tolist() == [1, 1, 0]
    # tau=2, need {2,3,5}: miss 3 -> min(stamp,slot) over {slot0 (1), slot1 (1)} = slot 0;
    # miss 5 -> only slot 1 holds an unneeded expert
    assert c.on_demand([5, 3, 2], 2) == [(3, 0, 4), (5, 1, 1)]
    assert c.expert.tolist() == [3, 5, 2] and c.stamp.tolist() == [2, 2, 2]
    # prefetch at tau=2: every slot is stamped 2 (not before the step) -> nothing placed
    assert c.prefetch([0, 1], 2) == []
    # prefetch at tau=3 in order [0,4,1]: slots 0, 1, 2 in turn (all stamped 2, lowest slot first)
    assert c.prefetch([0, 4, 1], 3) == [(0, 0, 3), (4, 1, 5), (1, 2, 2)]
    assert c.expert.tolist() == [0, 4, 1] and c.stamp.tolist() == [3, 3, 3]
    # tau=4, need {4,5}: miss 5; unneeded slots 0 (st 3) and 2 (st 3) -> slot 0
    assert c.on_demand([4, 5], 4) == [(5, 0, 0)]
    assert c.expert.tolist() == [5, 4, 1] and c.stamp.tolist() == [4, 4, 3]

    e = o.SlotCache(3, 8, [7])                            # [7, EMPTY, EMPTY]
    assert e.on_demand([2, 7], 1) == [(2, 1, o.EMPTY)]    # lowest EMPTY slot first
    assert e.expert.tolist() == [7, 2, -1] and e.stamp.tolist() == [1, 1, 0]
    # prefetch at tau=1: 5 takes the EMPTY slot 2; 6 finds no slot stamped before 1 -> stop
    assert e.prefetch([5, 6], 1) == [(5, 2, -1)]
    assert e.expert.tolist() == [7, 2, 5]

    # demand larger than S runs in rounds.  S=2, n=6, table [0,1] (stamps 0), need {1,2,3,4}:
    # round 0: miss 2 takes slot 0 (expert 0 is not needed); no victim is left for 3
    #          (slot 0 holds 2, slot 1 holds 1, both needed and not yet run) -> run [1, 2];
    # round 1: victims are slots whose expert already ran, lowest index first:
    #          3 -> slot 0 (evicts 2), 4 -> slot 1 (evicts 1) -> run [3, 4]; stamps of both -> 1
    r = o.SlotCache(2, 6, [0, 1])
    assert r.on_demand([4, 3, 2, 1], 1) == [(2, 0, 0), (3, 0, 2), (4, 1, 1)]
    assert r.rounds == [[1, 2], [3, 4]]
    assert r.run_slot == {1: 1, 2: 0, 3: 0, 4: 1}
    assert r.expert.tolist() == [3, 4] and r.stamp.tolist() == [1, 1]


# ------------------------------------------------------- decode loop ------

def _small_cfg(**kw):
    base = dict(name="s", L=3, D=64, n=10, K=3, I=24, r=6, S=5, windows=(1,), tokens=12,
                dtype="f32", seed=11)
    base.update(kw)
    return w.MoEConfig(**base)


def _adapter_variants(cfg, W):
    rng = np.random.default_rng(9)
    def zero(l):
        return np.zeros((cfg.r, cfg.D)), np.zeros((cfg.n, cfg.r))
    def rand(l):
        return rng.normal(size=(cfg.r, cfg.D)), rng.normal(size=(cfg.n, cfg.r))
    def reverse(l):
        A, B = W.adapter(l)
        return A, -B
    return {"svd": None, "zero": zero, "random": rand, "reversed": reverse}


def test_router_preservation_outputs_independent_of_policy():
    """Outputs never depend on M_max, the slot count or the adapter (paper: the
    native router stays authoritative; missing experts are loaded on demand)."""
    cfg = _small_cfg(batch=2, S=7)
    h0 = gen.hidden_states(cfg)
    W0 = o.OracleWeights(cfg)
    ref = np.stack(o.run_decode(cfg, W0, h0, M_max=-1).outputs)
    for name, ov in _adapter_variants(cfg, W0).items():
        W = o.OracleWeights(cfg, adapter_override=ov)
        for S in (cfg.K - 1, cfg.K * 2, 7, cfg.n):          # K-1: two-token demand runs in rounds
            for M in (0, 1, 2, 4, cfg.n):
                res = o.run_decode(cfg, W, h0, M_max=M, S=S)
                assert np.array_equal(np.stack(res.outputs), ref), (name, S, M)
                for st in res.steps:
                    table = st.table_after_demand
                    held = table[table != o.EMPTY]
                    assert len(set(held.tolist())) == len(held)            # no duplicates
                    if len(set(np.asarray(st.T).ravel().tolist())) <= S:
                        assert set(np.asarray(st.T).ravel().tolist()) <= set(held.tolist())
                    if len(set(np.asarray(st.T).ravel().tolist())) <= S:
                        for e, slot, ev in st.loads:
                            assert ev not in set(np.asarray(st.T).ravel().tolist())   # victim not needed
                    assert len(st.P) <= max(M, 0)
                    if st.P:
                        placed = [e for e, _, _ in st.P]
                        assert len(set(placed)) == len(placed)
                assert 0.0 <= res.ready_recall <= 1.0


def test_all_resident_and_no_prefetch_special_cases():
    cfg = _small_cfg()
    h0 = gen.hidden_states(cfg)
    W = o.OracleWeights(cfg)
    full = o.run_decode(cfg, W, h0, M_max=2, S=cfg.n)
    assert full.ready_recall == 1.0 and full.loads == 0 and full.prefetched == 0
    off = o.run_decode(cfg, W, h0, M_max=-1)
    pred0 = o.run_decode(cfg, W, h0, M_max=0)
    assert pred0.prefetched == 0
    assert pred0.ready_recall == off.ready_recall and pred0.loads == off.loads


def test_closed_form_exact_adapter_gives_perfect_recall():
    """Noise 0, rank r >= rank(W^{l+1}), zero down projections, no stand-in:
    h^{l+1} = h^l, so x^{l+1} = x^l and z_hat = W^{l+1} x^l = z^{l+1}; then
    R@K = 1, R@K/2 = 1/2 (the paper's maximum for half the budget) and R@(K+2) = 1."""
    cfg = w.get("c0")

    class ZeroDown(o.OracleWeights):
        def expert(self, l, e):
            Wg, Wu, Wd = super().expert(l, e)
            return Wg, Wu, np.zeros_like(Wd)

    W = ZeroDown(cfg, adapter_override=lambda l: tuple(
        o.decode(a, cfg.dtype) for a in gen.adapter_weights(cfg, l, noise=0.0)))
    res = o.run_decode(cfg, W, gen.hidden_states(cfg), M_max=1)
    K = cfg.K
    assert res.expert_recall[K] == 1.0
    assert res.expert_recall[K // 2] == 0.5
    assert res.expert_recall[K + 2] == 1.0


def test_metrics_recomputed_from_step_records():
    cfg = _small_cfg(batch=2, L=3, S=7)
    h0 = gen.hidden_states(cfg)
    W = o.OracleWeights(cfg)
    res = o.run_decode(cfg, W, h0, M_max=2)
    K, Ms = cfg.K, sorted(res.expert_recall)
    by_tl = {(s.t, s.l): s for s in res.steps}
    num = {m: 0 for m in Ms}
    ready, cnt = 0, 0
    for (t, l), st in by_tl.items():
        if l == 0:
            continue
        prev = by_tl[(t, l - 1)]
        for b in range(cfg.batch):
            Tb = set(int(e) for e in st.T[b])
            for m in Ms:
                order = sorted(range(cfg.n), key=lambda e: (-prev.s[e], e))[:m]
                num[m] += len(Tb & set(order))
            avail = set(int(e) for e in prev.next_table_after_prefetch if e != o.EMPTY)
            ready += len(Tb & avail)
            cnt += 1
    for m in Ms:
        assert res.expert_recall[m] == pytest.approx(num[m] / (cnt * K))
    assert res.ready_recall == pytest.approx(ready / (cnt * K))
    assert res.expert_recall[Ms[0]] <= res.expert_recall[Ms[1]] <= res.expert_recall[Ms[2]]
    assert res.expert_recall[Ms[0]] <= 0.5 + 1e-12          # K/2 candidates cover at most half
    # candidate set of all n experts covers everything
    for st in res.steps:
        if st.s is not None:
            assert set(o.candidate_set(st.s, cfg.n).tolist()) == set(range(cfg.n))


def test_layer_step_matches_decode_loop():
    cfg = _small_cfg()
    h0 = gen.hidden_states(cfg)
    W = o.OracleWeights(cfg)
    res = o.run_decode(cfg, W, h0, M_max=2, tokens=3)
    caches = [o.SlotCache(cfg.S, cfg.n, list(range(cfg.S))) for _ in range(cfg.L)]
    tau = 0
    for t in range(3):
        h = h0[t]
        for l in range(cfg.L):
            tau += 1
            st = o.layer_step(cfg, W, l, h, caches[l], caches[l + 1] if l + 1 < cfg.L else None, tau, 2)
            ref = res.steps[t * cfg.L + l]
            assert np.array_equal(st.T, ref.T) and np.array_equal(st.h_out, ref.h_out)
            assert st.P == ref.P and st.loads == ref.loads
            h = st.h_out


# ------------------------------------------------ Naive Prefetch (Table 5) --

@pytest.mark.parametrize("seed", range(20))
def test_naive_scores_brute_force(seed):
    """Gate mass per expert of the preceding step, accumulated independently."""
    rng = np.random.default_rng(100 + seed)
    n, B, K = int(rng.integers(4, 12)), int(rng.integers(1, 4)), 3
    K = min(K, n)
    T = np.stack([rng.choice(n, size=K, replace=False) for _ in range(B)])
    g = rng.random((B, K)).astype(np.float32)
    s = o.naive_scores(T, g, n)
    mass = {}
    for b in range(B):
        for k in range(K):
            mass[int(T[b, k])] = mass.get(int(T[b, k]), 0.0) + float(g[b, k])
    for e in range(n):
        if e in mass:
            assert s[e] == np.float32(mass[e])
        else:
            assert np.isneginf(s[e])
    assert np.isneginf(o.naive_scores(None, None, n)).all()        # no preceding step: no candidates


@pytest.mark.parametrize("seed", range(20))
def test_select_prefetch_never_picks_minus_inf(seed):
    rng = np.random.default_rng(200 + seed)
    n = int(rng.integers(2, 10))
    s = (rng.integers(0, 4, size=n) / 4).astype(np.float64)
    s[rng.random(n) < 0.5] = -np.inf
    occ = rng.random(n) < 0.3
    for M in range(0, n + 2):
        P = o.select_prefetch(s, occ, M)
        cand = [e for e in range(n) if not occ[e] and np.isfinite(s[e])]
        assert len(P) == min(M, len(cand)) and set(P) <= set(cand)
        want = sorted(cand, key=lambda e: (-s[e], e))[:M]
        assert P == want


def test_naive_prefetch_takes_only_the_preceding_steps_experts():
    """Naive Prefetch: every prefetched expert of target layer l+1 was routed
    there at the preceding step, never more than M_max; outputs equal the
    adapter policy's (router preservation holds across policies)."""
    cfg = _small_cfg(batch=2, S=4)
    h0 = gen.hidden_states(cfg)
    W = o.OracleWeights(cfg)
    ref = o.run_decode(cfg, W, h0, M_max=2)
    for M in (1, 2, 5):
        res = o.run_decode(cfg, W, h0, M_max=M, policy="naive")
        assert np.array_equal(np.stack(res.outputs), np.stack(ref.outputs))
        by = {(st.t, st.l): st for st in res.steps}
        issued = 0
        for st in res.steps:
            assert len(st.P) <= M
            issued += len(st.P)
            if st.P:
                prev = by[(st.t - 1, st.l + 1)]
                assert {e for e, _, _ in st.P} <= set(np.asarray(prev.T).ravel().tolist())
            if st.t == 0:
                assert not st.P                                   # nothing preceded the first step
        assert issued > 0
        assert all(np.isnan(v) for v in res.expert_recall.values())  # no adapter, no ExpertRecall


# ------------------------------------------------------ 4-bit expert codec --

def test_q4_decode_elementwise():
    """w = scale * (q - 8), one scale per 32 elements along D; checked element by element."""
    cfg = w.MoEConfig(name="q", L=2, D=64, n=4, K=2, I=5, r=4, S=4, windows=(1,), tokens=1, codec="q4", seed=3)
    gq, gs, uq, us, dq, ds = gen.expert_weights_q4(cfg, 0, 1)
    assert gq.dtype == np.uint8 and gq.max() <= 15 and gs.dtype == np.float16 and (gs > 0).all()
    Wg, Wu, Wd = o.q4_decode_expert(gq, gs, uq, us, dq, ds)
    for i in range(cfg.I):
        for d in range(cfg.D):
            assert Wg[i, d] == float(gs[i, d // 32]) * (int(gq[i, d]) - 8)
            assert Wu[i, d] == float(us[i, d // 32]) * (int(uq[i, d]) - 8)
            assert Wd[d, i] == float(ds[i, d // 32]) * (int(dq[d, i]) - 8)


def test_q4_expert_size_matches_the_papers_on_device_figure():
    """4-bit DeepSeek-VL2-Tiny experts occupy 1.94 MB (on-device evaluation)."""
    assert w.get("c3q4").blob_bytes == 1_935_360
    assert round(w.get("c3q4").blob_bytes / 1e6, 2) == 1.94


def test_q4_layer_against_torch_textbook_block():
    import torch
    cfg = w.MoEConfig(name="tq", L=2, D=64, n=6, K=2, I=32, r=4, S=6, windows=(1,), tokens=2, batch=2,
                      n_shared=1, codec="q4", seed=5)
    W = o.OracleWeights(cfg)
    h = o.decode(gen.hidden_states(cfg)[0], "bf16")
    cache = o.SlotCache(cfg.S, cfg.n, list(range(cfg.n)))
    u, x = o.layer_prologue(cfg, W, 0, h)
    T, g, z = o.route(W.router(0), x, cfg.K)
    assert cache.on_demand(o.batch_demand(T), 1) == []
    out = o.moe_output(cfg, W, 0, cache, u, x, T, g)

    def deq(parts):
        gq, gs, uq, us, dq, ds = (torch.tensor(np.asarray(p, dtype=np.float64)) for p in parts)
        rep = lambda sc: torch.repeat_interleave(sc, 32, dim=1)
        return (rep(gs) * (gq - 8), rep(us) * (uq - 8), rep(ds).T * (dq - 8))
    experts = [tuple(m.numpy() for m in deq(gen.expert_weights_q4(cfg, 0, e))) for e in range(cfg.n)]
    shared = [tuple(m.numpy() for m in deq(gen.shared_expert_weights_q4(cfg, 0, j))) for j in range(cfg.n_shared)]
    tT, tg, tout, tx = _torch_layer(h, W.router(0), cfg.K, experts, shared, cfg.rms_eps, None)
    assert np.array_equal(T, tT)
    np.testing.assert_allclose(out, tout, rtol=1e-11, atol=1e-12)


# --------------------------------------------------------------------------
# Section "Training Objective": the distillation loss and its gradient
# --------------------------------------------------------------------------

def _hand_pair():
    """D = r = 1, two experts: x = 1, A = 1, B = (ln 9, 0) give z_hat = (ln 9, 0)
    and pi_hat = (0.9, 0.1); the target logits (0, 0) give pi = (0.5, 0.5).
    KL(pi || pi_hat) = 0.5 ln(0.5/0.9) + 0.5 ln(0.5/0.1) = ln(5/3), while the
    reverse direction KL(pi_hat || pi) = 0.9 ln 1.8 + 0.1 ln 0.2 = 0.368..."""
    return (np.array([[1.0]]), np.array([[math.log(9.0)], [0.0]]), np.array([[1.0]]), np.array([[0.0, 0.0]]))


def _kl_pins_hold(loss_fn) -> bool:
    """The pins a KL(pi || pi_hat) implementation must meet: the hand pair's
    closed form, and scipy's relative entropy D(pi || pi_hat) on random rows."""
    A, B, X, Z = _hand_pair()
    if abs(loss_fn(A, B, X, Z) - math.log(5.0 / 3.0)) > 1e-14:
        return False
    import scipy.stats
    rng = np.random.default_rng(11)
    X = rng.normal(size=(9, 6))
    A, B = rng.normal(size=(3, 6)), rng.normal(size=(5, 3))
    Z = 2.0 * rng.normal(size=(9, 5))
    want = np.mean([scipy.stats.entropy(scipy.special.softmax(Z[i]), scipy.special.softmax(B @ (A @ X[i])))
                    for i in range(9)])
    return abs(loss_fn(A, B, X, Z) - want) <= 1e-12 * max(1.0, want)


def test_distill_loss_direction_hand_case_and_scipy():
    assert _kl_pins_hold(o.distill_pair_loss)
    A, B, X, Z = _hand_pair()
    reverse = 0.9 * math.log(1.8) + 0.1 * math.log(0.2)
    assert abs(o.distill_pair_loss(A, B, X, Z) - reverse) > 0.1        # the two directions differ here


def test_distill_pins_reject_a_reversed_kl():
    """A planted mistake in the oracle (the KL direction swapped) fails the pins."""
    def reversed_kl(A, B, X, Z):
        zhat = (np.asarray(X) @ np.asarray(A).T) @ np.asarray(B).T
        lp, lq = o.log_softmax(Z), o.log_softmax(zhat)
        return float(np.mean(np.sum(np.exp(lq) * (lq - lp), axis=-1)))
    assert not _kl_pins_hold(reversed_kl)
    assert _kl_pins_hold(o.distill_pair_loss)


def test_distill_grad_hand_case():
    """pi_hat - pi = (0.4, -0.4): dL/dB = (0.4, -0.4)^T a with a = 1, dL/dA = B^T (0.4, -0.4) x = 0.4 ln 9."""
    A, B, X, Z = _hand_pair()
    dA, dB = o.distill_pair_grad(A, B, X, Z)
    assert np.allclose(dB, [[0.4], [-0.4]], rtol=0, atol=1e-15)
    assert abs(dA[0, 0] - 0.4 * math.log(9.0)) < 1e-15


@pytest.mark.parametrize("seed", range(3))
def test_distill_grad_finite_differences(seed):
    """Central differences of the loss (fp64) against the closed-form gradient, every entry."""
    rng = np.random.default_rng(seed)
    N, D, r, n = 7, 5, 3, 6
    X = rng.normal(size=(N, D))
    A, B = 0.7 * rng.normal(size=(r, D)), 0.7 * rng.normal(size=(n, r))
    Z = 1.5 * rng.normal(size=(N, n))
    dA, dB = o.distill_pair_grad(A, B, X, Z)
    h = 1e-6
    for M, G in ((A, dA), (B, dB)):
        for idx in itertools.product(*map(range, M.shape)):
            keep = M[idx]
            M[idx] = keep + h
            up = o.distill_pair_loss(A, B, X, Z)
            M[idx] = keep - h
            dn = o.distill_pair_loss(A, B, X, Z)
            M[idx] = keep
            assert abs((up - dn) / (2 * h) - G[idx]) < 1e-8, idx


def test_distill_loss_invariants_and_pair_average():
    rng = np.random.default_rng(4)
    N, D, r, n = 20, 8, 3, 6
    X = rng.normal(size=(N, D))
    A, B = rng.normal(size=(r, D)), rng.normal(size=(n, r))
    # an exact adapter (the target logits are B A x plus a per-token shift): loss 0
    Z = (X @ A.T) @ B.T + rng.normal(size=(N, 1))
    assert abs(o.distill_pair_loss(A, B, X, Z)) < 1e-12
    Z2 = rng.normal(size=(N, n))
    v = o.distill_pair_loss(A, B, X, Z2)
    assert v > 0                                                        # Gibbs' inequality
    assert abs(o.distill_pair_loss(A, B, X, Z2 + 3.0) - v) < 1e-12        # logits up to a shift
    # L_pred averages the L - 1 pair losses (three layers: pairs 0->1 and 1->2)
    Xs = [X, rng.normal(size=(N, D)), rng.normal(size=(N, D))]
    Zs = [rng.normal(size=(N, n)) for _ in range(3)]
    ads = [(A, B), (rng.normal(size=(r, D)), rng.normal(size=(n, r)))]
    l01 = o.distill_pair_loss(ads[0][0], ads[0][1], Xs[0], Zs[1])
    l12 = o.distill_pair_loss(ads[1][0], ads[1][1], Xs[1], Zs[2])
    assert abs(o.distill_loss(ads, Xs, Zs) - (l01 + l12) / 2) < 1e-14
