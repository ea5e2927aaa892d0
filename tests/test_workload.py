"""The seeded input recipe: defaults unchanged by the routing-predictability
parameters, rank-k routers, scaled expert updates, and the recall the
calibrated recipe gives the SVD adapters (against the oracle)."""
import numpy as np

import oracle as o
import workload as w
from workload import gen

SMALL = w.MoEConfig(name="recipe_f32", L=2, D=256, n=16, K=4, I=64, r=8, S=16, windows=(2,), tokens=24,
                    dtype="f32", seed=5)


def test_default_parameters_keep_the_iid_recipe():
    a = gen.router_weight(SMALL, 0)
    b = gen.router_weight(SMALL.with_(router_rank=0, update_scale=1.0), 0)
    assert np.array_equal(a, b)
    assert np.linalg.matrix_rank(a.astype(np.float64)) == SMALL.n   # i.i.d.: full rank


def test_rank_k_router_has_rank_k_and_the_same_entry_scale():
    for dtype, tol in (("f32", 1e-5), ("bf16", 1e-2)):
        cfg = SMALL.with_(router_rank=3, dtype=dtype)
        W = o.decode(gen.router_weight(cfg, 1), dtype).astype(np.float64)
        sv = np.linalg.svd(W, compute_uv=False)
        assert sv[3] / sv[0] < tol                      # rank 3 up to the storage rounding
        assert abs(W.std() / cfg.w_std - 1.0) < 0.15


def test_update_scale_scales_only_the_down_projections():
    base, scaled = SMALL, SMALL.with_(update_scale=0.25)
    g0, u0, d0 = gen.expert_weights(base, 0, 3)
    g1, u1, d1 = gen.expert_weights(scaled, 0, 3)
    assert np.array_equal(g0, g1) and np.array_equal(u0, u1)
    np.testing.assert_allclose(d1, d0 * np.float32(0.25), rtol=1e-6)
    q = SMALL.with_(dtype="bf16", D=256, codec="q4")
    a = gen.expert_weights_q4(q, 0, 1)
    b = gen.expert_weights_q4(q.with_(update_scale=0.25), 0, 1)
    for i in range(5):
        assert np.array_equal(a[i], b[i])                # codes and gate/up scales unchanged
    np.testing.assert_allclose(b[5].astype(np.float64), (a[5].astype(np.float64) * 0.25), rtol=2e-3)


def test_calibrated_recipe_makes_the_next_routing_predictable():
    """With low-rank routers the rank-r SVD adapter predicts the next layer's
    routing far better than with i.i.d. routers (ExpertRecall@K)."""
    iid = SMALL.with_(r=4)
    cal = iid.with_(router_rank=4, update_scale=0.25)
    rec = {}
    for name, cfg in (("iid", iid), ("calibrated", cal)):
        res = o.run_decode(cfg, o.OracleWeights(cfg), gen.hidden_states(cfg), M_max=0, tokens=24)
        rec[name] = res.expert_recall[cfg.K]
    assert rec["calibrated"] > 0.9
    assert rec["calibrated"] > rec["iid"] + 0.2
