"""Lock-step parity driver: the device layer and the CPU oracle consume the same
stored hidden state and start from the same slot tables at every (token, layer).

Integer results (selected experts, on-demand loads, prefetch set and order,
slot tables, stamps) must match exactly.  The only exemption is a selection
boundary the oracle itself decides by a fp32 gap below 1e-6 (router logits
z_(K) - z_(K+1), or adjacent priorities among the eligible experts that the
prefetch set is cut from); then the device table is re-synchronised to the
oracle's and the case is logged.  Floating-point results are compared within
the stated tolerances.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List

import numpy as np

import oracle as o
from workload import gen

GAP_EXEMPT = 1e-6


@dataclass
class LockstepReport:
    layers: int = 0
    exempt: List[str] = field(default_factory=list)
    max_rel_h: float = 0.0        # max |gpu - ora| / max |ora| over layer outputs
    max_ulp_h: float = 0.0        # max elementwise |gpu - ora| / (spacing(ora) + 1e-6 max|ora|)
    max_err_g: float = 0.0
    max_err_s: float = 0.0
    max_err_x: float = 0.0
    prefetched: int = 0           # prefetch placements (oracle side) over the run


def _spacing(v: np.ndarray, dtype: str) -> np.ndarray:
    """Distance between adjacent representable values at |v| (bf16: 8 significant bits)."""
    a = np.abs(v)
    if dtype == "bf16":
        e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
        return 2.0 ** (e - 7)
    return np.spacing(a.astype(np.float32)).astype(np.float64)


def _topk_gap(z_row: np.ndarray, K: int) -> float:
    zs = np.sort(z_row)[::-1]
    return float(zs[K - 1] - zs[K]) if K < len(zs) else np.inf


def _prefetch_gap(s: np.ndarray, occupied: np.ndarray, M: int) -> float:
    elig = [e for e in range(len(s)) if not occupied[e] and np.isfinite(s[e])]
    vals = sorted((float(s[e]) for e in elig), reverse=True)[: M + 1]
    if len(vals) < 2:
        return np.inf
    return float(np.min(-np.diff(vals)))


def run_lockstep(stack, cfg, tokens: int, M_max: int, check_x: bool = True,
                 policy: str = "adapter", adapter_override=None, progress=None, h0=None) -> LockstepReport:
    """policy "naive": Naive Prefetch on both sides (the device via
    spp_set_prefetch_source); the oracle gets each layer's routing of the
    preceding step.  adapter_override(l) -> (A, B): the adapter values the
    oracle uses (those the stack was bound with, as stored).  progress(t, l):
    called after each compared layer.  h0: layer-0 hidden states [tokens,
    batch, D] in storage form (default: the workload's AR(1) states)."""
    from paper_2607_24787_amd import spp

    W = o.OracleWeights(cfg, cache_experts=cfg.host_layers * cfg.n + 8, adapter_override=adapter_override)
    W.warm()
    if h0 is None:
        h0 = gen.hidden_states(cfg, tokens=tokens)
    S = stack.S
    res = list(range(min(S, cfg.n)))
    caches = [o.SlotCache(S, cfg.n, res) for _ in range(cfg.L)]
    tol = 2e-2 if cfg.dtype == "bf16" else 1e-4
    rep = LockstepReport()
    spp.spp_set_prefetch_source(stack.ctx, spp.PREFETCH_PREV_TOKEN if policy == "naive" else spp.PREFETCH_ADAPTER)
    prev = [None] * cfg.L          # (T, g) of each layer at the preceding step (oracle side)
    tau = 0
    for t in range(tokens):
        h = h0[t]
        for l in range(cfg.L):
            tau += 1
            nxt = caches[l + 1] if l + 1 < cfg.L else None
            occ_next_before = nxt.occupied() if nxt is not None else None
            ref = o.layer_step(cfg, W, l, h, caches[l], nxt, tau, M_max, policy=policy,
                               next_prev=prev[l + 1] if l + 1 < cfg.L else None)
            prev[l] = (ref.T, ref.g)
            rep.prefetched += len(ref.P)
            stack.upload_hidden(h, 0)
            spp.spp_set_clock(stack.ctx, tau - 1)
            topk, gates, stats = stack.layer(l, 0, 1, M_max)
            h_gpu = stack.download(stack.hbuf[1])
            loads, pref = spp.spp_get_last_transfers(stack.ctx)
            tag = f"t={t} l={l}"
            resync = False
            for b in range(cfg.batch):
                if not np.array_equal(topk[b], ref.T[b]):
                    gap = _topk_gap(ref.z[b], cfg.K)
                    assert gap < GAP_EXEMPT, f"{tag} b={b}: top-k {topk[b]} != {ref.T[b]} (oracle gap {gap:.3g})"
                    rep.exempt.append(f"{tag} b={b} topk gap {gap:.3g}")
                    resync = True
                else:
                    rep.max_err_g = max(rep.max_err_g, float(np.max(np.abs(gates[b] - ref.g[b]))))
            if not resync:
                assert loads == ref.loads, f"{tag}: loads {loads} != {ref.loads}"
                assert stats.misses == len(ref.loads) and stats.token_hits == int(np.sum(ref.ready)), tag
                e, st = spp.spp_get_slot_table(stack.ctx, l, S)
                assert e.tolist() == ref.table_after_demand.tolist(), tag
                assert st.tolist() == ref.stamps_after_demand.tolist(), tag
            if ref.s is not None:
                s_gpu = spp.spp_get_last_priorities(stack.ctx, cfg.n)
                fin = np.isfinite(ref.s)
                assert np.array_equal(fin, np.isfinite(s_gpu)), f"{tag}: candidate sets differ"
                if fin.any():
                    rep.max_err_s = max(rep.max_err_s, float(np.max(np.abs(s_gpu[fin] - ref.s[fin]))))
                assert np.allclose(s_gpu[fin], ref.s[fin], rtol=1e-5, atol=2e-6), f"{tag}: priorities differ"
                if not resync and pref != ref.P:
                    gap = _prefetch_gap(ref.s, occ_next_before, max(M_max, 0))
                    assert gap < GAP_EXEMPT, f"{tag}: prefetch {pref} != {ref.P} (oracle gap {gap:.3g})"
                    rep.exempt.append(f"{tag} prefetch gap {gap:.3g}")
                    resync = True
                if not resync and nxt is not None:
                    assert stats.prefetched == len(ref.P), tag
                    e2, st2 = spp.spp_get_slot_table(stack.ctx, l + 1, S)
                    assert e2.tolist() == ref.next_table_after_prefetch.tolist(), tag
                    assert st2.tolist() == ref.next_stamps_after_prefetch.tolist(), tag
            if check_x and l == 0 and t < 4:
                x_gpu = spp.spp_get_last_router_input(stack.ctx, cfg.batch, cfg.D)
                rep.max_err_x = max(rep.max_err_x, float(np.max(np.abs(x_gpu - ref.x)) / np.max(np.abs(ref.x))))
                assert rep.max_err_x < 1e-5, f"{tag}: router input differs"
            if resync:
                spp.spp_set_slot_table(stack.ctx, l, ref.table_after_demand, ref.stamps_after_demand)
                if nxt is not None and ref.next_table_after_prefetch is not None:
                    spp.spp_set_slot_table(stack.ctx, l + 1, ref.next_table_after_prefetch,
                                           ref.next_stamps_after_prefetch)
            else:
                # outputs are compared only where the same experts ran
                og = o.decode(h_gpu, cfg.dtype)
                oo = o.decode(ref.h_out, cfg.dtype)
                rel = float(np.max(np.abs(og - oo)) / np.max(np.abs(oo)))
                ulp = float(np.max(np.abs(og - oo) / (_spacing(oo, cfg.dtype) + 1e-6 * np.max(np.abs(oo)))))
                rep.max_rel_h = max(rep.max_rel_h, rel)
                rep.max_ulp_h = max(rep.max_ulp_h, ulp)
                assert rel <= tol, f"{tag}: layer output rel err {rel:.3g} > {tol}"
            rep.layers += 1
            if progress is not None:
                progress(t, l)
            h = ref.h_out
    return rep
