"""Copy/compute fence tests on the device.

The FFN may read a slot only after the copy into it completed (RAW), and a
copy may overwrite a slot only after the last kernel that read it (WAR).  With
every copied slot poisoned with NaN bytes just before its copy, and every copy
held back by a bounded busy kernel on the copy stream, outputs must stay
bitwise identical to an unpoisoned, undelayed run, and contain no NaN.
"""
import sys

import numpy as np
import pytest

import oracle as o
import workload as w
from workload import gen

pytestmark = pytest.mark.gpu

RAGGED = w.MoEConfig(name="ragged_bf16_D640_n40_k5", L=3, D=640, n=40, K=5, I=100, r=12, S=11, windows=(2,),
                     tokens=16, seed=3)


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _run(cfg, M_max, tokens, poison=False, delay_us=0, engine=2, tier_us=0, overlap=False, splits=None,
         parallel=False):
    from paper_2607_24787_amd import spp
    from paper_2607_24787_amd.model import OffloadedMoEStack
    h0 = gen.hidden_states(cfg, tokens=tokens)
    st = OffloadedMoEStack(cfg)
    try:
        spp.spp_set_copy_engine(st.ctx, engine)
        spp.spp_set_ffn_overlap(st.ctx, 1 if overlap else 0)
        spp.spp_set_prefetch_parallel(st.ctx, 1 if parallel else 0)
        if tier_us:
            spp.spp_set_tier_delay(st.ctx, tier_us)
        spp.spp_debug_set_poison(st.ctx, poison)
        spp.spp_debug_set_copy_delay(st.ctx, delay_us)
        outs, on_time, needed, misses = [], 0, 0, 0
        for t in range(tokens):
            res = st.step(h0[t], M_max)
            for topk, _, stats in res:
                on_time += stats.ready_on_time
                distinct = len(set(topk.ravel().tolist()))
                needed += distinct
                misses += stats.misses
                # every routed expert was either ready when its FFN was enqueued or waited for
                assert stats.ready_on_time + stats.waited == distinct, (t, stats.ready_on_time, stats.waited)
            outs.append(st.download(st.hbuf[st.last_buf]))
        if splits is not None:
            splits.append(spp.spp_get_run_stats(st.ctx).ffn_split_launches)
        return np.stack(outs), on_time, needed, misses
    finally:
        st.close()


# batched, 6 slots for a demand of ~14 experts: the on-demand step runs in
# rounds and later rounds overwrite slots an earlier round's FFN read (WAR)
BATCH_ROUNDS = w.MoEConfig(name="batch5_bf16_D512_n24_k4_I160", L=2, D=512, n=24, K=4, I=160, r=8, S=6,
                           windows=(2,), tokens=6, batch=5, seed=13)


# 4-bit experts: a poisoned slot holds 0xFF bytes, i.e. NaN scales
Q4_FENCE = w.MoEConfig(name="q4_D256_n12_k3_I96", L=3, D=256, n=12, K=3, I=96, r=8, S=5, windows=(2,), tokens=12,
                       codec="q4", seed=21)


# copy engine 2: on-demand loads by the copy kernel, prefetches by DMA (the
# default); 0: every copy by the copy kernel; 1: every copy by DMA
@pytest.mark.parametrize("cfg,M_max,tokens,engine", [(RAGGED, 2, 12, 2), (w.get("c0"), 1, 16, 2),
                                                     (BATCH_ROUNDS, 2, 6, 2), (Q4_FENCE, 2, 12, 2),
                                                     (RAGGED, 2, 12, 0), (BATCH_ROUNDS, 2, 6, 0),
                                                     (RAGGED, 2, 12, 1), (BATCH_ROUNDS, 2, 6, 1)],
                         ids=["ragged", "c0", "batched_rounds", "q4", "ragged_kernel", "batched_rounds_kernel",
                              "ragged_sdma", "batched_rounds_sdma"])
def test_poisoned_delayed_copies_leave_outputs_unchanged(torch_cuda, cfg, M_max, tokens, engine):
    _log(f"[fences] {cfg.name} M_max={M_max} engine={engine}")
    ref, ref_on_time, needed, misses = _run(cfg, M_max, tokens, engine=engine)
    assert misses > 0, "the case must exercise on-demand loads"
    assert not np.isnan(o.decode(ref, cfg.dtype)).any()
    for poison, delay in [(True, 0), (True, 300), (False, 300)]:
        out, on_time, needed2, _ = _run(cfg, M_max, tokens, poison, delay, engine)
        assert needed2 == needed
        dec = o.decode(out, cfg.dtype)
        assert not np.isnan(dec).any(), (poison, delay)
        assert np.array_equal(out, ref), (poison, delay)
        if delay:
            # held-back copies were still in flight when the FFN was enqueued:
            # the compute stream had to wait on their events
            assert on_time < needed, (on_time, needed)
        _log(f"[fences] poison={poison} delay={delay}us ready_on_time={on_time}/{needed}")


def test_repeat_runs_are_bitwise_identical(torch_cuda):
    cfg = w.get("c1")
    a, _, _, _ = _run(cfg, cfg.window, 6)
    b, _, _, _ = _run(cfg, cfg.window, 6, poison=True)
    assert np.array_equal(a, b)
    for engine in (0, 1):   # every copy by the copy kernel, every copy by DMA: the same bytes
        c, _, _, _ = _run(cfg, cfg.window, 6, poison=True, engine=engine)
        assert np.array_equal(a, c), engine


@pytest.mark.parametrize("cfg,M_max,tokens", [(RAGGED, 4, 16), (w.get("c1q4"), 4, 6)], ids=["ragged", "qwen_q4"])
def test_parallel_prefetches_leave_outputs_unchanged(torch_cuda, cfg, M_max, tokens):
    """A layer's whole prefetch copies alternating the two copy streams, with
    poisoned and delayed copies: outputs bitwise those of the default run."""
    _log(f"[parallel] {cfg.name} M_max={M_max}")
    ref, _, needed, _ = _run(cfg, M_max, tokens)
    for poison, delay in [(True, 0), (True, 300)]:
        out, on_time, needed2, _ = _run(cfg, M_max, tokens, poison, delay, parallel=True)
        assert needed2 == needed
        assert not np.isnan(o.decode(out, cfg.dtype)).any(), (poison, delay)
        assert np.array_equal(out, ref), (poison, delay)


@pytest.mark.parametrize("cfg,M_max,tokens", [(RAGGED, 2, 16), (w.get("c0"), 1, 12)], ids=["ragged", "c0"])
def test_switching_copy_modes_between_tokens_keeps_the_bits(torch_cuda, cfg, M_max, tokens):
    """Copy engine and storage emulation changed before every token, with
    poisoned, delayed copies: split-engine prefetches go out whole on one copy
    stream, the other modes in halves on both, so a slot's earlier copy that
    was never waited on may still be in flight on the other stream when a new
    copy targets it (WAW).  Outputs stay bitwise those of the default run."""
    from paper_2607_24787_amd import spp
    from paper_2607_24787_amd.model import OffloadedMoEStack
    _log(f"[switch] {cfg.name} M_max={M_max}")
    ref, _, _, _ = _run(cfg, M_max, tokens)
    # (engine, tier delay in us, parallel): whole prefetches on one stream,
    # halves through the one storage queue, whole prefetches alternating the
    # streams, halves by DMA, whole again, halves by the copy kernel
    modes = [(2, 0, 0), (2, 300, 0), (2, 0, 1), (1, 0, 0), (2, 0, 1), (2, 0, 0), (0, 0, 0)]
    h0 = gen.hidden_states(cfg, tokens=tokens)
    st = OffloadedMoEStack(cfg)
    try:
        spp.spp_debug_set_poison(st.ctx, 1)
        outs = []
        for t in range(tokens):
            engine, tier_us, parallel = modes[t % len(modes)]
            spp.spp_set_copy_engine(st.ctx, engine)
            spp.spp_set_prefetch_parallel(st.ctx, parallel)
            spp.spp_set_tier_delay(st.ctx, tier_us)
            if not tier_us:
                spp.spp_debug_set_copy_delay(st.ctx, 300)
            st.step(h0[t], M_max)
            outs.append(st.download(st.hbuf[st.last_buf]))
        out = np.stack(outs)
    finally:
        st.close()
    assert not np.isnan(o.decode(out, cfg.dtype)).any()
    assert np.array_equal(out, ref)


@pytest.mark.parametrize("cfg,M_max,tokens", [(RAGGED, 2, 12), (BATCH_ROUNDS, 2, 6)], ids=["ragged", "batched_rounds"])
def test_storage_emulation_leaves_outputs_unchanged(torch_cuda, cfg, M_max, tokens):
    """Under storage emulation every expert read (on-demand loads included)
    goes through the copy streams' one queue, each behind its delay; outputs
    stay bitwise those of the default run."""
    _log(f"[tier] {cfg.name}")
    ref, _, needed, misses = _run(cfg, M_max, tokens)
    assert misses > 0
    out, on_time, needed2, _ = _run(cfg, M_max, tokens, poison=True, tier_us=300)
    assert needed2 == needed and on_time < needed
    assert np.array_equal(out, ref)


@pytest.mark.parametrize("cfg,M_max,tokens,poison,delay_us", [
    (RAGGED, 2, 12, False, 0),
    (RAGGED, 2, 12, True, 60),
    (Q4_FENCE, 2, 12, False, 0),
    (Q4_FENCE, 2, 12, True, 60),
    (w.get("c3q4").with_(L=3), 2, 4, False, 0),
    (w.get("c1"), 2, 4, False, 0),
], ids=["ragged", "ragged_poison_delay", "q4", "q4_poison_delay", "dsv2_q4", "qwen_full"])
def test_ffn_split_gives_the_single_launch_bits(torch_cuda, cfg, M_max, tokens, poison, delay_us):
    """With the FFN split on (resident experts beside the on-demand copies, late
    ones after them), every output is bitwise the same whichever experts are
    late -- the same as a single launch of the split's kernel, which runs every
    batch-1 FFN of the context while the split is on -- also with poisoned and
    delayed copies, which make more experts late; the split does happen."""
    _log(f"[split] {cfg.name} M_max={M_max} poison={poison} delay={delay_us}")
    splits = []
    base, _, _, _ = _run(cfg, M_max, tokens, overlap=True)
    got, _, _, misses = _run(cfg, M_max, tokens, poison=poison, delay_us=delay_us, overlap=True, splits=splits)
    assert not np.isnan(o.decode(got, cfg.dtype)).any()
    assert np.array_equal(base, got)
    assert misses > 0 and splits[0] > 0, (misses, splits)


def test_reads_wait_only_for_their_own_copies(torch_cuda):
    """Storage emulation on: every copy goes through the copy streams, each
    held about 20 ms.  Layer 1 loads its five routed experts as one group
    whose completion event belongs to slot 0 (the last load lands there); a
    prefetch then re-uses slot 0 while the group's copies may still be in
    flight, which re-records that event for the new copy.  The next call with
    the same routing must count the four experts still in their slots as
    ready on time (the first call's wait already covered their copies) and
    wait only for the one expert it reloads; the output bits stay the first
    call's."""
    from paper_2607_24787_amd import spp
    from paper_2607_24787_amd.model import OffloadedMoEStack
    cfg = RAGGED.with_(S=5)
    st = OffloadedMoEStack(cfg)
    try:
        h0 = gen.hidden_states(cfg, tokens=1)
        st.upload_hidden(h0[0], 0)
        st.layer(0, 0, 1, -1)                       # layer 1's input now sits in buffer 1
        T1, _, _ = st.layer(1, 1, 0, -1)
        need = sorted(set(T1.ravel().tolist()))
        assert len(need) == cfg.K
        others = [e for e in range(cfg.n) if e not in need]
        # slots hold experts the call does not need, stamps falling with the
        # slot index: the loads (ascending expert) take slots 4, 3, 2, 1, 0
        spp.spp_set_slot_table(st.ctx, 1, np.array(others[:5], np.int32), np.array([9, 7, 5, 3, 1], np.int64))
        spp.spp_set_clock(st.ctx, 20)
        spp.spp_set_tier_delay(st.ctx, 20000)
        _log("[own copies] call A: five loads in one group")
        _, _, sa = st.layer(1, 1, 0, -1)
        out_a = st.download(st.hbuf[0])
        loads, _ = spp.spp_get_last_transfers(st.ctx)
        assert [t[1] for t in loads] == [4, 3, 2, 1, 0]
        assert (sa.misses, sa.ready_on_time, sa.waited) == (5, 0, 5)
        # a hand-issued prefetch for layer 1 evicts the least recently stamped
        # slot, slot 0 (all stamps equal, lowest index), while nothing waits for it
        _log("[own copies] prefetch into slot 0")
        s = np.zeros(cfg.n, np.float32)
        s[others[0]] = 1.0
        assert spp.expert_cache_issue_prefetch(st.ctx, 1, s, 1) == [others[0]]
        e1, _ = spp.spp_get_slot_table(st.ctx, 1, cfg.S)
        assert int(e1[0]) == others[0]
        _log("[own copies] call B: same routing")
        _, _, sb = st.layer(1, 1, 0, -1)
        assert sb.misses == 1
        assert (sb.ready_on_time, sb.waited) == (4, 1), (sb.ready_on_time, sb.waited)
        out_b = st.download(st.hbuf[0])
        assert np.array_equal(out_a, out_b)
    finally:
        st.close()
