"""Host-side checks of libspp without a GPU: exports, budget rule, replacement policy.

The native slot policy (the same object every device context runs per layer)
is compared bit-exactly with the oracle's logical slot cache on random traces.
"""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle as o
from paper_2607_24787_amd import spp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "spp.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_0-9]+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_library_exports_every_declared_symbol():
    L = spp.lib()
    declared = _declared_functions()
    assert len(declared) >= 25
    for name in declared:
        assert hasattr(L, name), name
    assert set(declared) == set(spp.exported_symbols())


def test_select_prefetch_budget_matches_oracle_rule():
    rng = np.random.default_rng(0)
    cases = [(300.0, 150.0, 128), (299.9, 150.0, 128), (0.0, 1.0, 8), (-3.0, 1.0, 8), (1e9, 1.0, 64)]
    cases += [(float(rng.uniform(-50, 2000)), float(rng.uniform(0.5, 400)), int(rng.integers(0, 200)))
              for _ in range(300)]
    for W, c, n in cases:
        assert spp.select_prefetch_budget(W, c, n) == o.prefetch_budget(W, c, n)
    for W, c, n in [(1.0, 0.0, 8), (1.0, -2.0, 8), (math.nan, 1.0, 8), (1.0, math.inf, 8), (math.inf, 1.0, 8),
                    (1.0, 1.0, -1)]:
        with pytest.raises(spp.SppError) as e:
            spp.select_prefetch_budget(W, c, n)
        assert e.value.status == spp.SPP_EINVAL
        assert "finite" in spp.spp_last_error()


@pytest.mark.parametrize("seed", range(25))
def test_native_policy_matches_oracle_slot_cache(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(4, 40))
    S = int(rng.integers(1, n + 1))
    resident = list(rng.permutation(n)[: int(rng.integers(0, S + 1))])
    nat = spp.SlotPolicy(S, n, resident)
    ora = o.SlotCache(S, n, resident)
    tau = 0
    for step in range(60):
        tau += 1
        k = int(rng.integers(1, min(n, 2 * S) + 1))
        need = list(rng.integers(0, n, size=k))          # duplicates allowed; may exceed S (rounds)
        assert nat.on_demand(need, tau) == ora.on_demand(need, tau)
        e, t = nat.table()
        assert e.tolist() == ora.expert.tolist() and t.tolist() == ora.stamp.tolist()
        s = (rng.integers(0, 6, size=n) / 5).astype(np.float32)      # ties on purpose
        M = int(rng.integers(0, 6))
        if rng.random() < 0.5:
            tau += 1
        got = nat.prefetch(s, M, tau)
        want = ora.prefetch(o.select_prefetch(s.astype(np.float64), ora.occupied(), M), tau)
        assert got == want
        e, t = nat.table()
        assert e.tolist() == ora.expert.tolist() and t.tolist() == ora.stamp.tolist()


def test_native_policy_rejects_bad_input():
    with pytest.raises(spp.SppError):
        spp.SlotPolicy(2, 4, [0, 0])
    with pytest.raises(spp.SppError):
        spp.SlotPolicy(2, 4, [0, 1, 2])
    p = spp.SlotPolicy(2, 4, [0])
    with pytest.raises(spp.SppError):
        p.on_demand([5], 1)
    e, t = p.table()
    assert e.tolist() == [0, -1]                         # a failed call changes nothing
    # more distinct experts than slots run in rounds, as in the oracle's hand-worked trace
    q = spp.SlotPolicy(2, 6, [0, 1])
    assert q.on_demand([4, 3, 2, 1], 1) == [(2, 0, 0), (3, 0, 2), (4, 1, 1)]
    assert q.table()[0].tolist() == [3, 4]


def test_create_rejects_bad_shapes_without_touching_a_device():
    bad = [
        spp.make_desc(L=0, D=256, n=8, K=2, I=64, r=4, S=4),
        spp.make_desc(L=2, D=250, n=8, K=2, I=64, r=4, S=4),            # D*2 not a multiple of 16
        spp.make_desc(L=2, D=256, n=8, K=9, I=64, r=4, S=4),            # K > n
        spp.make_desc(L=2, D=256, n=8, K=2, I=64, r=300, S=4),          # r too large
        spp.make_desc(L=2, D=8192, n=8, K=2, I=64, r=4, S=4),           # D too large
        spp.make_desc(L=2, D=256, n=8, K=2, I=64, r=4, S=4, dtype=7),
        # fewer slots than one call's distinct routed experts, outside the tiled batched path
        spp.make_desc(L=2, D=256, n=8, K=2, I=64, r=4, S=1),                       # batch 1, S < K
        spp.make_desc(L=2, D=96, n=12, K=3, I=40, r=8, S=8, max_batch=3, dtype=spp.DTYPE_F32),  # S < K*B
        spp.make_desc(L=2, D=512, n=16, K=4, I=64, r=8, S=3, expert_codec=spp.CODEC_Q4),  # 4-bit, S < K
    ]
    for d in bad:
        with pytest.raises(spp.SppError) as e:
            spp.spp_create(d, 0)
        assert e.value.status == spp.SPP_EINVAL
    assert "S must be" in str(e.value)


def test_slot_count_check_depends_on_the_layout():
    """The create-time slot check is exactly S >= min(n, K * max_batch) for the
    contexts that cannot run a step in rounds; the tiled batched layout may
    hold fewer slots than a call's demand.  Only shapes the check refuses are
    created here (a shape it passes would reach the device)."""
    cases = [  # (desc kwargs, refused)
        (dict(L=2, D=256, n=8, K=2, I=64, r=4, S=1), True),
        (dict(L=2, D=96, n=12, K=3, I=40, r=8, S=8, max_batch=3, dtype=spp.DTYPE_F32), True),
        (dict(L=2, D=96, n=6, K=3, I=40, r=8, S=5, max_batch=3, dtype=spp.DTYPE_F32), True),   # min(n, K*B) = 6
        (dict(L=2, D=512, n=24, K=4, I=160, r=8, S=6, max_batch=5), False),  # tiled bf16: rounds
        (dict(L=2, D=96, n=12, K=3, I=40, r=8, S=9, max_batch=3, dtype=spp.DTYPE_F32), False),
        (dict(L=2, D=96, n=6, K=3, I=40, r=8, S=6, max_batch=3, dtype=spp.DTYPE_F32), False),
    ]
    for kw, refused in cases:
        d = spp.make_desc(**kw)
        tiled = spp.spp_blob_layout(d) == spp.LAYOUT_TILED
        assert refused == (not tiled and kw["S"] < min(kw["n"], kw["K"] * kw.get("max_batch", 1))), kw
        if refused:
            with pytest.raises(spp.SppError) as e:
                spp.spp_create(d, 0)
            assert e.value.status == spp.SPP_EINVAL and "S must be" in str(e.value), kw


def test_blob_stride():
    d = spp.make_desc(L=2, D=2048, n=128, K=8, I=768, r=64, S=32)
    assert spp.spp_blob_stride(d) == 9_437_184                 # 3*768*2048*2, already 4 KiB aligned
    d = spp.make_desc(L=2, D=96, n=12, K=3, I=40, r=8, S=12, dtype=spp.DTYPE_F32)
    assert spp.spp_blob_stride(d) == 49152                     # 46080 rounded up to 4 KiB


def _expected_blob(layout, G, U, Wd):
    """The blob the header's layout formulas describe, element by element."""
    I, D = G.shape
    out = np.zeros(3 * I * D, dtype=G.dtype)
    if layout == spp.LAYOUT_UNITS:
        for i in range(I):
            for d in range(D):
                out[(3 * i + 0) * D + d] = G[i, d]
                out[(3 * i + 1) * D + d] = U[i, d]
                out[(3 * i + 2) * D + d] = Wd[d, i]
        return out
    nb = D // 256
    for t in range(I // 16):
        for b in range(nb):
            for w, W in enumerate((G, U)):
                for j in range(8):
                    for l in range(64):
                        piece = (((t * nb + b) * 2 + w) * 8 + j) * 64 + l
                        row, col = 16 * t + l % 16, 256 * b + 32 * j + 8 * (l // 16)
                        out[piece * 8: piece * 8 + 8] = W[row, col: col + 8]
    for s in range(nb):
        for i in range(I):
            run = s * I + i
            out[2 * I * D + run * 256: 2 * I * D + run * 256 + 256] = Wd[256 * s: 256 * s + 256, i]
    return out


@pytest.mark.parametrize("case", ["units_f32", "units_bf16_batch1", "tiled_bf16"])
def test_pack_expert_places_every_element_where_the_header_says(case):
    if case == "units_f32":
        d, dt = spp.make_desc(L=2, D=96, n=12, K=3, I=40, r=8, S=12, dtype=spp.DTYPE_F32), np.float32
    elif case == "units_bf16_batch1":
        d, dt = spp.make_desc(L=2, D=512, n=12, K=3, I=32, r=8, S=12), np.uint16
    else:
        d, dt = spp.make_desc(L=2, D=512, n=12, K=3, I=32, r=8, S=12, max_batch=4), np.uint16
    want_layout = spp.LAYOUT_TILED if case == "tiled_bf16" else spp.LAYOUT_UNITS
    assert spp.spp_blob_layout(d) == want_layout
    I, D = d.I, d.D
    vals = np.arange(3 * I * D).astype(dt)                     # every element distinct
    G, U, Wd = vals[:I * D].reshape(I, D), vals[I * D:2 * I * D].reshape(I, D), vals[2 * I * D:].reshape(D, I)
    stride = spp.spp_blob_stride(d)
    out = np.full(stride, 0xAB, dtype=np.uint8)
    spp.spp_pack_expert(d, G, U, Wd, out=out)
    got = out[:3 * I * D * np.dtype(dt).itemsize].view(dt)
    assert np.array_equal(got, _expected_blob(want_layout, G, U, Wd))
    assert not out[3 * I * D * np.dtype(dt).itemsize:].any()   # padding zeroed
    # the tiled layout needs D % 256 == 0 and I % 16 == 0; other batched shapes keep the unit layout
    assert spp.spp_blob_layout(spp.make_desc(L=2, D=640, n=12, K=3, I=32, r=8, S=12, max_batch=4)) == spp.LAYOUT_UNITS
    assert spp.spp_blob_layout(spp.make_desc(L=2, D=512, n=12, K=3, I=40, r=8, S=12, max_batch=4)) == spp.LAYOUT_UNITS
    assert spp.lib().spp_pack_expert(None, None, None, None, None) == spp.SPP_EINVAL
    assert spp.lib().spp_pack_expert(ctypes.byref(d), None, None, None, out.ctypes.data) == spp.SPP_EINVAL
    with pytest.raises(ValueError):
        spp.spp_pack_expert(d, G.T, U, Wd)


@pytest.mark.parametrize("seed", range(10))
def test_native_prefetch_skips_minus_inf_like_the_oracle(seed):
    rng = np.random.default_rng(300 + seed)
    n = int(rng.integers(4, 30))
    S = int(rng.integers(1, n + 1))
    nat, ora = spp.SlotPolicy(S, n, []), o.SlotCache(S, n, [])
    tau = 0
    for step in range(30):
        tau += 1
        need = list(rng.integers(0, n, size=int(rng.integers(1, S + 1))))
        assert nat.on_demand(need, tau) == ora.on_demand(need, tau)
        s = (rng.integers(0, 5, size=n) / 4).astype(np.float32)
        s[rng.random(n) < 0.6] = -np.inf
        M = int(rng.integers(0, 6))
        got = nat.prefetch(s, M, tau)
        assert got == ora.prefetch(o.select_prefetch(s.astype(np.float64), ora.occupied(), M), tau)
        assert all(np.isfinite(s[e]) for e, _, _ in got)


def test_pack_expert_q4_places_codes_and_scales_where_the_header_says():
    d = spp.make_desc(L=2, D=256, n=6, K=2, I=5, r=4, S=6, expert_codec=spp.CODEC_Q4)
    assert spp.spp_blob_layout(d) == spp.LAYOUT_Q4_UNITS
    I, D, nb = d.I, d.D, d.D // 32
    unit = 3 * D // 2 + 3 * nb * 2
    assert spp.spp_blob_stride(d) == -(-I * unit // 4096) * 4096
    rng = np.random.default_rng(7)
    gq, uq = rng.integers(0, 16, size=(I, D)).astype(np.uint8), rng.integers(0, 16, size=(I, D)).astype(np.uint8)
    dq = rng.integers(0, 16, size=(D, I)).astype(np.uint8)
    gs, us, ds = (rng.uniform(0.001, 0.01, size=(I, nb)).astype(np.float16) for _ in range(3))
    blob = spp.spp_pack_expert_q4(d, gq, gs, uq, us, dq, ds)
    for i in range(I):
        u = blob[i * unit:(i + 1) * unit]
        for run, codes in enumerate((gq[i], uq[i], dq[:, i])):
            for e in range(D):
                byte = int(u[run * D // 2 + e // 2])
                assert (byte >> (4 * (e % 2))) & 0xF == codes[e]
        for run, sc in enumerate((gs[i], us[i], ds[i])):
            got = u[3 * D // 2 + run * nb * 2: 3 * D // 2 + (run + 1) * nb * 2].view(np.float16)
            assert np.array_equal(got, sc)
    assert not blob[I * unit:].any()
    bad = gq.copy()
    bad[0, 0] = 16
    with pytest.raises(spp.SppError):
        spp.spp_pack_expert_q4(d, bad, gs, uq, us, dq, ds)
    with pytest.raises(spp.SppError):                                  # plain packer refuses a 4-bit desc
        spp.spp_pack_expert(d, np.zeros((I, D), np.uint16), np.zeros((I, D), np.uint16), np.zeros((D, I), np.uint16))
    for kw in (dict(max_batch=2), dict(dtype=spp.DTYPE_F32), dict(D=320)):  # 4-bit needs bf16, batch 1, D % 256
        args = dict(L=2, D=256, n=6, K=2, I=5, r=4, S=6, expert_codec=spp.CODEC_Q4)
        args.update(kw)
        with pytest.raises(spp.SppError):
            spp.spp_create(spp.make_desc(**args), 0)


@pytest.mark.parametrize("cname,pyname", [("spp_model_desc", "ModelDesc"), ("spp_layer_stats", "LayerStats"),
                                          ("spp_run_stats", "RunStats")])
def test_binding_structs_match_the_header_layout(cname, pyname, tmp_path):
    """The ctypes structures have the size and field offsets a C compiler gives
    the header's structs (compiled here with gcc as plain C)."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("no C compiler")
    py = getattr(spp, pyname)
    fields = [f for f, _ in py._fields_]
    lines = [f'  printf("%zu\\n", offsetof({cname}, {f}));' for f in fields]
    src = tmp_path / "layout.c"
    src.write_text("#include <stddef.h>\n#include <stdio.h>\n#include \"spp.h\"\nint main(void) {\n"
                   f'  printf("%zu\\n", sizeof({cname}));\n' + "\n".join(lines) + "\n  return 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = [int(v) for v in subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split()]
    assert out[0] == ctypes.sizeof(py)
    assert out[1:] == [getattr(py, f).offset for f in fields]
