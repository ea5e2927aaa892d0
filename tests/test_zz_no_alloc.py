"""adapter_predict_static (no allocation, scratch in a static device array)
against adapter_predict (a context's scratch), through the C ABI: the same
priorities on two calls in a row, the second with a smaller batch, for batch-1
and batched launches; sizes above the static scratch are refused before any
device work."""
import sys

import numpy as np
import pytest

import oracle as o
import workload as w

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


# bf16 with a batched router (D % 16 == 0), rank 8 and rank 6; the Qwen-shaped adapter (n 128, r 64)
CASES = [w.MoEConfig(name="static_bf16_D256_n12_r8", L=2, D=256, n=12, K=3, I=64, r=8, S=12, windows=(2,),
                     tokens=2, batch=16, seed=9),
         w.MoEConfig(name="static_bf16_D256_n12_r6", L=2, D=256, n=12, K=3, I=64, r=6, S=12, windows=(2,),
                     tokens=2, batch=16, seed=10),
         w.get("c1").with_(L=2, batch=16, S=128, I=16)]


@pytest.mark.parametrize("cfg", CASES, ids=["r8", "r6", "qwen_shape"])
def test_static_scratch_entry_point_matches_adapter_predict(torch_cuda, cfg):
    import torch
    from paper_2607_24787_amd import spp
    from paper_2607_24787_amd.model import OffloadedMoEStack
    st = OffloadedMoEStack(cfg)
    try:
        rng = np.random.default_rng(3)
        A, Bm = st.adapter[0]
        A_ref, B_ref = o.OracleWeights(cfg).adapter(0)
        s_dev = torch.empty(cfg.n, dtype=torch.float32, device=st.device)
        for B in (cfg.batch, 5, 1):       # two calls in a row with a smaller batch after a larger one
            _log(f"[static] {cfg.name} B={B}")
            x = rng.normal(size=(B, cfg.D)).astype(np.float32)
            xd = torch.from_numpy(x).to(st.device)
            s_dev.fill_(float("nan"))
            spp.adapter_predict_static(A.data_ptr(), Bm.data_ptr(), st.dtype_code, cfg.D, cfg.n, cfg.r,
                                       xd.data_ptr(), B, s_dev.data_ptr(), st.stream.cuda_stream)
            torch.cuda.synchronize()
            got = s_dev.cpu().numpy()
            want = spp.adapter_predict(st.ctx, 0, xd.data_ptr(), B, cfg.n)
            assert np.array_equal(got, want), (B, np.max(np.abs(got - want)))
            _, _, s_ora = o.adapter_scores(A_ref, B_ref, x.astype(np.float64))
            np.testing.assert_allclose(got, s_ora, rtol=1e-5, atol=2e-6)
        # refused before any device work: too large for the static scratch, NULL or misaligned pointers
        big = spp.STATIC_SCRATCH_FLOATS // (cfg.n + cfg.r) + 1
        for args in ((A.data_ptr(), xd.data_ptr(), big), (0, xd.data_ptr(), 1), (A.data_ptr() + 8, xd.data_ptr(), 1),
                     (A.data_ptr(), xd.data_ptr() + 4, 1)):
            with pytest.raises(spp.SppError) as e:
                spp.adapter_predict_static(args[0], Bm.data_ptr(), st.dtype_code, cfg.D, cfg.n, cfg.r, args[1],
                                           args[2], s_dev.data_ptr(), st.stream.cuda_stream)
            assert e.value.status == spp.SPP_EINVAL
    finally:
        st.close()
