"""Assemble a synthetic offloaded-MoE decode stack on the device and drive it.

PyTorch is used for device memory, pinned host memory and the compute stream
only; every step of the hot path runs in libspp (see ``spp.py``).  Expert
weights are packed into the library's blob layout (unit i = [gate row i | up
row i | down column i]) inside one pinned host store per layer: the offload
tier.  Router, adapter, stand-in projection and shared-expert weights are
resident in HBM.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional, Sequence

import numpy as np

from . import spp


def _torch_from_storage(a: np.ndarray, device):
    import torch
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


class OffloadedMoEStack:
    """One spp context over a whole synthetic stack (all L layers).

    ``adapter_values(l) -> (A, B)`` optionally replaces the seeded adapters
    (values, rounded to the storage dtype here) for router-preservation tests.
    """

    def __init__(self, cfg, device: str = "cuda:0", S: Optional[int] = None,
                 resident: Optional[Sequence[int]] = None, adapter_values=None,
                 threads: Optional[int] = None):
        import torch
        from workload import gen

        self.cfg = cfg
        self.torch = torch
        self.device = torch.device(device)
        torch.cuda.set_device(self.device)
        self.stream = torch.cuda.current_stream(self.device)
        self.S = cfg.S if S is None else S
        self.dtype_code = spp.DTYPE_BF16 if cfg.dtype == "bf16" else spp.DTYPE_F32
        self.desc = spp.make_desc(cfg.L, cfg.D, cfg.n, cfg.K, cfg.I, cfg.r, self.S, max_batch=cfg.batch,
                                  n_shared=cfg.n_shared, dtype=self.dtype_code, has_proj=cfg.has_proj,
                                  rms_eps=cfg.rms_eps,
                                  expert_codec=spp.CODEC_Q4 if cfg.codec == "q4" else spp.CODEC_PLAIN)
        q4 = cfg.codec == "q4"
        self.stride = spp.spp_blob_stride(self.desc)
        self.elem = cfg.elem_bytes
        # a tied offload tier (cfg.expert_layers) shares one host store between the layers it ties
        self.host_layers = cfg.host_layers
        threads = threads or min(16, os.cpu_count() or 1)

        self.router, self.adapter, self.proj, self.shared, self.host = [], [], [], [], []
        for l in range(cfg.L):
            self.router.append(_torch_from_storage(gen.router_weight(cfg, l), self.device))
            if l < cfg.L - 1 and cfg.r > 0:
                if adapter_values is not None:
                    A, B = adapter_values(l)
                    A, B = self._to_storage(A), self._to_storage(B)
                else:
                    A, B = gen.adapter_weights(cfg, l)
                self.adapter.append((_torch_from_storage(A, self.device), _torch_from_storage(B, self.device)))
            else:
                self.adapter.append(None)
            self.proj.append(_torch_from_storage(gen.proj_weight(cfg, l), self.device) if cfg.has_proj else None)
            if cfg.n_shared:
                buf = np.zeros(cfg.n_shared * self.stride, dtype=np.uint8)
                for j in range(cfg.n_shared):
                    dst = buf[j * self.stride:(j + 1) * self.stride]
                    if q4:
                        spp.spp_pack_expert_q4(self.desc, *gen.shared_expert_weights_q4(cfg, l, j), out=dst)
                    else:
                        spp.spp_pack_expert(self.desc, *gen.shared_expert_weights(cfg, l, j), out=dst)
                self.shared.append(torch.from_numpy(buf).to(self.device))
            else:
                self.shared.append(None)

        # offload tier: pinned host stores, blobs packed in parallel
        for hl in range(self.host_layers):
            self.host.append(torch.empty(cfg.n * self.stride, dtype=torch.uint8, pin_memory=True))
        views = [h.numpy() for h in self.host]

        def fill(job):
            hl, e = job
            dst = views[hl][e * self.stride:(e + 1) * self.stride]
            if q4:
                spp.spp_pack_expert_q4(self.desc, *gen.expert_weights_q4(cfg, hl, e), out=dst)
            else:
                spp.spp_pack_expert(self.desc, *gen.expert_weights(cfg, hl, e), out=dst)

        jobs = [(hl, e) for hl in range(self.host_layers) for e in range(cfg.n)]
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(fill, jobs))

        self.ctx = spp.spp_create(self.desc, self.stream.cuda_stream)
        for l in range(cfg.L):
            ad = self.adapter[l]
            spp.spp_bind_layer(self.ctx, l, self.router[l].data_ptr(),
                               ad[0].data_ptr() if ad else 0, ad[1].data_ptr() if ad else 0,
                               self.proj[l].data_ptr() if self.proj[l] is not None else 0,
                               self.shared[l].data_ptr() if self.shared[l] is not None else 0,
                               self.host[l % self.host_layers].data_ptr())
        self.resident = list(range(min(self.S, cfg.n))) if resident is None else list(resident)
        self.reset()
        # ping-pong hidden-state buffers [B, D] in the storage dtype
        nbytes = cfg.batch * cfg.D * self.elem
        self.hbuf = [torch.empty(nbytes, dtype=torch.uint8, device=self.device) for _ in range(2)]

    def reset(self):
        """Initial slot tables (the resident set in slots 0.., stamp 0) and step clock 0."""
        for l in range(self.cfg.L):
            spp.spp_set_resident(self.ctx, l, self.resident)
        spp.spp_set_clock(self.ctx, 0)

    def _to_storage(self, v):
        from workload.gen import f32_to_bf16_bits
        v = np.asarray(v, dtype=np.float32)
        return f32_to_bf16_bits(v) if self.cfg.dtype == "bf16" else v

    # ---------------------------------------------------------------- data

    def upload_hidden(self, h_storage: np.ndarray, buf: int = 0):
        """Copy stored hidden states [B, D] into ping-pong buffer ``buf``."""
        a = np.ascontiguousarray(h_storage).reshape(-1).view(np.uint8)
        self.hbuf[buf].copy_(self.torch.from_numpy(a.copy()))
        return self.hbuf[buf]

    def download(self, t, B: Optional[int] = None) -> np.ndarray:
        B = self.cfg.batch if B is None else B
        self.torch.cuda.synchronize(self.device)
        raw = t[: B * self.cfg.D * self.elem].cpu().numpy()
        dt = np.uint16 if self.cfg.dtype == "bf16" else np.float32
        return raw.view(dt).reshape(B, self.cfg.D).copy()

    # ------------------------------------------------------------- compute

    def layer(self, l: int, src: int, dst: int, M_max: int, B: Optional[int] = None):
        B = self.cfg.batch if B is None else B
        return spp.moe_layer_forward(self.ctx, l, self.hbuf[src].data_ptr(), self.hbuf[dst].data_ptr(), B,
                                     self.cfg.K, M_max)

    def step(self, h_storage: Optional[np.ndarray], M_max: int, B: Optional[int] = None):
        """One decode step through all layers; returns the per-layer (topk, gates, stats)."""
        if h_storage is not None:
            self.upload_hidden(h_storage, 0)
        out = []
        src = 0
        for l in range(self.cfg.L):
            out.append(self.layer(l, src, 1 - src, M_max, B))
            src = 1 - src
        self.last_buf = src
        return out

    def step_from(self, h_in_ptr: int, M_max: int, B: Optional[int] = None):
        """One decode step whose layer-0 input is read from device address ``h_in_ptr``."""
        B = self.cfg.batch if B is None else B
        out = []
        src_ptr = h_in_ptr
        dst = 0
        for l in range(self.cfg.L):
            out.append(spp.moe_layer_forward(self.ctx, l, src_ptr, self.hbuf[dst].data_ptr(), B, self.cfg.K, M_max))
            src_ptr = self.hbuf[dst].data_ptr()
            dst = 1 - dst
        self.last_buf = 1 - dst
        return out

    def decode_step_from(self, h_in_ptr: int, M_max: int, B: Optional[int] = None):
        """One decode step through all layers in a single library call
        (spp_decode_step); the output lands in hbuf[0].  Returns the per-layer
        (topk, gates, stats) like step_from."""
        B = self.cfg.batch if B is None else B
        topk, gates, stats = spp.spp_decode_step(self.ctx, self.cfg.L, h_in_ptr, self.hbuf[0].data_ptr(),
                                                 self.hbuf[1].data_ptr(), B, self.cfg.K, M_max)
        self.last_buf = 0
        return [(topk[l], gates[l], stats[l]) for l in range(self.cfg.L)]

    def close(self):
        if getattr(self, "ctx", None):
            spp.spp_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
