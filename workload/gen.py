"""Seeded synthetic inputs for the offloaded-MoE decode hot path.

Every tensor is drawn from its own numpy PCG64 stream keyed by
``SeedSequence([seed, kind, layer, index])``, so any expert of any layer can be
regenerated on its own (random access, no multi-GB file).  Arrays are returned
in *storage* form: ``np.uint16`` bf16 bit patterns for bf16 configurations,
``np.float32`` for fp32 ones.  Decoding storage into arithmetic values is left
to each consumer.

Recipe (the paper trains adapters on real routers and evaluates on real
checkpoints; neither is available, so synthetic stand-ins take their place):

* router, expert (gate, up, down), shared-expert and stand-in projection
  weights: i.i.d. N(0, w_std^2) drawn in fp32, then rounded to bf16
  (round-to-nearest-even) for bf16 configurations; with router_rank k > 0 a
  router is instead G1 G2 w_std / sqrt(k) (G1 [n,k], G2 [k,D] i.i.d. N(0,1),
  a rank-k matrix with entries of std w_std), and down projections (routed
  and shared) are multiplied by update_scale;
* adapter of layer l (l < L-1): the rank-r truncated SVD of the *next* layer's
  stored router weights, W^{l+1} = U diag(sig) V^T, split symmetrically as
  A = diag(sqrt(sig_1..r)) V_r^T and B = U_r diag(sqrt(sig_1..r)) (zero rows /
  columns where r exceeds the rank), plus i.i.d. N(0, adapter_noise^2) on every
  entry; built once in fp64 and stored in the config dtype;
* 4-bit experts (codec "q4"): codes q = clip(round(N(0, 2.5^2)), -8, 7) + 8
  and per-block fp16 scales w_std/2.5 * U(0.75, 1.25), drawn directly (the
  codec is the workload's weight format; nothing is quantised here);
* layer-0 hidden states: an AR(1) sequence per batch element,
  h_0 = e_0, h_t = rho h_{t-1} + sigma e_t with e_t ~ N(0, I), built in fp64 and
  stored in the config dtype.
"""
from __future__ import annotations

import numpy as np

from .configs import Q4_BLOCK, MoEConfig

KIND_ROUTER = 1
KIND_ADAPTER_A = 2
KIND_ADAPTER_B = 3
KIND_GATE = 4
KIND_UP = 5
KIND_DOWN = 6
KIND_PROJ = 7
KIND_SHARED_GATE = 8
KIND_SHARED_UP = 9
KIND_SHARED_DOWN = 10
KIND_HIDDEN = 11
KIND_Q4_CODES = 12
KIND_Q4_SCALES = 13
KIND_SHARED_Q4_CODES = 14
KIND_SHARED_Q4_SCALES = 15


def _rng(cfg: MoEConfig, kind: int, layer: int, index: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, kind, layer, index])))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    b = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    return ((b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def _storage(cfg: MoEConfig, a32: np.ndarray) -> np.ndarray:
    return f32_to_bf16_bits(a32) if cfg.dtype == "bf16" else np.ascontiguousarray(a32, dtype=np.float32)


def _normal_weights(cfg: MoEConfig, kind: int, layer: int, index: int, shape, scale: float = 1.0) -> np.ndarray:
    g = _rng(cfg, kind, layer, index)
    a = g.standard_normal(int(np.prod(shape)), dtype=np.float32) * np.float32(cfg.w_std)
    if scale != 1.0:
        a = a * np.float32(scale)
    return _storage(cfg, a.reshape(shape))


def router_weight(cfg: MoEConfig, layer: int) -> np.ndarray:
    """Native router weights of a layer, [n, D]."""
    if cfg.router_rank <= 0:
        return _normal_weights(cfg, KIND_ROUTER, layer, 0, (cfg.n, cfg.D))
    k = cfg.router_rank
    g = _rng(cfg, KIND_ROUTER, layer, 0)
    g1 = g.standard_normal((cfg.n, k))
    g2 = g.standard_normal((k, cfg.D))
    a = (g1 @ g2) * (cfg.w_std / np.sqrt(k))
    return _storage(cfg, a.astype(np.float32))


def expert_weights(cfg: MoEConfig, layer: int, expert: int):
    """Routed expert ``expert`` of ``layer``: (gate [I,D], up [I,D], down [D,I])."""
    src = cfg.expert_layer(layer)
    return (_normal_weights(cfg, KIND_GATE, src, expert, (cfg.I, cfg.D)),
            _normal_weights(cfg, KIND_UP, src, expert, (cfg.I, cfg.D)),
            _normal_weights(cfg, KIND_DOWN, src, expert, (cfg.D, cfg.I), cfg.update_scale))


def _q4_expert(cfg: MoEConfig, kind_codes: int, kind_scales: int, layer: int, index: int):
    nb = cfg.D // Q4_BLOCK
    g = _rng(cfg, kind_codes, layer, index)
    codes = np.clip(np.rint(g.standard_normal((3, cfg.I, cfg.D)) * 2.5), -8, 7).astype(np.int16) + 8
    gs = _rng(cfg, kind_scales, layer, index)
    scales = cfg.w_std / 2.5 * gs.uniform(0.75, 1.25, size=(3, cfg.I, nb))
    if cfg.update_scale != 1.0:
        scales[2] *= cfg.update_scale
    scales = scales.astype(np.float16)
    # gate [I,D], its scales [I,D/32]; up alike; down [D,I] with scales [I,D/32] (blocks along D of column i)
    return (codes[0].astype(np.uint8), scales[0], codes[1].astype(np.uint8), scales[1],
            np.ascontiguousarray(codes[2].T.astype(np.uint8)), scales[2])


def expert_weights_q4(cfg: MoEConfig, layer: int, expert: int):
    """4-bit routed expert: (gate codes [I,D], gate scales [I,D/32], up codes,
    up scales, down codes [D,I], down scales [I,D/32]); codes uint8 in 0..15,
    scales float16."""
    return _q4_expert(cfg, KIND_Q4_CODES, KIND_Q4_SCALES, cfg.expert_layer(layer), expert)


def shared_expert_weights_q4(cfg: MoEConfig, layer: int, j: int):
    """4-bit always-resident shared expert ``j`` of ``layer`` (layout as expert_weights_q4)."""
    return _q4_expert(cfg, KIND_SHARED_Q4_CODES, KIND_SHARED_Q4_SCALES, layer, j)


def shared_expert_weights(cfg: MoEConfig, layer: int, j: int):
    """Always-resident shared expert ``j`` of ``layer``: (gate [I,D], up [I,D], down [D,I])."""
    return (_normal_weights(cfg, KIND_SHARED_GATE, layer, j, (cfg.I, cfg.D)),
            _normal_weights(cfg, KIND_SHARED_UP, layer, j, (cfg.I, cfg.D)),
            _normal_weights(cfg, KIND_SHARED_DOWN, layer, j, (cfg.D, cfg.I), cfg.update_scale))


def proj_weight(cfg: MoEConfig, layer: int) -> np.ndarray:
    """Dense stand-in projection of a layer (in place of attention), [D, D]."""
    return _normal_weights(cfg, KIND_PROJ, layer, 0, (cfg.D, cfg.D))


def _stored_values(cfg: MoEConfig, a: np.ndarray) -> np.ndarray:
    if cfg.dtype == "bf16":
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def adapter_weights(cfg: MoEConfig, layer: int, noise: float | None = None, rank: int | None = None):
    """Adapter (A [r,D], B [n,r]) attached to ``layer`` that predicts layer+1's logits.

    ``noise`` and ``rank`` override the configuration (used by special-case
    tests); the SVD is taken of the stored (rounded) next-layer router weights.
    """
    if not 0 <= layer < cfg.L - 1:
        raise ValueError("adapters exist for layers 0..L-2 only")
    r = cfg.r if rank is None else rank
    sd = cfg.adapter_noise if noise is None else noise
    W = _stored_values(cfg, router_weight(cfg, layer + 1))            # [n, D]
    U, sig, Vt = np.linalg.svd(W, full_matrices=False)                # U [n,k], Vt [k,D]
    k = min(r, sig.shape[0])
    root = np.sqrt(sig[:k])
    A = np.zeros((r, cfg.D))
    B = np.zeros((cfg.n, r))
    A[:k] = root[:, None] * Vt[:k]
    B[:, :k] = U[:, :k] * root[None, :]
    if sd > 0:
        A = A + sd * _rng(cfg, KIND_ADAPTER_A, layer).standard_normal(A.shape)
        B = B + sd * _rng(cfg, KIND_ADAPTER_B, layer).standard_normal(B.shape)
    return _storage(cfg, A.astype(np.float32)), _storage(cfg, B.astype(np.float32))


def hidden_states(cfg: MoEConfig, tokens: int | None = None) -> np.ndarray:
    """Layer-0 hidden states [tokens, batch, D] of ``batch`` independent AR(1) sequences."""
    T = cfg.tokens if tokens is None else tokens
    out = np.empty((T, cfg.batch, cfg.D), dtype=np.float64)
    for b in range(cfg.batch):
        g = _rng(cfg, KIND_HIDDEN, 0, b)
        eps = g.standard_normal((T, cfg.D))
        h = eps[0].copy()
        out[0, b] = h
        for t in range(1, T):
            h = cfg.rho * h + cfg.sigma * eps[t]
            out[t, b] = h
    return _storage(cfg, out.astype(np.float32))
