"""Synthetic GQA decode-step inputs with the shapes of the paper's workloads.

The paper measures on Llama-3.1-8B / Qwen3 attention states and on standard-normal random embeddings
(Appendix E.2). Neither the models nor their states are available, so every input here is synthetic
and seeded. Keys carry block structure so that within-block logit variation differs across blocks,
which is what CompKV's score is sensitive to (Sections 3.2 and 4.1):

* block beta has a centroid c_beta ~ N(0, I_d) and a spread sigma_beta;
* key j of block beta is k_j = c_beta + sigma_beta * eps_j with eps_j ~ N(0, I_d);
* values v_j ~ N(0, I_d); one query per head q ~ N(0, I_d) / sqrt(128).

Optional structure (per workload): a share of the non-mandatory blocks gets a shared key offset
along the unit's mean query, making them high-mass and low-variance; a share of the query heads
is made peaky by scaling. Every array is drawn in float32 and rounded to bf16 (round to nearest
even); consumers read the bf16 bits. Each (layer, batch element, KV head) unit is drawn from its
own seeded stream, so any unit can be regenerated alone.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, replace

import numpy as np

# stream tags of the per-unit seed sequences
_TAG_KNOISE, _TAG_V, _TAG_Q, _TAG_BLOCKS, _TAG_OFFSET, _TAG_PEAKY = 0, 1, 2, 3, 4, 5


@dataclass(frozen=True)
class Workload:
    """Shape and recipe of one synthetic decode workload.

    ``context`` is the number of tokens present when the measured decode step runs (the new token
    included). ``decode_steps`` extra rows of capacity are drawn for streaming appends.
    ``budget_blocks`` is the total number of exactly read blocks, mandatory blocks included.
    """

    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    context: int
    block_size: int
    budget_blocks: int
    n_var_groups: int = 4
    layers: int = 1
    sigma: str = "loguniform"  # "loguniform": [0.05, 1.0]; "lognormal": median 0.2, shape 1.0
    offset_frac: float = 0.0  # share of blocks given the shared high-mass key offset
    offset_logit: float = 3.0  # mean over the unit's heads of s*q.delta for the offset
    offset_sigma: float = 0.05  # spread of offset blocks
    peaky_frac: float = 0.0  # share of query heads scaled by peaky_scale
    peaky_scale: float = 4.0
    decode_steps: int = 0
    seed: int = 1000

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def capacity(self) -> int:
        return self.context + self.decode_steps

    @property
    def units(self) -> int:
        return self.batch * self.n_kv_heads

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def _w(**kw) -> Workload:
    return Workload(**kw)


# The synthetic decode workloads: a tiny case, a Llama-3-8B-shaped 32K layer, a 128K batch-4
# long-context case, a wide-GQA (64 query heads / 8 KV heads) batch-8 case, a streaming case, and two
# score-fidelity cases.
WORKLOADS = {
    "tiny_4k": _w(name="tiny_4k", batch=1, n_q_heads=8, n_kv_heads=2, head_dim=128, context=4096,
                  block_size=16, budget_blocks=16, seed=1000),
    "llama8b_32k": _w(name="llama8b_32k", batch=1, n_q_heads=32, n_kv_heads=8, head_dim=128,
                      context=32768, block_size=32, budget_blocks=65, offset_frac=0.05, seed=1001),
    "long_128k": _w(name="long_128k", batch=4, n_q_heads=32, n_kv_heads=8, head_dim=128,
                    context=131072, block_size=32, budget_blocks=64, sigma="lognormal", seed=1002),
    "wide_gqa_64k": _w(name="wide_gqa_64k", batch=8, n_q_heads=64, n_kv_heads=8, head_dim=128,
                       context=65536, block_size=64, budget_blocks=32, peaky_frac=0.1, seed=1003),
    "streaming_128k": _w(name="streaming_128k", batch=2, n_q_heads=32, n_kv_heads=8, head_dim=128,
                         context=131072, block_size=32, budget_blocks=128, layers=4,
                         decode_steps=256, seed=1004),
    # score fidelity against the exact residual (Appendix B.2 setting: 32 query / 8 KV heads, 16-token
    # blocks, a 512-token budget = 32 blocks of which 3 mandatory), on two key recipes
    "fidelity_16k": _w(name="fidelity_16k", batch=1, n_q_heads=32, n_kv_heads=8, head_dim=128, context=16384,
                       block_size=16, budget_blocks=32, offset_frac=0.05, seed=1005),
    "fidelity_lognormal_16k": _w(name="fidelity_lognormal_16k", batch=1, n_q_heads=32, n_kv_heads=8,
                                 head_dim=128, context=16384, block_size=16, budget_blocks=32,
                                 sigma="lognormal", seed=1006),
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even) and return the 16-bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 values (exact)."""
    return (np.ascontiguousarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(w: Workload, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.seed, *key])))


def _block_sigmas(w: Workload, rng: np.random.Generator, n_blocks: int) -> np.ndarray:
    if w.sigma == "loguniform":
        return np.exp(rng.uniform(math.log(0.05), math.log(1.0), n_blocks)).astype(np.float32)
    if w.sigma == "lognormal":
        return np.exp(math.log(0.2) + rng.standard_normal(n_blocks)).astype(np.float32)
    raise ValueError(f"unknown sigma recipe {w.sigma!r}")


def gen_queries(w: Workload, layer: int, b: int, step: int = 0) -> np.ndarray:
    """bf16 bits of the queries of batch element ``b`` at decode ``step``: [n_q_heads][head_dim]."""
    rng = _rng(w, layer, b, step, _TAG_Q)
    q = rng.standard_normal((w.n_q_heads, w.head_dim), dtype=np.float32) / np.float32(math.sqrt(128.0))
    if w.peaky_frac > 0:
        n_peaky = int(round(w.peaky_frac * w.n_q_heads))
        heads = _rng(w, layer, b, _TAG_PEAKY).choice(w.n_q_heads, size=n_peaky, replace=False)
        q[heads] *= np.float32(w.peaky_scale)
    return f32_to_bf16_bits(q)


def offset_blocks(w: Workload, layer: int, b: int, h: int) -> np.ndarray:
    """Ids of the blocks of one unit that carry the shared high-mass key offset (none unless
    ``offset_frac`` > 0); the sink block and the two most recent blocks are never chosen."""
    if w.offset_frac <= 0:
        return np.zeros(0, dtype=np.int64)
    x_ctx = -(-w.context // w.block_size)
    cand = np.arange(1, max(1, x_ctx - 2))
    n_off = min(len(cand), int(round(w.offset_frac * x_ctx)))
    return _rng(w, layer, b, h, _TAG_OFFSET).choice(cand, size=n_off, replace=False)


def gen_unit_kv(w: Workload, layer: int, b: int, h: int) -> tuple[np.ndarray, np.ndarray]:
    """bf16 bits of the keys and values of one (layer, batch element, KV head) unit.

    Returns two [capacity][head_dim] uint16 arrays. Rows past ``context`` are the tokens that
    streaming decode steps append, drawn from the same block recipe (token n lies in block n // B).
    """
    d, B, cap = w.head_dim, w.block_size, w.capacity
    n_blocks = -(-cap // B)
    rb = _rng(w, layer, b, h, _TAG_BLOCKS)
    centroids = rb.standard_normal((n_blocks, d), dtype=np.float32)
    sigmas = _block_sigmas(w, rb, n_blocks)
    offset = np.zeros((n_blocks, d), dtype=np.float32)
    if w.offset_frac > 0:
        # shared offset along the unit's mean query, sized so that the mean over the unit's
        # heads of (q_g . delta) / sqrt(d) equals offset_logit
        qs = bf16_bits_to_f32(gen_queries(w, layer, b, 0))[h * w.group:(h + 1) * w.group]
        qbar = qs.astype(np.float64).mean(axis=0)
        delta = w.offset_logit * math.sqrt(d) * qbar / float(qbar @ qbar)
        chosen = offset_blocks(w, layer, b, h)
        offset[chosen] = delta.astype(np.float32)
        sigmas[chosen] = np.float32(w.offset_sigma)
    blk = np.arange(cap) // B
    k = _rng(w, layer, b, h, _TAG_KNOISE).standard_normal((cap, d), dtype=np.float32)
    k *= sigmas[blk, None]
    k += centroids[blk]
    k += offset[blk]
    v = _rng(w, layer, b, h, _TAG_V).standard_normal((cap, d), dtype=np.float32)
    return f32_to_bf16_bits(k), f32_to_bf16_bits(v)


def gen_layer(w: Workload, layer: int = 0, threads: int = 8):
    """All units of one layer: K, V bits [batch][n_kv_heads][capacity][d], q bits [batch][Hq][d]."""
    K = np.empty((w.batch, w.n_kv_heads, w.capacity, w.head_dim), dtype=np.uint16)
    V = np.empty_like(K)

    def one(idx):
        b, h = divmod(idx, w.n_kv_heads)
        K[b, h], V[b, h] = gen_unit_kv(w, layer, b, h)

    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        list(ex.map(one, range(w.units)))
    q = np.stack([gen_queries(w, layer, b, 0) for b in range(w.batch)])
    return K, V, q
