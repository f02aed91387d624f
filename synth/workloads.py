"""Seeded synthetic attention-layer inputs with the shapes of the paper's models.

The paper measures on real prompts run through Qwen3 models; none of that is
available here, so these generators stand in for them.  Only the head counts,
head dimension, context lengths and block sizes follow the paper's models
(Qwen3-30B-A3B: 32 query / 4 KV heads; Qwen3-32B: 64 / 8; d = 128).  Keys are
built so that block radii vary (a per-block lognormal noise scale) and so that a
few "needle" keys are planted inside otherwise random blocks, aligned with a
later query: the mean-dilution situation the rescue branch is meant for.

Recipe (all streams numpy PCG64 seeded from (seed, stream tag, head index)):
  keys    k_t = mu_g + s_{g,b} * eps_t,  mu_g = 4 z/|z|,  s_{g,b} ~ LogNormal(mu, sigma)
  queries q_t = z_t + o_h,  o_h = 0.1 N(0, I) drawn once per query head
  values  v_t = z_t + o'_g, o'_g = 0.1 N(0, I) drawn once per KV head
  RoPE    NeoX rotate-half, theta_j = base^(-2j/d), positions 0..N-1, on Q and K
  needles key position p ~ U[B, N - 3B), target query position
          j ~ U[(floor(p/B) + n_local + 1) B, N), target query head h in the
          KV head's group; k_p = 3 q_j / |q_j| after RoPE
Everything is computed in float32 and rounded once to bf16 (nearest even).
"""

from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace

import numpy as np

from .bf16 import bf16_bits_from_f32, f32_from_bf16_bits

_TAG_KEYS, _TAG_QUERIES, _TAG_VALUES, _TAG_NEEDLES = 1, 2, 3, 4


@dataclass(frozen=True)
class Workload:
    name: str
    n_q_heads: int
    n_kv_heads: int
    seq_len: int
    block_size: int
    head_dim: int = 128
    rope: bool = False
    rope_base: float = 1.0e6
    needles_per_kv_head: int = 0
    needle_norm: float = 3.0   # |k_p| of a planted needle (the selector study also uses stronger ones)
    # (mu, sigma) of the lognormal per-block key-noise scale: one pair for all
    # KV heads, or one pair per KV head.
    key_noise: tuple = ((0.0, 0.5),)
    key_mean_norm: float = 4.0
    offset_scale: float = 0.1
    n_sink: int = 1
    n_local: int = 2
    n_recent: int = 0
    tau_base: float = 0.9
    tau_rescue: float = 0.95
    seed: int = 0
    note: str = field(default="", compare=False)

    @property
    def n_blocks(self) -> int:
        return -(-self.seq_len // self.block_size)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def noise_of(self, g: int) -> tuple:
        kn = self.key_noise
        return kn[g] if len(kn) > 1 else kn[0]

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def _qwen3_32b_noise() -> tuple:
    # KV heads 0-3: near-uniform small radii; 4-7: heavy-tailed radii.
    return tuple([(math.log(0.25), 0.02)] * 4 + [(0.0, 1.0)] * 4)


WORKLOADS = {
    # Small case the oracle finishes in seconds: 2 query heads share 1 KV head.
    "tiny-2k": Workload("tiny-2k", 2, 1, 2048, 64, rope=False, needles_per_kv_head=8,
                        note="seq 2048, GQA 2:1, B=64, 8 needles"),
    # Qwen3-30B-A3B-shaped layer.
    "qwen3-30b-a3b-32k": Workload("qwen3-30b-a3b-32k", 32, 4, 32768, 128, rope=True,
                                  needles_per_kv_head=64),
    "qwen3-30b-a3b-128k": Workload("qwen3-30b-a3b-128k", 32, 4, 131072, 128, rope=True,
                                   needles_per_kv_head=64),
    "qwen3-30b-a3b-128k-b64": Workload("qwen3-30b-a3b-128k-b64", 32, 4, 131072, 64, rope=True,
                                       needles_per_kv_head=64),
    "qwen3-30b-a3b-128k-b256": Workload("qwen3-30b-a3b-128k-b256", 32, 4, 131072, 256, rope=True,
                                        needles_per_kv_head=64),
    # Qwen3-32B-shaped layer with per-head radius heterogeneity.
    "qwen3-32b-64k": Workload("qwen3-32b-64k", 64, 8, 65536, 128, rope=True,
                              needles_per_kv_head=32, key_noise=_qwen3_32b_noise()),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def layer_schedule(n_layers: int = 48, master_seed: int = 48) -> list:
    """Per-layer variants of the 128K Qwen3-30B-A3B layer: the key-noise sigma
    and the needle count are drawn per layer so that density varies by layer."""
    rng = np.random.default_rng(master_seed)
    base = WORKLOADS["qwen3-30b-a3b-128k"]
    out = []
    for layer in range(n_layers):
        sigma = float(rng.uniform(0.25, 1.0))
        u = float(rng.uniform(-2.0, 2.0))
        n = int(round(64 * 2.0 ** u))
        out.append(base.with_(name=f"qwen3-30b-a3b-128k-layer{layer}", key_noise=((0.0, sigma),),
                              needles_per_kv_head=n, seed=1000 + layer))
    return out


def _rng(seed: int, tag: int, index: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(entropy=seed, spawn_key=(tag, index)))


def _rope_tables(n: int, d: int, base: float):
    half = d // 2
    inv = base ** (-2.0 * np.arange(half, dtype=np.float64) / d)
    ang = np.arange(n, dtype=np.float64)[:, None] * inv[None, :]
    return np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)


def _apply_rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    half = x.shape[-1] // 2
    x1, x2 = x[:, :half], x[:, half:]
    out = np.empty_like(x)
    out[:, :half] = x1 * cos - x2 * sin
    out[:, half:] = x2 * cos + x1 * sin
    return out


def _needle_plan(w: Workload) -> list:
    """[(g, key_pos, q_head, q_pos)] for every planted needle."""
    B, N = w.block_size, w.seq_len
    plan = []
    if w.needles_per_kv_head <= 0 or N < 4 * B:
        return plan
    for g in range(w.n_kv_heads):
        rng = _rng(w.seed, _TAG_NEEDLES, g)
        for _ in range(w.needles_per_kv_head):
            p = int(rng.integers(B, N - 3 * B))
            lo = min((p // B + w.n_local + 1) * B, N - 1)
            j = int(rng.integers(lo, N))
            h = g * w.group + int(rng.integers(w.group))
            plan.append((g, p, h, j))
    return plan


def make_inputs(w: Workload, threads: int | None = None) -> dict:
    """Return {"q", "k", "v"} as uint16 bf16 bit arrays [H][N][d] plus "needles"."""
    N, d, B = w.seq_len, w.head_dim, w.block_size
    M = w.n_blocks
    plan = _needle_plan(w)
    want = {}
    for (g, p, h, j) in plan:
        want.setdefault(h, set()).add(j)
    tables = _rope_tables(N, d, w.rope_base) if w.rope else None
    if threads is None:
        threads = max(1, min(8, len(os.sched_getaffinity(0))))

    q = np.empty((w.n_q_heads, N, d), dtype=np.uint16)
    k = np.empty((w.n_kv_heads, N, d), dtype=np.uint16)
    v = np.empty((w.n_kv_heads, N, d), dtype=np.uint16)
    needle_rows = {}

    def gen_q(h):
        rng = _rng(w.seed, _TAG_QUERIES, h)
        off = (w.offset_scale * rng.standard_normal(d)).astype(np.float32)
        x = rng.standard_normal((N, d), dtype=np.float32)
        x += off
        if tables is not None:
            x = _apply_rope(x, *tables)
        q[h] = bf16_bits_from_f32(x)
        return {j: x[j].copy() for j in want.get(h, ())}

    def gen_k(g):
        rng = _rng(w.seed, _TAG_KEYS, g)
        z = rng.standard_normal(d)
        mu = (w.key_mean_norm * z / np.linalg.norm(z)).astype(np.float32)
        m_ln, s_ln = w.noise_of(g)
        scales = rng.lognormal(m_ln, s_ln, size=M).astype(np.float32)
        x = rng.standard_normal((N, d), dtype=np.float32)
        x *= np.repeat(scales, B)[:N, None]
        x += mu
        if tables is not None:
            x = _apply_rope(x, *tables)
        for (gg, p, h, j) in plan:
            if gg == g:
                t = needle_rows[(h, j)]
                x[p] = w.needle_norm * t / np.linalg.norm(t)
        k[g] = bf16_bits_from_f32(x)

    def gen_v(g):
        rng = _rng(w.seed, _TAG_VALUES, g)
        off = (w.offset_scale * rng.standard_normal(d)).astype(np.float32)
        x = rng.standard_normal((N, d), dtype=np.float32)
        x += off
        v[g] = bf16_bits_from_f32(x)

    with ThreadPoolExecutor(threads) as ex:
        for h, rows in zip(range(w.n_q_heads), ex.map(gen_q, range(w.n_q_heads))):
            for j, row in rows.items():
                needle_rows[(h, j)] = row
        list(ex.map(gen_k, range(w.n_kv_heads)))
        list(ex.map(gen_v, range(w.n_kv_heads)))
    return {"q": q, "k": k, "v": v, "needles": plan}


def as_f32(bits: np.ndarray) -> np.ndarray:
    return f32_from_bf16_bits(bits)


def batch_workloads(base: Workload, seq_tokens, needles_per_2k: float | None = None) -> list:
    """One Workload per sequence of a batch: the base layer's heads and
    generator, the sequence's own length and seed (base.seed + s), and a needle
    count scaled to its length (needles_per_2k per 2048 tokens when given,
    else the base count)."""
    out = []
    for s, n in enumerate(seq_tokens):
        nd = base.needles_per_kv_head if needles_per_2k is None else int(round(needles_per_2k * n / 2048))
        out.append(base.with_(name=f"{base.name}-seq{s}", seq_len=int(n), seed=base.seed + s,
                              needles_per_kv_head=nd))
    return out


def make_batch_inputs(workloads: list, threads: int | None = None) -> dict:
    """Inputs of every sequence (make_inputs), packed along the token axis:
    {"q", "k", "v"} as [H][sum of N][d] bf16 bit arrays, plus "seq_tokens" and
    each sequence's "needles"."""
    parts = [make_inputs(w, threads) for w in workloads]
    return {x: np.concatenate([p[x] for p in parts], axis=1) for x in ("q", "k", "v")} | {
        "seq_tokens": [w.seq_len for w in workloads], "needles": [p["needles"] for p in parts]}
