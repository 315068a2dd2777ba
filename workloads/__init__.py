"""Seeded synthetic inputs for the ragged paged decode / chunked-prefill path.

This module is shared by the oracle-side tests and by the GPU path's tests and
benchmark.  It only draws random numbers and shapes; it contains none of the
method's arithmetic (no retained-length rule, no clustering, no page
accounting, no partitioning, no attention).  Quantities that depend on the
method, such as the number of pool pages a workload needs, are passed in by the
caller.

Workload recipes (the paper's models and SCBench traces are not available, so
these stand in for them; the retention structure follows the paper's
observation of an input-invariant head ranking with a narrow per-head band,
Section 3.2):

  1  tiny decode, fp32: L=1, B=2, H=4, Hq=8, d=64, N=512, fixed ratios
     {1.0, 0.5, 0.25, 0.125}, page 16, two groups of two heads.
  2  Llama-3.1-8B-shaped decode, bf16: L=1, B=32, Hq=32, H=8, d=128, N=8192,
     top 25 % of (layer, head) pairs ~U(0.7,1.0), rest ~U(0.05,0.2), per-request
     jitter U(-0.03,0.03) clipped to [0.02,1], groups of 2; Q~N(0,1), K,V~0.5 N(0,1).
  3  Qwen2.5-32B-shaped decode step, bf16: L=64, B=64, Hq=64, H=8, d=128,
     N ~ clip(round(exp(ln 16384 + 0.75 Z)), 2048, 65536), top 20 % of pairs
     ~U(0.6,1.0), rest ~U(0.03,0.15), jitter as above, groups of 2.
  4  load-balance stress, bf16: L=1, B=128, Hq=32, H=8, d=128,
     N ~ U{1024..131072}, one seeded head at ratio 1.0, the other seven at
     0.02, no jitter, groups of 4.
  5  ragged chunked prefill, bf16: L=1, B=16, Hq=32, H=8, d=128, chunk 512,
     compressed history of a 16384-token context with config 2's ratios,
     groups of 2; Q, K, V ~ N(0,1).

"Top x % of heads" selects max(1, round(x*L*H)) (layer, head) pairs with a
seeded permutation of all L*H pairs.  Random streams: SeedSequence(1000+cfg)
spawned into (ratios, contexts, free list, q, k, v, kv-pool, importance scores).

Compression of a prefill chunk (config 5's chunk, or scaled-down cases) takes
importance scores per (request, KV head, chunk token) standing in for a
compression method's scoring function: N(0,1) fp32, optionally with a share of
exact ties, signed zeros, infinities and NaNs.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

# Stream indices of SeedSequence(1000 + cfg).spawn(N_STREAMS).
S_RATIO, S_CTX, S_FREE, S_Q, S_K, S_V, S_POOL, S_SCORE = range(8)
N_STREAMS = 8


@dataclasses.dataclass(frozen=True)
class Geometry:
    num_layers: int
    num_kv_heads: int
    num_q_heads: int
    head_dim: int
    page_size: int
    heads_per_group: int

    @property
    def num_groups(self) -> int:
        return self.num_kv_heads // self.heads_per_group

    @property
    def gqa(self) -> int:
        return self.num_q_heads // self.num_kv_heads


@dataclasses.dataclass
class Workload:
    name: str
    seed: int
    geom: Geometry
    batch: int
    dtype: str                 # "f32" or "bf16": storage type of Q, K, V and outputs
    ctx_len: np.ndarray        # int32 [B], context length N_b of each request
    budget: np.ndarray         # float64 [L][H], static per-head budget profile
    ratio: np.ndarray          # float64 [B][L][H], ratio each request actually uses
    q_scale: float = 1.0
    kv_scale: float = 1.0
    chunk_len: int = 0         # prefill chunk length (0 for decode workloads)

    def streams(self):
        return np.random.SeedSequence(self.seed).spawn(N_STREAMS)

    def rng(self, stream: int) -> np.random.Generator:
        return np.random.default_rng(self.streams()[stream])

    def torch_seed(self, stream: int) -> int:
        return int(self.streams()[stream].generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1))


def _two_level_profile(rng, L, H, frac_hi, hi, lo):
    """Static per-(layer, head) budgets: a seeded subset of pairs is high."""
    n_pairs = L * H
    n_hi = max(1, int(round(frac_hi * n_pairs)))
    order = rng.permutation(n_pairs)
    is_hi = np.zeros(n_pairs, dtype=bool)
    is_hi[order[:n_hi]] = True
    vals = np.where(is_hi, rng.uniform(hi[0], hi[1], n_pairs), rng.uniform(lo[0], lo[1], n_pairs))
    return vals.reshape(L, H).astype(np.float64)


def _jitter(rng, budget, batch, amp=0.03, lo=0.02, hi=1.0):
    L, H = budget.shape
    j = rng.uniform(-amp, amp, size=(batch, L, H))
    return np.clip(budget[None, :, :] + j, lo, hi).astype(np.float64)


def config(cfg: int) -> Workload:
    """The five synthetic workloads, at full size."""
    seed = 1000 + cfg
    ss = np.random.SeedSequence(seed).spawn(N_STREAMS)
    r_ratio = np.random.default_rng(ss[S_RATIO])
    r_ctx = np.random.default_rng(ss[S_CTX])
    if cfg == 1:
        g = Geometry(1, 4, 8, 64, 16, 2)
        budget = np.array([[1.0, 0.5, 0.25, 0.125]])
        ratio = np.broadcast_to(budget, (2, 1, 4)).copy()
        ctx = np.full(2, 512, dtype=np.int32)
        return Workload("tiny-fp32", seed, g, 2, "f32", ctx, budget, ratio)
    if cfg == 2:
        g = Geometry(1, 8, 32, 128, 16, 2)
        budget = _two_level_profile(r_ratio, 1, 8, 0.25, (0.7, 1.0), (0.05, 0.2))
        ratio = _jitter(r_ratio, budget, 32)
        ctx = np.full(32, 8192, dtype=np.int32)
        return Workload("llama8b-decode-bf16", seed, g, 32, "bf16", ctx, budget, ratio,
                        q_scale=1.0, kv_scale=0.5)
    if cfg == 3:
        g = Geometry(64, 8, 64, 128, 16, 2)
        budget = _two_level_profile(r_ratio, 64, 8, 0.20, (0.6, 1.0), (0.03, 0.15))
        ratio = _jitter(r_ratio, budget, 64)
        z = r_ctx.standard_normal(64)
        ctx = np.clip(np.round(np.exp(math.log(16384.0) + 0.75 * z)), 2048, 65536).astype(np.int32)
        return Workload("qwen32b-decode-step-bf16", seed, g, 64, "bf16", ctx, budget, ratio)
    if cfg == 4:
        g = Geometry(1, 8, 32, 128, 16, 4)
        budget = _two_level_profile(r_ratio, 1, 8, 0.10, (1.0, 1.0), (0.02, 0.02))
        ratio = np.broadcast_to(budget, (128, 1, 8)).copy()
        ctx = r_ctx.integers(1024, 131072, size=128, endpoint=True).astype(np.int32)
        return Workload("loadbalance-stress-bf16", seed, g, 128, "bf16", ctx, budget, ratio)
    if cfg == 5:
        g = Geometry(1, 8, 32, 128, 16, 2)
        budget = _two_level_profile(r_ratio, 1, 8, 0.25, (0.7, 1.0), (0.05, 0.2))
        ratio = _jitter(r_ratio, budget, 16)
        ctx = np.full(16, 16384, dtype=np.int32)
        return Workload("chunked-prefill-bf16", seed, g, 16, "bf16", ctx, budget, ratio, chunk_len=512)
    raise ValueError(f"unknown config {cfg}")


# Decode-step shapes of the four models of the paper's planning-cost table (Table 1), with config 3's batch,
# contexts and retention structure: (layers, query heads, KV heads).
MODEL_SHAPES = {
    "qwen2.5-7b": (28, 28, 4),
    "llama3.1-8b": (32, 32, 8),
    "qwen3-32b": (64, 64, 8),
    "llama3.1-70b": (80, 64, 8),
}


def model_step(name: str) -> Workload:
    """A decode step of one of MODEL_SHAPES: B = 64, d = 128, bf16, page 16, groups of 2 heads, contexts
    clip(round(exp(ln 16384 + 0.75 Z)), 2048, 65536), 20 % of (layer, head) pairs ~U(0.6, 1.0), the rest
    ~U(0.03, 0.15), per-request jitter (config 3's recipe)."""
    L, Hq, H = MODEL_SHAPES[name]
    seed = 2000 + sorted(MODEL_SHAPES).index(name)
    ss = np.random.SeedSequence(seed).spawn(N_STREAMS)
    r_ratio = np.random.default_rng(ss[S_RATIO])
    r_ctx = np.random.default_rng(ss[S_CTX])
    g = Geometry(L, H, Hq, 128, 16, 2)
    budget = _two_level_profile(r_ratio, L, H, 0.20, (0.6, 1.0), (0.03, 0.15))
    ratio = _jitter(r_ratio, budget, 64)
    z = r_ctx.standard_normal(64)
    ctx = np.clip(np.round(np.exp(math.log(16384.0) + 0.75 * z)), 2048, 65536).astype(np.int32)
    return Workload(f"{name}-decode-step-bf16", seed, g, 64, "bf16", ctx, budget, ratio)


def retention_scores(seed: int, sample: int, num_layers: int, num_heads: int, n_tokens: int,
                     head_spread: float = 1.0, sample_jitter: float = 0.1) -> np.ndarray:
    """Importance scores [L][H][N] float32 of one calibration sample: head (l, h) scores its tokens
    a_{l,h} + d_{s,l,h} + N(0, 1), with a static head offset a ~ N(0, head_spread^2) drawn from `seed`
    alone (the input-invariant head ranking) and a per-sample offset d ~ N(0, sample_jitter^2) (the
    narrow per-input band).  Stands in for a compression method's scores on a pilot context."""
    a = np.random.default_rng(np.random.SeedSequence(seed).spawn(1)[0]).standard_normal(
        (num_layers, num_heads, 1)) * head_spread
    rng = np.random.default_rng(np.random.SeedSequence([seed, 1 + sample]))
    d = rng.standard_normal((num_layers, num_heads, 1)) * sample_jitter
    z = rng.standard_normal((num_layers, num_heads, n_tokens), dtype=np.float32)
    return (z + (a + d).astype(np.float32)).astype(np.float32)


def custom(seed: int, geom: Geometry, batch: int, dtype: str, ctx_len, budget=None, ratio=None,
           frac_hi=0.25, hi=(0.7, 1.0), lo=(0.05, 0.2), jitter=0.03, chunk_len=0,
           q_scale=1.0, kv_scale=1.0) -> Workload:
    """A scaled-down workload with the same structure, for parity tests."""
    ss = np.random.SeedSequence(seed).spawn(N_STREAMS)
    r_ratio = np.random.default_rng(ss[S_RATIO])
    r_ctx = np.random.default_rng(ss[S_CTX])
    L, H = geom.num_layers, geom.num_kv_heads
    if np.isscalar(ctx_len) or isinstance(ctx_len, tuple):
        if isinstance(ctx_len, tuple):
            ctx = r_ctx.integers(ctx_len[0], ctx_len[1], size=batch, endpoint=True).astype(np.int32)
        else:
            ctx = np.full(batch, int(ctx_len), dtype=np.int32)
    else:
        ctx = np.asarray(ctx_len, dtype=np.int32)
    if budget is None:
        budget = _two_level_profile(r_ratio, L, H, frac_hi, hi, lo)
    budget = np.asarray(budget, dtype=np.float64).reshape(L, H)
    if ratio is None:
        ratio = _jitter(r_ratio, budget, batch, amp=jitter) if jitter > 0 else \
            np.broadcast_to(budget, (batch, L, H)).copy()
    ratio = np.asarray(ratio, dtype=np.float64).reshape(batch, L, H)
    return Workload(f"custom-{seed}", seed, geom, batch, dtype, ctx, budget, ratio,
                    q_scale=q_scale, kv_scale=kv_scale, chunk_len=chunk_len)


def pool_pages_for(pages_needed: int) -> int:
    """Pool size used by every workload: 5 % slack plus 64 spare pages."""
    return int(math.ceil(1.05 * pages_needed)) + 64


def free_list(wl: Workload, pool_pages: int, identity: bool = False) -> np.ndarray:
    """The caller's free page list: a seeded permutation of all pool pages."""
    if identity:
        return np.arange(pool_pages, dtype=np.int32)
    return wl.rng(S_FREE).permutation(pool_pages).astype(np.int32)


def page_elems(geom: Geometry) -> int:
    """Elements in one physical page: H_p heads x {K, V} x P tokens x d."""
    return geom.heads_per_group * 2 * geom.page_size * geom.head_dim


# ---------------------------------------------------------------- host tensors

def host_normal(wl: Workload, stream: int, shape, scale: float) -> np.ndarray:
    """float32 N(0, scale^2) draws, on the host (small workloads)."""
    return (wl.rng(stream).standard_normal(size=shape, dtype=np.float32) * np.float32(scale))


def host_q_decode(wl: Workload) -> np.ndarray:
    L, B, Hq, d = wl.geom.num_layers, wl.batch, wl.geom.num_q_heads, wl.geom.head_dim
    return host_normal(wl, S_Q, (L, B, Hq, d), wl.q_scale)


def host_pool(wl: Workload, pool_pages: int) -> np.ndarray:
    return host_normal(wl, S_POOL, (pool_pages, page_elems(wl.geom)), wl.kv_scale)


def host_prefill_inputs(wl: Workload):
    g = wl.geom
    C = wl.chunk_len
    q = host_normal(wl, S_Q, (wl.batch, C, g.num_q_heads, g.head_dim), wl.q_scale)
    k = host_normal(wl, S_K, (wl.batch, C, g.num_kv_heads, g.head_dim), wl.kv_scale)
    v = host_normal(wl, S_V, (wl.batch, C, g.num_kv_heads, g.head_dim), wl.kv_scale)
    return q, k, v


def host_scores(wl: Workload, shape, special: bool = False) -> np.ndarray:
    """Importance scores [B][H][C] float32: N(0,1); with `special`, 30 % are rounded to
    multiples of 0.5 (exact ties), and some are -0.0, +-inf or NaN."""
    rng = wl.rng(S_SCORE)
    s = rng.standard_normal(size=shape, dtype=np.float32)
    if special:
        u = rng.random(size=shape)
        s = np.where(u < 0.3, np.round(s * 2) / 2, s).astype(np.float32)
        s[(u >= 0.30) & (u < 0.33)] = -0.0
        s[(u >= 0.33) & (u < 0.35)] = np.nan
        s[(u >= 0.35) & (u < 0.36)] = np.inf
        s[(u >= 0.36) & (u < 0.37)] = -np.inf
    return s


# -------------------------------------------------------------- device tensors

def device_normal_(t, wl: Workload, stream: int, scale: float, chunk_elems: int = 1 << 28):
    """Fill a device tensor in place with N(0, scale^2), chunk by chunk.

    Uses torch's device generator so multi-GB pools never pass through the host.
    """
    import torch
    gen = torch.Generator(device=t.device)
    gen.manual_seed(wl.torch_seed(stream))
    flat = t.view(-1)
    n = flat.numel()
    for s in range(0, n, chunk_elems):
        e = min(n, s + chunk_elems)
        tmp = torch.randn(e - s, generator=gen, device=t.device, dtype=torch.float32)
        if scale != 1.0:
            tmp.mul_(scale)
        flat[s:e].copy_(tmp)
        del tmp
    return t
