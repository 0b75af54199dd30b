"""Named synthetic workloads.

The shapes follow the paper's setting (RoPE full-attention models serving RAG
chunks and agent-memory records as context units, Sections 2.2, 3 and 6.1):
Llama-3-8B-shaped layers (32 query / 8 KV heads, head dim 128) for RAG and
agent memory, a Llama-3-70B-shaped layer (64 / 8 / 128) for long-context RAG,
and page size B = 16 (the fixed storage block of Section 5.1).  The datasets
and traces the paper replays are not available, so every workload is drawn
from seeded distributions that stand in for them: Zipf unit popularity,
a fixed count or Bernoulli draw of missing units, and a fixed recompute
window per reused unit (EPIC's chunk-initial window, Section 7).
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace


@dataclass(frozen=True)
class ModelShape:
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    page_size: int = 16
    kv_dtype: str = "bf16"      # "f32" | "bf16" | "e4m3"
    act_dtype: str = "bf16"     # "f32" | "bf16"
    rope_theta: float = 500000.0
    max_position: int = 65536


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    model: ModelShape
    seed: int
    n_requests: int
    # units per request: fixed count, or (lo, hi) inclusive uniform range
    units_per_request: int | tuple[int, int]
    # unit length: fixed, or (lo, hi) inclusive uniform range per unit id
    unit_tokens: int | tuple[int, int]
    pool_units: int                 # size of the unit universe (cache pool)
    zipf_s: float
    # missing units: exact count per request (int) or Bernoulli hit prob (float)
    n_missing: int | None = None
    hit_prob: float | None = None
    n_recompute: int = 16
    instruction_tokens: int = 64
    query_tokens: int = 32
    # explicit residency pattern for every request (overrides the draws)
    residency_pattern: tuple[int, ...] | None = None
    # unit ids per request in order (overrides the Zipf draw)
    unit_order: tuple[tuple[int, ...], ...] | None = None
    # retain newly computed units into the pool
    retain_misses: bool = True
    # miss scope of every request: "global" (missing units are rows of the
    # final pass over the whole prompt) or "local" (prefilled alone, then
    # composed with a recompute window like hits)
    miss_scope: str = "global"
    description: str = ""
    extra: dict = field(default_factory=dict)

    def with_(self, **kw) -> "WorkloadConfig":
        return replace(self, **kw)


_L8B = ModelShape(n_q_heads=32, n_kv_heads=8, head_dim=128, kv_dtype="bf16",
                  act_dtype="bf16", rope_theta=500000.0, max_position=65536)
_L70B = ModelShape(n_q_heads=64, n_kv_heads=8, head_dim=128, kv_dtype="bf16",
                   act_dtype="bf16", rope_theta=500000.0, max_position=65536)

CONFIGS: dict[str, WorkloadConfig] = {}


def _reg(cfg: WorkloadConfig) -> WorkloadConfig:
    CONFIGS[cfg.name] = cfg
    return cfg


# 1 request, one layer, 4q/4kv heads, head dim 64, fp32, theta 1e4.  Four
# 64-token units laid out [MISS, HIT, MISS, HIT] followed by a 16-token
# query: 272 prompt tokens, each reused unit recomputes its first 4 tokens.
TINY = _reg(WorkloadConfig(
    name="tiny", seed=0,
    model=ModelShape(n_q_heads=4, n_kv_heads=4, head_dim=64, kv_dtype="f32",
                     act_dtype="f32", rope_theta=10000.0, max_position=4096),
    n_requests=1, units_per_request=4, unit_tokens=64, pool_units=4,
    zipf_s=1.0, n_recompute=4, instruction_tokens=0, query_tokens=16,
    residency_pattern=(0, 1, 0, 1), unit_order=((0, 1, 2, 3),),
    description="1 request, 4 units x 64 tokens [M,H,M,H] + 16-token query, fp32"))

# Llama-3-8B-shaped RAG layer: 8 requests x 10 units x 512 tokens from a
# 2,000-unit pool with Zipf(1.1) popularity, 3 missing units per request,
# 64-token instruction + 32-token query, 16 recomputed tokens per reused unit.
RAG_8B = _reg(WorkloadConfig(
    name="rag8b", seed=1, model=_L8B, n_requests=8, units_per_request=10,
    unit_tokens=512, pool_units=2000, zipf_s=1.1, n_missing=3,
    n_recompute=16, instruction_tokens=64, query_tokens=32,
    description="RAG, 8 req x 10 units x 512 tok, Zipf 1.1 over 2,000 units, "
                "3 missing/req, bf16, 32q/8kv/d128"))

# Agent memory: 32 requests x U{20..60} records of U{64..256} tokens from a
# 20,000-record pool (Zipf 1.0), each record a hit with probability 0.75,
# 256-token instruction + 64-token query, 8 recomputed tokens per reused record.
AGENT_8B = _reg(WorkloadConfig(
    name="agent8b", seed=2, model=_L8B, n_requests=32,
    units_per_request=(20, 60), unit_tokens=(64, 256), pool_units=20000,
    zipf_s=1.0, hit_prob=0.75, n_recompute=8, instruction_tokens=256,
    query_tokens=64,
    description="agent memory, 32 req x U{20..60} records x U{64..256} tok, "
                "Zipf 1.0 over 20,000 records, hit p=0.75, bf16"))

# Long-context RAG, Llama-3-70B-shaped layer: 4 requests x 32 units x 1,024
# tokens (about 33k-token prompts), 3 missing units per request, 32 recomputed
# tokens per reused unit, pool of 3,125 units = 200k pages.
LONG_70B = _reg(WorkloadConfig(
    name="long70b", seed=3, model=_L70B, n_requests=4, units_per_request=32,
    unit_tokens=1024, pool_units=3125, zipf_s=1.1, n_missing=3,
    n_recompute=32, instruction_tokens=64, query_tokens=32,
    description="long-context RAG, 4 req x 32 units x 1,024 tok, 64q/8kv/d128"))

# fp8 KV pool: the 8B RAG config with e4m3 cached states and a per-page scale,
# batch 16, 16 units x 512 tokens, 3 of 16 missing per request.
FP8_RAG = _reg(WorkloadConfig(
    name="fp8rag", seed=4,
    model=replace(_L8B, kv_dtype="e4m3"), n_requests=16, units_per_request=16,
    unit_tokens=512, pool_units=2000, zipf_s=1.1, n_missing=3,
    n_recompute=16, instruction_tokens=64, query_tokens=32,
    description="fp8 e4m3 KV pool, 16 req x 16 units x 512 tok, bf16 activations"))

# ---- small parity cases: several tiles, ragged tails, unaligned offsets ----
_RAG_SMALL_SHAPE = replace(_L8B, max_position=8192)

SMALL_BF16 = _reg(WorkloadConfig(
    name="small_bf16", seed=11, model=_RAG_SMALL_SHAPE, n_requests=3,
    units_per_request=(3, 6), unit_tokens=(20, 150), pool_units=12,
    zipf_s=1.0, hit_prob=0.6, n_recompute=5, instruction_tokens=37,
    query_tokens=19,
    description="small bf16: unaligned offsets, ragged unit tails"))

SMALL_BF16_G8 = _reg(WorkloadConfig(
    name="small_bf16_g8", seed=12, model=replace(_L70B, max_position=8192),
    n_requests=2, units_per_request=4, unit_tokens=(40, 130), pool_units=8,
    zipf_s=1.1, n_missing=1, n_recompute=7, instruction_tokens=21,
    query_tokens=13,
    description="small bf16, 64q/8kv (GQA group 8)"))

SMALL_FP8 = _reg(WorkloadConfig(
    name="small_fp8", seed=14, model=replace(_RAG_SMALL_SHAPE, kv_dtype="e4m3"),
    n_requests=3, units_per_request=(3, 5), unit_tokens=(2, 9), pool_units=10,
    zipf_s=1.0, hit_prob=0.6, n_recompute=16, instruction_tokens=32,
    query_tokens=20, extra={"unit_tokens_multiple": 16},
    description="small e4m3 pool: page-aligned units of 32..144 tokens, "
                "ragged final page"))

SMALL_F32 = _reg(WorkloadConfig(
    name="small_f32", seed=13,
    model=ModelShape(n_q_heads=8, n_kv_heads=2, head_dim=128, kv_dtype="f32",
                     act_dtype="f32", rope_theta=10000.0, max_position=4096),
    n_requests=2, units_per_request=(2, 4), unit_tokens=(17, 90),
    pool_units=6, zipf_s=1.0, hit_prob=0.5, n_recompute=3,
    instruction_tokens=9, query_tokens=11,
    description="small fp32, GQA 4, ragged"))


def get_config(name: str) -> WorkloadConfig:
    try:
        return CONFIGS[name]
    except KeyError as e:
        raise KeyError(f"unknown workload {name!r}; have {sorted(CONFIGS)}") from e
