"""The five synthetic workloads the paged prefix-reuse attention path is measured and checked on.

Each workload stands in for a shape of the paper's semantic-operator pipelines (Section 2.1,
"Prefix sharing in semantic operators", and the workload table of Section 7.2): a downstream
operator's prompt `[S | C(t) | I_op]` reuses the cached KV of `[S | C(t)]` left by the upstream
operator and prefills only `I_op`, after which decode runs over the same cache. The paper's
datasets are not used; every tensor is a seeded N(0,1) draw rounded to bf16.

Readings where the workload text leaves a choice open:
  * uniform[a, b] is a discrete uniform over the integers a..b, both ends included, drawn
    independently per sequence;
  * a decode "context length" C is the number of tokens already cached; the step appends one
    token and attends over C + 1 keys;
  * the tiny workload's "64-block pool" is max(64, blocks needed); the pools of the decode,
    mixed and long-document workloads are ceil(1.25 x blocks needed);
  * the long-document lognormal has median 4096 and sigma ln 2 (so the clip bounds sit at
    +-2 sigma), drawn as round(exp(ln 4096 + sigma z)) and then clipped;
  * the shared operator prompt is 512 tokens = 32 full blocks referenced by every table.

This module holds no attention arithmetic: only sizes, distributions and seeds.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass

SEED_BASE = 2607_23815
BLOCK_SIZE = 16


@dataclass(frozen=True)
class Dist:
    """A length distribution: ("uniform", lo, hi), ("const", v) or
    ("lognormal", median, sigma, lo, hi)."""

    kind: str
    params: tuple

    @staticmethod
    def uniform(lo: int, hi: int) -> "Dist":
        return Dist("uniform", (int(lo), int(hi)))

    @staticmethod
    def const(v: int) -> "Dist":
        return Dist("const", (int(v),))

    @staticmethod
    def lognormal(median: float, sigma: float, lo: int, hi: int) -> "Dist":
        return Dist("lognormal", (float(median), float(sigma), int(lo), int(hi)))

    @property
    def max_value(self) -> int:
        if self.kind == "uniform":
            return self.params[1]
        if self.kind == "const":
            return self.params[0]
        return self.params[3]


@dataclass(frozen=True)
class BatchSpec:
    """One batch of sequences launched together.

    kind "prefill": each sequence has `prefix` cached tokens and `new` tokens to append and
    attend (new token j sees keys 0 .. prefix + j).
    kind "decode": each sequence has `prefix` = C cached tokens and appends one token, which
    attends over all C + 1 keys.
    """

    kind: str
    n_seqs: int
    prefix: Dist
    new: Dist


@dataclass(frozen=True)
class WorkloadSpec:
    name: str
    index: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    batches: tuple
    pool: tuple  # ("min", n) | ("fixed", n) | ("scale", factor)
    shared_prompt_tokens: int = 0
    block_size: int = BLOCK_SIZE
    description: str = ""

    @property
    def seed(self) -> int:
        return SEED_BASE + self.index

    def scaled(self, **n_seqs_per_kind) -> "WorkloadSpec":
        """The same distributions with fewer sequences (small enough for the oracle).
        Keyword arguments map a batch kind ("prefill"/"decode") to its new sequence count."""
        batches = tuple(
            dataclasses.replace(b, n_seqs=int(n_seqs_per_kind.get(b.kind, b.n_seqs)))
            for b in self.batches
        )
        pool = self.pool
        if pool[0] == "fixed":
            # keep the fixed pool's occupancy roughly as sparse as at full size
            full = sum(b.n_seqs for b in self.batches)
            small = sum(b.n_seqs for b in batches)
            pool = ("fixed", max(64, int(math.ceil(pool[1] * small / full))))
        return dataclasses.replace(self, batches=batches, pool=pool)


TINY = WorkloadSpec(
    name="tiny_prefix_reuse_prefill",
    index=1,
    num_q_heads=4,
    num_kv_heads=2,
    head_dim=64,
    batches=(BatchSpec("prefill", 8, Dist.uniform(32, 128), Dist.uniform(16, 64)),),
    pool=("min", 64),
    description="8 tuples, 4/2 heads, head_dim 64, prefix U[32,128], new U[16,64]",
)

LLAMA3_8B_PREFILL = WorkloadSpec(
    name="llama3_8b_prefix_reuse_prefill",
    index=2,
    num_q_heads=32,
    num_kv_heads=8,
    head_dim=128,
    batches=(BatchSpec("prefill", 256, Dist.uniform(256, 1024), Dist.uniform(64, 256)),),
    pool=("fixed", 40000),
    description="256 tuples, 32/8 heads, head_dim 128, prefix U[256,1024], new U[64,256], "
    "40k-block pool with random placement",
)

LLAMA3_8B_DECODE = WorkloadSpec(
    name="llama3_8b_paged_decode",
    index=3,
    num_q_heads=32,
    num_kv_heads=8,
    head_dim=128,
    batches=(BatchSpec("decode", 512, Dist.uniform(512, 2048), Dist.const(1)),),
    pool=("scale", 1.25),
    description="512 sequences, 32/8 heads, head_dim 128, context U[512,2048], one new token",
)

MIXED_70B = WorkloadSpec(
    name="mixed_70b_layer",
    index=4,
    num_q_heads=64,
    num_kv_heads=8,
    head_dim=128,
    batches=(
        BatchSpec("prefill", 128, Dist.uniform(512, 2048), Dist.uniform(128, 512)),
        BatchSpec("decode", 384, Dist.uniform(256, 4096), Dist.const(1)),
    ),
    pool=("scale", 1.25),
    description="128 prefill tuples (prefix U[512,2048], new U[128,512]) + 384 decode "
    "sequences (context U[256,4096]), 64/8 heads, head_dim 128, one pool",
)

LONG_DOC_SHARED_PROMPT = WorkloadSpec(
    name="long_doc_shared_prompt",
    index=5,
    num_q_heads=32,
    num_kv_heads=8,
    head_dim=128,
    batches=(
        BatchSpec(
            "prefill",
            64,
            Dist.lognormal(4096.0, math.log(2.0), 1024, 16384),
            Dist.uniform(128, 512),
        ),
    ),
    pool=("scale", 1.25),
    shared_prompt_tokens=512,
    description="64 tuples, 32/8 heads, head_dim 128, a 512-token prompt shared by every "
    "table, document prefix lognormal(median 4096) clipped [1024,16384], new U[128,512]",
)

ALL = (TINY, LLAMA3_8B_PREFILL, LLAMA3_8B_DECODE, MIXED_70B, LONG_DOC_SHARED_PROMPT)

# Beyond the five: a batch too small to fill the chip, made of very long cached documents
# with a short downstream suffix each (the case the prefill's key split is for).
LONG_PREFIX_FEW_TUPLES = WorkloadSpec(
    name="long_prefix_few_tuples",
    index=6,
    num_q_heads=32,
    num_kv_heads=8,
    head_dim=128,
    batches=(BatchSpec("prefill", 4, Dist.uniform(24576, 32768), Dist.uniform(64, 256)),),
    pool=("scale", 1.25),
    description="4 tuples, 32/8 heads, head_dim 128, prefix U[24576,32768], new U[64,256]",
)
EXTRA = (LONG_PREFIX_FEW_TUPLES,)
BY_NAME = {w.name: w for w in ALL + EXTRA}
