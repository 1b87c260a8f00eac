"""Seeded synthetic semantic-operator pipelines (inputs of the scheduler; no scheduling logic).

A pipeline is a list of stages; stage s runs one operator per task and, unless it is the last,
joins every surviving task with `fanout` right-side rows (a Cartesian product). Per task the
generator draws the tokens the stage appends (the operator's instruction plus the tuple or
right-side row it adds), the tokens the request generates, and whether the predicate drops the
tuple. These draws stand in for the paper's datasets, which are not available: the shapes
follow the workloads it describes (long reused tuple prefixes of about 400 to 2,700 tokens,
a fan-out of 17 hypotheses per contract, one- or two-token predicate answers, map outputs of
tens of tokens)."""
from dataclasses import dataclass

import numpy as np

from .configs import SEED_BASE, Dist
from .gen import _draw


@dataclass(frozen=True)
class StageSpec:
    suffix: Dist        # tokens the task appends to its parent's prefix
    out: Dist           # tokens its request generates (>= 1)
    keep: float = 1.0   # probability that the predicate keeps the tuple
    fanout: int = 1     # right-side rows joined with each surviving task (not the last stage)


@dataclass(frozen=True)
class PipelineSpec:
    name: str
    index: int
    num_tuples: int
    stages: tuple

    @property
    def seed(self) -> int:
        return SEED_BASE + 500 + self.index

    def scaled(self, num_tuples: int) -> "PipelineSpec":
        return PipelineSpec(self.name, self.index, num_tuples, self.stages)


def make_pipeline(spec: PipelineSpec, seed=None):
    """dict(fanout, suffix, out_len, filtered): per-stage int arrays in task order (task t of
    stage s + 1 is row t % fanout[s] joined with task t // fanout[s] of stage s)."""
    rng = np.random.default_rng(spec.seed if seed is None else seed)
    count = spec.num_tuples
    fanout, suffix, out_len, filtered = [], [], [], []
    for s, st in enumerate(spec.stages):
        suffix.append(_draw(st.suffix, count, rng).astype(np.int64))
        out_len.append(np.maximum(_draw(st.out, count, rng), 1).astype(np.int64))
        filtered.append((rng.random(count) >= st.keep).astype(np.int64))
        f = st.fanout if s + 1 < len(spec.stages) else 1
        fanout.append(f)
        count *= f
    return dict(fanout=fanout, suffix=suffix, out_len=out_len, filtered=filtered)


# filter -> map over clinical-note-sized tuples (about 400 tokens)
FILTER_MAP = PipelineSpec("filter_map", 0, 1000, (
    StageSpec(Dist.lognormal(400, 0.35, 120, 1200), Dist.uniform(1, 2), keep=0.5),
    StageSpec(Dist.uniform(40, 80), Dist.uniform(8, 60)),
))

# map over contract-sized documents, then a Cartesian product with 17 hypotheses judged by a
# short predicate
CP_FANOUT = PipelineSpec("cp_fanout", 1, 600, (
    StageSpec(Dist.lognormal(2145, 0.3, 800, 4000), Dist.uniform(4, 24), fanout=17),
    StageSpec(Dist.uniform(30, 45), Dist.uniform(1, 2), keep=0.4),
))

# filter -> map -> Cartesian product (fan-out 4) with a predicate
THREE_STAGE = PipelineSpec("three_stage", 2, 400, (
    StageSpec(Dist.lognormal(600, 0.4, 150, 2000), Dist.uniform(1, 2), keep=0.6),
    StageSpec(Dist.uniform(30, 60), Dist.uniform(10, 40), fanout=4),
    StageSpec(Dist.uniform(20, 40), Dist.uniform(1, 3), keep=0.5),
))

PIPELINES = (FILTER_MAP, CP_FANOUT, THREE_STAGE)
