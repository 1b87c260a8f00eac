"""CPU tier for the scheduler's C ABI (pkv_sched_run without a device): the library's C++
scheduler and the oracle's model produce the same event trace, counters and final budgets
over the synthetic pipelines, every policy, both pinning modes, both eviction orders, tight
and roomy pools; bad configurations are refused before anything runs."""
import random

import numpy as np
import pytest

from oracle.scheduler import Config, Pipeline, run_schedule
from workloads.pipelines import PIPELINES, make_pipeline

STAT_KEYS = ("steps", "launches", "retries", "hits", "misses", "prefill_tokens",
             "reused_tokens", "decode_tokens", "cow_copies", "max_batch", "evictions",
             "prefill_chunks")


@pytest.fixture(scope="module")
def lib():
    from paper_2607_23815_amd import lib as L
    return L


def _both(lib, d, **kw):
    pipe = Pipeline(**d)
    policy, nb = kw.pop("policy"), kw.pop("num_blocks")
    m = run_schedule(pipe, Config(policy, nb, **kw))
    st, tr, bud = lib.pkv_sched_run(lib.sched_config(policy, nb, **kw), d["fanout"],
                                    d["suffix"], d["out_len"], d["filtered"],
                                    max_events=len(m.trace) + 10)
    return m, st, tr, bud


CASES = []
for k, spec in enumerate(PIPELINES):
    for policy in range(5):
        CASES.append((spec, policy, k * 10 + policy))


@pytest.mark.parametrize("spec,policy,seed", CASES,
                         ids=[f"{c[0].name}-{c[1]}" for c in CASES])
def test_library_scheduler_matches_the_model(lib, spec, policy, seed):
    rnd = random.Random(seed)
    d = make_pipeline(spec.scaled(rnd.choice([16, 40])))
    pipe = Pipeline(**d)
    mb = max(-(-(max(a) + 64 + pipe.prefix[s][int(np.argmax(a))]) // 16)
             for s, a in enumerate(d["suffix"]))
    for trial in range(3):
        nb = rnd.choice([mb * pipe.S + 8, 3 * mb * pipe.S, 20 * mb])
        kw = dict(policy=policy, num_blocks=nb, max_out=64, initial_bound=[8] * pipe.S,
                  static_bound=[rnd.choice([0, 0, 2, 64]) for _ in range(pipe.S)],
                  max_batch=rnd.choice([4, 16, 64]), pinning=rnd.choice([0, 1]),
                  eviction=rnd.choice([0, 1]), delta=rnd.choice([0, 7, 40]),
                  alpha=rnd.choice([1.0, 0.8]), beta=rnd.choice([0.5, 0.2]),
                  breadth_share=rnd.choice([0.3, 0.6]), min_obs=rnd.choice([1, 8]),
                  max_step_tokens=rnd.choice([0, 0, 5, 100, 2048]))
        try:
            m, st, tr, bud = _both(lib, d, **kw)
        except ValueError:  # the pool is below the stages' minimum budgets
            with pytest.raises(lib.PkvError):
                lib.pkv_sched_run(lib.sched_config(**{**kw}), d["fanout"], d["suffix"],
                                  d["out_len"], d["filtered"])
            continue
        mt = np.asarray(m.trace, dtype=np.int64).reshape(-1, 5)
        assert st["num_events"] == len(m.trace)
        if not np.array_equal(tr, mt):
            k = next(i for i in range(min(len(tr), len(mt))) if not np.array_equal(tr[i], mt[i]))
            raise AssertionError(f"trial {trial} {kw}: first difference at event {k}: "
                                 f"library {tr[k].tolist()} model {mt[k].tolist()}")
        for key in STAT_KEYS:
            assert st[key] == m.stats[key], (key, kw)
        assert st["outputs"] == len(m.out)
        assert list(bud) == m.budget


def test_trace_buffer_overflow_counts_every_event(lib):
    d = make_pipeline(PIPELINES[0].scaled(12))
    cfg = lib.sched_config(0, 800, max_out=64, initial_bound=[8, 8])
    st, tr, _ = lib.pkv_sched_run(cfg, d["fanout"], d["suffix"], d["out_len"], d["filtered"],
                                  max_events=5)
    assert tr.shape == (5, 5) and st["num_events"] > 5
    st2, tr2, _ = lib.pkv_sched_run(cfg, d["fanout"], d["suffix"], d["out_len"],
                                    d["filtered"], max_events=st["num_events"])
    assert np.array_equal(tr2[:5], tr)


def test_bad_configurations_are_refused(lib):
    d = make_pipeline(PIPELINES[0].scaled(4))
    args = (d["fanout"], d["suffix"], d["out_len"], d["filtered"])
    for kw in (dict(policy=7, num_blocks=800, max_out=64),
               dict(policy=0, num_blocks=800, max_out=0),
               dict(policy=0, num_blocks=800, max_out=64, max_batch=0),
               dict(policy=0, num_blocks=800, max_out=64, alpha=0.0),
               dict(policy=2, num_blocks=800, max_out=64, breadth_share=1.5),
               dict(policy=0, num_blocks=10, max_out=64),      # below the minimum budgets
               dict(policy=0, num_blocks=800, max_out=8),      # an output longer than max_out
               dict(policy=0, num_blocks=800, max_out=64, max_step_tokens=-1)):
        with pytest.raises(lib.PkvError) as e:
            lib.pkv_sched_run(lib.sched_config(**kw), *args)
        assert e.value.status == lib.PKV_ERR_INVALID_ARG
    huge = [np.full(len(a), 1 << 30) for a in d["suffix"]]  # lengths past the int32 range
    with pytest.raises(lib.PkvError) as e:
        lib.pkv_sched_run(lib.sched_config(0, 800, max_out=64), d["fanout"], huge,
                          d["out_len"], d["filtered"])
    assert e.value.status == lib.PKV_ERR_INVALID_ARG
    bad = dict(d)
    bad["suffix"] = [d["suffix"][0], d["suffix"][1][:-1]]
    with pytest.raises(Exception):
        lib.pkv_sched_run(lib.sched_config(0, 800, max_out=64), bad["fanout"], bad["suffix"],
                          bad["out_len"], bad["filtered"])
