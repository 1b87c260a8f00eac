"""Pins of the scheduler model (oracle/scheduler.py) on the CPU, against what the paper's
definitions fix and against values worked out by hand:

  * the query's result does not depend on the schedule: every policy outputs exactly the
    final-stage tasks whose whole chain survived its predicates (brute force over the inputs);
  * every created task is launched once plus once per retry, and all memory is released at
    the end;
  * sequential depth-first execution runs one task at a time, so its step count is the sum of
    the tasks' output lengths (Section 5.3);
  * explicit pinning never loses a prefix its children need (Section 6): no cache misses;
    blocking execution over a table larger than the cache misses every prefix, and over a small
    table misses none (Section 2.2's cliff);
  * a request that hits its bound is retried with a doubled bound (Section 6), worked by hand;
  * the token bound is the nearest-rank 99th percentile of observed ratios, worked by hand;
  * rebalancing: the first transfers of a small two-stage run, worked by hand; budgets always
    sum to the pool and never drop below minBudget; every transfer's source was starving or a
    middle stage was saturated when it was made (Algorithm 1, Rebalance).
"""
import numpy as np
import pytest

from oracle.block_pool import EXPLICIT, VIRTUAL
from oracle.scheduler import (ADAPTIVE, BLOCKING, BREADTH_FIRST, DEPTH_FIRST, EV_LAUNCH,
                              EV_OUTPUT, EV_RETRY, EV_TRANSFER, SEQUENTIAL, Config, Pipeline,
                              SchedulerModel, run_schedule)
from workloads.pipelines import PIPELINES, make_pipeline

POLICIES = [ADAPTIVE, DEPTH_FIRST, BREADTH_FIRST, SEQUENTIAL, BLOCKING]


def surviving_outputs(d):
    """Brute force: final-stage tasks whose chain of ancestors all passed their predicates."""
    S = len(d["suffix"])

    def alive(s, t):
        if d["filtered"][s][t]:
            return False
        return s == 0 or alive(s - 1, t // d["fanout"][s - 1])

    return sorted((S - 1, t) for t in range(len(d["suffix"][S - 1])) if alive(S - 1, t))


def created_tasks(d):
    """Tasks that get created: all of stage 0, and the children of every surviving task."""
    S = len(d["suffix"])
    n = len(d["suffix"][0])
    alive = [not d["filtered"][0][t] for t in range(n)]
    total = n
    for s in range(1, S):
        f = d["fanout"][s - 1]
        kids = [alive[t // f] for t in range(len(d["suffix"][s]))]
        total += sum(kids)
        alive = [k and not d["filtered"][s][t] for t, k in enumerate(kids)]
    return total


def small(spec, n):
    d = make_pipeline(spec.scaled(n))
    return d, Pipeline(**d)


@pytest.mark.parametrize("spec", PIPELINES, ids=lambda s: s.name)
@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("pinning", [EXPLICIT, VIRTUAL])
def test_result_and_accounting_do_not_depend_on_the_schedule(spec, policy, pinning):
    d, pipe = small(spec, 24)
    cfg = Config(policy, 1200, max_out=64, initial_bound=[8] * pipe.S, max_batch=16,
                 pinning=pinning)
    m = run_schedule(pipe, cfg)
    assert sorted(m.out) == surviving_outputs(d)
    assert m.stats["launches"] == created_tasks(d) + m.stats["retries"]
    assert all(u == 0 for u in m.used)
    assert m.pool.seqs == {}
    assert sum(m.budget) == cfg.num_blocks
    assert all(e.pins == 0 for e in m.pool.entries.values())
    if policy == SEQUENTIAL:
        assert m.stats["max_batch"] == 1
    if pinning == EXPLICIT and policy != BLOCKING:
        assert m.stats["misses"] == 0


def test_sequential_steps_are_the_sum_of_output_lengths():
    d, pipe = small(PIPELINES[2], 20)
    cfg = Config(SEQUENTIAL, 900, max_out=64, static_bound=[64] * pipe.S)
    m = run_schedule(pipe, cfg)
    assert m.stats["retries"] == 0
    launched = [(e[2], e[3]) for e in m.trace if e[1] == EV_LAUNCH]
    assert m.stats["steps"] == sum(d["out_len"][s][t] for s, t in launched)


def test_blocking_execution_misses_every_prefix_once_the_table_outgrows_the_cache():
    """Two stages, fan-out 1: a map over tuples of 10 blocks, then a second operator that
    reuses each tuple's prefix. The pool holds about 12 tuples."""
    def run(n, policy):
        d = dict(fanout=[1, 1], suffix=[[150] * n, [8] * n], out_len=[[2] * n, [1] * n],
                 filtered=[[0] * n, [0] * n])
        cfg = Config(policy, 130, max_out=8, static_bound=[2, 1], max_batch=4,
                     pinning=VIRTUAL)
        return run_schedule(Pipeline(**d), cfg)
    small_run = run(6, BLOCKING)
    assert small_run.stats["misses"] == 0 and small_run.stats["hits"] == 6
    big_run = run(60, BLOCKING)
    assert big_run.stats["hits"] == 0 and big_run.stats["misses"] == 60
    # the memory-aware schedule keeps every prefix until its child has run
    assert run(60, ADAPTIVE).stats["misses"] == 0


def test_retry_doubles_the_bound_until_the_request_fits():
    # one tuple generating 5 tokens against a static bound of 2 (max_out 8): launched with
    # bound 2, interrupted after 2 tokens -> bound 4, interrupted after 4 -> bound 8, completes
    d = dict(fanout=[1], suffix=[[30]], out_len=[[5]], filtered=[[0]])
    m = run_schedule(Pipeline(**d), Config(ADAPTIVE, 64, max_out=8, static_bound=[2]))
    retries = [e for e in m.trace if e[1] == EV_RETRY]
    assert [(e[0], e[4]) for e in retries] == [(1, 4), (5, 8)]
    assert m.stats["launches"] == 3
    # steps: 2 (bound 2) + 4 (bound 4) + 5 (completes) = 11
    assert m.stats["steps"] == 11
    assert [e[1] for e in m.trace if e[1] == EV_OUTPUT] == [EV_OUTPUT]


def test_token_bound_is_the_nearest_rank_99th_percentile():
    d = dict(fanout=[1], suffix=[[128, 128]], out_len=[[1, 1]], filtered=[[0, 0]])
    m = SchedulerModel(Pipeline(**d), Config(ADAPTIVE, 64, max_out=500, initial_bound=[7],
                                             min_obs=8))
    from oracle.scheduler import _Task
    t = _Task(0, 0, None)
    m.ratios[0] = [k / 64 for k in range(1, 8)]  # 7 observations: still the initial bound
    assert m._bound(t) == 7
    m.ratios[0] = [k / 64 for k in range(100, 0, -1)]  # 100 ratios k/64
    # rank ceil(0.99 * 100) = 99 -> ratio 99/64; times the input length 128 -> 198
    assert m._bound(t) == 198
    m.ratios[0] = [k / 64 for k in range(1, 11)]  # n = 10: rank ceil(9.9) = 10 -> 10/64
    assert m._bound(t) == 20
    m.ratios[0] = [1000.0] * 10  # clamped to max_out
    assert m._bound(t) == 500


def _two_stage_for_rebalance():
    # stage 0: 144-token tuples, 1-token answers (static bound 1); stage 1: 16 more tokens,
    # 1-token answers. max_out 16: minBudget_0 = ceil(160/16) = 10; the stage-1 prefix is
    # 144 + 1 - 1 = 144 tokens, minBudget_1 = ceil((144 + 16 + 16)/16) = 11.
    n = 30
    d = dict(fanout=[1, 1], suffix=[[144] * n, [16] * n], out_len=[[1] * n, [1] * n],
             filtered=[[0] * n, [0] * n])
    return Pipeline(**d), Config(ADAPTIVE, 101, max_out=16, static_bound=[1, 1], delta=10)


def test_first_rebalancing_transfers_worked_by_hand():
    pipe, cfg = _two_stage_for_rebalance()
    m = SchedulerModel(pipe, cfg)
    assert m.min_budget == [10, 11] and m.budget == [10, 91]
    m.run()
    tr = [e for e in m.trace if e[1] == EV_TRANSFER]
    # step 0: stage 0 runs one task (charge ceil(145/16) = 10 = its whole budget); it ends and
    # enqueues its child. Stage 1 has 1 waiting < 0.5 * 91 / 11 = 4.14: starving, and can
    # give 10 (91 unused, 81 >= 11 left) -> stage 0 gets 10: budgets [20, 81].
    assert tr[0] == (0, EV_TRANSFER, 1, 0, 10)
    # step 1: stage 0 admits one more task (10 cached + 10 <= 20); stage 1 admits the child
    # (charge ceil(161/16) - floor(144/16) = 2). After the step, stage 1 waits on 1 task
    # < 0.5 * 81 / 11 = 3.68: starving again -> [30, 71].
    assert tr[1] == (1, EV_TRANSFER, 1, 0, 10)
    assert m.stats["misses"] == 0


@pytest.mark.parametrize("spec", PIPELINES, ids=lambda s: s.name)
def test_rebalancing_moves_budget_only_where_the_rules_say(spec):
    d, pipe = small(spec, 30)
    cfg = Config(ADAPTIVE, 1500, max_out=64, initial_bound=[8] * pipe.S, max_batch=16,
                 delta=16)
    m = SchedulerModel(pipe, cfg)
    seen = []
    orig = m.rebalance_budgets

    def observed():
        before = len(m.trace)
        waiting = [len(w) for w in m.waiting]
        budget = list(m.budget)
        orig()
        seen.append((waiting, budget, m.trace[before:]))
        assert sum(m.budget) == cfg.num_blocks
        assert all(b >= mb for b, mb in zip(m.budget, m.min_budget))

    m.rebalance_budgets = observed
    m.run()
    last = m.S - 1
    moves = 0
    for waiting, budget, events in seen:
        budget = list(budget)  # replayed event by event: each rule sees the budgets so far
        for e in events:
            assert e[1] == EV_TRANSFER and e[4] == cfg.delta
            moves += 1
            a, b = e[2], e[3]
            if b == a - 1:  # starvation: the giving stage was starving
                assert waiting[a] < cfg.beta * budget[a] / m.min_budget[a]
            else:  # saturation: to the last stage, while some middle stage was saturated
                assert b == last and a != last
                assert any(waiting[x] > cfg.alpha * budget[x] / m.min_budget[x]
                           for x in range(1, last))
            budget[a] -= e[4]
            budget[b] += e[4]
    assert moves > 0


def test_breadth_first_budget_split():
    d, pipe = small(PIPELINES[0], 10)
    m = SchedulerModel(pipe, Config(BREADTH_FIRST, 2000, max_out=64, breadth_share=0.3))
    assert m.budget[0] == 600 and m.budget[1] == 1400
    with pytest.raises(ValueError):
        SchedulerModel(pipe, Config(DEPTH_FIRST, 50, max_out=64))


@pytest.mark.parametrize("spec", PIPELINES, ids=lambda s: s.name)
def test_blocking_runs_each_stage_to_completion_first(spec):
    d, pipe = small(spec, 20)
    m = run_schedule(pipe, Config(BLOCKING, 1500, max_out=64, initial_bound=[8] * pipe.S,
                                  max_batch=8))
    for s in range(1, pipe.S):
        prev = [e[0] for e in m.trace if e[2] == s - 1 and e[1] != EV_TRANSFER]
        launches = [e[0] for e in m.trace if e[2] == s and e[1] == EV_LAUNCH]
        if launches:
            assert min(launches) > max(prev)


def test_charges_worked_by_hand():
    # stage 0: 150-token tuples, 2-token outputs (static bound 2): charge ceil(152/16) = 10.
    # Its KV: 150 + 2 - 1 = 151 tokens. Stage 1 appends 8 with bound 1: the reused prefix
    # covers 9 whole blocks (151 // 16) and the charge is ceil(160/16) - 9 = 1 (the copied
    # partial block; the new tokens fit in it).
    n = 3
    d = dict(fanout=[1, 1], suffix=[[150] * n, [8] * n], out_len=[[2] * n, [1] * n],
             filtered=[[0] * n, [0] * n])
    m = run_schedule(Pipeline(**d), Config(ADAPTIVE, 200, max_out=8, static_bound=[2, 1]))
    launches = {(e[2], e[3]): e[4] for e in m.trace if e[1] == EV_LAUNCH}
    assert all(launches[(0, t)] == 2 * 10 + 1 for t in range(n))
    assert all(launches[(1, t)] == 2 * 1 + 1 for t in range(n))
    assert m.stats["cow_copies"] == n


@pytest.mark.parametrize("pinning", [EXPLICIT, VIRTUAL])
def test_prefixes_are_pinned_exactly_while_children_need_them(pinning):
    from oracle.scheduler import task_key
    d, pipe = small(PIPELINES[1], 12)
    m = SchedulerModel(pipe, Config(ADAPTIVE, 2500, max_out=64, initial_bound=[8] * pipe.S,
                                    max_batch=16, pinning=pinning))
    tasks = {}
    orig = m.finish

    def complete(t, interrupted):
        tasks[(t.stage, t.idx)] = t
        orig(t, interrupted)
        for (s, i), u in tasks.items():
            e = m.pool.entries.get(task_key(s, i))
            if u.children_left > 0:  # completed, children still unreleased
                assert e is not None and e.pins == (1 if pinning == EXPLICIT else 0)
            elif e is not None:
                assert e.pins == 0

    m.finish = complete
    m.run()
    assert tasks


def test_chunked_prefill_worked_by_hand():
    # task A: 10-token prompt, 3 output tokens; task B: 50-token prompt, 1 output token;
    # budget 16 tokens per step, decodes first:
    #   step 0: A prefills 10 (token 1), B 6      step 1: A decodes (token 2), B 15 (21)
    #   step 2: A decodes (token 3: done), B 15 (36)   step 3: B 14 (50: token 1, done)
    d = dict(fanout=[1], suffix=[[10, 50]], out_len=[[3, 1]], filtered=[[0, 0]])
    m = run_schedule(Pipeline(**d), Config(ADAPTIVE, 64, max_out=8, static_bound=[8],
                                           max_step_tokens=16))
    outs = {e[3]: e[0] for e in m.trace if e[1] == EV_OUTPUT}
    assert outs == {0: 2, 1: 3}
    assert m.stats["prefill_chunks"] == 1 + 4 and m.stats["steps"] == 4
    assert m.stats["prefill_tokens"] == 60 and m.stats["decode_tokens"] == 2


@pytest.mark.parametrize("budget", [1, 7, 64, 512])
def test_chunked_prefill_keeps_the_result_and_the_budget(budget):
    d, pipe = small(PIPELINES[2], 20)
    kw = dict(max_out=64, static_bound=[64] * pipe.S, max_batch=16)
    ref = run_schedule(pipe, Config(ADAPTIVE, 1500, **kw))
    m = SchedulerModel(pipe, Config(ADAPTIVE, 1500, max_step_tokens=budget, **kw))
    per_step = []
    commit = m.pool.commit
    step_fn = m.engine_step

    def counted_commit(sid, n):
        per_step[-1] += n
        return commit(sid, n)

    def counted_step():
        per_step.append(0)
        return step_fn()

    m.pool.commit = counted_commit
    m.engine_step = counted_step
    m.run()
    assert max(per_step) <= budget
    assert sorted(m.out) == sorted(ref.out) == surviving_outputs(d)
    assert m.stats["prefill_tokens"] == ref.stats["prefill_tokens"]
    assert m.stats["decode_tokens"] == ref.stats["decode_tokens"]
    assert m.stats["misses"] == 0 and m.stats["retries"] == 0
    assert m.stats["prefill_chunks"] >= ref.stats["prefill_chunks"]
    assert all(u == 0 for u in m.used)
