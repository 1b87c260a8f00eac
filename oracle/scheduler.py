"""Plain model of the pipelined semantic-operator scheduler (oracle; test infrastructure only).

What it follows:
  * Section 5.1 (executing query plans): a pipeline of stages; a task runs one stage's operator on one
    tuple; a surviving task of a non-final stage is joined (Cartesian product) with the next
    stage's right-side table, creating dependent child tasks that reuse the task's cached
    prefix; a final-stage task's result is output; a filtered task ends its branch.
  * Algorithm 1 (Section 5.3), the adaptive memory-aware scheduler. Every iteration admits
    waiting tasks stage by stage, in queue order, while the memory manager finds room for the
    queue head in its stage's budget; then handles the tasks that finished (a retry raises the
    bound and queues the task again; a survivor of a non-final stage produces its children and
    keeps its memory until they are all done; results and filtered tasks release theirs); then
    adapts the budgets: a saturated stage other than the first and the last gives Delta to the
    last stage (from its own unused budget, or else from the first stage with Delta unused),
    and, from the last stage down to the second, a starving stage gives Delta to the one
    before it. A stage is saturated when more than alpha * budget_s / minBudget_s tasks wait,
    starving when fewer than beta * budget_s / minBudget_s do. Initial budgets: minBudget_s
    for every stage but the last, which takes the rest.
  * Section 6: each task carries a token bound (static per stage, or the 99th percentile of
    the output-to-input ratio of completed requests times the task's input length); a request
    that reaches its bound is interrupted, the bound is raised and the task re-enqueued.
    Explicit pinning pins a cached prefix until its children no longer need it; virtual pinning
    relies on the pool's eviction order.
  * Section 5.3's baselines: sequential depth-first (one task at a time, deepest stage first),
    parallel depth-first (the initial budgets, never rebalanced), parallel breadth-first (a
    static large first-stage budget), and blocking execution, the operator-at-a-time
    materialisation of Section 2.2 that Section 7.4 ablates (each stage runs to completion
    before the next starts; prefixes are left to the LRU cache).

Readings where the paper is silent (the library implements the same ones):
  * Memory is counted in 16-token KV blocks of the pool. A task's charge is the blocks it adds:
    ceil((P + suffix + bound) / 16) - floor(P / 16) when it reuses its parent's P cached tokens
    (the last, partly filled prefix block is copied on write), ceil((P + suffix + bound) / 16)
    when it recomputes them (a cache miss). Blocking execution charges every task its whole
    sequence, since no parent keeps a charge. minBudget_s is the largest miss charge of any
    stage-s task at the largest bound (max_out): one task with its prefix always fits.
  * A task's charge stays on its stage after it completes (its prefix is cached for its
    children) and is released when it is filtered, is a final-stage task, or when all of its
    children have been released; the release cascades up (Algorithm 1).
  * The engine is step-synchronous: each step, the first max_batch admitted tasks advance; a
    task's first step prefills its prompt (suffix, or prefix + suffix on a miss) and yields one
    output token; each later step appends the previous token's KV and yields one more. A task
    with out_len output tokens takes out_len steps and leaves P + suffix + out_len - 1 tokens of
    KV, the prefix its children reuse. With a per-step token budget (chunked prefill), the
    decoding tasks of the batch go first, one token each, in queue order, and the rest of the
    budget goes to prompt chunks, in queue order; a prompt yields its first token with its last
    chunk (a chunk attends over the cached prefix and the earlier chunks).
  * The bound is fixed when the task is admitted; before min_obs observations an estimated stage
    uses its initial bound; the 99th percentile is the nearest-rank one (rank ceil(0.99 n));
    the ratio and its product with the input length are computed in double precision and
    rounded up. A retried task's bound doubles (at most max_out) and is kept.
  * Completed prefixes are published under the key (stage << 40) | task and, under explicit
    pinning, pinned; released prefixes are unpinned and stay cached until evicted.
"""
from collections import deque

from .block_pool import EXPLICIT, LRU, BlockPoolModel, Status

ADAPTIVE, DEPTH_FIRST, BREADTH_FIRST, SEQUENTIAL, BLOCKING = 0, 1, 2, 3, 4

# trace events: (step, kind, stage, task, value)
EV_LAUNCH = 1     # value = 2 * charge + (1 if the prefix is reused else 0)
EV_DONE = 2       # completed and passed on; value = output tokens
EV_FILTERED = 3   # completed, dropped by its predicate
EV_OUTPUT = 4     # final-stage result
EV_RETRY = 5      # interrupted at its bound; value = the new bound
EV_RELEASE = 6    # charge released; value = blocks
EV_TRANSFER = 7   # budget moved: stage = from, task = to, value = blocks

BS = 16


def _cdiv(a, b):
    return -(-a // b)


def task_key(stage, idx):
    return (stage << 40) | idx


class Pipeline:
    """Per stage s: fanout[s] right-side rows joined with each surviving stage-s task (s < S-1);
    and per task t of stage s (t in 0..count_s-1, count_0 = number of input tuples,
    count_{s+1} = count_s * fanout[s], parent of (s+1, t) = (s, t // fanout[s])):
    suffix[s][t] tokens appended to the parent's prefix, out_len[s][t] >= 1 tokens generated,
    filtered[s][t] whether the predicate drops the tuple."""

    def __init__(self, fanout, suffix, out_len, filtered):
        self.S = len(suffix)
        self.fanout = [int(f) for f in fanout]
        self.suffix = [[int(x) for x in a] for a in suffix]
        self.out_len = [[int(x) for x in a] for a in out_len]
        self.filtered = [[int(x) for x in a] for a in filtered]
        for s in range(self.S - 1):
            if len(self.suffix[s + 1]) != len(self.suffix[s]) * self.fanout[s]:
                raise ValueError("stage sizes must follow the fanouts")
        # KV tokens cached in front of each task (its parent's final length)
        self.prefix = [[0] * len(self.suffix[0])]
        for s in range(1, self.S):
            f = self.fanout[s - 1]
            self.prefix.append([self.kv_len(s - 1, t // f) for t in range(len(self.suffix[s]))])

    def kv_len(self, s, t):
        return self.prefix[s][t] + self.suffix[s][t] + self.out_len[s][t] - 1


class Config:
    def __init__(self, policy, num_blocks, max_out, alpha=1.0, beta=0.5, delta=0,
                 pinning=EXPLICIT, eviction=LRU, breadth_share=0.5, static_bound=None,
                 initial_bound=None, min_obs=8, max_batch=256, max_steps=1_000_000,
                 max_step_tokens=0):
        self.policy = policy
        self.num_blocks = num_blocks
        self.max_out = max_out
        self.alpha, self.beta, self.delta = float(alpha), float(beta), int(delta)
        self.pinning, self.eviction = pinning, eviction
        self.breadth_share = float(breadth_share)
        self.static_bound = static_bound
        self.initial_bound = initial_bound
        self.min_obs, self.max_batch, self.max_steps = min_obs, max_batch, max_steps
        self.max_step_tokens = max_step_tokens  # 0: no budget (whole prompts)


class _Task:
    def __init__(self, stage, idx, parent):
        self.stage, self.idx, self.parent = stage, idx, parent
        self.bound = 0
        self.fixed_bound = False
        self.charge = 0
        self.hit = True
        self.seq = 0
        self.cached = 0      # prefix tokens reused from the cache
        self.prompt = 0      # prompt tokens to prefill
        self.prefilled = 0   # of which done
        self.generated = 0
        self.children_left = 0


class SchedulerModel:
    def __init__(self, pipe: Pipeline, cfg: Config):
        self.p, self.c = pipe, cfg
        S = pipe.S
        self.S = S
        self.pool = BlockPoolModel(cfg.num_blocks, BS)
        self.pool.set_eviction(cfg.eviction)
        self.pool.set_pinning(cfg.pinning)
        self.min_budget = [max(_cdiv(pipe.prefix[s][t] + pipe.suffix[s][t] + cfg.max_out, BS)
                               for t in range(len(pipe.suffix[s]))) for s in range(S)]
        self.delta = cfg.delta if cfg.delta > 0 else max(self.min_budget)
        self.budget = self._initial_budgets()
        self.used = [0] * S
        self.waiting = [deque() for _ in range(S)]
        self.running = []          # admitted tasks, in admission order (the engine's queue)
        self.ratios = [[] for _ in range(S)]
        self.trace, self.out = [], []
        self.step = 0
        self.stats = dict(steps=0, launches=0, retries=0, hits=0, misses=0, prefill_tokens=0,
                          reused_tokens=0, decode_tokens=0, cow_copies=0, max_batch=0,
                          prefill_chunks=0)

    # -- memory manager ---------------------------------------------------------------------
    def _initial_budgets(self):
        S, total, mb = self.S, self.c.num_blocks, self.min_budget
        if self.c.policy in (SEQUENTIAL, BLOCKING):
            return [total] + [0] * (S - 1)  # one budget for the whole pool (held by stage 0)
        b = list(mb)
        if self.c.policy == BREADTH_FIRST and S > 1:
            b[0] = max(mb[0], int(self.c.breadth_share * total))
        b[S - 1] = total - sum(b[:S - 1])
        if b[S - 1] < mb[S - 1]:
            raise ValueError("the pool is smaller than the stages' minimum budgets")
        return b

    def _bound(self, t):
        if t.fixed_bound:
            return t.bound
        s, c = t.stage, self.c
        static = c.static_bound[s] if c.static_bound else 0
        if static > 0:
            return min(static, c.max_out)
        r = self.ratios[s]
        if len(r) >= c.min_obs:
            srt = sorted(r)
            k = (99 * len(srt) + 99) // 100 - 1
            prompt = self.p.prefix[s][t.idx] + self.p.suffix[s][t.idx]
            b = int(-(-(srt[k] * prompt) // 1))  # ceil in double precision
            return max(1, min(b, c.max_out))
        init = c.initial_bound[s] if c.initial_bound and c.initial_bound[s] > 0 else c.max_out
        return max(1, min(init, c.max_out))

    def _size(self, t):
        """(charge, hit, bound) of admitting t now."""
        s, i = t.stage, t.idx
        P, suf = self.p.prefix[s][i], self.p.suffix[s][i]
        bound = self._bound(t)
        hit = s == 0 or self.pool.lookup(task_key(s - 1, i // self.p.fanout[s - 1])) > 0
        whole = _cdiv(P + suf + bound, BS)
        if self.c.policy == BLOCKING or not hit:
            return whole, hit, bound
        return whole - P // BS, hit, bound

    def fits_budget(self, stage, t):
        charge, _, _ = self._size(t)
        if self.c.policy == BLOCKING or self.c.policy == SEQUENTIAL:
            return sum(self.used) + charge <= self.c.num_blocks
        return self.used[stage] + charge <= self.budget[stage]

    def reserve_for(self, stage, t):
        charge, hit, bound = self._size(t)
        s, i, pool = t.stage, t.idx, self.pool
        P, suf = self.p.prefix[s][i], self.p.suffix[s][i]
        t.bound, t.charge, t.hit = bound, charge, hit
        if s == 0:
            _, t.seq = pool.create()
            assert pool.reserve(t.seq, suf + bound) == Status.OK
            t.cached, t.prompt = 0, suf
        elif hit:
            st, t.seq, tok = pool.attach(task_key(s - 1, i // self.p.fanout[s - 1]))
            assert st == Status.OK and tok == P
            st, copies = pool.reserve(t.seq, suf + bound, cow=True)
            assert st == Status.OK
            self.stats["cow_copies"] += len(copies)
            t.cached, t.prompt = P, suf
            self.stats["hits"] += 1
        else:
            _, t.seq = pool.create()
            assert pool.reserve(t.seq, P + suf + bound) == Status.OK
            t.cached, t.prompt = 0, P + suf
            self.stats["misses"] += 1
        self.used[self._charged_stage(t)] += charge
        t.generated = t.prefilled = 0
        self.stats["launches"] += 1
        self.trace.append((self.step, EV_LAUNCH, s, i, 2 * charge + (1 if hit else 0)))

    def return_charge(self, t):
        self.used[self._charged_stage(t)] -= t.charge
        self.trace.append((self.step, EV_RELEASE, t.stage, t.idx, t.charge))
        par = t.parent
        if par is not None and self.c.policy not in (BLOCKING,):
            par.children_left -= 1
            if par.children_left == 0:
                key = task_key(par.stage, par.idx)
                if self.c.pinning == EXPLICIT:
                    self.pool.unpin(key)  # the prefix stays cached, now evictable
                self.return_charge(par)

    def _charged_stage(self, t):
        return 0 if self.c.policy in (SEQUENTIAL, BLOCKING) else t.stage

    def saturated(self, s):
        return len(self.waiting[s]) > self.c.alpha * self.budget[s] / self.min_budget[s]

    def starving(self, s):
        return len(self.waiting[s]) < self.c.beta * self.budget[s] / self.min_budget[s]

    def _can_give(self, u):
        d = self.delta
        return self.budget[u] - self.used[u] >= d and self.budget[u] - d >= self.min_budget[u]

    def _move(self, a, b):
        self.budget[a] -= self.delta
        self.budget[b] += self.delta
        self.trace.append((self.step, EV_TRANSFER, a, b, self.delta))

    def relieve_saturation(self, s):
        last = self.S - 1
        if self._can_give(s):
            self._move(s, last)
            return
        for u in range(self.S - 1):
            if self._can_give(u):
                self._move(u, last)
                return

    def feed_previous(self, i):
        if self._can_give(i):
            self._move(i, i - 1)

    # -- the scheduling loop (Algorithm 1) ----------------------------------------------------
    def admit_waiting(self):
        pol = self.c.policy
        if pol == SEQUENTIAL:
            if self.running:
                return
            for s in reversed(range(self.S)):  # depth first: the deepest ready stage
                if self.waiting[s]:
                    t = self.waiting[s][0]
                    if self.fits_budget(s, t):
                        self.waiting[s].popleft()
                        self.reserve_for(s, t)
                        self.running.append(t)
                    return
            return
        stages = range(self.S)
        if pol == BLOCKING:  # one stage at a time: the first with unfinished work
            active = next(s for s in range(self.S)
                          if self.waiting[s] or any(t.stage == s for t in self.running))
            stages = [active]
        for s in stages:
            while self.waiting[s]:
                t = self.waiting[s][0]
                if self.fits_budget(s, t):
                    self.waiting[s].popleft()
                    self.reserve_for(s, t)
                    self.running.append(t)
                else:
                    break

    def engine_step(self):
        """Advance the first max_batch admitted tasks by one step; return the finished ones
        as (task, kind) in queue order, kind 0 = completed, 1 = interrupted at its bound."""
        batch = self.running[: self.c.max_batch]
        self.stats["max_batch"] = max(self.stats["max_batch"], len(batch))
        if self.c.max_step_tokens <= 0:
            take = {id(t): (t.prompt - t.prefilled if t.generated == 0 else 1) for t in batch}
        else:  # chunked prefill: decodes first, then prompt chunks, in queue order
            left = self.c.max_step_tokens
            take = {}
            for t in batch:
                if t.generated > 0 and left > 0:
                    take[id(t)] = 1
                    left -= 1
            for t in batch:
                if t.generated == 0:
                    rest = t.prompt - t.prefilled
                    if rest == 0 or left > 0:
                        take[id(t)] = min(rest, left)
                        left -= take[id(t)]
        done = []
        for t in batch:
            if id(t) not in take:
                continue
            n = take[id(t)]
            s, i = t.stage, t.idx
            if t.generated == 0:
                self.pool.commit(t.seq, n)
                self.stats["prefill_tokens"] += n
                if t.prefilled == 0:
                    self.stats["reused_tokens"] += t.cached
                self.stats["prefill_chunks"] += 1
                t.prefilled += n
                if t.prefilled < t.prompt:
                    continue
            else:
                self.pool.commit(t.seq, 1)
                self.stats["decode_tokens"] += 1
            t.generated += 1
            if t.generated == self.p.out_len[s][i]:
                done.append((t, 0))
            elif t.generated == t.bound:
                done.append((t, 1))
        return done

    def finish(self, t, interrupted):
        s, i, pool = t.stage, t.idx, self.pool
        self.running.remove(t)
        if interrupted:  # Section 6: raise the bound, re-enqueue
            pool.free_seq(t.seq)
            self.used[self._charged_stage(t)] -= t.charge
            t.bound = min(2 * t.bound, self.c.max_out)
            t.fixed_bound = True
            self.stats["retries"] += 1
            self.trace.append((self.step, EV_RETRY, s, i, t.bound))
            self.waiting[s].append(t)
            return
        prompt = self.p.prefix[s][i] + self.p.suffix[s][i]
        self.ratios[s].append(self.p.out_len[s][i] / prompt)
        filtered = self.p.filtered[s][i] != 0
        last = s == self.S - 1
        if not filtered:
            if not last:
                f = self.p.fanout[s]
                kids = [_Task(s + 1, i * f + r, t) for r in range(f)]
                self.waiting[s + 1].extend(kids)
                t.children_left = f  # its memory stays until these are done
                key = task_key(s, i)
                assert pool.publish(t.seq, key, self.p.kv_len(s, i)) == Status.OK
                if self.c.pinning == EXPLICIT and self.c.policy != BLOCKING:
                    pool.pin(key)
                pool.free_seq(t.seq)
                self.trace.append((self.step, EV_DONE, s, i, self.p.out_len[s][i]))
                if self.c.policy == BLOCKING:  # nothing tracks the children
                    self.used[0] -= t.charge
                    self.trace.append((self.step, EV_RELEASE, s, i, t.charge))
            else:
                self.out.append((s, i))
                self.trace.append((self.step, EV_OUTPUT, s, i, self.p.out_len[s][i]))
        else:
            self.trace.append((self.step, EV_FILTERED, s, i, self.p.out_len[s][i]))
        if filtered or last:
            pool.free_seq(t.seq)
            self.return_charge(t)

    def rebalance_budgets(self):
        for s in range(self.S):
            if s != 0 and s != self.S - 1 and self.saturated(s):
                self.relieve_saturation(s)
        for i in range(self.S - 1, 0, -1):
            if self.starving(i):
                self.feed_previous(i)

    def run(self):
        self.waiting[0].extend(_Task(0, t, None) for t in range(len(self.p.suffix[0])))
        while any(self.waiting) or self.running:
            if self.step >= self.c.max_steps:
                raise RuntimeError("step limit reached")
            self.admit_waiting()
            if not self.running:
                raise RuntimeError("no task can be admitted and none is running")
            done = self.engine_step()
            for t, kind in done:
                self.finish(t, kind == 1)
            if self.c.policy == ADAPTIVE:
                self.rebalance_budgets()
            self.step += 1
        self.stats["steps"] = self.step
        self.stats["evictions"] = self.pool.evictions
        return self


def run_schedule(pipe, cfg):
    return SchedulerModel(pipe, cfg).run()
