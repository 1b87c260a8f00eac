"""GPU tier for the pipeline scheduler's device mode: every engine step's attention work
(copy-on-write block copies, KV append, prefill and decode attention) runs through the
library's kernels. The schedule must be exactly the one the scheduling-only run (checked
against the oracle's model on the CPU) produces, the run must finish without a HIP error, and
its GPU time must be measured."""
import numpy as np
import pytest

from tests.gpu_util import say
from workloads.pipelines import PIPELINES, make_pipeline

pytestmark = pytest.mark.gpu


def _device(torch, num_blocks, hq=32, hkv=8, d=128, src_rows=8192, seed=0):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)

    def rnd(*shape):
        return torch.randn(*shape, generator=g, device="cuda", dtype=torch.float32).to(
            torch.bfloat16)
    return dict(k_cache=rnd(num_blocks, hkv, d // 8, 16, 8), v_cache=rnd(num_blocks, hkv, d, 16),
                q_src=rnd(src_rows, hq, d), k_src=rnd(src_rows, hkv, d),
                v_src=rnd(src_rows, hkv, d))


@pytest.mark.parametrize("spec", PIPELINES, ids=lambda s: s.name)
@pytest.mark.parametrize("policy,budget", [(0, 0), (4, 0), (0, 200)])
def test_device_mode_runs_the_same_schedule(gpu_lib, spec, policy, budget):
    """budget > 0: chunked prefill (prompt pieces attend over the cache and earlier pieces)."""
    import torch
    lib = gpu_lib
    say(f"[sched device] {spec.name} policy {policy} step budget {budget}")
    d = make_pipeline(spec.scaled(24))
    nb = 1500
    kw = dict(max_out=64, initial_bound=[8] * len(d["suffix"]), max_batch=16, pinning=1,
              max_step_tokens=budget)
    cfg = lib.sched_config(policy, nb, **kw)
    args = (d["fanout"], d["suffix"], d["out_len"], d["filtered"])
    st0, tr0, b0 = lib.pkv_sched_run(cfg, *args, max_events=200000)
    dev = _device(torch, nb)
    st1, tr1, b1 = lib.pkv_sched_run(cfg, *args, device=dev, max_events=200000)
    torch.cuda.synchronize()
    assert np.array_equal(tr0, tr1) and np.array_equal(b0, b1)
    for k in ("steps", "launches", "hits", "misses", "prefill_tokens", "cow_copies"):
        assert st0[k] == st1[k]
    assert st0["gpu_ms"] == 0.0 and st1["gpu_ms"] > 0.0
    say(f"  steps {st1['steps']} gpu {st1['gpu_ms']:.2f} ms wall {st1['wall_ms']:.1f} ms "
        f"hits {st1['hits']} misses {st1['misses']}")
    assert torch.isfinite(dev["k_cache"].float()).all()


def test_device_mode_refuses_short_sources(gpu_lib):
    import torch
    lib = gpu_lib
    d = make_pipeline(PIPELINES[1].scaled(4))  # contract-sized prompts (> 512 tokens)
    cfg = lib.sched_config(0, 1500, max_out=64, max_batch=16)
    dev = _device(torch, 1500, src_rows=512)
    with pytest.raises(lib.PkvError) as e:
        lib.pkv_sched_run(cfg, d["fanout"], d["suffix"], d["out_len"], d["filtered"],
                          device=dev)
    assert e.value.status == lib.PKV_ERR_INVALID_ARG
    torch.cuda.synchronize()
