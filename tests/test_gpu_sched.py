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


def _hip_d2h(ptr, nbytes):
    """Copy nbytes of device memory at a raw address (the group's output buffer) to the host."""
    import ctypes
    hip = None
    for name in ("libamdhip64.so", "libamdhip64.so.7", "libamdhip64.so.6"):
        try:
            hip = ctypes.CDLL(name)
            break
        except OSError:
            continue
    assert hip is not None, "libamdhip64 not found"
    buf = np.empty(nbytes, dtype=np.uint8)
    rc = hip.hipMemcpy(ctypes.c_void_p(buf.ctypes.data), ctypes.c_void_p(ptr),
                       ctypes.c_size_t(nbytes), ctypes.c_int(2))  # hipMemcpyDeviceToHost
    assert rc == 0, f"hipMemcpy failed ({rc})"
    return buf


@pytest.mark.parametrize("pidx,policy,budget", [(0, 0, 0), (1, 0, 0), (2, 4, 0), (0, 0, 200)])
def test_device_mode_results_match_the_oracle(gpu_lib, pidx, policy, budget):
    """The scheduler's device mode checked against the oracle: for a spread of the groups it
    launches (prefill groups, chunked prefill pieces, decode groups), the pool blocks the
    group touches are read before its append and after its attention; the append must be
    byte-exact (oracle.kv_append over the k_src / v_src rows the group names) and the
    attention output must match oracle.prefill_attention / decode_attention over the pool as
    it was before the append, within the attention bar."""
    import oracle
    import torch
    from tests.gpu_util import bf16_to_f64, compare, to_host_bits
    lib = gpu_lib
    spec = PIPELINES[pidx]
    say(f"[sched device vs oracle] {spec.name} policy {policy} step budget {budget}")
    d = make_pipeline(spec.scaled(24))
    nb, hq, hkv, dim = 1500, 32, 8, 128
    cfg = lib.sched_config(policy, nb, max_out=64, initial_bound=[8] * len(d["suffix"]),
                           max_batch=16, pinning=0, max_step_tokens=budget)
    dev = _device(torch, nb, hq, hkv, dim, seed=11)
    q_h, k_h, v_h = (to_host_bits(dev[n]) for n in ("q_src", "k_src", "v_src"))
    scale = 1.0 / np.sqrt(dim)
    seen = {False: 0, True: 0}
    checked = {False: 0, True: 0}
    state = {}
    failures = []

    def blocks(ids):
        idx = torch.as_tensor(ids, dtype=torch.int64, device="cuda")
        return (to_host_bits(dev["k_cache"].index_select(0, idx)),
                to_host_bits(dev["v_cache"].index_select(0, idx)))

    def hook(g):
        dec = g["decode"]
        if g["phase"] == 0:
            state.pop(dec, None)
            k = seen[dec]
            seen[dec] += 1
            cached, cu = g["cached"], g["cu_new"]
            n_new = np.diff(cu)
            cost = int(np.sum(n_new * (cached + n_new))) * hq
            if checked[dec] >= 3 or k % 4 != 0 or cost > 100_000_000:
                return
            used = [g["tables"][s, :-(-(int(cached[s]) + int(n_new[s])) // 16)]
                    for s in range(len(cached))]
            ids = np.unique(np.concatenate(used))
            state[dec] = (g, ids, blocks(ids))
            return
        if dec not in state:
            return
        g0, ids, (bk, bv) = state.pop(dec)
        try:
            cached, cu = g0["cached"], g0["cu_new"]
            n = len(cached)
            local = {int(b): j for j, b in enumerate(ids)}
            tab = np.full(g0["tables"].shape, -1, np.int32)
            for s in range(n):
                nblk = -(-(int(cached[s]) + int(cu[s + 1] - cu[s])) // 16)
                tab[s, :nblk] = [local[int(b)] for b in g0["tables"][s, :nblk]]
            rows = slice(int(cu[0]), int(cu[-1]))
            ek, ev = oracle.kv_append(bk, bv, tab, cached, cu - cu[0], k_h[rows], v_h[rows], 16)
            ak, av = blocks(ids)
            assert np.array_equal(ak, ek) and np.array_equal(av, ev), "append not byte-exact"
            nrow = n if dec else int(cu[-1])
            got = _hip_d2h(g["out_ptr"], nrow * hq * dim * 2).view(np.uint16).reshape(nrow, hq, dim)
            if dec:
                o, _ = oracle.decode_attention(bk, bv, tab, cached, q_h[:n], k_h[rows], v_h[rows],
                                               scale, 16)
            else:
                o, _ = oracle.prefill_attention(bk, bv, tab, cached, cu - cu[0], q_h[rows],
                                                k_h[rows], v_h[rows], scale, 16)
            compare(f"step {g0['step']} {'decode' if dec else 'prefill'} group of {n}",
                    bf16_to_f64(got), o)
            checked[dec] += 1
        except Exception as e:  # a hook cannot raise through the C call: collect
            failures.append(f"step {g0['step']}: {e}")

    args = (d["fanout"], d["suffix"], d["out_len"], d["filtered"])
    st, _, _ = lib.pkv_sched_run(cfg, *args, device=dev, group_hook=hook)
    torch.cuda.synchronize()
    say(f"  groups seen: prefill {seen[False]}, decode {seen[True]}; checked: prefill "
        f"{checked[False]}, decode {checked[True]}; gpu {st['gpu_ms']:.2f} ms")
    assert not failures, failures
    assert checked[False] >= 1 and checked[True] >= 1
