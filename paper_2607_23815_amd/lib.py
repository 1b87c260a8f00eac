"""Thin ctypes binding of libpkv.so (include/pkv.h), with the C names.

Argument marshalling only: tensors supply device pointers and torch's current stream supplies
the hipStream_t; every step of the path runs in the library's HIP kernels. There is no CPU
fallback: importing this module fails if libpkv.so is missing, and the device calls refuse
tensors that are not on the GPU. PKV_LIBRARY, if set, names another build of the library
to load instead of the in-tree one."""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_LIB_PATH = os.environ.get("PKV_LIBRARY") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libpkv.so")

if not os.path.exists(_LIB_PATH):
    raise ImportError(f"{_LIB_PATH} is missing: build it with "
                      "`python -m paper_2607_23815_amd.build` (needs hipcc)")
_lib = ctypes.CDLL(_LIB_PATH)

c_int32, c_int64, c_size_t, c_float, c_void_p = (ctypes.c_int32, ctypes.c_int64,
                                                  ctypes.c_size_t, ctypes.c_float,
                                                  ctypes.c_void_p)
P_int32 = ctypes.POINTER(c_int32)
P_int64 = ctypes.POINTER(c_int64)

PKV_OK = 0
PKV_ERR_INVALID_ARG = 1
PKV_ERR_OUT_OF_BLOCKS = 2
PKV_ERR_SHARED_BLOCK_WRITE = 3
PKV_ERR_UNSUPPORTED_SHAPE = 4
PKV_ERR_NOT_FOUND = 5
PKV_ERR_HIP = 6
PKV_ERR_KEY_EXISTS = 7
PKV_ERR_BAD_METADATA = 8
PKV_EVICT_LRU, PKV_EVICT_MRU = 0, 1
PKV_PIN_EXPLICIT, PKV_PIN_VIRTUAL = 0, 1


class PagedKV(ctypes.Structure):
    _fields_ = [("k_cache", c_void_p), ("v_cache", c_void_p), ("num_blocks", c_int32),
                ("block_size", c_int32), ("num_kv_heads", c_int32), ("head_dim", c_int32)]


class PoolStats(ctypes.Structure):
    _fields_ = [("num_free", c_int32), ("num_entries", c_int32), ("cached_blocks", c_int32),
                ("pinned_entries", c_int32), ("eviction", c_int32), ("pinning", c_int32),
                ("hits", c_int64), ("misses", c_int64), ("evictions", c_int64),
                ("cow_copies", c_int64)]


c_uint64 = ctypes.c_uint64
c_double = ctypes.c_double

PKV_MAX_STAGES = 8
(PKV_SCHED_ADAPTIVE, PKV_SCHED_DEPTH_FIRST, PKV_SCHED_BREADTH_FIRST, PKV_SCHED_SEQUENTIAL,
 PKV_SCHED_BLOCKING) = range(5)


class SchedConfig(ctypes.Structure):
    _fields_ = [("policy", c_int32), ("num_blocks", c_int32), ("max_out", c_int32),
                ("delta", c_int32), ("alpha", c_double), ("beta", c_double),
                ("breadth_share", c_double), ("pinning", c_int32), ("eviction", c_int32),
                ("min_obs", c_int32), ("max_batch", c_int32), ("max_steps", c_int64),
                ("max_step_tokens", c_int32),
                ("static_bound", c_int32 * PKV_MAX_STAGES),
                ("initial_bound", c_int32 * PKV_MAX_STAGES)]


class SchedStats(ctypes.Structure):
    _fields_ = [("steps", c_int64), ("launches", c_int64), ("retries", c_int64),
                ("hits", c_int64), ("misses", c_int64), ("prefill_tokens", c_int64),
                ("reused_tokens", c_int64), ("decode_tokens", c_int64),
                ("cow_copies", c_int64), ("evictions", c_int64), ("outputs", c_int64),
                ("prefill_chunks", c_int64), ("max_batch", c_int32), ("gpu_ms", c_double), ("wall_ms", c_double)]

class SchedGroup(ctypes.Structure):
    _fields_ = [("step", c_int64), ("phase", c_int32), ("decode", c_int32),
                ("num_seqs", c_int32), ("max_blocks", c_int32), ("tables", P_int32),
                ("cached", P_int32), ("cu_new", P_int32), ("out", c_void_p)]


SCHED_GROUP_HOOK = ctypes.CFUNCTYPE(None, c_void_p, ctypes.POINTER(SchedGroup))


class SchedDevice(ctypes.Structure):
    _fields_ = [("kv", PagedKV), ("num_q_heads", c_int32), ("q_src", c_void_p),
                ("k_src", c_void_p), ("v_src", c_void_p), ("src_rows", c_int32),
                ("stream", c_void_p), ("group_hook", SCHED_GROUP_HOOK),
                ("hook_user", c_void_p)]


_SIGS = {
    "pkv_last_error": (ctypes.c_char_p, []),
    "pkv_abi_version": (c_int32, []),
    "pkv_set_debug_validate": (c_int32, [c_int32]),
    "pkv_get_debug_validate": (c_int32, []),
    "pkv_pool_create": (c_int32, [c_int32, c_int32, P_int32, ctypes.POINTER(c_void_p)]),
    "pkv_pool_destroy": (None, [c_void_p]),
    "pkv_pool_num_free": (c_int32, [c_void_p]),
    "pkv_seq_create": (c_int32, [c_void_p, P_int64]),
    "pkv_seq_fork": (c_int32, [c_void_p, c_int64, c_int32, P_int64]),
    "pkv_seq_reserve": (c_int32, [c_void_p, c_int64, c_int32]),
    "pkv_seq_commit": (c_int32, [c_void_p, c_int64, c_int32]),
    "pkv_seq_free": (c_int32, [c_void_p, c_int64]),
    "pkv_seq_len": (c_int32, [c_void_p, c_int64, P_int32]),
    "pkv_fill_block_tables": (c_int32, [c_void_p, P_int64, c_int32, c_int32, P_int32, P_int32]),
    "pkv_pool_set_eviction": (c_int32, [c_void_p, c_int32]),
    "pkv_pool_set_pinning": (c_int32, [c_void_p, c_int32]),
    "pkv_pool_check_deadlock": (c_int32, [c_void_p, c_int32, c_int32, P_int32]),
    "pkv_prefix_publish": (c_int32, [c_void_p, c_int64, c_uint64, c_int32]),
    "pkv_prefix_attach": (c_int32, [c_void_p, c_uint64, P_int64, P_int32]),
    "pkv_prefix_lookup": (c_int32, [c_void_p, c_uint64, P_int32]),
    "pkv_prefix_pin": (c_int32, [c_void_p, c_uint64]),
    "pkv_prefix_unpin": (c_int32, [c_void_p, c_uint64]),
    "pkv_prefix_release": (c_int32, [c_void_p, c_uint64]),
    "pkv_seq_reserve_cow": (c_int32, [c_void_p, c_int64, c_int32, P_int32, c_int32, P_int32]),
    "pkv_pool_get_stats": (c_int32, [c_void_p, ctypes.POINTER(PoolStats)]),
    "pkv_copy_blocks": (c_int32, [ctypes.POINTER(PagedKV), c_void_p, c_int32, c_void_p]),
    "pkv_sched_run": (c_int32, [ctypes.POINTER(SchedConfig), c_int32, c_int32, P_int32,
                                c_int64, P_int32, P_int32, ctypes.POINTER(ctypes.c_uint8),
                                ctypes.POINTER(SchedDevice), P_int32, c_int64, P_int64,
                                P_int64, ctypes.POINTER(SchedStats)]),
    "pkv_kv_append": (c_int32, [ctypes.POINTER(PagedKV), c_void_p, c_void_p, c_void_p, c_int32,
                                c_void_p, c_void_p, c_int32, c_int32, c_int32, c_void_p]),
    "pkv_prefill_attention": (c_int32, [ctypes.POINTER(PagedKV), c_void_p, c_int32, c_void_p,
                                        c_int32, c_void_p, c_void_p, c_int32, c_int32, c_int32,
                                        c_int32, c_float, c_void_p, c_void_p, c_void_p,
                                        c_size_t, c_void_p]),
    "pkv_prefill_workspace_bytes": (c_size_t, [c_int32] * 7),
    "pkv_decode_attention": (c_int32, [ctypes.POINTER(PagedKV), c_void_p, c_int32, c_void_p,
                                       c_int32, c_void_p, c_int32, c_int32, c_float, c_void_p,
                                       c_void_p, c_void_p, c_size_t, c_void_p]),
    "pkv_decode_workspace_bytes": (c_size_t, [c_int32] * 5),
    "pkv_decode_attention_noalloc": (c_int32, [ctypes.POINTER(PagedKV), c_void_p, c_int32,
                                               c_void_p, c_int32, c_void_p, c_int32, c_int32,
                                               c_float, c_void_p, c_void_p, c_void_p]),
    "pkv_mixed_attention": (c_int32, [ctypes.POINTER(PagedKV), c_int32, c_float, c_void_p,
                                      c_void_p, c_int32, c_void_p, c_void_p, c_int32, c_int32,
                                      c_int32, c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                                      c_int32, c_void_p, c_int32, c_int32, c_void_p, c_void_p,
                                      c_void_p, c_size_t, c_void_p]),
    "pkv_gather_kv": (c_int32, [ctypes.POINTER(PagedKV), c_void_p, c_int32, c_void_p, c_void_p,
                                c_int32, c_int32, c_void_p, c_void_p, c_void_p]),
}

for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args

EXPORTED = tuple(_SIGS)


class PkvError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"[pkv status {status}] {message}")
        self.status = status


def _check(status: int) -> None:
    if status != PKV_OK:
        raise PkvError(status, _lib.pkv_last_error().decode())


def pkv_last_error() -> str:
    return _lib.pkv_last_error().decode()


def pkv_abi_version() -> int:
    return int(_lib.pkv_abi_version())


def pkv_set_debug_validate(on: bool) -> None:
    _check(_lib.pkv_set_debug_validate(1 if on else 0))


def pkv_get_debug_validate() -> bool:
    return bool(_lib.pkv_get_debug_validate())


# ----------------------------------------------------------------------------------------
# Block pool
# ----------------------------------------------------------------------------------------
class BlockPool:
    """Host bookkeeping of the KV block pool (pkv_pool_* / pkv_seq_*)."""

    def __init__(self, num_blocks: int, block_size: int = 16,
                 free_order: Optional[Sequence[int]] = None):
        handle = c_void_p()
        arr = None
        if free_order is not None:
            arr = np.ascontiguousarray(np.asarray(free_order, dtype=np.int32))
            ptr = arr.ctypes.data_as(P_int32)
        else:
            ptr = None
        _check(_lib.pkv_pool_create(num_blocks, block_size, ptr, ctypes.byref(handle)))
        self._h = handle
        self.num_blocks = num_blocks
        self.block_size = block_size

    def close(self):
        if self._h:
            _lib.pkv_pool_destroy(self._h)
            self._h = c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def num_free(self) -> int:
        return int(_lib.pkv_pool_num_free(self._h))

    def create(self) -> int:
        sid = c_int64()
        _check(_lib.pkv_seq_create(self._h, ctypes.byref(sid)))
        return sid.value

    def fork(self, parent: int, shared_tokens: int) -> int:
        sid = c_int64()
        _check(_lib.pkv_seq_fork(self._h, parent, shared_tokens, ctypes.byref(sid)))
        return sid.value

    def reserve(self, seq: int, n: int) -> int:
        """Returns the status (OK, OUT_OF_BLOCKS or SHARED_BLOCK_WRITE are expected outcomes);
        raises on argument errors."""
        st = _lib.pkv_seq_reserve(self._h, seq, n)
        if st not in (PKV_OK, PKV_ERR_OUT_OF_BLOCKS, PKV_ERR_SHARED_BLOCK_WRITE):
            _check(st)
        return st

    def reserve_cow(self, seq: int, n: int):
        """(status, [(source, copy), ...]); OK and OUT_OF_BLOCKS are expected outcomes."""
        s = self.seq_len(seq)  # raises on an unknown sequence
        del s
        room = max(1, -(-n // self.block_size) + 1)  # blocks a write of n tokens can touch
        buf = (c_int32 * (2 * room))()
        cnt = c_int32()
        st = _lib.pkv_seq_reserve_cow(self._h, seq, n, buf, room, ctypes.byref(cnt))
        if st not in (PKV_OK, PKV_ERR_OUT_OF_BLOCKS):
            _check(st)
        return st, [(buf[2 * k], buf[2 * k + 1]) for k in range(cnt.value)]

    def publish(self, seq: int, key: int, tokens: int) -> int:
        """Status: OK or KEY_EXISTS; raises on other errors."""
        st = _lib.pkv_prefix_publish(self._h, seq, key, tokens)
        if st not in (PKV_OK, PKV_ERR_KEY_EXISTS):
            _check(st)
        return st

    def attach(self, key: int):
        """(sequence id, tokens) on a hit, None on a miss."""
        sid, tok = c_int64(), c_int32()
        st = _lib.pkv_prefix_attach(self._h, key, ctypes.byref(sid), ctypes.byref(tok))
        if st == PKV_ERR_NOT_FOUND:
            return None
        _check(st)
        return sid.value, tok.value

    def lookup(self, key: int) -> int:
        tok = c_int32()
        _check(_lib.pkv_prefix_lookup(self._h, key, ctypes.byref(tok)))
        return tok.value

    def pin(self, key: int) -> None:
        _check(_lib.pkv_prefix_pin(self._h, key))

    def unpin(self, key: int) -> None:
        _check(_lib.pkv_prefix_unpin(self._h, key))

    def release(self, key: int) -> None:
        _check(_lib.pkv_prefix_release(self._h, key))

    def set_eviction(self, policy: int) -> None:
        _check(_lib.pkv_pool_set_eviction(self._h, policy))

    def set_pinning(self, mode: int) -> None:
        _check(_lib.pkv_pool_set_pinning(self._h, mode))

    def check_deadlock(self, waiting: int, running: int) -> bool:
        rec = c_int32()
        _check(_lib.pkv_pool_check_deadlock(self._h, waiting, running, ctypes.byref(rec)))
        return bool(rec.value)

    def stats(self) -> dict:
        st = PoolStats()
        _check(_lib.pkv_pool_get_stats(self._h, ctypes.byref(st)))
        return {name: int(getattr(st, name)) for name, _ in PoolStats._fields_}

    def commit(self, seq: int, n: int) -> None:
        _check(_lib.pkv_seq_commit(self._h, seq, n))

    def free(self, seq: int) -> None:
        _check(_lib.pkv_seq_free(self._h, seq))

    def seq_len(self, seq: int) -> int:
        n = c_int32()
        _check(_lib.pkv_seq_len(self._h, seq, ctypes.byref(n)))
        return n.value

    def block_tables(self, seq_ids: Sequence[int], max_blocks: int):
        """(tables int32 [n][max_blocks] padded -1, committed lengths int32 [n])."""
        ids = np.ascontiguousarray(np.asarray(seq_ids, dtype=np.int64))
        n = ids.shape[0]
        tables = np.empty((n, max_blocks), dtype=np.int32)
        lens = np.empty(n, dtype=np.int32)
        _check(_lib.pkv_fill_block_tables(self._h, ids.ctypes.data_as(P_int64), n, max_blocks,
                                          tables.ctypes.data_as(P_int32),
                                          lens.ctypes.data_as(P_int32)))
        return tables, lens


# ----------------------------------------------------------------------------------------
# Pipeline scheduler
# ----------------------------------------------------------------------------------------
def sched_config(policy, num_blocks, max_out, alpha=1.0, beta=0.5, delta=0, pinning=0,
                 eviction=0, breadth_share=0.5, static_bound=None, initial_bound=None,
                 min_obs=8, max_batch=256, max_steps=1_000_000,
                 max_step_tokens=0) -> SchedConfig:
    c = SchedConfig()
    c.policy, c.num_blocks, c.max_out, c.delta = policy, num_blocks, max_out, delta
    c.alpha, c.beta, c.breadth_share = alpha, beta, breadth_share
    c.pinning, c.eviction, c.min_obs, c.max_batch = pinning, eviction, min_obs, max_batch
    c.max_steps = max_steps
    c.max_step_tokens = max_step_tokens
    for s, v in enumerate(static_bound or []):
        c.static_bound[s] = int(v)
    for s, v in enumerate(initial_bound or []):
        c.initial_bound[s] = int(v)
    return c


def pkv_sched_run(cfg: SchedConfig, fanout, suffix, out_len, filtered, device=None,
                  max_events: int = 0, group_hook=None):
    """Run a pipeline (per-stage arrays, as the oracle's Pipeline takes them).
    Returns (stats dict, trace int32 [n][5] (None when max_events is 0), final budgets).
    device: None, or a dict(k_cache, v_cache, q_src, k_src, v_src[, stream]) of GPU tensors
    for device mode. group_hook (device mode): a callable receiving, for every group of
    sequences launched together, a dict(step, phase, decode, tables, cached, cu_new, out_ptr)
    with the host metadata as numpy copies (phase 0 before the group's append, 1 after its
    attention)."""
    S = len(suffix)
    fan = np.ascontiguousarray(np.asarray(list(fanout) + [1] * (S - len(fanout)),
                                          dtype=np.int32)[:S])
    suf = np.ascontiguousarray(np.concatenate([np.asarray(a) for a in suffix]).astype(np.int32))
    out = np.ascontiguousarray(np.concatenate([np.asarray(a) for a in out_len]).astype(np.int32))
    flt = np.ascontiguousarray(np.concatenate([np.asarray(a) for a in filtered]).astype(np.uint8))
    trace = np.zeros((max(max_events, 1), 5), dtype=np.int32)
    n_ev = c_int64()
    budgets = np.zeros(S, dtype=np.int64)
    stats = SchedStats()
    dev_arg = None
    if device is not None:
        import torch
        hq, d = int(device["q_src"].shape[1]), int(device["q_src"].shape[2])
        kv = paged_kv(device["k_cache"], device["v_cache"])
        dv = SchedDevice()
        dv.kv = kv
        dv.num_q_heads = hq
        dv.q_src = _dev_ptr(device["q_src"], "q_src", torch.bfloat16)
        dv.k_src = _dev_ptr(device["k_src"], "k_src", torch.bfloat16)
        dv.v_src = _dev_ptr(device["v_src"], "v_src", torch.bfloat16)
        dv.src_rows = int(min(device["q_src"].shape[0], device["k_src"].shape[0]))
        dv.stream = _stream(device.get("stream"))
        if int(device["k_src"].shape[2]) != d:
            raise ValueError("q_src / k_src head dims differ")
        if group_hook is not None:
            def _hook(_user, gp):
                g = gp.contents
                n, mb = int(g.num_seqs), int(g.max_blocks)
                group_hook(dict(
                    step=int(g.step), phase=int(g.phase), decode=bool(g.decode),
                    tables=np.ctypeslib.as_array(g.tables, shape=(n * mb,)).reshape(n, mb).copy(),
                    cached=np.ctypeslib.as_array(g.cached, shape=(n,)).copy(),
                    cu_new=np.ctypeslib.as_array(g.cu_new, shape=(n + 1,)).copy(),
                    out_ptr=int(g.out or 0)))
            dv.group_hook = SCHED_GROUP_HOOK(_hook)
        dev_arg = ctypes.byref(dv)
    if not (len(out) == len(suf) == len(flt)):
        raise ValueError("suffix, out_len and filtered must have the same lengths")
    _check(_lib.pkv_sched_run(ctypes.byref(cfg), S, int(len(suffix[0])),
                              fan.ctypes.data_as(P_int32), int(len(suf)),
                              suf.ctypes.data_as(P_int32),
                              out.ctypes.data_as(P_int32),
                              flt.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), dev_arg,
                              trace.ctypes.data_as(P_int32) if max_events else None,
                              max_events, ctypes.byref(n_ev),
                              budgets.ctypes.data_as(P_int64), ctypes.byref(stats)))
    st = {name: getattr(stats, name) for name, _ in SchedStats._fields_}
    tr = trace[: min(n_ev.value, max_events)] if max_events else None
    st["num_events"] = n_ev.value
    return st, tr, budgets


# ----------------------------------------------------------------------------------------
# Device calls (torch tensors on the GPU)
# ----------------------------------------------------------------------------------------
def _dev_ptr(t, name, dtype=None):
    import torch
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a GPU tensor (the library has no CPU path)")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return c_void_p(s.cuda_stream)


def paged_kv(k_cache, v_cache) -> PagedKV:
    """Describe a pool: k_cache bf16 [num_blocks][Hkv][D/8][16][8], v_cache bf16
    [num_blocks][Hkv][D][16]."""
    import torch
    if k_cache.dim() != 5 or v_cache.dim() != 4:
        raise ValueError("k_cache must be [nb][Hkv][D/8][bs][8] and v_cache [nb][Hkv][D][bs]")
    nb, hkv, nch, bs, e = k_cache.shape
    if e != 8 or tuple(v_cache.shape) != (nb, hkv, nch * 8, bs):
        raise ValueError("k_cache / v_cache shapes disagree")
    kp = _dev_ptr(k_cache, "k_cache", torch.bfloat16)
    vp = _dev_ptr(v_cache, "v_cache", torch.bfloat16)
    return PagedKV(kp, vp, nb, bs, hkv, nch * 8)


def pkv_kv_append(k_cache, v_cache, k_new, v_new, block_tables, cached_lens, cu_new_lens,
                  max_new_len: int, stream=None) -> None:
    import torch
    kv = paged_kv(k_cache, v_cache)
    b = int(cached_lens.shape[0])
    _check(_lib.pkv_kv_append(ctypes.byref(kv), _dev_ptr(k_new, "k_new", torch.bfloat16),
                              _dev_ptr(v_new, "v_new", torch.bfloat16),
                              _dev_ptr(block_tables, "block_tables", torch.int32),
                              int(block_tables.shape[1]),
                              _dev_ptr(cached_lens, "cached_lens", torch.int32),
                              _dev_ptr(cu_new_lens, "cu_new_lens", torch.int32), b,
                              int(k_new.shape[0]), int(max_new_len), _stream(stream)))


def pkv_prefill_workspace_bytes(num_seqs, total_new, num_q_heads, num_kv_heads, head_dim,
                                max_new_len, max_total_len) -> int:
    return int(_lib.pkv_prefill_workspace_bytes(num_seqs, total_new, num_q_heads, num_kv_heads,
                                                head_dim, max_new_len, max_total_len))


def pkv_prefill_attention(k_cache, v_cache, q, block_tables, cached_lens, cu_new_lens,
                          max_new_len: int, max_total_len: int, scale: float, out, lse=None,
                          workspace=None, stream=None) -> None:
    import torch
    kv = paged_kv(k_cache, v_cache)
    t, hq, d = q.shape
    b = int(cached_lens.shape[0])
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.pkv_prefill_attention(
        ctypes.byref(kv), _dev_ptr(q, "q", torch.bfloat16), hq,
        _dev_ptr(block_tables, "block_tables", torch.int32), int(block_tables.shape[1]),
        _dev_ptr(cached_lens, "cached_lens", torch.int32),
        _dev_ptr(cu_new_lens, "cu_new_lens", torch.int32), b, t, int(max_new_len),
        int(max_total_len), float(scale), _dev_ptr(out, "out", torch.bfloat16),
        _dev_ptr(lse, "lse", torch.float32), _dev_ptr(workspace, "workspace"), ws_bytes,
        _stream(stream)))


def pkv_decode_workspace_bytes(num_seqs, num_q_heads, num_kv_heads, head_dim,
                               max_seq_len) -> int:
    return int(_lib.pkv_decode_workspace_bytes(num_seqs, num_q_heads, num_kv_heads, head_dim,
                                               max_seq_len))


def pkv_decode_attention(k_cache, v_cache, q, block_tables, seq_lens, max_seq_len: int,
                         scale: float, out, lse=None, workspace=None, stream=None) -> None:
    import torch
    kv = paged_kv(k_cache, v_cache)
    b, hq, d = q.shape
    if workspace is None:  # convenience for one-off calls; timed callers pass their own
        workspace = alloc_workspace(pkv_decode_workspace_bytes(b, hq, int(k_cache.shape[1]), d,
                                                               int(max_seq_len)))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.pkv_decode_attention(
        ctypes.byref(kv), _dev_ptr(q, "q", torch.bfloat16), hq,
        _dev_ptr(block_tables, "block_tables", torch.int32), int(block_tables.shape[1]),
        _dev_ptr(seq_lens, "seq_lens", torch.int32), b, int(max_seq_len), float(scale),
        _dev_ptr(out, "out", torch.bfloat16), _dev_ptr(lse, "lse", torch.float32),
        _dev_ptr(workspace, "workspace"), ws_bytes, _stream(stream)))


PKV_DECODE_NOALLOC_MAX_BYTES = 32 << 20


def pkv_decode_attention_noalloc(k_cache, v_cache, q, block_tables, seq_lens, max_seq_len: int,
                                 scale: float, out, lse=None, stream=None) -> None:
    """pkv_decode_attention without a workspace argument: the library's fixed per-GPU
    scratch array serves instead (nothing is allocated here or in the library)."""
    import torch
    kv = paged_kv(k_cache, v_cache)
    b, hq, d = q.shape
    _check(_lib.pkv_decode_attention_noalloc(
        ctypes.byref(kv), _dev_ptr(q, "q", torch.bfloat16), hq,
        _dev_ptr(block_tables, "block_tables", torch.int32), int(block_tables.shape[1]),
        _dev_ptr(seq_lens, "seq_lens", torch.int32), b, int(max_seq_len), float(scale),
        _dev_ptr(out, "out", torch.bfloat16), _dev_ptr(lse, "lse", torch.float32),
        _stream(stream)))


def pkv_mixed_attention(k_cache, v_cache, scale: float,
                        q, block_tables, cached_lens, cu_new_lens, max_new_len: int,
                        max_total_len: int, out,
                        dq, d_block_tables, seq_lens, max_seq_len: int, d_out,
                        lse=None, d_lse=None, workspace=None, stream=None) -> None:
    """A prefill batch (as pkv_prefill_attention) and a decode batch (as
    pkv_decode_attention) in one fused launch."""
    import torch
    kv = paged_kv(k_cache, v_cache)
    t, hq, d = q.shape
    b = int(cached_lens.shape[0])
    bd = int(seq_lens.shape[0])
    if workspace is None:
        workspace = alloc_workspace(pkv_decode_workspace_bytes(bd, hq, int(k_cache.shape[1]), d,
                                                               int(max_seq_len)))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.pkv_mixed_attention(
        ctypes.byref(kv), hq, float(scale), _dev_ptr(q, "q", torch.bfloat16),
        _dev_ptr(block_tables, "block_tables", torch.int32), int(block_tables.shape[1]),
        _dev_ptr(cached_lens, "cached_lens", torch.int32),
        _dev_ptr(cu_new_lens, "cu_new_lens", torch.int32), b, t, int(max_new_len),
        int(max_total_len), _dev_ptr(out, "out", torch.bfloat16),
        _dev_ptr(lse, "lse", torch.float32), _dev_ptr(dq, "dq", torch.bfloat16),
        _dev_ptr(d_block_tables, "d_block_tables", torch.int32),
        int(d_block_tables.shape[1]), _dev_ptr(seq_lens, "seq_lens", torch.int32), bd,
        int(max_seq_len), _dev_ptr(d_out, "d_out", torch.bfloat16),
        _dev_ptr(d_lse, "d_lse", torch.float32), _dev_ptr(workspace, "workspace"), ws_bytes,
        _stream(stream)))


def pkv_copy_blocks(k_cache, v_cache, pairs, stream=None) -> None:
    """pairs: int32 GPU tensor [n][2] of (source block, copy)."""
    import torch
    kv = paged_kv(k_cache, v_cache)
    if pairs.dim() != 2 or pairs.shape[1] != 2:
        raise ValueError("pairs must be [n][2]")
    _check(_lib.pkv_copy_blocks(ctypes.byref(kv), _dev_ptr(pairs, "pairs", torch.int32),
                                int(pairs.shape[0]), _stream(stream)))


def pkv_gather_kv(k_cache, v_cache, block_tables, lens, cu_lens, max_len: int, k_out, v_out,
                  stream=None) -> None:
    import torch
    kv = paged_kv(k_cache, v_cache)
    _check(_lib.pkv_gather_kv(ctypes.byref(kv), _dev_ptr(block_tables, "block_tables",
                                                         torch.int32),
                              int(block_tables.shape[1]), _dev_ptr(lens, "lens", torch.int32),
                              _dev_ptr(cu_lens, "cu_lens", torch.int32), int(lens.shape[0]),
                              int(max_len), _dev_ptr(k_out, "k_out", torch.bfloat16),
                              _dev_ptr(v_out, "v_out", torch.bfloat16), _stream(stream)))


def alloc_workspace(nbytes: int, device="cuda"):
    """A byte tensor for the workspace argument (None when nbytes is 0)."""
    import torch
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=device)
