"""GPU tier for the opt-in metadata validation (PKV_DEBUG_VALIDATE), through the C ABI.

With validation on, every device call first checks its device metadata (block ids within the
pool, lengths within the host maxima and the table, token offsets starting at 0, never
decreasing, ending at the total) and refuses a call that fails with PKV_ERR_BAD_METADATA,
launching nothing else. Good metadata passes and gives the same bits as with validation off.
The malformed cases never reach the attention or copy kernels (and those kernels only bound
what they index in any case)."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import DevBatch, dev_pools, i32, say, scale_for, to_host_bits

pytestmark = pytest.mark.gpu


@pytest.fixture
def validating(gpu_lib):
    gpu_lib.pkv_set_debug_validate(True)
    assert gpu_lib.pkv_get_debug_validate()
    yield gpu_lib
    gpu_lib.pkv_set_debug_validate(False)


def _mixed_case():
    spec = W.MIXED_70B.scaled(prefill=3, decode=5)
    return W.make_case(spec)


def _refused(lib, fn, *args, what, **kw):
    with pytest.raises(lib.PkvError) as e:
        fn(*args, **kw)
    assert e.value.status == lib.PKV_ERR_BAD_METADATA, str(e.value)
    msg = lib.pkv_last_error()
    assert "PKV_DEBUG_VALIDATE" in msg and what in msg, msg
    say(f"  refused: {msg}")
    return msg


def test_good_metadata_passes_with_identical_results(gpu_lib):
    import torch
    lib = gpu_lib
    say("[validate] good metadata, validation on vs off")
    outs = []
    for on in (False, True):
        lib.pkv_set_debug_validate(on)
        try:
            case = _mixed_case()
            bp, bd = case.batches
            pk, pv = dev_pools(case)
            p, d = DevBatch(bp), DevBatch(bd)
            lib.pkv_kv_append(pk, pv, p.k_new, p.v_new, p.tables, p.cached, p.cu, p.max_new)
            lib.pkv_kv_append(pk, pv, d.k_new, d.v_new, d.tables, d.cached, d.cu, 1)
            op = torch.empty((bp.total_new, case.hq, case.d), dtype=torch.bfloat16, device="cuda")
            od = torch.empty((bd.n_seqs, case.hq, case.d), dtype=torch.bfloat16, device="cuda")
            sl = i32(bd.prefix_lens + 1)
            maxl = int(bd.prefix_lens.max()) + 1
            lib.pkv_prefill_attention(pk, pv, p.q, p.tables, p.cached, p.cu, p.max_new,
                                      p.max_total, scale_for(case.d), op)
            lib.pkv_decode_attention(pk, pv, d.q, d.tables, sl, maxl, scale_for(case.d), od)
            om = torch.empty_like(op)
            odm = torch.empty_like(od)
            lib.pkv_mixed_attention(pk, pv, scale_for(case.d), p.q, p.tables, p.cached, p.cu,
                                    p.max_new, p.max_total, om, d.q, d.tables, sl, maxl, odm)
            on_ = torch.empty_like(od)
            lib.pkv_decode_attention_noalloc(pk, pv, d.q, d.tables, sl, maxl, scale_for(case.d),
                                             on_)
            lens = bp.prefix_lens + bp.new_lens
            cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
            gk = torch.empty((int(cu[-1]), case.hkv, case.d), dtype=torch.bfloat16, device="cuda")
            gv = torch.empty_like(gk)
            lib.pkv_gather_kv(pk, pv, p.tables, i32(lens), i32(cu), int(lens.max()), gk, gv)
            torch.cuda.synchronize()
            outs.append([to_host_bits(x) for x in (op, od, om, odm, on_, gk, gv, pk, pv)])
        finally:
            lib.pkv_set_debug_validate(False)
    for a, b in zip(*outs):
        assert np.array_equal(a, b)


def test_malformed_metadata_is_refused(validating):
    import torch
    lib = validating
    say("[validate] malformed metadata")
    case = _mixed_case()
    bp, bd = case.batches
    pk, pv = dev_pools(case)
    p, d = DevBatch(bp), DevBatch(bd)
    nb = case.num_blocks
    scale = scale_for(case.d)
    op = torch.empty((bp.total_new, case.hq, case.d), dtype=torch.bfloat16, device="cuda")
    od = torch.empty((bd.n_seqs, case.hq, case.d), dtype=torch.bfloat16, device="cuda")
    sl_h = (bd.prefix_lens + 1).astype(np.int32)
    maxl = int(sl_h.max())
    before = (to_host_bits(pk), to_host_bits(pv))

    # a block id past the pool inside a prefill sequence's range (sequence 1)
    t = bp.block_tables.copy()
    t[1, 0] = nb
    msg = _refused(lib, lib.pkv_prefill_attention, pk, pv, p.q, i32(t), p.cached, p.cu,
                   p.max_new, p.max_total, scale, op, what="block id outside the pool")
    assert "sequence 1" in msg
    # the append checks the entries it writes: a bad id where sequence 1's new tokens go
    t = bp.block_tables.copy()
    t[1, int(bp.prefix_lens[1]) // 16] = nb + 3
    msg = _refused(lib, lib.pkv_kv_append, pk, pv, p.k_new, p.v_new, i32(t), p.cached, p.cu,
                   p.max_new, what="block id outside the pool")
    assert "sequence 1" in msg
    # -1 inside a decode sequence's range (sequence 2)
    t = bd.block_tables.copy()
    t[2, 0] = -1
    msg = _refused(lib, lib.pkv_decode_attention, pk, pv, d.q, i32(t), i32(sl_h), maxl, scale,
                   od, what="block id outside the pool")
    assert "sequence 2" in msg
    # decode lengths: above max_seq_len, and zero
    bad = sl_h.copy()
    bad[3] = maxl + 1
    _refused(lib, lib.pkv_decode_attention, pk, pv, d.q, d.tables, i32(bad), maxl, scale, od,
             what="length outside")
    bad = sl_h.copy()
    bad[0] = 0
    _refused(lib, lib.pkv_decode_attention_noalloc, pk, pv, d.q, d.tables, i32(bad), maxl,
             scale, od, what="length outside")
    # prefill: cached + new beyond max_total_len
    _refused(lib, lib.pkv_prefill_attention, pk, pv, p.q, p.tables, p.cached, p.cu, p.max_new,
             p.max_total - 1, scale, op, what="length outside")
    # token offsets: decreasing, and not ending at the total
    cu = bp.cu_new_lens.copy()
    cu[1], cu[2] = cu[2], cu[1]
    _refused(lib, lib.pkv_prefill_attention, pk, pv, p.q, p.tables, p.cached, i32(cu),
             p.max_total, p.max_total, scale, op, what="token offsets")
    cu = bp.cu_new_lens.copy()
    cu[-1] -= 1
    _refused(lib, lib.pkv_kv_append, pk, pv, p.k_new, p.v_new, p.tables, p.cached, i32(cu),
             p.max_new, what="token offsets")
    # mixed: the decode half is malformed
    t = bd.block_tables.copy()
    t[4, 0] = nb + 7
    msg = _refused(lib, lib.pkv_mixed_attention, pk, pv, scale, p.q, p.tables, p.cached, p.cu,
                   p.max_new, p.max_total, op, d.q, i32(t), i32(sl_h), maxl, od,
                   what="block id outside the pool")
    assert "decode batch" in msg and "sequence 4" in msg
    # gather: a length above max_len
    lens = (bp.prefix_lens + bp.new_lens).astype(np.int32)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    gk = torch.empty((int(cu[-1]), case.hkv, case.d), dtype=torch.bfloat16, device="cuda")
    gv = torch.empty_like(gk)
    _refused(lib, lib.pkv_gather_kv, pk, pv, p.tables, i32(lens), i32(cu), int(lens.max()) - 1,
             gk, gv, what="length outside")
    torch.cuda.synchronize()
    # nothing above was launched past its validation: the pool is unchanged
    assert np.array_equal(to_host_bits(pk), before[0])
    assert np.array_equal(to_host_bits(pv), before[1])
