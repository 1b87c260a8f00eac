"""GPU tier for the block-pool lifecycle: the device half of copy-on-write (pkv_copy_blocks,
bit-exact against the oracle), and a prefix published with a partly filled last block that
three sequences continue at once -- two attached from the cache and the publisher itself --
each through copy-on-write, then append and prefill attention (Section 2.1: the cached
prefix is reused and only the suffix computed). The cached prefix must come out untouched,
every pool byte must equal the oracle's, and attention must meet the attention bar."""
import numpy as np
import pytest

import oracle
from tests.gpu_util import bf16_to_f64, compare, i32, say, scale_for, to_dev_bits, to_host_bits
from tests.test_gpu_prefill import LSE_MAX, LSE_MEAN

pytestmark = pytest.mark.gpu


def _random_pool(rng, nb, hkv, d, bs=16):
    """Finite random bf16 bit patterns (no attention reads beyond what the tables name)."""
    def bits(shape):
        x = rng.standard_normal(shape).astype(np.float32)
        return (x.view(np.uint32) >> 16).astype(np.uint16)
    return bits((nb, hkv, d // 8, bs, 8)), bits((nb, hkv, d, bs))


@pytest.mark.parametrize("hkv,d", [(8, 128), (2, 64)])
def test_copy_blocks_bit_exact(gpu_lib, hkv, d):
    import torch
    lib = gpu_lib
    say(f"[copy_blocks] hkv={hkv} d={d}")
    rng = np.random.default_rng(7 + d)
    nb = 48
    pk_h, pv_h = _random_pool(rng, nb, hkv, d)
    pk, pv = to_dev_bits(pk_h), to_dev_bits(pv_h)
    perm = rng.permutation(nb)
    srcs, dsts = perm[:10], perm[10:20]
    pairs = [(int(s), int(t)) for s, t in zip(srcs, dsts)]
    pairs[3] = (int(srcs[0]), pairs[3][1])  # one source copied twice
    pairs += [(-1, int(perm[30])), (int(perm[31]), nb)]  # out-of-pool pairs are skipped
    lib.pkv_copy_blocks(pk, pv, i32(np.asarray(pairs, np.int32)))
    lib.pkv_copy_blocks(pk, pv, i32(np.zeros((0, 2), np.int32)))  # no pairs: a no-op
    torch.cuda.synchronize()
    ek, ev = oracle.copy_blocks(pk_h, pv_h, pairs)
    assert np.array_equal(to_host_bits(pk), ek)
    assert np.array_equal(to_host_bits(pv), ev)
    assert not np.array_equal(ek, pk_h)  # the copies did change something


def test_copy_on_write_continuations_of_a_cached_prefix(gpu_lib):
    import torch
    lib = gpu_lib
    say("[lifecycle] publish / attach / copy-on-write / append / prefill")
    rng = np.random.default_rng(2607)
    hq, hkv, d, bs, nb = 32, 8, 128, 16, 40
    prefix = 40  # blocks 0, 1 and half of block 2
    pk_h, pv_h = _random_pool(rng, nb, hkv, d)
    pool = lib.BlockPool(nb, bs, free_order=rng.permutation(nb))

    def bits(shape):
        x = rng.standard_normal(shape).astype(np.float32)
        return (x.view(np.uint32) >> 16).astype(np.uint16)

    # upstream operator: sequence a computes the tuple's prefix and publishes it
    a = pool.create()
    assert pool.reserve(a, prefix) == lib.PKV_OK
    k_pre, v_pre = bits((prefix, hkv, d)), bits((prefix, hkv, d))
    t_a, _ = pool.block_tables([a], 8)
    cu = np.array([0, prefix], np.int32)
    pk, pv = to_dev_bits(pk_h), to_dev_bits(pv_h)
    lib.pkv_kv_append(pk, pv, to_dev_bits(k_pre), to_dev_bits(v_pre), i32(t_a),
                      i32([0]), i32(cu), prefix)
    ref_k, ref_v = oracle.kv_append(pk_h, pv_h, t_a, [0], cu, k_pre, v_pre, bs)
    pool.commit(a, prefix)
    assert pool.publish(a, 0xC0FFEE, prefix) == lib.PKV_OK
    entry_row = t_a[0].copy()

    # downstream: two cache hits plus the publisher continue the same prefix
    b, nb_tok = pool.attach(0xC0FFEE)
    c, nc_tok = pool.attach(0xC0FFEE)
    assert nb_tok == nc_tok == prefix
    news = {a: 5, b: 30, c: 9}
    order = [a, b, c]
    pairs = []
    for s in order:
        assert pool.reserve(s, news[s]) == lib.PKV_ERR_SHARED_BLOCK_WRITE
        st, cp = pool.reserve_cow(s, news[s])
        assert st == lib.PKV_OK and len(cp) == 1 and cp[0][0] == entry_row[2]
        pairs += cp
    assert pool.stats()["cow_copies"] == 3
    lib.pkv_copy_blocks(pk, pv, i32(np.asarray(pairs, np.int32)))
    ref_k, ref_v = oracle.copy_blocks(ref_k, ref_v, pairs)

    tables, lens = pool.block_tables(order, 8)
    assert list(lens) == [prefix] * 3
    n = np.array([news[s] for s in order])
    cu_n = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    k_new, v_new = bits((int(n.sum()), hkv, d)), bits((int(n.sum()), hkv, d))
    q = bits((int(n.sum()), hq, d))
    lib.pkv_kv_append(pk, pv, to_dev_bits(k_new), to_dev_bits(v_new), i32(tables), i32(lens),
                      i32(cu_n), int(n.max()))
    out = torch.empty((int(n.sum()), hq, d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((int(n.sum()), hq), dtype=torch.float32, device="cuda")
    scale = scale_for(d)
    lib.pkv_prefill_attention(pk, pv, to_dev_bits(q), i32(tables), i32(lens), i32(cu_n),
                              int(n.max()), int((lens + n).max()), scale, out, lse=lse)
    torch.cuda.synchronize()

    # the pool byte for byte (copies, appends, and every block nobody wrote)
    ref_k, ref_v = oracle.kv_append(ref_k, ref_v, tables, lens, cu_n, k_new, v_new, bs)
    got_k, got_v = to_host_bits(pk), to_host_bits(pv)
    assert np.array_equal(got_k, ref_k) and np.array_equal(got_v, ref_v)
    # the cached prefix still holds exactly what the upstream operator wrote
    ck, cv = oracle.gather_seq(got_k, got_v, entry_row, prefix, bs)
    assert np.array_equal(ck, k_pre) and np.array_equal(cv, v_pre)
    # each continuation sees the shared prefix followed by its own suffix
    for i, s in enumerate(order):
        sk, sv = oracle.gather_seq(got_k, got_v, tables[i], prefix + n[i], bs)
        assert np.array_equal(sk[:prefix], k_pre)
        assert np.array_equal(sk[prefix:], k_new[cu_n[i]:cu_n[i + 1]])
        assert np.array_equal(sv[prefix:], v_new[cu_n[i]:cu_n[i + 1]])
    ro, rl = oracle.prefill_attention(ref_k, ref_v, tables, lens, cu_n, q, k_new, v_new, scale,
                                      bs)
    compare("cow prefill out", bf16_to_f64(to_host_bits(out)), ro)
    compare("cow prefill lse", lse.cpu().numpy().astype(np.float64), rl, atol_max=LSE_MAX,
            atol_mean=LSE_MEAN)

    for s in order:
        pool.free(s)
    assert pool.stats()["cached_blocks"] == 3  # the entry alone keeps its three blocks
    pool.release(0xC0FFEE)
    assert pool.num_free() == nb
