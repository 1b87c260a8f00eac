"""Pins of the CPU oracle against things other than itself (CPU only).

Each test names what fixes the expected value: a library routine (torch's scaled dot-product
attention in float64), the paper's prefix-reuse invariant, closed forms and special cases,
invariants, brute force, or a figure printed in the paper (tests/golden/)."""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from tests.paged_fixture import empty_pools, place, rand_bf16, widen

BS = 16
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _sdpa_reference(q_bits, k_bits, v_bits, visible, scale):
    """torch SDPA (CPU, float64) on contiguous tensors; K/V repeated to every query head."""
    n, hq, d = q_bits.shape
    hkv = k_bits.shape[1]
    g = hq // hkv
    q = torch.from_numpy(widen(q_bits)).permute(1, 0, 2)[None]            # [1][Hq][n][D]
    k = torch.from_numpy(widen(k_bits)).permute(1, 0, 2).repeat_interleave(g, 0)[None]
    v = torch.from_numpy(widen(v_bits)).permute(1, 0, 2).repeat_interleave(g, 0)[None]
    L = k_bits.shape[0]
    mask = torch.arange(L)[None, :] < torch.as_tensor(visible)[:, None]
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=scale)
    return o[0].permute(1, 0, 2).numpy()


def _paged_prefix_case(rng, p, n, hq, hkv, d, extra_blocks=3):
    """Contiguous K/V for p + n tokens; the first p placed in a pool at random blocks."""
    L = p + n
    nblk = -(-L // BS)
    num_blocks = nblk + extra_blocks
    table = rng.permutation(num_blocks)[:nblk].astype(np.int32)
    k_all = rand_bf16(rng, (L, hkv, d))
    v_all = rand_bf16(rng, (L, hkv, d))
    q = rand_bf16(rng, (n, hq, d))
    pk, pv = empty_pools(num_blocks, hkv, d, BS)
    place(pk, pv, table, k_all[:p], v_all[:p], BS)
    return dict(pk=pk, pv=pv, table=table[None, :], k_all=k_all, v_all=v_all, q=q, p=p, n=n)


MICRO = [(d, g, p, n) for d in (64, 128) for g in (1, 2, 4, 8)
         for p in (0, 1, 15, 16, 17) for n in (1, 2, 16, 33)]


@pytest.mark.parametrize("d,g,p,n", MICRO[::3] + [(128, 4, 17, 33), (64, 2, 16, 16)])
def test_pi1_prefill_equals_torch_sdpa(d, g, p, n):
    """Pi1: the oracle on a paged pool == torch SDPA (float64) on the unpaged tensors."""
    rng = np.random.default_rng(1000 + d + 10 * g + 100 * p + n)
    hkv = 2
    hq = hkv * g
    c = _paged_prefix_case(rng, p, n, hq, hkv, d)
    scale = 1.0 / math.sqrt(d)
    o, lse = oracle.prefill_attention(c["pk"], c["pv"], c["table"], [p], [0, n], c["q"],
                                      c["k_all"][p:], c["v_all"][p:], scale, BS)
    visible = p + np.arange(n) + 1
    ref = _sdpa_reference(c["q"], c["k_all"], c["v_all"], visible, scale)
    assert np.max(np.abs(o - ref)) <= 1e-12


def test_pi1_lse_equals_torch_logsumexp():
    rng = np.random.default_rng(7)
    p, n, hq, hkv, d = 17, 9, 4, 2, 64
    c = _paged_prefix_case(rng, p, n, hq, hkv, d)
    scale = 1.0 / math.sqrt(d)
    _, lse = oracle.prefill_attention(c["pk"], c["pv"], c["table"], [p], [0, n], c["q"],
                                      c["k_all"][p:], c["v_all"][p:], scale, BS)
    q = torch.from_numpy(widen(c["q"]))
    k = torch.from_numpy(widen(c["k_all"]))
    for j in range(n):
        for h in range(hq):
            s = scale * (k[: p + j + 1, h // 2] @ q[j, h])
            assert abs(float(torch.logsumexp(s, 0)) - lse[j, h]) <= 1e-12


def test_pi1_decode_equals_torch_sdpa():
    rng = np.random.default_rng(11)
    hq, hkv, d = 8, 2, 128
    ctx = [0, 5, 16, 31, 40]
    scale = 1.0 / math.sqrt(d)
    num_blocks = sum(-(-(c + 1) // BS) for c in ctx) + 4
    perm = rng.permutation(num_blocks)
    pk, pv = empty_pools(num_blocks, hkv, d, BS)
    tables = np.full((len(ctx), 4), -1, np.int32)
    q = rand_bf16(rng, (len(ctx), hq, d))
    kn = rand_bf16(rng, (len(ctx), hkv, d))
    vn = rand_bf16(rng, (len(ctx), hkv, d))
    fulls = []
    cur = 0
    for i, c in enumerate(ctx):
        nb = -(-(c + 1) // BS)
        tables[i, :nb] = perm[cur:cur + nb]
        cur += nb
        kk = rand_bf16(rng, (c, hkv, d))
        vv = rand_bf16(rng, (c, hkv, d))
        place(pk, pv, tables[i], kk, vv, BS)
        fulls.append((np.concatenate([kk, kn[i:i + 1]]), np.concatenate([vv, vn[i:i + 1]])))
    o, _ = oracle.decode_attention(pk, pv, tables, ctx, q, kn, vn, scale, BS)
    for i, c in enumerate(ctx):
        ref = _sdpa_reference(q[i:i + 1], fulls[i][0], fulls[i][1], [c + 1], scale)
        assert np.max(np.abs(o[i] - ref[0])) <= 1e-12


@pytest.mark.parametrize("p,n", [(1, 1), (15, 2), (16, 16), (17, 33), (40, 7)])
def test_pi2_prefix_reuse_equals_recompute(p, n):
    """Pi2 (Section 2.1, prefix sharing): prefill over a cached prefix of P tokens gives the
    same rows as recomputing the whole P + N prompt from scratch (rows P..P+N-1)."""
    rng = np.random.default_rng(p * 100 + n)
    hq, hkv, d = 8, 2, 64
    c = _paged_prefix_case(rng, p, n, hq, hkv, d)
    scale = 1.0 / math.sqrt(d)
    o_reuse, lse_reuse = oracle.prefill_attention(
        c["pk"], c["pv"], c["table"], [p], [0, n], c["q"], c["k_all"][p:], c["v_all"][p:],
        scale, BS)
    # recompute: empty cache, all P + N tokens are new; queries for the prefix are fresh draws
    q_full = np.concatenate([rand_bf16(rng, (p, hq, d)), c["q"]])
    pk0, pv0 = empty_pools(4, hkv, d, BS)
    o_full, lse_full = oracle.prefill_attention(
        pk0, pv0, np.full((1, 1), -1, np.int32), [0], [0, p + n], q_full, c["k_all"],
        c["v_all"], scale, BS)
    assert np.max(np.abs(o_reuse - o_full[p:])) <= 1e-12
    assert np.max(np.abs(lse_reuse - lse_full[p:])) <= 1e-12


def test_pi3_softmax_rows_sum_to_one_and_hide_future_keys():
    """Pi3: with V = identity, the output rows are the attention weights: non-negative,
    summing to 1, exactly zero on keys after the row's last visible key."""
    rng = np.random.default_rng(3)
    L, d = 37, 64
    q = rng.standard_normal((L, d))
    k = rng.standard_normal((L, d))
    visible = np.arange(L) + 1
    w, _ = oracle.softmax_attention(q, k, np.eye(L), visible, 0.125)
    assert np.all(w >= 0)
    assert np.max(np.abs(w.sum(axis=1) - 1.0)) <= 1e-12
    assert np.all(w[np.triu_indices(L, 1)] == 0.0)


def test_pi3_constant_values_give_constant_output():
    rng = np.random.default_rng(4)
    p, n, hq, hkv, d = 33, 12, 4, 2, 64
    c = _paged_prefix_case(rng, p, n, hq, hkv, d)
    one = np.uint16(0x3F80)  # bf16 1.0
    pv_one = np.where(c["pv"] == 0x7FC0, c["pv"], one).astype(np.uint16)
    o, _ = oracle.prefill_attention(c["pk"], pv_one, c["table"], [p], [0, n], c["q"],
                                    c["k_all"][p:], np.full_like(c["v_all"][p:], one), 0.125, BS)
    assert np.max(np.abs(o - 1.0)) <= 1e-12


def test_pi4_gqa_equals_mha_on_repeated_kv():
    """Pi4: query head h reads kv head h // g. Running the same data as multi-head attention
    with K/V repeated per query head gives the identical result."""
    rng = np.random.default_rng(5)
    p, n, hq, hkv, d = 21, 10, 8, 2, 64
    g = hq // hkv
    c = _paged_prefix_case(rng, p, n, hq, hkv, d)
    o_gqa, _ = oracle.prefill_attention(c["pk"], c["pv"], c["table"], [p], [0, n], c["q"],
                                        c["k_all"][p:], c["v_all"][p:], 0.125, BS)
    k_rep = np.repeat(c["k_all"], g, axis=1)
    v_rep = np.repeat(c["v_all"], g, axis=1)
    pk, pv = empty_pools(c["pk"].shape[0], hq, d, BS)
    place(pk, pv, c["table"][0], k_rep[:p], v_rep[:p], BS)
    o_mha, _ = oracle.prefill_attention(pk, pv, c["table"], [p], [0, n], c["q"], k_rep[p:],
                                        v_rep[p:], 0.125, BS)
    assert np.array_equal(o_gqa, o_mha)
    # and the mapping is h // g, not h % Hkv: swapping the two kv heads changes the output
    o_swapped, _ = oracle.prefill_attention(c["pk"][:, ::-1], c["pv"][:, ::-1], c["table"], [p],
                                            [0, n], c["q"], c["k_all"][p:, ::-1],
                                            c["v_all"][p:, ::-1], 0.125, BS)
    assert not np.allclose(o_gqa, o_swapped)


def test_pi5_single_key_returns_its_value():
    rng = np.random.default_rng(6)
    hq, hkv, d = 4, 2, 128
    q = rand_bf16(rng, (1, hq, d))
    kn = rand_bf16(rng, (1, hkv, d))
    vn = rand_bf16(rng, (1, hkv, d))
    pk, pv = empty_pools(2, hkv, d, BS)
    o, lse = oracle.prefill_attention(pk, pv, np.array([[1]], np.int32), [0], [0, 1], q, kn, vn,
                                      0.1, BS)
    for h in range(hq):
        assert np.array_equal(o[0, h], widen(vn[0, h // 2]))
        assert lse[0, h] == pytest.approx(0.1 * float(widen(q[0, h]) @ widen(kn[0, h // 2])),
                                          abs=1e-12)


def test_pi5_zero_query_averages_visible_values():
    rng = np.random.default_rng(8)
    p, n, hq, hkv, d = 19, 6, 4, 2, 64
    c = _paged_prefix_case(rng, p, n, hq, hkv, d)
    qz = np.zeros_like(c["q"])
    o, lse = oracle.prefill_attention(c["pk"], c["pv"], c["table"], [p], [0, n], qz,
                                      c["k_all"][p:], c["v_all"][p:], 0.125, BS)
    v = widen(c["v_all"])
    for j in range(n):
        mean = v[: p + j + 1].mean(axis=0)  # [Hkv][D]
        for h in range(hq):
            assert np.max(np.abs(o[j, h] - mean[h // 2])) <= 1e-12
            assert lse[j, h] == pytest.approx(math.log(p + j + 1), abs=1e-12)


def test_pi5_no_prefix_is_textbook_causal_attention():
    rng = np.random.default_rng(9)
    n, hq, hkv, d = 29, 4, 4, 64
    q = rand_bf16(rng, (n, hq, d))
    k = rand_bf16(rng, (n, hkv, d))
    v = rand_bf16(rng, (n, hkv, d))
    pk, pv = empty_pools(2, hkv, d, BS)
    o, _ = oracle.prefill_attention(pk, pv, np.array([[0, 1]], np.int32), [0], [0, n], q, k, v,
                                    0.125, BS)
    qt = torch.from_numpy(widen(q)).permute(1, 0, 2)[None]
    kt = torch.from_numpy(widen(k)).permute(1, 0, 2)[None]
    vt = torch.from_numpy(widen(v)).permute(1, 0, 2)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True, scale=0.125)
    assert np.max(np.abs(o - ref[0].permute(1, 0, 2).numpy())) <= 1e-12


def test_pi5_prefill_of_one_token_equals_decode():
    rng = np.random.default_rng(10)
    ctx = [3, 16, 47]
    hq, hkv, d = 8, 2, 64
    pk, pv = empty_pools(12, hkv, d, BS)
    tables = np.array([[0, -1, -1, -1], [1, 2, -1, -1], [3, 4, 5, 6]], np.int32)
    for i, c in enumerate(ctx):
        place(pk, pv, tables[i], rand_bf16(rng, (c, hkv, d)), rand_bf16(rng, (c, hkv, d)), BS)
    q = rand_bf16(rng, (3, hq, d))
    kn = rand_bf16(rng, (3, hkv, d))
    vn = rand_bf16(rng, (3, hkv, d))
    od, ld = oracle.decode_attention(pk, pv, tables, ctx, q, kn, vn, 0.125, BS)
    op, lp = oracle.prefill_attention(pk, pv, tables, ctx, [0, 1, 2, 3], q, kn, vn, 0.125, BS)
    assert np.array_equal(od, op) and np.array_equal(ld, lp)


def test_pi6_block_placement_does_not_change_results():
    """Pi6: the same logical data under two different physical placements gives bit-identical
    oracle outputs."""
    rng = np.random.default_rng(12)
    p, n, hq, hkv, d = 50, 20, 4, 2, 64
    c = _paged_prefix_case(rng, p, n, hq, hkv, d, extra_blocks=6)
    o1, l1 = oracle.prefill_attention(c["pk"], c["pv"], c["table"], [p], [0, n], c["q"],
                                      c["k_all"][p:], c["v_all"][p:], 0.125, BS)
    nb = c["pk"].shape[0]
    table2 = np.random.default_rng(99).permutation(nb)[: c["table"].shape[1]].astype(np.int32)
    pk2, pv2 = empty_pools(nb, hkv, d, BS)
    place(pk2, pv2, table2, c["k_all"][:p], c["v_all"][:p], BS)
    assert not np.array_equal(table2, c["table"][0])
    o2, l2 = oracle.prefill_attention(pk2, pv2, table2[None], [p], [0, n], c["q"], c["k_all"][p:],
                                      c["v_all"][p:], 0.125, BS)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_pi7_append_writes_exactly_the_new_slots():
    """Pi7: the append changes exactly T*Hkv*D elements of each pool (the new tokens' slots,
    NaN before), and gathering afterwards returns the cached prefix followed by the new rows."""
    rng = np.random.default_rng(13)
    hkv, d = 2, 64
    prefixes, news = [5, 16, 0, 31], [12, 1, 17, 40]
    num_blocks = 16
    perm = rng.permutation(num_blocks)
    pk, pv = empty_pools(num_blocks, hkv, d, BS)
    tables = np.full((4, 5), -1, np.int32)
    cur = 0
    pre_k, pre_v = [], []
    for i, (p, n) in enumerate(zip(prefixes, news)):
        nb = -(-(p + n) // BS)
        tables[i, :nb] = perm[cur:cur + nb]
        cur += nb
        kk, vv = rand_bf16(rng, (p, hkv, d)), rand_bf16(rng, (p, hkv, d))
        place(pk, pv, tables[i], kk, vv, BS)
        pre_k.append(kk)
        pre_v.append(vv)
    cu = np.concatenate([[0], np.cumsum(news)]).astype(np.int32)
    T = int(cu[-1])
    kn, vn = rand_bf16(rng, (T, hkv, d)), rand_bf16(rng, (T, hkv, d))
    pk2, pv2 = oracle.kv_append(pk, pv, tables, prefixes, cu, kn, vn, BS)
    assert int(np.sum(pk2 != pk)) == T * hkv * d
    assert int(np.sum(pv2 != pv)) == T * hkv * d
    for i, (p, n) in enumerate(zip(prefixes, news)):
        gk, gv = oracle.gather_seq(pk2, pv2, tables[i], p + n, BS)
        assert np.array_equal(gk, np.concatenate([pre_k[i], kn[cu[i]:cu[i + 1]]]))
        assert np.array_equal(gv, np.concatenate([pre_v[i], vn[cu[i]:cu[i + 1]]]))
    # the concatenated gather is the per-sequence gathers in order
    ck, cv = oracle.gather_kv(pk2, pv2, tables, np.add(prefixes, news), BS)
    assert ck.shape[0] == sum(prefixes) + T


def test_pi7_gather_kv_concatenates_sequences_in_order():
    """Pi7 for the multi-sequence gather: sequences of distinct lengths (0, one token, ends
    mid-block, whole blocks, several blocks) are placed into scattered blocks element by
    element by the test-side fixture; row r of the gathered K/V must be token r - start_i of
    sequence i, where start_i is the sum of the earlier lengths -- checked row by row against
    the contiguous tensors the pools were built from. Any other order, a dropped or repeated
    sequence, or a transposed chunk layout fails it."""
    rng = np.random.default_rng(23)
    hkv, d = 3, 64
    lens = [7, 0, 16, 1, 41, 33, 32]
    nblk = [-(-n // BS) for n in lens]
    num_blocks = sum(nblk) + 5
    perm = rng.permutation(num_blocks)
    tables = np.full((len(lens), max(nblk)), -1, np.int32)
    pk, pv = empty_pools(num_blocks, hkv, d, BS)
    cur = 0
    src_k, src_v = [], []
    for i, n in enumerate(lens):
        tables[i, :nblk[i]] = perm[cur:cur + nblk[i]]
        cur += nblk[i]
        kk, vv = rand_bf16(rng, (n, hkv, d)), rand_bf16(rng, (n, hkv, d))
        place(pk, pv, tables[i], kk, vv, BS)
        src_k.append(kk)
        src_v.append(vv)
    ck, cv = oracle.gather_kv(pk, pv, tables, lens, BS)
    assert ck.shape == (sum(lens), hkv, d) and cv.shape == ck.shape
    r = 0
    for i, n in enumerate(lens):
        for t in range(n):
            assert np.array_equal(ck[r], src_k[i][t]), (i, t)
            assert np.array_equal(cv[r], src_v[i][t]), (i, t)
            r += 1
    assert r == ck.shape[0]
    # no NaN canary (an unwritten slot) is gathered
    assert not np.any(ck == 0x7FC0) and not np.any(cv == 0x7FC0)


def test_pi8_kv_footprint_matches_paper():
    """Pi8: 2 * layers * kv_heads * head_dim * 2 bytes reproduces Section 2.2's 112 KB/token,
    84 MB per 750-token tuple and ~70 tuples in ~6 GB."""
    with open(os.path.join(GOLDEN, "kv_footprint.json")) as f:
        g = json.load(f)
    per_tok = oracle.kv_bytes_per_token(g["num_layers"], g["num_kv_heads"], g["head_dim"],
                                        g["bytes_per_element"])
    assert per_tok == g["paper_kb_per_token"] * 1024
    assert per_tok // 1024 * g["paper_tokens_per_tuple"] // 1000 == g["paper_mb_per_tuple"]
    tuples = int(g["paper_kv_space_gb"] * 1024 ** 3 // (per_tok * g["paper_tokens_per_tuple"]))
    assert abs(tuples - g["paper_max_tuples"]) <= 5


@pytest.mark.parametrize("where", ["last_visible", "first_hidden"])
def test_pi9_spike_key_probes_the_mask_boundary(where):
    """Pi9: a key planted parallel to query (j, h) with a large norm dominates that query's
    softmax if and only if it is visible to it (position <= P + j)."""
    rng = np.random.default_rng(14)
    p, n, hq, hkv, d = 20, 8, 4, 2, 64
    c = _paged_prefix_case(rng, p, n, hq, hkv, d)
    j, h = 3, 2
    t_star = p + j if where == "last_visible" else p + j + 1
    k_all = c["k_all"].copy()
    v_all = c["v_all"].copy()
    qj = widen(c["q"][j, h])
    spike = (qj * (40.0 / np.linalg.norm(qj)) * 8.0).astype(np.float32)
    k_all[t_star, h // 2] = (spike.view(np.uint32) >> 16).astype(np.uint16)
    v_all[t_star, h // 2] = np.uint16(0x4120)  # bf16 10.0
    o, _ = oracle.prefill_attention(c["pk"], c["pv"], c["table"], [p], [0, n], c["q"],
                                    k_all[p:], v_all[p:], 1.0 / 8.0, BS)
    if where == "last_visible":
        assert np.max(np.abs(o[j, h] - 10.0)) < 1e-6
    else:
        assert np.max(np.abs(o[j, h])) < 5.0
