"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these checks re-types an oracle formula: each one compares the oracle
with an independent formulation (bitwise integers, torch's fp64 attention on
contiguous K/V, brute-force enumeration, closed forms, invariants).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from synth.gen import pack_bits

HERE = os.path.dirname(os.path.abspath(__file__))


# ---------------------------------------------------------------------------
# tables (Sec. 3.2)
# ---------------------------------------------------------------------------
def _int_tables(masks, group_size, n_blocks):
    """Independent bitwise formulation: OR the raw words as Python ints."""
    B, Hq, nqb, W = masks.shape
    out = []
    for b in range(B):
        per_b = []
        for g in range(Hq // group_size):
            acc = 0
            for h in range(g * group_size, (g + 1) * group_size):
                for i in range(nqb):
                    for w in range(W):
                        acc |= int(masks[b, h, i, w]) << (64 * w)
            acc &= (1 << int(n_blocks[b])) - 1
            per_b.append([j for j in range(int(n_blocks[b])) if (acc >> j) & 1])
        out.append(per_b)
    return out


def test_tables_hand_worked_fixture():
    fx = json.load(open(os.path.join(HERE, "golden", "union_worked_example.json")))
    sel = fx["selected"]
    B, Hq, nqb = len(sel), len(sel[0]), len(sel[0][0])
    bits = np.zeros((B, Hq, nqb, fx["n_blocks"][0]), dtype=bool)
    for b in range(B):
        for h in range(Hq):
            for i in range(nqb):
                bits[b, h, i, sel[b][h][i]] = True
    masks = pack_bits(bits, 1)
    t = oracle.block_tables(masks, fx["group_size"], fx["n_blocks"])
    assert t == fx["expected_tables"]
    # per-head Q-block union = tables with groups of one head
    mbar = oracle.block_tables(masks, 1, fx["n_blocks"])
    assert [[row for row in per_b] for per_b in mbar] == fx["expected_mbar"]
    indptr, indices = oracle.tables_to_csr(t)
    assert indptr.tolist() == fx["expected_kv_indptr"]
    assert indices.tolist() == fx["expected_kv_indices"]


def test_tables_bruteforce_all_tiny_masks():
    """All 2^12 masks for 2 heads x 2 Q-blocks x 3 blocks, groups of 2 and 1."""
    for code in range(1 << 12):
        bits = np.array([(code >> k) & 1 for k in range(12)], dtype=bool).reshape(1, 2, 2, 3)
        masks = pack_bits(bits, 1)
        for gs in (1, 2):
            assert oracle.block_tables(masks, gs, [3]) == _int_tables(masks, gs, [3])


@pytest.mark.parametrize("nkb", [1, 31, 32, 33, 63, 64, 65, 127, 128, 129, 130])
def test_tables_random_word_edges(nkb):
    rng = np.random.default_rng(nkb)
    W = (nkb + 63) // 64 + 1        # one spare word full of garbage beyond nKB
    for density in (0.0, 0.02, 0.3, 1.0):
        raw = rng.integers(0, 2**63, size=(2, 8, 3, W), dtype=np.int64).astype(np.uint64)
        keep = rng.random((2, 8, 3, W * 64)) < density
        masks = pack_bits(keep, W) & raw | pack_bits(keep & (rng.random(keep.shape) < 0.5), W)
        # single bits on word edges
        for j in (0, 31, 32, 63, 64, nkb - 1):
            if 0 <= j < nkb:
                masks[1, 3, 2, j >> 6] |= np.uint64(1) << np.uint64(j & 63)
        n_blocks = [nkb, max(1, nkb // 2)]
        for gs in (1, 2, 4, 8):
            assert oracle.block_tables(masks, gs, n_blocks) == _int_tables(masks, gs, n_blocks)


def test_tables_coverage_and_minimality(workload_inputs):
    """Every selected bit lands in its group's table; every entry has a witness."""
    d = workload_inputs("tiny_gqa_1k")
    w = d["workload"]
    masks = d["masks"]
    nkb = [w.n_kv_blocks(b) for b in range(w.batch)]
    for gs in (1, 2, 4):
        T = oracle.block_tables(masks, gs, nkb)
        B, Hq, nqb, W = masks.shape
        for b in range(B):
            for g in range(Hq // gs):
                witnesses = set()
                for h in range(g * gs, (g + 1) * gs):
                    for i in range(nqb):
                        for j in range(nkb[b]):
                            if (int(masks[b, h, i, j // 64]) >> (j % 64)) & 1:
                                witnesses.add(j)
                                assert j in T[b][g]          # coverage
                assert set(T[b][g]) <= witnesses             # minimality
                assert T[b][g] == sorted(T[b][g])


def test_union_density_monotone(workload_inputs):
    d = workload_inputs("tiny_gqa_1k")
    w = d["workload"]
    dens = oracle.union_densities(d["masks"], 4, [w.n_cached_blocks(0)])
    assert dens["pre_union"] <= dens["q_union"] <= dens["group_union"] <= 1.0
    sub = oracle.union_densities(d["masks"], 2, [w.n_cached_blocks(0)])
    assert sub["group_union"] <= dens["group_union"]


# ---------------------------------------------------------------------------
# attention (Sec. 3.3, App. B.2)
# ---------------------------------------------------------------------------
def _bf16(x):
    return synth.bf16_round(np.asarray(x, dtype=np.float32))


def test_attention_hand_worked():
    """page = 2, D = 2, one cached block + a 2-token chunk; closed-form softmax."""
    e = math.e
    k = _bf16([[[1, 0], [0, 1]], [[1, 1], [0, 0]]])        # logical blocks 0, 1
    v = _bf16([[[1, 0], [0, 1]], [[2, 2], [4, 0]]])
    pt = np.array([[[1, 0]]], dtype=np.int32)               # block 0 -> page 1
    kp, vp = k[::-1].copy(), v[::-1].copy()
    q = _bf16([[[[1, 0]], [[0, 1]]]])                        # [B=1, C=2, Hq=1, D=2]
    out, lse = oracle.chunk_attention(q, kp, vp, pt, [2], [[[0, 1]]], 1, 1.0)
    np.testing.assert_allclose(out[0, 0, 0], [3 * e / (2 * e + 1), (1 + 2 * e) / (2 * e + 1)], rtol=1e-14)
    np.testing.assert_allclose(out[0, 1, 0], [(5 + 2 * e) / (2 * e + 2), 3 * e / (2 * e + 2)], rtol=1e-14)
    np.testing.assert_allclose(lse[0, 0], [math.log(2 * e + 1), math.log(2 * e + 2)], rtol=1e-14)
    # table with the chunk block only: causal masking still uses absolute positions
    out, lse = oracle.chunk_attention(q, kp, vp, pt, [2], [[[1]]], 1, 1.0)
    np.testing.assert_allclose(out[0, 0, 0], [2, 2], rtol=1e-14)
    np.testing.assert_allclose(out[0, 1, 0], [(2 * e + 4) / (e + 1), 2 * e / (e + 1)], rtol=1e-14)
    np.testing.assert_allclose(lse[0, 0], [1.0, math.log(e + 1)], rtol=1e-14)
    # a query that sees nothing: output 0, lse = -inf
    out, lse = oracle.chunk_attention(q, kp, vp, pt, [0], [[[1]]], 1, 1.0)
    assert np.all(out[0, 0, 0] == 0) and lse[0, 0, 0] == -np.inf
    # one cached token + the 2-token chunk: the sequence ends inside block 1,
    # whose second row (position 3) is not part of it and holds NaN
    kp2, vp2 = kp.copy(), vp.copy()
    kp2[0, 1, :] = 0x7FC0
    vp2[0, 1, :] = 0x7FC0
    out, lse = oracle.chunk_attention(q, kp2, vp2, pt, [1], [[[0, 1]]], 1, 1.0)
    np.testing.assert_allclose(out[0, 0, 0], [e / (e + 1), 1 / (e + 1)], rtol=1e-14)
    np.testing.assert_allclose(out[0, 1, 0], [1.0, 3 * e / (2 * e + 1)], rtol=1e-14)
    np.testing.assert_allclose(lse[0, 0], [math.log(e + 1), math.log(2 * e + 1)], rtol=1e-14)


def _contiguous_kv(d, b, kvh, nkb, seq_len=None):
    """The sequence's keys and values as contiguous [seq_len, D] tensors."""
    pt = d["page_table"][b, kvh, :nkb]
    K = oracle.bf16_to_f64(d["k_pool"][pt]).reshape(nkb * d["k_pool"].shape[1], -1)
    V = oracle.bf16_to_f64(d["v_pool"][pt]).reshape(nkb * d["v_pool"].shape[1], -1)
    if seq_len is not None:
        K, V = K[:seq_len], V[:seq_len]
    return torch.from_numpy(K), torch.from_numpy(V)


def _sdpa_ref(d, b, h, queries, keep_blocks=None):
    """torch fp64 SDPA over contiguous, unpaged K/V with an explicit mask."""
    w = d["workload"]
    ratio = w.num_q_heads // w.num_kv_heads
    nkb = w.n_kv_blocks(b)
    K, V = _contiguous_kv(d, b, h // ratio, nkb, w.seq_len(b))
    q = torch.from_numpy(oracle.bf16_to_f64(d["q"][b, queries, h, :]))
    kpos = torch.arange(w.seq_len(b))
    qpos = torch.as_tensor(w.cached_lens[b] + np.asarray(queries))
    allow = kpos[None, :] <= qpos[:, None]
    if keep_blocks is not None:
        kb = torch.zeros(nkb, dtype=torch.bool)
        kb[list(keep_blocks)] = True
        allow &= kb.repeat_interleave(w.page_size)[None, :w.seq_len(b)]
    o = torch.nn.functional.scaled_dot_product_attention(
        q[None, None], K[None, None], V[None, None], attn_mask=allow[None, None],
        scale=w.sm_scale)
    return o[0, 0].numpy()


def test_all_open_equals_dense_sdpa_tiny(workload_inputs):
    d = workload_inputs("tiny_gqa_1k")
    w = d["workload"]
    ones = np.full_like(d["masks"], np.uint64(0xFFFFFFFFFFFFFFFF))
    nkb = [w.n_kv_blocks(0)]
    T = oracle.block_tables(ones, 4, nkb)
    assert T == oracle.dense_tables(nkb, 1)
    out, lse = oracle.chunk_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                      d["cached_len"], T, 4, w.sm_scale)
    for h in range(4):
        ref = _sdpa_ref(d, 0, h, np.arange(w.chunk_len))
        np.testing.assert_allclose(out[0, :, h, :], ref, atol=1e-12, rtol=0)


def test_all_open_equals_dense_sdpa_32k_sampled(workload_inputs):
    d = workload_inputs("llama8b_32k")
    w = d["workload"]
    nkb = [w.n_kv_blocks(0)]
    T = oracle.dense_tables(nkb, w.num_groups)
    qs = np.array([0, 1, 63, 64, 1000, 2047])
    heads = [(0, 0), (0, 13), (0, 31)]
    out, _ = oracle.chunk_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                    d["cached_len"], T, w.group_size, w.sm_scale,
                                    heads=heads, queries=qs)
    for (_, h) in heads:
        np.testing.assert_allclose(out[0, qs, h, :], _sdpa_ref(d, 0, h, qs), atol=1e-12, rtol=0)


def test_no_cache_is_textbook_causal():
    """cached_len = 0 (first chunk): plain causal self-attention."""
    w = synth.get_workload("tiny_gqa_1k", cached_lens=(0,), max_kv_blocks=4)
    d = synth.make_inputs(w)
    T = oracle.block_tables(d["masks"], 4, [4])
    assert T == [[[0, 1, 2, 3]]]
    out, _ = oracle.chunk_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                    d["cached_len"], T, 4, w.sm_scale)
    K, V = _contiguous_kv(d, 0, 0, 4)
    for h in range(4):
        q = torch.from_numpy(oracle.bf16_to_f64(d["q"][0, :, h, :]))
        ref = torch.nn.functional.scaled_dot_product_attention(
            q[None, None], K[None, None], V[None, None], is_causal=True, scale=w.sm_scale)[0, 0]
        np.testing.assert_allclose(out[0, :, h, :], ref.numpy(), atol=1e-12, rtol=0)


def test_gathered_equals_masked_dense(workload_inputs):
    """Attention over gathered T[b,g] == dense attention with unselected blocks masked."""
    d = workload_inputs("tiny_gqa_1k")
    w = d["workload"]
    nc = w.n_cached_blocks(0)
    masks = synth.random_masks(11, 1, 4, w.n_qblocks, w.q_block, w.page_size,
                               [w.cached_lens[0]],
                               w.chunk_len, w.words, 0.04)
    for gs in (1, 2):
        T = oracle.block_tables(masks, gs, [w.n_kv_blocks(0)])
        out, _ = oracle.chunk_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                        d["cached_len"], T, gs, w.sm_scale)
        for h in range(4):
            assert len(T[0][h // gs]) < w.n_kv_blocks(0)      # genuinely sparse
            ref = _sdpa_ref(d, 0, h, np.arange(w.chunk_len), keep_blocks=T[0][h // gs])
            np.testing.assert_allclose(out[0, :, h, :], ref, atol=1e-12, rtol=0)


def test_page_permutation_invariance(workload_inputs):
    d = workload_inputs("tiny_gqa_1k")
    w = d["workload"]
    T = oracle.block_tables(d["masks"], 4, [w.n_kv_blocks(0)])
    base, lb = oracle.chunk_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                      d["cached_len"], T, 4, w.sm_scale)
    pi = np.random.default_rng(0).permutation(d["k_pool"].shape[0])
    kp = np.empty_like(d["k_pool"]); kp[pi] = d["k_pool"]
    vp = np.empty_like(d["v_pool"]); vp[pi] = d["v_pool"]
    pt = d["page_table"].copy()
    pt[pt >= 0] = pi[pt[pt >= 0]]
    out, lse = oracle.chunk_attention(d["q"], kp, vp, pt, d["cached_len"], T, 4, w.sm_scale)
    assert np.array_equal(out, base) and np.array_equal(lse, lb)


def test_block_sparse_rows_equal_masked_sdpa(workload_inputs):
    """Block-sparse arm: each (head, Q-block) row == torch fp64 SDPA with only
    that row's mask blocks open (independent of the gather/table code)."""
    d = workload_inputs("tiny_gqa_1k")
    w = d["workload"]
    nc = w.n_cached_blocks(0)
    masks = synth.random_masks(13, 1, 4, w.n_qblocks, w.q_block, w.page_size,
                               [w.cached_lens[0]],
                               w.chunk_len, w.words, 0.1)
    bits = oracle.unpack_masks(masks)
    out, lse = oracle.block_sparse_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                             d["cached_len"], bits, w.q_block, w.sm_scale)
    assert np.isfinite(lse).all()
    distinct = 0
    for h in range(4):
        for i in range(w.n_qblocks):
            keep = [j for j in range(w.n_kv_blocks(0)) if bits[0, h, i, j]]
            qs = np.arange(i * w.q_block, (i + 1) * w.q_block)
            ref = _sdpa_ref(d, 0, h, qs, keep_blocks=keep)
            np.testing.assert_allclose(out[0, qs, h, :], ref, atol=1e-12, rtol=0)
            distinct += keep != [j for j in range(w.n_kv_blocks(0)) if bits[0, 0, 0, j]]
    assert distinct > 0      # rows really differ from each other


def test_block_sparse_group_uniform_rows_equal_union(workload_inputs):
    """When every (head, Q-block) row of a group selects the same cached blocks,
    per-row execution and the group-union table give the same attention (the
    extra chunk blocks of the union are causally invisible)."""
    d = workload_inputs("tiny_gqa_1k")
    w = d["workload"]
    nc = w.n_cached_blocks(0)
    one = synth.random_masks(17, 1, 1, 1, w.q_block, w.page_size, [w.cached_lens[0]],
                             w.chunk_len, w.words, 0.2)
    sel = oracle.unpack_masks(one)[0, 0, 0, :nc]
    nkb = w.n_kv_blocks(0)
    bits = np.zeros((1, 4, w.n_qblocks, 64 * w.words), dtype=bool)
    for i in range(w.n_qblocks):
        bits[0, :, i, :nc] = sel
        last = nc + (i + 1) * w.q_block // w.page_size       # chunk-causal bits of Q-block i
        bits[0, :, i, nc:last] = True
    T = [[sorted(set(np.nonzero(sel)[0].tolist()) | set(range(nc, nkb)))]]
    bs, bl = oracle.block_sparse_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                           d["cached_len"], bits, w.q_block, w.sm_scale)
    un, ul = oracle.chunk_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                    d["cached_len"], T, 4, w.sm_scale)
    np.testing.assert_allclose(bs, un, atol=1e-12, rtol=0)
    np.testing.assert_allclose(bl, ul, atol=1e-12, rtol=0)


# ---------------------------------------------------------------------------
# estimator (the selector reading; see oracle/estimator.py)
# ---------------------------------------------------------------------------
def test_block_means_closed_form():
    """Q rows t -> Q-block means i*qb + (qb-1)/2; K rows r + d -> 31.5 + d (via pages)."""
    C, Hq, D, qb = 256, 2, 4, 64
    q = _bf16(np.broadcast_to(np.arange(C, dtype=np.float32)[None, :, None, None], (1, C, Hq, D)))
    qm = oracle.q_block_means(q, qb)
    for i in range(C // qb):
        assert np.all(qm[0, :, i, :] == i * qb + (qb - 1) / 2)
    page = np.arange(64, dtype=np.float32)[:, None] + np.arange(D, dtype=np.float32)[None, :]
    pool = np.stack([_bf16(page + 60 * p) for p in range(3)])      # page p offset 60p (exact in bf16)
    pt = np.array([[[2, 0, 1]]], dtype=np.int32)
    km = oracle.k_block_means(pool, pt, [3])
    for j, p in enumerate([2, 0, 1]):
        np.testing.assert_array_equal(km[0, 0, j], 31.5 + np.arange(D) + 60 * p)
    # a sequence ending 10 rows into block 2: that block's mean is over rows 0..9
    km = oracle.k_block_means(pool, pt, [3], seq_len=[2 * 64 + 10])
    np.testing.assert_array_equal(km[0, 0, 2], 4.5 + np.arange(D) + 60 * 1)
    np.testing.assert_array_equal(km[0, 0, 0], 31.5 + np.arange(D) + 60 * 2)
    # a chunk of 200 rows in Q-blocks of 64: four blocks, the last of rows 192..199
    q = _bf16(np.broadcast_to(np.arange(200, dtype=np.float32)[None, :, None, None],
                              (1, 200, Hq, D)))
    qm = oracle.q_block_means(q, qb)
    assert qm.shape == (1, Hq, 4, D)
    assert np.all(qm[0, :, 3, :] == 195.5) and np.all(qm[0, :, 2, :] == 128 + 31.5)


def test_block_scores_index_mapping():
    """One-hot pooled queries pick one coordinate of the right KV head's block means."""
    B, Hq, nqb, D, Hkv, nkb = 2, 4, 3, 8, 2, 5
    qm = np.zeros((B, Hq, nqb, D))
    km = np.random.default_rng(1).standard_normal((B, Hkv, nkb + 2, D))
    for b in range(B):
        for h in range(Hq):
            for i in range(nqb):
                qm[b, h, i, (b + 2 * h + 3 * i) % D] = 1.0
    sc = oracle.block_scores(qm, km, [nkb, nkb - 2])
    for b in range(B):
        assert sc[b].shape == (Hq, nqb, [nkb, nkb - 2][b])
        for h in range(Hq):
            for i in range(nqb):
                a = (b + 2 * h + 3 * i) % D
                np.testing.assert_array_equal(sc[b][h, i], km[b, h // 2, :sc[b].shape[2], a])


def _brute_topk(vals, k):
    """The unique k-subset whose members all beat all non-members (score desc, index asc)."""
    n = len(vals)
    beats = lambda a, b: (vals[a] > vals[b]) or (vals[a] == vals[b] and a < b)
    found = [s for s in itertools.combinations(range(n), k)
             if all(beats(a, b) for a in s for b in range(n) if b not in s)]
    assert len(found) == 1
    return list(found[0])


def test_topk_bruteforce_with_ties():
    s = synth.tied_scores(0, 60, 9, n_distinct=4)
    for r in range(s.shape[0]):
        for k in range(0, 10):
            got = oracle.select_top_blocks(s[r], k).tolist()
            assert got == _brute_topk(s[r].tolist(), k)


def test_topk_signed_zero_ties():
    s = np.array([0.0, -0.0, 0.0, -1.0, -0.0], dtype=np.float32)
    assert oracle.select_top_blocks(s, 3).tolist() == [0, 1, 2]
    s = np.array([-0.0, 0.0, -1.0], dtype=np.float32)
    assert oracle.select_top_blocks(s, 1).tolist() == [0]


def test_estimator_hand_built_case():
    """Pooled scores ranked by construction; sink, local window and causal bits by hand."""
    D, page, qb, C = 4, 64, 64, 128
    nc = 10
    # K block j has every row equal to (j%5 - 2) * e0  -> k_mean[j] = (j%5-2) e0
    kvals = [(j % 5) - 2 for j in range(nc + C // page)]
    pool = np.stack([_bf16(np.tile(np.array([v, 0, 0, 0], np.float32), (page, 1))) for v in kvals])
    pt = np.arange(len(kvals), dtype=np.int32)[None, None, :]
    q = _bf16(np.tile(np.array([1, 0, 0, 0], np.float32), (1, C, 1, 1)))   # q_mean = e0
    masks = oracle.estimate_masks(q, pool, pt, [nc * page], page, qb, C, 1,
                                  oracle.EstimatorParams(top_frac=0.25, sink_blocks=1, local_blocks=2))
    # scores over cached blocks: j%5-2 -> best are j=4, 9 (score 2) then j=3 (1); k = ceil(2.5) = 3
    sel = {4, 9, 3} | {0} | {8, 9}
    for i, causal in enumerate([{10}, {10, 11}]):
        want = sum(1 << j for j in sel | causal)
        assert int(masks[0, 0, i, 0]) == want


def test_estimator_hand_built_unaligned():
    """Block 10 holds the last 5 cached tokens and the first 59 of the chunk: it is a
    chunk block (open for every Q-block, never a top-k candidate); the 100-token
    chunk ends 41 rows into block 11; Q-block 1 holds 36 rows."""
    D, page, qb, C = 4, 64, 64, 100
    cl = 10 * page + 5
    nkb = oracle.n_kv_blocks(cl, C, page)
    assert nkb == 12
    kvals = [(j % 5) - 2 for j in range(nkb)]
    kvals[10] = 50                        # would win every top-k if it were a candidate
    pool = np.stack([_bf16(np.tile(np.array([v, 0, 0, 0], np.float32), (page, 1))) for v in kvals])
    pt = np.arange(nkb, dtype=np.int32)[None, None, :]
    q = _bf16(np.tile(np.array([1, 0, 0, 0], np.float32), (1, C, 1, 1)))
    masks = oracle.estimate_masks(q, pool, pt, [cl], page, qb, C, 1,
                                  oracle.EstimatorParams(top_frac=0.25, sink_blocks=1, local_blocks=2))
    assert masks.shape == (1, 1, 2, 1)
    sel = {4, 9, 3} | {0} | {8, 9}
    for i in range(2):
        assert int(masks[0, 0, i, 0]) == sum(1 << j for j in sel | {10, 11})


def test_unaligned_causal_bits_bruteforce(oracle_estimate, workload_inputs):
    """Chunk bits (j >= nC) of every mask row = the blocks, other than full cached
    ones, that hold a key some query of the Q-block may see, enumerated key by key;
    the cached bits hold between k and k + sink + local blocks."""
    name = "tiny_unaligned"
    d = workload_inputs(name)
    w = d["workload"]
    masks, _ = oracle_estimate(name)
    bits = oracle.unpack_masks(masks)
    assert w.n_qblocks == 4 and [w.n_kv_blocks(b) for b in range(3)] == [19, 4, 4]
    for b in range(w.batch):
        cl = w.cached_lens[b]
        nc = cl // w.page_size
        k = oracle.n_selected(w.top_frac, nc)
        for i in range(w.n_qblocks):
            want = set()
            for t in range(i * w.q_block, min((i + 1) * w.q_block, w.chunk_len)):
                for pos in range(cl + t + 1):
                    if pos // w.page_size >= nc:
                        want.add(pos // w.page_size)
            for h in range(w.num_q_heads):
                row = bits[b, h, i]
                assert set(np.nonzero(row[nc:])[0] + nc) == want
                cnt = int(row[:nc].sum())
                assert k <= cnt <= k + min(w.sink_blocks + w.local_blocks, nc)


def test_unaligned_all_open_equals_dense_sdpa(workload_inputs):
    """All-ones masks on sequences of 1000, 37 and 0 cached tokens + a 200-token
    chunk, NaN in every K/V row past each sequence end: the oracle equals torch's
    fp64 attention over the contiguous sequence, and no NaN gets through."""
    d = workload_inputs("tiny_unaligned")
    w = d["workload"]
    nkb = [w.n_kv_blocks(b) for b in range(w.batch)]
    ones = np.full((w.batch, w.num_q_heads, w.n_qblocks, w.words),
                   np.uint64(0xFFFFFFFFFFFFFFFF))
    T = oracle.block_tables(ones, w.group_size, nkb)
    assert T == oracle.dense_tables(nkb, w.num_groups)
    out, lse = oracle.chunk_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                      d["cached_len"], T, w.group_size, w.sm_scale)
    assert np.isfinite(out).all() and np.isfinite(lse).all()
    for b in range(w.batch):
        for h in range(w.num_q_heads):
            ref = _sdpa_ref(d, b, h, np.arange(w.chunk_len))
            np.testing.assert_allclose(out[b, :, h, :], ref, atol=1e-12, rtol=0)


def test_unaligned_block_sparse_rows_equal_masked_sdpa(workload_inputs):
    """Block-sparse execution of the estimator's raw mask rows on unaligned lengths
    == masked fp64 SDPA with that row's blocks open (partial last Q-block and page)."""
    d = workload_inputs("tiny_unaligned")
    w = d["workload"]
    masks = oracle.estimate_masks(d["q"], d["k_pool"], d["page_table"], d["cached_len"],
                                  w.page_size, w.q_block, w.chunk_len, w.words,
                                  oracle.EstimatorParams(w.top_frac, w.sink_blocks,
                                                         w.local_blocks))
    bits = oracle.unpack_masks(masks)
    out, _ = oracle.block_sparse_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                           d["cached_len"], bits, w.q_block, w.sm_scale)
    assert np.isfinite(out).all()
    for b in range(w.batch):
        for h in (0, 5):
            for i in range(w.n_qblocks):
                t = np.arange(i * w.q_block, min((i + 1) * w.q_block, w.chunk_len))
                keep = [j for j in range(w.n_kv_blocks(b)) if bits[b, h, i, j]]
                ref = _sdpa_ref(d, b, h, t, keep_blocks=keep)
                np.testing.assert_allclose(out[b, t, h, :], ref, atol=1e-12, rtol=0)


def test_estimator_recall_and_popcount(oracle_estimate, workload_inputs):
    """Needles are always selected by their target row; per-row cached popcount in [k, k+5]."""
    for name in ("llama8b_32k",):
        d = workload_inputs(name)
        w = d["workload"]
        masks, _ = oracle_estimate(name)
        bits = oracle.unpack_masks(masks)
        nc = w.n_cached_blocks(0)
        k = {480: 48}[nc]                 # top 10% of 480 cached blocks
        assert len(d["needles"]) == w.num_kv_heads * w.needles_per_kv_head
        for (b, kvh, j, h, i) in d["needles"]:
            assert bits[b, h, i, j]
        cnt = bits[0, :, :, :nc].sum(axis=-1)
        assert cnt.min() >= k and cnt.max() <= k + w.sink_blocks + w.local_blocks
        # whole chunk open after the Q-block union, causal staircase before it
        for i in range(w.n_qblocks):
            stair = bits[0, :, i, nc:w.n_kv_blocks(0)]
            assert stair[:, :(i + 1) * w.q_block // w.page_size].all()
            assert not stair[:, (i + 1) * w.q_block // w.page_size:].any()
        dens = oracle.union_densities(masks, w.group_size, [nc])
        assert dens["pre_union"] <= dens["q_union"] <= dens["group_union"]


# ---------------------------------------------------------------------------
# alpha-threshold selector (a reading; see oracle/estimator.py)
# ---------------------------------------------------------------------------
def test_threshold_selection_is_a_topk_prefix():
    """With distinct scores the kept set is the top-m set for m = its size, so it
    must equal the independent top-k selection at that k; it grows as the
    margin falls, keeps the maximum, and the limits are argmax / everything."""
    rng = np.random.default_rng(21)
    for n in (1, 2, 17, 64, 300):
        s = rng.standard_normal(n).astype(np.float32)
        s[rng.integers(n)] = s.max() + np.float32(1.0)         # a clear maximum
        prev = None
        for margin in (0.0, -0.01, -0.3, -1.0, -3.0, -np.inf):
            kept = oracle.select_threshold_blocks(s, np.float32(margin))
            assert s.argmax() in kept
            assert np.array_equal(kept, oracle.select_top_blocks(s, len(kept)))
            if prev is not None:
                assert set(prev) <= set(kept.tolist())
            prev = kept.tolist()
        assert prev == list(range(n))                          # -inf keeps every block
        assert oracle.select_threshold_blocks(s, np.float32(0.0)).tolist() == [int(s.argmax())]
    ties = np.array([1.0, 3.0, 3.0, -0.0, 0.0], dtype=np.float32)
    assert oracle.select_threshold_blocks(ties, np.float32(0.0)).tolist() == [1, 2]
    assert oracle.select_threshold_blocks(ties, np.float32(-3.0)).tolist() == [0, 1, 2, 3, 4]


def test_threshold_margin_matches_alpha_weight():
    """exp(temperature * sm_scale * margin) recovers alpha (the reading's definition)."""
    for alpha in (0.01, 0.06, 0.5):
        for tau in (1.0, 16.0):
            m = oracle.threshold_margin(alpha, tau, 1.0 / math.sqrt(128.0))
            assert m <= 0
            assert abs(math.exp(tau * float(m) / math.sqrt(128.0)) - alpha) < 1e-5 * alpha



def test_threshold_kept_blocks_are_the_alpha_heavy_softmax_blocks():
    """Through the softmax of the sharpened block scores (scipy), a block passes
    when its probability is at least alpha times the largest one; checked on
    every block not within 1e-4 (relative) of the cut."""
    from scipy.special import softmax
    rng = np.random.default_rng(23)
    sm = 1.0 / math.sqrt(128.0)
    for alpha, tau in ((0.01, 16.0), (0.06, 16.0), (0.3, 4.0), (0.9, 1.0)):
        s = (rng.standard_normal(500) * 3.0).astype(np.float32)
        kept = set(oracle.select_threshold_blocks(
            s, oracle.threshold_margin(alpha, tau, sm)).tolist())
        prob = softmax(tau * sm * s.astype(np.float64))
        ratio = prob / prob.max()
        clear = np.abs(ratio - alpha) > 1e-4 * alpha
        assert clear.sum() > 450
        want = set(np.nonzero((ratio >= alpha) & clear)[0].tolist())
        assert {j for j in kept if clear[j]} == want
        assert 0 < len(want) < 500


def _bits(word) -> set:
    w = int(word)
    return {j for j in range(64) if (w >> j) & 1}


def test_threshold_masks_hand_built_case():
    """masks_from_threshold on hand-picked float32 scores (10 cached blocks, a
    128-token chunk of two 64-query Q-blocks, margin -0.75, one sink block, a
    2-block local window); the kept blocks and the forced bits worked out by
    hand: the kept set is {j : s_j >= max + margin} (ties at the cut and at the
    maximum kept, -0.0 equal to +0.0), then the sink {0}, the local window
    {8, 9} and the chunk-causal blocks {10} (Q-block 0) or {10, 11} (Q-block 1)."""
    f = lambda *v: np.array(v, dtype=np.float32)
    s = np.zeros((2, 2, 10), dtype=np.float32)
    s[0, 0] = f(0, 1, 5, 2, 4.5, 0, 3, 5, 1, 0)                 # max 5, cut 4.25
    s[0, 1] = f(-1, -0.5, -0.5, -4, -1.25, -2, -3, -1.5, -9, -1.0)   # cut -1.25, kept exactly
    s[1, 0] = np.full(10, 7.0, dtype=np.float32)                  # all tie at the maximum
    s[1, 1] = f(-0.0, 0.0, -5, -5, -5, -5, -5, -5, -5, -5)        # signed zeros at the maximum
    masks = oracle.masks_from_threshold([s], [640], 128, 64, 64, 1, np.float32(-0.75),
                                        sink_blocks=1, local_blocks=2)
    assert masks.shape == (1, 2, 2, 1)
    want = {(0, 0): {0, 2, 4, 7, 8, 9, 10},
            (0, 1): {0, 1, 2, 4, 8, 9, 10, 11},
            (1, 0): set(range(11)),
            (1, 1): {0, 1, 8, 9, 10, 11}}
    for (h, i), bits in want.items():
        assert _bits(masks[0, h, i, 0]) == bits, (h, i)


def test_threshold_masks_hand_built_unaligned():
    """Three sequences with a 100-token chunk (Q-block 1 holds 36 queries):
    340 cached tokens (5 full cached blocks; block 5 holds the last 20 cached
    and the first 44 chunk tokens, so it is a chunk block, never a candidate),
    an empty cache, and 63 cached tokens (no full cached block; block 0 is
    shared).  Local window 3, sink 1, margin -0.75; every bit by hand."""
    f = lambda *v: np.array(v, dtype=np.float32)
    s0 = np.stack([f(1, 2, 3, 2.5, 0), f(9, 0, 0, 0, 0)])[None]  # [Hq=1, nQB=2, nC=5]
    empty = np.zeros((1, 2, 0), dtype=np.float32)
    masks = oracle.masks_from_threshold([s0, empty, empty], [340, 0, 63], 100, 64, 64, 1,
                                        np.float32(-0.75), sink_blocks=1, local_blocks=3)
    assert masks.shape == (3, 1, 2, 1)
    # b = 0: kept {2, 3} / {0}; sink {0}; local {2, 3, 4}; chunk blocks 5, 6 for both
    # Q-blocks (positions 340..403 and 404..439 end in block 6)
    assert _bits(masks[0, 0, 0, 0]) == {0, 2, 3, 4, 5, 6}
    assert _bits(masks[0, 0, 1, 0]) == {0, 2, 3, 4, 5, 6}
    # b = 1: no cache: Q-block 0 (positions 0..63) sees block 0, Q-block 1 (64..99) 0..1
    assert _bits(masks[1, 0, 0, 0]) == {0}
    assert _bits(masks[1, 0, 1, 0]) == {0, 1}
    # b = 2: 63 cached tokens: positions 63..126 -> blocks 0..1, 127..162 -> 0..2
    assert _bits(masks[2, 0, 0, 0]) == {0, 1}
    assert _bits(masks[2, 0, 1, 0]) == {0, 1, 2}


def test_union_densities_hand_built():
    """Densities of cached blocks before and after each union, worked out by hand.

    One sequence with nC = 4 cached blocks, 4 heads x 2 Q-blocks, groups of 2
    heads.  Kept cached blocks per (head, Q-block): h0 {0} {1}, h1 {0} {0},
    h2 {3} {}, h3 {2, 3} {2}; every row also holds chunk block 5, which no
    density counts.  Pre-union: 8 of 32 = 0.25.  Q-block union per head:
    {0,1} {0} {3} {2,3} = 6 of 16 = 0.375.  Group union: {0,1} {2,3} = 4 of 8
    = 0.5.  A second sequence with no cached block is left out of every mean."""
    rows = {(0, 0): [0], (0, 1): [1], (1, 0): [0], (1, 1): [0], (2, 0): [3], (2, 1): [],
            (3, 0): [2, 3], (3, 1): [2]}
    masks = np.zeros((2, 4, 2, 1), dtype=np.uint64)
    for (h, i), js in rows.items():
        for j in js + [5]:
            masks[0, h, i, 0] |= np.uint64(1) << np.uint64(j)
    masks[1, :, :, 0] = np.uint64(0b111)       # nC = 0: chunk blocks only
    dens = oracle.union_densities(masks, 2, [4, 0])
    assert dens == {"pre_union": 0.25, "q_union": 0.375, "group_union": 0.5}
    # groups of 4 heads: one group {0, 1, 2, 3} = 4 of 4
    assert oracle.union_densities(masks, 4, [4, 0])["group_union"] == 1.0
    # group size 1: the group union is the Q-block union
    assert oracle.union_densities(masks, 1, [4, 0])["group_union"] == 0.375
