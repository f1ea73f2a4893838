"""Execution-strategy arms at matched masks (Sec. 4.4): the copy arm (gather
the selected pages, then attention on contiguous pools) and the block-sparse
arm (each head x Q-block row runs its own mask row), through the C ABI.

The copy arm runs the zero-copy kernel on packed pools, so its output must be
bit-identical to the zero-copy path; the gather itself is checked against the
page-table definition.  Block-sparse tables are compared bit for bit with the
mask rows and the attention with the oracle's per-row execution.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from _helpers import (bf16_host_f64, compare_attention, device_inputs, i32_dev, rows_by_head,
                      sample_rows, u64_dev)

pytestmark = pytest.mark.gpu

ca = pytest.importorskip("paper_2605_16839_amd")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ca.load()


def _csr(masks, w):
    nkb = [w.n_kv_blocks(b) for b in range(w.batch)]
    return oracle.tables_to_csr(oracle.block_tables(masks, w.group_size, nkb))


def _bs_csr(bits, w):
    """CPU block-sparse tables: one row per (b, h, Q-block), set bits j < nKB_b."""
    indptr, indices = [0], []
    for b in range(w.batch):
        nkb = w.n_kv_blocks(b)
        for h in range(w.num_q_heads):
            for i in range(w.n_qblocks):
                row = np.nonzero(bits[b, h, i, :nkb])[0].tolist()
                indices += row
                indptr.append(len(indices))
    return np.array(indptr, dtype=np.int32), np.array(indices, dtype=np.int32)


@pytest.mark.parametrize("name,v_layout", [("tiny_gqa_1k", 0), ("llama8b_32k", 0),
                                           ("batched_ragged_4seq", 0), ("tiny_unaligned", 0),
                                           ("llama8b_unaligned", 0), ("tiny_unaligned", 1),
                                           ("llama8b_32k", 1)])
def test_copy_arm_gather_and_bitexact(name, v_layout, workload_inputs, oracle_estimate):
    """v_layout 0: token-major V pages, 1: transposed (the packed V pool keeps it)."""
    d = workload_inputs(name)
    w = d["workload"]
    p = ca.Problem.from_workload(w, v_layout=v_layout)
    x = device_inputs(d, v_layout)
    masks = d["masks"] if name == "tiny_gqa_1k" else oracle_estimate(name)[0]
    ip, ix = _csr(masks, w)
    tabs = (i32_dev(ip), i32_dev(ix))
    kp, vp = ca.gather_selected_pages(p, (x["k"], x["v"]), x["pt"], tabs, w.group_size)
    torch.cuda.synchronize()
    # the gather against its definition: packed page p = pool page of table entry p
    G = w.num_q_heads // w.group_size
    ratio = w.num_q_heads // w.num_kv_heads
    src = np.empty(ip[-1], dtype=np.int64)
    for r in range(w.batch * G):
        b, g = divmod(r, G)
        kvh = (g * w.group_size) // ratio
        src[ip[r]:ip[r + 1]] = d["page_table"][b, kvh, ix[ip[r]:ip[r + 1]]]
    pick = np.unique(np.linspace(0, ip[-1] - 1, 64).astype(np.int64))
    kh = kp[torch.as_tensor(pick, device="cuda")].view(torch.int16).cpu().numpy()
    vh = vp[torch.as_tensor(pick, device="cuda")].view(torch.int16).cpu().numpy()
    # bit patterns (NaN rows past a sequence end are copied as they are)
    assert np.array_equal(kh.view(np.uint16), d["k_pool"][src[pick]])
    v_want = d["v_pool"][src[pick]]
    if v_layout == 1:
        v_want = synth.v_pages_transposed(v_want)
    assert np.array_equal(vh.view(np.uint16), v_want)
    for splits in (1, 0):
        lse_z = torch.empty((p.batch, p.num_q_heads, p.chunk_len), dtype=torch.float32,
                            device="cuda")
        lse_c = torch.empty_like(lse_z)
        oz, _ = ca.chunk_attention(p, x["q"], (x["k"], x["v"]), x["pt"], tabs, w.group_size,
                                   w.sm_scale, num_splits=splits, lse=lse_z)
        oc, _ = ca.packed_chunk_attention(p, x["q"], (kp, vp), tabs, w.group_size, w.sm_scale,
                                          num_splits=splits, lse=lse_c)
        torch.cuda.synchronize()
        assert torch.equal(oz.view(torch.int16), oc.view(torch.int16))
        assert torch.equal(lse_z, lse_c)


def _union_rows_csr(masks, w):
    """CPU matched-table rows: T[b, g(h)] limited to the blocks Q-block i can see."""
    nkb = [w.n_kv_blocks(b) for b in range(w.batch)]
    T = oracle.block_tables(masks, w.group_size, nkb)
    indptr, indices = [0], []
    for b in range(w.batch):
        for h in range(w.num_q_heads):
            for i in range(w.n_qblocks):
                lim = oracle.causal_block_end(w.cached_lens[b], w.chunk_len, i, w.q_block,
                                              w.page_size)
                indices += [j for j in T[b][h // w.group_size] if j < lim]
                indptr.append(len(indices))
    return np.array(indptr, dtype=np.int32), np.array(indices, dtype=np.int32), T


@pytest.mark.parametrize("name", ["llama8b_32k", "batched_ragged_4seq", "llama8b_unaligned",
                                  "tiny_gqa_1k"])
def test_block_sparse_tables_bitexact(name, workload_inputs, oracle_estimate):
    """tiny_gqa_1k has a single group row (B = 1, one group of 4 heads): the
    per-row words then start at an 8-byte boundary past an odd count array."""
    d = workload_inputs(name)
    w = d["workload"]
    p = ca.Problem.from_workload(w)
    masks = d["masks"] if w.mask_kind == "bernoulli" else oracle_estimate(name)[0]
    ip, ix = ca.build_block_sparse_tables(p, u64_dev(masks))          # raw mask rows
    torch.cuda.synchronize()
    rip, rix = _bs_csr(oracle.unpack_masks(masks), w)
    assert np.array_equal(ip.cpu().numpy(), rip)
    assert np.array_equal(ix.cpu().numpy()[:rip[-1]], rix)
    ip, ix = ca.build_block_sparse_tables(p, u64_dev(masks), w.group_size)   # matched tables
    torch.cuda.synchronize()
    rip, rix, _ = _union_rows_csr(masks, w)
    assert np.array_equal(ip.cpu().numpy(), rip)
    assert np.array_equal(ix.cpu().numpy()[:rip[-1]], rix)


@pytest.mark.parametrize("name", ["llama8b_32k", "batched_ragged_4seq", "llama8b_unaligned"])
def test_block_sparse_matched_tables_attention(name, workload_inputs, oracle_estimate):
    """Block-sparse execution of the unioned tables computes the zero-copy result."""
    d = workload_inputs(name)
    w = d["workload"]
    p = ca.Problem.from_workload(w)
    x = device_inputs(d)
    masks, _ = oracle_estimate(name)
    _, _, T = _union_rows_csr(masks, w)
    tabs = ca.build_block_sparse_tables(p, u64_dev(masks), w.group_size)
    lse = torch.empty((p.batch, p.num_q_heads, p.chunk_len), dtype=torch.float32, device="cuda")
    out, _ = ca.block_sparse_chunk_attention(p, x["q"], (x["k"], x["v"]), x["pt"], tabs,
                                             w.sm_scale, lse=lse)
    torch.cuda.synchronize()
    rows = sample_rows(w.batch, w.num_q_heads, w.chunk_len, seed=w.seed + 9, heads_per_b=2,
                       n_random=8)
    ref = np.full((w.batch, w.chunk_len, w.num_q_heads, w.head_dim), np.nan)
    ref_lse = np.full((w.batch, w.num_q_heads, w.chunk_len), np.nan)
    for (b, h), ts in rows_by_head(rows).items():
        o, l = oracle.chunk_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                      d["cached_len"], T, w.group_size, w.sm_scale,
                                      heads=[(b, h)], queries=ts)
        ref[b, ts, h] = o[b, ts, h]
        ref_lse[b, h, ts] = l[b, h, ts]
    print(name, compare_attention(bf16_host_f64(out), lse.cpu().numpy().astype(np.float64), ref,
                                  ref_lse, rows))


def _bs_oracle_rows(d, bits, sm_scale, rows):
    w = d["workload"]
    ref = np.full((w.batch, w.chunk_len, w.num_q_heads, w.head_dim), np.nan)
    ref_lse = np.full((w.batch, w.num_q_heads, w.chunk_len), np.nan)
    for (b, h), ts in rows_by_head(rows).items():
        o, l = oracle.block_sparse_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                             d["cached_len"], bits, w.q_block, sm_scale,
                                             heads=[(b, h)], queries=ts)
        ref[b, ts, h] = o[b, ts, h]
        ref_lse[b, h, ts] = l[b, h, ts]
    return ref, ref_lse


@pytest.mark.parametrize("name,v_layout", [("llama8b_32k", 0), ("batched_ragged_4seq", 0),
                                           ("llama8b_unaligned", 0), ("llama8b_unaligned", 1)])
def test_block_sparse_attention_sampled(name, v_layout, workload_inputs, oracle_estimate):
    """v_layout 0: token-major V pages, 1: transposed (NaN past each sequence end)."""
    d = workload_inputs(name)
    w = d["workload"]
    p = ca.Problem.from_workload(w, v_layout=v_layout)
    x = device_inputs(d, v_layout)
    masks, _ = oracle_estimate(name)
    bits = oracle.unpack_masks(masks)
    tabs = ca.build_block_sparse_tables(p, u64_dev(masks))
    rows = sample_rows(w.batch, w.num_q_heads, w.chunk_len, seed=w.seed + 7, heads_per_b=2,
                       n_random=8)
    for scale_mult in (1.0, 8.0):
        lse = torch.empty((p.batch, p.num_q_heads, p.chunk_len), dtype=torch.float32,
                          device="cuda")
        out, _ = ca.block_sparse_chunk_attention(p, x["q"], (x["k"], x["v"]), x["pt"], tabs,
                                                 w.sm_scale * scale_mult, lse=lse)
        torch.cuda.synchronize()
        ref, ref_lse = _bs_oracle_rows(d, bits, w.sm_scale * scale_mult, rows)
        print(name, scale_mult,
              compare_attention(bf16_host_f64(out), lse.cpu().numpy().astype(np.float64), ref,
                                ref_lse, rows))


def test_block_sparse_rejects_64_query_blocks(workload_inputs):
    d = workload_inputs("tiny_gqa_1k")
    w = d["workload"]
    p = ca.Problem.from_workload(w)
    x = device_inputs(d)
    tabs = ca.build_block_sparse_tables(p, u64_dev(d["masks"]))
    with pytest.raises(ca.CAError) as e:
        ca.block_sparse_chunk_attention(p, x["q"], (x["k"], x["v"]), x["pt"], tabs, w.sm_scale)
    assert e.value.name == "CA_ERR_UNSUPPORTED"
