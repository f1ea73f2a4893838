"""The debug library (libcompactattn_debug.so, built with CA_DEBUG_CHECKS):
every attention call checks its tables and the page ids they reach before
launching.  On valid inputs its outputs equal the release library's bit for
bit; a malformed table is refused with CA_ERR_INVALID_TABLE before any launch.

The malformed cases here would read only valid pages even if they reached the
kernel (two entries swapped; an entry past the sequence, which the kernel drops
as past every tile's last visible block).  Out-of-range page ids are covered by
the host check's CPU tests (test_abi.py)."""
import os

import numpy as np
import pytest
import torch

import oracle
from _helpers import V_TRANSPOSED, device_inputs, i32_dev, u64_dev

pytestmark = pytest.mark.gpu

ca = pytest.importorskip("paper_2605_16839_amd")
from paper_2605_16839_amd import binding as B  # noqa: E402


@pytest.fixture(scope="module")
def dbg():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ca.load()
    if not os.path.exists(ca.DEBUG_LIB_PATH):
        pytest.fail("libcompactattn_debug.so is not built (run __graft_entry__.build())")
    return ca.load(ca.DEBUG_LIB_PATH)


def _tables(d, masks):
    w = d["workload"]
    nkb = [w.n_kv_blocks(b) for b in range(w.batch)]
    return oracle.tables_to_csr(oracle.block_tables(masks, w.group_size, nkb))


def _run(lib, p, x, ip, ix, w, dense=False, v=None):
    out = torch.empty_like(x["q"])
    lse = torch.empty((p.batch, p.num_q_heads, p.chunk_len), dtype=torch.float32, device="cuda")
    ws = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
    v = x["v"] if v is None else v
    P = B._ptr
    if dense:
        st = lib.ca_dense_paged_chunk_attention(p.ref, P(x["q"]), P(x["k"]), P(v), P(x["pt"]),
                                                w.sm_scale, 0, P(out), P(lse), P(ws), ws.numel(),
                                                B._stream(None))
    else:
        st = lib.ca_chunk_attention(p.ref, P(x["q"]), P(x["k"]), P(v), P(x["pt"]), P(ip), P(ix),
                                    w.group_size, w.sm_scale, 0, P(out), P(lse), P(ws),
                                    ws.numel(), B._stream(None))
    torch.cuda.synchronize()
    return st, out, lse


@pytest.mark.parametrize("name", ["tiny_gqa_1k", "llama8b_unaligned"])
def test_debug_library_matches_release(dbg, name, workload_inputs, oracle_estimate):
    d = workload_inputs(name)
    w = d["workload"]
    masks = d["masks"] if w.mask_kind == "bernoulli" else oracle_estimate(name)[0]
    ip, ix = _tables(d, masks)
    rel = ca.load()
    for v_layout in (0, V_TRANSPOSED):
        p = ca.Problem.from_workload(w, v_layout=v_layout)
        x = device_inputs(d, v_layout)
        tabs = (i32_dev(ip), i32_dev(np.concatenate([ix, np.zeros(1, np.int32)])))
        for dense in (False, True):
            s0, o0, l0 = _run(rel, p, x, *tabs, w, dense)
            s1, o1, l1 = _run(dbg, p, x, *tabs, w, dense)
            assert s0 == 0 and s1 == 0, (s0, s1, dbg.ca_last_error_detail())
            assert torch.equal(o0.view(torch.int16), o1.view(torch.int16))
            assert torch.equal(l0, l1)


def test_debug_library_refuses_malformed_tables(dbg, workload_inputs):
    d = workload_inputs("tiny_gqa_1k")
    w = d["workload"]
    p = ca.Problem.from_workload(w)
    x = device_inputs(d)
    ip, ix = _tables(d, d["masks"])
    assert ip[1] - ip[0] >= 3
    # two entries of row 0 swapped
    bad = ix.copy()
    bad[1], bad[2] = bad[2], bad[1]
    st, _, _ = _run(dbg, p, x, i32_dev(ip), i32_dev(bad), w)
    assert st == 7, st
    assert "row 0" in dbg.ca_last_error_detail().decode()
    # one more entry at the end of row 0: block nKB_0, past the sequence (a page
    # table with one spare column, pointing at page 0)
    nkb = w.n_kv_blocks(0)
    p2 = ca.Problem(w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.q_block,
                    w.chunk_len, w.max_kv_blocks + 1, list(w.cached_lens))
    pt2 = np.concatenate([d["page_table"], np.zeros(d["page_table"].shape[:2] + (1,), np.int32)],
                         axis=2)
    x2 = dict(x, pt=i32_dev(pt2))
    ip2 = ip.copy()
    ip2[1:] += 1
    ix2 = np.concatenate([ix[:ip[1]], [nkb], ix[ip[1]:]]).astype(np.int32)
    st, _, _ = _run(dbg, p2, x2, i32_dev(ip2), i32_dev(ix2), w)
    assert st == 7, st
    assert "nKB" in dbg.ca_last_error_detail().decode()
    st, _, _ = _run(dbg, p2, x2, i32_dev(ip), i32_dev(ix), w)     # the valid tables pass
    assert st == 0, dbg.ca_last_error_detail()
    # the release library does not check (it trusts the tables): only the debug one refuses
    st, _, _ = _run(ca.load(), p, x, i32_dev(ip), i32_dev(bad), w)
    assert st == 0


def test_debug_library_block_sparse_and_packed(dbg, workload_inputs, oracle_estimate):
    """The two other table layouts through the debug checks: equal to the release library."""
    name = "llama8b_unaligned"
    d = workload_inputs(name)
    w = d["workload"]
    p = ca.Problem.from_workload(w)
    x = device_inputs(d)
    masks, _ = oracle_estimate(name)
    rel = ca.load()
    P = B._ptr
    ws = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
    # block-sparse: one table per (b, h, Q-block) mask row
    bip, bix = ca.build_block_sparse_tables(p, u64_dev(masks))
    outs = []
    for lib in (rel, dbg):
        out = torch.empty_like(x["q"])
        st = lib.ca_block_sparse_chunk_attention(p.ref, P(x["q"]), P(x["k"]), P(x["v"]),
                                                 P(x["pt"]), P(bip), P(bix), w.sm_scale, 0,
                                                 P(out), None, P(ws), ws.numel(), B._stream(None))
        torch.cuda.synchronize()
        assert st == 0, (st, lib.ca_last_error_detail())
        outs.append(out)
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))
    # copy arm: packed pools in table order
    ip, ix = _tables(d, masks)
    tabs = (i32_dev(ip), i32_dev(ix))
    kp, vp = ca.gather_selected_pages(p, (x["k"], x["v"]), x["pt"], tabs, w.group_size)
    cap = kp.shape[0]
    outs = []
    for lib in (rel, dbg):
        out = torch.empty_like(x["q"])
        st = lib.ca_packed_chunk_attention(p.ref, P(x["q"]), P(kp), P(vp), P(tabs[0]),
                                           P(tabs[1]), w.group_size, w.sm_scale, 0, cap, P(out),
                                           None, P(ws), ws.numel(), B._stream(None))
        torch.cuda.synchronize()
        assert st == 0, (st, lib.ca_last_error_detail())
        outs.append(out)
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))
