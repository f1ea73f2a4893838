"""Merging split pieces (Sec. 3.3's attention over a table row cut into pieces,
the pieces' partial results merged by log-sum-exp).

The XCD-balanced split merges its two pieces inside the attention launch: the
second piece of a query tile to finish merges, in piece order, so the output
does not depend on which piece finishes second.  Its arrival counter lives in
the workspace, tagged per launch.  Uniform splits are merged by a second launch.
So, for both:
- the output is bit-identical whatever the workspace held on entry (zeros, all
  ones, random bytes), and a launch leaves every counter it used at zero;
- a launch on a workspace that still holds another launch's partial results
  gives bit-for-bit the output of a launch on a fresh workspace (a merge that
  read a stale partial through a cache would not);
- merged outputs still match the oracle (the parity tests cover every schedule;
  here two rows of every query tile per schedule)."""
import numpy as np
import pytest
import torch

import oracle
from _helpers import (bf16_host_f64, compare_attention, device_inputs, i32_dev, rows_by_head,
                      tile_rows)

pytestmark = pytest.mark.gpu

ca = pytest.importorskip("paper_2605_16839_amd")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ca.load()


def _counter_region(w, gs):
    """Byte range of the XCD-balanced split's arrival counters in the attention
    workspace: after the two partial outputs and log-sum-exps and the cut points,
    at the next 8-byte boundary, one uint64 per query tile (B*G rows x tiles)."""
    rows = w.batch * w.num_q_heads * w.chunk_len
    G = w.num_q_heads // gs
    at = 2 * rows * (w.head_dim + 1) * 4 + w.batch * G * 4
    at = (at + 7) & ~7
    tiles = w.batch * G * -(-w.chunk_len // (256 // gs))
    return at, at + 8 * tiles


_RT = {}


def _case(name, workload_inputs):
    """Inputs plus random group tables with rows of different lengths (every row
    cut by the XCD-balanced split), at 0.3 cached density."""
    if name not in _RT:
        d = workload_inputs(name)
        w = d["workload"]
        G = w.num_groups
        ncs = [w.n_cached_blocks(b) for b in range(w.batch)]
        nkbs = [w.n_kv_blocks(b) for b in range(w.batch)]
        T = []
        rng = np.random.default_rng(w.seed + 77)
        for b in range(w.batch):
            for g in range(G):
                nc = ncs[b]
                keep = rng.random(nc) < 0.2 + 0.2 * g / max(G - 1, 1)
                keep[0] = True
                T.append(sorted(set(np.nonzero(keep)[0].tolist()) | set(range(nc, nkbs[b]))))
        ip = np.zeros(len(T) + 1, dtype=np.int32)
        ip[1:] = np.cumsum([len(r) for r in T])
        ix = np.concatenate([np.asarray(r, dtype=np.int32) for r in T])
        _RT[name] = (d, T, ip, ix)
    return _RT[name]


# (workload, num_splits, dense): 0 on the 32K and batched shapes with tables of
# unequal lengths is the XCD-balanced two-piece split (merged in the launch);
# explicit splits run uniform pieces, merged by a second launch.  (With dense
# tables the batched rows are balanced over the XCDs already, one group of every
# sequence on each, and no row is cut.)
CASES = [
    ("llama8b_32k", 0, False),
    ("llama8b_32k", 2, False),
    ("llama8b_32k", 3, False),
    ("batched_ragged_4seq", 0, False),
    ("batched_ragged_4seq", 2, True),
    ("tiny_gqa_1k", 4, False),
]


def _run(ca_p, w, x, q, tables, gs, splits, dense, ws):
    out = torch.empty_like(q)
    lse = torch.empty((w.batch, w.num_q_heads, w.chunk_len), dtype=torch.float32, device="cuda")
    if dense:
        ca.dense_paged_chunk_attention(ca_p, q, (x["k"], x["v"]), x["pt"], w.sm_scale,
                                       num_splits=splits, out=out, lse=lse, ws=ws)
    else:
        ca.chunk_attention(ca_p, q, (x["k"], x["v"]), x["pt"], tables, gs, w.sm_scale,
                           num_splits=splits, out=out, lse=lse, ws=ws)
    torch.cuda.synchronize()
    return out.view(torch.int16).cpu().numpy(), lse.cpu().numpy()


def _same(a, b):
    assert np.array_equal(a[0], b[0]), "outputs differ"
    assert np.array_equal(a[1].view(np.int32), b[1].view(np.int32)), "lse differ"


@pytest.mark.parametrize("name,splits,dense", CASES)
def test_merge_independent_of_workspace(name, splits, dense, workload_inputs):
    d, T, ip, ix = _case(name, workload_inputs)
    w = d["workload"]
    gs = w.num_q_heads // w.num_kv_heads if dense else w.group_size
    p = ca.Problem.from_workload(w)
    x = device_inputs(d)
    tables = (i32_dev(ip), i32_dev(ix))
    nbytes = ca.attention_workspace_bytes(p, gs, splits)
    assert nbytes > 0
    xcd = splits == 0
    lo, hi = _counter_region(w, gs) if xcd else (0, 0)
    if xcd:
        assert hi == nbytes
    print(name, "splits", splits, "dense", dense, "ws bytes", nbytes, flush=True)

    ws0 = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    ref = _run(p, w, x, x["q"], tables, gs, splits, dense, ws0)
    assert not torch.any(ws0[lo:hi]), "a used counter was not left at zero"
    # the same launch again on the same workspace
    _same(_run(p, w, x, x["q"], tables, gs, splits, dense, ws0), ref)

    ones = torch.full((nbytes,), 255, dtype=torch.uint8, device="cuda")
    _same(_run(p, w, x, x["q"], tables, gs, splits, dense, ones), ref)
    if xcd:
        # counters of merged tiles back at 0; those of rows left whole untouched
        c = ones[lo:hi].cpu().numpy().view(np.uint64)
        assert set(np.unique(c).tolist()) <= {0, 2 ** 64 - 1}
        assert np.count_nonzero(c == 0) > 0, "no tile was merged"
    _same(_run(p, w, x, x["q"], tables, gs, splits, dense, ones), ref)

    g = torch.Generator().manual_seed(w.seed + 5)
    rnd = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, generator=g).to("cuda")
    _same(_run(p, w, x, x["q"], tables, gs, splits, dense, rnd), ref)


@pytest.mark.parametrize("name,splits,dense", CASES)
def test_merge_no_stale_partials(name, splits, dense, workload_inputs):
    """Launches on other queries in between: each output equals that of a launch
    on a fresh workspace, so no merge read a partial of an earlier launch."""
    d, T, ip, ix = _case(name, workload_inputs)
    w = d["workload"]
    gs = w.num_q_heads // w.num_kv_heads if dense else w.group_size
    p = ca.Problem.from_workload(w)
    x = device_inputs(d)
    tables = (i32_dev(ip), i32_dev(ix))
    nbytes = ca.attention_workspace_bytes(p, gs, splits)
    qs = [x["q"], torch.roll(x["q"], shifts=1, dims=1), -x["q"]]
    fresh = [_run(p, w, x, q, tables, gs, splits, dense,
                  torch.zeros(nbytes, dtype=torch.uint8, device="cuda")) for q in qs]
    assert not np.array_equal(fresh[0][0], fresh[1][0])
    ws = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    for i in (0, 1, 2, 1, 0, 2):
        _same(_run(p, w, x, qs[i], tables, gs, splits, dense, ws), fresh[i])


@pytest.mark.parametrize("name,splits,dense", CASES)
def test_merge_matches_oracle(name, splits, dense, workload_inputs):
    """Two rows of every (group row, query tile) against the fp64 oracle."""
    d, T, ip, ix = _case(name, workload_inputs)
    w = d["workload"]
    gs = w.num_q_heads // w.num_kv_heads if dense else w.group_size
    p = ca.Problem.from_workload(w)
    x = device_inputs(d)
    tables = (i32_dev(ip), i32_dev(ix))
    nbytes = ca.attention_workspace_bytes(p, gs, splits)
    out = torch.empty_like(x["q"])
    lse = torch.empty((w.batch, w.num_q_heads, w.chunk_len), dtype=torch.float32, device="cuda")
    ws = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    if dense:
        ca.dense_paged_chunk_attention(p, x["q"], (x["k"], x["v"]), x["pt"], w.sm_scale,
                                       num_splits=splits, out=out, lse=lse, ws=ws)
        nkb = [w.n_kv_blocks(b) for b in range(w.batch)]
        Tq = [list(range(nkb[r // w.num_kv_heads])) for r in range(w.batch * w.num_kv_heads)]
    else:
        ca.chunk_attention(p, x["q"], (x["k"], x["v"]), x["pt"], tables, gs, w.sm_scale,
                           num_splits=splits, out=out, lse=lse, ws=ws)
        Tq = T
    torch.cuda.synchronize()
    rows = tile_rows(w.batch, w.num_q_heads, w.chunk_len, gs, seed=w.seed, per_tile=2)
    if w.batch > 1:
        rows = rows[::4 if dense else 2]   # rows over up to 2016 blocks: a subset
    G = w.num_q_heads // gs
    tab = [[Tq[b * G + g] for g in range(G)] for b in range(w.batch)]
    ref = np.full((w.batch, w.chunk_len, w.num_q_heads, w.head_dim), np.nan)
    ref_lse = np.full((w.batch, w.num_q_heads, w.chunk_len), np.nan)
    for (b, h), ts in rows_by_head(rows).items():
        o, l = oracle.chunk_attention(d["q"], d["k_pool"], d["v_pool"], d["page_table"],
                                      d["cached_len"], tab, gs, w.sm_scale,
                                      heads=[(b, h)], queries=ts)
        ref[b, ts, h] = o[b, ts, h]
        ref_lse[b, h, ts] = l[b, h, ts]
    stats = compare_attention(bf16_host_f64(out), lse.cpu().numpy().astype(np.float64), ref,
                              ref_lse, rows=rows)
    print(name, splits, "dense" if dense else "selected", len(rows), "rows", stats)
