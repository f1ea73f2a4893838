"""Helpers shared by the GPU tests: device transfer and attention comparison."""
import numpy as np
import torch

import oracle
import synth

# Tolerances on bf16 attention outputs against the fp64 oracle.
MAX_ABS = 2e-2      # per element
MEAN_ABS = 2e-3     # mean over compared elements
REL_L2 = 1e-2       # ||got - ref|| / ||ref|| over compared rows
LSE_ABS = 1e-3      # natural-log log-sum-exp per row

DEV = "cuda"


def bf16_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV).view(torch.bfloat16)


def i32_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def u64_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint64).view(np.int64)).to(DEV)


def u64_host(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint64)


def bf16_host_f64(t: torch.Tensor) -> np.ndarray:
    return oracle.bf16_to_f64(t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16))


V_TOKEN_MAJOR, V_TRANSPOSED = 0, 1   # ca_problem.v_layout


def device_inputs(d: dict, v_layout: int = V_TOKEN_MAJOR) -> dict:
    """Q, K pool, V pool (token-major pages, or transposed ones) and page table on the GPU."""
    v = d["v_pool"] if v_layout == V_TOKEN_MAJOR else synth.v_pages_transposed(d["v_pool"])
    return dict(q=bf16_dev(d["q"]), k=bf16_dev(d["k_pool"]), v=bf16_dev(v),
                pt=i32_dev(d["page_table"]))


def compare_attention(got, got_lse, ref, ref_lse, rows=None, lse_tol=LSE_ABS):
    """got/ref: [B, C, Hq, D]; lse: [B, Hq, C].  ``rows`` = list of (b, h, t)."""
    if rows is None:
        g, r = got, ref
        gl, rl = got_lse, ref_lse
    else:
        bs, hs, ts = (np.array(x) for x in zip(*rows))
        g, r = got[bs, ts, hs, :], ref[bs, ts, hs, :]
        gl, rl = got_lse[bs, hs, ts], ref_lse[bs, hs, ts]
    err = np.abs(g - r)
    stats = dict(max_abs=float(err.max()), mean_abs=float(err.mean()),
                 rel_l2=float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-30)))
    fin = np.isfinite(rl)
    assert np.array_equal(fin, np.isfinite(gl)), "lse -inf pattern differs"
    stats["lse_abs"] = float(np.abs(gl[fin] - rl[fin]).max()) if fin.any() else 0.0
    assert stats["max_abs"] <= MAX_ABS, stats
    assert stats["mean_abs"] <= MEAN_ABS, stats
    assert stats["rel_l2"] <= REL_L2, stats
    assert stats["lse_abs"] <= lse_tol, stats
    return stats


def sample_rows(B, Hq, C, seed=0, heads_per_b=4, n_random=16):
    """(b, h, t) rows: chunk edges, tile edges and random queries on a few heads."""
    rng = np.random.default_rng(seed)
    fixed = [0, 1, 15, 16, 31, 32, 63, 64, 127, 128, C // 2, C - 65, C - 64, C - 2, C - 1]
    fixed = sorted({t for t in fixed if 0 <= t < C})
    rows = []
    for b in range(B):
        heads = sorted(set([0, Hq - 1] + rng.choice(Hq, size=heads_per_b, replace=False).tolist()))
        for h in heads:
            ts = sorted(set(fixed + rng.choice(C, size=n_random, replace=False).tolist()))
            rows += [(b, h, t) for t in ts]
    return rows


def tile_rows(B, Hq, C, group_size, seed=0, rows_per_tile=256, per_tile=2):
    """(b, h, t) rows covering every (sequence, execution group, query tile) of
    the attention kernel: a workgroup runs rows_per_tile (head, query) rows,
    i.e. rows_per_tile / group_size queries of every head of its group.  Each
    tile contributes per_tile queries (one on a tile edge, alternately the first
    and the last query, the others at random) on one head of the group, the
    head rotating from tile to tile so that every head of every group appears."""
    rng = np.random.default_rng(seed)
    qt = rows_per_tile // group_size
    rows = []
    for b in range(B):
        for g in range(Hq // group_size):
            for t in range(-(-C // qt)):
                h = g * group_size + (t + b + g) % group_size
                lo, hi = t * qt, min((t + 1) * qt, C)
                ts = {lo if t % 2 == 0 else hi - 1}
                while len(ts) < min(per_tile, hi - lo):
                    ts.add(int(rng.integers(lo, hi)))
                rows += [(b, h, x) for x in sorted(ts)]
    return rows


def rows_by_head(rows):
    heads, queries = {}, {}
    for (b, h, t) in rows:
        heads.setdefault((b, h), []).append(t)
    return heads
