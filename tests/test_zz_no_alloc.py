"""The allocation-free table builder (ca_build_block_tables_noalloc) against the
workspace one (ca_build_block_tables) through the C ABI: bit-exact tables on two
calls in a row, the second smaller, so the second reuses scratch that the first
left filled."""
import numpy as np
import pytest
import torch

from _helpers import u64_dev

pytestmark = pytest.mark.gpu

ca = pytest.importorskip("paper_2605_16839_amd")


def _case(seed, cached, Hq, Hkv, C, qb, and_words):
    """Masks whose bits are set with probability 2^-and_words (an AND of random
    words), every word of every row filled: the bits past a sequence's last
    block are garbage the builders must ignore."""
    rng = np.random.default_rng(seed)
    B = len(cached)
    nqb = -(-C // qb)
    maxkb = max(-(-(c + C) // 64) for c in cached)
    W = (maxkb + 63) // 64
    p = ca.Problem(B, Hq, Hkv, 128, qb, C, maxkb, cached)
    shape = (B, Hq, nqb, W)
    masks = np.full(shape, np.iinfo(np.uint64).max, dtype=np.uint64)
    for _ in range(and_words):
        masks &= rng.integers(0, 2**63, size=shape, dtype=np.int64).astype(np.uint64) | \
            (rng.integers(0, 2, size=shape, dtype=np.int64).astype(np.uint64) << np.uint64(63))
    return p, masks


@pytest.mark.parametrize("order", ["big_then_small"])
def test_noalloc_tables_equal_workspace_tables(order):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rng = np.random.default_rng(11)
    big_cached = [int(c) for c in rng.integers(0, 16384 * 64 - 2048, size=16)]
    cases = [
        # 16 sequences up to 1M tokens, 32/8 heads, groups of 4: 128 rows of up to 256 words
        (1, big_cached, 32, 8, 2048, 128, 5, 4),
        # then a smaller problem on the same scratch: 1 sequence, 4 heads on 1 KV head
        (2, [1000], 4, 1, 200, 64, 2, 2),
    ]
    for (seed, cached, Hq, Hkv, C, qb, and_words, gs) in cases:
        p, masks = _case(seed, cached, Hq, Hkv, C, qb, and_words)
        need = ca.tables_workspace_bytes(p, gs)
        print(f"case seed {seed}: B={len(cached)} rows={len(cached) * Hq // gs} "
              f"scratch bytes={need}", flush=True)
        m = u64_dev(masks)
        ref_ip, ref_ix = ca.build_block_tables(p, m, gs)
        got_ip, got_ix = ca.build_block_tables_noalloc(p, m, gs)
        torch.cuda.synchronize()
        rip, gip = ref_ip.cpu().numpy(), got_ip.cpu().numpy()
        assert np.array_equal(gip, rip)
        assert np.array_equal(got_ix.cpu().numpy()[:rip[-1]], ref_ix.cpu().numpy()[:rip[-1]])
        assert rip[-1] > 0
