"""The C-ABI library: it loads, exports every declared entry point, and its
host-side validation rejects bad problems before anything is enqueued.
No compute call is made here (no GPU in this tier)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "compactattn.h")

ca = pytest.importorskip("paper_2605_16839_amd")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = set(re.findall(r"\b(ca_[a-z_0-9]+)\s*\(", src))
    return names


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ca.LIB_PATH):
        pytest.fail("libcompactattn.so is not built (run __graft_entry__.build())")
    return ca.load()


def test_exports_every_declared_symbol(lib):
    declared = _declared()
    assert declared, "no declarations parsed"
    assert declared == set(ca.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name
    m = re.search(r"#define CA_ABI_VERSION (\d+)", open(HEADER).read())
    assert lib.ca_abi_version() == int(m.group(1))


def _prob(**kw):
    base = dict(batch=1, num_q_heads=32, num_kv_heads=8, head_dim=128, q_block=128,
                chunk_len=2048, max_kv_blocks=2048, cached_len=[129024], device=None)
    base.update(kw)
    return ca.Problem(**base)


def _status(p, group_size=4):
    return ca.load().ca_check_problem(p.ref, group_size)


def test_valid_problems(lib):
    assert _status(_prob()) == 0
    assert _status(_prob(batch=4, cached_len=[16384, 32768, 65536, 126976], max_kv_blocks=2016)) == 0
    assert _status(_prob(num_q_heads=4, num_kv_heads=1, head_dim=64, q_block=64, chunk_len=256,
                         max_kv_blocks=20, cached_len=[1024])) == 0
    assert _status(_prob(cached_len=[0])) == 0
    # any lengths: partial last Q-block and page, a block shared by cache and chunk
    assert _status(_prob(chunk_len=2000)) == 0
    assert _status(_prob(cached_len=[129000])) == 0          # 131048 tokens: 2048 blocks
    assert _status(_prob(chunk_len=1, cached_len=[1])) == 0


@pytest.mark.parametrize("kw,group,code", [
    (dict(head_dim=96), 4, "CA_ERR_UNSUPPORTED"),
    (dict(q_block=32), 4, "CA_ERR_UNSUPPORTED"),
    (dict(cached_len=[-64]), 4, "CA_ERR_SHAPE"),
    (dict(cached_len=[-1]), 4, "CA_ERR_SHAPE"),
    (dict(cached_len=[129088]), 4, "CA_ERR_SHAPE"),           # needs 2049 blocks
    (dict(cached_len=[129025]), 4, "CA_ERR_SHAPE"),           # 131073 tokens: 2049 blocks
    (dict(chunk_len=0), 4, "CA_ERR_SHAPE"),
    (dict(max_kv_blocks=20000, cached_len=[64]), 4, "CA_ERR_SHAPE"),
    (dict(num_kv_heads=5), 4, "CA_ERR_SHAPE"),
    (dict(), 3, "CA_ERR_GROUP"),
    (dict(), 8, "CA_ERR_GROUP"),
    (dict(batch=0, cached_len=[]), 4, "CA_ERR_SHAPE"),
])
def test_invalid_problems(lib, kw, group, code):
    s = _status(_prob(**kw), group)
    assert lib.ca_status_string(s).decode() == code
    assert lib.ca_last_error_detail().decode() != ""


def test_null_problem_and_null_buffers(lib):
    assert lib.ca_status_string(lib.ca_check_problem(None, 4)).decode() == "CA_ERR_NULL"
    p = _prob()
    # device cached_len missing: rejected before any launch
    s = lib.ca_build_block_tables(p.ref, None, 4, None, None, None, 0, None)
    assert lib.ca_status_string(s).decode() == "CA_ERR_NULL"
    s = lib.ca_chunk_attention(p.ref, None, None, None, None, None, None, 4, 0.1, 1,
                               None, None, None, 0, None)
    assert lib.ca_status_string(s).decode() == "CA_ERR_NULL"


def test_workspace_sizes(lib):
    p = _prob()
    # union words (8 rows x 32 words x 8 B) + 8 counts
    assert ca.tables_workspace_bytes(p, 4) == 8 * 32 * 8 + 8 * 4
    assert ca.attention_workspace_bytes(p, 4, 1) == 0
    assert ca.attention_workspace_bytes(p, 4, 2) == 2 * 32 * 2048 * 129 * 4
    # 256 query tiles fill the GPU and the 8 table rows spread over the 8 XCDs:
    # the automatic choice cuts every row in two (two partial sets + 8 cut
    # points + one 8-byte arrival counter per query tile, 8 rows x 32 tiles)
    assert ca.attention_workspace_bytes(p, 4, 0) == 2 * 32 * 2048 * 129 * 4 + 8 * 4 + 8 * 256
    # 6 table rows do not spread evenly over the XCDs: the uniform choice, here
    # 2 splits because 192 query tiles cannot fill the 256 resident workgroups
    six = _prob(num_q_heads=24, num_kv_heads=6)
    assert ca.attention_workspace_bytes(six, 4, 0) == 2 * 24 * 2048 * 129 * 4
    tiny = _prob(num_q_heads=4, num_kv_heads=1, head_dim=64, q_block=64, chunk_len=256,
                 max_kv_blocks=20, cached_len=[1024])
    assert ca.attention_workspace_bytes(tiny, 4, 0) > 0
    assert ca.tables_workspace_bytes(p, 3) == 0        # invalid group -> 0
    # block-sparse tables: one row per (b, h, Q-block) = 512 rows of 32 words + counts
    assert ca.block_sparse_tables_workspace_bytes(p) == 512 * 32 * 8 + 512 * 4
    assert ca.block_sparse_tables_workspace_bytes(p, 4) == (8 * 32 * 8 + 8 * 4) + (512 * 32 * 8 + 512 * 4)
    assert ca.block_sparse_tables_workspace_bytes(p, 3) == 0


def test_arm_validation(lib):
    """Host-side checks of the copy and block-sparse arms (nothing is launched)."""
    fake = ctypes.c_void_p(0x1000)    # never dereferenced: validation fails first
    tiny = _prob(num_q_heads=4, num_kv_heads=1, head_dim=64, q_block=64, chunk_len=256,
                 max_kv_blocks=20, cached_len=[1024])
    tiny.c.cached_len = fake.value
    # a 128-query tile of one head cannot follow 64-query Q-blocks
    s = lib.ca_block_sparse_chunk_attention(tiny.ref, fake, fake, fake, fake, fake, fake, 0.1, 1,
                                            fake, None, None, 0, None)
    assert lib.ca_status_string(s).decode() == "CA_ERR_UNSUPPORTED"
    p = _prob()
    p.c.cached_len = fake.value
    s = lib.ca_packed_chunk_attention(p.ref, fake, fake, fake, fake, fake, 4, 0.1, 1, 0,
                                      fake, None, None, 0, None)
    assert lib.ca_status_string(s).decode() == "CA_ERR_SHAPE"     # capacity 0
    s = lib.ca_gather_selected_pages(p.ref, fake, fake, fake, fake, fake, 4, fake, fake,
                                     8 * 2048 + 1, None)
    assert lib.ca_status_string(s).decode() == "CA_ERR_SHAPE"     # beyond B*G*max_kv_blocks
    s = lib.ca_gather_selected_pages(p.ref, fake, fake, fake, fake, fake, 3, fake, fake, 10, None)
    assert lib.ca_status_string(s).decode() == "CA_ERR_GROUP"


def test_threshold_validation(lib):
    """Threshold parameters are rejected on the host before any stage is enqueued
    (fake device pointers, never dereferenced)."""
    fake = ctypes.c_void_p(0x1000)
    p = _prob()
    p.c.cached_len = fake.value
    cases = [(0.0, 16.0, 0.1, 1, 4), (1.5, 16.0, 0.1, 1, 4), (float("nan"), 16.0, 0.1, 1, 4),
             (0.1, 0.0, 0.1, 1, 4), (0.1, 16.0, -0.1, 1, 4), (0.1, 16.0, 0.1, -1, 4)]
    for a, t, sm, sink, local in cases:
        s = lib.ca_select_blocks_threshold(p.ref, fake, a, t, sm, sink, local, fake, None)
        assert lib.ca_status_string(s).decode() == "CA_ERR_SHAPE", (a, t, sm, sink, local)
        s = lib.ca_estimate_masks_threshold(p.ref, fake, fake, fake, a, t, sm, sink, local, 0,
                                            fake, fake, fake, fake, None)
        assert lib.ca_status_string(s).decode() == "CA_ERR_SHAPE", (a, t, sm, sink, local)
    s = lib.ca_estimate_masks(p.ref, fake, fake, fake, 1.5, 1, 4, 0, fake, fake, fake, fake,
                              None)
    assert lib.ca_status_string(s).decode() == "CA_ERR_SHAPE"


def test_fused_tables_validation(lib):
    """ca_estimate_tables rejects a bad group, parameters and a short or
    misaligned workspace on the host (fake device pointers, never dereferenced)."""
    fake = ctypes.c_void_p(0x1000)
    p = _prob()
    p.c.cached_len = fake.value
    need = lib.ca_tables_workspace_bytes(p.ref, 4)
    assert need > 0

    def call(top=0.05, gs=4, ws=fake, nbytes=need, first=0):
        s = lib.ca_estimate_tables(p.ref, fake, fake, fake, top, 1, 4, first, gs, fake, fake,
                                   fake, fake, fake, ws, nbytes, None)
        return lib.ca_status_string(s).decode()

    assert call(gs=3) == "CA_ERR_GROUP"
    assert call(gs=0) == "CA_ERR_GROUP"
    assert call(top=1.5) == "CA_ERR_SHAPE"
    assert call(first=-1) == "CA_ERR_SHAPE"
    assert call(ws=None) == "CA_ERR_WORKSPACE"
    assert call(nbytes=8) == "CA_ERR_WORKSPACE"
    assert call(ws=ctypes.c_void_p(0x1004)) == "CA_ERR_WORKSPACE"



def test_unaligned_tensors_rejected(lib):
    """Every entry point rejects a bf16 / fp32 tensor that does not start on a
    16-byte boundary, on the host, before anything is enqueued (fake device
    pointers, never dereferenced)."""
    fake = ctypes.c_void_p(0x1000)
    odd = ctypes.c_void_p(0x1008)     # 8-byte aligned only
    p = _prob()
    p.c.cached_len = fake.value
    st = lambda s: lib.ca_status_string(s).decode()
    assert st(lib.ca_pool_q_blocks(p.ref, odd, fake, None)) == "CA_ERR_UNALIGNED"
    assert st(lib.ca_pool_k_blocks(p.ref, fake, fake, 0, odd, None)) == "CA_ERR_UNALIGNED"
    assert st(lib.ca_block_scores(p.ref, fake, fake, odd, None)) == "CA_ERR_UNALIGNED"
    assert st(lib.ca_estimate_masks(p.ref, fake, odd, fake, 0.05, 1, 4, 0, fake, fake, fake,
                                    fake, None)) == "CA_ERR_UNALIGNED"
    assert st(lib.ca_estimate_masks_threshold(p.ref, fake, fake, fake, 0.9, 1.0, 0.1, 1, 4, 0,
                                              odd, fake, fake, fake, None)) == "CA_ERR_UNALIGNED"
    need = lib.ca_tables_workspace_bytes(p.ref, 4)
    assert st(lib.ca_estimate_tables(p.ref, fake, fake, fake, 0.05, 1, 4, 0, 4, fake, fake, odd,
                                     fake, fake, fake, need, None)) == "CA_ERR_UNALIGNED"
    for args in ((odd, fake, fake, fake), (fake, odd, fake, fake), (fake, fake, odd, fake),
                 (fake, fake, fake, odd)):
        q, k, v, out = args
        assert st(lib.ca_chunk_attention(p.ref, q, k, v, fake, fake, fake, 4, 0.1, 1, out, None,
                                         None, 0, None)) == "CA_ERR_UNALIGNED"
    assert st(lib.ca_dense_paged_chunk_attention(p.ref, fake, fake, odd, fake, 0.1, 1, fake, None,
                                                 None, 0, None)) == "CA_ERR_UNALIGNED"
    assert st(lib.ca_gather_selected_pages(p.ref, fake, fake, fake, fake, fake, 4, fake, odd, 10,
                                           None)) == "CA_ERR_UNALIGNED"
    # the split-KV workspace holds fp32 partial rows written 16 bytes at a time
    ws = lib.ca_attention_workspace_bytes(p.ref, 4, 2)
    assert st(lib.ca_chunk_attention(p.ref, fake, fake, fake, fake, fake, fake, 4, 0.1, 2, fake,
                                     None, odd, ws, None)) == "CA_ERR_WORKSPACE"


def test_sm_scale_rejected(lib):
    """A zero, negative or non-finite softmax scale is rejected on the host by
    every attention entry point (it would turn masked scores into NaN / +inf
    weights); fake device pointers, never dereferenced."""
    fake = ctypes.c_void_p(0x1000)
    p = _prob()
    p.c.cached_len = fake.value
    st = lambda s: lib.ca_status_string(s).decode()
    for sm in (0.0, -0.125, float("nan"), float("inf"), -float("inf")):
        assert st(lib.ca_chunk_attention(p.ref, fake, fake, fake, fake, fake, fake, 4, sm, 1,
                                         fake, None, None, 0, None)) == "CA_ERR_SHAPE", sm
        assert st(lib.ca_dense_paged_chunk_attention(p.ref, fake, fake, fake, fake, sm, 1, fake,
                                                     None, None, 0, None)) == "CA_ERR_SHAPE", sm
        assert st(lib.ca_block_sparse_chunk_attention(p.ref, fake, fake, fake, fake, fake, fake,
                                                      sm, 1, fake, None, None, 0,
                                                      None)) == "CA_ERR_SHAPE", sm
        assert st(lib.ca_packed_chunk_attention(p.ref, fake, fake, fake, fake, fake, 4, sm, 1, 10,
                                                fake, None, None, 0, None)) == "CA_ERR_SHAPE", sm
    assert lib.ca_last_error_detail().decode().startswith("sm_scale")


def test_tables_workspace_alignment(lib):
    """The table builders keep uint64 union words in their workspace: a
    workspace that is not 8-byte aligned is rejected before any launch."""
    fake = ctypes.c_void_p(0x1000)
    odd = ctypes.c_void_p(0x1004)
    p = _prob()
    p.c.cached_len = fake.value
    st = lambda s: lib.ca_status_string(s).decode()
    need = lib.ca_tables_workspace_bytes(p.ref, 4)
    assert st(lib.ca_build_block_tables(p.ref, fake, 4, fake, fake, odd, need, None)) == \
        "CA_ERR_WORKSPACE"
    for gs in (0, 4):
        need = lib.ca_block_sparse_tables_workspace_bytes(p.ref, gs)
        assert st(lib.ca_build_block_sparse_tables(p.ref, fake, gs, fake, fake, odd, need,
                                                   None)) == "CA_ERR_WORKSPACE"


def test_v_layout_field(lib):
    """ca_problem.v_layout: 0 (token-major, the default) and 1 (transposed) are
    accepted, anything else is CA_ERR_SHAPE."""
    assert _status(_prob()) == 0
    assert _status(_prob(v_layout=ca.V_TRANSPOSED)) == 0
    for bad in (2, -1):
        s = _status(_prob(v_layout=bad))
        assert lib.ca_status_string(s).decode() == "CA_ERR_SHAPE"
        assert "v_layout" in lib.ca_last_error_detail().decode()


def test_block_sparse_workspace_one_group_row(lib):
    """One group row (B = 1, a single group of 4 heads): its words and count take
    12 bytes, so the per-(head, Q-block) words start at the next 8-byte boundary."""
    tiny = _prob(num_q_heads=4, num_kv_heads=1, head_dim=64, q_block=64, chunk_len=256,
                 max_kv_blocks=20, cached_len=[1024])
    assert ca.tables_workspace_bytes(tiny, 4) == 1 * 8 + 1 * 4
    rows = 4 * 4                         # heads x Q-blocks, one word each
    assert ca.block_sparse_tables_workspace_bytes(tiny, 4) == 16 + rows * 8 + rows * 4


def test_noalloc_tables_size_limit(lib):
    """The allocation-free table builder rejects, on the host and before any HIP
    call, a problem whose union words and counts exceed its fixed scratch
    (CA_NOALLOC_SCRATCH_BYTES); 512 group rows of 256 words need 1050624 bytes."""
    m = re.search(r"#define CA_NOALLOC_SCRATCH_BYTES \(1u << (\d+)\)", open(HEADER).read())
    limit = 1 << int(m.group(1))
    fake = ctypes.c_void_p(0x1000)
    big = _prob(batch=64, cached_len=[16384 * 64 - 2048] * 64, max_kv_blocks=16384)
    big.c.cached_len = fake.value
    assert ca.tables_workspace_bytes(big, 4) == 512 * (256 * 8 + 4) > limit
    s = lib.ca_build_block_tables_noalloc(big.ref, fake, 4, fake, fake, None)
    assert lib.ca_status_string(s).decode() == "CA_ERR_WORKSPACE"
    assert "scratch" in lib.ca_last_error_detail().decode()
    p = _prob()
    p.c.cached_len = fake.value
    st = lambda s: lib.ca_status_string(s).decode()
    assert st(lib.ca_build_block_tables_noalloc(p.ref, fake, 3, fake, fake, None)) == "CA_ERR_GROUP"
    assert st(lib.ca_build_block_tables_noalloc(p.ref, None, 4, fake, fake, None)) == "CA_ERR_NULL"


def _small_tables():
    """B = 2, Hq = 4, Hkv = 2, D = 64, q_block 64, C = 128, cached 100 / 256 tokens:
    nC = 1 / 4, nKB = 4 / 6; group_size 2 gives 4 rows (b, g), g reading KV head g."""
    p = ca.Problem(2, 4, 2, 64, 64, 128, 8, [100, 256], device=None)
    ip = np.array([0, 4, 8, 12, 16], dtype=np.int32)
    ix = np.array([0, 1, 2, 3, 0, 1, 2, 3, 0, 2, 4, 5, 1, 3, 4, 5], dtype=np.int32)
    pt = np.arange(2 * 2 * 8, dtype=np.int32).reshape(2, 2, 8)   # 32 distinct pages
    return p, ip, ix, pt


def _table_status(p, gs, ip, ix, pt=None, pages=0, chunk_open=0):
    ptr = lambda a: None if a is None else ctypes.c_void_p(np.ascontiguousarray(a).ctypes.data)
    arrs = [None if a is None else np.ascontiguousarray(a, dtype=np.int32) for a in (ip, ix, pt)]
    return ca.load().ca_check_tables_host(p.ref, gs, *[ptr(a) for a in arrs], pages, chunk_open)


def test_check_tables_host(lib):
    """The host table check that the debug build runs before every attention
    launch: CSR shape, entry order and range, chunk blocks, and page ids."""
    INV = 7
    p, ip, ix, pt = _small_tables()
    assert _table_status(p, 2, ip, ix) == 0
    assert _table_status(p, 2, ip, ix, pt, 32, 1) == 0
    ca.check_tables_host(p, 2, ip, ix, pt, 32, True)          # the Python wrapper
    bad = ix.copy(); bad[9], bad[10] = bad[10], bad[9]       # row 2 not ascending
    assert _table_status(p, 2, ip, bad) == INV
    bad = ix.copy(); bad[3] = 4                              # b = 0 has nKB = 4
    assert _table_status(p, 2, ip, bad) == INV
    bad = ix.copy(); bad[8] = -1
    assert _table_status(p, 2, ip, bad) == INV
    with pytest.raises(ca.CAError) as e:
        ca.check_tables_host(p, 2, ip, bad)
    assert e.value.name == "CA_ERR_INVALID_TABLE"
    # page ids: only the pages of listed blocks are checked, against [0, pool_pages)
    q = pt.copy(); q[1, 1, 3] = 32                           # row 3 lists block 3 of KV head 1
    assert _table_status(p, 2, ip, ix, q, 32) == INV
    assert _table_status(p, 2, ip, ix, q, 33) == 0
    q = pt.copy(); q[1, 0, 2] = -1                           # row 2 lists block 2 of KV head 0
    assert _table_status(p, 2, ip, ix, q, 32) == INV
    q = pt.copy(); q[1, 0, 1] = 999                          # block 1 of b = 1, KV head 0: not listed
    assert _table_status(p, 2, ip, ix, q, 32) == 0
    q = pt.copy(); q[0, 0, 7] = -5                           # past nKB: never read
    assert _table_status(p, 2, ip, ix, q, 32) == 0
    # chunk blocks 4, 5 of b = 1 must all be present when asked
    ip2 = np.array([0, 4, 8, 11, 15], dtype=np.int32)
    ix2 = np.array([0, 1, 2, 3, 0, 1, 2, 3, 0, 2, 4, 1, 3, 4, 5], dtype=np.int32)
    assert _table_status(p, 2, ip2, ix2) == 0
    assert _table_status(p, 2, ip2, ix2, chunk_open=1) == INV
    # CSR bounds
    bad_ip = ip.copy(); bad_ip[0] = 1
    assert _table_status(p, 2, bad_ip, ix) == INV
    bad_ip = ip.copy(); bad_ip[2] = 3                        # decreasing bound
    assert _table_status(p, 2, bad_ip, ix) == INV
    bad_ip = ip.copy(); bad_ip[4] = 4 * 8 + 1                # beyond B*G*max_kv_blocks
    assert _table_status(p, 2, bad_ip, ix) == INV
    # argument errors
    assert _table_status(p, -1, ip, ix) == 4                 # CA_ERR_GROUP
    assert _table_status(p, 3, ip, ix) == 4                  # 3 does not divide Hq / Hkv
    assert ca.load().ca_check_tables_host(p.ref, 2, None, None, None, 0, 0) == 1   # CA_ERR_NULL


def test_check_tables_host_block_sparse_rows(lib):
    """group_size 0: one row per (b, h, Q-block); row (b, h, i) reads KV head h / 2."""
    p, _, _, pt = _small_tables()
    nqb = 2
    rows = 2 * 4 * nqb
    ip = np.arange(rows + 1, dtype=np.int32)                 # every row lists block 0
    ix = np.zeros(rows, dtype=np.int32)
    assert _table_status(p, 0, ip, ix, pt, 32) == 0
    q = pt.copy(); q[1, 1, 0] = 40                           # (b = 1, h = 2 or 3) rows
    assert _table_status(p, 0, ip, ix, q, 32) == 7
    q = pt.copy(); q[1, 1, 1] = 40                           # block 1: listed by no row
    assert _table_status(p, 0, ip, ix, q, 32) == 0
