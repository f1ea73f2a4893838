"""Thin ctypes binding of libcompactattn (include/compactattn.h).

Argument marshalling only: every step of the path runs in the HIP kernels of
the shared library.  torch is used for device memory and streams; tensors are
passed by ``data_ptr()`` and every call is enqueued on torch's current stream.
If the library has not been built, loading fails loudly -- there is no CPU
fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libcompactattn.so")
# the same sources built with CA_DEBUG_CHECKS: table and page-id checks before
# every attention launch (see ca_check_tables_host in include/compactattn.h)
DEBUG_LIB_PATH = os.path.join(_PKG, "libcompactattn_debug.so")

_c_i32p = ctypes.POINTER(ctypes.c_int32)

EXPORTED = (
    "ca_abi_version", "ca_status_string", "ca_last_error_detail", "ca_check_problem",
    "ca_pool_q_blocks", "ca_pool_k_blocks", "ca_block_scores", "ca_select_blocks",
    "ca_estimate_masks", "ca_tables_workspace_bytes", "ca_build_block_tables",
    "ca_attention_workspace_bytes", "ca_chunk_attention",
    "ca_dense_paged_chunk_attention", "ca_validate_tables",
    "ca_block_sparse_tables_workspace_bytes", "ca_build_block_sparse_tables",
    "ca_block_sparse_chunk_attention", "ca_gather_selected_pages", "ca_packed_chunk_attention",
    "ca_select_blocks_threshold", "ca_estimate_masks_threshold", "ca_estimate_tables",
    "ca_build_block_tables_noalloc", "ca_check_tables_host",
)


class CAProblem(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("q_block", ctypes.c_int32),
        ("chunk_len", ctypes.c_int32),
        ("max_kv_blocks", ctypes.c_int32),
        ("cached_len_host", _c_i32p),
        ("cached_len", ctypes.c_void_p),
        ("v_layout", ctypes.c_int32),
    ]


# ca_problem.v_layout: V pages token-major [P, page, D] (the paper's layout, as
# the K pages) or transposed [P, D, page]
V_TOKEN_MAJOR = 0
V_TRANSPOSED = 1


class CAError(RuntimeError):
    def __init__(self, status: int, name: str, detail: str):
        super().__init__(f"{name}: {detail}")
        self.status = status
        self.name = name
        self.detail = detail


_lib = None


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Load the shared library (raises if it has not been built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it first (__graft_entry__.build() or "
                           "python -m paper_2605_16839_amd.build)")
    lib = ctypes.CDLL(p)
    P = ctypes.POINTER(CAProblem)
    vp, i32, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
    i64 = ctypes.c_int64
    sig = {
        "ca_abi_version": ([], ctypes.c_int),
        "ca_status_string": ([ctypes.c_int], ctypes.c_char_p),
        "ca_last_error_detail": ([], ctypes.c_char_p),
        "ca_check_problem": ([P, i32], ctypes.c_int),
        "ca_pool_q_blocks": ([P, vp, vp, vp], ctypes.c_int),
        "ca_pool_k_blocks": ([P, vp, vp, i32, vp, vp], ctypes.c_int),
        "ca_block_scores": ([P, vp, vp, vp, vp], ctypes.c_int),
        "ca_select_blocks": ([P, vp, f32, i32, i32, vp, vp], ctypes.c_int),
        "ca_estimate_masks": ([P, vp, vp, vp, f32, i32, i32, i32, vp, vp, vp, vp, vp], ctypes.c_int),
        "ca_tables_workspace_bytes": ([P, i32], sz),
        "ca_build_block_tables": ([P, vp, i32, vp, vp, vp, sz, vp], ctypes.c_int),
        "ca_build_block_tables_noalloc": ([P, vp, i32, vp, vp, vp], ctypes.c_int),
        "ca_attention_workspace_bytes": ([P, i32, i32], sz),
        "ca_chunk_attention": ([P, vp, vp, vp, vp, vp, vp, i32, f32, i32, vp, vp, vp, sz, vp],
                               ctypes.c_int),
        "ca_dense_paged_chunk_attention": ([P, vp, vp, vp, vp, f32, i32, vp, vp, vp, sz, vp],
                                           ctypes.c_int),
        "ca_validate_tables": ([P, i32, vp, vp, i32, vp], ctypes.c_int),
        "ca_check_tables_host": ([P, i32, vp, vp, vp, i64, i32], ctypes.c_int),
        "ca_select_blocks_threshold": ([P, vp, f32, f32, f32, i32, i32, vp, vp], ctypes.c_int),
        "ca_estimate_masks_threshold": ([P, vp, vp, vp, f32, f32, f32, i32, i32, i32, vp, vp, vp,
                                         vp, vp], ctypes.c_int),
        "ca_estimate_tables": ([P, vp, vp, vp, f32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp,
                                sz, vp], ctypes.c_int),
        "ca_block_sparse_tables_workspace_bytes": ([P, i32], sz),
        "ca_build_block_sparse_tables": ([P, vp, i32, vp, vp, vp, sz, vp], ctypes.c_int),
        "ca_block_sparse_chunk_attention": ([P, vp, vp, vp, vp, vp, vp, f32, i32, vp, vp, vp,
                                             sz, vp], ctypes.c_int),
        "ca_gather_selected_pages": ([P, vp, vp, vp, vp, vp, i32, vp, vp, i64, vp],
                                     ctypes.c_int),
        "ca_packed_chunk_attention": ([P, vp, vp, vp, vp, vp, i32, f32, i32, i64, vp, vp, vp,
                                       sz, vp], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    if path is None:
        _lib = lib
    return lib


def _check(status: int) -> None:
    if status != 0:
        lib = load()
        raise CAError(status, lib.ca_status_string(status).decode(),
                      lib.ca_last_error_detail().decode())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Problem:
    """Sizes of one chunk step plus the per-sequence cached lengths.

    Holds the ca_problem struct, the host copy of cached_len that it points
    to, and the device copy (on ``device``; None for host-only validation).
    ``v_layout`` names the layout of the V pages the attention calls read.
    """

    def __init__(self, batch: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
                 q_block: int, chunk_len: int, max_kv_blocks: int,
                 cached_len: Sequence[int], page_size: int = 64,
                 device: Optional[str] = "cuda", v_layout: int = V_TOKEN_MAJOR):
        self.batch, self.num_q_heads, self.num_kv_heads = batch, num_q_heads, num_kv_heads
        self.head_dim, self.q_block, self.chunk_len = head_dim, q_block, chunk_len
        self.page_size, self.max_kv_blocks = page_size, max_kv_blocks
        self.v_layout = v_layout
        self._host = (ctypes.c_int32 * len(cached_len))(*[int(c) for c in cached_len])
        self.cached_len = [int(c) for c in cached_len]
        self.cached_len_dev = (torch.tensor(self.cached_len, dtype=torch.int32, device=device)
                               if device is not None else None)
        self.c = CAProblem(batch, num_q_heads, num_kv_heads, head_dim, page_size, q_block,
                           chunk_len, max_kv_blocks,
                           ctypes.cast(self._host, _c_i32p),
                           self.cached_len_dev.data_ptr() if self.cached_len_dev is not None else None,
                           v_layout)

    @classmethod
    def from_workload(cls, w, device: Optional[str] = "cuda",
                      v_layout: int = V_TOKEN_MAJOR) -> "Problem":
        return cls(w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.q_block, w.chunk_len,
                   w.max_kv_blocks, w.cached_lens, w.page_size, device, v_layout)

    @property
    def ref(self):
        return ctypes.byref(self.c)

    @property
    def n_qblocks(self) -> int:
        return -(-self.chunk_len // self.q_block)

    @property
    def words(self) -> int:
        return (self.max_kv_blocks + 63) // 64

    def n_groups(self, group_size: int) -> int:
        return self.num_q_heads // group_size


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------
def abi_version() -> int:
    return load().ca_abi_version()


def check_problem(p: Problem, group_size: int = 0) -> None:
    _check(load().ca_check_problem(p.ref, group_size))


def _dev(p: Problem):
    return p.cached_len_dev.device


def pool_q_blocks(p: Problem, q: torch.Tensor, q_mean: Optional[torch.Tensor] = None, stream=None):
    if q_mean is None:
        q_mean = torch.empty((p.batch, p.num_q_heads, p.n_qblocks, p.head_dim),
                             dtype=torch.float32, device=q.device)
    _check(load().ca_pool_q_blocks(p.ref, _ptr(q), _ptr(q_mean), _stream(stream)))
    return q_mean


def pool_k_blocks(p: Problem, k_pool: torch.Tensor, page_table: torch.Tensor,
                  k_mean: Optional[torch.Tensor] = None, first_block: int = 0, stream=None):
    if k_mean is None:
        k_mean = torch.zeros((p.batch, p.num_kv_heads, p.max_kv_blocks, p.head_dim),
                             dtype=torch.float32, device=k_pool.device)
    _check(load().ca_pool_k_blocks(p.ref, _ptr(k_pool), _ptr(page_table), first_block,
                                   _ptr(k_mean), _stream(stream)))
    return k_mean


def block_scores(p: Problem, q_mean: torch.Tensor, k_mean: torch.Tensor,
                 scores: Optional[torch.Tensor] = None, stream=None):
    if scores is None:
        scores = torch.full((p.batch, p.num_q_heads, p.n_qblocks, p.max_kv_blocks), float("nan"),
                            dtype=torch.float32, device=q_mean.device)
    _check(load().ca_block_scores(p.ref, _ptr(q_mean), _ptr(k_mean), _ptr(scores),
                                  _stream(stream)))
    return scores


def select_blocks(p: Problem, scores: torch.Tensor, top_frac: float, sink_blocks: int = 1,
                  local_blocks: int = 4, masks: Optional[torch.Tensor] = None, stream=None):
    if masks is None:
        masks = torch.empty((p.batch, p.num_q_heads, p.n_qblocks, p.words), dtype=torch.int64,
                            device=scores.device)
    _check(load().ca_select_blocks(p.ref, _ptr(scores), top_frac, sink_blocks, local_blocks,
                                   _ptr(masks), _stream(stream)))
    return masks


def estimate_masks(p: Problem, q: torch.Tensor, k_pool: torch.Tensor, page_table: torch.Tensor,
                   top_frac: float, sink_blocks: int = 1, local_blocks: int = 4,
                   k_mean: Optional[torch.Tensor] = None, k_mean_first_block: int = 0,
                   bufs: Optional[dict] = None, stream=None):
    """Returns (masks int64-bits [B,Hq,nQB,W], dict of q_mean, k_mean, scores)."""
    dev = q.device
    b = bufs if bufs is not None else {}
    if "q_mean" not in b:
        b["q_mean"] = torch.empty((p.batch, p.num_q_heads, p.n_qblocks, p.head_dim),
                                  dtype=torch.float32, device=dev)
    if k_mean is not None:
        b["k_mean"] = k_mean
    elif "k_mean" not in b:
        b["k_mean"] = torch.zeros((p.batch, p.num_kv_heads, p.max_kv_blocks, p.head_dim),
                                  dtype=torch.float32, device=dev)
    if "scores" not in b:
        b["scores"] = torch.empty((p.batch, p.num_q_heads, p.n_qblocks, p.max_kv_blocks),
                                  dtype=torch.float32, device=dev)
    if "masks" not in b:
        b["masks"] = torch.empty((p.batch, p.num_q_heads, p.n_qblocks, p.words),
                                 dtype=torch.int64, device=dev)
    _check(load().ca_estimate_masks(p.ref, _ptr(q), _ptr(k_pool), _ptr(page_table), top_frac,
                                    sink_blocks, local_blocks, k_mean_first_block,
                                    _ptr(b["q_mean"]), _ptr(b["k_mean"]), _ptr(b["scores"]),
                                    _ptr(b["masks"]), _stream(stream)))
    return b["masks"], b


def estimate_masks_threshold(p: Problem, q: torch.Tensor, k_pool: torch.Tensor,
                             page_table: torch.Tensor, alpha: float, temperature: float,
                             sm_scale: float, sink_blocks: int = 1, local_blocks: int = 4,
                             k_mean: Optional[torch.Tensor] = None, k_mean_first_block: int = 0,
                             bufs: Optional[dict] = None, stream=None):
    """Alpha-threshold selector: (masks, buffers) like estimate_masks."""
    dev = q.device
    b = bufs if bufs is not None else {}
    if "q_mean" not in b:
        b["q_mean"] = torch.empty((p.batch, p.num_q_heads, p.n_qblocks, p.head_dim),
                                  dtype=torch.float32, device=dev)
    if k_mean is not None:
        b["k_mean"] = k_mean
    elif "k_mean" not in b:
        b["k_mean"] = torch.zeros((p.batch, p.num_kv_heads, p.max_kv_blocks, p.head_dim),
                                  dtype=torch.float32, device=dev)
    if "scores" not in b:
        b["scores"] = torch.empty((p.batch, p.num_q_heads, p.n_qblocks, p.max_kv_blocks),
                                  dtype=torch.float32, device=dev)
    if "masks" not in b:
        b["masks"] = torch.empty((p.batch, p.num_q_heads, p.n_qblocks, p.words),
                                 dtype=torch.int64, device=dev)
    _check(load().ca_estimate_masks_threshold(p.ref, _ptr(q), _ptr(k_pool), _ptr(page_table),
                                              alpha, temperature, sm_scale, sink_blocks,
                                              local_blocks, k_mean_first_block,
                                              _ptr(b["q_mean"]), _ptr(b["k_mean"]),
                                              _ptr(b["scores"]), _ptr(b["masks"]),
                                              _stream(stream)))
    return b["masks"], b


def select_blocks_threshold(p: Problem, scores: torch.Tensor, alpha: float, temperature: float,
                            sm_scale: float, sink_blocks: int = 1, local_blocks: int = 4,
                            masks: Optional[torch.Tensor] = None, stream=None):
    if masks is None:
        masks = torch.empty((p.batch, p.num_q_heads, p.n_qblocks, p.words), dtype=torch.int64,
                            device=scores.device)
    _check(load().ca_select_blocks_threshold(p.ref, _ptr(scores), alpha, temperature, sm_scale,
                                             sink_blocks, local_blocks, _ptr(masks),
                                             _stream(stream)))
    return masks


def tables_workspace_bytes(p: Problem, group_size: int) -> int:
    return load().ca_tables_workspace_bytes(p.ref, group_size)


def build_block_tables(p: Problem, masks: torch.Tensor, group_size: int,
                       out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None,
                       ws: Optional[torch.Tensor] = None, stream=None):
    """masks -> tables = (kv_indptr [B*G+1], kv_indices [B*G*max_kv_blocks]) int32."""
    dev = masks.device
    R = p.batch * p.n_groups(group_size)
    if out is None:
        out = (torch.empty(R + 1, dtype=torch.int32, device=dev),
               torch.empty(R * p.max_kv_blocks, dtype=torch.int32, device=dev))
    nbytes = tables_workspace_bytes(p, group_size)
    if ws is None:
        ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    _check(load().ca_build_block_tables(p.ref, _ptr(masks), group_size, _ptr(out[0]),
                                        _ptr(out[1]), _ptr(ws), ws.numel() * ws.element_size(),
                                        _stream(stream)))
    return out


def build_block_tables_noalloc(p: Problem, masks: torch.Tensor, group_size: int,
                               out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None,
                               stream=None):
    """build_block_tables without a workspace (the library's fixed scratch); the
    caller still owns the output tables (allocated here when ``out`` is None)."""
    R = p.batch * p.n_groups(group_size)
    if out is None:
        out = (torch.empty(R + 1, dtype=torch.int32, device=masks.device),
               torch.empty(R * p.max_kv_blocks, dtype=torch.int32, device=masks.device))
    _check(load().ca_build_block_tables_noalloc(p.ref, _ptr(masks), group_size, _ptr(out[0]),
                                                _ptr(out[1]), _stream(stream)))
    return out


def estimate_tables(p: Problem, q: torch.Tensor, k_pool: torch.Tensor, page_table: torch.Tensor,
                    top_frac: float, group_size: int, sink_blocks: int = 1,
                    local_blocks: int = 4, k_mean: Optional[torch.Tensor] = None,
                    k_mean_first_block: int = 0, bufs: Optional[dict] = None,
                    out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None,
                    ws: Optional[torch.Tensor] = None, stream=None):
    """Fused estimator -> union -> CSR: returns (tables, buffers); no masks."""
    dev = q.device
    b = bufs if bufs is not None else {}
    if "q_mean" not in b:
        b["q_mean"] = torch.empty((p.batch, p.num_q_heads, p.n_qblocks, p.head_dim),
                                  dtype=torch.float32, device=dev)
    if k_mean is not None:
        b["k_mean"] = k_mean
    elif "k_mean" not in b:
        b["k_mean"] = torch.zeros((p.batch, p.num_kv_heads, p.max_kv_blocks, p.head_dim),
                                  dtype=torch.float32, device=dev)
    if "scores" not in b:
        b["scores"] = torch.empty((p.batch, p.num_q_heads, p.n_qblocks, p.max_kv_blocks),
                                  dtype=torch.float32, device=dev)
    R = p.batch * p.n_groups(group_size)
    if out is None:
        out = (torch.empty(R + 1, dtype=torch.int32, device=dev),
               torch.empty(R * p.max_kv_blocks, dtype=torch.int32, device=dev))
    if ws is None:
        ws = torch.empty(max(tables_workspace_bytes(p, group_size), 8), dtype=torch.uint8,
                         device=dev)
    _check(load().ca_estimate_tables(p.ref, _ptr(q), _ptr(k_pool), _ptr(page_table), top_frac,
                                     sink_blocks, local_blocks, k_mean_first_block, group_size,
                                     _ptr(b["q_mean"]), _ptr(b["k_mean"]), _ptr(b["scores"]),
                                     _ptr(out[0]), _ptr(out[1]), _ptr(ws),
                                     ws.numel() * ws.element_size(), _stream(stream)))
    return out, b


def attention_workspace_bytes(p: Problem, group_size: int, num_splits: int) -> int:
    return load().ca_attention_workspace_bytes(p.ref, group_size, num_splits)


def _attn_ws(p, group_size, num_splits, ws, dev):
    if ws is not None:
        return ws
    n = attention_workspace_bytes(p, group_size, num_splits)
    return torch.empty(n, dtype=torch.uint8, device=dev) if n else None


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def chunk_attention(p: Problem, q_chunk: torch.Tensor, kv_pool: Tuple[torch.Tensor, torch.Tensor],
                    page_table: torch.Tensor, tables: Tuple[torch.Tensor, torch.Tensor],
                    group_size: int, sm_scale: float, num_splits: int = 0,
                    out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                    ws: Optional[torch.Tensor] = None, stream=None):
    """Attention of the chunk over its groups' tables; returns (out bf16, lse fp32 or None).

    ``kv_pool`` = (k_pool ``[P, page, D]``, v_pool ``[P, page, D]``, or
    ``[P, D, page]`` when ``p.v_layout == V_TRANSPOSED``)."""
    k_pool, v_pool = kv_pool
    if out is None:
        out = torch.empty_like(q_chunk)
    ws = _attn_ws(p, group_size, num_splits, ws, q_chunk.device)
    _check(load().ca_chunk_attention(p.ref, _ptr(q_chunk), _ptr(k_pool), _ptr(v_pool),
                                     _ptr(page_table), _ptr(tables[0]), _ptr(tables[1]),
                                     group_size, sm_scale, num_splits, _ptr(out), _ptr(lse),
                                     _ptr(ws), _nbytes(ws), _stream(stream)))
    return out, lse


def dense_paged_chunk_attention(p: Problem, q_chunk: torch.Tensor,
                                kv_pool: Tuple[torch.Tensor, torch.Tensor],
                                page_table: torch.Tensor, sm_scale: float, num_splits: int = 0,
                                out: Optional[torch.Tensor] = None,
                                lse: Optional[torch.Tensor] = None,
                                ws: Optional[torch.Tensor] = None, stream=None):
    k_pool, v_pool = kv_pool
    if out is None:
        out = torch.empty_like(q_chunk)
    gs = p.num_q_heads // p.num_kv_heads
    ws = _attn_ws(p, gs, num_splits, ws, q_chunk.device)
    _check(load().ca_dense_paged_chunk_attention(p.ref, _ptr(q_chunk), _ptr(k_pool),
                                                 _ptr(v_pool), _ptr(page_table), sm_scale,
                                                 num_splits, _ptr(out), _ptr(lse), _ptr(ws),
                                                 _nbytes(ws), _stream(stream)))
    return out, lse


def block_sparse_tables_workspace_bytes(p: Problem, group_size: int = 0) -> int:
    return load().ca_block_sparse_tables_workspace_bytes(p.ref, group_size)


def build_block_sparse_tables(p: Problem, masks: torch.Tensor, group_size: int = 0,
                              out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None,
                              ws: Optional[torch.Tensor] = None, stream=None):
    """One table per (b, h, Q-block) row: its own mask row (group_size = 0) or the
    causally limited union of its execution group (group_size > 0)."""
    dev = masks.device
    R = p.batch * p.num_q_heads * p.n_qblocks
    if out is None:
        out = (torch.empty(R + 1, dtype=torch.int32, device=dev),
               torch.empty(R * p.max_kv_blocks, dtype=torch.int32, device=dev))
    nbytes = block_sparse_tables_workspace_bytes(p, group_size)
    if ws is None:
        ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    _check(load().ca_build_block_sparse_tables(p.ref, _ptr(masks), group_size, _ptr(out[0]),
                                               _ptr(out[1]), _ptr(ws), _nbytes(ws),
                                               _stream(stream)))
    return out


def block_sparse_chunk_attention(p: Problem, q_chunk: torch.Tensor,
                                 kv_pool: Tuple[torch.Tensor, torch.Tensor],
                                 page_table: torch.Tensor, tables: Tuple[torch.Tensor, torch.Tensor],
                                 sm_scale: float, num_splits: int = 0,
                                 out: Optional[torch.Tensor] = None,
                                 lse: Optional[torch.Tensor] = None,
                                 ws: Optional[torch.Tensor] = None, stream=None):
    """Attention of every (head, Q-block) over its own mask row's blocks."""
    k_pool, v_pool = kv_pool
    if out is None:
        out = torch.empty_like(q_chunk)
    ws = _attn_ws(p, 1, num_splits, ws, q_chunk.device)
    _check(load().ca_block_sparse_chunk_attention(p.ref, _ptr(q_chunk), _ptr(k_pool),
                                                  _ptr(v_pool), _ptr(page_table),
                                                  _ptr(tables[0]), _ptr(tables[1]), sm_scale,
                                                  num_splits, _ptr(out), _ptr(lse), _ptr(ws),
                                                  _nbytes(ws), _stream(stream)))
    return out, lse


def gather_selected_pages(p: Problem, kv_pool: Tuple[torch.Tensor, torch.Tensor],
                          page_table: torch.Tensor, tables: Tuple[torch.Tensor, torch.Tensor],
                          group_size: int, capacity_pages: Optional[int] = None,
                          out: Optional[Tuple[torch.Tensor, torch.Tensor]] = None, stream=None):
    """Copy arm: pack every group's selected K/V pages contiguously in table order."""
    k_pool, v_pool = kv_pool
    if capacity_pages is None:
        capacity_pages = p.batch * p.n_groups(group_size) * p.max_kv_blocks
    if out is None:
        out = (torch.empty((capacity_pages,) + tuple(k_pool.shape[1:]), dtype=k_pool.dtype,
                           device=k_pool.device),
               torch.empty((capacity_pages,) + tuple(v_pool.shape[1:]), dtype=v_pool.dtype,
                           device=v_pool.device))
    _check(load().ca_gather_selected_pages(p.ref, _ptr(k_pool), _ptr(v_pool), _ptr(page_table),
                                           _ptr(tables[0]), _ptr(tables[1]), group_size,
                                           _ptr(out[0]), _ptr(out[1]), capacity_pages,
                                           _stream(stream)))
    return out


def packed_chunk_attention(p: Problem, q_chunk: torch.Tensor,
                           packed: Tuple[torch.Tensor, torch.Tensor],
                           tables: Tuple[torch.Tensor, torch.Tensor], group_size: int,
                           sm_scale: float, num_splits: int = 0,
                           out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                           ws: Optional[torch.Tensor] = None, stream=None):
    """Copy arm: attention over the packed pools (table entry p = packed page p)."""
    k_packed, v_packed = packed
    if out is None:
        out = torch.empty_like(q_chunk)
    ws = _attn_ws(p, group_size, num_splits, ws, q_chunk.device)
    _check(load().ca_packed_chunk_attention(p.ref, _ptr(q_chunk), _ptr(k_packed),
                                            _ptr(v_packed), _ptr(tables[0]), _ptr(tables[1]),
                                            group_size, sm_scale, num_splits,
                                            k_packed.shape[0], _ptr(out), _ptr(lse), _ptr(ws),
                                            _nbytes(ws), _stream(stream)))
    return out, lse


def check_tables_host(p: Problem, group_size: int, kv_indptr, kv_indices, page_table=None,
                      pool_pages: int = 0, require_chunk_open: bool = False) -> None:
    """Host-only check of host (numpy int32) tables and, with a page table, of the
    page ids they reach; group_size 0 = the block-sparse (b, h, Q-block) rows."""
    import numpy as np

    arr = [None if a is None else np.ascontiguousarray(a, dtype=np.int32)
           for a in (kv_indptr, kv_indices, page_table)]
    ptr = lambda a: None if a is None else ctypes.c_void_p(a.ctypes.data)
    _check(load().ca_check_tables_host(p.ref, group_size, ptr(arr[0]), ptr(arr[1]), ptr(arr[2]),
                                       int(pool_pages), int(require_chunk_open)))


def validate_tables(p: Problem, group_size: int, tables, require_chunk_open: bool = True,
                    stream=None) -> None:
    _check(load().ca_validate_tables(p.ref, group_size, _ptr(tables[0]), _ptr(tables[1]),
                                     int(require_chunk_open), _stream(stream)))
