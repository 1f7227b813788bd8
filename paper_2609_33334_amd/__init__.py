"""MI355X (gfx950) eviction step of Draft-Guided Eviction (arxiv 2609.33334).

Thin Python binding over the C ABI of ``libdge.so`` (include/dge.h).  Functions
here only marshal arguments: they take torch tensors that already live on the
GPU, pass their device pointers and the current HIP stream to the library, and
allocate outputs/workspaces with torch when the caller does not pass them.
Every step of the path runs in the library's HIP kernels.

Names follow the C ABI: ``score`` (dge_score), ``select_topb``,
``select_streaming``, ``compact``, ``h2o_colsum``, ``pyramid_budgets``,
``workspace_size``; ``evict_layer`` chains score -> select_topb -> compact.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

from . import _lib
from ._lib import (DGE_BF16, DGE_F32, OP_H2O, OP_SCORE, OP_SELECT, ROWS_DRAFT,  # noqa: F401
                   ROWS_WINDOW, ROWS_WINDOW_DRAFT, DGEError, Geom)

__all__ = ["Geometry", "score", "score_noalloc", "score_with_lse", "score_lse", "evicted_mass", "select_topb", "select_compact",
           "select_compact_layers", "select_streaming", "compact", "compact_inplace",
           "cache_attention",
           "rope", "project_rope", "project_rope_workspace", "retained_runs", "h2o_colsum",
           "pyramid_budgets", "workspace_size", "evict_layer", "DGEError", "ROWS_WINDOW_DRAFT",
           "ROWS_DRAFT", "ROWS_WINDOW", "n_scoring_rows"]


def _torch():
    import torch
    return torch


def n_scoring_rows(window: int, k_draft: int, rows: int) -> int:
    return {ROWS_WINDOW_DRAFT: window + k_draft, ROWS_DRAFT: k_draft, ROWS_WINDOW: window}[rows]


@dataclass
class Geometry:
    """One layer's cache geometry (dge_geom_t) with the offsets kept alive.

    ``kv_lens`` are the cached rows N_b = L_b + k of each sequence.  K and V are
    [H_kv][sum N_b][head_dim] (``kv_head_stride`` elements between heads).
    """
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    window: int
    k_draft: int
    kv_lens: Sequence[int]
    dtype: int = DGE_BF16
    kv_head_stride: Optional[int] = None
    device: str = "cuda"

    def __post_init__(self):
        torch = _torch()
        self.offsets_host = np.concatenate([[0], np.cumsum(np.asarray(self.kv_lens, np.int64))]).astype(np.int64)
        self.offsets_dev = torch.tensor(self.offsets_host, dtype=torch.int64, device=self.device)
        if self.kv_head_stride is None:
            self.kv_head_stride = int(self.offsets_host[-1]) * self.head_dim
        self._c = Geom(len(self.kv_lens), self.n_q_heads, self.n_kv_heads, self.head_dim,
                       self.window, self.k_draft, self.offsets_dev.data_ptr(),
                       self.offsets_host.ctypes.data, int(self.kv_head_stride), int(self.dtype))

    @property
    def batch(self) -> int:
        return len(self.kv_lens)

    @property
    def total_rows(self) -> int:
        return int(self.offsets_host[-1])

    @property
    def c(self) -> Geom:
        return self._c

    @property
    def elt_dtype(self):
        torch = _torch()
        return torch.bfloat16 if self.dtype == DGE_BF16 else torch.float32


def _ptr(t) -> Optional[int]:
    """Device address of a tensor handed to the library (None for NULL); a host tensor
    is refused, since every pointer argument of the C ABI is a device pointer."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"a {tuple(t.shape)} tensor on {t.device} passed where the library "
                         "needs a GPU tensor")
    return t.data_ptr()


def _need(t, name: str, dtypes, min_numel: int = 0, optional: bool = False):
    """Argument check before anything reaches the library: a contiguous tensor of one of
    the given dtypes with at least min_numel elements (the C ABI sees raw pointers only, so
    a wrong element type or a short buffer would be misread).  The device is checked when
    the pointer is taken (_ptr)."""
    torch = _torch()
    if t is None:
        if optional:
            return
        raise ValueError(f"{name}: a tensor is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
    if t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype} not in {[str(d) for d in dtypes]}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if t.numel() < min_numel:
        raise ValueError(f"{name}: {t.numel()} elements, at least {min_numel} needed")


def _f32():
    return (_torch().float32,)


def _i32():
    return (_torch().int32,)


def _stream(stream) -> int:
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def workspace_size(geom: Geometry, op: int) -> int:
    n = ctypes.c_size_t(0)
    _lib.check(_lib.lib().dge_workspace_size(ctypes.byref(geom.c), op, ctypes.byref(n)),
               "dge_workspace_size")
    return int(n.value)


def _workspace(geom: Geometry, op: int, ws):
    torch = _torch()
    if ws is None:
        ws = torch.empty(workspace_size(geom, op), dtype=torch.uint8, device=geom.device)
    return ws


def score(geom: Geometry, rows: int, q, k, raw=None, ws=None, stream=None):
    """dge_score: raw[h][j] for every cached key.  Returns raw [H_kv][T] float32."""
    torch = _torch()
    nr = n_scoring_rows(geom.window, geom.k_draft, rows)
    _need(q, "q", (geom.elt_dtype,), geom.n_q_heads * geom.batch * nr * geom.head_dim)
    _need(k, "k", (geom.elt_dtype,), (geom.n_kv_heads - 1) * geom.kv_head_stride
          + geom.total_rows * geom.head_dim)
    if raw is None:
        raw = torch.empty(geom.n_kv_heads, geom.total_rows, dtype=torch.float32, device=geom.device)
    _need(raw, "raw", _f32(), geom.n_kv_heads * geom.total_rows)
    ws = _workspace(geom, OP_SCORE, ws)
    _lib.check(_lib.lib().dge_score(ctypes.byref(geom.c), rows, _ptr(q), _ptr(k), _ptr(raw),
                                    _ptr(ws), ws.numel(), _stream(stream)), "dge_score")
    return raw


def score_with_lse(geom: Geometry, rows: int, q, k, raw=None, row_lse=None, ws=None,
                   stream=None):
    """dge_score_with_lse: raw scores and the scoring rows' full-cache log-partitions.
    Returns (raw [H_kv][T], row_lse [H_q][batch * n_rows] natural log)."""
    torch = _torch()
    nr = n_scoring_rows(geom.window, geom.k_draft, rows)
    _need(q, "q", (geom.elt_dtype,), geom.n_q_heads * geom.batch * nr * geom.head_dim)
    _need(k, "k", (geom.elt_dtype,), (geom.n_kv_heads - 1) * geom.kv_head_stride
          + geom.total_rows * geom.head_dim)
    if raw is None:
        raw = torch.empty(geom.n_kv_heads, geom.total_rows, dtype=torch.float32, device=geom.device)
    if row_lse is None:
        row_lse = torch.empty(geom.n_q_heads, geom.batch * nr, dtype=torch.float32,
                              device=geom.device)
    _need(raw, "raw", _f32(), geom.n_kv_heads * geom.total_rows)
    _need(row_lse, "row_lse", _f32(), geom.n_q_heads * geom.batch * nr)
    ws = _workspace(geom, OP_SCORE, ws)
    _lib.check(_lib.lib().dge_score_with_lse(ctypes.byref(geom.c), rows, _ptr(q), _ptr(k),
                                             _ptr(raw), _ptr(row_lse), _ptr(ws), ws.numel(),
                                             _stream(stream)), "dge_score_with_lse")
    return raw, row_lse


def evicted_mass(geom: Geometry, q, n_q: int, q_from_end: int, k_c, n_select: int, n_tail: int,
                 n_kept, lse_full, rho=None, beta=None, l_match=None, stream=None):
    """dge_evicted_mass: per-row evicted mass rho [H_q][batch*n_q], and per (sequence, KV
    head) its mean beta and the attention-matching loss l_match ([batch][H_kv] each)."""
    torch = _torch()
    rows = geom.batch * n_q
    _need(q, "q", (geom.elt_dtype,), geom.n_q_heads * rows * geom.head_dim)
    _need(k_c, "k_c", (geom.elt_dtype,),
          geom.batch * geom.n_kv_heads * (n_select + n_tail) * geom.head_dim)
    _need(n_kept, "n_kept", _i32(), geom.batch)
    _need(lse_full, "lse_full", _f32(), geom.n_q_heads * rows)
    if rho is None:
        rho = torch.empty(geom.n_q_heads, rows, dtype=torch.float32, device=geom.device)
    if beta is None:
        beta = torch.empty(geom.batch, geom.n_kv_heads, dtype=torch.float32, device=geom.device)
    if l_match is None:
        l_match = torch.empty(geom.batch, geom.n_kv_heads, dtype=torch.float32, device=geom.device)
    _need(rho, "rho", _f32(), geom.n_q_heads * rows)
    _need(beta, "beta", _f32(), geom.batch * geom.n_kv_heads)
    _need(l_match, "l_match", _f32(), geom.batch * geom.n_kv_heads)
    _lib.check(_lib.lib().dge_evicted_mass(ctypes.byref(geom.c), _ptr(q), n_q, q_from_end,
                                           _ptr(k_c), n_select, n_tail, _ptr(n_kept),
                                           _ptr(lse_full), _ptr(rho), _ptr(beta), _ptr(l_match),
                                           _stream(stream)), "dge_evicted_mass")
    return rho, beta, l_match


def score_noalloc(geom: Geometry, rows: int, q, k, raw=None, stream=None):
    """dge_score_noalloc: dge_score with the library's fixed per-GPU scratch instead of a
    workspace (no device allocation inside the call; calls on one GPU must not overlap).
    Returns raw [H_kv][T] float32."""
    torch = _torch()
    nr = n_scoring_rows(geom.window, geom.k_draft, rows)
    _need(q, "q", (geom.elt_dtype,), geom.n_q_heads * geom.batch * nr * geom.head_dim)
    _need(k, "k", (geom.elt_dtype,), (geom.n_kv_heads - 1) * geom.kv_head_stride
          + geom.total_rows * geom.head_dim)
    if raw is None:
        raw = torch.empty(geom.n_kv_heads, geom.total_rows, dtype=torch.float32, device=geom.device)
    _need(raw, "raw", _f32(), geom.n_kv_heads * geom.total_rows)
    _lib.check(_lib.lib().dge_score_noalloc(ctypes.byref(geom.c), rows, _ptr(q), _ptr(k),
                                            _ptr(raw), _stream(stream)), "dge_score_noalloc")
    return raw


def score_lse(geom: Geometry, rows: int, q, k, row_lse, raw=None, stream=None):
    """dge_score_lse: dge_score with caller-supplied scoring-row log-sum-exp (one pass
    over K).  row_lse is [H_q][batch * n_rows] float32.  Returns raw [H_kv][T]."""
    torch = _torch()
    nr = n_scoring_rows(geom.window, geom.k_draft, rows)
    _need(q, "q", (geom.elt_dtype,), geom.n_q_heads * geom.batch * nr * geom.head_dim)
    _need(k, "k", (geom.elt_dtype,), (geom.n_kv_heads - 1) * geom.kv_head_stride
          + geom.total_rows * geom.head_dim)
    _need(row_lse, "row_lse", _f32(), geom.n_q_heads * geom.batch * nr)
    if raw is None:
        raw = torch.empty(geom.n_kv_heads, geom.total_rows, dtype=torch.float32, device=geom.device)
    _need(raw, "raw", _f32(), geom.n_kv_heads * geom.total_rows)
    _lib.check(_lib.lib().dge_score_lse(ctypes.byref(geom.c), rows, _ptr(q), _ptr(k), _ptr(row_lse),
                                        _ptr(raw), _stream(stream)), "dge_score_lse")
    return raw


def select_topb(geom: Geometry, scores, pool_kernel: int, n_tail: int, n_select: int,
                idx=None, n_kept=None, ws=None, stream=None):
    """dge_select_topb: per-head top-n_select after max-pooling.  Returns (idx, n_kept)."""
    torch = _torch()
    if idx is None:
        idx = torch.empty(geom.batch, geom.n_kv_heads, max(n_select, 0), dtype=torch.int32,
                          device=geom.device)
    if n_kept is None:
        n_kept = torch.empty(max(geom.batch, 4), dtype=torch.int32, device=geom.device)
    _need(scores, "scores", _f32(), geom.n_kv_heads * geom.total_rows)
    _need(idx, "idx", _i32(), geom.batch * geom.n_kv_heads * max(n_select, 0))
    _need(n_kept, "n_kept", _i32(), geom.batch)
    ws = _workspace(geom, OP_SELECT, ws)
    _lib.check(_lib.lib().dge_select_topb(ctypes.byref(geom.c), _ptr(scores), pool_kernel, n_tail,
                                          n_select, _ptr(idx), _ptr(n_kept), _ptr(ws), ws.numel(),
                                          _stream(stream)), "dge_select_topb")
    return idx, n_kept[:geom.batch]


def select_compact(geom: Geometry, scores, pool_kernel: int, n_tail: int, n_select: int, k, v,
                   idx=None, n_kept=None, k_out=None, v_out=None, ws=None, stream=None):
    """dge_select_compact: select_topb and compact in one call.
    Returns (idx, n_kept, k_out, v_out)."""
    torch = _torch()
    if idx is None:
        idx = torch.empty(geom.batch, geom.n_kv_heads, max(n_select, 0), dtype=torch.int32,
                          device=geom.device)
    if n_kept is None:
        n_kept = torch.empty(max(geom.batch, 4), dtype=torch.int32, device=geom.device)
    shape = (geom.batch, geom.n_kv_heads, n_select + n_tail, geom.head_dim)
    if k_out is None:
        k_out = torch.empty(shape, dtype=k.dtype, device=geom.device)
    if v_out is None:
        v_out = torch.empty(shape, dtype=v.dtype, device=geom.device)
    kv_min = (geom.n_kv_heads - 1) * geom.kv_head_stride + geom.total_rows * geom.head_dim
    _need(scores, "scores", _f32(), geom.n_kv_heads * geom.total_rows)
    _need(idx, "idx", _i32(), geom.batch * geom.n_kv_heads * max(n_select, 0))
    _need(n_kept, "n_kept", _i32(), geom.batch)
    _need(k, "k", (geom.elt_dtype,), kv_min)
    _need(v, "v", (geom.elt_dtype,), kv_min)
    _need(k_out, "k_out", (geom.elt_dtype,), k_out_numel := geom.batch * geom.n_kv_heads
          * (n_select + n_tail) * geom.head_dim)
    _need(v_out, "v_out", (geom.elt_dtype,), k_out_numel)
    ws = _workspace(geom, OP_SELECT, ws)
    _lib.check(_lib.lib().dge_select_compact(ctypes.byref(geom.c), _ptr(scores), pool_kernel,
                                             n_tail, n_select, _ptr(idx), _ptr(n_kept), _ptr(k),
                                             _ptr(v), _ptr(k_out), _ptr(v_out), _ptr(ws),
                                             ws.numel(), _stream(stream)), "dge_select_compact")
    return idx, n_kept[:geom.batch], k_out, v_out


def select_compact_layers(geom: Geometry, scores, pool_kernel: int, n_tail: int, n_select,
                          k, v, idx=None, n_kept=None, k_out=None, v_out=None, ws=None,
                          stream=None):
    """dge_select_compact_layers: select + compact for len(n_select) layers of a
    layer-major cache in one launch (geom describes one layer).  Returns lists of
    per-layer views (idx [batch][H_kv][n_select[l]], k_out / v_out
    [batch][H_kv][n_select[l] + n_tail][d]) and n_kept [n_layers][batch]; the packed
    buffers may be passed in as flat tensors."""
    torch = _torch()
    n_sel = [int(x) for x in n_select]
    nl = len(n_sel)
    nb = geom.batch * geom.n_kv_heads
    tot_idx = nb * sum(n_sel)
    tot_rows = nb * sum(x + n_tail for x in n_sel)
    if idx is None:
        idx = torch.empty(max(tot_idx, 4), dtype=torch.int32, device=geom.device)
    if n_kept is None:
        n_kept = torch.empty(max(nl * geom.batch, 4), dtype=torch.int32, device=geom.device)
    if k_out is None:
        k_out = torch.empty(tot_rows, geom.head_dim, dtype=k.dtype, device=geom.device)
    if v_out is None:
        v_out = torch.empty(tot_rows, geom.head_dim, dtype=v.dtype, device=geom.device)
    kv_min = ((nl * geom.n_kv_heads - 1) * geom.kv_head_stride + geom.total_rows * geom.head_dim)
    _need(scores, "scores", _f32(), nl * geom.n_kv_heads * geom.total_rows)
    _need(idx, "idx", _i32(), tot_idx)
    _need(n_kept, "n_kept", _i32(), nl * geom.batch)
    _need(k, "k", (geom.elt_dtype,), kv_min)
    _need(v, "v", (geom.elt_dtype,), kv_min)
    _need(k_out, "k_out", (geom.elt_dtype,), tot_rows * geom.head_dim)
    _need(v_out, "v_out", (geom.elt_dtype,), tot_rows * geom.head_dim)
    ws = _workspace(geom, OP_SELECT, ws)
    arr = (ctypes.c_int32 * nl)(*n_sel)
    _lib.check(_lib.lib().dge_select_compact_layers(
        ctypes.byref(geom.c), nl, _ptr(scores), pool_kernel, n_tail, arr, _ptr(idx),
        _ptr(n_kept), _ptr(k), _ptr(v), _ptr(k_out), _ptr(v_out), _ptr(ws), ws.numel(),
        _stream(stream)), "dge_select_compact_layers")
    idx_l, k_l, v_l = [], [], []
    io = ro = 0
    for x in n_sel:
        idx_l.append(idx[io:io + nb * x].view(geom.batch, geom.n_kv_heads, x))
        rows = nb * (x + n_tail)
        shape = (geom.batch, geom.n_kv_heads, x + n_tail, geom.head_dim)
        k_l.append(k_out.view(-1, geom.head_dim)[ro:ro + rows].view(shape))
        v_l.append(v_out.view(-1, geom.head_dim)[ro:ro + rows].view(shape))
        io += nb * x
        ro += rows
    return idx_l, n_kept[:nl * geom.batch].view(nl, geom.batch), k_l, v_l


def select_streaming(geom: Geometry, n_sink: int, n_recent: int, idx=None, n_kept=None,
                     stream=None):
    """dge_select_streaming: StreamingLLM sinks.  Returns (idx, n_kept)."""
    torch = _torch()
    if idx is None:
        idx = torch.empty(geom.batch, geom.n_kv_heads, max(n_sink, 1), dtype=torch.int32,
                          device=geom.device)
    if n_kept is None:
        n_kept = torch.empty(max(geom.batch, 4), dtype=torch.int32, device=geom.device)
    _lib.check(_lib.lib().dge_select_streaming(ctypes.byref(geom.c), n_sink, n_recent, _ptr(idx),
                                               _ptr(n_kept), _stream(stream)),
               "dge_select_streaming")
    return idx[..., :n_sink], n_kept[:geom.batch]


def compact(geom: Geometry, idx, n_kept, n_select: int, n_tail: int, k, v, k_out=None,
            v_out=None, stream=None):
    """dge_compact: [retained past] || [tail] per (b, h).  Returns (k_out, v_out)
    shaped [batch][H_kv][n_select + n_tail][head_dim]."""
    torch = _torch()
    shape = (geom.batch, geom.n_kv_heads, n_select + n_tail, geom.head_dim)
    if k_out is None:
        k_out = torch.empty(shape, dtype=k.dtype, device=geom.device)
    if v_out is None:
        v_out = torch.empty(shape, dtype=v.dtype, device=geom.device)
    kv_min = (geom.n_kv_heads - 1) * geom.kv_head_stride + geom.total_rows * geom.head_dim
    _need(idx, "idx", _i32(), geom.batch * geom.n_kv_heads * max(n_select, 0))
    _need(n_kept, "n_kept", _i32(), geom.batch)
    _need(k, "k", (geom.elt_dtype,), kv_min)
    _need(v, "v", (geom.elt_dtype,), kv_min)
    _need(k_out, "k_out", (geom.elt_dtype,), n_out := geom.batch * geom.n_kv_heads
          * (n_select + n_tail) * geom.head_dim)
    _need(v_out, "v_out", (geom.elt_dtype,), n_out)
    _lib.check(_lib.lib().dge_compact(ctypes.byref(geom.c), _ptr(idx), _ptr(n_kept), n_select,
                                      n_tail, _ptr(k), _ptr(v), _ptr(k_out), _ptr(v_out),
                                      _stream(stream)), "dge_compact")
    return k_out, v_out


def compact_inplace(geom: Geometry, idx, n_kept, n_select: int, n_tail: int, k, v,
                    stream=None):
    """dge_compact_inplace: the compacted rows overwrite the first n_kept[b] + n_tail rows
    of each (sequence, KV head) segment of k and v.  Returns (k, v)."""
    kv_min = (geom.n_kv_heads - 1) * geom.kv_head_stride + geom.total_rows * geom.head_dim
    _need(idx, "idx", _i32(), geom.batch * geom.n_kv_heads * max(n_select, 0))
    _need(n_kept, "n_kept", _i32(), geom.batch)
    _need(k, "k", (geom.elt_dtype,), kv_min)
    _need(v, "v", (geom.elt_dtype,), kv_min)
    _lib.check(_lib.lib().dge_compact_inplace(ctypes.byref(geom.c), _ptr(idx), _ptr(n_kept),
                                              n_select, n_tail, _ptr(k), _ptr(v),
                                              _stream(stream)), "dge_compact_inplace")
    return k, v


def cache_attention(geom: Geometry, q, n_q: int, q_from_end: int, k_c, v_c, n_select: int,
                    n_tail: int, n_kept, out=None, lse=None, stream=None):
    """dge_cache_attention: attention of query rows over compacted caches (the layout of
    compact / select_compact).  Returns (out [H_q][batch*n_q][d] float32,
    lse [H_q][batch*n_q] float32, natural log)."""
    torch = _torch()
    rows = geom.batch * n_q
    if out is None:
        out = torch.empty(geom.n_q_heads, rows, geom.head_dim, dtype=torch.float32,
                          device=geom.device)
    if lse is None:
        lse = torch.empty(geom.n_q_heads, rows, dtype=torch.float32, device=geom.device)
    n_c = geom.batch * geom.n_kv_heads * (n_select + n_tail) * geom.head_dim
    _need(q, "q", (geom.elt_dtype,), geom.n_q_heads * rows * geom.head_dim)
    _need(k_c, "k_c", (geom.elt_dtype,), n_c)
    _need(v_c, "v_c", (geom.elt_dtype,), n_c)
    _need(n_kept, "n_kept", _i32(), geom.batch)
    _need(out, "out", _f32(), geom.n_q_heads * rows * geom.head_dim)
    _need(lse, "lse", _f32(), geom.n_q_heads * rows)
    _lib.check(_lib.lib().dge_cache_attention(ctypes.byref(geom.c), _ptr(q), n_q, q_from_end,
                                              _ptr(k_c), _ptr(v_c), n_select, n_tail,
                                              _ptr(n_kept), _ptr(out), _ptr(lse),
                                              _stream(stream)), "dge_cache_attention")
    return out, lse


def rope(x, positions, theta: float = 500000.0, stream=None):
    """dge_rope: rotary position embedding of the rows of x ([heads][rows][head_dim],
    bf16 or float32, contiguous) at the given int32 positions, in place.  Returns x."""
    torch = _torch()
    if not isinstance(x, torch.Tensor) or x.dim() != 3:
        raise ValueError("x: expected a [heads][rows][head_dim] tensor")
    # element types first (an fp16 x would be read as float32, int64 positions as pairs
    # of int32), then sizes and devices
    if x.dtype not in (torch.bfloat16, torch.float32):
        raise TypeError(f"x: dtype {x.dtype}; rope takes bfloat16 or float32 rows")
    if not isinstance(positions, torch.Tensor) or positions.dtype != torch.int32:
        raise TypeError("positions: expected an int32 tensor")
    _need(x, "x", (torch.bfloat16, torch.float32))
    _need(positions, "positions", _i32(), x.shape[1])
    dt = DGE_BF16 if x.dtype == torch.bfloat16 else DGE_F32
    _lib.check(_lib.lib().dge_rope(x.shape[0], x.shape[1], x.shape[2], dt,
                                   x.shape[1] * x.shape[2], _ptr(positions), float(theta),
                                   _ptr(x), _stream(stream)), "dge_rope")
    return x


def project_rope_workspace(n_rows: int, hidden: int, n_heads: int, head_dim: int) -> int:
    """dge_project_rope_workspace: bytes of workspace dge_project_rope needs (0 for none)."""
    n = ctypes.c_size_t(0)
    _lib.check(_lib.lib().dge_project_rope_workspace(n_rows, hidden, n_heads, head_dim,
                                                     ctypes.byref(n)), "dge_project_rope_workspace")
    return int(n.value)


def project_rope(x, w, positions, n_heads: int, head_dim: int, theta: float = 500000.0,
                 out=None, ws=None, stream=None):
    """dge_project_rope: out = RoPE(x W^T) per head, x [n_rows][hidden] bf16, w
    [n_heads*head_dim][hidden] bf16 (a Linear weight), int32 positions [n_rows].  Returns
    out [n_heads][n_rows][head_dim] bf16."""
    torch = _torch()
    if not isinstance(x, torch.Tensor) or x.dim() != 2 or not isinstance(w, torch.Tensor) or w.dim() != 2:
        raise ValueError("x: [n_rows][hidden] and w: [n_heads * head_dim][hidden] expected")
    n_rows, hidden = x.shape
    if w.shape[0] != n_heads * head_dim or w.shape[1] != hidden:
        raise ValueError(f"w: shape {tuple(w.shape)}, expected ({n_heads * head_dim}, {hidden})")
    _need(x, "x", (torch.bfloat16,))
    _need(w, "w", (torch.bfloat16,))
    if not isinstance(positions, torch.Tensor) or positions.dtype != torch.int32:
        raise TypeError("positions: expected an int32 tensor")
    _need(positions, "positions", _i32(), n_rows)
    if out is None:
        out = torch.empty(n_heads, n_rows, head_dim, dtype=torch.bfloat16, device=x.device)
    _need(out, "out", (torch.bfloat16,), n_heads * n_rows * head_dim)
    need = project_rope_workspace(n_rows, hidden, n_heads, head_dim)
    if ws is None and need > 0:
        ws = torch.empty(need, dtype=torch.uint8, device=x.device)
    _lib.check(_lib.lib().dge_project_rope(n_rows, hidden, _ptr(x), n_heads, head_dim, _ptr(w),
                                           _ptr(positions), float(theta), _ptr(out), _ptr(ws),
                                           0 if ws is None else ws.numel() * ws.element_size(),
                                           _stream(stream)), "dge_project_rope")
    return out


def retained_runs(geom: Geometry, idx, n_kept, runs=None, mean_len=None, stream=None):
    """dge_retained_runs: contiguity of the selected sets.  idx [batch][H_kv][n_select]
    int32 (ascending rows, as select_topb writes them), n_kept [batch].  Returns
    (runs [batch][H_kv] int32, mean_len [batch][H_kv] float32)."""
    torch = _torch()
    n_select = int(idx.shape[-1])
    if runs is None:
        runs = torch.empty(geom.batch, geom.n_kv_heads, dtype=torch.int32, device=geom.device)
    if mean_len is None:
        mean_len = torch.empty(geom.batch, geom.n_kv_heads, dtype=torch.float32,
                               device=geom.device)
    _need(idx, "idx", _i32(), geom.batch * geom.n_kv_heads * n_select)
    _need(n_kept, "n_kept", _i32(), geom.batch)
    _lib.check(_lib.lib().dge_retained_runs(ctypes.byref(geom.c), _ptr(idx), _ptr(n_kept),
                                            n_select, _ptr(runs), _ptr(mean_len),
                                            _stream(stream)), "dge_retained_runs")
    return runs, mean_len


def h2o_colsum(geom: Geometry, q_all, k, lse=None, colsum=None, ws=None, stream=None):
    """dge_h2o_colsum: H2O accumulated attention.  Returns colsum [H_kv][T] float32."""
    torch = _torch()
    if colsum is None:
        colsum = torch.empty(geom.n_kv_heads, geom.total_rows, dtype=torch.float32,
                             device=geom.device)
    _need(q_all, "q_all", (geom.elt_dtype,), geom.n_q_heads * geom.total_rows * geom.head_dim)
    _need(k, "k", (geom.elt_dtype,), (geom.n_kv_heads - 1) * geom.kv_head_stride
          + geom.total_rows * geom.head_dim)
    _need(lse, "lse", _f32(), geom.n_q_heads * geom.total_rows, optional=True)
    _need(colsum, "colsum", _f32(), geom.n_kv_heads * geom.total_rows)
    ws = _workspace(geom, OP_H2O, ws)
    nbytes = ws.numel()
    _lib.check(_lib.lib().dge_h2o_colsum(ctypes.byref(geom.c), _ptr(q_all), _ptr(k), _ptr(lse),
                                         _ptr(colsum), _ptr(ws), nbytes, _stream(stream)),
               "dge_h2o_colsum")
    return colsum


def pyramid_budgets(B: int, w: int, n_layers: int, beta: int = 20) -> list:
    """dge_pyramid_budgets (host): PyramidKV per-layer total budgets B_l."""
    out = (ctypes.c_int32 * max(n_layers, 1))()
    _lib.check(_lib.lib().dge_pyramid_budgets(B, w, n_layers, beta, out), "dge_pyramid_budgets")
    return list(out)[:n_layers]


def evict_layer(geom: Geometry, q, k, v, budget: int, pool_kernel: int, rows: int = ROWS_WINDOW_DRAFT,
                stream=None, ws_score=None, ws_select=None, out=None, fused: bool = True):
    """score -> select (B - w, tail w + k) -> compact for one layer.

    ``fused`` runs selection and compaction as dge_select_compact, otherwise as
    dge_select_topb then dge_compact.  Returns dict(raw, idx, n_kept, k, v); ``out``
    may hold preallocated tensors under the same keys.
    """
    out = out or {}
    n_tail = geom.window + geom.k_draft
    n_select = budget - geom.window
    raw = score(geom, rows, q, k, raw=out.get("raw"), ws=ws_score, stream=stream)
    if fused:
        idx, n_kept, k_out, v_out = select_compact(
            geom, raw, pool_kernel, n_tail, n_select, k, v, idx=out.get("idx"),
            n_kept=out.get("n_kept"), k_out=out.get("k"), v_out=out.get("v"), ws=ws_select,
            stream=stream)
    else:
        idx, n_kept = select_topb(geom, raw, pool_kernel, n_tail, n_select, idx=out.get("idx"),
                                  n_kept=out.get("n_kept"), ws=ws_select, stream=stream)
        k_out, v_out = compact(geom, idx, n_kept, n_select, n_tail, k, v, k_out=out.get("k"),
                               v_out=out.get("v"), stream=stream)
    return dict(raw=raw, idx=idx, n_kept=n_kept, k=k_out, v=v_out)
