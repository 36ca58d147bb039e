"""Thin Python binding of liblsa.so (the C-ABI in include/lsa.h).

Argument marshalling only: every step of the hot path runs in the HIP library. PyTorch provides
device memory and the current stream. Importing this module does not load the library; the
first call does, and raises if liblsa.so has not been built (there is no fallback).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblsa.so")

LSA_KEY_BF16 = 0
LSA_KEY_FP8_E4M3FN = 1
POOLING = {"mean": 0, "minmax": 1}   # lsa_pooling


class LSAError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        super().__init__(f"{where}: {message} (status {status})")
        self.status = status


class _IndexParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_heads", "head_dim", "key_dtype", "page", "sub_block", "keep_pages",
        "k_sparse", "k_sink", "k_swa", "run_align", "pooling", "hi_min_kv")]


class _AttnParams(ctypes.Structure):
    _fields_ = [("n_heads", ctypes.c_int32), ("d_qk", ctypes.c_int32), ("d_v", ctypes.c_int32),
                ("latent", ctypes.c_int32), ("sm_scale", ctypes.c_float)]


@dataclass(frozen=True)
class IndexParams:
    """Indexer hyper-parameters (Sec. 3.1 and 3.3 of the paper); see lsa_index_params."""
    n_heads: int
    head_dim: int
    fp8: bool
    page: int
    sub_block: int
    keep_pages: int
    k_sparse: int
    k_sink: int
    k_swa: int
    run_align: int
    pooling: str = "mean"    # coarse-stage block summary: "mean" (Eq. 9) or "minmax" (Eq. 13)
    hi_min_kv: int = 0       # adaptive dispatch: caches of at most this many tokens are indexed flat

    @property
    def k_cap(self) -> int:
        return self.k_sink + self.k_swa + self.k_sparse

    @property
    def block_width(self) -> int:
        """Columns of one block-cache row: d_I (mean keys) or 2 d_I ([k_max | k_min])."""
        return 2 * self.head_dim if self.pooling == "minmax" else self.head_dim

    def c(self) -> _IndexParams:
        return _IndexParams(self.n_heads, self.head_dim, LSA_KEY_FP8_E4M3FN if self.fp8 else LSA_KEY_BF16,
                            self.page, self.sub_block, self.keep_pages, self.k_sparse, self.k_sink,
                            self.k_swa, self.run_align, POOLING[self.pooling], self.hi_min_kv)


@dataclass(frozen=True)
class AttnParams:
    n_heads: int
    d_qk: int
    d_v: int
    latent: bool
    sm_scale: float

    def c(self) -> _AttnParams:
        return _AttnParams(self.n_heads, self.d_qk, self.d_v, int(self.latent), self.sm_scale)


MLA = dict(n_heads=64, d_qk=576, d_v=512, latent=True)
MQA = dict(n_heads=16, d_qk=128, d_v=128, latent=False)

_lib = None
_vp, _i32, _i64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t


def lib() -> ctypes.CDLL:
    """Load liblsa.so (once). Raises when it is missing: the product path has no fallback."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing; build it with `python -m paper_2608_01662_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER(_IndexParams)
        A = ctypes.POINTER(_AttnParams)
        L.lsa_index_k_cap.argtypes = [P]
        L.lsa_index_k_cap.restype = _i32
        L.lsa_index_workspace_size.argtypes = [P, _i64, _i64]
        L.lsa_index_workspace_size.restype = _sz
        L.lsa_block_means.argtypes = [P, _i64, _vp, _vp, _vp, _vp]
        L.lsa_block_means.restype = _i32
        L.lsa_block_minmax.argtypes = [P, _i64, _vp, _vp, _vp, _vp]
        L.lsa_block_minmax.restype = _i32
        L.lsa_block_keys_update.argtypes = [P, _i64, _vp, _i64, _vp, _vp, _vp, _vp]
        L.lsa_block_keys_update.restype = _i32
        L.lsa_index_prefill.argtypes = [P, _i64, _i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                        _vp, _sz, _vp]
        L.lsa_index_prefill.restype = _i32
        L.lsa_index_decode.argtypes = [P, _i32, _vp, _vp, _i32, _i32, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                       _vp, _vp, _vp, _vp, _sz, _vp]
        L.lsa_index_decode.restype = _i32
        L.lsa_index_decode_static.argtypes = [P, _i32, _vp, _vp, _i32, _i32, _i64, _vp, _vp, _vp, _vp, _vp, _vp,
                                              _vp, _vp, _vp, _vp, _vp]
        L.lsa_index_decode_static.restype = _i32
        L.lsa_sparse_attn_workspace_size.argtypes = [A, _i64, _i32, _i32]
        L.lsa_sparse_attn_workspace_size.restype = _sz
        L.lsa_sparse_attn.argtypes = [A, _i64, _vp, _vp, _vp, _i64, _vp, _vp, _i32, _vp, _i32, _i32, _i32, _vp,
                                      _vp, _vp, _sz, _vp]
        L.lsa_sparse_attn.restype = _i32
        L.lsa_sparse_attn_runs_workspace_size.argtypes = [A, _i64, _i32, _i32]
        L.lsa_sparse_attn_runs_workspace_size.restype = _sz
        L.lsa_sparse_attn_runs.argtypes = [A, _i64, _vp, _vp, _vp, _i64, _vp, _vp, _i32, _vp, _i32, _i32, _i32,
                                           _vp, _vp, _vp, _sz, _vp]
        L.lsa_sparse_attn_runs.restype = _i32
        L.lsa_hfa_attn_workspace_size.argtypes = [A, _i64]
        L.lsa_hfa_attn_workspace_size.restype = _sz
        L.lsa_hfa_attn.argtypes = [A, _i64, _vp, _vp, _i64, _vp, _vp, _i32, _i64, _i32, _vp, _vp, _vp, _sz, _vp]
        L.lsa_hfa_attn.restype = _i32
        L.lsa_status_string.argtypes = [_i32]
        L.lsa_status_string.restype = ctypes.c_char_p
        L.lsa_last_error.argtypes = []
        L.lsa_last_error.restype = ctypes.c_char_p
        L.lsa_version.argtypes = []
        L.lsa_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(status: int, where: str) -> None:
    if status != 0:
        L = lib()
        raise LSAError(status, where, (L.lsa_last_error() or b"").decode() or
                       L.lsa_status_string(status).decode())


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


_BF16, _F32, _I32, _I64, _U8 = (torch.bfloat16,), (torch.float32,), (torch.int32,), (torch.int64,), (torch.uint8,)


def _need(name: str, t, dtypes, shape=None, device=None, min_rows: int | None = None):
    """The C ABI receives bare pointers, so the sizes it is told must match the tensors behind
    them: `t` must be a contiguous CUDA tensor of one of `dtypes` on `device`, of exactly `shape`
    (None entries match any size), with at least `min_rows` rows. Raises ValueError otherwise."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if not t.is_cuda or (device is not None and t.device != torch.device(device)):
        raise ValueError(f"{name} must be a CUDA tensor on {device or 'a GPU'} (got {t.device})")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {' or '.join(str(d) for d in dtypes)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and (t.dim() != len(shape) or any(s is not None and d != s for d, s in zip(t.shape, shape))):
        want = tuple("*" if s is None else s for s in shape)
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {want}")
    if min_rows is not None and t.shape[0] < min_rows:
        raise ValueError(f"{name} has {t.shape[0]} rows, at least {min_rows} needed")
    return t


def _need_opt(name: str, t, *args, **kw):
    return None if t is None else _need(name, t, *args, **kw)


def _key_dtypes(prm: "IndexParams"):
    return _U8 if prm.fp8 else _BF16


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _keys_u8_or_bf16(k: torch.Tensor) -> torch.Tensor:
    if k.dtype == torch.float8_e4m3fn:
        return k.view(torch.uint8)
    return k


def _workspace(nbytes: int, device, ws):
    if nbytes == 0:
        return None, 0
    if ws is not None:
        _need("workspace", ws, tuple({ws.dtype}), device=device)
        return ws, ws.numel() * ws.element_size()
    return torch.empty(nbytes, dtype=torch.uint8, device=device), nbytes


def index_workspace_size(prm: IndexParams, n_rows: int, max_kv: int) -> int:
    return int(lib().lsa_index_workspace_size(ctypes.byref(prm.c()), n_rows, max_kv))


def attn_workspace_size(prm: AttnParams, n_rows: int, k_cap: int, paged: bool) -> int:
    return int(lib().lsa_sparse_attn_workspace_size(ctypes.byref(prm.c()), n_rows, k_cap, int(paged)))


def block_means(prm: IndexParams, k: torch.Tensor, k_scale: torch.Tensor | None = None,
                out: torch.Tensor | None = None) -> torch.Tensor:
    """Mean-key cache of the coarse stage: [n_tok // sub_block, head_dim] bf16."""
    k = _need("k", _keys_u8_or_bf16(k), _key_dtypes(prm), (None, prm.head_dim))
    n_tok = k.shape[0]
    _need_opt("k_scale", k_scale, _F32, (n_tok,), k.device)
    if out is None:
        out = torch.empty((n_tok // prm.sub_block, prm.head_dim), dtype=torch.bfloat16, device=k.device)
    _need("out", out, _BF16, (n_tok // prm.sub_block, prm.head_dim), k.device)
    _check(lib().lsa_block_means(ctypes.byref(prm.c()), n_tok, _p(k), _p(k_scale), _p(out), _stream(k.device)),
           "lsa_block_means")
    return out


def block_minmax(prm: IndexParams, k: torch.Tensor, k_scale: torch.Tensor | None = None,
                 out: torch.Tensor | None = None) -> torch.Tensor:
    """Min-max block cache (Eq. 13): [n_tok // sub_block, 2 * head_dim] bf16 rows [k_max | k_min]."""
    k = _need("k", _keys_u8_or_bf16(k), _key_dtypes(prm), (None, prm.head_dim))
    n_tok = k.shape[0]
    _need_opt("k_scale", k_scale, _F32, (n_tok,), k.device)
    if out is None:
        out = torch.empty((n_tok // prm.sub_block, 2 * prm.head_dim), dtype=torch.bfloat16, device=k.device)
    _need("out", out, _BF16, (n_tok // prm.sub_block, 2 * prm.head_dim), k.device)
    _check(lib().lsa_block_minmax(ctypes.byref(prm.c()), n_tok, _p(k), _p(k_scale), _p(out), _stream(k.device)),
           "lsa_block_minmax")
    return out


def block_keys(prm: IndexParams, k: torch.Tensor, k_scale: torch.Tensor | None = None,
               out: torch.Tensor | None = None) -> torch.Tensor:
    """The block cache the coarse stage of `prm` reads: mean keys or min-max extrema."""
    return (block_minmax if prm.pooling == "minmax" else block_means)(prm, k, k_scale, out)


def block_keys_update(prm: IndexParams, rows: torch.Tensor, k: torch.Tensor, k_scale: torch.Tensor | None,
                      block: torch.Tensor) -> torch.Tensor:
    """Recompute, in place, the block-cache rows of the sub-blocks holding token rows `rows` (int64)."""
    k = _need("k", _keys_u8_or_bf16(k), _key_dtypes(prm), (None, prm.head_dim))
    _need("rows", rows, _I64, (None,), k.device)
    _need_opt("k_scale", k_scale, _F32, (k.shape[0],), k.device)
    _need("block", block, _BF16, (k.shape[0] // prm.sub_block, prm.block_width), k.device)
    _check(lib().lsa_block_keys_update(ctypes.byref(prm.c()), rows.numel(), _p(rows), k.shape[0], _p(k),
                                       _p(k_scale), _p(block), _stream(k.device)), "lsa_block_keys_update")
    return block


def _index_outputs(prm: IndexParams, n_rows: int, device, runs: bool, pages: bool, out: dict | None):
    out = dict(out or {})
    kc = prm.k_cap
    out.setdefault("idx", torch.empty((n_rows, kc), dtype=torch.int32, device=device))
    out.setdefault("count", torch.empty((n_rows,), dtype=torch.int32, device=device))
    if runs:
        out.setdefault("runs", torch.empty((n_rows, kc, 2), dtype=torch.int32, device=device))
        out.setdefault("run_count", torch.empty((n_rows,), dtype=torch.int32, device=device))
    if pages and prm.keep_pages > 0:
        out.setdefault("pages", torch.empty((n_rows, prm.keep_pages), dtype=torch.int32, device=device))
    shapes = {"idx": (n_rows, kc), "count": (n_rows,), "runs": (n_rows, kc, 2), "run_count": (n_rows,),
              "pages": (n_rows, prm.keep_pages)}
    for key, t in out.items():
        if key not in shapes:
            raise ValueError(f"unknown output {key!r} (expected {', '.join(shapes)})")
        _need(f"out[{key!r}]", t, _I32, shapes[key], device)
    return out


def index_prefill(prm: IndexParams, q: torch.Tensor, w: torch.Tensor, k: torch.Tensor,
                  k_scale: torch.Tensor | None, block_keys: torch.Tensor | None, q_start: int,
                  n_kv: int | None = None, runs: bool = True, pages: bool = False,
                  workspace: torch.Tensor | None = None, out: dict | None = None) -> dict:
    """LSA indexer for query rows at positions q_start .. q_start + n_q - 1 (lsa_index_prefill)."""
    k = _keys_u8_or_bf16(k)
    _need("q", q, _BF16, (None, prm.n_heads, prm.head_dim))
    n_q, dev = q.shape[0], q.device
    n_kv = k.shape[0] if n_kv is None else n_kv
    _need("w", w, _F32, (n_q, prm.n_heads), dev)
    _need("k", k, _key_dtypes(prm), (None, prm.head_dim), dev, min_rows=n_kv)
    if prm.fp8:
        _need("k_scale", k_scale, _F32, (None,), dev, min_rows=n_kv)
    _need_opt("block_keys", block_keys, _BF16, (None, prm.block_width), dev, min_rows=n_kv // prm.sub_block)
    o = _index_outputs(prm, n_q, q.device, runs, pages, out)
    ws, wsb = _workspace(index_workspace_size(prm, n_q, n_kv), q.device, workspace)
    _check(lib().lsa_index_prefill(ctypes.byref(prm.c()), q_start, n_q, n_kv, _p(q), _p(w), _p(k), _p(k_scale),
                                   _p(block_keys), _p(o["idx"]), _p(o["count"]), _p(o.get("runs")),
                                   _p(o.get("run_count")), _p(o.get("pages")), _p(ws), wsb, _stream(q.device)),
           "lsa_index_prefill")
    return o


def index_decode(prm: IndexParams, ctx_len: torch.Tensor, page_table: torch.Tensor, kv_page_size: int,
                 n_phys: int, q: torch.Tensor, w: torch.Tensor, k: torch.Tensor, k_scale: torch.Tensor | None,
                 block_keys: torch.Tensor | None, runs: bool = True, pages: bool = False,
                 workspace: torch.Tensor | None = None, out: dict | None = None) -> dict:
    """LSA indexer for one new token per sequence over a paged key cache (lsa_index_decode)."""
    k = _keys_u8_or_bf16(k)
    _need("page_table", page_table, _I32, (None, None))
    batch, max_pages = page_table.shape
    dev = page_table.device
    _need("ctx_len", ctx_len, _I32, (batch,), dev)
    _need("q", q, _BF16, (batch, prm.n_heads, prm.head_dim), dev)
    _need("w", w, _F32, (batch, prm.n_heads), dev)
    n_cached = n_phys * kv_page_size
    _need("k", k, _key_dtypes(prm), None, dev)
    if k.shape[-1] != prm.head_dim or k.numel() < n_cached * prm.head_dim:
        raise ValueError(f"k must hold n_phys * kv_page_size = {n_cached} key rows of {prm.head_dim}")
    if prm.fp8:
        _need("k_scale", k_scale, _F32, None, dev)
        if k_scale.numel() < n_cached:
            raise ValueError(f"k_scale must hold {n_cached} scales")
    _need_opt("block_keys", block_keys, _BF16, (None, prm.block_width), dev, min_rows=n_cached // prm.sub_block)
    o = _index_outputs(prm, batch, q.device, runs, pages, out)
    ws, wsb = _workspace(index_workspace_size(prm, batch, max_pages * kv_page_size), q.device, workspace)
    _check(lib().lsa_index_decode(ctypes.byref(prm.c()), batch, _p(ctx_len), _p(page_table), max_pages,
                                  kv_page_size, n_phys, _p(q), _p(w), _p(k), _p(k_scale), _p(block_keys),
                                  _p(o["idx"]), _p(o["count"]), _p(o.get("runs")), _p(o.get("run_count")),
                                  _p(o.get("pages")), _p(ws), wsb, _stream(q.device)),
           "lsa_index_decode")
    return o


def index_decode_static(prm: IndexParams, ctx_len: torch.Tensor, page_table: torch.Tensor, kv_page_size: int,
                        n_phys: int, q: torch.Tensor, w: torch.Tensor, k: torch.Tensor, k_scale: torch.Tensor | None,
                        block_keys: torch.Tensor | None, out: dict) -> dict:
    """lsa_index_decode_static: the decode indexer with its scratch in the library's fixed device
    array (no workspace). `out` holds preallocated outputs (idx, count, and optionally runs +
    run_count and pages), so that this call allocates nothing either."""
    k = _keys_u8_or_bf16(k)
    _need("page_table", page_table, _I32, (None, None))
    batch, max_pages = page_table.shape
    dev = page_table.device
    _need("ctx_len", ctx_len, _I32, (batch,), dev)
    _need("q", q, _BF16, (batch, prm.n_heads, prm.head_dim), dev)
    _need("w", w, _F32, (batch, prm.n_heads), dev)
    n_cached = n_phys * kv_page_size
    _need("k", k, _key_dtypes(prm), None, dev)
    if k.shape[-1] != prm.head_dim or k.numel() < n_cached * prm.head_dim:
        raise ValueError(f"k must hold n_phys * kv_page_size = {n_cached} key rows of {prm.head_dim}")
    if prm.fp8:
        _need("k_scale", k_scale, _F32, None, dev)
        if k_scale.numel() < n_cached:
            raise ValueError(f"k_scale must hold {n_cached} scales")
    _need_opt("block_keys", block_keys, _BF16, (None, prm.block_width), dev, min_rows=n_cached // prm.sub_block)
    if out is None or "idx" not in out or "count" not in out:
        raise ValueError("index_decode_static needs preallocated outputs (out['idx'], out['count'])")
    o = _index_outputs(prm, batch, q.device, "runs" in out, "pages" in out, out)
    _check(lib().lsa_index_decode_static(ctypes.byref(prm.c()), batch, _p(ctx_len), _p(page_table), max_pages,
                                         kv_page_size, n_phys, _p(q), _p(w), _p(k), _p(k_scale), _p(block_keys),
                                         _p(o["idx"]), _p(o["count"]), _p(o.get("runs")), _p(o.get("run_count")),
                                         _p(o.get("pages")), _stream(q.device)),
           "lsa_index_decode_static")
    return o


def _attn_io(prm: AttnParams, q, kv, out, lse, paged: bool):
    """Checks q and kv, allocates out / lse when asked to; returns (n_rows, n_kv_rows, out, lse)."""
    _need("q", q, _BF16, (None, prm.n_heads, prm.d_qk))
    n_rows, dev = q.shape[0], q.device
    _need("kv", kv, _BF16, (None, None, prm.d_qk) if paged else (None, prm.d_qk), dev)
    n_kv_rows = kv.shape[0] * (kv.shape[1] if paged else 1)
    if out is None:
        out = torch.empty((n_rows, prm.n_heads, prm.d_v), dtype=torch.bfloat16, device=dev)
    _need("out", out, _BF16, (n_rows, prm.n_heads, prm.d_v), dev)
    if lse is True:
        lse = torch.empty((n_rows, prm.n_heads), dtype=torch.float32, device=dev)
    elif lse is False:
        lse = None
    _need_opt("lse", lse, _F32, (n_rows, prm.n_heads), dev)
    return n_rows, n_kv_rows, out, lse


def sparse_attn(prm: AttnParams, q: torch.Tensor, kv: torch.Tensor, v: torch.Tensor | None,
                idx: torch.Tensor, count: torch.Tensor, page_table: torch.Tensor | None = None,
                kv_page_size: int = 0, rows_per_seq: int = 1, out: torch.Tensor | None = None,
                lse: torch.Tensor | bool | None = True, workspace: torch.Tensor | None = None):
    """Sparse attention over idx (lsa_sparse_attn). Returns (out [n_rows, H, d_v] bf16, lse or None).

    kv: contiguous [n_kv_rows, d_qk] or paged [n_phys, page, d_qk] (then page_table is required)."""
    paged = page_table is not None
    n_rows, n_kv_rows, out, lse = _attn_io(prm, q, kv, out, lse, paged)
    dev = q.device
    if prm.latent:
        if v is not None:
            raise ValueError("v must be None with a latent cache (V is the first d_v columns of kv)")
    else:
        _need("v", v, _BF16, tuple(kv.shape[:-1]) + (prm.d_v,), dev)
    _need("idx", idx, _I32, (n_rows, None), dev)
    k_cap = idx.shape[1]
    _need("count", count, _I32, (n_rows,), dev)
    if paged:
        if kv.shape[1] != kv_page_size:
            raise ValueError(f"paged kv has pages of {kv.shape[1]} rows, kv_page_size is {kv_page_size}")
        if rows_per_seq < 1:
            raise ValueError("rows_per_seq must be >= 1")
        _need("page_table", page_table, _I32, (None, None), dev, min_rows=-(-n_rows // rows_per_seq))
    max_pages = page_table.shape[1] if paged else 0
    ws, wsb = _workspace(attn_workspace_size(prm, n_rows, k_cap, page_table is not None), q.device, workspace)
    _check(lib().lsa_sparse_attn(ctypes.byref(prm.c()), n_rows, _p(q), _p(kv), _p(v), n_kv_rows, _p(idx),
                                 _p(count), k_cap, _p(page_table), max_pages, kv_page_size, rows_per_seq,
                                 _p(out), _p(lse), _p(ws), wsb, _stream(q.device)),
           "lsa_sparse_attn")
    return out, lse


def attn_runs_workspace_size(prm: AttnParams, n_rows: int, k_cap: int, paged: bool) -> int:
    return int(lib().lsa_sparse_attn_runs_workspace_size(ctypes.byref(prm.c()), n_rows, k_cap, int(paged)))


def sparse_attn_runs(prm: AttnParams, q: torch.Tensor, kv: torch.Tensor, runs: torch.Tensor, run_count: torch.Tensor,
                     out: torch.Tensor | None = None, lse: torch.Tensor | bool | None = True,
                     workspace: torch.Tensor | None = None, v: torch.Tensor | None = None,
                     page_table: torch.Tensor | None = None, kv_page_size: int = 0, rows_per_seq: int = 1):
    """Sparse attention over the run form of the lists (lsa_sparse_attn_runs): runs [n_rows, k_cap, 2]
    int32 (start, length) as the indexer returns them, run_count [n_rows]. Other arguments as
    sparse_attn. Returns (out, lse or None)."""
    paged = page_table is not None
    n_rows, n_kv_rows, out, lse = _attn_io(prm, q, kv, out, lse, paged)
    dev = q.device
    if prm.latent:
        if v is not None:
            raise ValueError("v must be None with a latent cache (V is the first d_v columns of kv)")
    else:
        _need("v", v, _BF16, tuple(kv.shape[:-1]) + (prm.d_v,), dev)
    _need("runs", runs, _I32, (n_rows, None, 2), dev)
    k_cap = runs.shape[1]
    _need("run_count", run_count, _I32, (n_rows,), dev)
    if paged:
        if kv.shape[1] != kv_page_size:
            raise ValueError(f"paged kv has pages of {kv.shape[1]} rows, kv_page_size is {kv_page_size}")
        if rows_per_seq < 1:
            raise ValueError("rows_per_seq must be >= 1")
        _need("page_table", page_table, _I32, (None, None), dev, min_rows=-(-n_rows // rows_per_seq))
    max_pages = page_table.shape[1] if paged else 0
    ws, wsb = _workspace(attn_runs_workspace_size(prm, n_rows, k_cap, paged), dev, workspace)
    _check(lib().lsa_sparse_attn_runs(ctypes.byref(prm.c()), n_rows, _p(q), _p(kv), _p(v), n_kv_rows, _p(runs),
                                      _p(run_count), k_cap, _p(page_table), max_pages, kv_page_size, rows_per_seq,
                                      _p(out), _p(lse), _p(ws), wsb, _stream(dev)),
           "lsa_sparse_attn_runs")
    return out, lse


def hfa_workspace_size(prm: AttnParams, n_rows: int) -> int:
    return int(lib().lsa_hfa_attn_workspace_size(ctypes.byref(prm.c()), n_rows))


def hfa_attn(prm: AttnParams, q: torch.Tensor, kv: torch.Tensor, idx: torch.Tensor, count: torch.Tensor,
             q_start: int, k_swa: int, out: torch.Tensor | None = None, lse: torch.Tensor | bool | None = True,
             workspace: torch.Tensor | None = None):
    """Split attention (lsa_hfa_attn): listed non-window part and contiguous window on two streams,
    merged by log-sum-exp rescaling. Returns (out, lse or None) as sparse_attn."""
    n_rows, n_kv_rows, out, lse = _attn_io(prm, q, kv, out, lse, False)
    _need("idx", idx, _I32, (n_rows, None), q.device)
    k_cap = idx.shape[1]
    _need("count", count, _I32, (n_rows,), q.device)
    ws, wsb = _workspace(hfa_workspace_size(prm, n_rows), q.device, workspace)
    _check(lib().lsa_hfa_attn(ctypes.byref(prm.c()), n_rows, _p(q), _p(kv), n_kv_rows, _p(idx), _p(count), k_cap,
                              q_start, k_swa, _p(out), _p(lse), _p(ws), wsb, _stream(q.device)), "lsa_hfa_attn")
    return out, lse


def version() -> str:
    return lib().lsa_version().decode()
