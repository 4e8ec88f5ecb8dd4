"""ctypes binding of libconduit (include/conduit.h) over torch device tensors.

Argument marshalling only: every step of the refresh step runs in the HIP
library.  torch provides device memory and the current stream; no torch
compute is used on the path.  If the library is missing, the first call raises
ConduitError (there is no fallback).
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libconduit.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(5)
F32, BF16 = 0, 1
NORM_CAUSAL_ROW, NORM_VISUAL_ONLY = 0, 1
AGG_MEAN, AGG_RMS = 0, 1
RANK_COMPOSITE, RANK_ATTENTION, RANK_EXPLICIT = 0, 1, 2
MAX_IMAGES = 256

EXPORTS = [
    "conduit_budget", "conduit_score_workspace_bytes", "conduit_score",
    "conduit_select_workspace_bytes", "conduit_select_topk", "conduit_scatter_kv",
    "conduit_refresh_workspace_bytes", "conduit_refresh_attn", "conduit_status_str",
    "conduit_last_error", "conduit_version", "conduit_profile_enable", "conduit_profile_count",
    "conduit_profile_read", "conduit_value_norms", "conduit_residual_workspace_bytes",
    "conduit_residual_error", "conduit_score_noalloc", "conduit_scatter_kv_layers",
    "conduit_refresh_layers_workspace_bytes", "conduit_refresh_attn_layers",
    "conduit_score_layers_workspace_bytes", "conduit_score_layers", "conduit_merge_refresh_attn",
]
SCORE_NOALLOC_MAX_BYTES = 16 << 20


class ConduitError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        super().__init__(f"{_status_name(status)}: {detail}")


class KV(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("k_stride", ctypes.c_int64),
                ("v_stride", ctypes.c_int64), ("n_ctx", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("block_table", ctypes.c_void_p),
                ("n_pages", ctypes.c_int32)]


class Images(ctypes.Structure):
    _fields_ = [("n_images", ctypes.c_int32), ("n_vis", ctypes.c_int32),
                ("img_pos", ctypes.POINTER(ctypes.c_int32)),
                ("img_off", ctypes.POINTER(ctypes.c_int32))]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libconduit.so (built in-tree by __graft_entry__.build())."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ConduitError(ERR_HIP, f"{LIB_PATH} is not built (run __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, f32, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                 ctypes.c_size_t)
        pkv, pimg = ctypes.POINTER(KV), ctypes.POINTER(Images)
        L.conduit_budget.argtypes = [i64, i64, i64]
        L.conduit_budget.restype = i64
        L.conduit_score_workspace_bytes.argtypes = [pkv, i32, pimg]
        L.conduit_score_workspace_bytes.restype = sz
        L.conduit_score.argtypes = [pkv, vp, i32, i32, pimg, ctypes.c_int, ctypes.c_int, f32, vp, vp,
                                    vp, vp, vp, i32, vp, vp, vp, sz, vp]
        L.conduit_score.restype = ctypes.c_int
        L.conduit_score_noalloc.argtypes = [pkv, vp, i32, i32, pimg, ctypes.c_int, ctypes.c_int, f32, vp,
                                            vp, vp, vp, vp, i32, vp, vp, vp]
        L.conduit_score_noalloc.restype = ctypes.c_int
        L.conduit_select_workspace_bytes.argtypes = [i32, i32]
        L.conduit_select_workspace_bytes.restype = sz
        L.conduit_select_topk.argtypes = [vp, vp, i32, pimg, f32, ctypes.c_int, i32, vp, vp, vp, vp,
                                          vp, vp, vp, sz, vp]
        L.conduit_value_norms.argtypes = [pkv, pimg, vp, vp]
        L.conduit_residual_workspace_bytes.argtypes = [pkv, i32, pimg, i32, i32]
        L.conduit_residual_workspace_bytes.restype = sz
        L.conduit_residual_error.argtypes = [pkv, vp, i32, i32, pimg, f32, vp, vp, vp, i32, f32, vp, vp,
                                             sz, vp]
        L.conduit_residual_error.restype = ctypes.c_int
        L.conduit_value_norms.restype = ctypes.c_int
        L.conduit_select_topk.restype = ctypes.c_int
        L.conduit_scatter_kv.argtypes = [pkv, vp, i32, vp, vp, vp, vp, vp]
        L.conduit_scatter_kv.restype = ctypes.c_int
        L.conduit_refresh_workspace_bytes.argtypes = [pkv, i32]
        L.conduit_refresh_workspace_bytes.restype = sz
        L.conduit_refresh_attn.argtypes = [pkv, vp, vp, i32, f32, vp, vp, vp, sz, vp]
        L.conduit_refresh_attn.restype = ctypes.c_int
        L.conduit_merge_refresh_attn.argtypes = [pkv, vp, i32, vp, vp, vp, f32, vp, vp, vp, sz, vp]
        L.conduit_merge_refresh_attn.restype = ctypes.c_int
        pvp = ctypes.POINTER(ctypes.c_void_p)
        L.conduit_scatter_kv_layers.argtypes = [pkv, i32, vp, i32, pvp, pvp, vp]
        L.conduit_scatter_kv_layers.restype = ctypes.c_int
        L.conduit_refresh_layers_workspace_bytes.argtypes = [pkv, i32, i32]
        L.conduit_refresh_layers_workspace_bytes.restype = sz
        L.conduit_refresh_attn_layers.argtypes = [pkv, i32, pvp, vp, i32, f32, pvp, pvp, vp, sz, vp]
        L.conduit_refresh_attn_layers.restype = ctypes.c_int
        L.conduit_score_layers_workspace_bytes.argtypes = [pkv, i32, pimg, i32]
        L.conduit_score_layers_workspace_bytes.restype = sz
        L.conduit_score_layers.argtypes = [pkv, i32, pvp, i32, i32, pimg, ctypes.c_int, ctypes.c_int, f32, pvp,
                                           vp, vp, i32, vp, sz, vp]
        L.conduit_score_layers.restype = ctypes.c_int
        L.conduit_status_str.argtypes = [ctypes.c_int]
        L.conduit_status_str.restype = ctypes.c_char_p
        L.conduit_last_error.argtypes = []
        L.conduit_last_error.restype = ctypes.c_char_p
        L.conduit_version.argtypes = []
        L.conduit_version.restype = ctypes.c_char_p
        L.conduit_profile_enable.argtypes = [i32]
        L.conduit_profile_enable.restype = ctypes.c_int
        L.conduit_profile_count.argtypes = []
        L.conduit_profile_count.restype = i32
        L.conduit_profile_read.argtypes = [i32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(f32)]
        L.conduit_profile_read.restype = ctypes.c_int
        _lib = L
    return _lib


def _status_name(status: int) -> str:
    try:
        return lib().conduit_status_str(status).decode()
    except Exception:  # noqa: BLE001 - naming must never mask the real error
        return f"status {status}"


def _check(status: int) -> None:
    if status != OK:
        raise ConduitError(status, lib().conduit_last_error().decode())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise ConduitError(ERR_UNSUPPORTED, f"cache dtype {t.dtype} (bfloat16 or float32)")


def kv_desc(k: torch.Tensor, v: torch.Tensor, n_q_heads: int) -> KV:
    """Descriptor of one layer's cache: k, v are [n_ctx, H_kv, d] device tensors
    whose last two dims are dense (any token stride)."""
    for t in (k, v):
        if t.dim() != 3 or t.stride(2) != 1 or t.stride(1) != t.shape[2]:
            raise ConduitError(ERR_INVALID_ARG, "cache tensors must be [n_ctx, H_kv, d], rows dense")
    if k.shape != v.shape or k.dtype != v.dtype:
        raise ConduitError(ERR_INVALID_ARG, "k and v must match in shape and dtype")
    n_ctx, hkv, d = k.shape
    return KV(k.data_ptr(), v.data_ptr(), k.stride(0), v.stride(0), n_ctx, n_q_heads, hkv, d,
              _dtype_code(k), 0, None, 0)


def kv_desc_paged(k_pages: torch.Tensor, v_pages: torch.Tensor, block_table: torch.Tensor,
                  n_ctx: int, n_q_heads: int) -> KV:
    """Descriptor of one layer's paged cache: k_pages, v_pages are
    [n_pages, page_size, H_kv, d] device tensors (last two dims dense, pages
    evenly strided); block_table is a device int32 tensor whose entry i is the
    page holding tokens i*page_size .. (i+1)*page_size - 1."""
    for t in (k_pages, v_pages):
        if t.dim() != 4 or t.stride(3) != 1 or t.stride(2) != t.shape[3] or \
                t.stride(0) != t.shape[1] * t.stride(1):
            raise ConduitError(ERR_INVALID_ARG, "page tensors must be [n_pages, page, H_kv, d], rows dense")
    if k_pages.shape != v_pages.shape or k_pages.dtype != v_pages.dtype:
        raise ConduitError(ERR_INVALID_ARG, "k and v pages must match in shape and dtype")
    n_pages, page, hkv, d = k_pages.shape
    if block_table.dtype != torch.int32 or block_table.dim() != 1 or \
            block_table.numel() < -(-n_ctx // page):
        raise ConduitError(ERR_INVALID_ARG, "block_table must be int32 with ceil(n_ctx / page) entries")
    return KV(k_pages.data_ptr(), v_pages.data_ptr(), k_pages.stride(1), v_pages.stride(1), n_ctx,
              n_q_heads, hkv, d, _dtype_code(k_pages), page, block_table.data_ptr(), n_pages)


class ImageTable:
    """Host image table (Eq. 1) kept alive for the duration of calls."""

    def __init__(self, img_pos: Sequence[int], img_off: Sequence[int]):
        self.pos = np.ascontiguousarray(img_pos, dtype=np.int32)
        self.off = np.ascontiguousarray(img_off, dtype=np.int32)
        self.desc = Images(len(self.pos), int(self.off[-1]) if len(self.off) else 0,
                           self.pos.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                           self.off.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))

    @property
    def n_vis(self) -> int:
        return int(self.desc.n_vis)

    @property
    def n_images(self) -> int:
        return int(self.desc.n_images)


def _workspace(nbytes: int, device, ws: Optional[torch.Tensor]) -> Optional[torch.Tensor]:
    if nbytes == 0:
        return ws
    if ws is not None and ws.numel() * ws.element_size() >= nbytes:
        return ws
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def _nbytes(t: Optional[torch.Tensor]) -> int:
    return 0 if t is None else t.numel() * t.element_size()


# ---------------------------------------------------------------------------
# The four entry points
# ---------------------------------------------------------------------------

def conduit_budget(n_vis: int, r_num: int, r_den: int) -> int:
    return int(lib().conduit_budget(n_vis, r_num, r_den))


def score_workspace_bytes(kv: KV, n_q: int, img: ImageTable) -> int:
    return int(lib().conduit_score_workspace_bytes(ctypes.byref(kv), n_q, ctypes.byref(img.desc)))


def conduit_score(kv: KV, q: torch.Tensor, q_pos0: int, img: ImageTable, s_acc: torch.Tensor,
                  a_acc: torch.Tensor, accumulate: bool = False, norm: int = NORM_CAUSAL_ROW,
                  scale: Optional[float] = None, row_lse_in: Optional[torch.Tensor] = None,
                  row_lse_out: Optional[torch.Tensor] = None, a_out: Optional[torch.Tensor] = None,
                  vnorm_out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                  stream=None, agg: int = AGG_MEAN,
                  vnorm_in: Optional[torch.Tensor] = None) -> None:
    """Scoring pass of one layer (Eq. 4/6-7); see conduit_score in conduit.h."""
    n_q = q.shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(kv.head_dim)
    ws = _workspace(score_workspace_bytes(kv, n_q, img), q.device, ws)
    _check(lib().conduit_score(ctypes.byref(kv), q.data_ptr(), n_q, q_pos0, ctypes.byref(img.desc),
                               norm, agg, scale, _ptr(row_lse_in), _ptr(row_lse_out), _ptr(vnorm_in),
                               s_acc.data_ptr(), a_acc.data_ptr(), int(accumulate), _ptr(a_out),
                               _ptr(vnorm_out), _ptr(ws), _nbytes(ws), _stream(stream)))


def score_layers_workspace_bytes(kv: KV, n_q: int, img: "ImageTable", n_layers: int) -> int:
    return int(lib().conduit_score_layers_workspace_bytes(ctypes.byref(kv), n_q, ctypes.byref(img.desc), n_layers))


def conduit_score_layers(kvs, qs, q_pos0: int, img: "ImageTable", s_acc: torch.Tensor, a_acc: torch.Tensor,
                         accumulate: bool = False, norm: int = NORM_CAUSAL_ROW, scale: Optional[float] = None,
                         agg: int = AGG_MEAN, vnorm_in=None, ws: Optional[torch.Tensor] = None,
                         stream=None) -> None:
    """Scoring pass over several layers, accumulated (Eq. 6-7); see conduit_score_layers."""
    n, n_q = len(kvs), qs[0].shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(kvs[0].head_dim)
    ws = _workspace(score_layers_workspace_bytes(kvs[0], n_q, img, n), qs[0].device, ws)
    arr = (KV * n)(*kvs)
    vn = None if vnorm_in is None else _ptr_array(vnorm_in)
    _check(lib().conduit_score_layers(arr, n, _ptr_array(qs), n_q, q_pos0, ctypes.byref(img.desc), norm, agg,
                                      scale, vn, s_acc.data_ptr(), a_acc.data_ptr(), int(accumulate), _ptr(ws),
                                      _nbytes(ws), _stream(stream)))


def conduit_score_noalloc(kv: KV, q: torch.Tensor, q_pos0: int, img: ImageTable, s_acc: torch.Tensor,
                          a_acc: torch.Tensor, accumulate: bool = False, norm: int = NORM_CAUSAL_ROW,
                          scale: Optional[float] = None, row_lse_in: Optional[torch.Tensor] = None,
                          row_lse_out: Optional[torch.Tensor] = None, a_out: Optional[torch.Tensor] = None,
                          vnorm_out: Optional[torch.Tensor] = None, stream=None, agg: int = AGG_MEAN,
                          vnorm_in: Optional[torch.Tensor] = None) -> None:
    """conduit_score on the library's fixed device scratch (no workspace, no
    allocation); see conduit_score_noalloc in conduit.h."""
    n_q = q.shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(kv.head_dim)
    _check(lib().conduit_score_noalloc(ctypes.byref(kv), q.data_ptr(), n_q, q_pos0, ctypes.byref(img.desc),
                                       norm, agg, scale, _ptr(row_lse_in), _ptr(row_lse_out),
                                       _ptr(vnorm_in), s_acc.data_ptr(), a_acc.data_ptr(), int(accumulate),
                                       _ptr(a_out), _ptr(vnorm_out), _stream(stream)))


def conduit_value_norms(kv: KV, img: ImageTable, vnorm_out: torch.Tensor, stream=None) -> None:
    """Value-norm table of one layer (Eq. 7 proxy, Sec. 4.3); see conduit_value_norms."""
    _check(lib().conduit_value_norms(ctypes.byref(kv), ctypes.byref(img.desc), vnorm_out.data_ptr(),
                                     _stream(stream)))


def residual_workspace_bytes(kv: KV, n_q: int, img: ImageTable, n_samples: int, iso: bool) -> int:
    return int(lib().conduit_residual_workspace_bytes(ctypes.byref(kv), n_q, ctypes.byref(img.desc),
                                                      n_samples, int(iso)))


def conduit_residual_error(kv: KV, q: torch.Tensor, q_pos0: int, img: ImageTable,
                           row_lse: torch.Tensor, refreshed: torch.Tensor, err_out: torch.Tensor,
                           z: Optional[torch.Tensor] = None, kappa: float = 0.5,
                           scale: Optional[float] = None, ws: Optional[torch.Tensor] = None,
                           stream=None) -> None:
    """Residual value-write error of a refresh set (Eq. 3, App. D.1/D.3); see
    conduit_residual_error.  z [M, N_vis, H_kv, d] gives the isotropic
    estimator's draws; without z the projected error is computed."""
    n_q = q.shape[0]
    n_samples = 1 if z is None else z.shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(kv.head_dim)
    need = residual_workspace_bytes(kv, n_q, img, n_samples, z is not None)
    if ws is None:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    _check(lib().conduit_residual_error(ctypes.byref(kv), q.data_ptr(), n_q, q_pos0, ctypes.byref(img.desc),
                                        scale, row_lse.data_ptr(), refreshed.data_ptr(), _ptr(z), n_samples,
                                        kappa, err_out.data_ptr(), ws.data_ptr(), ws.numel(),
                                        _stream(stream)))


def conduit_select_topk(s_acc: torch.Tensor, a_acc: torch.Tensor, n_layers: int, img: ImageTable,
                        lam: float, k: int, idx_out: torch.Tensor, pos_out: torch.Tensor,
                        mask_out: Optional[torch.Tensor] = None,
                        shat_out: Optional[torch.Tensor] = None,
                        c_out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                        stream=None, rule: int = RANK_COMPOSITE,
                        quota_out: Optional[torch.Tensor] = None) -> None:
    """Reweighting and top-k (Eq. 8-11, or a variant rule); see conduit_select_topk."""
    need = int(lib().conduit_select_workspace_bytes(img.n_vis, img.n_images))
    ws = _workspace(need, s_acc.device, ws)
    _check(lib().conduit_select_topk(s_acc.data_ptr(), a_acc.data_ptr(), n_layers,
                                     ctypes.byref(img.desc), lam, rule, k, _ptr(idx_out),
                                     _ptr(pos_out), _ptr(mask_out), _ptr(shat_out), _ptr(c_out),
                                     _ptr(quota_out), _ptr(ws), _nbytes(ws), _stream(stream)))


def conduit_scatter_kv(kv: KV, pos: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
                       k_old_out: Optional[torch.Tensor] = None,
                       v_old_out: Optional[torch.Tensor] = None, stream=None) -> None:
    """Cache merge of one layer; see conduit_scatter_kv."""
    _check(lib().conduit_scatter_kv(ctypes.byref(kv), pos.data_ptr(), pos.numel(),
                                    _ptr(k_new), _ptr(v_new), _ptr(k_old_out), _ptr(v_old_out),
                                    _stream(stream)))


def refresh_workspace_bytes(kv: KV, k: int) -> int:
    return int(lib().conduit_refresh_workspace_bytes(ctypes.byref(kv), k))


def _ptr_array(ts) -> ctypes.Array:
    return (ctypes.c_void_p * len(ts))(*[None if t is None else t.data_ptr() for t in ts])


def conduit_scatter_kv_layers(kvs, pos: torch.Tensor, k_new, v_new, stream=None) -> None:
    """Cache merge of several layers with the same rows; see conduit_scatter_kv_layers."""
    arr = (KV * len(kvs))(*kvs)
    _check(lib().conduit_scatter_kv_layers(arr, len(kvs), pos.data_ptr(), pos.numel(), _ptr_array(k_new),
                                           _ptr_array(v_new), _stream(stream)))


def refresh_layers_workspace_bytes(kv: KV, k: int, n_layers: int) -> int:
    return int(lib().conduit_refresh_layers_workspace_bytes(ctypes.byref(kv), k, n_layers))


def conduit_refresh_attn_layers(kvs, q_sel, pos: torch.Tensor, o_out, lse_out=None,
                                scale: Optional[float] = None, ws: Optional[torch.Tensor] = None,
                                stream=None) -> None:
    """Refresh attention of the same rows in several layers; see conduit_refresh_attn_layers."""
    k, n = pos.numel(), len(kvs)
    if scale is None:
        scale = 1.0 / math.sqrt(kvs[0].head_dim)
    ws = _workspace(refresh_layers_workspace_bytes(kvs[0], k, n), q_sel[0].device, ws)
    arr = (KV * n)(*kvs)
    lse = None if lse_out is None else ctypes.cast(_ptr_array(lse_out), ctypes.POINTER(ctypes.c_void_p))
    _check(lib().conduit_refresh_attn_layers(arr, n, _ptr_array(q_sel), pos.data_ptr(), k, scale,
                                             _ptr_array(o_out), lse, _ptr(ws), _nbytes(ws), _stream(stream)))


def conduit_refresh_attn(kv: KV, q_sel: torch.Tensor, pos: torch.Tensor, o_out: torch.Tensor,
                         lse_out: Optional[torch.Tensor] = None, scale: Optional[float] = None,
                         ws: Optional[torch.Tensor] = None, stream=None) -> None:
    """Refresh attention of the selected rows over the merged cache."""
    k = pos.numel()
    if scale is None:
        scale = 1.0 / math.sqrt(kv.head_dim)
    ws = _workspace(refresh_workspace_bytes(kv, k), q_sel.device, ws)
    _check(lib().conduit_refresh_attn(ctypes.byref(kv), q_sel.data_ptr(), pos.data_ptr(), k,
                                      scale, o_out.data_ptr(), _ptr(lse_out), _ptr(ws), _nbytes(ws),
                                      _stream(stream)))


def conduit_merge_refresh_attn(kv: KV, pos: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
                               q_sel: torch.Tensor, o_out: torch.Tensor, lse_out: Optional[torch.Tensor] = None,
                               scale: Optional[float] = None, ws: Optional[torch.Tensor] = None,
                               stream=None) -> None:
    """Cache merge and refresh attention of the same rows in one call; see
    conduit_merge_refresh_attn."""
    k = pos.numel()
    if scale is None:
        scale = 1.0 / math.sqrt(kv.head_dim)
    ws = _workspace(refresh_workspace_bytes(kv, k), q_sel.device, ws)
    _check(lib().conduit_merge_refresh_attn(ctypes.byref(kv), pos.data_ptr(), k, k_new.data_ptr(), v_new.data_ptr(),
                                            q_sel.data_ptr(), scale, o_out.data_ptr(), _ptr(lse_out), _ptr(ws),
                                            _nbytes(ws), _stream(stream)))


def profile_enable(enabled: bool) -> None:
    """Turn per-launch kernel timing on (clearing the record) or off, for the
    calling thread (conduit_profile_enable)."""
    _check(lib().conduit_profile_enable(1 if enabled else 0))


def profile_records() -> list:
    """[(kernel name, ms)] of the launches recorded since timing was enabled;
    waits for each to finish (conduit_profile_read)."""
    L = lib()
    out = []
    name, ms = ctypes.c_char_p(), ctypes.c_float()
    for i in range(L.conduit_profile_count()):
        _check(L.conduit_profile_read(i, ctypes.byref(name), ctypes.byref(ms)))
        out.append((name.value.decode(), ms.value))
    return out


# ---------------------------------------------------------------------------
# A whole refresh step over preallocated buffers
# ---------------------------------------------------------------------------

class RefreshStep:
    """Buffers and calls for one refresh step: score every layer, select once,
    then merge and refresh every layer (the order of Algorithm 1 followed by
    the selective recompute).

    layers: list of dicts of device tensors {"k", "v", "q"} per scored layer
    (k, v [n_ctx, H_kv, d]; q [n_q, H_q, d]).  Fresh rows for the selection
    are passed to `refresh` as {"k_new", "v_new", "q_sel"} per layer.
    """

    def __init__(self, layers, n_q_heads: int, q_pos0: int, img: ImageTable, k: int,
                 lam: float = 1.0, norm: int = NORM_CAUSAL_ROW, device="cuda",
                 agg: int = AGG_MEAN, rule: int = RANK_COMPOSITE, vnorm_tables=None):
        """vnorm_tables: optional per-layer value-norm tables (conduit_value_norms)."""
        self.layers = layers
        self.kvs = [kv_desc(L["k"], L["v"], n_q_heads) for L in layers]
        self.q_pos0, self.img, self.k, self.lam, self.norm = q_pos0, img, k, lam, norm
        self.agg, self.rule, self.vnorm_tables = agg, rule, vnorm_tables
        self.n_q = layers[0]["q"].shape[0]
        nv = img.n_vis
        f32 = dict(dtype=torch.float32, device=device)
        self.s_acc = torch.zeros(nv, **f32)
        self.a_acc = torch.zeros(nv, **f32)
        self.shat = torch.zeros(nv, **f32)
        self.c = torch.zeros(img.n_images, **f32)
        self.quota = torch.zeros(img.n_images, dtype=torch.int32, device=device)
        self.idx = torch.zeros(max(k, 1), dtype=torch.int32, device=device)
        self.pos = torch.zeros(max(k, 1), dtype=torch.int32, device=device)
        self.mask = torch.zeros(nv, dtype=torch.uint8, device=device)
        ws_bytes = score_layers_workspace_bytes(self.kvs[0], self.n_q, img, len(self.kvs))
        self.ws_score = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=device)
        sb = int(lib().conduit_select_workspace_bytes(nv, img.n_images))
        self.ws_select = torch.empty(max(sb, 1), dtype=torch.uint8, device=device)
        rb = refresh_layers_workspace_bytes(self.kvs[0], k, len(self.kvs)) if k > 0 else 0
        self.ws_refresh = torch.empty(max(rb, 1), dtype=torch.uint8, device=device)
        L0 = layers[0]
        self.out = [torch.empty((max(k, 1), n_q_heads, L0["k"].shape[2]), dtype=L0["k"].dtype,
                                device=device) for _ in layers]
        self.lse = [torch.empty((max(k, 1), n_q_heads), **f32) for _ in layers]

    def score_and_select(self, stream=None):
        if self.k == 0:
            conduit_select_topk(self.s_acc, self.a_acc, len(self.layers), self.img, self.lam, 0,
                                self.idx, self.pos, mask_out=self.mask, stream=stream,
                                rule=self.rule)
            return
        if len(self.kvs) > 1:  # every layer in a few launches, summed in layer order
            conduit_score_layers(self.kvs, [L["q"] for L in self.layers], self.q_pos0, self.img, self.s_acc,
                                 self.a_acc, norm=self.norm, agg=self.agg, vnorm_in=self.vnorm_tables,
                                 ws=self.ws_score, stream=stream)
        else:
            conduit_score(self.kvs[0], self.layers[0]["q"], self.q_pos0, self.img, self.s_acc, self.a_acc,
                          norm=self.norm, ws=self.ws_score, stream=stream, agg=self.agg,
                          vnorm_in=None if self.vnorm_tables is None else self.vnorm_tables[0])
        conduit_select_topk(self.s_acc, self.a_acc, len(self.layers), self.img, self.lam, self.k,
                            self.idx, self.pos, mask_out=self.mask, shat_out=self.shat,
                            c_out=self.c, ws=self.ws_select, stream=stream, rule=self.rule,
                            quota_out=self.quota)

    def refresh(self, fresh, stream=None, k_old=None, v_old=None):
        if self.k == 0:
            return
        pos = self.pos[: self.k]
        if len(self.kvs) > 1 and k_old is None and v_old is None:
            # every layer in a few launches: one merge and one plan for up to 16 layers
            conduit_scatter_kv_layers(self.kvs, pos, [F["k_new"] for F in fresh], [F["v_new"] for F in fresh],
                                      stream=stream)
            conduit_refresh_attn_layers(self.kvs, [F["q_sel"] for F in fresh], pos,
                                        [o[: self.k] for o in self.out], lse_out=[x[: self.k] for x in self.lse],
                                        ws=self.ws_refresh, stream=stream)
            return
        for li, (kv, F) in enumerate(zip(self.kvs, fresh)):
            if k_old is None and v_old is None:  # merge and refresh in one call
                conduit_merge_refresh_attn(kv, pos, F["k_new"], F["v_new"], F["q_sel"], self.out[li][: self.k],
                                           lse_out=self.lse[li][: self.k], ws=self.ws_refresh, stream=stream)
                continue
            conduit_scatter_kv(kv, pos, F["k_new"], F["v_new"],
                               None if k_old is None else k_old[li],
                               None if v_old is None else v_old[li], stream=stream)
            conduit_refresh_attn(kv, F["q_sel"], pos, self.out[li][: self.k],
                                 lse_out=self.lse[li][: self.k], ws=self.ws_refresh, stream=stream)
