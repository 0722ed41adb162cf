"""ctypes binding of libhsa.so (include/hsa.h).

Argument marshalling only: tensors are passed as raw device pointers, the
per-head budgets as a host int32 array, and the stream as the current torch
stream. Every step of the computation runs in the library's HIP kernels.
There is no fallback: if the library is not built, loading it raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lib", "libhsa.so")

HSA_DTYPE_BF16 = 0
HSA_DTYPE_F32 = 1
STATUS = {0: "HSA_OK", 1: "HSA_ERR_INVALID_ARG", 2: "HSA_ERR_UNSUPPORTED",
          3: "HSA_ERR_OUT_OF_RANGE", 4: "HSA_ERR_WORKSPACE", 5: "HSA_ERR_DEVICE",
          6: "HSA_ERR_IO"}

c_i32, c_vp, c_sz = ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t


class HsaConfig(ctypes.Structure):
    _fields_ = [("batch", c_i32), ("num_heads", c_i32), ("head_dim", c_i32),
                ("page_size", c_i32), ("dtype", c_i32), ("sm_scale", ctypes.c_float),
                ("gate_dims", c_i32)]


class HsaTierStats(ctypes.Structure):
    _fields_ = [("evictions", ctypes.c_int64), ("fetches", ctypes.c_int64),
                ("spills", ctypes.c_int64), ("reloads", ctypes.c_int64),
                ("prefetched", ctypes.c_int64), ("backups", ctypes.c_int64)]


class HsaKvPool(ctypes.Structure):
    _fields_ = [("k", c_vp), ("v", c_vp), ("page_table", c_vp),
                ("num_slots", c_i32), ("max_pages", c_i32)]


class HsaError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {STATUS.get(status, status)}")
        self.status = status


class LibraryNotBuilt(RuntimeError):
    pass


_lib = None


def lib():
    """The loaded libhsa.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise LibraryNotBuilt(f"{LIB_PATH} missing: build it with `python -m paper_2609_34606_amd.build`")
    # torch's HIP runtime first: the library's libamdhip64.so.7 then binds to
    # that copy (same soname). Loaded the other way round, torch loads its own
    # copy beside the system one, and memory and streams of one runtime are
    # not valid in the other (the library's launches then fail).
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    L.hsa_status_string.restype = ctypes.c_char_p
    L.hsa_status_string.argtypes = [ctypes.c_int]
    for n, extra in (("hsa_state_update_workspace_size", [c_i32]),
                     ("hsa_page_select_workspace_size", [c_i32]),
                     ("hsa_sparse_attn_workspace_size", [c_i32, c_i32, c_i32]),
                     ("hsa_forward_workspace_size", [c_i32, c_i32, c_i32]),
                     ("hsa_adaptive_workspace_size", [c_i32, c_i32, c_i32])):
        f = getattr(L, n)
        f.restype = c_sz
        f.argtypes = [P(HsaConfig)] + extra
    for n, extra in (("hsa_linformer_compress_workspace_size", [c_i32, c_i32]),
                     ("hsa_linformer_workspace_size", [c_i32, c_i32, c_i32])):
        f = getattr(L, n)
        f.restype = c_sz
        f.argtypes = [P(HsaConfig)] + extra
    L.hsa_linformer_compress.restype = ctypes.c_int
    L.hsa_linformer_compress.argtypes = [P(HsaConfig), P(HsaKvPool), c_vp, c_vp, c_i32, c_i32,
                                         c_i32, c_vp, c_vp, c_vp, c_sz, c_vp]
    L.hsa_forward_linformer.restype = ctypes.c_int
    L.hsa_forward_linformer.argtypes = [P(HsaConfig), c_vp, c_i32, P(HsaKvPool), c_vp, c_vp, c_i32,
                                        c_i32, c_i32, c_vp, c_i32, ctypes.c_double,
                                        ctypes.c_double, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_sz,
                                        c_vp]
    L.hsa_retrieval_workspace_size.restype = c_sz
    L.hsa_retrieval_workspace_size.argtypes = [P(HsaConfig), c_i32, c_i32, c_i32]
    L.hsa_chunk_select.restype = ctypes.c_int
    L.hsa_chunk_select.argtypes = [P(HsaConfig), c_vp, c_vp, c_i32, c_i32, c_vp, c_i32, c_vp, c_vp,
                                   c_vp, c_vp]
    L.hsa_forward_retrieval.restype = ctypes.c_int
    L.hsa_forward_retrieval.argtypes = [P(HsaConfig), c_vp, c_i32, P(HsaKvPool), c_vp, c_vp, c_i32,
                                        c_i32, c_vp, c_i32, c_i32, c_vp, c_i32, c_vp, c_vp, c_vp,
                                        c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]
    L.hsa_tier_create.restype = ctypes.c_int
    L.hsa_tier_create.argtypes = [P(HsaConfig), P(HsaKvPool), c_vp, c_vp, c_i32, ctypes.c_char_p,
                                  c_i32, c_i32, P(c_vp)]
    L.hsa_tier_destroy.restype = None
    L.hsa_tier_destroy.argtypes = [c_vp]
    L.hsa_tier_place.restype = ctypes.c_int
    L.hsa_tier_place.argtypes = [c_vp, c_i32, c_i32, P(c_i32), c_vp]
    L.hsa_tier_fetch.restype = ctypes.c_int
    L.hsa_tier_fetch.argtypes = [c_vp, c_vp, c_i32, c_vp]
    L.hsa_tier_prefetch.restype = ctypes.c_int
    L.hsa_tier_prefetch.argtypes = [c_vp, c_vp, c_i32, c_vp]
    L.hsa_tier_commit.restype = ctypes.c_int
    L.hsa_tier_commit.argtypes = [c_vp, c_vp]
    L.hsa_tier_drop.restype = ctypes.c_int
    L.hsa_tier_drop.argtypes = [c_vp, c_vp]
    L.hsa_tier_locate.restype = c_i32
    L.hsa_tier_locate.argtypes = [c_vp, c_i32, c_i32]
    L.hsa_tier_stats.restype = None
    L.hsa_tier_stats.argtypes = [c_vp, P(HsaTierStats)]
    L.hsa_forward_noalloc_bytes.restype = c_sz
    L.hsa_forward_noalloc_bytes.argtypes = [P(HsaConfig), c_i32, c_i32, c_i32, c_vp, c_i32]
    L.hsa_forward_noalloc.restype = ctypes.c_int
    L.hsa_forward_noalloc.argtypes = [P(HsaConfig), c_vp, c_i32, P(HsaKvPool), c_i32, c_i32, c_vp,
                                      c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp]
    L.hsa_page_write.restype = ctypes.c_int
    L.hsa_page_write.argtypes = [P(HsaConfig), P(HsaKvPool), c_vp, c_vp, c_i32, c_i32, c_vp, c_vp]
    L.hsa_cube_order.restype = c_i32
    L.hsa_cube_order.argtypes = [c_i32, c_i32, c_i32, c_i32, c_i32, c_i32, c_vp]
    L.hsa_attention_plan.restype = ctypes.c_int
    L.hsa_attention_plan.argtypes = [P(HsaConfig), c_i32, c_vp, c_i32, c_vp, c_vp, c_vp]
    L.hsa_block_count.restype = c_i32
    L.hsa_block_count.argtypes = [P(HsaConfig), c_i32, c_i32]
    c_f64 = ctypes.c_double
    L.hsa_block_select.restype = ctypes.c_int
    L.hsa_block_select.argtypes = [P(HsaConfig), c_vp, c_i32, P(HsaKvPool), c_vp, c_i32, c_i32,
                                   c_i32, c_f64, c_f64, c_vp, c_vp, c_vp, c_vp, c_vp, c_i32, c_vp,
                                   c_sz, c_vp]
    L.hsa_sparse_attn_adaptive.restype = ctypes.c_int
    L.hsa_sparse_attn_adaptive.argtypes = [P(HsaConfig), c_vp, c_i32, P(HsaKvPool), c_vp, c_i32,
                                           c_vp, c_i32, c_i32, c_f64, c_f64, c_vp, c_vp, c_vp,
                                           c_sz, c_vp]
    L.hsa_forward_adaptive.restype = ctypes.c_int
    L.hsa_forward_adaptive.argtypes = [P(HsaConfig), c_vp, c_i32, P(HsaKvPool), c_i32, c_i32, c_vp,
                                       c_i32, c_f64, c_f64, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp,
                                       c_vp, c_vp, c_sz, c_vp]
    L.hsa_state_update.restype = ctypes.c_int
    L.hsa_state_update.argtypes = [P(HsaConfig), P(HsaKvPool), c_i32, c_i32, c_vp, c_vp, c_vp,
                                   c_vp, c_sz, c_vp]
    L.hsa_page_select.restype = ctypes.c_int
    L.hsa_page_select.argtypes = [P(HsaConfig), c_vp, c_i32, c_vp, c_i32, c_i32, c_vp, c_i32,
                                  c_vp, c_vp, c_vp, c_sz, c_vp]
    L.hsa_sparse_attn.restype = ctypes.c_int
    L.hsa_sparse_attn.argtypes = [P(HsaConfig), c_vp, c_i32, P(HsaKvPool), c_vp, c_i32, c_vp,
                                  c_i32, c_i32, c_vp, c_vp, c_vp, c_sz, c_vp]
    L.hsa_forward.restype = ctypes.c_int
    L.hsa_forward.argtypes = [P(HsaConfig), c_vp, c_i32, P(HsaKvPool), c_i32, c_i32, c_vp,
                              c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]
    L.hsa_forward_selected.restype = ctypes.c_int
    L.hsa_forward_selected.argtypes = [P(HsaConfig), c_vp, c_i32, P(HsaKvPool), c_vp, c_i32, c_vp,
                                       c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]
    _lib = L
    return L


# ------------------------------------------------------------------ helpers
def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if hasattr(t, "data_ptr"):
        if not t.is_contiguous():
            raise ValueError("tensor arguments must be contiguous")
        return t.data_ptr()
    return int(t)


def _out(t, n: int, dtype: str, what: str) -> Optional[int]:
    """Pointer of an optional output of at least n elements of dtype
    ('int32' or 'float64'), or None."""
    if t is None:
        return None
    if hasattr(t, "dtype") and str(t.dtype) != f"torch.{dtype}":
        raise ValueError(f"{what}: expected {dtype}, got {t.dtype}")
    if hasattr(t, "numel") and t.numel() < n:
        raise ValueError(f"{what}: {t.numel()} elements, need {n}")
    return _ptr(t)


def _gate(cfg, g, n_q: int) -> Optional[int]:
    """Pointer of a gate-logit tensor after checking that it holds what the
    kernels read: fp32, [B, n_q, H] or, with cfg.gate_dims = d, [B, n_q, H, d]."""
    if g is None:
        return None
    per = cfg.head_dim if cfg.gate_dims > 1 else 1
    want = cfg.batch * n_q * cfg.num_heads * per
    if hasattr(g, "numel"):
        if g.numel() != want or str(g.dtype) != "torch.float32":
            raise ValueError(f"gate logits must be {want} fp32 values ([B, n_q, H"
                             f"{', d' if per > 1 else ''}]), got {tuple(g.shape)} {g.dtype}")
    return _ptr(g)


def _elem_dtype(cfg) -> str:
    return "torch.bfloat16" if cfg.dtype == HSA_DTYPE_BF16 else "torch.float32"


def _rows(cfg, t, n_q: int, what: str, fp32: bool = False) -> Optional[int]:
    """Pointer of a [B, n_q, H, d] tensor (queries or outputs) after checking
    its size and element type against the config (the kernels index it with
    these sizes and read or write elements of the config's dtype; fp32 = True
    for the fp32 sparse-branch output)."""
    if t is not None and hasattr(t, "numel"):
        want = cfg.batch * n_q * cfg.num_heads * cfg.head_dim
        if t.numel() != want:
            raise ValueError(f"{what} must hold [B, n_q, H, d] = {want} values, "
                             f"got {tuple(t.shape)}")
        dt = "torch.float32" if fp32 else _elem_dtype(cfg)
        if str(t.dtype) != dt:
            raise ValueError(f"{what} must be {dt}, got {t.dtype}")
    return _ptr(t)


def _stream(stream) -> Optional[int]:
    """A HIP stream handle: an int, a torch stream, or None for torch's
    current stream."""
    if stream is not None:
        return int(getattr(stream, "cuda_stream", stream))
    import torch
    return torch.cuda.current_stream().cuda_stream


def _budgets(k_h: Optional[Sequence[int]]):
    if k_h is None:
        return None, None
    arr = np.ascontiguousarray(np.asarray(k_h, dtype=np.int32))
    return arr, arr.ctypes.data_as(c_vp)


def _check(fn: str, status: int):
    if status != 0:
        raise HsaError(fn, status)


def _workspace(nbytes: int, device):
    import torch
    if nbytes == 0:
        return None
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def config(batch: int, num_heads: int, head_dim: int, page_size: int, dtype,
           sm_scale: float = 0.0, gate_dims: int = 0) -> HsaConfig:
    """gate_dims: 0 for gate logits per (query, head), head_dim for logits per
    (query, head, dim)."""
    if not isinstance(dtype, int):
        dtype = HSA_DTYPE_BF16 if str(dtype).endswith("bfloat16") or dtype == "bf16" else HSA_DTYPE_F32
    return HsaConfig(batch, num_heads, head_dim, page_size, dtype, sm_scale, gate_dims)


def kv_pool(k_pool, v_pool, page_table, cfg: Optional[HsaConfig] = None) -> HsaKvPool:
    """The pool descriptor. With cfg, the tensors are checked against it
    first: k_pool [slots, H, P, d] and v_pool [slots, H, d, P] of the config's
    dtype, page_table [B, max_pages] int32."""
    if cfg is not None:
        H, P, d = cfg.num_heads, cfg.page_size, cfg.head_dim
        slots = int(k_pool.shape[0])
        dt = _elem_dtype(cfg)
        for name, t, shape in (("k_pool", k_pool, (slots, H, P, d)), ("v_pool", v_pool, (slots, H, d, P))):
            if tuple(t.shape) != shape or str(t.dtype) != dt:
                raise ValueError(f"{name} must be {dt} {shape}, got {t.dtype} {tuple(t.shape)}")
        if page_table.dim() != 2 or page_table.shape[0] != cfg.batch or str(page_table.dtype) != "torch.int32":
            raise ValueError(f"page_table must be int32 [B={cfg.batch}, max_pages], got "
                             f"{page_table.dtype} {tuple(page_table.shape)}")
    return HsaKvPool(_ptr(k_pool), _ptr(v_pool), _ptr(page_table), int(k_pool.shape[0]),
                     int(page_table.shape[-1]))


# ------------------------------------------------------------------ C ABI calls
def hsa_state_update_workspace_size(cfg: HsaConfig, n_pages: int) -> int:
    return lib().hsa_state_update_workspace_size(ctypes.byref(cfg), n_pages)


def hsa_page_select_workspace_size(cfg: HsaConfig, n_q: int) -> int:
    return lib().hsa_page_select_workspace_size(ctypes.byref(cfg), n_q)


def hsa_sparse_attn_workspace_size(cfg: HsaConfig, n_q: int, k_max: int, n_cur_pages: int) -> int:
    return lib().hsa_sparse_attn_workspace_size(ctypes.byref(cfg), n_q, k_max, n_cur_pages)


def hsa_forward_workspace_size(cfg: HsaConfig, n_q: int, k_max: int, n_cur_pages: int) -> int:
    return lib().hsa_forward_workspace_size(ctypes.byref(cfg), n_q, k_max, n_cur_pages)


def hsa_adaptive_workspace_size(cfg: HsaConfig, n_q: int, k_max: int, n_cur_pages: int) -> int:
    return lib().hsa_adaptive_workspace_size(ctypes.byref(cfg), n_q, k_max, n_cur_pages)


def hsa_block_count(cfg: HsaConfig, n_hist_pages: int, n_cur_pages: int) -> int:
    return lib().hsa_block_count(ctypes.byref(cfg), n_hist_pages, n_cur_pages)


def hsa_status_string(status: int) -> str:
    return lib().hsa_status_string(status).decode()


def hsa_state_update(cfg, pool, first_page, n_pages, kv_state, k_state, page_kmean,
                     ws=None, stream=None, check=True) -> int:
    if ws is None:
        ws = _workspace(hsa_state_update_workspace_size(cfg, n_pages), kv_state.device)
    st = lib().hsa_state_update(ctypes.byref(cfg), ctypes.byref(pool), first_page, n_pages,
                                _ptr(kv_state), _ptr(k_state), _ptr(page_kmean), _ptr(ws),
                                0 if ws is None else ws.numel(), _stream(stream))
    if check:
        _check("hsa_state_update", st)
    return st


def hsa_page_write(cfg, pool, k_src, v_src, first_page, n_pages, src_of=None, stream=None,
                   check=True) -> int:
    """Append pages: k_src / v_src [B, n_pages * P, H, d] (raster order) into
    the pool slots of logical pages [first_page, first_page + n_pages),
    optionally permuted by src_of (device int32 [P], e.g. from
    hsa_cube_order)."""
    want = cfg.batch * n_pages * cfg.page_size * cfg.num_heads * cfg.head_dim
    for name, t in (("k_src", k_src), ("v_src", v_src)):
        if hasattr(t, "numel") and (t.numel() != want or str(t.dtype) != _elem_dtype(cfg)):
            raise ValueError(f"{name} must hold {want} values of {_elem_dtype(cfg)} "
                             f"([B, n_pages * P, H, d]), got {tuple(t.shape)} {t.dtype}")
    if src_of is not None and hasattr(src_of, "numel"):
        if src_of.numel() != cfg.page_size or str(src_of.dtype) != "torch.int32":
            raise ValueError("src_of must be int32 [P]")
    st = lib().hsa_page_write(ctypes.byref(cfg), ctypes.byref(pool), _ptr(k_src), _ptr(v_src),
                              first_page, n_pages, _ptr(src_of), _stream(stream))
    if check:
        _check("hsa_page_write", st)
    return st


def hsa_cube_order(frames: int, height: int, width: int, cube=(4, 8, 4)):
    """(src_of, whole): src_of[i] = raster index of the token stored at
    position i of a page in cube order (int32 numpy array), and the number of
    positions covered by whole cubes."""
    n = frames * height * width
    out = np.empty(n, np.int32)
    whole = lib().hsa_cube_order(frames, height, width, int(cube[0]), int(cube[1]), int(cube[2]),
                                 out.ctypes.data_as(c_vp))
    if whole < 0:
        raise ValueError("invalid cube order sizes")
    return out, whole


def hsa_page_select(cfg, q, n_q, page_kmean, max_pages, n_cand, k_h, k_max, sel,
                    sel_score=None, ws=None, stream=None, check=True) -> int:
    if ws is None:
        ws = _workspace(hsa_page_select_workspace_size(cfg, n_q), q.device)
    _keep, kp = _budgets(k_h)
    st = lib().hsa_page_select(ctypes.byref(cfg), _rows(cfg, q, n_q, "q"), n_q, _ptr(page_kmean), max_pages,
                               n_cand, kp, k_max, _ptr(sel), _ptr(sel_score), _ptr(ws),
                               0 if ws is None else ws.numel(), _stream(stream))
    if check:
        _check("hsa_page_select", st)
    return st


def hsa_sparse_attn(cfg, q, n_q, pool, sel, k_max, k_h, cur_first_page, n_cur_pages, o_sp,
                    lse=None, ws=None, stream=None, check=True) -> int:
    if ws is None:
        ws = _workspace(hsa_sparse_attn_workspace_size(cfg, n_q, k_max, n_cur_pages), q.device)
    _keep, kp = _budgets(k_h)
    qp, op = _rows(cfg, q, n_q, "q"), _rows(cfg, o_sp, n_q, "o_sp", fp32=True)
    st = lib().hsa_sparse_attn(ctypes.byref(cfg), qp, n_q, ctypes.byref(pool), _ptr(sel),
                               k_max, kp, cur_first_page, n_cur_pages, op, _ptr(lse),
                               _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream))
    if check:
        _check("hsa_sparse_attn", st)
    return st


def hsa_forward(cfg, q, n_q, pool, n_cand, n_cur_pages, k_h, k_max, kv_state, k_state,
                page_kmean, g_lin, g_sp, o, sel_out=None, ws=None, stream=None,
                check=True) -> int:
    if ws is None:
        ws = _workspace(hsa_forward_workspace_size(cfg, n_q, k_max, n_cur_pages), q.device)
    _keep, kp = _budgets(k_h)
    qp, op = _rows(cfg, q, n_q, "q"), _rows(cfg, o, n_q, "o")
    glp, gsp = _gate(cfg, g_lin, n_q), _gate(cfg, g_sp, n_q)
    st = lib().hsa_forward(ctypes.byref(cfg), qp, n_q, ctypes.byref(pool), n_cand,
                           n_cur_pages, kp, k_max, _ptr(kv_state), _ptr(k_state),
                           _ptr(page_kmean), glp, gsp, op, _ptr(sel_out),
                           _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream))
    if check:
        _check("hsa_forward", st)
    return st


def hsa_forward_selected(cfg, q, n_q, pool, sel, k_max, k_h, n_cand, n_cur_pages, kv_state,
                         k_state, g_lin, g_sp, o, ws=None, stream=None, check=True) -> int:
    if ws is None:
        ws = _workspace(hsa_forward_workspace_size(cfg, n_q, k_max, n_cur_pages), q.device)
    _keep, kp = _budgets(k_h)
    qp, op = _rows(cfg, q, n_q, "q"), _rows(cfg, o, n_q, "o")
    glp, gsp = _gate(cfg, g_lin, n_q), _gate(cfg, g_sp, n_q)
    st = lib().hsa_forward_selected(ctypes.byref(cfg), qp, n_q, ctypes.byref(pool), _ptr(sel),
                                    k_max, kp, n_cand, n_cur_pages, _ptr(kv_state), _ptr(k_state),
                                    glp, gsp, op, _ptr(ws),
                                    0 if ws is None else ws.numel(), _stream(stream))
    if check:
        _check("hsa_forward_selected", st)
    return st


def hsa_forward_noalloc_bytes(cfg, n_q, n_cand, n_cur_pages, k_h, k_max) -> int:
    _keep, kp = _budgets(k_h)
    return lib().hsa_forward_noalloc_bytes(ctypes.byref(cfg), n_q, n_cand, n_cur_pages, kp, k_max)


def hsa_forward_noalloc(cfg, q, n_q, pool, n_cand, n_cur_pages, k_h, k_max, kv_state, k_state,
                        page_kmean, g_lin, g_sp, o, sel_out=None, stream=None, check=True) -> int:
    """hsa_forward with the library's static per-GPU workspace (no device
    allocation by the library or by this binding)."""
    _keep, kp = _budgets(k_h)
    qp, op = _rows(cfg, q, n_q, "q"), _rows(cfg, o, n_q, "o")
    glp, gsp = _gate(cfg, g_lin, n_q), _gate(cfg, g_sp, n_q)
    st = lib().hsa_forward_noalloc(ctypes.byref(cfg), qp, n_q, ctypes.byref(pool), n_cand,
                                   n_cur_pages, kp, k_max, _ptr(kv_state), _ptr(k_state),
                                   _ptr(page_kmean), glp, gsp, op, _ptr(sel_out), _stream(stream))
    if check:
        _check("hsa_forward_noalloc", st)
    return st


# Paper's setting of the coverage thresholds (tau_max, tau_min) = (1.00, 0.35).
TAU_MIN, TAU_MAX = 0.35, 1.00
BLOCK_Q = 64  # queries per query block (HSA_BLOCK_Q)


def hsa_block_select(cfg, q, n_q, pool, sel, k_max, cur_first_page, n_cur_pages,
                     tau_min=TAU_MIN, tau_max=TAU_MAX, gini=None, tau=None, n_kept=None,
                     kept=None, pooled=None, kept_len=0, ws=None, stream=None,
                     check=True) -> int:
    if ws is None:
        ws = _workspace(hsa_adaptive_workspace_size(cfg, n_q, k_max, n_cur_pages), q.device)
    bh = cfg.batch * cfg.num_heads
    n_qb = -(-n_q // BLOCK_Q)
    st = lib().hsa_block_select(ctypes.byref(cfg), _rows(cfg, q, n_q, "q"), n_q, ctypes.byref(pool), _ptr(sel),
                                k_max, cur_first_page, n_cur_pages, float(tau_min),
                                float(tau_max), _out(gini, bh, "float64", "gini"),
                                _out(tau, bh, "float64", "tau"),
                                _out(n_kept, bh * n_qb, "int32", "n_kept"),
                                _out(kept, bh * n_qb * kept_len, "int32", "kept"),
                                _out(pooled, bh * n_qb * kept_len, "float64", "pooled"), kept_len,
                                _ptr(ws), 0 if ws is None else ws.numel(), _stream(stream))
    if check:
        _check("hsa_block_select", st)
    return st


def hsa_sparse_attn_adaptive(cfg, q, n_q, pool, sel, k_max, k_h, cur_first_page, n_cur_pages,
                             o_sp, lse=None, tau_min=TAU_MIN, tau_max=TAU_MAX, ws=None,
                             stream=None, check=True) -> int:
    if ws is None:
        ws = _workspace(hsa_adaptive_workspace_size(cfg, n_q, k_max, n_cur_pages), q.device)
    _keep, kp = _budgets(k_h)
    st = lib().hsa_sparse_attn_adaptive(ctypes.byref(cfg), _rows(cfg, q, n_q, "q"), n_q,
                                        ctypes.byref(pool), _ptr(sel), k_max, kp, cur_first_page,
                                        n_cur_pages, float(tau_min), float(tau_max),
                                        _rows(cfg, o_sp, n_q, "o_sp", fp32=True), _ptr(lse),
                                        _ptr(ws), 0 if ws is None else ws.numel(),
                                        _stream(stream))
    if check:
        _check("hsa_sparse_attn_adaptive", st)
    return st


def hsa_forward_adaptive(cfg, q, n_q, pool, n_cand, n_cur_pages, k_h, k_max, kv_state, k_state,
                         page_kmean, g_lin, g_sp, o, tau_min=TAU_MIN, tau_max=TAU_MAX,
                         sel_out=None, ws=None, stream=None, check=True) -> int:
    if ws is None:
        ws = _workspace(hsa_adaptive_workspace_size(cfg, n_q, k_max, n_cur_pages), q.device)
    _keep, kp = _budgets(k_h)
    qp, op = _rows(cfg, q, n_q, "q"), _rows(cfg, o, n_q, "o")
    glp, gsp = _gate(cfg, g_lin, n_q), _gate(cfg, g_sp, n_q)
    st = lib().hsa_forward_adaptive(ctypes.byref(cfg), qp, n_q, ctypes.byref(pool), n_cand,
                                    n_cur_pages, kp, k_max, float(tau_min), float(tau_max),
                                    _ptr(kv_state), _ptr(k_state), _ptr(page_kmean), glp,
                                    gsp, op, _ptr(sel_out), _ptr(ws),
                                    0 if ws is None else ws.numel(), _stream(stream))
    if check:
        _check("hsa_forward_adaptive", st)
    return st


def hsa_linformer_compress_workspace_size(cfg: HsaConfig, rank: int, n_pages: int) -> int:
    return lib().hsa_linformer_compress_workspace_size(ctypes.byref(cfg), rank, n_pages)


def hsa_linformer_workspace_size(cfg: HsaConfig, n_q: int, k_max: int, n_cur_pages: int) -> int:
    return lib().hsa_linformer_workspace_size(ctypes.byref(cfg), n_q, k_max, n_cur_pages)


def hsa_linformer_compress(cfg, pool, e_k, e_v, rank, first_page, n_pages, ck, cv, ws=None,
                           stream=None, check=True) -> int:
    if ws is None:
        ws = _workspace(hsa_linformer_compress_workspace_size(cfg, rank, n_pages), ck.device)
    st = lib().hsa_linformer_compress(ctypes.byref(cfg), ctypes.byref(pool), _ptr(e_k), _ptr(e_v),
                                      rank, first_page, n_pages, _ptr(ck), _ptr(cv), _ptr(ws),
                                      0 if ws is None else ws.numel(), _stream(stream))
    if check:
        _check("hsa_linformer_compress", st)
    return st


def hsa_forward_linformer(cfg, q, n_q, pool, ck, cv, rank, n_cand, n_cur_pages, k_h, k_max,
                          page_kmean, g_lin, g_sp, o, tau_min=TAU_MIN, tau_max=TAU_MAX,
                          sel_out=None, ws=None, stream=None, check=True) -> int:
    if ws is None:
        ws = _workspace(hsa_linformer_workspace_size(cfg, n_q, k_max, n_cur_pages), q.device)
    _keep, kp = _budgets(k_h)
    qp, op = _rows(cfg, q, n_q, "q"), _rows(cfg, o, n_q, "o")
    glp, gsp = _gate(cfg, g_lin, n_q), _gate(cfg, g_sp, n_q)
    st = lib().hsa_forward_linformer(ctypes.byref(cfg), qp, n_q, ctypes.byref(pool), _ptr(ck),
                                     _ptr(cv), rank, n_cand, n_cur_pages, kp, k_max,
                                     float(tau_min), float(tau_max), _ptr(page_kmean), glp,
                                     gsp, op, _ptr(sel_out), _ptr(ws),
                                     0 if ws is None else ws.numel(), _stream(stream))
    if check:
        _check("hsa_forward_linformer", st)
    return st


def hsa_retrieval_workspace_size(cfg: HsaConfig, n_q: int, k_max: int, n_cur_pages: int) -> int:
    return lib().hsa_retrieval_workspace_size(ctypes.byref(cfg), n_q, k_max, n_cur_pages)


def hsa_chunk_select(cfg, prompt_emb, chunk_emb, emb_dim, n_chunks, chunk_first, n_cand,
                     cand_range, chunk_out=None, chunk_score=None, stream=None,
                     check=True) -> int:
    st = lib().hsa_chunk_select(ctypes.byref(cfg), _ptr(prompt_emb), _ptr(chunk_emb), emb_dim,
                                n_chunks, _ptr(chunk_first), n_cand, _ptr(chunk_out),
                                _ptr(chunk_score), _ptr(cand_range), _stream(stream))
    if check:
        _check("hsa_chunk_select", st)
    return st


def hsa_forward_retrieval(cfg, q, n_q, pool, prompt_emb, chunk_emb, emb_dim, n_chunks,
                          chunk_first, n_cand, n_cur_pages, k_h, k_max, kv_state, k_state,
                          page_kmean, g_lin, g_sp, o, chunk_out=None, sel_out=None, ws=None,
                          stream=None, check=True) -> int:
    if ws is None:
        ws = _workspace(hsa_retrieval_workspace_size(cfg, n_q, k_max, n_cur_pages), q.device)
    _keep, kp = _budgets(k_h)
    qp, op = _rows(cfg, q, n_q, "q"), _rows(cfg, o, n_q, "o")
    glp, gsp = _gate(cfg, g_lin, n_q), _gate(cfg, g_sp, n_q)
    st = lib().hsa_forward_retrieval(ctypes.byref(cfg), qp, n_q, ctypes.byref(pool),
                                     _ptr(prompt_emb), _ptr(chunk_emb), emb_dim, n_chunks,
                                     _ptr(chunk_first), n_cand, n_cur_pages, kp, k_max,
                                     _ptr(kv_state), _ptr(k_state), _ptr(page_kmean), glp,
                                     gsp, op, _ptr(chunk_out), _ptr(sel_out), _ptr(ws),
                                     0 if ws is None else ws.numel(), _stream(stream))
    if check:
        _check("hsa_forward_retrieval", st)
    return st


class HsaTier:
    """Host-managed tiers of a layer's KV pool (include/hsa.h, hsa_tier_*):
    logical pages live in the pool's slots (L1), in pinned host slots (L2) or
    in slots of an unnamed file under ``l3_dir`` (L3). ``pool`` None makes a
    plan-only tier (bookkeeping without copies). ``backup`` keeps a copy of
    every page in the file (``commit`` writes new pages, ``drop`` releases
    the pool and host copies)."""

    def __init__(self, cfg: HsaConfig, pool: Optional[HsaKvPool], l2_slots: int, host_k=None,
                 host_v=None, num_slots: int = 0, max_pages: int = 0, l3_dir: Optional[str] = None,
                 l3_slots: int = 0, backup: bool = False):
        if pool is None:
            pool = HsaKvPool(None, None, None, num_slots, max_pages)
        self._keep = (cfg, pool, host_k, host_v)
        h = c_vp()
        _check("hsa_tier_create", lib().hsa_tier_create(
            ctypes.byref(cfg), ctypes.byref(pool), _ptr(host_k), _ptr(host_v), l2_slots,
            None if l3_dir is None else str(l3_dir).encode(), l3_slots, int(bool(backup)),
            ctypes.byref(h)))
        self._h = h

    def close(self):
        if self._h:
            lib().hsa_tier_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _stream(self, stream):
        return None if self._keep[1].k is None else _stream(stream)

    def place(self, b: int, page: int, stream=None, check=True):
        slot = c_i32(-1)
        st = lib().hsa_tier_place(self._h, b, page, ctypes.byref(slot), self._stream(stream))
        if check:
            _check("hsa_tier_place", st)
            return slot.value
        return st, slot.value

    def _move(self, fn, pages, stream, check):
        arr = np.ascontiguousarray(np.asarray(pages, dtype=np.int32))
        n = arr.shape[-1] if arr.ndim else 0
        st = getattr(lib(), fn)(self._h, arr.ctypes.data_as(c_vp), n, self._stream(stream))
        if check:
            _check(fn, st)
        return st

    def fetch(self, pages, stream=None, check=True) -> int:
        return self._move("hsa_tier_fetch", pages, stream, check)

    def prefetch(self, pages, stream=None, check=True) -> int:
        return self._move("hsa_tier_prefetch", pages, stream, check)

    def commit(self, stream=None, check=True) -> int:
        st = lib().hsa_tier_commit(self._h, self._stream(stream))
        if check:
            _check("hsa_tier_commit", st)
        return st

    def drop(self, stream=None, check=True) -> int:
        st = lib().hsa_tier_drop(self._h, self._stream(stream))
        if check:
            _check("hsa_tier_drop", st)
        return st

    def locate(self, b: int, page: int) -> int:
        return lib().hsa_tier_locate(self._h, b, page)

    def stats(self) -> dict:
        s = HsaTierStats()
        lib().hsa_tier_stats(self._h, ctypes.byref(s))
        return {k: getattr(s, k) for k, _ in HsaTierStats._fields_}

    def counters(self):
        """(pages moved out of the pool, pages brought into it)."""
        s = self.stats()
        return s["evictions"], s["fetches"]
