"""Device buffers of one HSA attention layer, driven through the C ABI."""
from __future__ import annotations

from typing import Optional, Sequence

from . import hsa as _h


class HsaLayer:
    """Paged KV pool, page table, linear state and page index of one layer.

    Shapes follow include/hsa.h: k_pool [slots,H,P,d], v_pool [slots,H,d,P],
    page_table [B,max_pages], kv_state [B,H,d,d], k_state [B,H,d],
    page_kmean [B,H,max_pages,d]; gate logits [B,n_q,H], or [B,n_q,H,d] with
    gate_dims = d.
    """

    def __init__(self, batch: int, heads: int, head_dim: int, page_size: int,
                 dtype, device, k_pool=None, v_pool=None, page_table=None,
                 num_slots: int = 0, max_pages: int = 0, sm_scale: float = 0.0,
                 gate_dims: int = 0):
        import torch
        self.torch = torch
        self.device = torch.device(device)
        self.dtype = dtype
        self.cfg = _h.config(batch, heads, head_dim, page_size, dtype, sm_scale, gate_dims)
        if k_pool is None:
            k_pool = torch.empty((num_slots, heads, page_size, head_dim), dtype=dtype, device=device)
            v_pool = torch.empty((num_slots, heads, head_dim, page_size), dtype=dtype, device=device)
        if page_table is None:
            page_table = torch.full((batch, max_pages), -1, dtype=torch.int32, device=device)
        self.k_pool, self.v_pool, self.page_table = k_pool, v_pool, page_table
        self.max_pages = int(page_table.shape[-1])
        self.kv_state = torch.zeros((batch, heads, head_dim, head_dim), dtype=torch.float32, device=device)
        self.k_state = torch.zeros((batch, heads, head_dim), dtype=torch.float32, device=device)
        self.page_kmean = torch.zeros((batch, heads, self.max_pages, head_dim), dtype=torch.float64,
                                      device=device)
        self._ws = {}

    @property
    def pool(self) -> _h.HsaKvPool:
        return _h.kv_pool(self.k_pool, self.v_pool, self.page_table, self.cfg)

    def workspace(self, key, nbytes: int):
        if nbytes == 0:
            return None
        w = self._ws.get(key)
        if w is None or w.numel() < nbytes:
            w = self.torch.empty(nbytes, dtype=self.torch.uint8, device=self.device)
            self._ws[key] = w
        return w

    def set_projections(self, e_k, e_v):
        """Linformer projections ([H, rank, P] each, e[h][j][t] = E^(h)[t][j])
        and a compressed pool for every slot of the layer's pool."""
        torch = self.torch
        H, rank = e_k.shape[0], e_k.shape[1]
        self.e_k, self.e_v, self.rank = e_k, e_v, rank
        slots = self.k_pool.shape[0]
        d = self.k_pool.shape[-1]
        self.ck = torch.empty((slots, H, rank, d), dtype=self.k_pool.dtype, device=self.device)
        self.cv = torch.empty((slots, H, d, rank), dtype=self.k_pool.dtype, device=self.device)

    def compress(self, first_page: int, n_pages: int, stream=None):
        """Compress logical pages [first, first+n) with the Linformer projections."""
        ws = self.workspace("compress", _h.hsa_linformer_compress_workspace_size(
            self.cfg, self.rank, n_pages))
        _h.hsa_linformer_compress(self.cfg, self.pool, self.e_k, self.e_v, self.rank, first_page,
                                  n_pages, self.ck, self.cv, ws=ws, stream=stream)

    def reset_state(self):
        self.kv_state.zero_()
        self.k_state.zero_()

    def fold(self, first_page: int, n_pages: int, stream=None):
        """Fold logical pages [first, first+n) into the state and page index."""
        ws = self.workspace("state", _h.hsa_state_update_workspace_size(self.cfg, n_pages))
        _h.hsa_state_update(self.cfg, self.pool, first_page, n_pages, self.kv_state,
                            self.k_state, self.page_kmean, ws=ws, stream=stream)

    def forward(self, q, n_cand: int, n_cur: int, k_h: Sequence[int], k_max: Optional[int] = None,
                g_lin=None, g_sp=None, out=None, sel_out=None, stream=None):
        B, n_q = q.shape[0], q.shape[1]
        k_max = max(1, max(k_h)) if k_max is None else k_max
        if out is None:
            out = self.torch.empty_like(q)
        ws = self.workspace("fwd", _h.hsa_forward_workspace_size(self.cfg, n_q, k_max, n_cur))
        _h.hsa_forward(self.cfg, q, n_q, self.pool, n_cand, n_cur, k_h, k_max, self.kv_state,
                       self.k_state, self.page_kmean, g_lin, g_sp, out, sel_out=sel_out, ws=ws,
                       stream=stream)
        return out

    def forward_selected(self, q, sel, n_cand: int, n_cur: int, k_h: Sequence[int],
                         k_max: Optional[int] = None, g_lin=None, g_sp=None, out=None, stream=None):
        """The forward pass for a selection already in `sel` ([B,H,k_max] int32)."""
        B, n_q = q.shape[0], q.shape[1]
        k_max = int(sel.shape[-1]) if k_max is None else k_max
        if out is None:
            out = self.torch.empty_like(q)
        ws = self.workspace("fwd", _h.hsa_forward_workspace_size(self.cfg, n_q, k_max, n_cur))
        _h.hsa_forward_selected(self.cfg, q, n_q, self.pool, sel, k_max, k_h, n_cand, n_cur,
                                self.kv_state, self.k_state, g_lin, g_sp, out, ws=ws, stream=stream)
        return out

    def forward_adaptive(self, q, n_cand: int, n_cur: int, k_h: Sequence[int],
                         k_max: Optional[int] = None, tau_min: float = _h.TAU_MIN,
                         tau_max: float = _h.TAU_MAX, g_lin=None, g_sp=None, out=None,
                         sel_out=None, stream=None):
        """The forward pass with the head-adaptive block-sparse sparse branch."""
        B, n_q = q.shape[0], q.shape[1]
        k_max = max(1, max(k_h)) if k_max is None else k_max
        if out is None:
            out = self.torch.empty_like(q)
        ws = self.workspace("fwd_adaptive", _h.hsa_adaptive_workspace_size(self.cfg, n_q, k_max, n_cur))
        _h.hsa_forward_adaptive(self.cfg, q, n_q, self.pool, n_cand, n_cur, k_h, k_max,
                                self.kv_state, self.k_state, self.page_kmean, g_lin, g_sp, out,
                                tau_min=tau_min, tau_max=tau_max, sel_out=sel_out, ws=ws,
                                stream=stream)
        return out

    def forward_linformer(self, q, n_cand: int, n_cur: int, k_h: Sequence[int],
                          k_max: Optional[int] = None, tau_min: float = _h.TAU_MIN,
                          tau_max: float = _h.TAU_MAX, g_lin=None, g_sp=None, out=None,
                          sel_out=None, stream=None):
        """The forward pass with the Linformer linear branch over the compressed
        pages and the head-adaptive block-sparse sparse branch."""
        B, n_q = q.shape[0], q.shape[1]
        k_max = max(1, max(k_h)) if k_max is None else k_max
        if out is None:
            out = self.torch.empty_like(q)
        ws = self.workspace("fwd_linformer", _h.hsa_linformer_workspace_size(self.cfg, n_q, k_max, n_cur))
        _h.hsa_forward_linformer(self.cfg, q, n_q, self.pool, self.ck, self.cv, self.rank, n_cand,
                                 n_cur, k_h, k_max, self.page_kmean, g_lin, g_sp, out,
                                 tau_min=tau_min, tau_max=tau_max, sel_out=sel_out, ws=ws,
                                 stream=stream)
        return out
