"""fp64 reference of the Linformer linear branch (TEST INFRASTRUCTURE).

This module is the checker, not the product. Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it. It shares no code with the HIP library.

Paper passages followed (WorldAttention, arxiv 2609.34606):
  * Sec. 3.3 "Linear branch": per head h two projections E_K^(h), E_V^(h)
    in R^{L x r} compress keys and values along the sequence,
    K~ = E_K^T K and V~ = E_V^T V (r x d each), and the branch output is
    softmax(Q K~^T / sqrt(d)) V~.
  * App. "Linear Branch": a growing KV sequence is cut into segments of the
    projection length L; each segment is projected on its own and the
    compressed segments are concatenated into one compressed context; the
    projection works at page level.
  * Sec. 3.3 "Gated fusion": o = sigmoid(g_lin) O_lin + sigmoid(g_sp) O_sp.

Readings (listed in the design notes):
  * a segment is one page (L = P), so a page is compressed once, when it is
    written, with the head's fixed projections;
  * the branch attends over the compressed versions of the pages HSA works
    on: the selected history pages and the current pages (the active KV of
    Sec. 3.2), the same list as the sparse branch;
  * the projections are inputs (the trained weights are not available); the
    softmax scale is that of the sparse branch;
  * the sparse branch is the head-adaptive block-sparse one of
    ``hsa_blocks_oracle`` (with tau = 1 it is the page-level one).

Pinning: ``tests/test_oracle_linformer_pins.py``.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np

from oracle import hsa_blocks_oracle as BO
from oracle import hsa_oracle as O


def compress(e: np.ndarray, x_page: np.ndarray) -> np.ndarray:
    """E^T X for one page (a segment of L = P tokens): e [r, P] holds E^T,
    x_page [P, d] the page's keys or values -> [r, d]."""
    return np.asarray(e, np.float64) @ np.asarray(x_page, np.float64)


def linformer_branch(q: np.ndarray, ck: Sequence[np.ndarray], cv: Sequence[np.ndarray],
                     scale: float):
    """softmax(q [ck_1; ck_2; ...]^T * scale) [cv_1; cv_2; ...] and its
    log-sum-exp, over the concatenated compressed pages."""
    return O.sparse_branch(np.asarray(q, np.float64), np.concatenate(ck, 0),
                           np.concatenate(cv, 0), scale)


def hsa_forward_linformer(q, k_pool, v_pool, page_table, e_k, e_v, n_cand: int, n_cur: int,
                          k_h: Sequence[int], tau_min: float = BO.TAU_MIN,
                          tau_max: float = BO.TAU_MAX, g_lin=None, g_sp=None,
                          sm_scale: Optional[float] = None,
                          heads: Optional[Sequence[int]] = None,
                          query_blocks: Optional[Sequence[int]] = None) -> Dict[str, object]:
    """HSA forward with the Linformer linear branch and the head-adaptive
    block-sparse sparse branch, gated as in Sec. 3.3.

    e_k, e_v: [H, r, P] (E^T of each head). Output rows are those of
    ``query_blocks`` (every query block by default)."""
    q = np.asarray(q)
    B, n_q, H, d = q.shape
    scale = (1.0 / np.sqrt(d)) if not sm_scale else float(sm_scale)
    heads = list(range(H)) if heads is None else list(heads)
    qb = BO.page_blocks(n_q, BO.BLOCK_Q)
    qsel = range(len(qb)) if query_blocks is None else list(query_blocks)
    rows = np.concatenate([np.arange(*qb[i]) for i in qsel]) if len(qsel) else np.zeros(0, np.int64)
    sp = BO.hsa_forward_adaptive(q, k_pool, v_pool, page_table, n_cand, n_cur, k_h, tau_min,
                                 tau_max, sm_scale=sm_scale, heads=heads, query_blocks=qsel,
                                 linear=False)
    out = {"O": np.zeros((B, len(rows), H, d)), "O_lin": np.zeros((B, len(rows), H, d)),
           "lse_lin": np.zeros((B, H, len(rows))), "O_sp": sp["O_sp"], "sel": sp["sel"],
           "kept": sp["kept"], "gini": sp["gini"], "tau": sp["tau"], "rows": rows}
    cur_pages = list(range(n_cand, n_cand + n_cur))
    for b in range(B):
        for h in heads:
            sel = [int(x) for x in sp["sel"][b, h] if x >= 0]
            ck, cv = [], []
            for p in sel + cur_pages:
                k_page, v_page = O.page_kv(k_pool, v_pool, page_table, b, h, p)
                ck.append(compress(e_k[h], k_page))
                cv.append(compress(e_v[h], v_page))
            o_lin, lse = linformer_branch(np.asarray(q[b, rows, h], np.float64), ck, cv, scale)
            out["O_lin"][b, :, h] = o_lin
            out["lse_lin"][b, h] = lse
            gl = None if g_lin is None else np.asarray(g_lin)[b, rows, h]
            gs = None if g_sp is None else np.asarray(g_sp)[b, rows, h]
            out["O"][b, :, h] = O.gated_merge(o_lin, sp["O_sp"][b, :, h], gl, gs)
    return out
