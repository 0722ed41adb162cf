"""fp64 reference of the head-adaptive block-sparse sparse branch (TEST INFRASTRUCTURE).

This module is the checker, not the product. Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it. It shares no code with the HIP library.

Paper passages followed (WorldAttention, arxiv 2609.34606):
  * Sec. 3.3 "Sparse branch": tokens of the retrieved pages are cut into
    blocks of B tokens; a pooled (block-level) attention map picks, per head,
    the blocks each query block attends to; attention then runs at token
    resolution inside the chosen blocks only. History pages use blocks of
    B_inter = 128 tokens, the current chunk blocks of B_intra = 64.
  * App. "Sparse Branch": for query block i of head h, the blocks sorted by
    descending block weight p_{i,:}; the kept set is the shortest prefix of
    that order whose summed weight reaches the head's coverage threshold
    tau_h; the Gini coefficient of the sorted weights, averaged over query
    blocks, sets tau_h = tau_min + G (tau_max - tau_min).
  * Sec. 4.5 (HSA ablation table): (tau_max, tau_min) = (1.00, 0.35) is the
    paper's chosen setting.

Readings (where the paper leaves a choice open; listed in the design notes):
  * the pooled map is the row softmax over key blocks of the scaled dot
    product of mean-pooled query and key blocks (scale 1/sqrt(d));
  * blocks are consecutive runs of B tokens inside each page (the last block
    of a page is shorter when B does not divide the page); pages are never
    merged into one block; query blocks are consecutive runs of 64 queries;
  * the kept prefix uses the order (weight descending, block index
    ascending); if rounding keeps the total below tau_h, every block is kept,
    and tau_h >= 1 keeps every block (the running sum may round to 1 early);
  * key blocks of one head are numbered page by page in list order (the
    selected history pages first, then the current chunk's pages).

Pinning: ``tests/test_oracle_blocks_pins.py``.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from oracle import hsa_oracle as O

BLOCK_Q = 64        # queries per query block
BLOCK_HIST = 128    # tokens per key block of a retrieved history page (B_inter)
BLOCK_CUR = 64      # tokens per key block of a current-chunk page (B_intra)
TAU_MIN, TAU_MAX = 0.35, 1.00


def page_blocks(P: int, B: int) -> List[Tuple[int, int]]:
    """[start, end) token ranges of the blocks of one page of P tokens."""
    return [(s, min(s + B, P)) for s in range(0, P, B)]


def list_blocks(n_hist: int, n_cur: int, P: int, b_hist: int = BLOCK_HIST,
                b_cur: int = BLOCK_CUR) -> List[Tuple[int, int, int]]:
    """Key blocks of one head's page list: (list position, start, end).

    The first n_hist list positions are retrieved history pages (blocks of
    b_hist tokens), the next n_cur the current chunk's pages (b_cur).
    """
    out = []
    for li in range(n_hist + n_cur):
        B = b_hist if li < n_hist else b_cur
        out += [(li, s, e) for s, e in page_blocks(P, B)]
    return out


def block_means(x: np.ndarray, bounds: Sequence[Tuple[int, int]]) -> np.ndarray:
    """Mean of rows [s, e) of x for each (s, e): [len(bounds), d] (fp64)."""
    x = np.asarray(x, np.float64)
    return np.stack([x[s:e].mean(axis=0) for s, e in bounds]) if len(bounds) else np.zeros((0, x.shape[1]))


def pooled_map(qbar: np.ndarray, kbar: np.ndarray, scale: float) -> np.ndarray:
    """Block attention weights: row softmax of qbar kbar^T * scale. [NQ,N].

    Each score is its own sum over d (not a blocked matrix product), so equal
    key blocks get bit-equal weights and their tie falls to the block id."""
    qbar = np.asarray(qbar, np.float64)
    kbar = np.asarray(kbar, np.float64)
    s = (qbar[:, None, :] * kbar[None, :, :]).sum(axis=-1) * scale
    s -= s.max(axis=1, keepdims=True)
    e = np.exp(s)
    return e / e.sum(axis=1, keepdims=True)


def block_order(p_row: np.ndarray) -> np.ndarray:
    """Block indices by weight descending, ties by lower index."""
    n = p_row.shape[0]
    return np.lexsort((np.arange(n), -p_row))


def gini(pm: np.ndarray) -> float:
    """Gini coefficient of a head's pooled map, averaged over query blocks:
    E_i[(1/N) sum_m (N - 2m + 1) p_{i,sigma_i(m)}] with m = 1..N over the
    descending order."""
    pm = np.asarray(pm, np.float64)
    nq, n = pm.shape
    if nq == 0 or n == 0:
        return 0.0
    w = (n - 2.0 * np.arange(1, n + 1) + 1.0) / n
    return float(np.mean([np.dot(w, row[block_order(row)]) for row in pm]))


def coverage_threshold(g: float, tau_min: float = TAU_MIN, tau_max: float = TAU_MAX) -> float:
    """tau_h = tau_min + G (tau_max - tau_min)."""
    return tau_min + g * (tau_max - tau_min)


def select_blocks(p_row: np.ndarray, tau: float) -> np.ndarray:
    """Shortest prefix of the descending order whose running sum (in that
    order) reaches tau; all blocks when it never does. A threshold of 1 or
    more is the whole mass, so it keeps every block whatever the rounding of
    the running sum."""
    order = block_order(p_row)
    if tau >= 1.0:
        return order
    c = np.cumsum(np.asarray(p_row, np.float64)[order])
    hit = np.nonzero(c >= tau)[0]
    k = (hit[0] + 1) if hit.size else order.size
    return order[:k]


def adaptive_head(q: np.ndarray, k_list: Sequence[np.ndarray], v_list: Sequence[np.ndarray],
                  n_hist: int, scale: float, tau_min: float = TAU_MIN, tau_max: float = TAU_MAX,
                  block_q: int = BLOCK_Q, b_hist: int = BLOCK_HIST, b_cur: int = BLOCK_CUR,
                  query_blocks: Optional[Sequence[int]] = None) -> Dict[str, object]:
    """Sparse branch of one head with head-adaptive block selection.

    q [n_q,d]; k_list/v_list: the [P,d] keys and values of each list page
    (history pages first). Returns the pooled map, G, tau, the kept blocks of
    every query block, and O_sp / lse for the rows of ``query_blocks`` (all
    by default), in row order.
    """
    q = np.asarray(q, np.float64)
    n_q, d = q.shape
    n_list = len(k_list)
    P = k_list[0].shape[0] if n_list else 0
    blocks = list_blocks(n_hist, n_list - n_hist, P, b_hist, b_cur)
    # mean key of every block, page by page in list order
    kbar = np.concatenate([block_means(k_list[li], page_blocks(P, b_hist if li < n_hist else b_cur))
                           for li in range(n_list)], 0) if blocks else np.zeros((0, d))
    qb = page_blocks(n_q, block_q)
    qbar = block_means(q, qb)
    pm = pooled_map(qbar, kbar, scale) if blocks else np.zeros((len(qb), 0))
    g = gini(pm)
    tau = coverage_threshold(g, tau_min, tau_max)
    kept = [select_blocks(pm[i], tau) for i in range(len(qb))]
    qsel = range(len(qb)) if query_blocks is None else list(query_blocks)
    rows, o_sp, lse = [], [], []
    for i in qsel:
        s, e = qb[i]
        ks = np.concatenate([np.asarray(k_list[blocks[j][0]], np.float64)[blocks[j][1]:blocks[j][2]]
                             for j in kept[i]], 0)
        vs = np.concatenate([np.asarray(v_list[blocks[j][0]], np.float64)[blocks[j][1]:blocks[j][2]]
                             for j in kept[i]], 0)
        o, l = O.sparse_branch(q[s:e], ks, vs, scale)
        rows.append(np.arange(s, e))
        o_sp.append(o)
        lse.append(l)
    return {"blocks": blocks, "pooled": pm, "gini": g, "tau": tau, "kept": kept,
            "rows": np.concatenate(rows) if rows else np.zeros(0, np.int64),
            "O_sp": np.concatenate(o_sp, 0) if o_sp else np.zeros((0, d)),
            "lse": np.concatenate(lse) if lse else np.zeros(0)}


def hsa_forward_adaptive(q, k_pool, v_pool, page_table, n_cand: int, n_cur: int,
                         k_h: Sequence[int], tau_min: float = TAU_MIN, tau_max: float = TAU_MAX,
                         g_lin=None, g_sp=None, sm_scale: Optional[float] = None,
                         heads: Optional[Sequence[int]] = None,
                         query_blocks: Optional[Sequence[int]] = None,
                         state_pages: Optional[Sequence[int]] = None,
                         linear: bool = True) -> Dict[str, object]:
    """HSA forward with the head-adaptive block-sparse sparse branch.

    Steps 1-4 (page index, chunk summary, top-k_h pages, page list) and the
    linear branch are those of ``hsa_oracle.hsa_forward``; the sparse branch
    attends, for each query block, to its kept key blocks only. Output rows
    are those of ``query_blocks`` (all query blocks by default). With
    ``linear=False`` the kernelised linear branch and the merge are skipped
    ("O" stays zero) for callers that bring their own linear branch.
    """
    q = np.asarray(q)
    B, n_q, H, d = q.shape
    scale = (1.0 / np.sqrt(d)) if not sm_scale else float(sm_scale)
    heads = list(range(H)) if heads is None else list(heads)
    if state_pages is None:
        state_pages = range(n_cand + n_cur)
    state_pages = list(state_pages)
    qb = page_blocks(n_q, BLOCK_Q)
    qsel = range(len(qb)) if query_blocks is None else list(query_blocks)
    rows = np.concatenate([np.arange(*qb[i]) for i in qsel]) if len(qsel) else np.zeros(0, np.int64)
    nr = len(rows)
    cur_pages = list(range(n_cand, n_cand + n_cur))
    out = {"O": np.zeros((B, nr, H, d)), "O_sp": np.zeros((B, nr, H, d)), "lse": np.zeros((B, H, nr)),
           "sel": np.full((B, H, max(1, max(k_h))), -1, np.int64), "gini": np.zeros((B, H)),
           "tau": np.zeros((B, H)), "kept": {}, "pooled": {}, "rows": rows}
    for b in range(B):
        for h in heads:
            cand = [O.page_key_mean(k_pool[int(page_table[b, p]), h]) for p in range(n_cand)]
            qbar = O.query_mean(q[b, :, h])
            alpha = O.page_scores(qbar, np.stack(cand)) if n_cand else np.zeros(0)
            sel = O.select_top_pages(alpha, k_h[h]) if n_cand else np.zeros(0, np.int64)
            out["sel"][b, h, :len(sel)] = sel
            pages = list(sel) + cur_pages
            kv = [O.page_kv(k_pool, v_pool, page_table, b, h, p) for p in pages]
            r = adaptive_head(q[b, :, h], [x[0] for x in kv], [x[1] for x in kv], len(sel), scale,
                              tau_min, tau_max, query_blocks=qsel)
            out["gini"][b, h], out["tau"][b, h] = r["gini"], r["tau"]
            out["kept"][(b, h)] = r["kept"]
            out["pooled"][(b, h)] = r["pooled"]
            out["O_sp"][b, :, h] = r["O_sp"]
            out["lse"][b, h] = r["lse"]
            if not linear:
                continue
            kl, vl = O.gather_pages(k_pool, v_pool, page_table, b, h, state_pages)
            S, z = O.linear_state(kl, vl)
            o_lin = O.linear_branch(np.asarray(q[b, rows, h], np.float64), S, z)
            gl = None if g_lin is None else np.asarray(g_lin)[b, rows, h]
            gs = None if g_sp is None else np.asarray(g_sp)[b, rows, h]
            out["O"][b, :, h] = O.gated_merge(o_lin, r["O_sp"], gl, gs)
    return out
