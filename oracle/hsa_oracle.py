"""fp64 reference computation of the HSA forward pass (TEST INFRASTRUCTURE).

This module is the checker, not the product. Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
it. It shares no code with the HIP library: it reads the same input arrays
(in the layout the C ABI documents) and recomputes every quantity from the
paper's definitions in plain numpy float64, one batch entry and one head at a
time, with no blocking or fusion.

Paper passages followed (WorldAttention, arxiv 2609.34606):
  * Sec. 3.2 "Stage 2: page-level retrieval": a page is scored by the scaled
    dot product of the chunk's average query and the page's average key;
    the top pages by that score are kept.
  * Sec. 3.2 "Active KV construction": the kept pages are concatenated.
  * Sec. 3.3 "Sparse branch": exact softmax attention restricted to the
    selected key set, i.e. App. A.1 eq. (attention) with a zero mask on it.
  * Sec. 3.3 "Gated fusion of two branches": the two branch outputs are
    weighted by sigmoid gates and summed.
  * The linear branch is the kernelised running-state form with feature map
    elu(x)+1 (a reading: the paper's own linear branch is a Linformer
    projection; see the readings list in the design notes).

Pinning: every function here is checked in ``tests/test_oracle_pins.py``
against something other than itself (a library routine, a brute-force
enumeration, the quadratic form, closed forms, invariants).
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np


# --------------------------------------------------------------------------
# elementary steps
# --------------------------------------------------------------------------

def phi(x: np.ndarray) -> np.ndarray:
    """Linear-branch feature map elu(x) + 1: x + 1 for x > 0, exp(x) otherwise."""
    x = np.asarray(x, dtype=np.float64)
    return np.where(x > 0.0, x + 1.0, np.exp(np.minimum(x, 0.0)))


def page_key_mean(k_page: np.ndarray) -> np.ndarray:
    """Average key of one page (Sec. 3.2, Stage 2): mean over its tokens. [P,d] -> [d]."""
    return np.asarray(k_page, dtype=np.float64).mean(axis=0)


def query_mean(q: np.ndarray) -> np.ndarray:
    """Average query of the current chunk (Sec. 3.2, Stage 2). [n_q,d] -> [d]."""
    return np.asarray(q, dtype=np.float64).mean(axis=0)


def page_scores(qbar: np.ndarray, kbar: np.ndarray) -> np.ndarray:
    """Stage-2 similarity: alpha_p = qbar . kbar_p / sqrt(d_k). kbar [N,d] -> [N]."""
    d = qbar.shape[-1]
    return (np.asarray(kbar, np.float64) @ np.asarray(qbar, np.float64)) / np.sqrt(d)


def select_top_pages(alpha: np.ndarray, k_h: int) -> np.ndarray:
    """Top-k_h candidate pages by score (Sec. 3.2, Stage 2).

    Ordered by (alpha descending, page index ascending): equal scores keep
    the lower (older) logical page first. At most len(alpha) pages.
    """
    n = alpha.shape[0]
    k_eff = max(0, min(int(k_h), n))
    order = np.lexsort((np.arange(n), -alpha))
    return order[:k_eff].astype(np.int64)


def linear_state(k: np.ndarray, v: np.ndarray):
    """Running state of the kernelised linear branch over keys k, values v [N,d].

    S = sum_t phi(k_t) v_t^T  ([d_k, d_v]) and z = sum_t phi(k_t)  ([d_k]).
    """
    fk = phi(k)
    return fk.T @ np.asarray(v, np.float64), fk.sum(axis=0)


def linear_branch(q: np.ndarray, S: np.ndarray, z: np.ndarray) -> np.ndarray:
    """O_lin[i] = phi(q_i)^T S / (phi(q_i) . z). q [n,d] -> [n,d_v]."""
    fq = phi(q)
    return (fq @ S) / (fq @ z)[:, None]


def sparse_branch(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float):
    """Exact softmax attention of q over the key set (k, v).

    App. A.1 eq. (attention) with M = 0 on the selected keys:
    S = q k^T * scale, A = softmax(S) row-wise, O = A v. Also returns the
    row log-sum-exp of S (natural log).
    """
    s = (np.asarray(q, np.float64) @ np.asarray(k, np.float64).T) * scale
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    den = e.sum(axis=1, keepdims=True)
    o = (e @ np.asarray(v, np.float64)) / den
    return o, (m + np.log(den))[:, 0]


def sigmoid(g: np.ndarray) -> np.ndarray:
    g = np.asarray(g, np.float64)
    return 1.0 / (1.0 + np.exp(-g))


def gated_merge(o_lin, o_sp, g_lin=None, g_sp=None):
    """O = O_lin * sigmoid(G_lin) + O_sp * sigmoid(G_sp) (Sec. 3.3, gated fusion).

    The paper leaves the gate shape open (head-level gates, yet an
    element-wise product with the branch outputs). A gate array with one axis
    fewer than the outputs is per query and head and broadcast over the head
    dimension; one with the outputs' shape is element-wise. Absent gates mean
    logit 0, i.e. weight 1/2 each.
    """
    def weight(g):
        if g is None:
            return 0.5
        w = sigmoid(g)
        return w if w.ndim == np.ndim(o_lin) else w[..., None]
    return weight(g_lin) * o_lin + weight(g_sp) * o_sp


# --------------------------------------------------------------------------
# pool access (layout only: [slot,H,P,d] keys, [slot,H,d,P] values)
# --------------------------------------------------------------------------

def page_kv(k_pool, v_pool, page_table, b: int, h: int, p: int):
    slot = int(page_table[b, p])
    k = np.asarray(k_pool[slot, h], np.float64)          # [P, d]
    v = np.asarray(v_pool[slot, h], np.float64).T        # [P, d]
    return k, v


def gather_pages(k_pool, v_pool, page_table, b, h, pages: Sequence[int]):
    """Active KV of one head: concatenation of the listed pages (Sec. 3.2)."""
    d = k_pool.shape[-1]
    if len(pages) == 0:
        return np.zeros((0, d)), np.zeros((0, d))
    ks, vs = zip(*(page_kv(k_pool, v_pool, page_table, b, h, p) for p in pages))
    return np.concatenate(ks, 0), np.concatenate(vs, 0)


# --------------------------------------------------------------------------
# whole pass
# --------------------------------------------------------------------------

def hsa_forward(q, k_pool, v_pool, page_table, n_cand: int, n_cur: int,
                k_h: Sequence[int], g_lin=None, g_sp=None,
                sm_scale: Optional[float] = None, k_max: Optional[int] = None,
                heads: Optional[Sequence[int]] = None,
                query_rows: Optional[Sequence[int]] = None,
                state_pages: Optional[Sequence[int]] = None,
                cand_range: Optional[Sequence[Sequence[int]]] = None) -> Dict[str, np.ndarray]:
    """HSA forward for one chunk.

    q [B,n_q,H,d]; history (candidate) pages are logical pages [0, n_cand);
    the current chunk's pages are [n_cand, n_cand+n_cur). Per head h:
      1. page index: mean key of every candidate page;
      2. chunk summary: mean query over all n_q queries;
      3. scores alpha = qbar . kbar / sqrt(d) and the top-k_h pages;
      4. active keys: the selected pages followed by the current pages;
      5. sparse branch: exact softmax attention over the active keys;
      6. linear branch over the state of ``state_pages`` (default: every page
         up to and including the current chunk);
      7. gated merge.
    ``query_rows`` restricts steps 5-7 to some queries (step 2 always uses
    all of them); ``heads`` restricts everything to some heads.
    ``cand_range[b] = (lo, hi)`` restricts the candidates of batch entry b
    to logical pages [lo, hi) within the history (Stage-1 retrieval picks
    one chunk); ``alpha`` then holds scores at those positions only.
    """
    q = np.asarray(q)
    B, n_q, H, d = q.shape
    scale = (1.0 / np.sqrt(d)) if not sm_scale else float(sm_scale)
    heads = list(range(H)) if heads is None else list(heads)
    rows = np.arange(n_q) if query_rows is None else np.asarray(query_rows)
    k_max = max(k_h) if k_max is None else int(k_max)
    if state_pages is None:
        state_pages = range(n_cand + n_cur)
    state_pages = list(state_pages)
    cur_pages = list(range(n_cand, n_cand + n_cur))
    nr = len(rows)
    out = {
        "O": np.zeros((B, nr, H, d)), "O_lin": np.zeros((B, nr, H, d)),
        "O_sp": np.zeros((B, nr, H, d)), "lse": np.zeros((B, H, nr)),
        "sel": -np.ones((B, H, k_max), np.int64),
        "sel_score": np.zeros((B, H, k_max)),
        "alpha": np.zeros((B, H, n_cand)), "qbar": np.zeros((B, H, d)),
        "kbar": np.zeros((B, H, n_cand + n_cur, d)),
        "S": np.zeros((B, H, d, d)), "z": np.zeros((B, H, d)),
    }
    for b in range(B):
        for h in heads:
            kbar = np.stack([page_key_mean(k_pool[int(page_table[b, p]), h])
                             for p in range(n_cand + n_cur)]) if n_cand + n_cur else np.zeros((0, d))
            qbar = query_mean(q[b, :, h, :])
            lo, hi = (0, n_cand) if cand_range is None else (int(cand_range[b][0]), int(cand_range[b][1]))
            alpha = np.zeros(n_cand)
            alpha[lo:hi] = page_scores(qbar, kbar[lo:hi])
            sel = lo + select_top_pages(alpha[lo:hi], k_h[h])
            out["kbar"][b, h] = kbar
            out["qbar"][b, h] = qbar
            out["alpha"][b, h] = alpha
            out["sel"][b, h, :len(sel)] = sel
            out["sel_score"][b, h, :len(sel)] = alpha[sel]
            k_act, v_act = gather_pages(k_pool, v_pool, page_table, b, h,
                                        list(sel) + cur_pages)
            qh = np.asarray(q[b, rows, h, :], np.float64)
            o_sp, lse = sparse_branch(qh, k_act, v_act, scale)
            k_st, v_st = gather_pages(k_pool, v_pool, page_table, b, h, state_pages)
            S, z = linear_state(k_st, v_st)
            o_lin = linear_branch(qh, S, z)
            gl = None if g_lin is None else np.asarray(g_lin)[b, rows, h]
            gs = None if g_sp is None else np.asarray(g_sp)[b, rows, h]
            out["O_sp"][b, :, h] = o_sp
            out["O_lin"][b, :, h] = o_lin
            out["O"][b, :, h] = gated_merge(o_lin, o_sp, gl, gs)
            out["lse"][b, h] = lse
            out["S"][b, h], out["z"][b, h] = S, z
    return out
