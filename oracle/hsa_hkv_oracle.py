"""fp64 reference of the two-stage retrieval of the hierarchical KV cache
(TEST INFRASTRUCTURE).

This module is the checker, not the product. Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it. It shares no code with the HIP library.

Paper passages followed (WorldAttention, arxiv 2609.34606):
  * Sec. 3.2 "Global KV bank initialization": the bank is a sequence of KV
    chunks C_1..C_M, one per video segment, each cut into pages.
  * Sec. 3.2 "Stage 1: prompt-level retrieval": the cosine similarity
    between the current prompt embedding and every previous chunk's prompt
    embedding selects the top-1 chunk, whose pages are the Stage-2
    candidates.
  * Sec. 3.2 "Stage 2: page-level retrieval" and the rest of the forward
    pass: those of ``hsa_oracle.hsa_forward`` with the candidates restricted
    to the chosen chunk's pages.

Readings (listed in the design notes):
  * chunk m covers the logical pages [chunk_first[m], chunk_first[m+1]) of
    the history, chunks in generation order;
  * the top-1 chunk breaks ties by the lower chunk index; an embedding of
    norm 0 has cosine 0 with everything;
  * the linear branch still covers every page written so far (the state is
    folded at write time, before any page can move to a lower tier).

Pinning: ``tests/test_oracle_hkv_pins.py``.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np

from oracle import hsa_oracle as O


def cosine_scores(prompt: np.ndarray, chunks: np.ndarray) -> np.ndarray:
    """cos(prompt, c_m) for every row c_m of chunks [M, E] (fp64). Each dot
    product is its own sum over E, so chunks that differ by an exact scale
    factor get bit-equal cosines and their tie falls to the lower index."""
    p = np.asarray(prompt, np.float64)
    c = np.asarray(chunks, np.float64)
    num = (c * p[None, :]).sum(axis=1)
    den = np.linalg.norm(c, axis=1) * np.linalg.norm(p)
    out = np.zeros(c.shape[0])
    ok = den > 0
    out[ok] = num[ok] / den[ok]
    return out


def select_chunk(scores: np.ndarray) -> int:
    """Top-1 chunk, ties to the lower index."""
    return int(np.argmax(np.asarray(scores, np.float64)))


def hsa_forward_retrieval(q, k_pool, v_pool, page_table, prompt_emb, chunk_emb, chunk_first,
                          n_cur: int, k_h: Sequence[int], g_lin=None, g_sp=None,
                          sm_scale: Optional[float] = None, k_max: Optional[int] = None,
                          heads: Optional[Sequence[int]] = None,
                          query_rows: Optional[Sequence[int]] = None) -> Dict[str, object]:
    """Stage-1 chunk retrieval, then the HSA forward with the Stage-2
    candidates restricted to the chosen chunk's pages.

    prompt_emb [B, E], chunk_emb [B, M, E], chunk_first [B, M+1]; the history
    is logical pages [0, chunk_first[b][M]) (the same for every b)."""
    B = np.asarray(q).shape[0]
    chunk_first = np.asarray(chunk_first)
    n_cand = int(chunk_first[0, -1])
    chunk, score, ranges = [], [], []
    for b in range(B):
        sc = cosine_scores(prompt_emb[b], chunk_emb[b])
        m = select_chunk(sc)
        chunk.append(m)
        score.append(sc[m])
        ranges.append((int(chunk_first[b, m]), int(chunk_first[b, m + 1])))
    out = O.hsa_forward(q, k_pool, v_pool, page_table, n_cand, n_cur, k_h, g_lin, g_sp,
                        sm_scale=sm_scale, k_max=k_max, heads=heads, query_rows=query_rows,
                        cand_range=ranges)
    out["chunk"] = np.array(chunk, np.int64)
    out["chunk_score"] = np.array(score)
    return out
