"""Seeded generators for HSA inputs, in the C ABI's memory layout.

Layouts (shared with the library header):
  q          [B, n_q, H, d]              token-major, as a projection writes it
  k_pool     [num_slots, H, P, d]        one page of one head is P rows of d
  v_pool     [num_slots, H, d, P]        value pages are stored d-major
  page_table [B, max_pages] int32        logical page -> physical slot
  g_lin/g_sp [B, n_q, H] float32         gate logits (optional)

Every tensor is drawn from its own stream,
``SeedSequence([workload_seed, layer, chunk, tensor_id])``, so draws do not
depend on generation order. bf16 workloads round fp32 draws to bf16 with
round-to-nearest-even; the returned arrays hold those bf16 values as fp32.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

from .configs import Workload

# tensor ids inside a (seed, layer, chunk) stream family
T_Q, T_K, T_V, T_PERM, T_GLIN, T_GSP, T_CENTROIDS, T_ASSIGN, T_EK, T_EV, T_PROMPT = range(11)


def _ss(wl: Workload, layer: int, chunk: int, tid: int) -> np.random.SeedSequence:
    return np.random.SeedSequence([wl.seed, layer, chunk, tid])


def seed_int(wl: Workload, layer: int, chunk: int, tid: int) -> int:
    """A 63-bit integer seed for generators that take one (torch)."""
    return int(_ss(wl, layer, chunk, tid).generate_state(2, np.uint64)[0] >> np.uint64(1))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _round(wl: Workload, x: np.ndarray) -> np.ndarray:
    x = x.astype(np.float32, copy=False)
    if wl.dtype == "bf16":
        return bf16_bits_to_f32(f32_to_bf16_bits(x))
    return x


@dataclasses.dataclass
class Case:
    wl: Workload
    q: np.ndarray
    k_pool: np.ndarray
    v_pool: np.ndarray
    page_table: np.ndarray
    k_h: np.ndarray
    g_lin: Optional[np.ndarray] = None
    g_sp: Optional[np.ndarray] = None
    meta: Dict = dataclasses.field(default_factory=dict)

    @property
    def num_slots(self) -> int:
        return self.k_pool.shape[0]


def slot_permutation(wl: Workload, layer: int = 0, chunk: int = 0) -> np.ndarray:
    n = wl.batch * wl.n_pages
    return np.random.default_rng(_ss(wl, layer, chunk, T_PERM)).permutation(n).astype(np.int32)


def _cluster_layout(wl: Workload, layer: int, chunk: int):
    """Clustered pages: 32 per-head centroids of norm 4, runs of 10 pages.

    The run 100 pages before the end of the history gets cluster c*; no later
    run uses c*. The query chunk and the current pages are drawn near c*.
    """
    H, d = wl.heads, wl.head_dim
    rc = np.random.default_rng(_ss(wl, layer, chunk, T_CENTROIDS))
    cent = rc.standard_normal((H, 32, d))
    cent *= 4.0 / np.linalg.norm(cent, axis=-1, keepdims=True)
    ra = np.random.default_rng(_ss(wl, layer, chunk, T_ASSIGN))
    c_star = int(ra.integers(32))
    runs = max(1, (wl.n_cand + 9) // 10)
    assign = ra.integers(0, 32, runs)
    star_run = max(0, runs - 10)
    assign[star_run] = c_star
    others = np.array([c for c in range(32) if c != c_star])
    if runs > star_run + 1:
        assign[star_run + 1:] = ra.choice(others, runs - star_run - 1)
    page_cluster = np.array([assign[p // 10] for p in range(wl.n_cand)], dtype=np.int64)
    return cent.astype(np.float32), c_star, page_cluster


def make_case(wl: Workload, layer: int = 0, chunk: int = 0) -> Case:
    """Host (numpy) inputs for one layer and one chunk of a workload."""
    B, H, d, P, nq = wl.batch, wl.heads, wl.head_dim, wl.page_size, wl.n_q
    npg = wl.n_pages
    rq = np.random.default_rng(_ss(wl, layer, chunk, T_Q))
    rk = np.random.default_rng(_ss(wl, layer, chunk, T_K))
    rv = np.random.default_rng(_ss(wl, layer, chunk, T_V))
    s = np.float32(wl.value_scale)
    meta: Dict = {}
    if wl.structure == "clusters":
        cent, c_star, page_cluster = _cluster_layout(wl, layer, chunk)
        meta.update(c_star=c_star, page_cluster=page_cluster)
        noise = np.float32(0.5)
        q = rq.standard_normal((B, nq, H, d), dtype=np.float32) * noise
        q += cent[None, None, np.arange(H), c_star, :]
        k_log = rk.standard_normal((B, npg, H, P, d), dtype=np.float32) * noise
        for p in range(npg):
            c = page_cluster[p] if p < wl.n_cand else c_star
            k_log[:, p] += cent[None, :, c, None, :]
    elif wl.structure == "gaussian":
        q = rq.standard_normal((B, nq, H, d), dtype=np.float32) * s
        k_log = rk.standard_normal((B, npg, H, P, d), dtype=np.float32) * s
    else:
        raise ValueError(wl.structure)
    v_log = rv.standard_normal((B, npg, H, d, P), dtype=np.float32) * s
    perm = slot_permutation(wl, layer, chunk)
    nslots = B * npg
    k_pool = np.empty((nslots, H, P, d), np.float32)
    v_pool = np.empty((nslots, H, d, P), np.float32)
    k_pool[perm] = _round(wl, k_log.reshape(nslots, H, P, d))
    v_pool[perm] = _round(wl, v_log.reshape(nslots, H, d, P))
    del k_log, v_log
    page_table = perm.reshape(B, npg).astype(np.int32)
    g_lin = g_sp = None
    if wl.gates:
        g_lin = np.random.default_rng(_ss(wl, layer, chunk, T_GLIN)).standard_normal(
            (B, nq, H), dtype=np.float32)
        g_sp = np.random.default_rng(_ss(wl, layer, chunk, T_GSP)).standard_normal(
            (B, nq, H), dtype=np.float32)
    return Case(wl, _round(wl, q), k_pool, v_pool, page_table,
                np.array(wl.budgets(), np.int32), g_lin, g_sp, meta)


def make_case_torch(wl: Workload, device, layer: int = 0, chunk: int = 0,
                    k_pool=None, v_pool=None, slot_base: int = 0):
    """Device inputs drawn with torch generators (for full-size workloads).

    Values differ from ``make_case`` (a different generator) but follow the
    same recipe. Returns a dict of device tensors in the ABI layout, with
    ``q``/``k_pool``/``v_pool`` in the workload dtype. When ``k_pool`` and
    ``v_pool`` are given, the new pages are written into slots
    ``slot_base + perm`` of those pools instead of fresh ones.
    """
    import torch

    B, H, d, P, nq = wl.batch, wl.heads, wl.head_dim, wl.page_size, wl.n_q
    npg = wl.n_pages
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32

    def gen(tid):
        g = torch.Generator(device=device)
        g.manual_seed(seed_int(wl, layer, chunk, tid))
        return g

    s = float(wl.value_scale)
    meta = {}
    perm = torch.from_numpy(slot_permutation(wl, layer, chunk).astype(np.int64)).to(device)
    nslots = B * npg
    if k_pool is None:
        k_pool = torch.empty((nslots, H, P, d), dtype=dt, device=device)
        v_pool = torch.empty((nslots, H, d, P), dtype=dt, device=device)
    slots = perm + slot_base
    gk, gv = gen(T_K), gen(T_V)
    if wl.structure == "clusters":
        cent, c_star, page_cluster = _cluster_layout(wl, layer, chunk)
        meta.update(c_star=c_star, page_cluster=page_cluster)
        cent_t = torch.from_numpy(cent).to(device)
        q = torch.randn((B, nq, H, d), generator=gen(T_Q), device=device) * 0.5
        q += cent_t[torch.arange(H, device=device), c_star][None, None]
    else:
        q = torch.randn((B, nq, H, d), generator=gen(T_Q), device=device) * s
    # pages are drawn one logical page at a time to bound temporary memory
    for b in range(B):
        for p in range(npg):
            lp = b * npg + p
            kk = torch.randn((H, P, d), generator=gk, device=device)
            if wl.structure == "clusters":
                c = int(page_cluster[p]) if p < wl.n_cand else c_star
                kk = kk * 0.5 + cent_t[:, c, None, :]
            else:
                kk = kk * s
            vv = torch.randn((H, d, P), generator=gv, device=device) * s
            k_pool[slots[lp]] = kk.to(dt)
            v_pool[slots[lp]] = vv.to(dt)
    page_table = slots.reshape(B, npg).to(torch.int32)
    out = dict(q=q.to(dt).contiguous(), k_pool=k_pool, v_pool=v_pool,
               page_table=page_table.contiguous(),
               k_h=np.array(wl.budgets(), np.int32), meta=meta)
    if wl.gates:
        out["g_lin"] = torch.randn((B, nq, H), generator=gen(T_GLIN), device=device)
        out["g_sp"] = torch.randn((B, nq, H), generator=gen(T_GSP), device=device)
    return out


def make_projections(wl: Workload, rank: int, kind: str = "gaussian", layer: int = 0):
    """Compression weights of a Linformer-style linear branch, per head, in
    the layout the library reads: e[h][j][t] for rank j and token t of a
    page ([H, rank, P], the transpose of an L x r projection with L = P).

    The trained weights are not available, so they are drawn:
      * "gaussian": N(0, 1/P) entries, so that a compressed token of unit
        variance inputs has unit variance;
      * "meanpool": row j holds 1/n on its own run of n = P / rank
        consecutive tokens (P a multiple of rank) and 0 elsewhere.
    Returns (e_k, e_v) as float32 arrays holding workload-dtype values.
    """
    H, P = wl.heads, wl.page_size
    if kind == "gaussian":
        s = np.float32(1.0 / np.sqrt(P))
        e_k = np.random.default_rng(_ss(wl, layer, 0, T_EK)).standard_normal(
            (H, rank, P), dtype=np.float32) * s
        e_v = np.random.default_rng(_ss(wl, layer, 0, T_EV)).standard_normal(
            (H, rank, P), dtype=np.float32) * s
    elif kind == "meanpool":
        if P % rank:
            raise ValueError("meanpool needs P to be a multiple of rank")
        n = P // rank
        e_k = np.zeros((H, rank, P), np.float32)
        for j in range(rank):
            e_k[:, j, j * n:(j + 1) * n] = np.float32(1.0 / n)
        e_v = e_k.copy()
    else:
        raise ValueError(kind)
    return _round(wl, e_k), _round(wl, e_v)


def make_prompts(wl: Workload, emb_dim: int = 4096, layer: int = 0, chunk: int = 0):
    """Prompt embeddings of the KV bank's chunks and of the current chunk.

    Chunks are runs of consecutive history pages: the clustered workload's
    runs of 10 pages (one prompt per run), otherwise generation chunks of
    n_cur pages. Each cluster (or chunk) gets a seeded N(0,1) direction; a
    chunk's embedding is its direction plus N(0, 0.3^2) noise, and the
    current prompt is the direction of the current chunk's cluster (the
    clustered workload) or of a random chunk, plus noise.
    Returns (prompt_emb [B, E], chunk_emb [B, M, E], chunk_first [B, M+1]
    int32) as float32 / int32 arrays.
    """
    B = wl.batch
    rng = np.random.default_rng(_ss(wl, layer, chunk, T_PROMPT))
    if wl.structure == "clusters":
        run = 10
        _, c_star, page_cluster = _cluster_layout(wl, layer, chunk)
        first = list(range(0, wl.n_cand, run)) + [wl.n_cand]
        labels = [int(page_cluster[f]) for f in first[:-1]]
        target = c_star
        n_dir = 32
    else:
        run = max(1, wl.n_cur)
        first = list(range(0, wl.n_cand, run)) + [wl.n_cand]
        labels = list(range(len(first) - 1))
        n_dir = max(1, len(labels))
        target = int(rng.integers(n_dir))
    dirs = rng.standard_normal((n_dir, emb_dim)).astype(np.float32)
    M = len(labels)
    chunk_emb = np.empty((B, M, emb_dim), np.float32)
    prompt = np.empty((B, emb_dim), np.float32)
    for b in range(B):
        chunk_emb[b] = dirs[labels] + np.float32(0.3) * rng.standard_normal((M, emb_dim), dtype=np.float32)
        prompt[b] = dirs[target] + np.float32(0.3) * rng.standard_normal(emb_dim, dtype=np.float32)
    chunk_first = np.tile(np.asarray(first, np.int32), (B, 1))
    return prompt, chunk_emb, chunk_first
