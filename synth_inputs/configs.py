"""Workload shapes for the HSA forward pass.

The video-model shapes come from the paper's setting (Wan2.1 at 480p): one
latent frame is 1560 tokens, a generation chunk is three latent frames
(4680 query tokens), and a page holds the keys and values of consecutive
frames (Sec. "Hierarchical KV Cache", Stage-2 page-level retrieval). Here a
page is one latent frame (1560 tokens) unless a workload says otherwise.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    heads: int
    head_dim: int
    n_q: int               # queries in the current chunk
    page_size: int         # tokens per KV page
    n_cand: int            # history pages (retrieval candidates)
    n_cur: int             # pages holding the current chunk's own keys/values
    k_h: Optional[Tuple[int, ...]]  # per-head page budget; None -> draw_k_h
    dtype: str             # "bf16" or "f32"
    seed: int
    value_scale: float = 1.0       # q, k, v are drawn as N(0,1) * value_scale
    structure: str = "gaussian"    # "gaussian" or "clusters"
    k_h_choices: Tuple[int, ...] = ()
    layers: int = 1
    chunks: int = 1
    gates: bool = False            # draw N(0,1) gate logits

    @property
    def n_pages(self) -> int:
        return self.n_cand + self.n_cur

    @property
    def k_max(self) -> int:
        return max(self.budgets())

    def budgets(self) -> Tuple[int, ...]:
        if self.k_h is not None:
            return tuple(int(x) for x in self.k_h)
        rng = np.random.default_rng(np.random.SeedSequence([self.seed, 0, 0, 99]))
        return tuple(int(x) for x in rng.choice(np.array(self.k_h_choices), self.heads))

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # Tiny fp32 case that the oracle finishes in well under a second.
    "c1": Workload("c1_tiny_f32", batch=1, heads=2, head_dim=64, n_q=256,
                   page_size=256, n_cand=8, n_cur=1, k_h=(2, 2), dtype="f32",
                   seed=0, value_scale=64 ** -0.25),
    # One layer: 21 history frames, 3-frame query chunk, k_h = 4.
    "c2": Workload("c2_single_layer_bf16", batch=1, heads=12, head_dim=128,
                   n_q=4680, page_size=1560, n_cand=21, n_cur=3,
                   k_h=(4,) * 12, dtype="bf16", seed=1),
    # Long history (187,200 history keys), head-adaptive budgets.
    "c3": Workload("c3_long_history_bf16", batch=1, heads=12, head_dim=128,
                   n_q=4680, page_size=1560, n_cand=120, n_cur=3, k_h=None,
                   k_h_choices=(2, 4, 8, 16), dtype="bf16", seed=2),
    # Prompt switch: clustered pages, the query chunk matches a cluster last
    # seen 100 pages back.
    "c4": Workload("c4_prompt_switch_bf16", batch=1, heads=12, head_dim=128,
                   n_q=4680, page_size=1560, n_cand=240, n_cur=3, k_h=None,
                   k_h_choices=(4, 8), dtype="bf16", seed=3,
                   structure="clusters"),
    # Streaming: 30 independent layers, 60 chunks of 3 pages each; the
    # history before chunk t (1-based) is 3(t-1) pages.
    "c5": Workload("c5_streaming_30layer_bf16", batch=1, heads=12,
                   head_dim=128, n_q=4680, page_size=1560, n_cand=177,
                   n_cur=3, k_h=(8,) * 12, dtype="bf16", seed=4, layers=30,
                   chunks=60),
}


def get_workload(name: str) -> Workload:
    if name in WORKLOADS:
        return WORKLOADS[name]
    for w in WORKLOADS.values():
        if w.name == name:
            return w
    raise KeyError(name)


def streaming_chunk(wl: Workload, t: int) -> Workload:
    """Shape of streaming chunk t (1-based): 3(t-1) history pages."""
    return wl.replace(n_cand=wl.n_cur * (t - 1), layers=1, chunks=1)
