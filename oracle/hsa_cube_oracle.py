"""fp64-free reference of the cube token order of a page (TEST INFRASTRUCTURE).

This module is the checker, not the product. Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use
it. It shares no code with the HIP library.

Paper passages followed (WorldAttention, arxiv 2609.34606):
  * App. "Block Sparse Attention": a (T, H, W) latent is cut into
    (C_t, C_h, C_w) cubes of B = C_t C_h C_w tokens, and a token at (t, h, w)
    is given the flattened index
        n = (floor(t/C_t) N_h N_w + floor(h/C_h) N_w + floor(w/C_w)) B
            + (t mod C_t) C_h C_w + (h mod C_h) C_w + (w mod C_w)
    with (N_t, N_h, N_w) the cube counts, so that every run of B consecutive
    tokens is one cube;
  * Sec. 3.3 "Inter- and intra-chunk sparse granularity": (4, 8, 4), B = 128,
    for retrieved history and (4, 4, 4), B = 64, for the current chunk.

Reading (listed in the design notes): the paper assumes the cube divides the
latent; a 480p frame is 30 x 52 tokens and a chunk 3 frames, so it does not.
The tokens of whole cubes take the positions the formula gives them with
(N_t, N_h, N_w) the counts of whole cubes; the remaining tokens (those of the
cubes truncated along the far edges) follow, ordered by the cube they fall in
(cube index along t, then h, then w) and inside it by (t, h, w).

Pinning: ``tests/test_oracle_cube_pins.py``.
"""
from __future__ import annotations

import numpy as np


def cube_positions(T: int, H: int, W: int, ct: int, ch: int, cw: int):
    """(pos, whole): pos[raster index] = stored position of that token, and
    the number of positions taken by whole cubes."""
    t, h, w = np.meshgrid(np.arange(T), np.arange(H), np.arange(W), indexing="ij")
    t, h, w = t.ravel(), h.ravel(), w.ravel()
    Nt, Nh, Nw = T // ct, H // ch, W // cw
    B = ct * ch * cw
    inside = (t < Nt * ct) & (h < Nh * ch) & (w < Nw * cw)
    pos = np.empty(T * H * W, np.int64)
    # the paper's index for tokens of whole cubes
    pos[inside] = ((t[inside] // ct) * Nh * Nw + (h[inside] // ch) * Nw + (w[inside] // cw)) * B \
        + (t[inside] % ct) * ch * cw + (h[inside] % ch) * cw + (w[inside] % cw)
    whole = Nt * Nh * Nw * B
    # the rest: by cube, then (t, h, w), after the whole cubes
    rest = np.nonzero(~inside)[0]
    key = np.lexsort((w[rest], h[rest], t[rest], w[rest] // cw, h[rest] // ch, t[rest] // ct))
    pos[rest[key]] = whole + np.arange(rest.size)
    return pos, whole


def cube_order(T: int, H: int, W: int, ct: int, ch: int, cw: int):
    """(src_of, whole): src_of[i] = raster index (t H + h) W + w of the token
    stored at position i."""
    pos, whole = cube_positions(T, H, W, ct, ch, cw)
    src_of = np.empty_like(pos)
    src_of[pos] = np.arange(pos.size)
    return src_of, whole


def permute_page(x_raster: np.ndarray, src_of: np.ndarray) -> np.ndarray:
    """A page's tokens [P, ...] from raster order to stored order."""
    return np.asarray(x_raster)[np.asarray(src_of)]
