"""Pins of the Linformer linear-branch oracle against things other than
itself: projections that make the compressed context equal to (a subset
of) the page tokens reduce the branch to dense attention computed by torch;
mean pooling over groups of equal tokens is exact; order invariance; the
gated forward in the limits where both branches see the same keys."""
import numpy as np
import pytest
import torch
from scipy.special import expit

from oracle import hsa_linformer_oracle as LO

F = torch.nn.functional


def _pages(seed, n_pages=3, P=48, d=16):
    rng = np.random.default_rng(seed)
    ks = [rng.standard_normal((P, d)) for _ in range(n_pages)]
    vs = [rng.standard_normal((P, d)) for _ in range(n_pages)]
    q = rng.standard_normal((40, d))
    return q, ks, vs


def _sdpa(q, k, v, scale):
    return F.scaled_dot_product_attention(torch.from_numpy(q)[None], torch.from_numpy(k)[None],
                                          torch.from_numpy(v)[None], scale=scale)[0].numpy()


def test_identity_projection_is_dense_attention():
    q, ks, vs = _pages(1)
    e = np.eye(ks[0].shape[0])                       # r = P, E = I
    ck = [LO.compress(e, k) for k in ks]
    cv = [LO.compress(e, v) for v in vs]
    o, lse = LO.linformer_branch(q, ck, cv, 0.3)
    ref = _sdpa(q, np.concatenate(ks), np.concatenate(vs), 0.3)
    np.testing.assert_allclose(o, ref, rtol=1e-10, atol=1e-12)
    s = q @ np.concatenate(ks).T * 0.3
    np.testing.assert_allclose(lse, np.log(np.exp(s).sum(1)), rtol=1e-12)


@pytest.mark.parametrize("g", [2, 4, 8])
def test_mean_pooling_over_equal_tokens_is_exact(g):
    # every run of g tokens of a page repeats one key and one value: full
    # attention weights each distinct token g times, which cancels; the
    # mean-pooling projection recovers exactly the distinct tokens
    rng = np.random.default_rng(g)
    P, d, n_pages = 48, 16, 3
    r = P // g
    ks = [np.repeat(rng.standard_normal((r, d)), g, axis=0) for _ in range(n_pages)]
    vs = [np.repeat(rng.standard_normal((r, d)), g, axis=0) for _ in range(n_pages)]
    q = rng.standard_normal((33, d))
    e = np.zeros((r, P))
    for j in range(r):
        e[j, j * g:(j + 1) * g] = 1.0 / g
    o, _ = LO.linformer_branch(q, [LO.compress(e, k) for k in ks], [LO.compress(e, v) for v in vs],
                               0.25)
    ref = _sdpa(q, np.concatenate(ks), np.concatenate(vs), 0.25)
    np.testing.assert_allclose(o, ref, rtol=1e-10, atol=1e-12)


def test_token_selecting_projection_attends_to_the_selected_tokens():
    q, ks, vs = _pages(3)
    P = ks[0].shape[0]
    pick = np.array([0, 5, 17, 31, 47])
    e = np.zeros((len(pick), P))
    e[np.arange(len(pick)), pick] = 1.0
    o, _ = LO.linformer_branch(q, [LO.compress(e, k) for k in ks], [LO.compress(e, v) for v in vs],
                               0.2)
    ref = _sdpa(q, np.concatenate([k[pick] for k in ks]), np.concatenate([v[pick] for v in vs]), 0.2)
    np.testing.assert_allclose(o, ref, rtol=1e-10, atol=1e-12)


def test_compressed_page_order_does_not_matter_and_compression_is_per_page():
    q, ks, vs = _pages(4, n_pages=4)
    rng = np.random.default_rng(9)
    e = rng.standard_normal((8, ks[0].shape[0])) / np.sqrt(ks[0].shape[0])
    ck = [LO.compress(e, k) for k in ks]
    cv = [LO.compress(e, v) for v in vs]
    a, la = LO.linformer_branch(q, ck, cv, 0.25)
    perm = [2, 0, 3, 1]
    b, lb = LO.linformer_branch(q, [ck[i] for i in perm], [cv[i] for i in perm], 0.25)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(la, lb, rtol=1e-14)
    # a page's compression depends on that page only: the projection of the
    # concatenation of two pages with a block-diagonal E is the pair
    both = LO.compress(np.block([[e, np.zeros_like(e)], [np.zeros_like(e), e]]),
                       np.concatenate(ks[:2]))
    np.testing.assert_allclose(both, np.concatenate(ck[:2]), rtol=1e-12, atol=1e-14)


def test_forward_merges_gates_and_reduces_to_twice_dense_attention():
    # tau = 1 keeps every block and E = I keeps every token: both branches
    # are dense attention over the same pages, so O = (s(g_lin) + s(g_sp)) O_sp
    rng = np.random.default_rng(5)
    B, n_q, H, d, P, n_cand, n_cur = 1, 70, 2, 16, 24, 3, 1
    npg = n_cand + n_cur
    q = rng.standard_normal((B, n_q, H, d))
    kp = rng.standard_normal((npg, H, P, d))
    vp = rng.standard_normal((npg, H, d, P))
    pt = rng.permutation(npg).reshape(B, npg).astype(np.int32)
    e = np.stack([np.eye(P)] * H)
    gl = rng.standard_normal((B, n_q, H))
    gs = rng.standard_normal((B, n_q, H))
    r = LO.hsa_forward_linformer(q, kp, vp, pt, e, e, n_cand, n_cur, [2, 3], 1.0, 1.0, gl, gs)
    np.testing.assert_allclose(r["O_lin"], r["O_sp"], rtol=1e-10, atol=1e-12)
    w = (expit(gl) + expit(gs))[..., None]
    np.testing.assert_allclose(r["O"], w * r["O_sp"], rtol=1e-10, atol=1e-12)
