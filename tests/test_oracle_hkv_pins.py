"""Pins of the two-stage retrieval oracle: cosine similarity against its
closed forms and scipy, the top-1 chunk against brute force with ties, and
the restricted forward against the unrestricted one in the cases where they
must agree."""
import numpy as np
import pytest
from scipy.spatial.distance import cosine as scipy_cosine_distance

from oracle import hsa_hkv_oracle as HK
from oracle import hsa_oracle as O


def test_cosine_closed_forms_and_scipy():
    rng = np.random.default_rng(1)
    p = rng.standard_normal(64)
    C = rng.standard_normal((9, 64))
    C[3] = 2.5 * p                    # parallel: 1
    C[4] = -p                         # antiparallel: -1
    C[5] = 0.0                        # zero norm: 0 by the reading
    u = rng.standard_normal(64)
    C[6] = u - (u @ p) / (p @ p) * p  # orthogonal: 0
    sc = HK.cosine_scores(p, C)
    assert sc[3] == pytest.approx(1.0, abs=1e-15) and sc[4] == pytest.approx(-1.0, abs=1e-15)
    assert sc[5] == 0.0 and abs(sc[6]) < 1e-14
    for m in (0, 1, 2, 7, 8):
        assert sc[m] == pytest.approx(1.0 - scipy_cosine_distance(p, C[m]), abs=1e-14)
    # invariant to positive scaling of either side
    np.testing.assert_allclose(HK.cosine_scores(3.0 * p, 0.5 * C), sc, rtol=1e-14, atol=1e-15)


def test_top1_chunk_brute_force_and_ties():
    rng = np.random.default_rng(2)
    for _ in range(20):
        s = rng.integers(-3, 4, 7).astype(float)          # many exact ties
        m = HK.select_chunk(s)
        assert s[m] == s.max() and all(s[j] < s.max() for j in range(m))


def _bank(seed, B=1, H=2, d=16, P=24, pages_per_chunk=(3, 2, 4), n_cur=1, E=32):
    rng = np.random.default_rng(seed)
    n_cand = sum(pages_per_chunk)
    npg = n_cand + n_cur
    q = rng.standard_normal((B, 40, H, d))
    kp = rng.standard_normal((B * npg, H, P, d))
    vp = rng.standard_normal((B * npg, H, d, P))
    pt = rng.permutation(B * npg).reshape(B, npg).astype(np.int32)
    cf = np.concatenate([[0], np.cumsum(pages_per_chunk)])[None].repeat(B, 0)
    ce = rng.standard_normal((B, len(pages_per_chunk), E))
    pe = rng.standard_normal((B, E))
    return q, kp, vp, pt, cf, ce, pe, n_cand


def test_one_chunk_holding_the_history_is_the_plain_forward():
    q, kp, vp, pt, _, ce, pe, n_cand = _bank(3)
    cf = np.array([[0, n_cand]])
    a = HK.hsa_forward_retrieval(q, kp, vp, pt, pe, ce[:, :1], cf, 1, [2, 3])
    b = O.hsa_forward(q, kp, vp, pt, n_cand, 1, [2, 3])
    np.testing.assert_array_equal(a["sel"], b["sel"])
    np.testing.assert_allclose(a["O"], b["O"], rtol=1e-12, atol=1e-14)


def test_selection_stays_inside_the_chosen_chunk():
    q, kp, vp, pt, cf, ce, pe, n_cand = _bank(4)
    ce[0, 1] = 7.0 * pe[0]            # chunk 1 (pages 3, 4) is the prompt's
    r = HK.hsa_forward_retrieval(q, kp, vp, pt, pe, ce, cf, 1, [1, 5])
    assert r["chunk"][0] == 1 and r["chunk_score"][0] == pytest.approx(1.0, abs=1e-14)
    for h, k in enumerate([1, 5]):
        s = r["sel"][0, h]
        s = s[s >= 0]
        assert len(s) == min(k, 2) and set(s.tolist()) <= {3, 4}
    # the same pages as a forward over a bank that holds only that chunk,
    # relabelled: the chunk's pages become the whole history
    pt2 = np.concatenate([pt[:, 3:5], pt[:, n_cand:]], 1)
    b = O.hsa_forward(q, kp, vp, pt2, 2, 1, [1, 5], state_pages=[])
    for h in range(2):
        np.testing.assert_array_equal(r["sel"][0, h][r["sel"][0, h] >= 0] - 3,
                                      b["sel"][0, h][b["sel"][0, h] >= 0])
    np.testing.assert_allclose(r["O_sp"], b["O_sp"], rtol=1e-12, atol=1e-14)


def test_scaled_chunks_tie_exactly():
    rng = np.random.default_rng(5)
    p = rng.standard_normal(100)
    C = rng.standard_normal((4, 100))
    C[1] = 0.5 * p
    C[3] = 4.0 * p
    sc = HK.cosine_scores(p, C)
    assert sc[1] == sc[3] and HK.select_chunk(sc) == 1
