"""Pins of the block-sparse (head-adaptive) oracle against things other than
itself: closed forms of the Gini coefficient, brute-force minimal subsets,
the full-coverage limit (dense attention), partitions and invariances."""
import itertools

import numpy as np
import pytest
import torch

from oracle import hsa_blocks_oracle as BO
from oracle import hsa_oracle as O


def test_page_blocks_partition_each_page():
    for P, B in [(1560, 128), (1560, 64), (256, 64), (200, 128), (8, 64), (64, 64)]:
        b = BO.page_blocks(P, B)
        assert b[0][0] == 0 and b[-1][1] == P
        assert all(e1 == s2 for (_, e1), (s2, _) in zip(b, b[1:]))        # contiguous
        assert all(s % B == 0 and 0 < e - s <= B for s, e in b)            # aligned, short last
        assert len(b) == -(-P // B)


def test_list_blocks_history_then_current():
    bl = BO.list_blocks(2, 1, 1560)
    assert len(bl) == 2 * 13 + 25
    assert bl[0] == (0, 0, 128) and bl[12] == (0, 1536, 1560) and bl[26] == (2, 0, 64)


@pytest.mark.parametrize("n", [1, 2, 7, 64, 283])
def test_gini_closed_forms(n):
    rng = np.random.default_rng(n)
    uniform = np.full((3, n), 1.0 / n)
    assert abs(BO.gini(uniform)) < 1e-14                               # uniform -> 0
    onehot = np.zeros((3, n))
    onehot[np.arange(3), rng.integers(0, n, 3)] = 1.0
    assert abs(BO.gini(onehot) - (n - 1) / n) < 1e-14                  # one-hot -> (N-1)/N
    for k in {1, max(1, n // 3), n}:
        # mass spread evenly over k blocks (any positions): G = (N - k) / N
        pm = np.zeros((2, n))
        for r in range(2):
            pm[r, rng.permutation(n)[:k]] = 1.0 / k
        assert abs(BO.gini(pm) - (n - k) / n) < 1e-13


def test_gini_is_the_mean_over_query_blocks():
    n = 9
    a = np.full(n, 1.0 / n)
    b = np.zeros(n)
    b[4] = 1.0
    assert abs(BO.gini(np.stack([a, b])) - 0.5 * (n - 1) / n) < 1e-14


def test_coverage_threshold_endpoints_from_data():
    n = 12
    assert BO.coverage_threshold(BO.gini(np.full((2, n), 1.0 / n))) == pytest.approx(BO.TAU_MIN, abs=1e-14)
    oh = np.eye(n)[:3]
    g = BO.gini(oh)
    assert BO.coverage_threshold(g, 0.35, 1.0) == pytest.approx(0.35 + 0.65 * (n - 1) / n, abs=1e-14)


@pytest.mark.parametrize("seed", range(6))
def test_select_blocks_is_the_minimal_heaviest_subset(seed):
    # brute force over all subsets of a small row: the kept set has the
    # smallest size whose mass can reach tau, and the largest mass among
    # subsets of that size
    rng = np.random.default_rng(seed)
    n = 8
    p = rng.dirichlet(np.full(n, 0.5))
    for tau in [0.05, 0.35, 0.6, 0.9, 0.999]:
        kept = BO.select_blocks(p, tau)
        best_k = next(k for k in range(1, n + 1)
                      if max(sum(p[list(c)]) for c in itertools.combinations(range(n), k)) >= tau)
        assert len(kept) == best_k
        best_mass = max(sum(p[list(c)]) for c in itertools.combinations(range(n), best_k))
        assert abs(p[kept].sum() - best_mass) < 1e-12


def test_select_blocks_ties_keep_lower_index_and_thresholds_nest():
    p = np.array([0.2, 0.1, 0.2, 0.3, 0.1, 0.1])
    assert list(BO.select_blocks(p, 0.45)) == [3, 0]
    assert list(BO.select_blocks(p, 0.65)) == [3, 0, 2]
    assert list(BO.select_blocks(p, 0.75)) == [3, 0, 2, 1]
    prev = []
    for tau in np.linspace(0.01, 1.0, 25):
        cur = list(BO.select_blocks(p, tau))
        assert cur[:len(prev)] == prev        # a larger threshold extends the prefix
        prev = cur


def test_select_blocks_full_coverage_keeps_everything():
    p = np.full(7, 1.0 / 7)          # sums to slightly less or more than 1 in fp64
    assert len(BO.select_blocks(p, 1.0)) == 7


def test_pooled_map_rows_are_distributions_matching_torch():
    rng = np.random.default_rng(3)
    qb, kb = rng.standard_normal((5, 16)), rng.standard_normal((11, 16))
    pm = BO.pooled_map(qb, kb, 0.25)
    ref = torch.softmax(torch.from_numpy(qb) @ torch.from_numpy(kb).T * 0.25, dim=1).numpy()
    np.testing.assert_allclose(pm, ref, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(pm.sum(1), 1.0, rtol=1e-14)


def _head(seed, n_q=150, P=200, n_hist=2, n_cur=1, d=16):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((n_q, d))
    ks = [rng.standard_normal((P, d)) for _ in range(n_hist + n_cur)]
    vs = [rng.standard_normal((P, d)) for _ in range(n_hist + n_cur)]
    return q, ks, vs


def test_full_coverage_equals_dense_attention_over_the_list():
    # tau = 1 keeps every block: the block-sparse branch is exact attention
    # over all keys of the listed pages (torch SDPA as the reference)
    q, ks, vs = _head(5)
    r = BO.adaptive_head(q, ks, vs, n_hist=2, scale=0.25, tau_min=1.0, tau_max=1.0, b_hist=128, b_cur=64)
    assert all(len(k) == len(r["blocks"]) for k in r["kept"])
    K, V = np.concatenate(ks), np.concatenate(vs)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None], torch.from_numpy(K)[None], torch.from_numpy(V)[None], scale=0.25)[0].numpy()
    np.testing.assert_allclose(r["O_sp"], ref, rtol=1e-10, atol=1e-12)


def test_block_sparse_branch_equals_masked_dense_attention():
    # each query block attends exactly to the tokens of its kept blocks:
    # dense attention with an explicit -inf mask elsewhere
    q, ks, vs = _head(7)
    r = BO.adaptive_head(q, ks, vs, n_hist=2, scale=0.3, tau_min=0.3, tau_max=0.6, b_hist=128, b_cur=64)
    K, V = np.concatenate(ks), np.concatenate(vs)
    P = ks[0].shape[0]
    s = q @ K.T * 0.3
    mask = np.full(s.shape, -np.inf)
    for i, (qs, qe) in enumerate(BO.page_blocks(q.shape[0], BO.BLOCK_Q)):
        for j in r["kept"][i]:
            li, a, b = r["blocks"][j]
            mask[qs:qe, li * P + a: li * P + b] = 0.0
    a_ = np.exp(s + mask - (s + mask).max(1, keepdims=True))
    ref = (a_ @ V) / a_.sum(1, keepdims=True)
    np.testing.assert_allclose(r["O_sp"], ref, rtol=1e-10, atol=1e-12)
    assert 0 < np.mean([len(k) for k in r["kept"]]) < len(r["blocks"])


def test_planted_block_is_kept_first():
    q, ks, vs = _head(9)
    qm = q[:64].mean(0)
    ks[0][128:200] = qm * 40.0             # block 1 of page 0 aligned with query block 0
    r = BO.adaptive_head(q, ks, vs, n_hist=2, scale=0.25)
    assert r["kept"][0][0] == 1


def test_gini_of_peaked_maps_raises_the_threshold():
    q, ks, vs = _head(11)
    flat = BO.adaptive_head(q * 0.0, ks, vs, n_hist=2, scale=0.25)
    q2 = q.copy()
    for i in range(0, q.shape[0], 64):
        q2[i:i + 64] += ks[0][0:128].mean(0) * 800.0   # block 0 dominates every row
    peaked = BO.adaptive_head(q2, ks, vs, n_hist=2, scale=0.25)
    n = len(peaked["blocks"])
    assert flat["gini"] < 1e-12 and flat["tau"] == pytest.approx(BO.TAU_MIN)
    assert peaked["gini"] > 0.9 * (n - 1) / n and peaked["tau"] > 0.9
    assert all(list(k) == [0] for k in peaked["kept"][:2])


def test_forward_adaptive_full_coverage_matches_hsa_forward():
    # with tau = 1 every query block keeps every block, so the whole pass is
    # the page-level HSA forward of the base oracle
    rng = np.random.default_rng(2)
    B, n_q, H, d, P, n_cand, n_cur = 1, 130, 2, 16, 72, 4, 1
    npg = n_cand + n_cur
    q = rng.standard_normal((B, n_q, H, d))
    kp = rng.standard_normal((npg, H, P, d))
    vp = rng.standard_normal((npg, H, d, P))
    pt = rng.permutation(npg).reshape(B, npg).astype(np.int32)
    a = BO.hsa_forward_adaptive(q, kp, vp, pt, n_cand, n_cur, [2, 3], tau_min=1.0, tau_max=1.0)
    b = O.hsa_forward(q, kp, vp, pt, n_cand, n_cur, [2, 3])
    np.testing.assert_array_equal(a["sel"], b["sel"])
    np.testing.assert_allclose(a["O"], b["O"], rtol=1e-10, atol=1e-12)


def test_equal_key_blocks_get_equal_weights_and_tie_to_lower_id():
    rng = np.random.default_rng(21)
    qb = rng.standard_normal((3, 32))
    kb = rng.standard_normal((40, 32))
    kb[[5, 17, 33]] = kb[29]
    pm = BO.pooled_map(qb, kb, 0.2)
    assert (pm[:, 5] == pm[:, 29]).all() and (pm[:, 17] == pm[:, 33]).all()
    for row in pm:
        order = list(BO.block_order(row))
        pos = [order.index(j) for j in (5, 17, 29, 33)]
        assert pos == sorted(pos) and pos[-1] - pos[0] == 3


def test_threshold_one_keeps_every_block_even_if_the_sum_rounds_early():
    # weights whose running sum reaches 1.0 in fp64 before the last block
    p = np.array([0.5, 0.5 - 2.0 ** -54, 2.0 ** -54, 1e-300])
    assert np.cumsum(p)[1] == 1.0 or np.cumsum(p)[2] == 1.0
    assert len(BO.select_blocks(p, 1.0)) == 4
    assert len(BO.select_blocks(p, 0.75)) == 2


def test_block_means_equal_reshaped_page_means():
    # on a page that the block size divides, the block means are the means of
    # the page reshaped into [P / B, B, d]
    rng = np.random.default_rng(7)
    for P, B in [(1536, 128), (1536, 64), (256, 64)]:
        x = rng.standard_normal((P, 16))
        got = BO.block_means(x, BO.page_blocks(P, B))
        np.testing.assert_allclose(got, x.reshape(-1, B, 16).mean(1), rtol=0, atol=1e-15)


def _blocky_head(rng, n_hist, n_cur, P, d, n_q, b_hist=BO.BLOCK_HIST, b_cur=BO.BLOCK_CUR):
    """Keys constant inside every key block (a distinct random vector per
    block, page by page in list order) and queries constant inside every
    query block."""
    k_list, v_list = [], []
    for li in range(n_hist + n_cur):
        B = b_hist if li < n_hist else b_cur
        k = np.zeros((P, d))
        for s, e in BO.page_blocks(P, B):
            k[s:e] = rng.standard_normal(d) * 1.5
        k_list.append(k)
        v_list.append(rng.standard_normal((P, d)))
    q = np.zeros((n_q, d))
    for s, e in BO.page_blocks(n_q, BO.BLOCK_Q):
        q[s:e] = rng.standard_normal(d) * 1.5
    return q, k_list, v_list


def _token_mass(q, k_list, scale, blocks):
    """Softmax over every token of the list (torch, fp64) for each query, the
    mass it puts on each key block: [n_q, n_blocks]."""
    keys = torch.from_numpy(np.concatenate(k_list, 0))
    p = torch.softmax(torch.from_numpy(q) @ keys.T * scale, dim=-1)
    off = np.cumsum([0] + [k.shape[0] for k in k_list])
    cols = [p[:, off[li] + s: off[li] + e].sum(-1) for li, s, e in blocks]
    return torch.stack(cols, -1).numpy()


@pytest.mark.parametrize("seed", range(3))
def test_pooled_map_equals_token_softmax_mass_on_blocky_inputs(seed):
    # With keys constant inside equal-size key blocks and queries constant
    # inside each query block, the softmax of a query over all tokens puts on
    # block j exactly the weight that the pooled (block-level) map gives it:
    # each token of block j has score s q.k_j, so the block's mass is
    # B exp(s q.k_j) / sum_j' B exp(s q.k_j'). This fixes the pooling to the
    # mean (sum pooling scales every score by B), the scale, and which page
    # and rows each block id stands for.
    rng = np.random.default_rng(100 + seed)
    d, n_q, P = 32, 200, 384            # history blocks of 128 divide the page
    q, k_list, v_list = _blocky_head(rng, 3, 0, P, d, n_q)
    scale = 1.0 / np.sqrt(d)
    r = BO.adaptive_head(q, k_list, v_list, 3, scale, query_blocks=[])
    mass = _token_mass(q, k_list, scale, r["blocks"])
    for i, (s, e) in enumerate(BO.page_blocks(n_q, BO.BLOCK_Q)):
        np.testing.assert_allclose(mass[s:e], np.broadcast_to(r["pooled"][i], mass[s:e].shape),
                                   rtol=1e-12, atol=1e-15)


def test_pooled_map_against_token_mass_with_unequal_block_sizes():
    # History blocks hold 128 tokens and current-chunk blocks 64, so the
    # token-level mass of block j is proportional to n_j exp(s q.k_j) while
    # the pooled weight is proportional to exp(s q.k_j): dividing the mass by
    # the block size and renormalising gives the pooled map.
    rng = np.random.default_rng(9)
    d, n_q, P = 32, 130, 256
    q, k_list, v_list = _blocky_head(rng, 2, 2, P, d, n_q)
    scale = 0.2
    r = BO.adaptive_head(q, k_list, v_list, 2, scale, query_blocks=[])
    mass = _token_mass(q, k_list, scale, r["blocks"])
    sizes = np.array([e - s for _, s, e in r["blocks"]], np.float64)
    assert set(sizes.tolist()) == {64.0, 128.0}
    per = mass / sizes
    per /= per.sum(-1, keepdims=True)
    for i, (s, e) in enumerate(BO.page_blocks(n_q, BO.BLOCK_Q)):
        np.testing.assert_allclose(per[s:e], np.broadcast_to(r["pooled"][i], per[s:e].shape),
                                   rtol=1e-12, atol=1e-15)
