"""Pins of the fp64 oracle against things other than itself.

Each test ties one oracle function to a library routine, a brute-force
enumeration, an alternative formula, a closed form or an invariant, so that a
dropped term, a wrong sign or index, or a transposed operand fails one of them.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import hsa_oracle as O
from synth_inputs import make_case
from synth_inputs.configs import Workload

HERE = os.path.dirname(os.path.abspath(__file__))
rng0 = np.random.default_rng(1234)


def small_wl(**kw):
    base = dict(name="pin", batch=1, heads=3, head_dim=16, n_q=24, page_size=8,
                n_cand=6, n_cur=2, k_h=(2, 3, 6), dtype="f32", seed=7)
    base.update(kw)
    return Workload(**base)


def run(case, **kw):
    wl = case.wl
    return O.hsa_forward(case.q, case.k_pool, case.v_pool, case.page_table,
                         wl.n_cand, wl.n_cur, list(case.k_h), case.g_lin,
                         case.g_sp, **kw)


# ---------------------------------------------------------------- feature map
def test_phi_is_elu_plus_one():
    x = rng0.standard_normal(10000) * 5
    ref = torch.nn.functional.elu(torch.from_numpy(x), alpha=1.0).numpy() + 1.0
    np.testing.assert_allclose(O.phi(x), ref, rtol=1e-15, atol=1e-15)
    assert (O.phi(x) > 0).all()


def test_phi_mean_closed_form():
    # For x ~ N(0,1): E[elu(x)+1] = 1/2 + 1/sqrt(2 pi) + e^{1/2} Phi(-1).
    from scipy.stats import norm
    expect = 0.5 + 1 / math.sqrt(2 * math.pi) + math.exp(0.5) * norm.cdf(-1.0)
    x = np.random.default_rng(5).standard_normal((400000, 4))
    _, z = O.linear_state(x, np.ones_like(x))
    assert abs(z.mean() / x.shape[0] - expect) < 3e-3
    assert abs(expect - 1.16052) < 1e-4


# ---------------------------------------------------------------- linear branch
def test_linear_branch_matches_quadratic_form():
    # O_lin[i] = sum_j (phi(q_i).phi(k_j)) v_j / sum_j phi(q_i).phi(k_j),
    # written as explicit loops over (i, j): the attention-matrix form.
    r = np.random.default_rng(11)
    q, k, v = r.standard_normal((5, 4)), r.standard_normal((7, 4)), r.standard_normal((7, 3))
    S, z = O.linear_state(k, v)
    got = O.linear_branch(q, S, z)
    for i in range(5):
        num = np.zeros(3)
        den = 0.0
        for j in range(7):
            w = 0.0
            for c in range(4):
                a = q[i, c] + 1 if q[i, c] > 0 else math.exp(q[i, c])
                b = k[j, c] + 1 if k[j, c] > 0 else math.exp(k[j, c])
                w += a * b
            num += w * v[j]
            den += w
        np.testing.assert_allclose(got[i], num / den, rtol=1e-13)


def test_linear_state_is_additive_over_pages():
    r = np.random.default_rng(12)
    k, v = r.standard_normal((30, 4)), r.standard_normal((30, 4))
    S, z = O.linear_state(k, v)
    S1, z1 = O.linear_state(k[:11], v[:11])
    S2, z2 = O.linear_state(k[11:], v[11:])
    np.testing.assert_allclose(S, S1 + S2, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(z, z1 + z2, rtol=1e-13)


# ---------------------------------------------------------------- sparse branch
def test_sparse_branch_matches_torch_sdpa():
    r = np.random.default_rng(13)
    q, k, v = r.standard_normal((9, 16)), r.standard_normal((21, 16)), r.standard_normal((21, 16))
    got, lse = O.sparse_branch(q, k, v, 1 / math.sqrt(16))
    t = lambda a: torch.from_numpy(a)[None, None]
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v))[0, 0].numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)
    ref_lse = torch.logsumexp(t(q) @ t(k).transpose(-1, -2) / 4.0, -1)[0, 0].numpy()
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-13)


def test_sparse_branch_matches_explicit_loops():
    r = np.random.default_rng(14)
    q, k, v = r.standard_normal((3, 4)), r.standard_normal((5, 4)), r.standard_normal((5, 2))
    got, _ = O.sparse_branch(q, k, v, 0.5)
    for i in range(3):
        w = [math.exp(0.5 * sum(q[i, c] * k[j, c] for c in range(4))) for j in range(5)]
        ref = [sum(w[j] * v[j, e] for j in range(5)) / sum(w) for e in range(2)]
        np.testing.assert_allclose(got[i], ref, rtol=1e-13)


# ---------------------------------------------------------------- scores
def test_page_score_is_mean_pairwise_scaled_dot():
    # qbar.kbar/sqrt(d) equals the average of q_i.k_t/sqrt(d) over all pairs.
    r = np.random.default_rng(15)
    q, k = r.standard_normal((6, 8)), r.standard_normal((10, 8))
    a = O.page_scores(O.query_mean(q), O.page_key_mean(k)[None])[0]
    pair = np.mean([[float(q[i] @ k[t]) for t in range(10)] for i in range(6)]) / math.sqrt(8)
    assert abs(a - pair) < 1e-13


# ---------------------------------------------------------------- selection
def _brute_topk(alpha, k):
    """Among k-subsets of maximal score sum, the lexicographically smallest."""
    n = len(alpha)
    best, best_sum = None, None
    for T in itertools.combinations(range(n), k):
        s = sum(alpha[t] for t in T)
        if best is None or s > best_sum or (s == best_sum and T < best):
            best, best_sum = T, s
    return best


@pytest.mark.parametrize("n", [1, 4, 7, 9])
def test_selection_matches_subset_enumeration(n):
    r = np.random.default_rng(100 + n)
    for trial in range(20):
        # small integers: plenty of exact ties, sums are exact in fp64
        alpha = r.integers(-3, 4, n).astype(np.float64)
        for k in range(0, n + 2):
            sel = O.select_top_pages(alpha, k)
            ref = _brute_topk(alpha, min(k, n))
            assert tuple(sorted(sel.tolist())) == ref
            # rank order: score descending, then index ascending
            keys = [(-alpha[p], p) for p in sel]
            assert keys == sorted(keys)


def test_duplicate_page_tie_keeps_lower_index():
    wl = small_wl(heads=1, k_h=(1,), n_cand=5, n_cur=1)
    case = make_case(wl)
    # make logical pages 1 and 3 identical and strongly aligned with the queries
    qdir = case.q[0, :, 0, :].mean(0)
    for p in (1, 3):
        case.k_pool[case.page_table[0, p], 0] = np.tile(qdir * 3, (wl.page_size, 1))
    out = run(case)
    assert out["alpha"][0, 0, 1] == out["alpha"][0, 0, 3]
    assert out["sel"][0, 0, 0] == 1


# ---------------------------------------------------------------- merge
def test_sigmoid_and_gate_limits():
    from scipy.special import expit
    g = rng0.standard_normal(50) * 10
    np.testing.assert_allclose(O.sigmoid(g), expit(g), rtol=1e-14)
    a, b = rng0.standard_normal((4, 3, 5)), rng0.standard_normal((4, 3, 5))
    one = np.full((4, 3), 40.0)
    np.testing.assert_allclose(O.gated_merge(a, b, one, -one), a, atol=1e-15)
    np.testing.assert_allclose(O.gated_merge(a, b, -one, one), b, atol=1e-15)
    np.testing.assert_allclose(O.gated_merge(a, b), 0.5 * (a + b), rtol=1e-15)


def test_elementwise_gate_limits_pick_a_branch_per_element():
    # element-wise gates (the outputs' shape): a per-element choice of branch
    # in the saturated limit, and a gate constant over the last axis equals
    # the per-(query, head) gate
    a, b = rng0.standard_normal((4, 3, 5)), rng0.standard_normal((4, 3, 5))
    mask = rng0.random((4, 3, 5)) < 0.5
    g = np.where(mask, 40.0, -40.0)
    np.testing.assert_allclose(O.gated_merge(a, b, g, -g), np.where(mask, a, b), atol=1e-15)
    gh = rng0.standard_normal((4, 3))
    ge = np.repeat(gh[..., None], 5, axis=-1)
    np.testing.assert_array_equal(O.gated_merge(a, b, ge, -ge), O.gated_merge(a, b, gh, -gh))


def test_forward_with_elementwise_gates_picks_branches_per_element():
    wl = small_wl(gates=True)
    case = make_case(wl)
    d = wl.head_dim
    mask = np.random.default_rng(5).random(case.g_lin.shape + (d,)) < 0.5
    g = np.where(mask, 40.0, -40.0).astype(np.float32)
    out = O.hsa_forward(case.q, case.k_pool, case.v_pool, case.page_table, wl.n_cand, wl.n_cur,
                        list(case.k_h), g, -g)
    np.testing.assert_allclose(out["O"], np.where(mask, out["O_lin"], out["O_sp"]), atol=1e-14)
    # constant over d: the head-wise result
    ge = np.repeat(case.g_lin[..., None], d, axis=-1)
    se = np.repeat(case.g_sp[..., None], d, axis=-1)
    e = O.hsa_forward(case.q, case.k_pool, case.v_pool, case.page_table, wl.n_cand, wl.n_cur,
                      list(case.k_h), ge, se)
    h = O.hsa_forward(case.q, case.k_pool, case.v_pool, case.page_table, wl.n_cand, wl.n_cur,
                      list(case.k_h), case.g_lin, case.g_sp)
    np.testing.assert_array_equal(e["O"], h["O"])


# ---------------------------------------------------------------- whole pass
def test_full_budget_equals_dense_attention_over_all_pages():
    wl = small_wl(k_h=(6, 9, 100))
    case = make_case(wl)
    out = run(case)
    d = wl.head_dim
    for h in range(wl.heads):
        k, v = O.gather_pages(case.k_pool, case.v_pool, case.page_table, 0, h,
                              range(wl.n_pages))
        t = lambda a: torch.from_numpy(np.asarray(a, np.float64))[None, None]
        ref = torch.nn.functional.scaled_dot_product_attention(
            t(case.q[0, :, h]), t(k), t(v))[0, 0].numpy()
        np.testing.assert_allclose(out["O_sp"][0, :, h], ref, rtol=1e-11, atol=1e-12)
        assert sorted(out["sel"][0, h][out["sel"][0, h] >= 0].tolist()) == list(range(wl.n_cand))
        # the linear state covers every page
        S, z = O.linear_state(k, v)
        np.testing.assert_allclose(out["S"][0, h], S, rtol=1e-12)
    assert d == 16


def test_slot_permutation_invariance_is_exact():
    wl = small_wl()
    case = make_case(wl)
    a = run(case)
    perm = np.random.default_rng(3).permutation(case.num_slots)
    inv = np.argsort(perm)
    k2, v2 = case.k_pool[perm], case.v_pool[perm]
    pt2 = inv[case.page_table].astype(np.int32)
    b = O.hsa_forward(case.q, k2, v2, pt2, wl.n_cand, wl.n_cur, list(case.k_h))
    for key in ("O", "sel", "alpha", "S"):
        np.testing.assert_array_equal(a[key], b[key])


def test_key_permutation_within_page_invariance():
    wl = small_wl()
    case = make_case(wl)
    a = run(case)
    perm = np.random.default_rng(4).permutation(wl.page_size)
    k2 = case.k_pool[:, :, perm, :]
    v2 = case.v_pool[:, :, :, perm]
    b = O.hsa_forward(case.q, k2, v2, case.page_table, wl.n_cand, wl.n_cur, list(case.k_h))
    np.testing.assert_array_equal(a["sel"], b["sel"])
    np.testing.assert_allclose(a["O"], b["O"], rtol=1e-12, atol=1e-13)


def test_logical_page_relabelling():
    wl = small_wl()
    case = make_case(wl)
    a = run(case)
    perm = np.random.default_rng(5).permutation(wl.n_cand)   # new logical p <- old perm[p]
    pt2 = case.page_table.copy()
    pt2[0, :wl.n_cand] = case.page_table[0, perm]
    b = O.hsa_forward(case.q, case.k_pool, case.v_pool, pt2, wl.n_cand, wl.n_cur, list(case.k_h))
    inv = np.argsort(perm)
    for h in range(wl.heads):
        sa = a["sel"][0, h][a["sel"][0, h] >= 0]
        sb = b["sel"][0, h][b["sel"][0, h] >= 0]
        np.testing.assert_array_equal(inv[sa], sb)
    np.testing.assert_allclose(a["O"], b["O"], rtol=1e-12, atol=1e-13)


def test_query_permutation_equivariance():
    wl = small_wl()
    case = make_case(wl)
    a = run(case)
    perm = np.random.default_rng(6).permutation(wl.n_q)
    b = O.hsa_forward(case.q[:, perm], case.k_pool, case.v_pool, case.page_table,
                      wl.n_cand, wl.n_cur, list(case.k_h))
    np.testing.assert_array_equal(a["sel"], b["sel"])
    np.testing.assert_allclose(a["O"][:, perm], b["O"], rtol=1e-12, atol=1e-13)


def test_zero_budget_attends_current_chunk_only():
    wl = small_wl(k_h=(0, 0, 0))
    case = make_case(wl)
    out = run(case)
    assert (out["sel"] == -1).all()
    for h in range(wl.heads):
        k, v = O.gather_pages(case.k_pool, case.v_pool, case.page_table, 0, h,
                              range(wl.n_cand, wl.n_pages))
        ref, _ = O.sparse_branch(case.q[0, :, h], k, v, 1 / math.sqrt(wl.head_dim))
        np.testing.assert_allclose(out["O_sp"][0, :, h], ref, rtol=1e-13)


def test_constant_values_give_constant_output():
    wl = small_wl(gates=True)
    case = make_case(wl)
    case.v_pool[:] = 0.75
    out = run(case)
    np.testing.assert_allclose(out["O_sp"], 0.75, rtol=1e-13)
    np.testing.assert_allclose(out["O_lin"], 0.75, rtol=1e-13)
    wsum = O.sigmoid(case.g_lin)[..., None] + O.sigmoid(case.g_sp)[..., None]
    np.testing.assert_allclose(out["O"], 0.75 * np.broadcast_to(wsum, out["O"].shape), rtol=1e-13)


def test_linearity_in_values():
    wl = small_wl(gates=True)
    case = make_case(wl)
    a = run(case)
    case.v_pool *= -2.0   # exact in fp32
    b = run(case)
    np.testing.assert_allclose(b["O"], -2.0 * a["O"], rtol=1e-12, atol=1e-14)


def test_no_history():
    wl = small_wl(n_cand=0, k_h=(2, 2, 2))
    case = make_case(wl)
    out = run(case)
    assert (out["sel"] == -1).all()
    assert np.isfinite(out["O"]).all()


def test_planted_cluster_recall():
    # Clustered pages; the query chunk sits near the cluster of the run 100
    # pages back. Every selected page must come from that cluster.
    wl = Workload("c4_small", batch=1, heads=2, head_dim=128, n_q=64, page_size=16,
                  n_cand=240, n_cur=1, k_h=(4, 8), dtype="bf16", seed=3,
                  structure="clusters")
    case = make_case(wl)
    out = run(case, query_rows=[0, 1])
    pc = case.meta["page_cluster"]
    cs = case.meta["c_star"]
    star_pages = set(np.nonzero(pc == cs)[0].tolist())
    assert set(range(140, 150)) <= star_pages
    for h in range(2):
        sel = out["sel"][0, h][out["sel"][0, h] >= 0]
        assert len(sel) == wl.k_h[h]
        assert set(sel.tolist()) <= star_pages


def test_paper_geometry_fixture():
    # Stage-2 retrieval with K_p pages of 8 frames x 1560 tokens: the active
    # history has the size the paper states.
    with open(os.path.join(HERE, "golden", "paper_geometry.json")) as f:
        g = json.load(f)
    P = g["frames_per_page"] * g["tokens_per_frame"]
    wl = Workload("geom", batch=1, heads=1, head_dim=4, n_q=2, page_size=P,
                  n_cand=6, n_cur=0, k_h=(g["k_p"],), dtype="f32", seed=0)
    case = make_case(wl)
    out = run(case)
    sel = out["sel"][0, 0]
    k, _ = O.gather_pages(case.k_pool, case.v_pool, case.page_table, 0, 0, sel[sel >= 0])
    assert k.shape[0] == g["active_tokens"]
