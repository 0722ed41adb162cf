"""GPU parity: the HIP library against the fp64 oracle on the same inputs.

Selections are compared bit-exact (including -1 padding); floating-point
outputs within the tolerances of hsa_testlib (bf16: max-abs 2e-2, rel-L2
5e-3; fp32: max-abs 1e-4, rel-L2 2e-5). Small cases cover every output
element; full-size workloads compare every selection and state entry and a
sample of query rows that includes the first and the ragged last tile.
"""
import numpy as np
import pytest

from synth_inputs import WORKLOADS, make_case
from synth_inputs.configs import Workload

from hsa_testlib import compare, elementwise_gates, run_library, run_oracle, say, upload

pytestmark = pytest.mark.gpu


def _case_dict(case):
    return dict(q=case.q, k_pool=case.k_pool, v_pool=case.v_pool, page_table=case.page_table,
                g_lin=case.g_lin, g_sp=case.g_sp)


def _run_small(wl, k_max=None, sm_scale=0.0, mutate=None):
    say(f"[case] {wl}")
    case = make_case(wl)
    if mutate:
        mutate(case)
    dev = upload(case)
    gpu, _ = run_library(wl, dev, case.k_h, k_max=k_max, sm_scale=sm_scale)
    ref = run_oracle(_case_dict(case), wl, case.k_h, k_max=k_max or max(1, max(case.k_h)),
                     sm_scale=sm_scale or None)
    compare(gpu, ref, wl, case.k_h)
    return gpu, ref


SMALL = Workload("small", batch=1, heads=3, head_dim=128, n_q=300, page_size=200, n_cand=7,
                 n_cur=2, k_h=(0, 3, 9), dtype="bf16", seed=11, gates=True)


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_small_ragged(d, dtype):
    # 3 query tiles with a ragged tail, pages that straddle 64-key tiles,
    # a head with no budget and a head whose budget exceeds the history.
    _run_small(SMALL.replace(head_dim=d, dtype=dtype))


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_elementwise_gates(d, dtype):
    # one gate logit per output element (cfg.gate_dims = d), in the fused
    # epilogue of the walk and of the split combine
    _run_small(SMALL.replace(head_dim=d, dtype=dtype, seed=23), mutate=elementwise_gates)
    _run_small(SMALL.replace(head_dim=d, dtype=dtype, batch=2, heads=2, k_h=(2, 5), n_q=129,
                             seed=24), mutate=elementwise_gates)


def test_batch_two_and_gates():
    _run_small(SMALL.replace(batch=2, heads=2, k_h=(2, 5), n_q=129, seed=12))


@pytest.mark.parametrize("P", [8, 64, 136])
def test_page_sizes(P):
    _run_small(SMALL.replace(page_size=P, n_cand=11, k_h=(1, 4, 6), seed=13 + P))


def test_single_query_and_no_history():
    _run_small(SMALL.replace(n_q=1, seed=14))
    _run_small(SMALL.replace(n_cand=0, k_h=(0, 0, 0), seed=15), k_max=2)


def test_explicit_softmax_scale():
    _run_small(SMALL.replace(seed=16), sm_scale=0.05)


@pytest.mark.parametrize("d", [128, 64])
def test_one_and_two_tile_walks(d):
    # The page walk's first and last slots: a single 64-key tile (one current
    # page, no history), two tiles (one selected page), and a page shorter
    # than a tile, each with a query tile of one query at the end (n_q = 257).
    base = SMALL.replace(head_dim=d, n_q=257, page_size=64, n_cur=1, seed=17)
    _run_small(base.replace(n_cand=0, k_h=(0, 0, 0)), k_max=1)
    _run_small(base.replace(n_cand=2, k_h=(1, 0, 1), seed=18))
    _run_small(base.replace(page_size=40, n_cand=2, k_h=(1, 2, 0), seed=19))


def test_duplicate_pages_tie_to_lower_index():
    wl = SMALL.replace(heads=2, k_h=(1, 2), n_cand=9, seed=17)

    def dup(case):
        # pages 2, 5 and 7 identical and aligned with the mean query of each head
        for h in range(wl.heads):
            qd = case.q[0, :, h, :].mean(0)
            page = np.tile(qd * 2.0, (wl.page_size, 1)).astype(np.float32)
            from synth_inputs import bf16_bits_to_f32, f32_to_bf16_bits
            page = bf16_bits_to_f32(f32_to_bf16_bits(page))
            for p in (2, 5, 7):
                case.k_pool[case.page_table[0, p], h] = page

    gpu, ref = _run_small(wl, mutate=dup)
    assert gpu["sel"][0, 0, 0] == 2
    assert list(gpu["sel"][0, 1, :2]) == [2, 5]


def test_c1_tiny_f32():
    _run_small(WORKLOADS["c1"])


def _rows(n_q, k=192, seed=0):
    r = np.random.default_rng(seed).choice(n_q, size=min(k, n_q), replace=False)
    tail = [0, 1, 31, 32, 127, 128, n_q - 1, n_q - 2, (n_q // 128) * 128]
    return np.unique(np.concatenate([r, [t for t in tail if 0 <= t < n_q]]))


def _full_size(name, rows_k=160):
    import torch
    from synth_inputs import make_case_torch
    wl = WORKLOADS[name]
    say(f"[case] full-size {wl.name}")
    dev = make_case_torch(wl, "cuda:0")
    torch.cuda.synchronize()
    k_h = dev["k_h"]
    gpu, _ = run_library(wl, dev, k_h)
    host = {k: (None if v is None else v.float().cpu().numpy())
            for k, v in dev.items() if k in ("q", "k_pool", "v_pool")}
    host["page_table"] = dev["page_table"].cpu().numpy()
    rows = _rows(wl.n_q, rows_k)
    ref = run_oracle(host, wl, k_h, rows=rows)
    compare(gpu, ref, wl, k_h, rows=rows)
    return gpu, ref, dev


def test_c2_single_layer_full_size():
    _full_size("c2")


def test_c3_long_history_full_size():
    _full_size("c3")


def test_c4_prompt_switch_recall_full_size():
    gpu, ref, dev = _full_size("c4", rows_k=96)
    pc, cs = dev["meta"]["page_cluster"], dev["meta"]["c_star"]
    star = set(np.nonzero(pc == cs)[0].tolist())
    for h in range(gpu["sel"].shape[1]):
        s = gpu["sel"][0, h][gpu["sel"][0, h] >= 0]
        assert set(s.tolist()) <= star, (h, s)
        assert any(140 <= p < 150 for p in s)


def test_determinism():
    import torch
    wl = SMALL.replace(seed=21)
    case = make_case(wl)
    dev = upload(case)
    a, _ = run_library(wl, dev, case.k_h)
    b, _ = run_library(wl, dev, case.k_h)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)
    torch.cuda.synchronize()


def test_forward_selected_matches_forward():
    import torch
    from paper_2609_34606_amd import HsaLayer
    wl = SMALL.replace(seed=31)
    case = make_case(wl)
    dev = upload(case)
    say(f"[case] forward_selected {wl}")
    B, n_q, H, d = dev["q"].shape
    layer = HsaLayer(B, H, d, wl.page_size, dev["q"].dtype, dev["q"].device, k_pool=dev["k_pool"],
                     v_pool=dev["v_pool"], page_table=dev["page_table"])
    layer.fold(0, wl.n_pages)
    k_h = list(case.k_h)
    sel = torch.empty((B, H, max(k_h)), dtype=torch.int32, device=dev["q"].device)
    a = layer.forward(dev["q"], wl.n_cand, wl.n_cur, k_h, g_lin=dev["g_lin"], g_sp=dev["g_sp"],
                      sel_out=sel)
    b = layer.forward_selected(dev["q"], sel, wl.n_cand, wl.n_cur, k_h, g_lin=dev["g_lin"],
                               g_sp=dev["g_sp"])
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_streaming_incremental_state_and_outputs():
    # Chunks of 3 pages appended one by one; at chunk t the history is the
    # 3(t-1) earlier pages and the state covers every page written so far.
    import torch
    from oracle import hsa_oracle as O
    from paper_2609_34606_amd import HsaLayer
    T = 4
    wl = SMALL.replace(heads=2, n_q=150, page_size=200, n_cand=3 * (T - 1), n_cur=3, k_h=(2, 5),
                       seed=41)
    case = make_case(wl)            # pages 0..11 of the whole stream
    dev = upload(case)
    B, _, H, d = dev["q"].shape
    layer = HsaLayer(B, H, d, wl.page_size, dev["q"].dtype, dev["q"].device, k_pool=dev["k_pool"],
                     v_pool=dev["v_pool"], page_table=dev["page_table"])
    for t in range(1, T + 1):
        say(f"[case] streaming chunk {t}")
        qc = make_case(wl, chunk=t).q   # a fresh query chunk
        q = torch.from_numpy(qc).to("cuda:0").to(torch.bfloat16)
        n_cand = 3 * (t - 1)
        layer.fold(n_cand, 3)
        sel = torch.full((B, H, 5), -7, dtype=torch.int32, device="cuda:0")
        o = layer.forward(q, n_cand, 3, list(case.k_h), k_max=5, sel_out=sel)
        torch.cuda.synchronize()
        ref = O.hsa_forward(qc, case.k_pool, case.v_pool, case.page_table, n_cand, 3,
                            list(case.k_h), k_max=5, state_pages=range(3 * t))
        np.testing.assert_array_equal(sel.cpu().numpy(), ref["sel"])
        from hsa_testlib import BF16_TOL, assert_close
        assert_close(f"O chunk {t}", o.float().cpu().numpy(), ref["O"], **BF16_TOL)
    # the incremental state equals a cold fold of the same pages
    cold = HsaLayer(B, H, d, wl.page_size, dev["q"].dtype, dev["q"].device, k_pool=dev["k_pool"],
                    v_pool=dev["v_pool"], page_table=dev["page_table"])
    cold.fold(0, 3 * T)
    torch.cuda.synchronize()
    np.testing.assert_allclose(layer.kv_state.cpu().numpy(), cold.kv_state.cpu().numpy(),
                               rtol=1e-5, atol=1e-4)
    np.testing.assert_allclose(layer.k_state.cpu().numpy(), cold.k_state.cpu().numpy(), rtol=1e-6)
    np.testing.assert_array_equal(layer.page_kmean.cpu().numpy(), cold.page_kmean.cpu().numpy())


def test_c5_last_chunk_full_size():
    # streaming workload at its longest history: chunk 60, 177 history pages
    from synth_inputs.configs import streaming_chunk
    wl = streaming_chunk(WORKLOADS["c5"], 60)
    WORKLOADS["_c5_t60"] = wl
    try:
        _full_size("_c5_t60", rows_k=96)
    finally:
        del WORKLOADS["_c5_t60"]
