"""GPU parity of the two-stage retrieval (Stage-1 chunk, Stage-2 pages
inside it) against the fp64 oracle, and of the forward pass at the paper's
page geometry (pages of 8 latent frames = 12,480 tokens, K_p = 4).

The chosen chunk and the page selection are compared bit-exact (fp64 on both
sides), the chunk's cosine within 1e-12, outputs within the bf16 / fp32 bars
of hsa_testlib."""
import numpy as np
import pytest

from synth_inputs import WORKLOADS, make_case, make_prompts
from synth_inputs.configs import Workload

from hsa_testlib import BF16_TOL, F32_TOL, assert_close, compare, run_library, run_oracle, say
from hsa_testlib import to_host, upload
from oracle import hsa_hkv_oracle as HK

pytestmark = pytest.mark.gpu

SMALL = Workload("small_retrieval", batch=1, heads=3, head_dim=128, n_q=300, page_size=200,
                 n_cand=9, n_cur=3, k_h=(0, 2, 5), dtype="bf16", seed=81, gates=True)


def _run(wl, host, dev, k_h, prompts, rows=None, mutate_prompts=None):
    import torch
    from paper_2609_34606_amd import HsaLayer, hsa_chunk_select
    pe, ce, cf = prompts
    if mutate_prompts:
        mutate_prompts(pe, ce)
    cuda = dev["q"].device
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(cuda)
    pe_d, ce_d, cf_d = t(pe), t(ce), t(cf)
    B, n_q, H, d = dev["q"].shape
    M, E = ce.shape[1], ce.shape[2]
    k_max = max(1, max(k_h))
    layer = HsaLayer(B, H, d, wl.page_size, dev["q"].dtype, cuda, k_pool=dev["k_pool"],
                     v_pool=dev["v_pool"], page_table=dev["page_table"])
    layer.fold(0, wl.n_pages)
    o = torch.empty_like(dev["q"])
    sel = torch.full((B, H, k_max), -7, dtype=torch.int32, device=cuda)
    chunk = torch.full((B,), -7, dtype=torch.int32, device=cuda)
    from paper_2609_34606_amd import hsa_forward_retrieval
    hsa_forward_retrieval(layer.cfg, dev["q"], n_q, layer.pool, pe_d, ce_d, E, M, cf_d, wl.n_cand,
                          wl.n_cur, list(k_h), k_max, layer.kv_state, layer.k_state,
                          layer.page_kmean, dev.get("g_lin"), dev.get("g_sp"), o, chunk_out=chunk,
                          sel_out=sel)
    score = torch.zeros((B,), dtype=torch.float64, device=cuda)
    rng_ = torch.zeros((B, 2), dtype=torch.int32, device=cuda)
    hsa_chunk_select(layer.cfg, pe_d, ce_d, E, M, cf_d, wl.n_cand, rng_, chunk_score=score)
    torch.cuda.synchronize()
    ref = HK.hsa_forward_retrieval(host["q"], host["k_pool"], host["v_pool"], host["page_table"],
                                   pe, ce, cf, wl.n_cur, list(k_h), host.get("g_lin"),
                                   host.get("g_sp"), k_max=k_max, query_rows=rows)
    say(f"  chunk {to_host(chunk).tolist()} (oracle {ref['chunk'].tolist()}), cos {to_host(score).tolist()}")
    np.testing.assert_array_equal(to_host(chunk), ref["chunk"])
    np.testing.assert_allclose(to_host(score), ref["chunk_score"], rtol=0, atol=1e-12)
    r = to_host(rng_)
    for b in range(B):
        m = int(ref["chunk"][b])
        assert r[b].tolist() == [int(cf[b, m]), int(cf[b, m + 1])]
    np.testing.assert_array_equal(to_host(sel), ref["sel"])
    tol = BF16_TOL if wl.dtype == "bf16" else F32_TOL
    go = to_host(o) if rows is None else to_host(o)[:, rows]
    assert_close("O", go, ref["O"], **tol)
    return ref


def _small(wl, mutate_prompts=None, emb_dim=256):
    say(f"[case] retrieval {wl}")
    case = make_case(wl)
    host = dict(q=case.q, k_pool=case.k_pool, v_pool=case.v_pool, page_table=case.page_table,
                g_lin=case.g_lin, g_sp=case.g_sp)
    return _run(wl, host, upload(case), list(case.k_h), make_prompts(wl, emb_dim),
                mutate_prompts=mutate_prompts)


@pytest.mark.parametrize("d", [128, 64])
def test_small_bf16(d):
    _small(SMALL.replace(head_dim=d))


def test_small_fp32():
    # c1: chunks of one page, so every head keeps a single page
    _small(WORKLOADS["c1"])


def test_tied_chunks_pick_the_lower_index():
    def tie(pe, ce):
        ce[0, 2] = pe[0] * 2.0
        ce[0, 1] = pe[0] * 0.5   # the same cosine (1), lower index
    ref = _small(SMALL.replace(seed=82), mutate_prompts=tie)
    assert ref["chunk"][0] == 1


@pytest.mark.parametrize("emb_dim", [1000, 2102])
def test_many_chunks_ragged_embedding(emb_dim):
    # 40 one-page chunks (more than one per wave of the Stage-1 workgroup)
    # and embedding sizes that end inside a round of a lane's loads (1000:
    # 16-byte loads, 2102: 4-byte loads)
    _small(SMALL.replace(page_size=64, n_cand=40, n_cur=1, k_h=(1, 0, 1), seed=83), emb_dim=emb_dim)


def test_c4_prompt_switch_full_size():
    import torch
    from synth_inputs import make_case_torch
    wl = WORKLOADS["c4"]
    say(f"[case] retrieval full-size {wl.name}")
    dev = make_case_torch(wl, "cuda:0")
    torch.cuda.synchronize()
    host = {k: dev[k].float().cpu().numpy() for k in ("q", "k_pool", "v_pool")}
    host["page_table"] = dev["page_table"].cpu().numpy()
    rows = np.unique(np.concatenate([np.arange(0, 4680, 97), [4679]]))
    ref = _run(wl, host, dev, list(dev["k_h"]), make_prompts(wl), rows=rows)
    # the chosen chunk holds the current chunk's cluster
    pc, cs = dev["meta"]["page_cluster"], dev["meta"]["c_star"]
    m = int(ref["chunk"][0])
    assert (pc[10 * m:10 * m + 10] == cs).all()


def test_paper_page_geometry():
    # a page is 8 latent frames of 1560 tokens (12,480 keys) and K_p = 4
    # pages are retrieved: 4 x 8 x 1560 = 49,920 history keys per head
    wl = Workload("paper_geometry", batch=1, heads=2, head_dim=128, n_q=520, page_size=8 * 1560,
                  n_cand=6, n_cur=1, k_h=(4, 4), dtype="bf16", seed=83, gates=True)
    say(f"[case] paper geometry {wl}")
    case = make_case(wl)
    dev = upload(case)
    gpu, _ = run_library(wl, dev, case.k_h)
    rows = np.unique(np.concatenate([np.arange(0, 520, 13), [519]]))
    ref = run_oracle(dict(q=case.q, k_pool=case.k_pool, v_pool=case.v_pool,
                          page_table=case.page_table, g_lin=case.g_lin, g_sp=case.g_sp),
                     wl, case.k_h, rows=rows)
    assert (gpu["sel"] >= 0).sum(-1).tolist() == [[4, 4]]
    compare(gpu, ref, wl, case.k_h, rows=rows)
