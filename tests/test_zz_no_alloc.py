"""hsa_forward_noalloc (the entry point for callers that cannot allocate)
against hsa_forward on the same inputs: two calls in a row on the same
GPU's static workspace, the second with a smaller input (fewer heads,
queries and pages), so stale contents of the first call must not leak into
the second. Both run the same kernels with the same schedule, so the
selection and the output must match bit for bit (the parity bar for bf16
outputs, max-abs 2e-2 / rel-L2 5e-3, is then met trivially; it is checked
too)."""
import numpy as np
import pytest

from synth_inputs.configs import Workload

from hsa_testlib import BF16_TOL, assert_close, say

pytestmark = pytest.mark.gpu

# first call: uneven budgets so that the schedule splits long lists and the
# split partials land in the static workspace
BIG = Workload("noalloc_big", batch=1, heads=12, head_dim=128, n_q=4680, page_size=1560,
               n_cand=40, n_cur=3, k_h=(16, 2, 8, 16, 4, 2, 8, 16, 2, 4, 8, 16), dtype="bf16",
               seed=71, gates=True)
SMALL = Workload("noalloc_small", batch=1, heads=3, head_dim=128, n_q=300, page_size=200,
                 n_cand=7, n_cur=2, k_h=(0, 3, 9), dtype="bf16", seed=72, gates=True)


def _both(wl):
    import torch
    from paper_2609_34606_amd import HsaLayer, hsa_forward_noalloc, hsa_forward_noalloc_bytes
    from synth_inputs import make_case_torch
    say(f"[case] noalloc vs forward {wl}")
    dev = make_case_torch(wl, "cuda:0")
    q = dev["q"]
    B, n_q, H, d = q.shape
    k_h = [int(x) for x in dev["k_h"]]
    k_max = max(1, max(k_h))
    layer = HsaLayer(B, H, d, wl.page_size, q.dtype, q.device, k_pool=dev["k_pool"],
                     v_pool=dev["v_pool"], page_table=dev["page_table"])
    layer.fold(0, wl.n_pages)
    need = hsa_forward_noalloc_bytes(layer.cfg, n_q, wl.n_cand, wl.n_cur, k_h, k_max)
    assert 0 < need <= (128 << 20), need
    sel_a = torch.full((B, H, k_max), -7, dtype=torch.int32, device=q.device)
    sel_b = torch.full_like(sel_a, -9)
    o_a = layer.forward(q, wl.n_cand, wl.n_cur, k_h, k_max=k_max, g_lin=dev["g_lin"],
                        g_sp=dev["g_sp"], sel_out=sel_a)
    o_b = torch.full_like(o_a, float("nan"))
    hsa_forward_noalloc(layer.cfg, q, n_q, layer.pool, wl.n_cand, wl.n_cur, k_h, k_max,
                        layer.kv_state, layer.k_state, layer.page_kmean, dev["g_lin"], dev["g_sp"],
                        o_b, sel_out=sel_b)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(sel_b.cpu().numpy(), sel_a.cpu().numpy())
    assert_close("O noalloc vs forward", o_b.float().cpu().numpy(), o_a.float().cpu().numpy(),
                 **BF16_TOL)
    assert torch.equal(o_a.view(torch.int16), o_b.view(torch.int16)), "outputs differ in some bits"
    # without sel_out the selection goes to the static workspace too
    o_c = torch.full_like(o_a, float("nan"))
    hsa_forward_noalloc(layer.cfg, q, n_q, layer.pool, wl.n_cand, wl.n_cur, k_h, k_max,
                        layer.kv_state, layer.k_state, layer.page_kmean, dev["g_lin"], dev["g_sp"],
                        o_c)
    torch.cuda.synchronize()
    assert torch.equal(o_a.view(torch.int16), o_c.view(torch.int16))


def test_noalloc_matches_forward_twice_second_smaller():
    _both(BIG)
    _both(SMALL)
