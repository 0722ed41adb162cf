"""GPU runs of the optional argument checks (HSA_CHECK=1): page-table entries
and selected pages that name no slot of the pool are reported as
HSA_ERR_OUT_OF_RANGE before any kernel is launched, and a valid call gives
the same bits as without the checks."""
import os

import numpy as np
import pytest

from synth_inputs import make_case
from synth_inputs.configs import Workload

from hsa_testlib import say, upload

pytestmark = pytest.mark.gpu

WL = Workload("small_checks", batch=1, heads=2, head_dim=128, n_q=200, page_size=64, n_cand=5,
              n_cur=2, k_h=(2, 3), dtype="bf16", seed=91, gates=False)


@pytest.fixture
def checks_on():
    old = os.environ.get("HSA_CHECK")
    os.environ["HSA_CHECK"] = "1"
    yield
    if old is None:
        del os.environ["HSA_CHECK"]
    else:
        os.environ["HSA_CHECK"] = old


def _layer(dev):
    from paper_2609_34606_amd import HsaLayer
    B, n_q, H, d = dev["q"].shape
    return HsaLayer(B, H, d, WL.page_size, dev["q"].dtype, dev["q"].device, k_pool=dev["k_pool"],
                    v_pool=dev["v_pool"], page_table=dev["page_table"])


def test_checked_call_matches_unchecked():
    import torch
    say("[case] HSA_CHECK valid call")
    case = make_case(WL)
    dev = upload(case)
    a = _layer(dev)
    a.fold(0, WL.n_pages)
    oa = a.forward(dev["q"], WL.n_cand, WL.n_cur, list(WL.k_h))
    os.environ["HSA_CHECK"] = "1"
    try:
        b = _layer(dev)
        b.fold(0, WL.n_pages)
        ob = b.forward(dev["q"], WL.n_cand, WL.n_cur, list(WL.k_h))
    finally:
        del os.environ["HSA_CHECK"]
    torch.cuda.synchronize()
    assert torch.equal(oa.view(torch.int16), ob.view(torch.int16))
    assert torch.equal(a.kv_state, b.kv_state)


def test_bad_slot_in_current_pages_is_out_of_range(checks_on):
    import torch
    from paper_2609_34606_amd.hsa import HsaError
    say("[case] HSA_CHECK bad current-page slot")
    case = make_case(WL)
    dev = upload(case)
    layer = _layer(dev)
    layer.fold(0, WL.n_pages)
    bad = dev["page_table"].clone()
    bad[0, WL.n_cand + 1] = case.num_slots + 3   # a current page beyond the pool
    layer.page_table.copy_(bad)
    with pytest.raises(HsaError) as e:
        layer.forward(dev["q"], WL.n_cand, WL.n_cur, list(WL.k_h))
    assert e.value.status == 3
    with pytest.raises(HsaError) as e:
        layer.fold(WL.n_cand, WL.n_cur)
    assert e.value.status == 3
    torch.cuda.synchronize()


def test_selected_page_with_bad_slot_is_out_of_range(checks_on):
    import torch
    from paper_2609_34606_amd.hsa import HsaError
    say("[case] HSA_CHECK bad selected-page slot")
    case = make_case(WL)
    dev = upload(case)
    layer = _layer(dev)
    layer.fold(0, WL.n_pages)
    layer.page_table[0, 1] = -5                    # history page 1 maps to no slot
    sel = torch.tensor([[[0, 1, -1], [3, 4, 0]]], dtype=torch.int32, device=dev["q"].device)
    with pytest.raises(HsaError) as e:
        layer.forward_selected(dev["q"], sel, WL.n_cand, WL.n_cur, list(WL.k_h), k_max=3)
    assert e.value.status == 3
    # the same page table is fine when the bad page is not selected
    sel_ok = torch.tensor([[[0, 2, -1], [3, 4, 0]]], dtype=torch.int32, device=dev["q"].device)
    o = layer.forward_selected(dev["q"], sel_ok, WL.n_cand, WL.n_cur, list(WL.k_h), k_max=3)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(o.float()).all())
