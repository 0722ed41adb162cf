"""Helpers shared by the GPU parity tests: upload a synthetic case, run the
library through its C ABI, run the oracle, compare."""
from __future__ import annotations

import sys
from typing import Dict, Optional, Sequence

import numpy as np

from oracle import hsa_oracle as O

BF16_TOL = dict(max_abs=2e-2, rel_l2=5e-3)   # bf16 outputs
F32_TOL = dict(max_abs=1e-4, rel_l2=2e-5)    # fp32 end to end


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def err(got, ref) -> Dict[str, float]:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    d = got - ref
    nr = np.linalg.norm(ref)
    return {"max_abs": float(np.abs(d).max()) if d.size else 0.0,
            "rel_l2": float(np.linalg.norm(d) / nr) if nr > 0 else float(np.linalg.norm(d))}


def assert_close(name, got, ref, max_abs, rel_l2):
    e = err(got, ref)
    say(f"  {name}: max_abs={e['max_abs']:.3e} rel_l2={e['rel_l2']:.3e}")
    assert np.isfinite(np.asarray(got, np.float64)).all(), f"{name}: non-finite output"
    assert e["max_abs"] <= max_abs, f"{name}: max_abs {e['max_abs']:.3e} > {max_abs}"
    assert e["rel_l2"] <= rel_l2, f"{name}: rel_l2 {e['rel_l2']:.3e} > {rel_l2}"
    return e


def torch_dtype(wl):
    import torch
    return torch.bfloat16 if wl.dtype == "bf16" else torch.float32


def upload(case, device="cuda:0"):
    """Device copies of a host case (bf16 values are exact in fp32)."""
    import torch
    dt = torch_dtype(case.wl)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
    out = dict(q=t(case.q).to(dt), k_pool=t(case.k_pool).to(dt), v_pool=t(case.v_pool).to(dt),
               page_table=t(case.page_table).to(torch.int32))
    out["g_lin"] = None if case.g_lin is None else t(case.g_lin)
    out["g_sp"] = None if case.g_sp is None else t(case.g_sp)
    return out


def to_host(x):
    import torch
    if x is None:
        return None
    if x.dtype == torch.bfloat16:
        x = x.float()
    return x.cpu().numpy()


def gate_dims_of(dev: Dict) -> int:
    """head_dim when the case carries element-wise gate logits [B, n_q, H, d],
    else 0 (one logit per query and head)."""
    for k in ("g_lin", "g_sp"):
        g = dev.get(k)
        if g is not None and g.dim() == 4:
            return int(g.shape[-1])
    return 0


def elementwise_gates(case, seed=23):
    """Replace a case's gate logits by seeded N(0,1) logits per output element."""
    r = np.random.default_rng(seed)
    B, n_q, H, d = case.q.shape
    case.g_lin = r.standard_normal((B, n_q, H, d)).astype(np.float32)
    case.g_sp = r.standard_normal((B, n_q, H, d)).astype(np.float32)


def run_library(wl, dev: Dict, k_h: Sequence[int], k_max: Optional[int] = None,
                sm_scale: float = 0.0, with_parts: bool = True):
    """Cold state over every page, then the full forward; optionally also the
    standalone selection (with scores) and sparse-branch calls."""
    import torch
    from paper_2609_34606_amd import HsaLayer, hsa_page_select, hsa_sparse_attn

    B, n_q, H, d = dev["q"].shape
    k_max = max(1, max(k_h)) if k_max is None else k_max
    layer = HsaLayer(B, H, d, wl.page_size, dev["q"].dtype, dev["q"].device,
                     k_pool=dev["k_pool"], v_pool=dev["v_pool"], page_table=dev["page_table"],
                     sm_scale=sm_scale, gate_dims=gate_dims_of(dev))
    layer.fold(0, wl.n_cand + wl.n_cur)
    sel = torch.full((B, H, k_max), -7, dtype=torch.int32, device=dev["q"].device)
    o = layer.forward(dev["q"], wl.n_cand, wl.n_cur, list(k_h), k_max=k_max,
                      g_lin=dev.get("g_lin"), g_sp=dev.get("g_sp"), sel_out=sel)
    res = dict(O=o, sel=sel, S_T=layer.kv_state, z=layer.k_state, kmean=layer.page_kmean)
    if with_parts:
        sel2 = torch.full_like(sel, -7)
        score = torch.zeros((B, H, k_max), dtype=torch.float64, device=sel.device)
        hsa_page_select(layer.cfg, dev["q"], n_q, layer.page_kmean, layer.max_pages, wl.n_cand,
                        list(k_h), k_max, sel2, sel_score=score)
        o_sp = torch.zeros((B, n_q, H, d), dtype=torch.float32, device=sel.device)
        lse = torch.zeros((B, H, n_q), dtype=torch.float32, device=sel.device)
        hsa_sparse_attn(layer.cfg, dev["q"], n_q, layer.pool, sel2, k_max, list(k_h),
                        wl.n_cand, wl.n_cur, o_sp, lse=lse)
        res.update(sel2=sel2, score=score, O_sp=o_sp, lse=lse)
    torch.cuda.synchronize()
    return {k: to_host(v) for k, v in res.items()}, layer


def run_oracle(case_like, wl, k_h, k_max=None, rows=None, heads=None, sm_scale=None):
    return O.hsa_forward(case_like["q"], case_like["k_pool"], case_like["v_pool"],
                         case_like["page_table"], wl.n_cand, wl.n_cur, list(k_h),
                         case_like.get("g_lin"), case_like.get("g_sp"), sm_scale=sm_scale,
                         k_max=k_max, query_rows=rows, heads=heads)


def compare(gpu, ref, wl, k_h, rows=None, tol=None, state_tol=4e-3, heads=None):
    """Compare every library output with the oracle's."""
    tol = tol or (BF16_TOL if wl.dtype == "bf16" else F32_TOL)
    heads = list(range(gpu["O"].shape[2])) if heads is None else list(heads)
    r = slice(None) if rows is None else np.asarray(rows)
    # selection: bit-exact, including -1 padding
    np.testing.assert_array_equal(gpu["sel"][:, heads], ref["sel"][:, heads])
    if "sel2" in gpu:
        np.testing.assert_array_equal(gpu["sel2"][:, heads], ref["sel"][:, heads])
        np.testing.assert_allclose(gpu["score"][:, heads], ref["sel_score"][:, heads],
                                   rtol=1e-12, atol=1e-14)
    # page index: fp64
    npg = wl.n_cand + wl.n_cur
    np.testing.assert_allclose(gpu["kmean"][:, heads, :npg], ref["kbar"][:, heads],
                               rtol=1e-12, atol=1e-15)
    # linear state (library stores the transpose)
    S_ref = np.swapaxes(ref["S"], -1, -2)[:, heads]
    st_tol = state_tol if wl.dtype == "bf16" else 1e-5
    assert_close("kv_state", gpu["S_T"][:, heads], S_ref, max_abs=np.inf, rel_l2=st_tol)
    assert_close("k_state", gpu["z"][:, heads], ref["z"][:, heads], max_abs=np.inf, rel_l2=1e-5)
    go = gpu["O"][:, r][:, :, heads]
    assert_close("O", go, ref["O"][:, :, heads], **tol)
    if "O_sp" in gpu:
        assert_close("O_sp", gpu["O_sp"][:, r][:, :, heads], ref["O_sp"][:, :, heads], **tol)
        lse_g = gpu["lse"][:, heads][:, :, r]
        np.testing.assert_allclose(lse_g, ref["lse"][:, heads], atol=2e-3 if wl.dtype == "bf16" else 1e-4)
