"""GPU check of the host-managed KV tiers: a pool with fewer slots than
logical pages, pages placed in generation order (moving the least recently
used ones to pinned host memory and from there to a file), Stage-2 selection
on the page index, a fetch of the selected and current pages, the forward
pass, and a prefetch on a side stream issued while that forward runs (it
moves pages the forward does not read). Because the kernels only read pages
that are in the pool, the result must equal, bit for bit, the forward with
every page resident (same pages folded in the same order); it is also
checked against the oracle."""
import numpy as np
import pytest

from synth_inputs import make_case
from synth_inputs.configs import Workload

from hsa_testlib import BF16_TOL, assert_close, say, to_host, upload
from oracle import hsa_oracle as O

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("l2,l3", [(9, 0), (3, 6), (1, 8)])
def test_forward_over_fetched_pages_is_bit_exact(l2, l3, tmp_path):
    import torch
    from paper_2609_34606_amd import HsaLayer, HsaTier, hsa_page_select
    wl = Workload("tier", batch=1, heads=3, head_dim=128, n_q=300, page_size=200, n_cand=15,
                  n_cur=3, k_h=(1, 2, 3), dtype="bf16", seed=91, gates=True)
    case = make_case(wl)
    dev = upload(case)
    H, d, P, npg = wl.heads, wl.head_dim, wl.page_size, wl.n_pages
    cuda = dev["q"].device
    k_h, k_max = list(wl.k_h), max(wl.k_h)
    # two chunks: the first sees 12 history pages, the second 15
    chunks = [(12, 3), (15, 3)]
    n_slots = 10                 # 18 pages fit: 10 + l2 + l3 - 1
    pool_k = torch.empty((n_slots, H, P, d), dtype=torch.bfloat16, device=cuda)
    pool_v = torch.empty((n_slots, H, d, P), dtype=torch.bfloat16, device=cuda)
    table = torch.full((1, npg + 3), -1, dtype=torch.int32, device=cuda)
    host_k = torch.empty((l2, H, P, d), dtype=torch.bfloat16, pin_memory=True)
    host_v = torch.empty((l2, H, d, P), dtype=torch.bfloat16, pin_memory=True)
    layer = HsaLayer(1, H, d, P, torch.bfloat16, cuda, k_pool=pool_k, v_pool=pool_v,
                     page_table=table)
    tier = HsaTier(layer.cfg, layer.pool, l2, host_k, host_v, l3_dir=tmp_path if l3 else None,
                   l3_slots=l3)
    side = torch.cuda.Stream()
    # the second chunk's queries are a fresh draw
    qs = [dev["q"], torch.from_numpy(make_case(wl, chunk=1).q).to(cuda).to(torch.bfloat16)]
    placed = 0
    for ci, (n_cand, n_cur) in enumerate(chunks):
        say(f"[case] tier chunk {ci}: {n_cand} history pages, pool of {n_slots}, host {l2}, file {l3}")
        # pages arrive in generation order; each is written into the slot the
        # tier gives it and folded at once (state and page index)
        for p in range(placed, n_cand + n_cur):
            lp = p % npg                      # source data of logical page p
            slot = tier.place(0, p)
            pool_k[slot] = dev["k_pool"][case.page_table[0, lp]]
            pool_v[slot] = dev["v_pool"][case.page_table[0, lp]]
            layer.fold(p, 1)
        placed = n_cand + n_cur
        q = qs[ci]
        sel = torch.full((1, H, k_max), -7, dtype=torch.int32, device=cuda)
        hsa_page_select(layer.cfg, q, wl.n_q, layer.page_kmean, layer.max_pages, n_cand, k_h,
                        k_max, sel)
        torch.cuda.synchronize()
        pages = np.concatenate([to_host(sel).reshape(1, -1),
                                np.arange(n_cand, n_cand + n_cur, dtype=np.int32)[None]], 1)
        tier.fetch(pages)
        o = layer.forward_selected(q, sel, n_cand, n_cur, k_h, g_lin=dev["g_lin"], g_sp=dev["g_sp"])
        # while the forward runs: bring back up to two pages from the lowest
        # tier holding any (the file first), moving pages the forward does not
        # read (the pool holds those and the prefetched ones together)
        room = n_slots - len(set(pages[pages >= 0].tolist()))
        lows = sorted(range(placed), key=lambda p: tier.locate(0, p))[:min(2, room)]
        lows = [p for p in lows if tier.locate(0, p) < -1]
        if lows:
            tier.prefetch([lows], stream=side)
            assert all(tier.locate(0, p) >= 0 for p in pages.ravel() if p >= 0)
        torch.cuda.synchronize()
        # the resident reference: the same pages folded in the same order
        if ci == 0:
            ref_table = torch.tensor([[case.page_table[0, p % npg] for p in range(npg + 3)]],
                                     dtype=torch.int32, device=cuda)
            ref = HsaLayer(1, H, d, P, torch.bfloat16, cuda, k_pool=dev["k_pool"],
                           v_pool=dev["v_pool"], page_table=ref_table)
            ref_done = 0
        for p in range(ref_done, n_cand + n_cur):
            ref.fold(p, 1)
        ref_done = n_cand + n_cur
        sel_r = torch.full_like(sel, -7)
        o_r = ref.forward(q, n_cand, n_cur, k_h, k_max=k_max, g_lin=dev["g_lin"], g_sp=dev["g_sp"],
                          sel_out=sel_r)
        torch.cuda.synchronize()
        say(f"  {tier.stats()}; selected {to_host(sel).tolist()}")
        assert torch.equal(sel, sel_r)
        assert torch.equal(layer.kv_state, ref.kv_state) and torch.equal(layer.page_kmean[:, :, :placed],
                                                                          ref.page_kmean[:, :, :placed])
        assert torch.equal(o.view(torch.int16), o_r.view(torch.int16))
        # and the oracle, on the logical pages as written
        lt = np.array([[case.page_table[0, p % npg] for p in range(n_cand + n_cur)]], np.int32)
        oref = O.hsa_forward(to_host(q), case.k_pool, case.v_pool, lt, n_cand, n_cur, k_h,
                             case.g_lin, case.g_sp, k_max=k_max)
        np.testing.assert_array_equal(to_host(sel), oref["sel"])
        assert_close(f"O chunk {ci}", to_host(o), oref["O"], **BF16_TOL)
    st = tier.stats()
    assert st["evictions"] > 0 and st["fetches"] > 0 and st["prefetched"] > 0
    if l3:
        assert st["spills"] > 0 and st["reloads"] > 0
    tier.close()


def test_every_page_restored_from_the_file_backup(tmp_path):
    """Backup mode: pages written to the file by commits (once per chunk of
    three), every pool and host copy dropped and overwritten with NaN, then
    each page fetched back from its file slot bit for bit, and the forward
    over restored pages equal to the one with every page resident."""
    import torch
    from paper_2609_34606_amd import HsaLayer, HsaTier, hsa_page_select
    wl = Workload("tier-backup", batch=1, heads=3, head_dim=128, n_q=300, page_size=200, n_cand=15,
                  n_cur=3, k_h=(1, 2, 3), dtype="bf16", seed=92, gates=True)
    case = make_case(wl)
    dev = upload(case)
    H, d, P, npg = wl.heads, wl.head_dim, wl.page_size, wl.n_pages
    cuda = dev["q"].device
    k_h, k_max = list(wl.k_h), max(wl.k_h)
    n_slots, l2 = 10, 2          # the forward's fetch: up to 6 selected + 3 current pages
    pool_k = torch.empty((n_slots, H, P, d), dtype=torch.bfloat16, device=cuda)
    pool_v = torch.empty((n_slots, H, d, P), dtype=torch.bfloat16, device=cuda)
    table = torch.full((1, npg), -1, dtype=torch.int32, device=cuda)
    host_k = torch.empty((l2, H, P, d), dtype=torch.bfloat16, pin_memory=True)
    host_v = torch.empty((l2, H, d, P), dtype=torch.bfloat16, pin_memory=True)
    layer = HsaLayer(1, H, d, P, torch.bfloat16, cuda, k_pool=pool_k, v_pool=pool_v,
                     page_table=table)
    tier = HsaTier(layer.cfg, layer.pool, l2, host_k, host_v, l3_dir=tmp_path, l3_slots=npg,
                   backup=True)
    src = [int(case.page_table[0, p]) for p in range(npg)]
    say(f"[case] tier backup: {npg} pages, pool of {n_slots}, host {l2}, file {npg}")
    for p in range(npg):
        slot = tier.place(0, p)
        pool_k[slot] = dev["k_pool"][src[p]]
        pool_v[slot] = dev["v_pool"][src[p]]
        layer.fold(p, 1)
        if p % 3 == 2:
            tier.commit()
    st0 = tier.stats()
    say(f"  after placing: {st0}")
    assert st0["backups"] == npg
    tier.drop()
    torch.cuda.synchronize()
    assert [tier.locate(0, p) for p in range(npg)] == [-(2 + l2 + p) for p in range(npg)]
    assert bool((table == -1).all())
    for t in (pool_k, pool_v, host_k, host_v):
        t.fill_(float("nan"))
    torch.cuda.synchronize()
    for i in range(0, npg, n_slots):
        grp = list(range(i, min(npg, i + n_slots)))
        tier.fetch([grp])
        torch.cuda.synchronize()
        tab = to_host(table)[0]
        for p in grp:
            s = tier.locate(0, p)
            assert s >= 0 and tab[p] == s
            assert torch.equal(pool_k[s].view(torch.int16), dev["k_pool"][src[p]].view(torch.int16)), p
            assert torch.equal(pool_v[s].view(torch.int16), dev["v_pool"][src[p]].view(torch.int16)), p
    st1 = tier.stats()
    say(f"  after restoring: {st1}")
    assert st1["reloads"] - st0["reloads"] == npg and st1["backups"] == npg
    # the forward over restored pages
    n_cand, n_cur = wl.n_cand, wl.n_cur
    q = dev["q"]
    sel = torch.full((1, H, k_max), -7, dtype=torch.int32, device=cuda)
    hsa_page_select(layer.cfg, q, wl.n_q, layer.page_kmean, layer.max_pages, n_cand, k_h, k_max, sel)
    torch.cuda.synchronize()
    pages = np.concatenate([to_host(sel).reshape(1, -1),
                            np.arange(n_cand, n_cand + n_cur, dtype=np.int32)[None]], 1)
    tier.fetch(pages)
    o = layer.forward_selected(q, sel, n_cand, n_cur, k_h, g_lin=dev["g_lin"], g_sp=dev["g_sp"])
    ref_table = torch.tensor([src], dtype=torch.int32, device=cuda)
    ref = HsaLayer(1, H, d, P, torch.bfloat16, cuda, k_pool=dev["k_pool"], v_pool=dev["v_pool"],
                   page_table=ref_table)
    for p in range(npg):
        ref.fold(p, 1)
    sel_r = torch.full_like(sel, -7)
    o_r = ref.forward(q, n_cand, n_cur, k_h, k_max=k_max, g_lin=dev["g_lin"], g_sp=dev["g_sp"],
                      sel_out=sel_r)
    torch.cuda.synchronize()
    assert torch.equal(sel, sel_r)
    assert torch.equal(o.view(torch.int16), o_r.view(torch.int16))
    tier.close()
