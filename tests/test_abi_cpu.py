"""Host-side checks of libhsa.so that need no GPU: the library loads, exports
every function include/hsa.h declares, and rejects bad arguments before any
launch (none of these calls reaches a kernel)."""
import ctypes
import os
import re

import pytest

import paper_2609_34606_amd as P
from paper_2609_34606_amd import hsa as H

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "hsa.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(hsa_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = P.lib()
    names = declared_functions()
    assert len(names) >= 9, names
    for n in names:
        assert hasattr(lib, n), n


def test_missing_library_fails_loudly(monkeypatch):
    monkeypatch.setattr(H, "_lib", None)
    monkeypatch.setattr(H, "LIB_PATH", "/nonexistent/libhsa.so")
    with pytest.raises(H.LibraryNotBuilt):
        H.lib()


def test_status_strings():
    for code, name in H.STATUS.items():
        assert P.hsa_status_string(code) == name


def test_workspace_sizes():
    cfg = P.config(1, 12, 128, 1560, "bf16")
    s123 = P.hsa_state_update_workspace_size(cfg, 123)
    assert s123 > 0 and s123 % 256 == 0
    assert P.hsa_state_update_workspace_size(cfg, 0) == 0
    assert P.hsa_page_select_workspace_size(cfg, 4680) >= 4680 // 32 * 12 * 128 * 8
    assert P.hsa_forward_workspace_size(cfg, 4680, 16, 3) >= P.hsa_page_select_workspace_size(cfg, 4680)
    bad = P.config(1, 12, 96, 1560, "bf16")
    assert P.hsa_state_update_workspace_size(bad, 3) == 0


def _pool(num_slots=4, max_pages=4):
    # fake non-NULL device pointers: validation fails before any use
    return H.HsaKvPool(0x1000, 0x2000, 0x3000, num_slots, max_pages)


def test_validation_errors_without_launch():
    lib = P.lib()
    cfg = P.config(1, 2, 64, 256, "f32")
    pool = _pool()
    by = ctypes.byref
    fake = ctypes.c_void_p(0x4000)
    # NULL config / pool / outputs
    assert lib.hsa_state_update(None, by(pool), 0, 1, fake, fake, fake, None, 0, None) == 1
    assert lib.hsa_state_update(by(cfg), None, 0, 1, fake, fake, fake, None, 0, None) == 1
    assert lib.hsa_state_update(by(cfg), by(pool), 0, 1, None, fake, fake, None, 0, None) == 1
    # page range beyond the page table
    assert lib.hsa_state_update(by(cfg), by(pool), 2, 3, fake, fake, fake, None, 0, None) == 3
    # workspace missing / misaligned
    assert lib.hsa_state_update(by(cfg), by(pool), 0, 2, fake, fake, fake, None, 0, None) == 4
    assert lib.hsa_state_update(by(cfg), by(pool), 0, 2, fake, fake, fake,
                                ctypes.c_void_p(0x4004), 1 << 30, None) == 4
    # unsupported shapes
    for c in (P.config(1, 2, 96, 256, "f32"), P.config(1, 2, 64, 12, "f32"),
              P.config(1, 65, 64, 256, "f32"), P.config(1, 2, 64, 256, 7)):
        assert lib.hsa_state_update(by(c), by(pool), 0, 1, fake, fake, fake, None, 0, None) == 2
    # selection: budget above k_max, history beyond the page table
    import numpy as np
    kh = np.array([3, 1], np.int32)
    khp = kh.ctypes.data_as(ctypes.c_void_p)
    assert lib.hsa_page_select(by(cfg), fake, 8, fake, 4, 2, khp, 2, fake, None, fake, 1 << 20,
                               None) == 1
    assert lib.hsa_page_select(by(cfg), fake, 8, fake, 4, 5, khp, 4, fake, None, fake, 1 << 20,
                               None) == 3
    # forward: a head with no active page
    kh0 = np.array([0, 1], np.int32)
    assert lib.hsa_forward(by(cfg), fake, 8, by(pool), 2, 0, kh0.ctypes.data_as(ctypes.c_void_p),
                           1, fake, fake, fake, None, None, fake, None, fake, 1 << 20, None) == 1
    # sparse branch: empty key set everywhere
    assert lib.hsa_sparse_attn(by(cfg), fake, 8, by(pool), None, 0, None, 0, 0, fake, None, None,
                               0, None) == 1
    # list longer than the kernels hold
    assert lib.hsa_sparse_attn(by(cfg), fake, 8, by(_pool(4, 4000)), fake, 1020, None, 0, 8, fake,
                               None, None, 0, None) == 2
    # negative scale
    neg = P.config(1, 2, 64, 256, "f32", sm_scale=-1.0)
    assert lib.hsa_state_update(by(neg), by(pool), 0, 1, fake, fake, fake, None, 0, None) == 1
    # gate shape: one logit per (query, head) (0 or 1) or per element (head_dim)
    for gd, want in ((1, 0), (64, 0), (5, 1), (128, 1), (-1, 1)):
        g = P.config(1, 2, 64, 256, "f32", gate_dims=gd)
        assert lib.hsa_state_update(by(g), by(pool), 0, 2, fake, fake, fake, None, 0, None) == (
            4 if want == 0 else 1), gd


def test_adaptive_entry_points_validate_before_launch():
    import numpy as np
    lib = P.lib()
    by = ctypes.byref
    fake = ctypes.c_void_p(0x4000)
    cfg = P.config(1, 2, 128, 1560, "bf16")
    pool = _pool(64, 64)
    # block counts: 13 blocks of <= 128 per history page, 25 of <= 64 per current page
    assert P.hsa_block_count(cfg, 4, 3) == 4 * 13 + 3 * 25
    assert P.hsa_block_count(cfg, -1, 3) == -1
    ws = P.hsa_adaptive_workspace_size(cfg, 4680, 16, 3)
    assert ws > P.hsa_sparse_attn_workspace_size(cfg, 4680, 16, 3) and ws % 256 == 0
    kh = np.array([4, 4], np.int32)
    khp = kh.ctypes.data_as(ctypes.c_void_p)
    big = 1 << 30
    # thresholds outside 0 <= tau_min <= tau_max <= 1
    for tmin, tmax in ((-0.1, 1.0), (0.5, 0.4), (0.3, 1.5), (float("nan"), 1.0)):
        assert lib.hsa_sparse_attn_adaptive(by(cfg), fake, 64, by(pool), fake, 4, khp, 10, 3,
                                            tmin, tmax, fake, None, fake, big, None) == 1
        assert lib.hsa_forward_adaptive(by(cfg), fake, 64, by(pool), 10, 3, khp, 4, tmin, tmax,
                                        fake, fake, fake, None, None, fake, None, fake, big,
                                        None) == 1
    # kept rows shorter than the block count
    assert lib.hsa_block_select(by(cfg), fake, 64, by(pool), fake, 4, 10, 3, 0.35, 1.0, None, None,
                                None, fake, None, 4 * 13 + 3 * 25 - 1, fake, big, None) == 1
    # more key blocks than a head's list may hold
    long_pool = _pool(4, 1000)
    assert lib.hsa_sparse_attn_adaptive(by(cfg), fake, 64, by(long_pool), fake, 320, None, 0, 3,
                                        0.35, 1.0, fake, None, fake, big, None) == 2
    # workspace too small
    assert lib.hsa_sparse_attn_adaptive(by(cfg), fake, 64, by(pool), fake, 4, khp, 10, 3, 0.35,
                                        1.0, fake, None, fake, 1024, None) == 4


def test_library_shares_torchs_hip_runtime():
    # loading the library first (before any torch call) must not leave two
    # HIP runtimes in the process: the binding imports torch before it
    import subprocess
    import sys
    code = ("import paper_2609_34606_amd.hsa as H; H.lib(); "
            "m = open('/proc/self/maps').read(); "
            "print(len({l.split()[-1] for l in m.splitlines() if 'libamdhip64' in l}))")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                         cwd=os.path.dirname(os.path.dirname(os.path.abspath(__file__))), timeout=300)
    assert out.returncode == 0, out.stderr[-2000:]
    assert out.stdout.strip().splitlines()[-1] == "1"


def test_tier_policy_plan_only():
    # 4 pool slots, 6 host slots, 10 logical pages: pages leave the pool least
    # recently used first; a fetch brings listed pages back and pins them
    cfg = P.config(1, 2, 64, 256, "bf16")
    t = P.HsaTier(cfg, None, 6, num_slots=4, max_pages=10)
    slots = [t.place(0, p) for p in range(4)]
    assert sorted(slots) == [0, 1, 2, 3] and t.counters() == (0, 0)
    assert t.place(0, 4) == slots[0] and t.locate(0, 0) == -2     # page 0 -> host slot 0
    assert t.place(0, 5) == slots[1] and t.locate(0, 1) == -3
    t.fetch([[0, 2]])                  # 0 comes back into the LRU slot (page 3's); 2 is pinned
    assert t.locate(0, 0) >= 0 and t.locate(0, 2) >= 0 and t.locate(0, 3) < -1
    assert t.counters() == (3, 1)
    t.place(0, 6)                      # LRU among 4, 5, 0, 2: page 4
    assert t.locate(0, 4) < -1
    # more pages listed than the pool holds
    assert t.fetch([[0, 1, 2, 3, 5]], check=False) == 2
    # a page never placed, a page out of range
    assert t.fetch([[9]], check=False) == 1 and t.fetch([[10]], check=False) == 3
    assert t.place(0, 6, check=False)[0] == 1                       # placed twice
    # capacity: pool + host slots - 1 (one host slot stays free for swaps)
    t2 = P.HsaTier(cfg, None, 2, num_slots=2, max_pages=10)
    t2.place(0, 0), t2.place(0, 1), t2.place(0, 2)
    assert t2.place(0, 3, check=False)[0] == 2
    t2.fetch([[0, 1]])                 # both back in the pool through the spare slot
    assert t2.locate(0, 0) >= 0 and t2.locate(0, 1) >= 0 and t2.locate(0, 2) < -1
    t.close(), t2.close()


def test_tier_three_levels_and_prefetch_plan_only():
    # 2 pool slots, 2 host slots, 3 file slots (capacity 2 + 2 + 3 - 1 = 6):
    # L1 evicts its least recently used page to L2, a full L2 spills its own
    # to L3, a page read back from L3 frees its slot for the spill it causes
    cfg = P.config(1, 2, 64, 256, "bf16")
    with pytest.raises(P.HsaError):
        P.HsaTier(cfg, None, 0, num_slots=2, max_pages=10, l3_slots=3)   # L3 needs L2
    t = P.HsaTier(cfg, None, 2, num_slots=2, max_pages=10, l3_slots=3)
    L2 = lambda i: -(i + 2)
    L3 = lambda i: -(2 + 2 + i)
    for p in range(6):
        t.place(0, p)
    assert t.place(0, 6, check=False)[0] == 2
    assert [t.locate(0, p) for p in range(6)] == [L3(0), L3(1), L2(0), L2(1), 0, 1]
    assert t.stats() == dict(evictions=4, fetches=0, spills=2, reloads=0, prefetched=0, backups=0)
    t.fetch([[0]])                 # p0: L3 -> L1; p4 -> L2; p2 -> L3 (the freed slot)
    assert [t.locate(0, p) for p in range(6)] == [0, L3(1), L3(0), L2(1), L2(0), 1]
    # a prefetch leaves the fetched page where it is and moves the other
    t.prefetch([[1]])
    assert [t.locate(0, p) for p in range(6)] == [0, 1, L3(0), L3(1), L2(0), L2(1)]
    assert t.stats() == dict(evictions=6, fetches=2, spills=4, reloads=2, prefetched=1, backups=0)
    # the fetched page plus two more do not fit in two slots
    assert t.prefetch([[2, 3]], check=False) == 2
    # a fetch may move anything it does not list
    t.fetch([[2, 3]])
    assert [t.locate(0, p) for p in range(6)] == [L2(0), L2(1), 0, 1, L3(0), L3(1)]
    assert t.stats() == dict(evictions=8, fetches=4, spills=6, reloads=4, prefetched=1, backups=0)
    # a fetch swaps: each page it brings from L2 trades places with the page
    # it displaces, which takes its host slot
    t.fetch([[0, 1]])
    assert [t.locate(0, p) for p in range(6)] == [0, 1, L2(0), L2(1), L3(0), L3(1)]
    assert t.stats() == dict(evictions=10, fetches=6, spills=6, reloads=4, prefetched=1, backups=0)
    t.close()
    # one host slot, holding a page the fetch lists: the pool's least
    # recently used page goes straight to a free file slot
    t = P.HsaTier(cfg, None, 1, num_slots=2, max_pages=10, l3_slots=3)
    L3 = lambda i: -(2 + 1 + i)
    for p in range(5):
        t.place(0, p)
    assert [t.locate(0, p) for p in range(5)] == [L3(0), L3(1), L2(0), 1, 0]
    t.fetch([[0, 2]])
    assert [t.locate(0, p) for p in range(5)] == [1, L3(1), 0, L3(0), L2(0)]
    assert t.stats() == dict(evictions=5, fetches=2, spills=3, reloads=1, prefetched=0, backups=0)
    t.close()


def test_tier_backup_plan_only():
    # backup mode: 2 pool slots, 1 host slot, 5 file slots, one per page
    cfg = P.config(1, 2, 64, 256, "bf16")
    with pytest.raises(P.HsaError):
        P.HsaTier(cfg, None, 1, num_slots=2, max_pages=10, backup=True)   # needs file slots
    t = P.HsaTier(cfg, None, 1, num_slots=2, max_pages=10, l3_slots=5, backup=True)
    L2 = lambda i: -(i + 2)
    L3 = lambda i: -(2 + 1 + i)
    for p in range(5):
        t.place(0, p)
    assert t.place(0, 5, check=False)[0] == 2           # one file slot per page
    # p0 and p1 left L2 before any commit: written to their own slots then
    assert [t.locate(0, p) for p in range(5)] == [L3(0), L3(1), L2(0), 1, 0]
    assert t.stats() == dict(evictions=3, fetches=0, spills=2, reloads=0, prefetched=0, backups=2)
    t.commit()                          # the other three: p2 from L2, p3 and p4 from the pool
    assert t.stats()["backups"] == 5
    t.commit()                          # nothing left to write
    assert t.stats()["backups"] == 5
    # p0 back from its file slot (the copy stays there); p3 -> L2, and p2
    # leaves L2 for its own file slot without a write
    t.fetch([[0]])
    assert [t.locate(0, p) for p in range(5)] == [1, L3(1), L3(2), L2(0), 0]
    assert t.stats() == dict(evictions=4, fetches=1, spills=3, reloads=1, prefetched=0, backups=5)
    # drop every pool and host copy: each page in its own file slot only
    t.drop()
    assert [t.locate(0, p) for p in range(5)] == [L3(p) for p in range(5)]
    t.fetch([[3, 4]])                   # both restored from the file
    assert t.locate(0, 3) >= 0 and t.locate(0, 4) >= 0
    assert t.stats() == dict(evictions=4, fetches=3, spills=3, reloads=3, prefetched=0, backups=5)
    # without a host tier the pool's page goes straight to its file slot
    t2 = P.HsaTier(cfg, None, 0, num_slots=2, max_pages=10, l3_slots=3, backup=True)
    t2.place(0, 0), t2.place(0, 1), t2.place(0, 2)
    assert t2.locate(0, 0) == -2 and t2.stats()["backups"] == 1 and t2.stats()["spills"] == 1
    t2.fetch([[0, 2]])                  # p1 leaves for its slot, p0 comes back
    assert t2.locate(0, 1) == -3 and t2.stats()["backups"] == 2 and t2.stats()["reloads"] == 1
    # commit and drop need backup mode
    t3 = P.HsaTier(cfg, None, 2, num_slots=2, max_pages=10)
    assert t3.commit(check=False) == 1 and t3.drop(check=False) == 1
    t.close(), t2.close(), t3.close()


def test_tier_fetch_swaps_and_prefetch_reuses_the_slot_freed_first_plan_only():
    # a fetch swaps the page it brings from L2 with the page it displaces (one
    # host slot, in place); a prefetch copies the displaced page to the free
    # host slot freed longest ago, not the one its incoming page just left
    cfg = P.config(1, 2, 64, 256, "bf16")
    t = P.HsaTier(cfg, None, 4, num_slots=2, max_pages=10)
    for p in range(4):
        t.place(0, p)                   # p0 -> host 0, p1 -> host 1
    assert t.locate(0, 0) == -2 and t.locate(0, 1) == -3
    t.fetch([[0]])                      # p0 <-> p2: p2 takes host 0
    assert t.locate(0, 0) >= 0 and t.locate(0, 2) == -2
    t.prefetch([[1]])                   # p3 -> host 2 (free, never used); host 1 freed
    assert t.locate(0, 3) == -4
    t.prefetch([[2]])                   # p1 -> host 3 (never used), not host 1; host 0 freed
    assert t.locate(0, 1) == -5
    t.prefetch([[3]])                   # p2 -> host 1 (freed before host 0)
    assert t.locate(0, 2) == -3
    t.close()


def test_gate_tensors_are_checked_against_the_gate_shape():
    import torch
    from paper_2609_34606_amd import hsa as H
    head = P.config(2, 3, 64, 256, "bf16")
    elem = P.config(2, 3, 64, 256, "bf16", gate_dims=64)
    n_q = 5
    assert H._gate(head, None, n_q) is None
    assert H._gate(head, torch.zeros((2, n_q, 3)), n_q) is not None
    assert H._gate(elem, torch.zeros((2, n_q, 3, 64)), n_q) is not None
    for cfg, g in ((head, torch.zeros((2, n_q, 3, 64))), (elem, torch.zeros((2, n_q, 3))),
                   (head, torch.zeros((2, n_q + 1, 3))), (head, torch.zeros((2, n_q, 3), dtype=torch.float64))):
        with pytest.raises(ValueError):
            H._gate(cfg, g, n_q)


def test_query_and_output_tensors_are_checked_against_the_config():
    import torch
    from paper_2609_34606_amd import hsa as H
    cfg = P.config(2, 3, 64, 256, "bf16")
    bf = torch.bfloat16
    assert H._rows(cfg, torch.zeros((2, 5, 3, 64), dtype=bf), 5, "q") is not None
    for t in (torch.zeros((2, 6, 3, 64), dtype=bf), torch.zeros((2, 5, 3, 128), dtype=bf),
              torch.zeros((1, 5, 3, 64), dtype=bf)):
        with pytest.raises(ValueError):
            H._rows(cfg, t, 5, "q")
    # element type: the kernels read and write the config's dtype (twice the
    # bytes for fp32), so a mismatch is rejected before any pointer is passed
    with pytest.raises(ValueError):
        H._rows(cfg, torch.zeros((2, 5, 3, 64)), 5, "q")
    f32 = P.config(2, 3, 64, 256, "f32")
    assert H._rows(f32, torch.zeros((2, 5, 3, 64)), 5, "q") is not None
    with pytest.raises(ValueError):
        H._rows(f32, torch.zeros((2, 5, 3, 64), dtype=bf), 5, "o")
    # the sparse-branch output is fp32 under either config
    assert H._rows(cfg, torch.zeros((2, 5, 3, 64)), 5, "o_sp", fp32=True) is not None
    with pytest.raises(ValueError):
        H._rows(cfg, torch.zeros((2, 5, 3, 64), dtype=bf), 5, "o_sp", fp32=True)


def test_block_select_outputs_are_checked_for_size_and_type():
    import torch
    from paper_2609_34606_amd import hsa as H
    assert H._out(None, 10, "int32", "x") is None
    assert H._out(torch.zeros(10, dtype=torch.int32), 10, "int32", "x") is not None
    assert H._out(torch.zeros(12, dtype=torch.float64), 10, "float64", "x") is not None
    for t, dt in ((torch.zeros(9, dtype=torch.int32), "int32"), (torch.zeros(10), "float64"),
                  (torch.zeros(10, dtype=torch.int64), "int32")):
        with pytest.raises(ValueError):
            H._out(t, 10, dt, "x")


def test_pool_tensors_are_checked_against_the_config():
    import torch
    from paper_2609_34606_amd import hsa as H
    cfg = P.config(2, 3, 64, 16, "bf16")
    bf = torch.bfloat16
    k = torch.zeros((5, 3, 16, 64), dtype=bf)
    v = torch.zeros((5, 3, 64, 16), dtype=bf)
    pt = torch.zeros((2, 4), dtype=torch.int32)
    pool = H.kv_pool(k, v, pt, cfg)
    assert (pool.num_slots, pool.max_pages) == (5, 4)
    bad = [(k.float(), v, pt), (k, v.float(), pt), (k.transpose(2, 3).contiguous(), v, pt),
           (k, v.transpose(2, 3).contiguous(), pt), (k[:, :2].contiguous(), v, pt),
           (k, v, pt.long()), (k, v, pt[:1].contiguous())]
    for a, b, c in bad:
        with pytest.raises(ValueError):
            H.kv_pool(a, b, c, cfg)



def test_attention_planner_fits_its_chunk_table():
    # The planner's chunk table holds HSA_PLAN_MAX_CHUNKS entries. Long page
    # lists split heads into several key ranges and every (head, split) group
    # is cut into chunks of query tiles; with many heads the plan must still
    # fit (a coarser cut or fewer splits), for every head count the config
    # accepts, both walks and P = 1560 as well as short pages.
    lib = P.lib()
    n_items, n_chunks, widest = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    rng = __import__("numpy").random.default_rng(5)
    checked = 0
    for H_ in list(range(1, 65, 3)) + [17, 32, 63, 64]:
        for n_q in (1, 257, 2560, 4680, 20000):
            for lens in ((50,) * H_, tuple(int(x) for x in rng.integers(1, 120, H_)), (1,) * H_):
                for adaptive in (0, 1):
                    cfg = P.config(1, H_, 128, 1560 if adaptive == 0 else 512, "bf16")
                    arr = (ctypes.c_int32 * H_)(*lens)
                    st = lib.hsa_attention_plan(ctypes.byref(cfg), n_q, arr, adaptive,
                                                ctypes.byref(n_items), ctypes.byref(n_chunks),
                                                ctypes.byref(widest))
                    assert st == 0, (H_, n_q, lens[:3], adaptive, st)
                    if adaptive == 0 and n_items.value >= 1024:
                        # many items: one workgroup per whole item
                        assert n_chunks.value == n_items.value and widest.value == 1
                    else:
                        assert 1 <= n_chunks.value <= 256, (H_, n_q, n_chunks.value)
                    waves = 4 if adaptive else 8
                    assert n_items.value >= H_ * -(-n_q // (32 * waves))
                    # tile lists split a head's pages; the page walk's ranges
                    # cut an item (its list's 64-key tiles) into pieces
                    most = max(lens) * (1 if adaptive else -(-1560 // 64))
                    assert 1 <= widest.value <= most
                    checked += 1
    assert checked > 500
    cfg = P.config(1, 4, 128, 1560, "bf16")
    bad = (ctypes.c_int32 * 4)(3, 0, 3, 3)
    assert lib.hsa_attention_plan(ctypes.byref(cfg), 100, bad, 0, None, None, None) == 1


def _stream_k_segments(B, H, n_q, P, lens, G, whole=False):
    """The page walk's segments as its kernel derives them: the launch's
    tiles (items b, h, 256-query tile; max(1, lens[h]) x ceil(P / 64) tiles
    each) cut into G ranges (the first T % G of them one tile longer), or
    with whole, range i = item i; yields (range, item, first tile, end tile,
    rotation, item start)."""
    nqt, tpp = -(-n_q // 256), -(-P // 64)
    off = [0]
    for h in range(H):
        off.append(off[-1] + nqt * max(1, lens[h]) * tpp)
    per_b = off[H]
    T = B * per_b
    if whole:
        for i in range(B * H * nqt):
            b, rest = divmod(i, H * nqt)
            h, qt = divmod(rest, nqt)
            n = max(1, lens[h]) * tpp
            t0 = b * per_b + off[h] + qt * n
            yield i, (b, h, qt), 0, n, 0, t0
        return
    q, rm = divmod(T, G)
    start = lambda i: i * q + min(i, rm)
    range_of = lambda t: t // (q + 1) if t < rm * (q + 1) else rm + (t - rm * (q + 1)) // q
    for r in range(G):
        t, t_end = start(r), start(r + 1)
        while t < t_end:
            b = t // per_b
            tb = t - b * per_b
            h = 0
            while h + 1 < H and off[h + 1] <= tb:
                h += 1
            n = max(1, lens[h]) * tpp
            qt, a = divmod(tb - off[h], n)
            item0 = t - a
            e = min(n, t_end - item0)
            # rotation: the larger of the first two pieces (or the one piece)
            # runs in step with its range
            r0 = range_of(item0)
            s1 = start(r0 + 1)
            rs = s1
            if item0 + n <= s1 or (item0 + n <= start(r0 + 2) and s1 - item0 >= item0 + n - s1):
                rs = start(r0)
            yield r, (b, h, qt), a, e, (item0 - rs) % n, item0
            t = item0 + e


def _walked_keys(a, e, sigma, n, n_real):
    """Key tiles the kernel walks for the segment [a, e) of an item of n
    tiles rotated by sigma, with n_real real tiles: its count and start as the
    kernel computes them, then the tiles, wrapping at n_real."""
    length = e - a
    S = a + sigma if a + sigma < n else a + sigma - n
    c1 = max(0, min(S + length, n_real) - S)
    c2 = min(S + length - n, n_real) if S + length > n else 0
    k = S if c1 > 0 else 0
    keys = []
    for _ in range(c1 + c2):
        keys.append(k)
        k = k + 1 if k + 1 < n_real else 0
    return keys


def test_stream_k_ranges_cover_every_tile_once():
    # The page walk cuts the launch's tiles into the planner's ranges (one
    # workgroup each). Every tile must be walked exactly once; an item cut
    # into pieces must sit in consecutive ranges, only as a range's first or
    # last segment (its partial slot 0 or 1), with no two pieces sharing a
    # slot; the planner's widest cut must be the largest piece count. Each
    # item's rotated, wrapping walk must visit every key tile of its real
    # list (which may be shorter than the planned one) exactly once, and a
    # piece that is in step with its range must walk key tile = time.
    lib = P.lib()
    n_items, n_chunks, widest = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    rng = __import__("numpy").random.default_rng(9)
    cases = [(1, 12, 4680, 1560, None), (2, 64, 600, 64, None), (3, 5, 300, 96, None),
             (1, 17, 2560, 64, None), (4, 12, 4680, 1560, None), (1, 1, 1, 64, (1,)),
             (1, 3, 257, 64, (1, 1, 1)), (2, 7, 20000, 40, None), (1, 12, 4680, 1560, (7,) * 12),
             (1, 12, 4680, 1560, (4, 19, 11, 5, 5, 19, 5, 11, 11, 11, 7, 11)),
             (30, 12, 4680, 1560, (11,) * 12), (5, 12, 4680, 1560, None), (4, 12, 4680, 1560, (9,) * 12),
             (1, 12, 4680, 64, (5, 7, 11, 19, 5, 19, 5, 11, 11, 11, 7, 11)), (1, 3, 600, 64, (2, 9, 30))]
    for B, H_, n_q, page, lens in cases:
        lens = lens or tuple(int(x) for x in rng.integers(1, 120, H_))
        cfg = P.config(B, H_, 128, page, "bf16")
        arr = (ctypes.c_int32 * H_)(*lens)
        assert lib.hsa_attention_plan(ctypes.byref(cfg), n_q, arr, 0, ctypes.byref(n_items),
                                      ctypes.byref(n_chunks), ctypes.byref(widest)) == 0
        G = n_chunks.value
        items = B * n_items.value
        tpp = -(-page // 64)
        T = items // H_ * sum(max(1, x) * tpp for x in lens)
        g_sk = max(1, min(256, T // 16, 2 * items))
        if len(set(max(1, x) for x in lens)) == 1:
            k = -(-items // 256)
            if items % k == 0 and 8 * (items // k) >= 7 * 256:
                g_sk = items // k
        max_len = max(max(1, x) for x in lens) * tpp
        # one workgroup per whole item: many items, or few short ones
        whole = items >= 1024 or (items <= 256 and max_len <= T // g_sk + 4)
        if whole:
            assert G == B * n_items.value and widest.value == 1
        else:
            assert 1 <= G <= 256, G
        if len(set(max(1, x) for x in lens)) == 1 and 224 <= B * n_items.value <= 256:
            assert G == B * n_items.value and widest.value == 1  # whole items, none cut
        # workgroup w runs on XCD w % 8: each XCD's ranges are contiguous and
        # every range has one workgroup
        xcd_ranges = {}
        for w in range(G):
            x = w % 8
            xcd_ranges.setdefault(x, []).append(x * (G // 8) + min(x, G % 8) + w // 8)
        flat = [r for x in sorted(xcd_ranges) for r in xcd_ranges[x]]
        assert flat == list(range(G))
        segs = list(_stream_k_segments(B, H_, n_q, page, lens, G, whole))
        tpp = -(-page // 64)
        # real lists: the planned length, or fewer pages for some heads
        real = [max(0, x - int(rng.integers(0, 3))) if h % 2 else x for h, x in enumerate(lens)]
        range_start = {}
        for r, _, a, _, _, item0 in segs:
            range_start.setdefault(r, item0 + a)
        pieces, walked, keys, in_step = {}, 0, {}, set()
        for r, item, a, e, sigma, item0 in segs:
            assert 0 <= a < e
            walked += e - a
            pieces.setdefault(item, []).append((r, a, e))
            n = max(1, lens[item[1]]) * tpp
            ks = _walked_keys(a, e, sigma, n, real[item[1]] * tpp)
            keys.setdefault(item, []).extend(ks)
            if (a + sigma) % n == (item0 + a - range_start[r]) % n:
                in_step.add(item)
                if real[item[1]] == lens[item[1]]:
                    assert ks == [(item0 + v - range_start[r]) % n for v in range(a, e)]
        assert in_step == set(pieces)  # every item has a piece in step
        assert walked == B * n_items.value // H_ * sum(max(1, x) * tpp for x in lens)
        assert len(pieces) == B * n_items.value
        for item, ks in keys.items():
            assert sorted(ks) == list(range(real[item[1]] * tpp)), item
        first = {}
        last = {}
        for r, item, a, e, _, _ in segs:
            first.setdefault(r, item)
            last[r] = item
        slots = set()
        most = 1
        for item, ps in pieces.items():
            n = max(1, lens[item[1]]) * tpp
            assert ps[0][1] == 0 and ps[-1][2] == n
            assert all(x[2] == y[1] for x, y in zip(ps, ps[1:]))  # contiguous tiles
            assert [x[0] for x in ps] == list(range(ps[0][0], ps[0][0] + len(ps)))
            most = max(most, len(ps))
            if len(ps) == 1:
                continue
            for k, (r, a, e) in enumerate(ps):
                slot = 1 if k == 0 and a == 0 and first[r] != item else 0
                assert (first[r] == item) if slot == 0 else (last[r] == item)
                assert (r, slot) not in slots
                slots.add((r, slot))
        assert most == widest.value, (B, H_, n_q, page, most, widest.value)


def test_noalloc_rejects_calls_beyond_its_static_workspace():
    # host-side: the size check comes before any device call, so fake
    # non-NULL pointers are enough
    lib = P.lib()
    kh = (ctypes.c_int32 * 12)(*([16] * 12))
    small = P.config(1, 12, 128, 1560, "bf16")
    need = lib.hsa_forward_noalloc_bytes(ctypes.byref(small), 4680, 120, 3, kh, 16)
    assert 0 < need <= (128 << 20)
    big = P.config(8, 12, 128, 1560, "bf16")     # 8 x 60,000 queries: 184 MB of query sums
    need_big = lib.hsa_forward_noalloc_bytes(ctypes.byref(big), 60000, 120, 3, kh, 16)
    assert need_big > (128 << 20)
    pool = H.HsaKvPool(0x1000, 0x2000, 0x3000, 8 * 123, 123)
    st = lib.hsa_forward_noalloc(ctypes.byref(big), 0x4000, 60000, ctypes.byref(pool), 120, 3, kh, 16,
                                 0x5000, 0x6000, 0x7000, None, None, 0x8000, None, None)
    assert st == 4  # HSA_ERR_WORKSPACE
    st = lib.hsa_forward_noalloc(ctypes.byref(small), None, 4680, ctypes.byref(pool), 120, 3, kh, 16,
                                 0x5000, 0x6000, 0x7000, None, None, 0x8000, None, None)
    assert st == 1  # HSA_ERR_INVALID_ARG
