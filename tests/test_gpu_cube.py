"""GPU parity of the page writer and of the head-adaptive path on pages
stored in cube order (App. "Block Sparse Attention", the flattening of
(C_t, C_h, C_w) cubes; Sec. 3.3 "Inter- and intra-chunk sparse granularity").

Pages are produced token-major in raster order (frame, row, column), as a
projection writes them, and appended with hsa_page_write. The pool must equal
the oracle's permutation of the same tokens bit for bit. The adaptive forward
at the paper's page geometry (8 latent frames of 30 x 52 tokens = 12,480,
history cubes (4, 8, 4), current cubes (4, 4, 4)) is then compared with the
oracle run on a pool the oracle permuted itself: selections and kept blocks
bit-exact, outputs within the bf16 bar."""
import numpy as np
import pytest

from oracle import hsa_blocks_oracle as BO
from oracle import hsa_cube_oracle as CO
from synth_inputs import bf16_bits_to_f32, f32_to_bf16_bits

from hsa_testlib import say

pytestmark = pytest.mark.gpu


def _round(x, dtype):
    x = x.astype(np.float32)
    return bf16_bits_to_f32(f32_to_bf16_bits(x)) if dtype == "bf16" else x


def _raster_pages(rng, n_pages, frames, Hh, Ww, heads, d, dtype, structured):
    """[n_pages * P, heads, d] keys and values in raster order; with
    `structured`, keys carry a vector per coarse spatio-temporal region, so
    that blocks of neighbouring tokens differ in their mean key."""
    P = frames * Hh * Ww
    k = rng.standard_normal((n_pages, frames, Hh, Ww, heads, d)).astype(np.float32) * 0.6
    if structured:
        reg = rng.standard_normal((n_pages, 2, 4, 4, heads, d)).astype(np.float32) * 1.2
        t = np.arange(frames) * 2 // frames
        hh = np.arange(Hh) * 4 // Hh
        ww = np.arange(Ww) * 4 // Ww
        k += reg[:, t][:, :, hh][:, :, :, ww]
    v = rng.standard_normal((n_pages, frames, Hh, Ww, heads, d)).astype(np.float32)
    return _round(k.reshape(n_pages * P, heads, d), dtype), _round(v.reshape(n_pages * P, heads, d), dtype)


def _host_pool(kr, vr, table, orders, P):
    """The oracle's pool: page p of the raster arrays, permuted by orders[p]."""
    n_pages, heads, d = len(orders), kr.shape[1], kr.shape[2]
    kp = np.zeros((n_pages, heads, P, d), np.float32)
    vp = np.zeros((n_pages, heads, d, P), np.float32)
    for p in range(n_pages):
        kk = CO.permute_page(kr[p * P:(p + 1) * P], orders[p])
        vv = CO.permute_page(vr[p * P:(p + 1) * P], orders[p])
        kp[table[p]] = np.transpose(kk, (1, 0, 2))
        vp[table[p]] = np.transpose(vv, (1, 2, 0))
    return kp, vp


def _write(cfg_args, kr, vr, table, n_hist, n_cur, orders_lib, dtype):
    import torch
    from paper_2609_34606_amd import HsaLayer, hsa_page_write
    B, heads, d, P = cfg_args
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    cuda = "cuda:0"
    n_pages = n_hist + n_cur
    layer = HsaLayer(B, heads, d, P, dt, cuda, num_slots=n_pages, max_pages=n_pages)
    layer.k_pool.fill_(float("nan"))
    layer.v_pool.fill_(float("nan"))
    layer.page_table.copy_(torch.from_numpy(table.astype(np.int32))[None])
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(cuda).to(dt)[None]
    for first, n, order in ((0, n_hist, orders_lib[0]), (n_hist, n_cur, orders_lib[1])):
        if n == 0:
            continue
        src = None if order is None else torch.from_numpy(order.astype(np.int32)).to(cuda)
        hsa_page_write(layer.cfg, layer.pool, t(kr[first * P:(first + n) * P]),
                       t(vr[first * P:(first + n) * P]), first, n, src_of=src)
    torch.cuda.synchronize()
    return layer


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("bf16", 64), ("f32", 128)])
@pytest.mark.parametrize("cube", [None, (4, 8, 4)])
def test_page_writer_is_the_oracle_permutation(dtype, d, cube):
    import paper_2609_34606_amd as P_
    frames, Hh, Ww, heads, n_pages = 2, 30, 52, 3, 3
    P = frames * Hh * Ww
    say(f"[case] page writer {dtype} d={d} cube={cube} P={P}")
    rng = np.random.default_rng(91)
    kr, vr = _raster_pages(rng, n_pages, frames, Hh, Ww, heads, d, dtype, False)
    table = rng.permutation(n_pages)
    lib_order = None if cube is None else P_.hsa_cube_order(frames, Hh, Ww, cube)[0]
    ref_order = np.arange(P) if cube is None else CO.cube_order(frames, Hh, Ww, *cube)[0]
    layer = _write((1, heads, d, P), kr, vr, table, n_pages, 0, (lib_order, None), dtype)
    kp, vp = _host_pool(kr, vr, table, [ref_order] * n_pages, P)
    np.testing.assert_array_equal(layer.k_pool.float().cpu().numpy(), kp)
    np.testing.assert_array_equal(layer.v_pool.float().cpu().numpy(), vp)


def test_adaptive_forward_on_cube_ordered_pages_paper_geometry():
    import torch
    import paper_2609_34606_amd as P_
    from test_gpu_adaptive import compare, run_library
    from synth_inputs.configs import Workload
    frames, Hh, Ww = 8, 30, 52
    P = frames * Hh * Ww                       # 12,480 tokens, the paper's page
    wl = Workload("cube_paper_geometry", batch=1, heads=2, head_dim=128, n_q=520, page_size=P,
                  n_cand=6, n_cur=1, k_h=(4, 3), dtype="bf16", seed=93, gates=True)
    say(f"[case] adaptive on cube-ordered pages {wl}")
    rng = np.random.default_rng(wl.seed)
    n_pages = wl.n_pages
    kr, vr = _raster_pages(rng, n_pages, frames, Hh, Ww, wl.heads, wl.head_dim, "bf16", True)
    table = rng.permutation(n_pages)
    hist_lib, whole_h = P_.hsa_cube_order(frames, Hh, Ww, (4, 8, 4))
    cur_lib, whole_c = P_.hsa_cube_order(frames, Hh, Ww, (4, 4, 4))
    assert (whole_h, whole_c) == (78 * 128, 182 * 64)
    layer = _write((1, wl.heads, wl.head_dim, P), kr, vr, table, wl.n_cand, wl.n_cur,
                   (hist_lib, cur_lib), "bf16")
    # queries near the mean key of one region of the newest history page
    q = rng.standard_normal((1, wl.n_q, wl.heads, wl.head_dim)).astype(np.float32) * 0.6
    q += kr[(wl.n_cand - 1) * P:(wl.n_cand - 1) * P + 4 * Hh * Ww].mean(0)[None, None] * 1.5
    q = _round(q, "bf16")
    g_lin = rng.standard_normal((1, wl.n_q, wl.heads)).astype(np.float32)
    g_sp = rng.standard_normal((1, wl.n_q, wl.heads)).astype(np.float32)
    cuda = "cuda:0"
    tt = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(cuda)
    dev = dict(q=tt(q).to(torch.bfloat16), k_pool=layer.k_pool, v_pool=layer.v_pool,
               page_table=layer.page_table, g_lin=tt(g_lin), g_sp=tt(g_sp))
    gpu = run_library(wl, dev, wl.k_h)
    hist_ref = CO.cube_order(frames, Hh, Ww, 4, 8, 4)[0]
    cur_ref = CO.cube_order(frames, Hh, Ww, 4, 4, 4)[0]
    kp, vp = _host_pool(kr, vr, table, [hist_ref] * wl.n_cand + [cur_ref] * wl.n_cur, P)
    qbs = [0, 3, 8]
    ref = BO.hsa_forward_adaptive(q, kp, vp, table[None], wl.n_cand, wl.n_cur, list(wl.k_h),
                                  g_lin=g_lin, g_sp=g_sp, query_blocks=qbs)
    fr = compare(gpu, ref, wl, wl.k_h, query_blocks=qbs)
    assert min(fr) < 1.0   # the selection keeps a subset of the blocks
