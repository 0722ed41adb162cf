"""Pins of the cube token order (oracle/hsa_cube_oracle.py) by properties the
paper states for it, not by its formula: the order is a permutation; every
run of B stored tokens of the whole-cube prefix is exactly one aligned
(C_t, C_h, C_w) box, with its tokens in (t, h, w) order and the boxes in
cube order; the truncated cubes follow, each contiguous. And the library's
host-side table (hsa_cube_order) equals the oracle's."""
import numpy as np
import pytest

from oracle import hsa_cube_oracle as CO

SHAPES = [(8, 32, 52, (4, 8, 4)), (8, 30, 52, (4, 8, 4)), (8, 30, 52, (4, 4, 4)),
          (3, 30, 52, (4, 4, 4)), (1, 30, 52, (4, 8, 4)), (4, 8, 8, (2, 4, 4)), (5, 7, 9, (2, 3, 4))]


def _coords(src, H, W):
    return src // (H * W), (src // W) % H, src % W


@pytest.mark.parametrize("T,H,W,cube", SHAPES)
def test_order_is_a_permutation(T, H, W, cube):
    src, whole = CO.cube_order(T, H, W, *cube)
    assert np.array_equal(np.sort(src), np.arange(T * H * W))
    B = cube[0] * cube[1] * cube[2]
    assert whole % B == 0 and whole == (T // cube[0]) * (H // cube[1]) * (W // cube[2]) * B


@pytest.mark.parametrize("T,H,W,cube", SHAPES)
def test_every_run_of_b_tokens_in_the_prefix_is_one_cube(T, H, W, cube):
    ct, ch, cw = cube
    B = ct * ch * cw
    src, whole = CO.cube_order(T, H, W, *cube)
    t, h, w = _coords(src, H, W)
    prev = None
    for r in range(whole // B):
        sl = slice(r * B, (r + 1) * B)
        tt, hh, ww = t[sl], h[sl], w[sl]
        # an aligned box of the cube's extents
        assert tt.min() % ct == 0 and hh.min() % ch == 0 and ww.min() % cw == 0
        assert (tt.max() - tt.min(), hh.max() - hh.min(), ww.max() - ww.min()) == (ct - 1, ch - 1, cw - 1)
        assert len(set(src[sl].tolist())) == B
        # inside the cube: (t, h, w) order, i.e. increasing raster index
        assert (np.diff(src[sl]) > 0).all()
        # cubes in order of (cube t, cube h, cube w)
        cur = (tt.min() // ct, hh.min() // ch, ww.min() // cw)
        assert prev is None or cur > prev
        prev = cur


@pytest.mark.parametrize("T,H,W,cube", SHAPES)
def test_truncated_cubes_follow_each_contiguous(T, H, W, cube):
    ct, ch, cw = cube
    src, whole = CO.cube_order(T, H, W, *cube)
    t, h, w = _coords(src[whole:], H, W)
    cid = [(a // ct, b // ch, c // cw) for a, b, c in zip(t, h, w)]
    # every token here lies outside the whole-cube region
    assert all(a >= T // ct or b >= H // ch or c >= W // cw for a, b, c in cid)
    # cube ids non-decreasing (each truncated cube contiguous, in cube order)
    assert all(x <= y for x, y in zip(cid, cid[1:]))
    for k in set(cid):
        idx = [i for i, c in enumerate(cid) if c == k]
        assert idx == list(range(idx[0], idx[-1] + 1))
        assert (np.diff(src[whole:][idx]) > 0).all()


def test_divisible_latent_has_no_truncated_cube_and_paper_block_count():
    # 8 frames of 32 x 52 tokens with the history cube (4, 8, 4): 2 x 4 x 13
    # cubes of 128 tokens
    src, whole = CO.cube_order(8, 32, 52, 4, 8, 4)
    assert whole == 8 * 32 * 52 == 104 * 128


def test_library_table_equals_the_oracle():
    import paper_2609_34606_amd as P
    for T, H, W, cube in SHAPES:
        got, whole = P.hsa_cube_order(T, H, W, cube)
        ref, rwhole = CO.cube_order(T, H, W, *cube)
        assert whole == rwhole
        np.testing.assert_array_equal(got, ref)
