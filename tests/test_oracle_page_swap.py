"""Pins of the page-swap oracle (CPU): a hand-worked case, round trips and
invariants that a slip in the copy (wrong block, wrong direction, a dropped
scale, a partial block) would break."""
import numpy as np
import pytest

import oracle


def _pool(n, hkv=2, p=4, d=8, seed=0, dtype=np.uint16):
    g = np.random.default_rng(seed)
    return g.integers(0, 1 << (8 * np.dtype(dtype).itemsize), size=(n, hkv, p, d)).astype(dtype)


def test_hand_worked_case():
    # pool pages hold their own id everywhere; host blocks start at -1
    k = np.arange(5, dtype=np.int32)[:, None, None, None] * np.ones((5, 1, 2, 3), np.int32)
    v = 10 + k
    hk = -np.ones((3, 1, 2, 3), np.int32)
    hv = hk.copy()
    out_k, out_v, _, _ = oracle.swap_out(k, v, None, None, [4, 1], hk, hv, None, None, [2, 0])
    assert out_k[:, 0, 0, 0].tolist() == [1, -1, 4]
    assert out_v[:, 0, 0, 0].tolist() == [11, -1, 14]
    # back into pages 0 and 3 of a zeroed pool
    z = np.zeros_like(k)
    nk, nv, _, _ = oracle.swap_in(out_k, out_v, None, None, [0, 2], z, z, None, None, [3, 0])
    assert nk[:, 0, 0, 0].tolist() == [4, 0, 0, 1, 0]
    assert nv[:, 0, 0, 0].tolist() == [14, 0, 0, 11, 0]
    assert (k[:, 0, 0, 0] == np.arange(5)).all()  # inputs untouched


@pytest.mark.parametrize("dtype", [np.uint16, np.uint8])
def test_round_trip_restores_the_pool(dtype):
    k, v = _pool(40, dtype=dtype, seed=1), _pool(40, dtype=dtype, seed=2)
    ks = np.random.default_rng(3).random((40, 2)).astype(np.float32)
    vs = np.random.default_rng(4).random((40, 2)).astype(np.float32)
    pages = [7, 31, 0, 12, 39]
    host = [3, 0, 4, 1, 2]
    hk, hv = np.zeros((5, 2, 4, 8), dtype), np.zeros((5, 2, 4, 8), dtype)
    hks, hvs = np.zeros((5, 2), np.float32), np.zeros((5, 2), np.float32)
    hk, hv, hks, hvs = oracle.swap_out(k, v, ks, vs, pages, hk, hv, hks, hvs, host)
    # every listed page landed whole in its host block, scales included
    for p_, h_ in zip(pages, host):
        assert (hk[h_] == k[p_]).all() and (hv[h_] == v[p_]).all()
        assert (hks[h_] == ks[p_]).all() and (hvs[h_] == vs[p_]).all()
    # clobber the pages, swap back: the pool is restored bit for bit
    k2, v2, ks2, vs2 = k.copy(), v.copy(), ks.copy(), vs.copy()
    for p_ in pages:
        k2[p_] = 0; v2[p_] = 0; ks2[p_] = 0; vs2[p_] = 0
    rk, rv, rks, rvs = oracle.swap_in(hk, hv, hks, hvs, host, k2, v2, ks2, vs2, pages)
    assert (rk == k).all() and (rv == v).all() and (rks == ks).all() and (rvs == vs).all()


def test_swap_in_to_other_pages_moves_exactly_those_pages():
    k, v = _pool(20, seed=5), _pool(20, seed=6)
    pages, host = [2, 5, 9], [0, 1, 2]
    hk, hv, _, _ = oracle.swap_out(k, v, None, None, pages, np.zeros((3, 2, 4, 8), np.uint16),
                                   np.zeros((3, 2, 4, 8), np.uint16), None, None, host)
    new_pages = [11, 3, 17]
    nk, nv, _, _ = oracle.swap_in(hk, hv, None, None, host, k, v, None, None, new_pages)
    for old, new in zip(pages, new_pages):
        assert (nk[new] == k[old]).all() and (nv[new] == v[old]).all()
    untouched = [i for i in range(20) if i not in new_pages]
    assert (nk[untouched] == k[untouched]).all() and (nv[untouched] == v[untouched]).all()


def test_repeated_sources_are_fine_repeated_destinations_are_not():
    k, v = _pool(6, seed=7), _pool(6, seed=8)
    hk = np.zeros((2, 2, 4, 8), np.uint16)
    out_k, _, _, _ = oracle.swap_out(k, v, None, None, [3, 3], hk, hk, None, None, [0, 1])
    assert (out_k[0] == k[3]).all() and (out_k[1] == k[3]).all()
    with pytest.raises(ValueError):
        oracle.swap_out(k, v, None, None, [1, 2], hk, hk, None, None, [0, 0])
    with pytest.raises(ValueError):
        oracle.swap_out(k, v, None, None, [6], hk, hk, None, None, [0])
