"""Pins for oracle.gather: marker blocks make every copy traceable."""
import numpy as np

from oracle.gather import kv_gather


def _marked(layers, blocks, elems, base):
    # every element of block b in layer l of a plane holds base + 1000*l + b
    a = np.empty((layers, blocks, elems), dtype=np.int64)
    for l in range(layers):
        for b in range(blocks):
            a[l, b] = base + 1000 * l + b
    return a


def test_markers_follow_the_plan():
    layers, nsrc, ndst, elems = 3, 7, 11, 32
    sk, sv = _marked(layers, nsrc, elems, 10**6), _marked(layers, nsrc, elems, 2 * 10**6)
    dk, dv = _marked(layers, ndst, elems, 3 * 10**6), _marked(layers, ndst, elems, 4 * 10**6)
    src = np.array([4, 0, 6, 2])
    dst = np.array([9, 1, 3, 10])
    ok, ov = kv_gather(sk, sv, dk, dv, src, dst, layer0=1, n_layers=2)
    for l in range(layers):
        for b in range(ndst):
            if l in (1, 2) and b in dst:
                s = src[list(dst).index(b)]
                assert np.all(ok[l, b] == 10**6 + 1000 * l + s)     # K from K, same layer
                assert np.all(ov[l, b] == 2 * 10**6 + 1000 * l + s)  # V from V
            else:                                                   # untouched canary
                assert np.all(ok[l, b] == 3 * 10**6 + 1000 * l + b)
                assert np.all(ov[l, b] == 4 * 10**6 + 1000 * l + b)
    # inputs are not modified
    assert np.all(dk == _marked(layers, ndst, elems, 3 * 10**6))


def test_empty_plan_is_identity():
    d = np.arange(2 * 5 * 4).reshape(2, 5, 4)
    ok, ov = kv_gather(d, d, d, d + 1, np.zeros(0, int), np.zeros(0, int))
    assert np.array_equal(ok, d) and np.array_equal(ov, d + 1)


def test_round_trip_restores_staging():
    rng = np.random.default_rng(0)
    layers, nsrc, ndst, elems = 2, 6, 9, 16
    sk = rng.integers(0, 2**16, (layers, nsrc, elems))
    sv = rng.integers(0, 2**16, (layers, nsrc, elems))
    dk = rng.integers(0, 2**16, (layers, ndst, elems))
    dv = rng.integers(0, 2**16, (layers, ndst, elems))
    src = rng.permutation(nsrc)
    dst = rng.permutation(ndst)[:nsrc]
    pk, pv = kv_gather(sk, sv, dk, dv, src, dst)
    bk, bv = kv_gather(pk, pv, np.zeros_like(sk), np.zeros_like(sv), dst, src)
    assert np.array_equal(bk, sk) and np.array_equal(bv, sv)
