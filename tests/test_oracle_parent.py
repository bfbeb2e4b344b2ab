"""Pins of the oracle's intersection of a sub-domain's intermediate bounds with its parent's
(a reading where the paper is silent: a parent's bounds hold on its children, which are subsets
of it).  Checked against what does not come from the oracle: loose parents and a parent equal to
the child's own bounds change nothing; the intersected bounds never exceed the parent's; and the
bounds are sound on the child sub-domain itself -- on sampled points of the box that satisfy the
child's split constraints on the real network, every pre-activation lies in [l, u] and the
output is above lb."""
import numpy as np

from oracle import ref
from paper_2011_13824_amd import workloads as wl
from tests import helpers as H


def test_loose_and_own_parents_change_nothing():
    w = wl.tiny()
    net = ref.RefNet(w.layers)
    split = w.splits(ref.root_unstable(net, w.x0, w.eps, w.C))
    lb, l, u, code = ref.bound(net, w.x0, w.eps, w.C, split)
    big = np.full(l.shape, 1e30, np.float32)
    got = ref.bound_child(net, w.x0, w.eps, w.C, split, None, -big, big)
    for a, b in zip(got, (lb, l, u, code)):
        assert np.array_equal(a, b)
    # own bounds as the parent's (rounded to fp32 outward, so that they contain the fp64 ones)
    lp = np.nextafter(l.astype(np.float32), np.float32(-np.inf))
    up = np.nextafter(u.astype(np.float32), np.float32(np.inf))
    lp = np.where(lp.astype(np.float64) <= l, lp, np.nextafter(lp, np.float32(-np.inf)))
    up = np.where(up.astype(np.float64) >= u, up, np.nextafter(up, np.float32(np.inf)))
    got = ref.bound_child(net, w.x0, w.eps, w.C, split, None, lp, up)
    for a, b in zip(got, (lb, l, u, code)):
        assert np.array_equal(a, b)


def parent_child_cases(layers, x0, eps, C, nsub, seed):
    """Sub-domains with 1-3 splits drawn from the root-unstable neurons, and their parents (the
    same splits without the last one)."""
    net = ref.RefNet(layers)
    cand = ref.root_unstable(net, x0, eps, C)
    rng = np.random.default_rng(seed)
    child = np.zeros((nsub, net.n_relu), np.int8)
    parent = np.zeros_like(child)
    for b in range(nsub):
        idx = rng.choice(cand, size=int(rng.integers(1, 4)), replace=False)
        sg = rng.choice(np.array([-1, 1], np.int8), size=idx.size)
        child[b, idx] = sg
        parent[b, idx[:-1]] = sg[:-1]
    return net, parent, child


def test_intersected_bounds_are_sound_on_the_child():
    w = wl.tiny()
    eps = 0.2
    net, parent, child = parent_child_cases(w.layers, w.x0, eps, w.C, 16, 4)
    _, lp, up, _ = ref.bound(net, w.x0, eps, w.C, parent)
    lb, l, u, code = ref.bound_child(net, w.x0, eps, w.C, child, None, lp, up)
    lb0, l0, u0, _ = ref.bound(net, w.x0, eps, w.C, child)
    assert np.all(l >= lp.astype(np.float32) - 1e-12) and np.all(u <= up.astype(np.float32) + 1e-12)
    assert (l > l0 + 1e-9).any() or (u < u0 - 1e-9).any(), "the intersection must bite somewhere"
    X = H.box_samples(w.x0, eps, 200000, np.random.default_rng(0))
    out, pre = H.torch_forward(w.layers, X, return_pre=True)
    checked = 0
    for b in range(child.shape[0]):
        ok = np.ones(X.shape[0], bool)
        for j in np.flatnonzero(child[b]):
            ok &= (pre[:, j] >= 0) if child[b, j] > 0 else (pre[:, j] < 0)
        if ok.sum() < 100:
            continue
        checked += 1
        P = pre[ok]
        assert np.all(P >= l[b] - 1e-9) and np.all(P <= u[b] + 1e-9), f"sub-domain {b}: l, u"
        assert lb[b, 0] <= (out[ok] @ w.C[0].astype(np.float64)).min() + 1e-9, f"sub-domain {b}"
    assert checked >= 8, checked


def test_intersected_bounds_are_sound_on_a_conv_child():
    layers = wl.random_net(H.small_conv_arch(), 21)
    x0 = np.random.default_rng(21).uniform(0, 1, wl.n_in(layers[0])).astype(np.float32)
    C = wl.margin_spec(3, 2)
    eps = 0.05
    net, parent, child = parent_child_cases(layers, x0, eps, C, 12, 5)
    _, lp, up, _ = ref.bound(net, x0, eps, C, parent)
    lb, l, u, _ = ref.bound_child(net, x0, eps, C, child, None, lp, up)
    X = H.box_samples(x0, eps, 50000, np.random.default_rng(1))
    out, pre = H.torch_forward(layers, X, return_pre=True)
    checked = 0
    for b in range(child.shape[0]):
        ok = np.ones(X.shape[0], bool)
        for j in np.flatnonzero(child[b]):
            ok &= (pre[:, j] >= 0) if child[b, j] > 0 else (pre[:, j] < 0)
        if ok.sum() < 50:
            continue
        checked += 1
        assert np.all(pre[ok] >= l[b] - 1e-9) and np.all(pre[ok] <= u[b] + 1e-9)
        assert np.all(lb[b] <= (out[ok] @ C.T.astype(np.float64)).min(0) + 1e-9)
    assert checked >= 6, checked
