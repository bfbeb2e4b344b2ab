"""Pins of the oracle's branch and bound (Algorithm 1 without LP) against what the paper and
brute force fix: the App. A.1 counter-example (pure LiRPA BaB ends with the global lower bound
-1 and cannot verify), a 1-D net whose violation is found by the upper bound f_hi < 0 of
Algorithm 1's loop condition, properties that need branching to be verified (soundness against
sampled minima), and the branching rule on a hand case."""
import json
import os

import numpy as np

from oracle import bab, ref
from paper_2011_13824_amd import workloads as wl
from tests import helpers as H

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def app_a1():
    g = json.load(open(os.path.join(GOLDEN, "app_a1_counterexample.json")))
    layers = [dict(wl.fc(1, 2), W=np.array(g["W1"], np.float32), b=np.array(g["b1"], np.float32)),
              dict(wl.fc(2, 1), W=np.array(g["W2"], np.float32), b=np.array(g["b2"], np.float32))]
    return layers, np.array(g["x0"], np.float32), g["eps"]


def test_app_a1_pure_lirpa_bab_reports_minus_one():
    """App. A.1: after splitting h1 and h2, sub-domains (1) and (2) are verified (range [0,0])
    and (3), (4) keep the range [-1, 1] with no neuron left to split: the global lower bound
    is -1 and the property (true: f = 0) cannot be verified without LP."""
    layers, x0, eps = app_a1()
    r = bab.bab(ref.RefNet(layers), x0, eps, np.array([1.0], np.float32), 8, 100, 10)
    assert r["status"] == bab.UNKNOWN_STUCK
    assert r["f_lo"] == -1.0 and r["f_hi"] == 1.0
    assert (r["iterations"], r["domains_bounded"], r["domains_left"]) == (2, 7, 2)


def test_branching_rule_hand_case():
    l = np.array([-1.0, -2.0, 1.0, -3.0])
    u = np.array([1.0, 1.0, 2.0, 3.0])
    code = np.array([5, 5, 4, 1])  # the last is split: never chosen
    # intercepts -l u / (u - l): 0.5, 2/3, (active), (split)
    assert bab.branch_neuron(l, u, code) == 1
    assert bab.branch_neuron(np.array([-1.0, -1.0]), np.array([1.0, 1.0]), [5, 5]) == 0  # tie
    assert bab.branch_neuron(l, u, np.array([4, 3, 4, 2])) == -1


def test_violation_found_by_upper_bound():
    """f(x) = ReLU(x) + ReLU(-x) - 1/2 on [-1, 1]: min f = -1/2 at x = 0.  After h1 and h2 are
    split active together, f_s = -1/2 on the box and its upper bound -1/2 < 0 ends the loop."""
    layers = [dict(wl.fc(1, 2), W=np.array([[1.0], [-1.0]], np.float32), b=np.zeros(2, np.float32)),
              dict(wl.fc(2, 1), W=np.array([[1.0, 1.0]], np.float32),
                   b=np.array([-0.5], np.float32))]
    r = bab.bab(ref.RefNet(layers), np.zeros(1, np.float32), 1.0, np.array([1.0], np.float32),
                8, 100, 10)
    assert r["status"] == bab.VIOLATED and r["f_hi"] == -0.5 and r["iterations"] == 2
    X = np.linspace(-1, 1, 2001)[:, None]
    assert H.torch_forward(layers, X).min() == -0.5


def random_net_case(seed):
    layers = wl.random_net([wl.fc(2, 8), wl.fc(8, 8), wl.fc(8, 1)], seed)
    x0 = np.random.default_rng(seed).uniform(-1, 1, 2).astype(np.float32)
    return layers, x0


def test_verified_after_branching_is_sound():
    for seed, eps, c, iters in ((55, 0.4, -1.0, 2), (28, 0.2, -1.0, 1), (40, 0.2, 1.0, 1)):
        layers, x0 = random_net_case(seed)
        net = ref.RefNet(layers)
        cs = np.array([c], np.float32)
        root, *_ = ref.bound(net, x0, eps, cs[None], B=1)
        assert root[0, 0] < 0, "the root alone must not verify it"
        r = bab.bab(net, x0, eps, cs, 1024, 4000, 30)
        assert r["status"] == bab.VERIFIED and r["iterations"] == iters
        X = H.box_samples(x0, eps, 100000, np.random.default_rng(seed))
        vals = c * H.torch_forward(layers, X)[:, 0]
        assert 0 <= r["f_lo"] <= vals.min(), (seed, r["f_lo"], vals.min())
        # with optimised slopes the verdict is the same and still sound
        r2 = bab.bab(net, x0, eps, cs, 1024, 4000, 30, root_steps=20, steps=5)
        assert r2["status"] == bab.VERIFIED and 0 <= r2["f_lo"] <= vals.min()


def test_tiny_violation_is_real():
    w = wl.tiny()
    c = np.array([-1.0, 1.0], np.float32)
    r = bab.bab(ref.RefNet(w.layers), w.x0, 0.2, c, 1024, 4000, 30)
    assert r["status"] == bab.VIOLATED and r["iterations"] > 0
    X = H.box_samples(w.x0, 0.2, 100000, np.random.default_rng(1))
    assert (H.torch_forward(w.layers, X) @ c.astype(np.float64)).min() < 0
