"""Upper bounds (Eq. 8: f_hi = max_x of the upper linear function U) and their optimisation
(Eq. 9) against the fp64 oracle: ub = -lb(-C) of the oracle's own lower bound (no separate
oracle arithmetic), with the bound tolerance 1e-4 abs + 1e-4 rel; soundness against points
sampled in the box: lb <= C f_s(x) <= ub."""
import numpy as np
import pytest
import torch

from oracle import ref
from paper_2011_13824_amd import lirpa
from paper_2011_13824_amd import workloads as wl
from tests import helpers as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lirpa.load()


def dev(a):
    return None if a is None else torch.as_tensor(np.ascontiguousarray(a)).cuda()


def check(name, got, want):
    excess = np.abs(got - want) - (1e-4 + 1e-4 * np.abs(want))
    print(f"{name}: max |gpu - oracle| = {np.abs(got - want).max():.3g}", flush=True)
    assert np.all(np.isfinite(got)) and np.all(excess <= 0), \
        f"{name}: exceeds tolerance by {excess.max():.3g}"


def cases():
    small = wl.random_net(H.small_conv_arch(), 21)
    x0s = np.random.default_rng(21).uniform(0, 1, wl.n_in(small[0])).astype(np.float32)
    return {"tiny": (wl.tiny(), None), "small": (None, (small, x0s, 0.05, wl.margin_spec(3, 2))),
            "base": (wl.base(), None), "wide": (wl.wide(), None)}


@pytest.mark.parametrize("name", ["tiny", "small", "base", "wide"])
def test_bound_ul_matches_oracle(name):
    w, raw = cases()[name]
    if w is not None:
        layers, x0, eps, C = w.layers, w.x0, w.eps, w.C
    else:
        layers, x0, eps, C = raw
    rnet = ref.RefNet(layers)
    B = 24
    split = wl.make_splits(B, rnet.n_relu, 8, 5, ref.root_unstable(rnet, x0, eps, C))
    alpha = np.random.default_rng(6).uniform(0, 1, (B, rnet.n_relu)).astype(np.float32)
    net = lirpa.Network(layers)
    for al in (None, alpha):
        lb, ub = net.bound_ul(dev(x0), eps, dev(C), dev(split), dev(al))
        lb, ub = lb.cpu().double().numpy(), ub.cpu().double().numpy()
        lr, *_ = ref.bound(rnet, x0, eps, C, split, al)
        ln, *_ = ref.bound(rnet, x0, eps, -C, split, al)
        tag = f"{name}{'' if al is None else '+alpha'}"
        check(f"{tag} lb", lb, lr)
        check(f"{tag} ub", ub, -ln)
        assert np.all(ub >= lb)
        # the lower side equals lirpa_bound's
        lb1 = net.bound(dev(x0), eps, dev(C), dev(split), dev(al)).cpu().double().numpy()
        check(f"{tag} lb vs lirpa_bound", lb, lb1)
    X = H.box_samples(x0, eps, 20000 if name in ("tiny", "small") else 1000,
                      np.random.default_rng(2))
    for b in range(0, B, 5):
        vals = H.torch_forward(layers, X, split[b]) @ C.T.astype(np.float64)
        assert np.all(lb[b] <= vals.min(0) + 1e-5) and np.all(vals.max(0) <= ub[b] + 1e-5), \
            f"{name}[{b}]: a sample outside [lb, ub]"


ADAM = {k: float(np.float32(x)) for k, x in
        (("lr", 0.1), ("beta1", 0.9), ("beta2", 0.999), ("eps_adam", 1e-8))}


def test_optimize_ul_sides():
    """Each side of lirpa_optimize_ul is lirpa_optimize on C (lower) and on -C (upper, negated),
    bit for bit; the oracle's own fresh-start trajectories agree within the bound tolerance."""
    w = wl.wide_opt()
    B, steps = 4, 3
    rnet = ref.RefNet(w.layers)
    split = w.splits(ref.root_unstable(rnet, w.x0, w.eps, w.C), B=B)
    net = lirpa.Network(w.layers)
    x0, C, sp = dev(w.x0), dev(w.C), dev(split)
    lb, ub, st = net.optimize_ul(x0, w.eps, C, sp, steps=steps, lr=ADAM["lr"])
    alpha = torch.empty((B, w.n_relu), dtype=torch.float32, device="cuda")
    lo = net.optimize(x0, w.eps, C, sp, alpha.clone(), steps=steps, lr=ADAM["lr"], fresh=True)
    up = net.optimize(x0, w.eps, -C, sp, alpha.clone(), steps=steps, lr=ADAM["lr"], fresh=True)
    assert torch.equal(lb, lo) and torch.equal(ub, -up)
    lb, ub = lb.cpu().double().numpy(), ub.cpu().double().numpy()
    for nm, spec, got, sgn in (("lower", w.C, lb, 1.0), ("upper", -w.C, ub, -1.0)):
        _, l, u, _ = ref.bound(rnet, w.x0, w.eps, spec, split)
        a0 = np.where((l < 0) & (u > 0), u / np.where(u - l > 0, u - l, 1),
                      np.where(l >= 0, 1.0, 0.0))
        r = ref.optimize(rnet, w.x0, w.eps, spec, split, a0, steps, **ADAM)
        check(f"optimised {nm}", got, sgn * r["lb_best"])
    h_lb, h_ub = net.bound_ul(x0, w.eps, C, sp)
    assert np.all(lb >= h_lb.cpu().double().numpy() - 1e-6)
    assert np.all(ub <= h_ub.cpu().double().numpy() + 1e-6)
    assert (ub < h_ub.cpu().double().numpy()).any(), "the upper side did not improve"


def test_optimize_ul_tiny_sound_and_tighter():
    w = wl.tiny()
    rnet = ref.RefNet(w.layers)
    split = w.splits(ref.root_unstable(rnet, w.x0, w.eps, w.C))
    net = lirpa.Network(w.layers)
    x0, C, sp = dev(w.x0), dev(w.C), dev(split)
    h_lb, h_ub = (t.cpu().double().numpy() for t in net.bound_ul(x0, w.eps, C, sp))
    lb, ub, st = net.optimize_ul(x0, w.eps, C, sp, steps=20)
    # resume: 10 more steps from the returned state never loosen the best bounds much
    lb2, ub2, _ = net.optimize_ul(x0, w.eps, C, sp, steps=10, state=st)
    lb, ub = lb.cpu().double().numpy(), ub.cpu().double().numpy()
    assert np.all(lb >= h_lb - 1e-6) and np.all(ub <= h_ub + 1e-6)
    assert lb.sum() > h_lb.sum() and ub.sum() < h_ub.sum()
    X = H.box_samples(w.x0, w.eps, 50000, np.random.default_rng(4))
    for b in range(w.B):
        vals = H.torch_forward(w.layers, X, split[b]) @ w.C.T.astype(np.float64)
        assert lb[b, 0] <= vals.min() + 1e-5 and vals.max() <= ub[b, 0] + 1e-5
        assert lb2[b, 0].item() <= vals.min() + 1e-5 and vals.max() <= ub2[b, 0].item() + 1e-5
