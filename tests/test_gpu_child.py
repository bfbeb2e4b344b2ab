"""lirpa_bound_child (intermediate bounds intersected with the parent sub-domain's) against the
oracle's ref_bound_child: lb, l, u within the bound tolerance, stability codes byte for byte as in
the plain parity tests.  The parent bounds come from the oracle's own bound of the parent
sub-domains (the child's splits without its last one), given to both sides as the same fp32
arrays; they pass through every path that relaxes a layer (the relaxation-parameter kernel,
the receptive-field pass 2 and the fused pass-3 kernel)."""
import numpy as np
import pytest
import torch

from oracle import ref
from paper_2011_13824_amd import lirpa
from paper_2011_13824_amd import workloads as wl
from tests import helpers as H
from tests.test_gpu_parity import check, check_codes
from tests.test_oracle_parent import parent_child_cases

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lirpa.load()


def dev(a):
    return None if a is None else torch.as_tensor(np.ascontiguousarray(a)).cuda()


def problem(name):
    if name == "small":
        layers = wl.random_net(H.small_conv_arch(), 21)
        x0 = np.random.default_rng(21).uniform(0, 1, wl.n_in(layers[0])).astype(np.float32)
        return layers, x0, 0.05, wl.margin_spec(3, 2)
    w = wl.get(name)
    eps = 0.2 if name == "tiny" else w.eps
    return w.layers, w.x0, eps, w.C


@pytest.mark.parametrize("name", ["tiny", "small", "base", "wide", "deep"])
def test_bound_child_matches_oracle(name):
    layers, x0, eps, C = problem(name)
    B = 16 if name in ("tiny", "small") else 6
    rnet, parent, child = parent_child_cases(layers, x0, eps, C, B, 9)
    _, lp, up, _ = ref.bound(rnet, x0, eps, C, parent)
    lp, up = lp.astype(np.float32), up.astype(np.float32)
    alpha = np.random.default_rng(3).uniform(0, 1, (B, rnet.n_relu)).astype(np.float32)
    net = lirpa.Network(layers)
    for al in (None, alpha):
        lb, l, u, code = (t.cpu().numpy() for t in net.bound_child(
            dev(x0), eps, dev(C), dev(child), dev(al), dev(lp), dev(up)))
        lb, l, u = lb.astype(np.float64), l.astype(np.float64), u.astype(np.float64)
        lr, llr, ulr, cr = ref.bound_child(rnet, x0, eps, C, child, al, lp, up)
        tag = f"{name}{'' if al is None else '+alpha'} child"
        check(f"{tag} lb", lb, lr)
        check(f"{tag} l", l, llr)
        check(f"{tag} u", u, ulr)
        check_codes(f"{tag} codes", code, cr, l, u, llr, ulr, child)
        assert np.all(l >= lp) and np.all(u <= up), "intersected bounds outside the parent's"
        # the intersection changes the result (it is not a no-op on these cases)
        l0 = net.bound(dev(x0), eps, dev(C), dev(child), dev(al), want_lu=True)[1]
        print(f"{tag}: {int((l > l0.cpu().numpy() + 1e-7).sum())} lower bounds tightened",
              flush=True)
