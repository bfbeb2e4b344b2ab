"""lirpa_bound_noalloc (the entry point for callers that cannot allocate device memory) against
lirpa_bound on the same inputs, through the C ABI: two calls in a row, the second with a smaller
batch, and a batch larger than the scratch array (run in chunks).  Results must be bitwise
identical: the same kernels run with a different workspace and chunking, and every reduction
has a fixed order."""
import numpy as np
import pytest
import torch

from oracle import ref
from paper_2011_13824_amd import lirpa
from paper_2011_13824_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lirpa.load()


def dev(a):
    return None if a is None else torch.as_tensor(np.ascontiguousarray(a)).cuda()


def outputs(B, S, n_relu):
    return (torch.empty((B, S), dtype=torch.float32, device="cuda"),
            torch.empty((B, n_relu), dtype=torch.float32, device="cuda"),
            torch.empty((B, n_relu), dtype=torch.float32, device="cuda"),
            torch.empty((B, n_relu), dtype=torch.int8, device="cuda"))


def both(net, w, split, alpha=None):
    B, S = split.shape[0], w.S
    x0, C, sp, al = dev(w.x0), dev(w.C), dev(split), dev(alpha)
    ref_out = outputs(B, S, net.n_relu)
    ws, ws_bytes = net.workspace(S, B, 0, 64 << 30)
    lirpa.lirpa_bound(net.handle, x0, w.eps, C, S, B, sp, al, *ref_out, ws, ws_bytes)
    got = outputs(B, S, net.n_relu)
    # poison the outputs: every entry must be written
    for t in got:
        t.fill_(-7)
    lirpa.lirpa_bound_noalloc(net.handle, x0, w.eps, C, S, B, sp, al, *got)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in ref_out], [t.cpu().numpy() for t in got]


@pytest.mark.parametrize("name,B2", [("base", 37), ("tiny", 5)])
def test_noalloc_matches_bound_twice(name, B2):
    w = wl.get(name)
    rnet = ref.RefNet(w.layers)
    split = w.splits(ref.root_unstable(rnet, w.x0, w.eps, w.C))
    net = lirpa.Network(w.layers)
    alpha = np.random.default_rng(2).uniform(0, 1, (w.B, w.n_relu)).astype(np.float32)
    for k, (sp, al) in enumerate(((split, None), (split[:B2], alpha[:B2]))):
        want, got = both(net, w, sp, al)
        print(f"{name} call {k + 1}: B = {sp.shape[0]}", flush=True)
        for nm, a, b in zip(("lb", "l", "u", "code"), want, got):
            assert np.array_equal(a, b), f"{name} call {k + 1}: {nm} differs"
        lr, *_ = ref.bound(rnet, w.x0, w.eps, w.C, sp, al)
        err = np.abs(got[0] - lr) - (1e-4 + 1e-4 * np.abs(lr))
        assert np.all(err <= 0), f"{name} call {k + 1}: lb off the oracle by {err.max():.3g}"


def test_noalloc_chunks_a_batch_beyond_the_scratch_array():
    w = wl.wide()
    rnet = ref.RefNet(w.layers)
    split = w.splits(ref.root_unstable(rnet, w.x0, w.eps, w.C))
    net = lirpa.Network(w.layers)
    need = lirpa.lirpa_workspace_bytes(net.handle, w.S, w.B, 0)
    assert need > 128 << 20, "the batch must not fit the scratch array"
    want, got = both(net, w, split)
    for nm, a, b in zip(("lb", "l", "u", "code"), want, got):
        assert np.array_equal(a, b), f"wide: {nm} differs"
    print(f"wide: B = {w.B}, {need / 2**20:.0f} MiB of workspace in chunks of the 128 MiB "
          f"scratch array, identical", flush=True)


def test_noalloc_rejects_a_sub_domain_beyond_the_scratch_array():
    # one Linear layer of 2^23 features: a single sub-domain's workspace exceeds 128 MiB
    layers = [wl.fc(4, 1 << 23), wl.fc(1 << 23, 1)]
    for t in layers:
        t["W"] = np.zeros(wl.weight_shape(t), np.float32)
        t["b"] = np.zeros(t["out_c"], np.float32)
    net = lirpa.Network(layers)
    lb = torch.empty((1, 1), dtype=torch.float32, device="cuda")
    with pytest.raises(lirpa.LirpaError) as ei:
        lirpa.lirpa_bound_noalloc(net.handle, dev(np.zeros(4, np.float32)), 0.1,
                                  dev(np.ones((1, 1), np.float32)), 1, 1, None, None, lb, None,
                                  None, None)
    assert ei.value.code == lirpa.LIRPA_ENOMEM and "128 MiB" in str(ei.value)
