"""Algorithmic work that bench.py charges to the reverse-sweep kernels (CPU only).

The stage figures of the benchmark line divide these counts by measured kernel time, so a count
that includes data the kernel never has to touch shows up as a rate above the hardware's.  The
counts below are derived by hand for the Wide net (Conv 3->16 and 16->32, k4 s2 p1 on 32x32,
FC 2048->100, FC 100->10; 2048 sub-domains, 9 specs).
"""
import os
import sys

import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import bench  # noqa: E402
from paper_2011_13824_amd import workloads as wl  # noqa: E402

N0, N1, N2, N3 = 3 * 32 * 32, 16 * 16 * 16, 32 * 8 * 8, 100
B, S = 2048, 9


@pytest.fixture(scope="module")
def layers():
    return wl.get("wide_opt").layers


def test_dense_counts_without_fractions(layers):
    work = bench.grad_work(layers, S, B)
    Q3, Q4 = B * 2 * N3, B * S
    # pass-3 gathers: 3 floats per neuron and group of 8 rows, plus 3 per (sub-domain, neuron)
    assert work["grad_gather[layer1,pass3]"][1] == pytest.approx(12.0 * N1 * Q3 / 8 + 12.0 * B * N1)
    # final-pass reduction: the tape and G entries of every row of every neuron
    assert work["grad_reduce[layer1,pass4]"][1] == pytest.approx(8.0 * N1 * Q4 + 12.0 * B * N1)
    # fused pass-3 forward: signs (1 byte per input), tape over g^(1), partial sums of both layers
    assert work["fwd12[layer1,pass3]"][1] == pytest.approx(
        N0 * Q3 + 4.0 * N1 * Q3 + 12.0 * (N1 + N2) * Q3 / 8)
    # its flops: both convolutions dense, 2 * MACs per row
    macs1, macs2 = N1 * 3 * 16, N2 * 16 * 16
    assert work["fwd12[layer1,pass3]"][0] == pytest.approx(2.0 * Q3 * (macs1 + macs2))


def test_unstable_fractions_scale_only_the_sparse_reads(layers):
    fr = [0.1, 0.25, 0.8]
    dense = bench.grad_work(layers, S, B, (0.25, 0.5))
    work = bench.grad_work(layers, S, B, (0.25, 0.5), fr)
    Q3, Q4 = B * 2 * N3, B * S
    nu1, nu2 = 0.1 * N1, 0.25 * N2
    assert work["grad_gather[layer1,pass3]"][1] == pytest.approx(12.0 * nu1 * Q3 / 8 + 12.0 * B * nu1)
    assert work["grad_gather[layer2,pass3]"][1] == pytest.approx(12.0 * nu2 * Q3 / 8 + 12.0 * B * nu2)
    # the final pass has R = 9 <= 64 rows per sub-domain: the segmented reduction skips stable rows
    assert work["grad_reduce[layer1,pass4]"][1] == pytest.approx(8.0 * nu1 * Q4 + 12.0 * B * nu1)
    # 32 channels on T_2: the fused forward writes the unstable neurons' sums only
    assert work["fwd12[layer1,pass3]"][1] == pytest.approx(
        N0 * Q3 + 4.0 * N1 * Q3 + 12.0 * (nu1 + nu2) * Q3 / 8)
    # T_2 flops at the unstable layer-2 neurons; the tiles computed are the executed work
    macs1, macs2 = N1 * 3 * 16, N2 * 16 * 16
    assert work["fwd12[layer1,pass3]"][0] == pytest.approx(2.0 * Q3 * (macs1 + 0.25 * macs2))
    assert work["executed"]["fwd12[layer1,pass3]"] == pytest.approx(2.0 * Q3 * (macs1 + 0.5 * macs2))
    # pass-2 gather: every layer-1 code, then for an unstable neuron the partials of the windows
    # covering it (4 row groups of 8 channels x 2 x 2 taps) and its gradient entry
    assert work["pass2_grad_gather[layer1,pass2]"][1] == pytest.approx(
        B * N1 * (1.0 + 0.1 * (4.0 * 16 + 8.0)))
    # the witness forwards themselves do not change
    for k in ("fwd[layer1,pass4]", "fwd[layer2,pass4]", "pass2_window_grad[layer1,pass2]"):
        assert work[k] == dense[k]


def test_pass_rows_above_the_segment_limit_read_every_neuron(layers):
    # pass 3 has R = 200 rows per sub-domain, so a reduction there is the per-neuron kernel,
    # which reads every neuron's rows
    work = bench.grad_work(layers, S, B, None, [0.1, 0.25, 0.8])
    Q3 = B * 2 * N3
    assert work["grad_reduce[layer1,pass3]"][1] == pytest.approx(8.0 * N1 * Q3 + 12.0 * B * 0.1 * N1)


def test_relax_params_reads_alpha_of_unstable_neurons_only(layers):
    # l, u (8), split (1), a_lo, a_up, b_up and the code (13) per neuron; alpha (4) only where
    # the neuron is unstable, since every other neuron's slope is fixed
    plain = bench.stage_work(layers, S, B)
    opt = bench.stage_work(layers, S, B, [0.1, 0.25, 0.8])
    assert plain["relax_params[layer1,pass1]"][1] == pytest.approx(22.0 * B * N1)
    assert opt["relax_params[layer1,pass1]"][1] == pytest.approx((22.0 + 0.4) * B * N1)
    assert opt["relax_params[layer2,pass2]"][1] == pytest.approx((22.0 + 1.0) * B * N2)
