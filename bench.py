#!/usr/bin/env python
"""Throughput of batched LiRPA sub-domain bounds on one MI355X.

Default workload: alpha-optimised bounds of the wide conv net Conv(3->16, k4 s2 p1)-Conv(16->32,
k4 s2 p1)-FC(2048->100)-FC(100->10) on 3x32x32 inputs, 2048 sub-domains with up to 16 splits
each, 9 margin specs.  One step = one lirpa_optimize call over the whole batch: a heuristic bound
pass, then 20 projected Adam steps on the lower slopes (each a bound with every intermediate
pass recomputed under the sub-domain's splits and its gradient through those bounds), the best
bound of the 21 iterates kept.  --workload picks the plain-bound workloads instead (one step =
one lirpa_bound call: layer-1 bounds, every intermediate pass and the final pass).  Inputs are
synthetic and resident in HBM before the timed region.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "subdomain lower bounds/sec (batched LiRPA) + % MFMA / HBM roofline"
PEAK_FP32_TFLOPS = 157.3   # MI355X dense fp32 (MFMA)
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E


def stage_work(layers, S, B, fr=None):
    """Algorithmic work of one step per kernel class: {class: (flop, bytes)}.

    A backward stage through layer m carries Q = B*R rows (R = 2 n_k for pass k, S for the final
    pass).  Its flops are 2 * Q * MACs(T_m) with MACs(T_m) = n_out * in_c * k^2 for a conv
    (every kernel tap, the dense count of the forward convolution) and out_c * in_c for a
    linear layer.  Its bytes are the fp32 slab it reads ([n_m, Q]) plus, for a relaxing stage,
    the slab it writes ([n_{m-1}, Q]); a concretising stage writes Q floats.  The pass
    initialisation writes its relaxed [n_{k-1}, Q] slab."""
    from paper_2011_13824_amd import workloads as wl
    L = len(layers)
    n = [wl.n_in(layers[0])] + [wl.n_out(t) for t in layers]

    def macs(t):
        if t["kind"] == wl.CONV:
            return wl.n_out(t) * t["in_c"] * t["k"] * t["k"]
        return t["out_c"] * t["in_c"]

    work = {}

    def add(cls, flop, byt):
        f, b = work.get(cls, (0.0, 0.0))
        work[cls] = (f + flop, b + byt)

    if L >= 3 and layers[0]["kind"] == wl.CONV and layers[1]["kind"] == wl.CONV:
        # pass 2 restricted to each row's receptive field (launched instead of the dense pass
        # when the library has a kernel for the shapes): a row +-e_j of h^(2) carries the
        # C1 x K2 x K2 window of W_2 through the relaxation of layer 1 and T_1^T, each window
        # entry reaching in_c x K1 x K1 inputs.  Bytes: the layer-1 relaxation parameters read
        # (3 floats per neuron) and l, u of layer 2 written.
        t1, t2 = layers[0], layers[1]
        Q2 = B * 2 * n[2]
        wmacs = t1["out_c"] * t2["k"] ** 2 * t1["in_c"] * t1["k"] ** 2
        add("pass2_window[layer1,pass2]", 2.0 * Q2 * wmacs, 4.0 * (3 * B * n[1] + Q2))
    if L >= 4 and all(layers[i]["kind"] == wl.CONV for i in (0, 1, 2)) \
            and layers[1]["stride"] == 1 and layers[2]["stride"] == 1:
        # pass 3 restricted to receptive fields: each of the C2 x K3 x K3 entries of a row's
        # window on g^(2) reaches C1 x K2 x K2 entries of g^(1), and each of the C1 x W1 x W1
        # entries of the g^(1) window (W1 = K3 + K2 - 1) reaches in_c x K1 x K1 inputs
        t1, t2, t3 = layers[0], layers[1], layers[2]
        Q3 = B * 2 * n[3]
        w1 = t3["k"] + t2["k"] - 1
        wmacs = (t2["out_c"] * t3["k"] ** 2 * t1["out_c"] * t2["k"] ** 2
                 + t1["out_c"] * w1 * w1 * t1["in_c"] * t1["k"] ** 2)
        add("pass3_window[layer1,pass3]", 2.0 * Q3 * wmacs,
            4.0 * (3 * B * (n[1] + n[2]) + Q3))
    if L >= 5 and all(layers[i]["kind"] == wl.CONV for i in (0, 1, 2, 3)) \
            and layers[1]["stride"] == 1 and layers[2]["stride"] == 1:
        # pass 4 restricted to receptive fields: the C3 x K4 x K4 entries of a row's window on
        # g^(3) each reach C2 x K3 x K3 entries of g^(2); the C2 x W2 x W2 entries of that window
        # (W2 = K4 + K3 - 1) each reach C1 x K2 x K2 of g^(1); the C1 x W1 x W1 entries of the
        # g^(1) window (W1 = W2 + K2 - 1) each reach in_c x K1 x K1 inputs
        t1, t2, t3, t4 = layers[0], layers[1], layers[2], layers[3]
        Q4 = B * 2 * n[4]
        w2 = t4["k"] + t3["k"] - 1
        w1 = w2 + t2["k"] - 1
        wmacs = (t3["out_c"] * t4["k"] ** 2 * t2["out_c"] * t3["k"] ** 2
                 + t2["out_c"] * w2 * w2 * t1["out_c"] * t2["k"] ** 2
                 + t1["out_c"] * w1 * w1 * t1["in_c"] * t1["k"] ** 2)
        add("pass4_window[layer1,pass4]", 2.0 * Q4 * wmacs,
            4.0 * (3 * B * (n[1] + n[2] + n[3]) + Q4))
    for m in range(1, L):
        # relaxation parameters of layer m (elementwise): l, u read or, for layer 1, copied from
        # the shared bounds and written (8 bytes), the split byte read, (a_lo, a_up, b_up) and
        # the stability code written (13 bytes) per neuron and sub-domain; with optimised
        # slopes (fr = the fraction of the layer's neurons unstable), alpha read (4 bytes) for
        # the unstable neurons, the only ones whose slope is free
        fa = 0.0 if fr is None else fr[m - 1]
        add(f"relax_params[layer{m},pass{m}]", 0.0, (22.0 + 4.0 * fa) * B * n[m])
    if L >= 3 and layers[L - 2]["kind"] == wl.FC:
        # the final pass's spec rows through T_L and T_{L-1} in one kernel: T_{L-1}^T's flops;
        # bytes: the relaxations of layers L-1 and L-2 read (3 floats per neuron and
        # sub-domain), the relaxed slab over g^(L-2) written
        Qf = B * S
        add(f"final_fc[layer{L - 1},pass{L}]", 2.0 * Qf * macs(layers[L - 2]),
            4.0 * 3 * B * (n[L - 1] + n[L - 2]) + 4.0 * n[L - 2] * Qf)
    if L == 4 and layers[2]["kind"] == wl.FC and all(layers[i]["kind"] == wl.CONV for i in (0, 1)):
        # the whole final pass in one kernel (launched for the shapes the library covers): the
        # spec rows through T_3^T, T_2^T and T_1^T; bytes: the relaxations of layers 1 to 3
        # read (3 floats per neuron and sub-domain), W_3 and z1, one float per row written
        Qf = B * S
        add(f"spec_bound[layer2,pass{L}]",
            2.0 * Qf * (macs(layers[2]) + macs(layers[1]) + macs(layers[0])),
            4.0 * (3 * B * (n[1] + n[2] + n[3]) + n[3] * n[2] + n[1]) + 4.0 * Qf)
    for k in range(2, L + 1):
        R = 2 * n[k] if k < L else S
        Q = B * R
        mtop = k - 1 if k < L else L
        if k < L:
            add(f"init_rows[layer{k},pass{k}]", 0.0, 4.0 * n[k - 1] * Q)
        if 3 <= k < L and layers[k - 1]["kind"] == wl.FC and layers[k - 2]["kind"] == wl.CONV:
            # the pass opened at a fully connected layer inside the stage through layer k-1
            # (launched instead of init_rows + that stage for the shapes the library covers): its
            # flops; bytes: the rows of W_k and the relaxation of layer k-1 (3 floats per neuron
            # and sub-domain) read, the relaxed slab over g^(k-2) written
            t = layers[k - 2]
            add(f"convT_relax_fc[layer{k - 1},pass{k}]", 2.0 * Q * macs(t),
                4.0 * (n[k] * n[k - 1] + 3 * B * n[k - 1]) + 4.0 * n[k - 2] * Q)
            if k == 3 and layers[0]["kind"] == wl.CONV:
                # the whole pass in one kernel (launched instead of the FC-opened stage and the
                # bound stage for the shapes the library covers): both convolutions' flops;
                # bytes: the rows of W_3, the relaxations of layers 2 and 1 (3 floats per
                # neuron and sub-domain, and z1), one float per row written
                add(f"convT_fc_bound[layer{k - 1},pass{k}]",
                    2.0 * Q * (macs(t) + macs(layers[0])),
                    4.0 * (n[k] * n[k - 1] + 3 * B * (n[k - 1] + n[1]) + n[1]) + 4.0 * Q)
        for m in range(mtop, 0, -1):
            t = layers[m - 1]
            kind = "fcT" if t["kind"] == wl.FC else "convT"
            sfx = "_relax" if m > 1 else "_bound"
            out_bytes = 4.0 * n[m - 1] * Q if m > 1 else 4.0 * Q
            add(f"{kind}{sfx}[layer{m},pass{k}]", 2.0 * Q * macs(t), 4.0 * n[m] * Q + out_bytes)
        if mtop >= 2 and all(layers[i]["kind"] == wl.CONV for i in (0, 1)):
            # the last two stages fused in one kernel (launched instead of the pair for the
            # shapes the library covers): both stages' flops; the slab over h^(2) read and one
            # float per row written
            add(f"convT2_bound[layer2,pass{k}]", 2.0 * Q * (macs(layers[1]) + macs(layers[0])),
                4.0 * n[2] * Q + 4.0 * Q)
            # the same pair in the kernel that also runs pass 3 from W_3 (slab source): the same
            # flops; bytes as above plus the layer-1 relaxation (3 floats per neuron and
            # sub-domain, and z1)
            add(f"convT_slab_bound[layer2,pass{k}]",
                2.0 * Q * (macs(layers[1]) + macs(layers[0])),
                4.0 * n[2] * Q + 4.0 * Q + 4.0 * (3 * B * n[1] + n[1]))
    return work


def grad_work(layers, S, B, l2=None, fr=None):
    """Algorithmic work per launch of the reverse-sweep kernel classes: {class: (flop, bytes)}.

    Pass P (rows Q = B*R) is swept from its witnesses forward.  The witness forward through
    layer m costs 2 * Q * MACs(T_m) flops; its bytes are its input per row (the sign of A_x, one
    byte per input, for m = 1; the relaxed activations over g^(m-1) otherwise), the recorded
    coefficients over g^(m) and its output over g^(m) (4 bytes per entry each).  The adjoint
    sums read per (sub-domain, neuron) what the forward left (3 floats per group of 8 rows).
    The receptive-field pass 2 rebuilds each row's relaxed window and its A_x on MFMA and runs
    W_1 over the window's witness: twice the window flops of the bound pass; bytes: the layer-1
    relaxation read (3 floats per neuron and sub-domain) and one partial sum written per
    (window, window neuron).

    The fused two-layer forward of pass 3 needs T_2 only at the layer-2 neurons that are
    unstable (elsewhere the adjoint terms it feeds are not used); with 32 channels it computes
    just those (in tiles of 16 channels per pair of positions).  l2 = (fraction of layer-2
    neurons unstable, fraction of the dense T_2 tiles computed), from the batch's stability
    codes: its algorithmic flops count T_2 at the unstable neurons only, and the executed MFMA
    flops (the tiles computed) are returned under the key "executed".

    fr[m - 1] is the fraction of layer-m neurons unstable over the batch.  Only unstable neurons
    get adjoint terms, so the gathers read the partial sums of those neurons alone, the
    segmented reduction (R <= 64 rows per sub-domain) reads only their rows, and with 32
    channels on T_2 the fused pass-3 forward writes only their partial sums."""
    from paper_2011_13824_amd import workloads as wl
    L = len(layers)
    n = [wl.n_in(layers[0])] + [wl.n_out(t) for t in layers]

    def macs(t):
        if t["kind"] == wl.CONV:
            return wl.n_out(t) * t["in_c"] * t["k"] * t["k"]
        return t["out_c"] * t["in_c"]

    fr = [1.0] * L if fr is None else list(fr) + [1.0] * (L - len(fr))
    work = {}
    for P in range(L, 1, -1):
        R = S if P == L else 2 * n[P]
        Q = B * R
        if P == 2 and P < L and layers[0]["kind"] == wl.CONV and layers[1]["kind"] == wl.CONV:
            t1, t2 = layers[0], layers[1]
            wmacs = t1["out_c"] * t2["k"] ** 2 * t1["in_c"] * t1["k"] ** 2
            parts = B * (t2["out_c"] // 8) * t2["out_h"] * t2["out_w"] * t1["out_c"] * t2["k"] ** 2
            # (only the rows of unstable layer-2 neurons carry weight, and only those are run)
            f2 = l2[0] if l2 is not None else 1.0
            work["pass2_window_grad[layer1,pass2]"] = (4.0 * Q * wmacs * f2,
                                                       4.0 * (3 * B * n[1] + parts))
            # the gather reads every layer-1 code (a byte) and, for an unstable neuron, one
            # partial per covering window (NG groups x (K2 / S2)^2 taps) and its gradient entry
            taps = (t2["k"] + t2["stride"] - 1) // t2["stride"]
            cover = (t2["out_c"] // 8) * taps * taps
            work["pass2_grad_gather[layer1,pass2]"] = (
                0.0, B * n[1] * (1.0 + fr[0] * (4.0 * cover + 8.0)))
            continue
        if P == 3 and P < L and all(layers[i]["kind"] == wl.CONV for i in (0, 1)) \
                and layers[2]["kind"] == wl.FC:
            # both convolutions of pass 3's witness forward in one kernel (launched for the
            # shapes the library covers): their flops; bytes: the signs of A_x (one byte per
            # input), the recorded coefficients over g^(1), the adjoint partial sums of both
            # layers (3 floats per neuron and group of 8 rows)
            f2, tiles = (1.0, 1.0)
            compact = layers[1]["out_c"] == 32
            if compact and l2 is not None:
                f2, tiles = l2
            sums = fr[0] * n[1] + fr[1] * n[2] if compact else n[1] + n[2]
            work[f"fwd12[layer1,pass{P}]"] = (
                2.0 * Q * (macs(layers[0]) + f2 * macs(layers[1])),
                n[0] * Q + 4.0 * n[1] * Q + 12.0 * sums * Q / 8)
            work.setdefault("executed", {})[f"fwd12[layer1,pass{P}]"] = \
                2.0 * Q * (macs(layers[0]) + tiles * macs(layers[1]))
        for m in range(1, P):
            t = layers[m - 1]
            inb = n[0] * Q if m == 1 else 4.0 * n[m - 1] * Q
            work[f"fwd[layer{m},pass{P}]"] = (2.0 * Q * macs(t), inb + 8.0 * n[m] * Q)
            nu = fr[m - 1] * n[m]  # unstable neurons per sub-domain
            work[f"grad_gather[layer{m},pass{P}]"] = (0.0, 12.0 * nu * Q / 8 + 12.0 * B * nu)
            rows = nu if R <= 64 else n[m]  # (the segmented reduction skips stable neurons)
            work[f"grad_reduce[layer{m},pass{P}]"] = (0.0, 8.0 * rows * Q + 12.0 * B * nu)
    return work


def layer2_stats(net, x0, w, C, split, alpha):
    """(fraction of layer-2 neurons unstable, fraction of the dense T_2 tiles the fused pass-3
    forward computes) over the batch at the given slopes, or None when T_2 is not a
    convolution.  The second is 1 unless T_2 has 32 channels on an 8x8 map: then a row's 8
    positions are paired by their number of unstable channels (most with fewest, ties by
    position), a tile is 16 channels at a pair, and a pair takes ceil(n / 16) tiles, at least
    one, for its n channels unstable at either position."""
    t2 = w.layers[1]
    if t2.get("kind") != 1:
        return None
    from paper_2011_13824_amd import workloads as wl
    off2, n2 = wl.n_out(w.layers[0]), wl.n_out(t2)
    _, code = net.bound(x0, w.eps, C, split=split, alpha=alpha, want_codes=True)
    u = code[:, off2:off2 + n2].cpu().numpy() == 5
    if t2["out_c"] != 32 or (t2["out_h"], t2["out_w"]) != (8, 8):
        return float(u.mean()), 1.0
    u = u.reshape(-1, 32, 8, 8).transpose(0, 2, 3, 1)  # [B, row, position, channel]
    key = u.sum(axis=3) * 8 + np.arange(8)  # unique per position
    order = np.argsort(key, axis=2)  # positions by rank
    lo = np.take_along_axis(u, order[:, :, :4, None], axis=2)
    hi = np.take_along_axis(u, order[:, :, ::-1][:, :, :4, None], axis=2)
    per_pair = (lo | hi).sum(axis=3)  # [B, row, pair]
    tiles = np.maximum(1, (per_pair + 15) // 16)
    return float(u.mean()), float(tiles.mean() / 2.0)


def unstable_fractions(net, x0, w, C, split, alpha):
    """Fraction of the neurons of each ReLU layer that are unstable over the batch at the
    given slopes, from the library's stability codes."""
    from paper_2011_13824_amd import workloads as wl
    _, code = net.bound(x0, w.eps, C, split=split, alpha=alpha, want_codes=True)
    u = code.cpu().numpy() == 5
    fr, off = [], 0
    for t in w.layers[:-1]:
        k = wl.n_out(t)
        fr.append(float(u[:, off:off + k].mean()))
        off += k
    return fr


def traffic_record(workload, kernel):
    """HBM bytes per launch of a kernel class, as measured by rocprofv3 (FETCH_SIZE and
    WRITE_SIZE, scaled by a copy of known size) and recorded under profiles/ for this exact
    library build (sha256 of lirpa.hip followed by build.py); None when no record matches."""
    import glob
    import hashlib
    pkg = os.path.join(ROOT, "paper_2011_13824_amd")
    h = hashlib.sha256()
    for f in (os.path.join(pkg, "csrc", "lirpa.hip"), os.path.join(pkg, "build.py")):
        with open(f, "rb") as fh:
            h.update(fh.read())
    sha = h.hexdigest()
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        with open(path) as fh:
            for line in fh:
                if not line.startswith("traffic-record: "):
                    continue
                rec = json.loads(line[len("traffic-record: "):])
                if (rec.get("workload"), rec.get("kernel"), rec.get("source_sha256")) == \
                        (workload, kernel, sha):
                    return rec["read_bytes"] + rec["write_bytes"]
    return None


def cpu_baseline(w, budget_s=20.0):
    """The fp64 oracle, as it is, on a bounded sample of the same workload recipe."""
    from oracle import ref
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or os.cpu_count()
    rnet = ref.RefNet(w.layers)
    cand = ref.root_unstable(rnet, w.x0, w.eps, w.C)
    split = w.splits(cand)
    if w.steps > 0:
        # the same work per sub-domain as the GPU step: a heuristic bound pass for the fresh
        # start, then the projected Adam loop (a bound and a gradient per step, one more bound)
        n = min(16, w.B)
        t0 = time.perf_counter()
        _, l, u, _ = ref.bound(rnet, w.x0, w.eps, w.C, split[:n], nthreads=threads)
        a0 = np.where((l < 0) & (u > 0), u / np.where(u - l > 0, u - l, 1),
                      np.where(l >= 0, 1.0, 0.0))
        ref.optimize(rnet, w.x0, w.eps, w.C, split[:n], a0, w.steps, lr=w.lr, nthreads=threads)
        dt = time.perf_counter() - t0
        return {"value": round(n / dt, 4), "unit": "subdomains/s", "cores": threads,
                "kind": "oracle",
                "sample": f"first {n} of the {w.B} sub-domains of the {w.name} batch, heuristic "
                          f"start and {w.steps} Adam steps (fp64 C oracle, OpenMP, "
                          f"{dt:.1f} s wall)"}
    probe = min(8, w.B)
    t0 = time.perf_counter()
    ref.bound(rnet, w.x0, w.eps, w.C, split[:probe], nthreads=threads)
    per = (time.perf_counter() - t0) / probe
    n = int(min(w.B, max(probe, budget_s / max(per, 1e-9))))
    t0 = time.perf_counter()
    ref.bound(rnet, w.x0, w.eps, w.C, split[:n], nthreads=threads)
    dt = time.perf_counter() - t0
    return {"value": round(n / dt, 3), "unit": "subdomains/s", "cores": threads,
            "kind": "oracle",
            "sample": f"first {n} of the {w.B} sub-domains of the {w.name} batch "
                      f"(fp64 C oracle, OpenMP, {dt:.1f} s wall)"}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="wide_opt",
                    choices=["tiny", "base", "wide", "deep", "wide_opt"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0, help="seconds of oracle time")
    ap.add_argument("--max-ws-gib", type=float, default=64.0)
    ap.add_argument("--batch", type=int, default=0, help="override the workload's batch size")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only copy a device buffer of this many MiB 3 times (a known-size "
                         "kernel for scaling HBM byte counters) and exit")
    args = ap.parse_args()

    if args.copy_calibration_mib > 0:
        import torch
        n = args.copy_calibration_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "copies": 3}), flush=True)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(sub-domains shard across GPUs with no exchange; see the design notes). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2011_13824_amd import lirpa, workloads as wl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    w = wl.get(args.workload)
    if args.batch:
        w.B = args.batch
    B, S = w.B, w.S
    net = lirpa.Network(w.layers, device=dev)
    x0 = torch.as_tensor(w.x0).to(dev)
    C = torch.as_tensor(w.C).to(dev)

    # split masks: neurons unstable at the root, from this library's own root bound
    _, l0, u0 = net.bound(x0, w.eps, C, B=1, want_lu=True)
    l0, u0 = l0.cpu().numpy()[0], u0.cpu().numpy()[0]
    cand = np.flatnonzero((l0 < 0) & (u0 > 0))
    split = torch.as_tensor(w.splits(cand)).to(dev)

    optimise = w.steps > 0
    ws, ws_bytes = net.workspace(S, B, 1 if optimise else 0, int(args.max_ws_gib * (1 << 30)))
    lb = torch.empty((B, S), dtype=torch.float32, device=dev)
    if optimise:
        alpha = torch.empty((B, w.n_relu), dtype=torch.float32, device=dev)
        adam_m = torch.empty_like(alpha)
        adam_v = torch.empty_like(alpha)
        # fresh start: alpha from the library's own heuristic pass, zero Adam moments
        params = lirpa.lirpa_opt_params(w.steps, w.lr, 0.9, 0.999, 1e-8, 0, 1)

    def step():
        if optimise:
            # one optimised bound of the whole batch: a heuristic pass, then 20 Adam steps
            # (21 bounds and 20 gradients through the recomputed intermediate bounds)
            lirpa.lirpa_optimize(net.handle, x0, w.eps, C, S, B, split, alpha, adam_m, adam_v,
                                 params, lb, None, ws, ws_bytes)
        else:
            lirpa.lirpa_bound(net.handle, x0, w.eps, C, S, B, split, None, lb, None, None,
                              None, ws, ws_bytes)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    value = B / (ms / 1e3)

    # per-kernel event timing over the same number of steps
    lirpa.lirpa_timing_begin()
    for _ in range(args.steps):
        step()
    times = lirpa.lirpa_timing_end()
    torch.cuda.synchronize()
    fr = unstable_fractions(net, x0, w, C, split, alpha) if optimise else None
    work = stage_work(w.layers, S, B, fr)
    executed = {}
    if optimise:
        work.update(grad_work(w.layers, S, B, layer2_stats(net, x0, w, C, split, alpha), fr))
        executed = work.pop("executed", {})
    stages = {}
    for cls, (tot_ms, launches) in sorted(times.items(), key=lambda kv: -kv[1][0]):
        f, b = work.get(cls, (0.0, 0.0))
        f, b = f * launches, b * launches
        sec = tot_ms / 1e3
        stages[cls] = {"ms_per_step": round(tot_ms / args.steps, 4),
                       "launches_per_step": launches / args.steps,
                       "tflops": round(f / sec / 1e12, 3) if f else None,
                       "gbs": round(b / sec / 1e9, 1) if b else None}
        if cls in executed:
            stages[cls]["executed_tflops"] = round(executed[cls] * launches / sec / 1e12, 3)
    dom = max(times, key=lambda c: times[c][0])
    tot_ms, launches = times[dom]
    f, b = work.get(dom, (0.0, 0.0))
    f, b = f * launches, b * launches
    if f > 0 and (b == 0 or f / b >= PEAK_FP32_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)):
        achieved = f / launches / (tot_ms / launches / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_FP32_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_FP32_TFLOPS, 4)}
    else:
        achieved = b / (tot_ms / 1e3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    roof["kernel"] = dom
    roof["avg_launch_ms"] = round(tot_ms / launches, 4)
    if dom in executed:
        # the MFMA work the kernel actually issues (it skips T_2 where nothing uses it)
        roof["executed_tflops"] = round(executed[dom] / (tot_ms / launches / 1e3) / 1e12, 3)
    roof["traffic"] = None if args.batch else traffic_record(w.name, dom)

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "subdomains/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "net": w.extra.get("arch"), "B": B, "S": S,
                   "n_relu": w.n_relu, "max_splits": w.max_splits, "eps": w.eps,
                   "alpha": (f"{w.steps} Adam steps (lr {w.lr}) from the upper slope"
                             if optimise else "upper slope"),
                   "ws_gib": round(ws_bytes / 2**30, 2)},
        "path_tflops": round(sum(work.get(c, (0.0, 0.0))[0] * times[c][1] for c in times)
                             / args.steps / (ms / 1e3) / 1e12, 3),
        "roofline": roof,
        "stages": stages,
        "cpu_baseline": None if args.no_cpu_baseline else cpu_baseline(w, args.cpu_budget),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
