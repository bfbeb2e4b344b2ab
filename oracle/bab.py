"""ORACLE -- test infrastructure only.

Plain Python branch and bound over the fp64 oracle's bounds: Algorithm 1 of Xu et al., "Fast and
Complete" (ICLR 2021), Sec. 3.3 (batch splits) and Sec. 3.4 (the complete framework), without
the LP fallback of its lines 11-13.  Only the tests may import this module; it shares nothing
with the GPU library.

Steps, in the order of Algorithm 1:
* line 2: optimised LiRPA at the root gives (f_lo, f_hi);
* line 3: P, the set of unverified sub-domains, starts as the root;
* line 5, batch_pick_out: the n sub-domains of P with the lowest f_lo (ties: the order in which
  they entered P) are taken out of P;
* line 6, batch_split: each is split on one unstable ReLU neuron into a child with the neuron
  forced active (split +1) and one with it forced inactive (split -1);
* line 7: optimised LiRPA bounds every child; a child starts from its parent's slopes alpha;
* line 8, Domain_Filter: children with f_lo >= 0 are verified and dropped; the rest join P;
* lines 9-10: f_lo = min over P of the lower bounds, f_hi = min over P of the upper bounds;
* line 4: the loop ends when f_lo >= 0 (P empty: verified) or f_hi < 0 (a sub-domain whose
  upper bound is negative: a violation).

Readings where the paper is silent:
* the branching rule: BaBSR's score is not given in the paper.  The stand-in scores each
  unstable, unsplit neuron of the sub-domain by the intercept -l u / (u - l) of its upper
  relaxation line (Eq. 5) under the sub-domain's own bounds, and splits the highest score,
  the lowest flat neuron index on ties;
* f_hi of a sub-domain is the upper bound at the slopes the lower side ended with (one
  bound of -C at those slopes);
* without LP the loop also stops when a picked sub-domain has no unstable unsplit neuron left
  ("stuck", line 12's case (2)) or when P outgrows eta or the iteration limit is reached
  (line 11).
"""
from __future__ import annotations

import numpy as np

from oracle import ref

VERIFIED, VIOLATED, UNKNOWN_STUCK, UNKNOWN_LIMIT = 1, 2, 3, 4


def heuristic_alpha(l, u):
    """The fresh-start slopes: the upper slope u/(u-l) of unstable neurons, 1 active, 0 inactive."""
    return np.where((l < 0) & (u > 0), u / np.where(u - l > 0, u - l, 1.0),
                    np.where(l >= 0, 1.0, 0.0))


def branch_neuron(l, u, code):
    """The stand-in branching rule: argmax of -l u / (u - l) over unstable unsplit neurons."""
    best, j_best = -np.inf, -1
    for j in range(l.size):
        if code[j] != ref.ST_UNSTABLE:
            continue
        score = -l[j] * u[j] / (u[j] - l[j])
        if score > best:
            best, j_best = score, j
    return j_best


def bound_domains(net, x0, eps, c, splits, alphas, steps, fresh, adam):
    """Optimised LiRPA on a batch of sub-domains: (lb, ub, alpha, l, u, code) per sub-domain.

    steps = 0 takes the heuristic slopes (alpha None) or the given ones; otherwise projected
    Adam from alphas (or from the heuristic start when fresh) with zero moments."""
    C = np.asarray(c, dtype=np.float32)[None, :]
    if steps == 0:
        lb, l, u, code = ref.bound(net, x0, eps, C, splits, alphas)
        ubn, _, _, _ = ref.bound(net, x0, eps, -C, splits, alphas)
        return lb[:, 0], -ubn[:, 0], alphas, l, u, code
    if fresh:
        _, l, u, _ = ref.bound(net, x0, eps, C, splits)
        alphas = heuristic_alpha(l, u)
    r = ref.optimize(net, x0, eps, C, splits, alphas, steps, **adam)
    a = r["alpha"].astype(np.float32)
    _, l, u, code = ref.bound(net, x0, eps, C, splits, a)
    ubn, _, _, _ = ref.bound(net, x0, eps, -C, splits, a)
    return r["lb_best"][:, 0], -ubn[:, 0], a, l, u, code


def bab(net, x0, eps, c, batch, max_domains, max_iters, root_steps=0, steps=0, lr=0.1,
        beta1=0.9, beta2=0.999, eps_adam=1e-8):
    """Algorithm 1 without LP on the property c^T f(x) >= 0 over ||x - x0||_inf <= eps.

    Returns dict(status, f_lo, f_hi, iterations, domains_bounded, domains_left)."""
    adam = dict(lr=lr, beta1=beta1, beta2=beta2, eps_adam=eps_adam)
    n = net.n_relu
    root = np.zeros((1, n), dtype=np.int8)
    lb, ub, al, l, u, code = bound_domains(net, x0, eps, c, root, None, root_steps, True, adam)
    bounded = 1
    P = []  # entries: (lb, ub, split, alpha, branch neuron), in the order they entered P
    leaf_lo = leaf_hi = np.inf  # lowest bounds of the verified (dropped) sub-domains
    if lb[0] >= 0:
        leaf_lo, leaf_hi = lb[0], ub[0]
    else:
        P.append((lb[0], ub[0], root[0], None if al is None else al[0],
                  branch_neuron(l[0], u[0], code[0])))
    it = 0
    while True:
        if not P:
            return dict(status=VERIFIED, f_lo=float(leaf_lo), f_hi=float(leaf_hi),
                        iterations=it, domains_bounded=bounded, domains_left=0)
        f_lo = min(d[0] for d in P)
        f_hi = min(d[1] for d in P)
        status = None
        if f_hi < 0:
            status = VIOLATED
        elif len(P) > max_domains or it >= max_iters:
            status = UNKNOWN_LIMIT
        else:
            k = min(batch, len(P))
            order = sorted(range(len(P)), key=lambda i: (P[i][0], i))  # stable
            picked = [P[i] for i in order[:k]]
            if any(d[4] < 0 for d in picked):
                status = UNKNOWN_STUCK
        if status is not None:
            return dict(status=status, f_lo=float(f_lo), f_hi=float(f_hi), iterations=it,
                        domains_bounded=bounded, domains_left=len(P))
        P = [P[i] for i in order[k:]]
        # batch_split: child 2i forces the neuron active, child 2i + 1 inactive
        splits = np.zeros((2 * k, n), dtype=np.int8)
        alphas = None if picked[0][3] is None else np.zeros((2 * k, n), dtype=np.float32)
        for i, d in enumerate(picked):
            for s_, sgn in ((2 * i, 1), (2 * i + 1, -1)):
                splits[s_] = d[2]
                splits[s_, d[4]] = sgn
                if alphas is not None:
                    alphas[s_] = d[3]
        lb, ub, al, l, u, code = bound_domains(net, x0, eps, c, splits, alphas, steps, False,
                                               adam)
        bounded += 2 * k
        for s_ in range(2 * k):  # Domain_Filter
            if lb[s_] >= 0:
                leaf_lo, leaf_hi = min(leaf_lo, lb[s_]), min(leaf_hi, ub[s_])
            else:
                P.append((lb[s_], ub[s_], splits[s_], None if al is None else al[s_],
                          branch_neuron(l[s_], u[s_], code[s_])))
        it += 1
