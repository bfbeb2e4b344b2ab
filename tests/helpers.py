"""Test-side helpers: an independent fp64 network evaluation (torch CPU ops), closed forms and
small network builders.  None of this is used by the product path."""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as F

from paper_2011_13824_amd import workloads as wl


def torch_forward(layers, X, split=None, return_pre=False):
    """f_s(X) for a batch X [N, n0] in fp64 with torch's own conv2d / linear.

    split (optional, [n_relu] int) replaces split-active ReLUs by the identity and
    split-inactive ReLUs by zero.  Returns the output [N, n_L] (and the pre-activations of
    every ReLU layer, concatenated, when return_pre)."""
    a = torch.as_tensor(np.asarray(X, dtype=np.float64))
    N = a.shape[0]
    pres = []
    off = 0
    for m, t in enumerate(layers):
        W = torch.as_tensor(t["W"].astype(np.float64))
        b = torch.as_tensor(t["b"].astype(np.float64))
        if t["kind"] == wl.CONV:
            a = F.conv2d(a.reshape(N, t["in_c"], t["in_h"], t["in_w"]), W, b,
                         stride=t["stride"], padding=t["pad"]).reshape(N, -1)
        else:
            a = a.reshape(N, -1) @ W.T + b
        if m < len(layers) - 1:
            pres.append(a.clone())
            n = a.shape[1]
            if split is not None:
                s = torch.as_tensor(np.asarray(split[off:off + n], dtype=np.int64))
                a = torch.where(s > 0, a, torch.where(s < 0, torch.zeros_like(a), a.clamp(min=0)))
            else:
                a = a.clamp(min=0)
            off += n
    out = a.numpy()
    if return_pre:
        return out, torch.cat(pres, dim=1).numpy()
    return out


def affine_map_of_split_net(layers, split):
    """M, c with f_s(x) = M x + c, for a split vector that fixes every ReLU (built forward)."""
    n0 = wl.n_in(layers[0])
    X = np.vstack([np.zeros((1, n0)), np.eye(n0)])
    Y = torch_forward(layers, X, split)
    c = Y[0]
    M = (Y[1:] - c).T
    return M, c


def box_min_of_affine(Cspec, M, c, x0, eps):
    """min over ||x - x0||_inf <= eps of C (M x + c), in closed form (eps taken as fp32)."""
    eps = np.float64(np.float32(eps))
    CM = Cspec.astype(np.float64) @ M
    return CM @ x0.astype(np.float64) + Cspec.astype(np.float64) @ c - eps * np.abs(CM).sum(1)


def box_samples(x0, eps, n, rng):
    eps = np.float64(np.float32(eps))
    x0 = np.asarray(x0, dtype=np.float64)
    return x0 + eps * rng.uniform(-1.0, 1.0, size=(n, x0.size))


def small_conv_arch():
    """A small convolutional chain: strided and unit-stride convs, odd padding, FC head."""
    return [wl.conv(2, 9, 4, 3, 2, 1), wl.conv(4, 5, 3, 2, 1, 0), wl.fc(48, 7), wl.fc(7, 3)]
