"""Helpers for GPU tests: move seeded inputs to the device and build descriptors."""
from __future__ import annotations

import numpy as np


def to_device(x, device="cuda"):
    """Inputs -> dict of torch tensors holding exactly the stored bits."""
    import torch

    def t(a):
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(device)
        return torch.from_numpy(np.ascontiguousarray(a)).to(device)

    return dict(Q=t(x.Q), K=t(x.K), V=t(x.V), dO=t(x.dO), W1=t(x.W1), W2=t(x.W2), tau=t(x.tau))


def to_f64(t):
    import torch
    return t.detach().to(torch.float64).cpu().numpy()


def desc_of(wl, segments=0, sigma=1.0, chunk=0):
    import paper_2606_27748_amd as F
    return F.make_desc(wl.B, wl.H, wl.N, wl.d, wl.m, wl.variant, wl.causal, wl.io, dv=wl.dv,
                       sigma=sigma, segments=segments, chunk=chunk)
