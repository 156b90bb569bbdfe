"""Independent float64 check of the oracle: plain PyTorch CPU autograd.

Unlike the oracle, this embeds *every occurrence* separately (no dedup), pools
with per-sample torch ops, and lets autograd derive all gradients.  It is used
only as a pin for the oracle on small inputs.
"""
from __future__ import annotations

import numpy as np
import torch


def _f64(x):
    if isinstance(x, torch.Tensor):
        return x.detach().to(torch.float64).cpu()
    return torch.as_tensor(np.asarray(x), dtype=torch.float64)


def step_autograd(batch, T, Ws, bs, mode: str, final_relu: bool = False):
    """Loss L = sum(g_u * U) + sum(g_a * A) and its gradients, per occurrence.

    T: full table (indexable by image ID).  Returns dict with U, A, E_occ,
    ge (dL/dE per occurrence), dW, db.
    """
    seg = np.asarray(batch["seg_off"], dtype=np.int64)
    beh = np.asarray(batch["beh_ids"], dtype=np.int64)
    ad = np.asarray(batch["ad_ids"], dtype=np.int64)
    occ = np.concatenate([beh, ad])
    n_beh = beh.size
    B = seg.size - 1
    Tt = _f64(T)
    X = Tt[torch.as_tensor(occ)]                       # every occurrence, no dedup
    W = [_f64(w).requires_grad_() for w in Ws]
    b = [_f64(x).requires_grad_() for x in bs]
    h = X
    for l in range(len(W)):
        h = torch.nn.functional.linear(h, W[l], b[l])
        if l < len(W) - 1 or final_relu:
            h = torch.relu(h)
    E_occ = h
    E_occ.retain_grad()
    A = E_occ[n_beh:]
    outs = []
    for i in range(B):
        e = E_occ[seg[i]:seg[i + 1]]
        if e.shape[0] == 0:
            outs.append(torch.zeros(E_occ.shape[1], dtype=torch.float64))
        elif mode == "sum":
            outs.append(e.sum(0))
        elif mode == "max":
            outs.append(e.max(0).values)
        elif mode == "att":
            w = torch.softmax(e @ A[i], dim=0)
            outs.append(w @ e)
        else:
            raise ValueError(mode)
    U = torch.stack(outs) if B else torch.zeros((0, E_occ.shape[1]), dtype=torch.float64)
    gU = _f64(batch["g_u"])
    gA = _f64(batch["g_a"]) if batch.get("g_a") is not None else torch.zeros_like(A)
    L = (gU * U).sum() + (gA * A).sum()
    L.backward()
    return {
        "U": U.detach().numpy(), "A": A.detach().numpy(), "E_occ": E_occ.detach().numpy(),
        "ge": E_occ.grad.numpy(), "L": float(L.detach()),
        "dW": [w.grad.numpy() for w in W], "db": [x.grad.numpy() for x in b],
    }
