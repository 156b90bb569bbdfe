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


def joint_autograd(batch, jb, T, Ws, bs, id_tables, ctr_Ws, ctr_bs, mode: str = "att", query_table=None):
    """The joint step in float64 autograd, every occurrence embedded on its own.

    Image path as step_autograd (no dedup); each ID table is bag-summed over a
    sample's behaviors and its ad with torch's embedding_bag; the CTR MLP (ReLU
    between layers) runs on [U, A, bag_0, bag_1, ...] and the loss is torch's
    mean softmax cross-entropy.  With query_table t_q, a second attentive
    channel takes the ad's row of ID table t_q as its query (U2_i =
    softmax(e_j . Q_i) weighted sum of the behaviors' e_j) and the CTR input
    is [U, U2, A, bags...].  T and id_tables are whole tables.  Returns the
    loss, U, A, the bags, X, the gradient of X, the image-model and CTR
    gradients, and the dense gradient of every ID table.
    """
    seg = np.asarray(batch["seg_off"], dtype=np.int64)
    beh = np.asarray(batch["beh_ids"], dtype=np.int64)
    ad = np.asarray(batch["ad_ids"], dtype=np.int64)
    occ = np.concatenate([beh, ad])
    n_beh = beh.size
    B = seg.size - 1
    X_img = _f64(T)[torch.as_tensor(occ)]
    W = [_f64(w).requires_grad_() for w in Ws]
    b = [_f64(x).requires_grad_() for x in bs]
    h = X_img
    for l in range(len(W)):
        h = torch.nn.functional.linear(h, W[l], b[l])
        if l < len(W) - 1:
            h = torch.relu(h)
    E_occ = h
    A = E_occ[n_beh:]
    outs = []
    for i in range(B):
        e = E_occ[seg[i]:seg[i + 1]]
        if mode == "sum":
            outs.append(e.sum(0))
        elif mode == "att":
            outs.append(torch.softmax(e @ A[i], dim=0) @ e)
        else:
            raise ValueError(mode)
    U = torch.stack(outs)
    tabs = [_f64(x).requires_grad_() for x in id_tables]
    bags = []
    for t, tab in enumerate(tabs):
        bt = np.asarray(jb["beh_ids"][t], np.int64)
        at = np.asarray(jb["ad_ids"][t], np.int64)
        # one bag per sample: its behaviors' IDs then its ad's ID
        flat, offs = [], []
        for i in range(B):
            offs.append(len(flat))
            flat.extend(bt[seg[i]:seg[i + 1]].tolist())
            flat.append(int(at[i]))
        bags.append(torch.nn.functional.embedding_bag(torch.as_tensor(flat), tab, torch.as_tensor(offs),
                                                      mode="sum"))
    users = [U]
    if query_table is not None:
        Q = tabs[query_table][torch.as_tensor(np.asarray(jb["ad_ids"][query_table], np.int64))]
        users.append(torch.stack([torch.softmax(E_occ[seg[i]:seg[i + 1]] @ Q[i], dim=0) @ E_occ[seg[i]:seg[i + 1]]
                                  for i in range(B)]))
    X = torch.cat(users + [A] + bags, dim=1)
    X.retain_grad()
    cW = [_f64(w).requires_grad_() for w in ctr_Ws]
    cb = [_f64(x).requires_grad_() for x in ctr_bs]
    z = X
    for l in range(len(cW)):
        z = torch.nn.functional.linear(z, cW[l], cb[l])
        if l < len(cW) - 1:
            z = torch.relu(z)
    loss = torch.nn.functional.cross_entropy(z, torch.as_tensor(np.asarray(jb["labels"], np.int64)))
    loss.backward()
    return {
        "loss": float(loss.detach()), "U": U.detach().numpy(), "A": A.detach().numpy(),
        "bags": [x.detach().numpy() for x in bags], "X": X.detach().numpy(), "dX": X.grad.numpy(),
        "dW": [w.grad.numpy() for w in W], "db": [x.grad.numpy() for x in b],
        "ctr_dW": [w.grad.numpy() for w in cW], "ctr_db": [x.grad.numpy() for x in cb],
        "id_grad": [x.grad.numpy() for x in tabs],
    }
