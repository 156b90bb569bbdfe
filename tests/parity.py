"""Helpers for the GPU-vs-oracle parity tests.

Tolerance (per tensor): every element must satisfy
    |x - r| <= rtol * max(|r|, rms(r))
i.e. relative above the tensor's RMS, absolute (rtol * RMS) below it.
rtol = 1e-4 for float32 storage, 2e-2 for bfloat16 storage.  For tensors
whose rows are D-wide vectors (embeddings E, pooled U, ad A, embedding
gradients dE) the floor is taken per row as well, max(|r|, rms(r), rms(r_row)):
a row of dE is the gradient of one image and a sum over all its occurrences,
and for a hot image it is the residue of heavy cancellation whose absolute
error scales with the row, not with its smallest entry.

Decisions taken in floating point (a ReLU mask, the max-pool argmax) can land
on either side of a near-tie when the GPU's float32 value and the oracle's
float64 value differ by rounding.  Such a decision is accepted when the
oracle's own value is within `tau` of the tie; its effect on the gradients is
then bounded from oracle quantities (absolute values propagated through the
absolute weights) and added to the tolerance of the affected elements.  The
expected values themselves always come from the oracle.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import oracle
from paper_1711_06505_amd import ams, synth

RTOL = {"f32": 1e-4, "f32x3": 1e-4, "bf16": 2e-2}


def f64(x):
    if isinstance(x, torch.Tensor):
        return x.detach().float().cpu().numpy().astype(np.float64)
    return np.asarray(x, dtype=np.float64)


def assert_close(x, r, rtol, name, extra=None, rows=False):
    x, r = f64(x), f64(r)
    assert x.shape == r.shape, (name, x.shape, r.shape)
    if r.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(r * r)))
    scale = np.maximum(np.abs(r), rms)
    if rows:
        scale = np.maximum(scale, np.sqrt(np.mean(r * r, axis=1, keepdims=True)))
    bound = rtol * scale
    if extra is not None:
        bound = bound + extra
    err = np.abs(x - r)
    bad = ~(err <= bound)
    if bad.any():
        idx = np.argwhere(bad)[:5].tolist()
        raise AssertionError(f"{name}: {int(bad.sum())}/{r.size} elements beyond tolerance; "
                             f"worst rel {float(np.max(err / np.maximum(scale, 1e-300))):.3e}; e.g. {idx}")
    return float(np.max(err / np.maximum(scale, 1e-300)))


def assert_close_sensitive(x, ref, pert, rtol, name, extra=None, rows=False):
    """End-to-end check of a result downstream of float32 intermediates: x
    against the oracle's exact value ref, held to rtol plus twice
    |pert - ref|, where pert is the oracle's own computation of the same
    result on the GPU's intermediates (its E, its forward values).  The
    extra tolerance is the oracle's measured sensitivity of this result to
    float32-sized changes of its inputs, including decisions (ReLU or PReLU
    branches, attention) that sit near a tie; it is zero where the chain is
    well-conditioned, and the GPU must then meet rtol alone."""
    bound = 2 * np.abs(f64(pert) - f64(ref))
    return assert_close(x, ref, rtol, name + " (end to end)", extra=bound if extra is None else bound + extra,
                        rows=rows)


# --------------------------------------------------------------- inputs

def device_batch(batch):
    occ = synth.occurrences(batch)
    return {
        "ids": torch.from_numpy(occ).cuda(),
        "seg_off": torch.from_numpy(batch["seg_off"]).cuda(),
        "dU": torch.from_numpy(batch["g_u"]).cuda(),
        "dA": torch.from_numpy(batch["g_a"]).cuda(),
        "n_beh": int(batch["seg_off"][-1]),
        "B": batch["seg_off"].size - 1,
    }


def run_gpu_step(w, batch, T_dev, Ws, bs, mode, final_relu=False, cap=None):
    db = device_batch(batch)
    st = ams.Step(w.dims, w.dtype, mode, db["B"], db["n_beh"], final_relu=final_relu, cap=cap)
    Wd = [W.cuda() for W in Ws]
    bd = [b.cuda() for b in bs]
    st.run(db["ids"], w.n_images, T_dev, Wd, bd, db["seg_off"], db["dU"], db["dA"])
    torch.cuda.synchronize()
    return st


def gpu_outputs(st):
    n_u = int(st.n_uniq.item())
    out = {
        "n_uniq": n_u, "dev_status": int(st.dev_status.item()),
        "uniq": st.uniq[:n_u].cpu().numpy(), "inv": st.inv[:st.n_occ].cpu().numpy(),
        "occ_perm": st.occ_perm[:st.n_occ].cpu().numpy(), "uniq_off": st.uniq_off[:n_u + 1].cpu().numpy(),
        "E": f64(st.E[:n_u]), "H1": f64(st.H1[:n_u]), "U": f64(st.U[:st.B]), "A": f64(st.A[:st.B]),
        "dE": f64(st.dE[:n_u]), "dW": [f64(x) for x in st.dW], "db": [f64(x) for x in st.db],
    }
    if st.H2 is not None:
        out["H2"] = f64(st.H2[:n_u])
    if st.mode == "att":
        out["w"] = f64(st.saved[:st.n_beh])
    elif st.mode == "max":
        out["argmax"] = st.saved[:st.B].cpu().numpy()
    return out


# ------------------------------------------------------- decision checks

def relu_flips(z_orc, h_gpu, tau_rel):
    """(u, m) pairs where the GPU's ReLU decision differs from the oracle's;
    each must be a near-tie |z| <= tau_rel * rms(z)."""
    z = np.asarray(z_orc)
    flips = np.argwhere((z > 0) != (np.asarray(h_gpu) > 0))
    if flips.size:
        rms = float(np.sqrt(np.mean(z * z)))
        worst = float(np.max(np.abs(z[tuple(flips.T)])))
        assert worst <= tau_rel * rms, f"ReLU decision flipped at |z| = {worst:.3e} (rms {rms:.3e})"
    return flips


def max_flips(seg_off, inv, E_orc, am_gpu, am_orc, tau_rel):
    """(i, d) where the GPU's first-argmax differs from the oracle's; the
    GPU's pick must be within tau of the oracle's maximum."""
    bad = np.argwhere(am_gpu != am_orc)
    if bad.size:
        rms = float(np.sqrt(np.mean(E_orc * E_orc)))
        for i, d in bad:
            jg, jo = int(am_gpu[i, d]), int(am_orc[i, d])
            assert seg_off[i] <= jg < seg_off[i + 1], "argmax outside the sample"
            gap = E_orc[inv[jo], d] - E_orc[inv[jg], d]
            assert 0 <= gap <= tau_rel * max(abs(E_orc[inv[jo], d]), rms), (i, d, gap)
    return bad


def grad_flip_bounds(dims, Ws, Xrows, orc_fwd, orc_bwd, flips1, flips2, dE_delta=None):
    """Elementwise bounds on how much the weight gradients may move when the
    ReLU decisions in flips1 (layer 1) / flips2 (layer 2) go the other way, or
    when dE changes by |dE_delta| (n_u x D, from argmax near-ties).

    Absolute values are propagated through absolute weights, so the bound
    holds whichever way each decision went."""
    L = len(dims) - 1
    n_u = orc_fwd["E"].shape[0]
    aW = [np.abs(f64(W)) for W in Ws]
    X = np.abs(f64(Xrows))
    h = [X] + [np.maximum(z, 0) for z in orc_fwd["Z"][:-1]]
    dZ = orc_bwd["dZ"]
    extra_W = [np.zeros((o, i)) for i, o in zip(dims[:-1], dims[1:])]
    extra_b = [np.zeros(o) for o in dims[1:]]
    # perturbation of pre-activation gradients, layer by layer from the top
    dz_delta = [np.zeros((n_u, o)) for o in dims[1:]]
    if dE_delta is not None:
        dz_delta[L - 1] += np.abs(dE_delta)
    # a flipped decision moves dz by at most the unmasked gradient |dh|
    for layer, flips in ((0, flips1), (1, flips2)):
        if flips is None or len(flips) == 0 or layer >= L - 1:
            continue
        dh = np.abs(dZ[layer + 1] @ f64(Ws[layer + 1]))       # unmasked gradient into layer's output
        for u, m in flips:
            dz_delta[layer][u, m] += dh[u, m]
    for l in range(L - 1, -1, -1):
        extra_W[l] += dz_delta[l].T @ np.abs(h[l])
        extra_b[l] += dz_delta[l].sum(0)
        if l > 0:
            # bounded change reaching the layer below (mask taken as open)
            dz_delta[l - 1] += dz_delta[l] @ aW[l]
    # a layer-1 flip changes only its own row of dW1 / db1 (covered above);
    # grow by a factor 2 for rounding in the perturbed terms themselves
    return [2 * e for e in extra_W], [2 * e for e in extra_b]


def large_grid_workload():
    """The long-sequence shapes at 6144 samples: 1.12M occurrences, 17.5k
    chunks of 64 positions, the hottest image's run 1.6k chunks long.  Past
    16,384 chunks the pooling backward switches to its large-grid kernels
    (several chunks per wave in the stable-order pass, 64 chunks per wave in
    the fix-up), which smaller batches never reach."""
    import dataclasses
    return dataclasses.replace(synth.get("c3_long"), name="long_6144", index=33, batch=6144, stream=-1)
