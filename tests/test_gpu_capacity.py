"""A unique-row capacity below the batch's real unique count.

The pooling calls are told E and dE hold `cap` rows while the dedup found
n_u > cap distinct images.  Every call must stay inside those rows: the
buffers here are slices of larger ones whose rows past `cap` hold a sentinel
pattern, so a write past the capacity shows up as a changed sentinel (and a
read past it could only touch this same allocation).  Where the definition
still fixes the answer (sum pooling: a row's gradient does not depend on E)
the rows below the capacity are checked against the oracle as well.
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_1711_06505_amd import ams, synth
from tests.parity import assert_close, device_batch, f64

pytestmark = pytest.mark.gpu

SENTINEL = -12345.5
SPARE = 64


def cuda_i32(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).cuda()


def guarded(rows, D, fill=None):
    """A [rows x D] view of a [rows + SPARE x D] buffer whose spare rows hold the sentinel."""
    big = torch.full((rows + SPARE, D), SENTINEL, device="cuda")
    if fill is not None:
        big[:rows] = fill
    return big, big[:rows]


@pytest.mark.parametrize("mode", ["sum", "max", "att"])
def test_pool_with_capacity_below_unique_count(mode):
    w = synth.get("tiny")
    batch = synth.make_batch(w)
    dd = oracle.dedup(synth.occurrences(batch), w.n_images)
    n_u, D = dd["n_uniq"], w.out_dim
    cap = n_u - 57
    print(f"capacity {mode}: n_u={n_u} cap={cap}", flush=True)
    rng = np.random.default_rng(3)
    E32 = rng.standard_normal((n_u, D)).astype(np.float32)
    db = device_batch(batch)
    B, n_beh = db["B"], db["n_beh"]
    E_big, E = guarded(cap, D, torch.from_numpy(E32[:cap]).cuda())
    dE_big, dE = guarded(cap, D)
    inv = cuda_i32(dd["inv"])
    U = torch.zeros((B, D), device="cuda")
    A = torch.zeros((B, D), device="cuda")
    saved = (torch.zeros((B, D), dtype=torch.int32, device="cuda") if mode == "max" else
             torch.zeros(n_beh, device="cuda") if mode == "att" else None)
    ams.ams_pool_fwd(mode, db["seg_off"], n_beh, inv, E, U, A, saved)
    nu = torch.tensor([n_u], dtype=torch.int32, device="cuda")
    ws = torch.empty(max(ams.ams_pool_workspace(mode, B, n_beh, D, cap), 256), dtype=torch.uint8, device="cuda")
    ams.ams_pool_bwd(mode, db["seg_off"], n_beh, inv, cuda_i32(dd["occ_perm"]), cuda_i32(dd["uniq_off"]), nu,
                     cap, E, U, A, saved, db["dU"], db["dA"], dE, ws)
    torch.cuda.synchronize()
    # nothing written past the capacity
    assert torch.all(E_big[cap:] == SENTINEL) and torch.all(dE_big[cap:] == SENTINEL)
    assert torch.isfinite(U).all() and torch.isfinite(A).all() and torch.isfinite(dE).all()
    # rows past the capacity read as zero rows
    E_zero = E32.copy()
    E_zero[cap:] = 0
    pf = oracle.pool_fwd(mode, batch["seg_off"], dd["inv"], E_zero)
    assert_close(f64(A), pf["A"], 1e-6, "A")
    if mode == "sum":
        assert_close(f64(U), pf["U"], 1e-5, "U")
        # a sum-pooled image's gradient does not depend on E: rows below cap are exact
        pb = oracle.pool_bwd("sum", batch["seg_off"], dd["inv"], n_u, E32, pf, batch["g_u"], batch["g_a"])
        assert_close(f64(dE), pb["dE"][:cap], 1e-5, "dE below the capacity")


def test_embed_and_step_with_capacity_below_unique_count():
    w = synth.get("tiny")
    batch = synth.make_batch(w)
    dd = oracle.dedup(synth.occurrences(batch), w.n_images)
    cap = dd["n_uniq"] - 40
    db = device_batch(batch)
    Ws, bs = synth.make_weights(w)
    T = synth.table_full(w, device="cuda")
    st = ams.Step(w.dims, w.dtype, "att", db["B"], db["n_beh"], cap=cap, cap_checked=True)
    # the Step's buffers hold exactly `cap` rows; guard them with sentinel rows
    keep = {}
    for name in ("E", "dE"):
        big, view = guarded(cap, w.out_dim)
        setattr(st, name, view)
        keep[name] = big
    occ = torch.from_numpy(synth.occurrences(batch)).cuda()
    st.run(occ, w.n_images, T, [x.cuda() for x in Ws], [x.cuda() for x in bs], db["seg_off"], db["dU"], db["dA"])
    torch.cuda.synchronize()
    assert not st.capacity_ok()
    for name, big in keep.items():
        assert torch.all(big[cap:] == SENTINEL), name
    assert int(st.dev_status.item()) == 0
