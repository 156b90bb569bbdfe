"""GPU parity of multiple-query attentive pooling (section 5.2) through the C
ABI against the float64 oracle: the ID channel (a query per sample) forward
and backward, and the two channels of one step merged into one dE (the image
channel's ams_pool_bwd, then the ID channel with accumulate = 1).  Per call:
both sides get the same dedup, embeddings and queries (float32 values), at the
tiny, the 1024-sample and the long-sequence batch shapes (hot images whose
runs cross many 64-position chunks), and the long-sequence shapes at 6144
samples, where the backward takes its large-grid kernels."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_1711_06505_amd import ams, synth
from tests.parity import RTOL, assert_close, f64, large_grid_workload

pytestmark = pytest.mark.gpu
F32 = RTOL["f32"]


def cuda(x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x))
    return (t.to(dtype) if dtype is not None else t).cuda()


@pytest.mark.parametrize("name", ["tiny", "c1_f32", "c3_long", "large_grid"])
def test_two_channel_pooling_matches_oracle(name):
    w = large_grid_workload() if name == "large_grid" else synth.get(name)
    batch = synth.make_batch(w)
    occ = synth.occurrences(batch)
    dd = oracle.dedup(occ, w.n_images)
    seg = batch["seg_off"]
    B, n_beh, n_u, D = w.batch, int(seg[-1]), dd["n_uniq"], 12
    print(f"mqap {name}: n_beh={n_beh} n_u={n_u}", flush=True)
    rng = np.random.default_rng(3)
    E = (rng.standard_normal((n_u, D)) * 0.5).astype(np.float32)
    Q = (rng.standard_normal((B, D)) * 0.5).astype(np.float32)
    g1 = rng.standard_normal((B, D)).astype(np.float32)
    g2 = rng.standard_normal((B, D)).astype(np.float32)
    gA = rng.standard_normal((B, D)).astype(np.float32)
    E64, Q64 = E.astype(np.float64), Q.astype(np.float64)
    # oracle: the image channel (ad query) and the ID channel (given query)
    f1 = oracle.pool_fwd("att", seg, dd["inv"], E64)
    f2 = oracle.pool_query_fwd(seg, dd["inv"], E64, Q64)
    b1 = oracle.pool_bwd("att", seg, dd["inv"], n_u, E64, f1, g1, gA)
    b2 = oracle.pool_query_bwd(seg, dd["inv"], n_u, E64, Q64, f2, g2)
    # GPU, same inputs
    i32 = torch.int32
    seg_d, inv_d = cuda(seg, i32), cuda(dd["inv"], i32)
    perm_d, off_d = cuda(dd["occ_perm"], i32), cuda(dd["uniq_off"], i32)
    nu_d = torch.tensor([n_u], dtype=i32, device="cuda")
    E_d, Q_d = cuda(E), cuda(Q)
    U1, A1 = torch.empty((B, D), device="cuda"), torch.empty((B, D), device="cuda")
    w1 = torch.empty(max(n_beh, 1), device="cuda")
    U2, w2 = torch.empty((B, D), device="cuda"), torch.empty(max(n_beh, 1), device="cuda")
    ams.ams_pool_fwd("att", seg_d, n_beh, inv_d, E_d, U1, A1, w1)
    ams.ams_pool_query_fwd(seg_d, n_beh, inv_d, E_d, Q_d, U2, w2)
    torch.cuda.synchronize()
    assert_close(U2, f2["U"], F32, "U (ID channel)", rows=True)
    assert_close(w2[:n_beh], f2["w"], F32, "w (ID channel)")
    cap = n_u + 33
    E_cap = torch.zeros((cap, D), device="cuda")        # E and dE hold `cap` rows
    E_cap[:n_u] = E_d
    ws = torch.empty(max(ams.ams_pool_workspace("att", B, n_beh, D, cap), 256), dtype=torch.uint8, device="cuda")
    dE = torch.full((cap, D), 7.0, device="cuda")
    dQ = torch.full((B, D), 7.0, device="cuda")
    # backward on the oracle's forward values (identical inputs for both sides)
    U1o, A1o, w1o = cuda(f1["U"].astype(np.float32)), cuda(f1["A"].astype(np.float32)), cuda(f1["w"].astype(np.float32))
    U2o, w2o = cuda(f2["U"].astype(np.float32)), cuda(f2["w"].astype(np.float32))
    ams.ams_pool_query_bwd(seg_d, n_beh, inv_d, perm_d, off_d, nu_d, cap, E_cap, Q_d, U2o, w2o, cuda(g2), dQ, dE,
                           False, ws)
    torch.cuda.synchronize()
    assert_close(dE[:n_u], b2["dE"], F32, "dE (ID channel alone)", rows=True)
    assert_close(dQ, b2["dQ"], F32, "dQ", rows=True)
    # both channels into one dE: image channel first, then the ID channel accumulated
    ams.ams_pool_bwd("att", seg_d, n_beh, inv_d, perm_d, off_d, nu_d, cap, E_cap, U1o, A1o, w1o, cuda(g1), cuda(gA),
                     dE, ws)
    ams.ams_pool_query_bwd(seg_d, n_beh, inv_d, perm_d, off_d, nu_d, cap, E_cap, Q_d, U2o, w2o, cuda(g2), dQ, dE,
                           True, ws)
    torch.cuda.synchronize()
    assert_close(dE[:n_u], b1["dE"] + b2["dE"], F32, "dE (both channels)", rows=True)
