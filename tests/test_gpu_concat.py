"""GPU parity of the concatenate aggregator (section 5.2) through the C ABI
against the float64 oracle: U and A are copies and must be bit-exact; dE is
a sum per unique image (1e-4 relative).  Batch shapes: the tiny one, the
1024-sample one and the long-sequence one (lengths up to 500 against Lc = 64,
so most lists are truncated, and hot images whose runs cross many 64-position
chunks), the same shapes at 6144 samples (the backward's large-grid
kernels), plus Lc larger than every list (pure padding)."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_1711_06505_amd import ams, synth
from tests.parity import RTOL, assert_close, large_grid_workload

pytestmark = pytest.mark.gpu
F32 = RTOL["f32"]


def cuda(x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x))
    return (t.to(dtype) if dtype is not None else t).cuda()


@pytest.mark.parametrize("name,Lc", [("tiny", 3), ("tiny", 40), ("c1_f32", 20), ("c3_long", 64),
                                     ("large_grid", 16)])
def test_concat_pooling_matches_oracle(name, Lc):
    w = large_grid_workload() if name == "large_grid" else synth.get(name)
    batch = synth.make_batch(w)
    occ = synth.occurrences(batch)
    dd = oracle.dedup(occ, w.n_images)
    seg = batch["seg_off"]
    B, n_beh, n_u, D = w.batch, int(seg[-1]), dd["n_uniq"], 12
    print(f"concat {name} Lc={Lc}: n_beh={n_beh} n_u={n_u}", flush=True)
    rng = np.random.default_rng(Lc)
    E = (rng.standard_normal((n_u, D)) * 0.5).astype(np.float32)
    gU = rng.standard_normal((B, Lc * D)).astype(np.float32)
    gA = rng.standard_normal((B, D)).astype(np.float32)
    f = oracle.pool_concat_fwd(seg, dd["inv"], E, Lc)
    dE_ref = oracle.pool_concat_bwd(seg, dd["inv"], n_u, D, Lc, gU, gA)
    i32 = torch.int32
    seg_d, inv_d = cuda(seg, i32), cuda(dd["inv"], i32)
    U = torch.full((B, Lc * D), float("nan"), device="cuda")
    A = torch.full((B, D), float("nan"), device="cuda")
    ams.ams_pool_concat_fwd(Lc, seg_d, n_beh, inv_d, cuda(E), U, A)
    torch.cuda.synchronize()
    assert torch.equal(U.cpu(), torch.from_numpy(f["U"].astype(np.float32))), "U"
    assert torch.equal(A.cpu(), torch.from_numpy(f["A"].astype(np.float32))), "A"
    cap = n_u + 17
    dE = torch.full((cap, D), float("nan"), device="cuda")
    ws = torch.empty(ams.load().ams_pool_workspace(0, B, n_beh, D, cap), dtype=torch.uint8, device="cuda")
    nu_d = torch.tensor([n_u], dtype=i32, device="cuda")
    ams.ams_pool_concat_bwd(Lc, seg_d, n_beh, inv_d, cuda(dd["occ_perm"], i32), cuda(dd["uniq_off"], i32), nu_d, cap,
                            cuda(gU), cuda(gA), dE, ws)
    torch.cuda.synchronize()
    assert_close(dE[:n_u], dE_ref, F32, "dE (concat)", rows=True)
