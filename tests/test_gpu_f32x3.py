"""GPU parity of AMS_F32_X3 (float32 storage; the 4096-wide forward product
on bf16 MFMA with every float32 operand split exactly into three bf16 parts
and six of the nine part products kept) against the float64 oracle at the
float32 tolerance, 1e-4 relative.

Forward at the 96-sample 4096-256-64-12 batch (cap past n_u, ragged last
tile) and at the benchmarked 1024-sample batch at full size (tiles cut
between stream-K workers); rows whose ID is out of range; PReLU (the saved
pre-activations); whole steps end to end.  The split's error is also held to
that of the float32-MFMA path on the same inputs: the three part products it
leaves out are below 2^-22 of each product, about one float32 rounding."""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import oracle
from paper_1711_06505_amd import ams, synth
from tests.parity import RTOL, assert_close, f64
from tests.test_gpu_parity import compare_step, step_case

pytestmark = pytest.mark.gpu
TOL = RTOL["f32x3"]


def workload(name):
    base = synth.get("c1_f32")
    if name == "mid":
        base = dataclasses.replace(base, index=11, batch=96, n_images=20_000, stream=-1)
    return dataclasses.replace(base, name=f"{name}_f32x3", dtype="f32x3")


def case(w):
    batch = synth.make_batch(w)
    dd = oracle.dedup(synth.occurrences(batch), w.n_images)
    Ws, bs = synth.make_weights(w)
    return dd, Ws, bs


def gpu_fwd(w, uniq_np, Ws, bs, dtype, cap_extra=77, slopes=None):
    n_u = len(uniq_np)
    cap = n_u + cap_extra
    T_dev = synth.table_rows(w, np.arange(w.n_images), device="cuda")
    uniq = torch.zeros(cap, dtype=torch.int32, device="cuda")
    uniq[:n_u] = torch.from_numpy(np.asarray(uniq_np, np.int32)).cuda()
    nu = torch.tensor([n_u], dtype=torch.int32, device="cuda")
    mlp = ams.make_mlp(w.dims, dtype)
    H1 = torch.full((cap, w.dims[1]), float("nan"), device="cuda")
    H2 = torch.full((cap, w.dims[2]), float("nan"), device="cuda")
    E = torch.full((cap, w.out_dim), float("nan"), device="cuda")
    ws = torch.empty(ams.ams_embed_workspace(mlp, cap), dtype=torch.uint8, device="cuda")
    ams.ams_embed_fwd(mlp, T_dev, uniq, nu, cap, [W.cuda() for W in Ws], [b.cuda() for b in bs], H1, H2, E, ws,
                      slopes=None if slopes is None else [torch.from_numpy(s).cuda() for s in slopes])
    torch.cuda.synchronize()
    return {"E": f64(E[:n_u]), "H1": f64(H1[:n_u]), "H2": f64(H2[:n_u])}


def rel_err(g, o):
    return float(np.abs(g - o).max() / max(np.abs(o).max(), 1e-30))


@pytest.mark.parametrize("name", ["mid", "c1"])
def test_x3_forward_matches_oracle(name):
    w = workload(name)
    dd, Ws, bs = case(w)
    print(f"f32x3 fwd {name}: n_u={dd['n_uniq']}", flush=True)
    g = gpu_fwd(w, dd["uniq"], Ws, bs, "f32x3")
    T_u = synth.table_rows(w, dd["uniq"])
    o = oracle.mlp_fwd(T_u, np.arange(dd["n_uniq"]), Ws, bs)
    assert_close(g["H1"], np.maximum(o["Z"][0], 0), TOL, "H1")
    assert_close(g["H2"], np.maximum(o["Z"][1], 0), TOL, "H2")
    assert_close(g["E"], o["E"], TOL, "E", rows=True)


def test_x3_error_tracks_float32_mfma():
    """Max error of H1 against the float64 oracle: the split within 4x of the
    float32-MFMA path (both are float32-rounding sized)."""
    w = workload("mid")
    dd, Ws, bs = case(w)
    T_u = synth.table_rows(w, dd["uniq"])
    o = np.maximum(oracle.mlp_fwd(T_u, np.arange(dd["n_uniq"]), Ws, bs)["Z"][0], 0)
    e3 = rel_err(gpu_fwd(w, dd["uniq"], Ws, bs, "f32x3")["H1"], o)
    e1 = rel_err(gpu_fwd(w, dd["uniq"], Ws, bs, "f32")["H1"], o)
    print(f"H1 max rel error: split {e3:.3g}, float32 MFMA {e1:.3g}", flush=True)
    assert e3 <= max(4 * e1, 1e-6)


def test_x3_out_of_range_rows_read_zero():
    w = workload("mid")
    Ws, bs = synth.make_weights(w)
    ids = np.arange(0, 3000, 7, dtype=np.int32)                 # 429 rows: 4 tiles, ragged
    ids[[5, 200, 428]] = [w.n_images + 3, -2, w.n_images]
    g = gpu_fwd(w, ids, Ws, bs, "f32x3")
    X = synth.table_rows(w, np.clip(ids, 0, w.n_images - 1)).double()
    X[[5, 200, 428]] = 0
    o = oracle.mlp_fwd(X, np.arange(len(ids)), Ws, bs)
    assert_close(g["E"], o["E"], TOL, "E", rows=True)


def test_x3_prelu_forward():
    w = workload("mid")
    dd, Ws, bs = case(w)
    rng = np.random.default_rng(3)
    sl = [rng.uniform(-0.25, 0.5, d).astype(np.float32) for d in w.dims[1:-1]]
    g = gpu_fwd(w, dd["uniq"], Ws, bs, "f32x3", slopes=sl)
    X = synth.table_rows(w, dd["uniq"]).double().numpy()
    Z = oracle.dense_fwd(X, Ws, bs, sl)
    assert_close(g["H1"], Z[0], TOL, "Z1 (saved)")
    assert_close(g["H2"], Z[1], TOL, "Z2 (saved)")
    assert_close(g["E"], Z[-1], TOL, "E", rows=True)


@pytest.mark.parametrize("name,mode", [("mid", "att"), ("mid", "max"), ("c1", "att")])
def test_x3_step_end_to_end(name, mode):
    w = workload(name)
    print(f"f32x3 step {name} {mode}", flush=True)
    batch, Ws, T_u, g, o = step_case(w, mode)
    compare_step(w, mode, batch, Ws, T_u, g, o)
