"""GPU parity of the image embedding model with PReLU between its layers
(section 7.2: a learnable slope per channel) through the C ABI against the
float64 oracle's dense net (the same definition the CTR model's PReLU is
pinned on), at 1e-4 relative.

Forward: E and the saved pre-activations Z1, Z2 (which the library keeps in
H1_save / H2_save in PReLU mode) at the tiny batch (256-64-16: the
one-tile-per-block first layer), the 96-sample 4096-256-64-12 batch and the
benchmarked 1024-sample batch at full size (the stream-K first layer with
tiles cut between workers).  Backward, per call as in the ReLU tests: the
GPU gets the oracle's pre-activations (rounded to float32, so both sides take
the same branches) and a random dE; every weight, bias and slope gradient is
compared.  Slopes of both signs; slope 0 reproduces the ReLU path.

bf16 storage (table and weights bf16, float32 accumulation): the same checks
on the stream-K first layer (96 and 1024 samples) and the row-split one (a
capacity past 131,072 rows).  Z1 is kept as its bf16 rounding, so the
forward's E is held to 1e-4 and Z1 to bf16 rounding; the backward gets the
oracle's Z1 rounded to bf16 (the oracle takes the same values) and is held
to the bf16 tolerance, as the ReLU bf16 backward is."""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import oracle
from paper_1711_06505_amd import ams, synth
from tests.parity import RTOL, assert_close, assert_close_sensitive, f64

pytestmark = pytest.mark.gpu
F32 = RTOL["f32"]
BF16 = RTOL["bf16"]
# from this capacity on the bf16 first layer runs the row-split kernel
ROW_SPLIT_CAP = 2 * 256 * 256


def workload(name):
    if name in ("mid_f32", "mid_bf16"):
        base = synth.get("c1_f32" if name == "mid_f32" else "c2_bf16")
        return dataclasses.replace(base, name=name, index=11, batch=96, n_images=20_000, stream=-1)
    return synth.get(name)


def case(w, seed=3, zero=False):
    batch = synth.make_batch(w)
    dd = oracle.dedup(synth.occurrences(batch), w.n_images)
    Ws, bs = synth.make_weights(w)
    rng = np.random.default_rng(seed)
    sl = [np.zeros(d, np.float32) if zero else rng.uniform(-0.25, 0.5, d).astype(np.float32)
          for d in w.dims[1:-1]]
    return dd, Ws, bs, sl


def setup(w, dd, cap_extra=77, cap=None):
    n_u = dd["n_uniq"]
    cap = n_u + cap_extra if cap is None else cap
    T_dev = synth.table_rows(w, np.arange(w.n_images), device="cuda")
    uniq = torch.zeros(cap, dtype=torch.int32, device="cuda")
    uniq[:n_u] = torch.from_numpy(dd["uniq"].astype(np.int32)).cuda()
    nu = torch.tensor([n_u], dtype=torch.int32, device="cuda")
    return T_dev, uniq, nu, cap


def gpu_fwd(w, dd, Ws, bs, sl, cap=None):
    T_dev, uniq, nu, cap = setup(w, dd, cap=cap)
    mlp = ams.make_mlp(w.dims, w.dtype)
    h1dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    H1 = torch.full((cap, w.dims[1]), float("nan"), dtype=h1dt, device="cuda")
    H2 = torch.full((cap, w.dims[2]), float("nan"), device="cuda") if w.n_layers == 3 else None
    E = torch.full((cap, w.out_dim), float("nan"), device="cuda")
    ws = torch.empty(ams.ams_embed_workspace(mlp, cap), dtype=torch.uint8, device="cuda")
    ams.ams_embed_fwd(mlp, T_dev, uniq, nu, cap, [W.cuda() for W in Ws], [b.cuda() for b in bs], H1, H2, E, ws,
                      slopes=None if sl is None else [torch.from_numpy(s).cuda() for s in sl])
    torch.cuda.synchronize()
    n_u = dd["n_uniq"]
    return {"E": f64(E[:n_u]), "H1": f64(H1[:n_u]), "H2": f64(H2[:n_u]) if H2 is not None else None}


@pytest.mark.parametrize("name", ["tiny", "mid_f32", "c1_f32"])
def test_embed_prelu_forward(name):
    w = workload(name)
    dd, Ws, bs, sl = case(w)
    print(f"embed prelu fwd {name}: n_u={dd['n_uniq']}", flush=True)
    g = gpu_fwd(w, dd, Ws, bs, sl)
    X = synth.table_rows(w, dd["uniq"]).double().numpy()
    Z = oracle.dense_fwd(X, Ws, bs, sl)
    assert_close(g["H1"], Z[0], F32, "Z1 (saved)")
    if w.n_layers == 3:
        assert_close(g["H2"], Z[1], F32, "Z2 (saved)")
    assert_close(g["E"], Z[-1], F32, "E", rows=True)


def test_embed_prelu_slope_zero_is_relu():
    w = workload("mid_f32")
    dd, Ws, bs, sl = case(w, zero=True)
    p = gpu_fwd(w, dd, Ws, bs, sl)
    r = gpu_fwd(w, dd, Ws, bs, None)
    assert_close(p["E"], r["E"], 1e-6, "E (slope 0 vs ReLU)")
    assert_close(np.maximum(p["H1"], 0), r["H1"], 1e-6, "H1")


@pytest.mark.parametrize("name", ["tiny", "mid_f32"])
def test_embed_prelu_backward(name):
    w = workload(name)
    dd, Ws, bs, sl = case(w, seed=4)
    n_u = dd["n_uniq"]
    print(f"embed prelu bwd {name}: n_u={n_u}", flush=True)
    X = synth.table_rows(w, dd["uniq"]).double().numpy()
    Z = oracle.dense_fwd(X, Ws, bs, sl)
    Zf = [z.astype(np.float32) for z in Z[:-1]]             # what the GPU holds
    rng = np.random.default_rng(5)
    dE32 = rng.standard_normal((n_u, w.out_dim)).astype(np.float32)
    ref = oracle.dense_bwd(X, Ws, sl, [z.astype(np.float64) for z in Zf] + [Z[-1]], dE32)
    T_dev, uniq, nu, cap = setup(w, dd, cap_extra=40)
    mlp = ams.make_mlp(w.dims, "f32")
    H1 = torch.zeros((cap, w.dims[1]), device="cuda")
    H1[:n_u] = torch.from_numpy(Zf[0]).cuda()
    H2 = None
    if w.n_layers == 3:
        H2 = torch.zeros((cap, w.dims[2]), device="cuda")
        H2[:n_u] = torch.from_numpy(Zf[1]).cuda()
    dE = torch.zeros((cap, w.out_dim), device="cuda")
    dE[:n_u] = torch.from_numpy(dE32).cuda()
    dW = [torch.full((o, i), float("nan"), device="cuda") for i, o in zip(w.dims[:-1], w.dims[1:])]
    db = [torch.full((o,), float("nan"), device="cuda") for o in w.dims[1:]]
    ds = [torch.full((d,), float("nan"), device="cuda") for d in w.dims[1:-1]]
    ws = torch.empty(ams.ams_embed_workspace(mlp, cap), dtype=torch.uint8, device="cuda")
    ams.ams_embed_bwd(mlp, T_dev, uniq, nu, cap, [W.cuda() for W in Ws], H1, H2, None, dE, dW, db, ws,
                      slopes=[torch.from_numpy(s).cuda() for s in sl], dslopes=ds)
    torch.cuda.synchronize()
    for l in range(w.n_layers):
        assert_close(dW[l], ref["dW"][l], F32, f"dW{l + 1}")
        assert_close(db[l], ref["db"][l], F32, f"db{l + 1}")
    for l in range(w.n_layers - 1):
        assert_close(ds[l], ref["dslope"][l], F32, f"dslope{l + 1}")


def test_prelu_step_end_to_end_attentive():
    """A whole step with PReLU through Step.run (dedup, embed, attentive
    pooling and their backward) on the 96-sample 4096-256-64-12 batch.  The
    forward against the oracle's dense net and pooling.  The backward end to
    end against the oracle's whole chain (its pooling backward on its own
    forward, its dense backward on its own pre-activations), held to 1e-4
    plus twice the oracle's own sensitivity: the difference between that
    chain and the same chain on the GPU's forward outputs and saved
    pre-activations (which covers a PReLU branch taken the other way at a
    near-zero pre-activation).  That chained computation is also checked
    directly, at 1e-4, for every weight, bias and slope gradient."""
    w = workload("mid_f32")
    batch = synth.make_batch(w)
    Ws, bs = synth.make_weights(w)
    rng = np.random.default_rng(9)
    sl = [rng.uniform(-0.25, 0.5, d).astype(np.float32) for d in w.dims[1:-1]]
    n_beh, B = int(batch["seg_off"][-1]), w.batch
    T_dev = synth.table_rows(w, np.arange(w.n_images), device="cuda")
    st = ams.Step(w.dims, "f32", "att", B, n_beh, prelu=True)
    ids = torch.from_numpy(synth.occurrences(batch).astype(np.int32)).cuda()
    seg = torch.from_numpy(batch["seg_off"].astype(np.int32)).cuda()
    gU = torch.from_numpy(batch["g_u"]).cuda()
    gA = torch.from_numpy(batch["g_a"]).cuda()
    st.run(ids, w.n_images, T_dev, [W.cuda() for W in Ws], [b.cuda() for b in bs], seg, gU, gA,
           slopes=[torch.from_numpy(s).cuda() for s in sl])
    torch.cuda.synchronize()
    od = oracle.dedup(synth.occurrences(batch), w.n_images)
    n_u = od["n_uniq"]
    assert int(st.n_uniq.item()) == n_u and int(st.dev_status.item()) == 0
    np.testing.assert_array_equal(st.uniq[:n_u].cpu().numpy(), od["uniq"])
    X = synth.table_rows(w, od["uniq"]).double().numpy()
    Z = oracle.dense_fwd(X, Ws, bs, sl)
    E_g = f64(st.E[:n_u])
    assert_close(E_g, Z[-1], F32, "E", rows=True)
    pf = oracle.pool_fwd("att", batch["seg_off"], od["inv"], Z[-1])
    assert_close(st.U[:B], pf["U"], F32, "U", rows=True)
    # backward, chained on the GPU's own forward
    gfwd = {"U": f64(st.U[:B]), "A": f64(st.A[:B]), "w": f64(st.saved[:n_beh]),
            "argmax": np.full((B, w.out_dim), -1, np.int32)}
    pb = oracle.pool_bwd("att", batch["seg_off"], od["inv"], n_u, E_g, gfwd, batch["g_u"], batch["g_a"])
    assert_close(st.dE[:n_u], pb["dE"], F32, "dE", rows=True)
    Zg = [f64(st.H1[:n_u]), f64(st.H2[:n_u]), E_g]
    ref = oracle.dense_bwd(X, Ws, sl, Zg, f64(st.dE[:n_u]))
    for l in range(w.n_layers):
        assert_close(st.dW[l], ref["dW"][l], F32, f"dW{l + 1}")
        assert_close(st.db[l], ref["db"][l], F32, f"db{l + 1}")
    for l in range(w.n_layers - 1):
        assert_close(st.dslope[l], ref["dslope"][l], F32, f"dslope{l + 1}")
    # end to end: the whole float64 chain on the oracle's own values
    pb_o = oracle.pool_bwd("att", batch["seg_off"], od["inv"], n_u, Z[-1], pf, batch["g_u"], batch["g_a"])
    ref_o = oracle.dense_bwd(X, Ws, sl, Z, pb_o["dE"])
    assert_close_sensitive(st.dE[:n_u], pb_o["dE"], pb["dE"], F32, "dE", rows=True)
    for l in range(w.n_layers):
        assert_close_sensitive(st.dW[l], ref_o["dW"][l], ref["dW"][l], F32, f"dW{l + 1}")
        assert_close_sensitive(st.db[l], ref_o["db"][l], ref["db"][l], F32, f"db{l + 1}")
    for l in range(w.n_layers - 1):
        assert_close_sensitive(st.dslope[l], ref_o["dslope"][l], ref["dslope"][l], F32, f"dslope{l + 1}")


# ------------------------------------------------------------------ bf16

def f64w(Ws):
    """bf16 weights as the float64 arrays the oracle takes (exact)."""
    return [W.double().numpy() for W in Ws]


@pytest.mark.parametrize("name", ["mid_bf16", "c2_bf16", "row_split"])
def test_embed_prelu_forward_bf16(name):
    w = workload("mid_bf16" if name == "row_split" else name)
    dd, Ws, bs, sl = case(w)
    cap = ROW_SPLIT_CAP + 13 if name == "row_split" else None
    print(f"embed prelu fwd bf16 {name}: n_u={dd['n_uniq']} cap={cap}", flush=True)
    g = gpu_fwd(w, dd, Ws, bs, sl, cap=cap)
    X = synth.table_rows(w, dd["uniq"]).double().numpy()
    Z = oracle.dense_fwd(X, f64w(Ws), bs, sl)
    assert_close(g["H1"], Z[0], BF16, "Z1 (saved, bf16)")
    assert_close(g["H2"], Z[1], F32, "Z2 (saved)")
    assert_close(g["E"], Z[-1], F32, "E", rows=True)           # float32 accumulation throughout


def test_embed_prelu_slope_zero_is_relu_bf16():
    w = workload("mid_bf16")
    dd, Ws, bs, sl = case(w, zero=True)
    p = gpu_fwd(w, dd, Ws, bs, sl)
    r = gpu_fwd(w, dd, Ws, bs, None)
    assert_close(p["E"], r["E"], 1e-5, "E (slope 0 vs ReLU)")
    assert_close(np.maximum(p["H1"], 0), r["H1"], 1e-6, "H1")


def test_embed_prelu_backward_bf16():
    w = workload("mid_bf16")
    dd, Ws, bs, sl = case(w, seed=4)
    n_u = dd["n_uniq"]
    print(f"embed prelu bwd bf16: n_u={n_u}", flush=True)
    X = synth.table_rows(w, dd["uniq"]).double().numpy()
    Z = oracle.dense_fwd(X, f64w(Ws), bs, sl)
    Z1b = torch.from_numpy(Z[0]).to(torch.bfloat16)                      # what the GPU holds
    Z2f = Z[1].astype(np.float32)
    rng = np.random.default_rng(5)
    dE32 = rng.standard_normal((n_u, w.out_dim)).astype(np.float32)
    ref = oracle.dense_bwd(X, f64w(Ws), sl, [Z1b.double().numpy(), Z2f.astype(np.float64), Z[-1]], dE32)
    T_dev, uniq, nu, cap = setup(w, dd, cap_extra=40)
    mlp = ams.make_mlp(w.dims, "bf16")
    H1 = torch.zeros((cap, w.dims[1]), dtype=torch.bfloat16, device="cuda")
    H1[:n_u] = Z1b.cuda()
    H2 = torch.zeros((cap, w.dims[2]), device="cuda")
    H2[:n_u] = torch.from_numpy(Z2f).cuda()
    dE = torch.zeros((cap, w.out_dim), device="cuda")
    dE[:n_u] = torch.from_numpy(dE32).cuda()
    dW = [torch.full((o, i), float("nan"), device="cuda") for i, o in zip(w.dims[:-1], w.dims[1:])]
    db = [torch.full((o,), float("nan"), device="cuda") for o in w.dims[1:]]
    ds = [torch.full((d,), float("nan"), device="cuda") for d in w.dims[1:-1]]
    ws = torch.empty(ams.ams_embed_workspace(mlp, cap), dtype=torch.uint8, device="cuda")
    ams.ams_embed_bwd(mlp, T_dev, uniq, nu, cap, [W.cuda() for W in Ws], H1, H2, None, dE, dW, db, ws,
                      slopes=[torch.from_numpy(s).cuda() for s in sl], dslopes=ds)
    torch.cuda.synchronize()
    for l in range(w.n_layers):
        assert_close(dW[l], ref["dW"][l], BF16, f"dW{l + 1}")
        assert_close(db[l], ref["db"][l], BF16, f"db{l + 1}")
    for l in range(w.n_layers - 1):
        assert_close(ds[l], ref["dslope"][l], BF16, f"dslope{l + 1}")


def test_prelu_step_bf16_attentive():
    """Step.run with PReLU in bf16 on the 96-sample batch: forward against the
    oracle's dense net and pooling; backward chained on the GPU's own forward
    outputs and saved pre-activations (the oracle's dense backward on them)."""
    w = workload("mid_bf16")
    batch = synth.make_batch(w)
    Ws, bs = synth.make_weights(w)
    rng = np.random.default_rng(9)
    sl = [rng.uniform(-0.25, 0.5, d).astype(np.float32) for d in w.dims[1:-1]]
    n_beh, B = int(batch["seg_off"][-1]), w.batch
    T_dev = synth.table_rows(w, np.arange(w.n_images), device="cuda")
    st = ams.Step(w.dims, "bf16", "att", B, n_beh, prelu=True)
    ids = torch.from_numpy(synth.occurrences(batch).astype(np.int32)).cuda()
    seg = torch.from_numpy(batch["seg_off"].astype(np.int32)).cuda()
    gU = torch.from_numpy(batch["g_u"]).cuda()
    gA = torch.from_numpy(batch["g_a"]).cuda()
    st.run(ids, w.n_images, T_dev, [W.cuda() for W in Ws], [b.cuda() for b in bs], seg, gU, gA,
           slopes=[torch.from_numpy(s).cuda() for s in sl])
    torch.cuda.synchronize()
    od = oracle.dedup(synth.occurrences(batch), w.n_images)
    n_u = od["n_uniq"]
    assert int(st.n_uniq.item()) == n_u and int(st.dev_status.item()) == 0
    X = synth.table_rows(w, od["uniq"]).double().numpy()
    Z = oracle.dense_fwd(X, f64w(Ws), bs, sl)
    E_g = f64(st.E[:n_u])
    assert_close(E_g, Z[-1], F32, "E", rows=True)
    pf = oracle.pool_fwd("att", batch["seg_off"], od["inv"], Z[-1])
    assert_close(st.U[:B], pf["U"], F32, "U", rows=True)
    gfwd = {"U": f64(st.U[:B]), "A": f64(st.A[:B]), "w": f64(st.saved[:n_beh]),
            "argmax": np.full((B, w.out_dim), -1, np.int32)}
    pb = oracle.pool_bwd("att", batch["seg_off"], od["inv"], n_u, E_g, gfwd, batch["g_u"], batch["g_a"])
    assert_close(st.dE[:n_u], pb["dE"], F32, "dE", rows=True)
    Zg = [f64(st.H1[:n_u]), f64(st.H2[:n_u]), E_g]
    ref = oracle.dense_bwd(X, f64w(Ws), sl, Zg, f64(st.dE[:n_u]))
    for l in range(w.n_layers):
        assert_close(st.dW[l], ref["dW"][l], BF16, f"dW{l + 1}")
        assert_close(st.db[l], ref["db"][l], BF16, f"db{l + 1}")
    for l in range(w.n_layers - 1):
        assert_close(st.dslope[l], ref["dslope"][l], BF16, f"dslope{l + 1}")
