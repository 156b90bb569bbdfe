"""Pins for the float64 oracle, each against something other than the oracle.

Pins used: numpy.unique / stable argsort (dedup), a brute-force dict, torch
float64 nn.functional.linear and autograd over every occurrence (no dedup),
numpy reduceat (sum/max pooling), closed forms and special cases of attentive
pooling, central finite differences, and invariants that hold by the method's
definition (dedup is exact; gradients merged per image equal the sum of
per-occurrence gradients).
"""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_1711_06505_amd import synth
from tests.torch_ref import step_autograd


def small_case(seed=3, B=12, n_ids=40, dims=(64, 32, 16, 12), dtype="f32", lens=None):
    """A small batch with repeated IDs inside samples and ads among behaviors."""
    rng = np.random.default_rng(seed)
    if lens is None:
        lens = rng.integers(1, 9, size=B)
    seg = np.zeros(B + 1, np.int32)
    seg[1:] = np.cumsum(lens)
    beh = rng.integers(0, n_ids, size=int(seg[-1])).astype(np.int32)
    ad = rng.integers(0, n_ids, size=B).astype(np.int32)
    ad[0] = beh[0]  # an ad image that is also a behavior image
    D = dims[-1]
    batch = {"seg_off": seg, "beh_ids": beh, "ad_ids": ad,
             "g_u": rng.standard_normal((B, D)).astype(np.float32),
             "g_a": rng.standard_normal((B, D)).astype(np.float32)}
    T = torch.from_numpy(rng.standard_normal((n_ids, dims[0])).astype(np.float32))
    Ws, bs = [], []
    for fi, fo in zip(dims[:-1], dims[1:]):
        lim = np.sqrt(6.0 / (fi + fo))
        Ws.append(torch.from_numpy(rng.uniform(-lim, lim, (fo, fi)).astype(np.float32)))
        bs.append(torch.from_numpy(rng.uniform(-0.1, 0.1, fo).astype(np.float32)))
    if dtype == "bf16":
        T = T.to(torch.bfloat16)
        Ws = [W.to(torch.bfloat16) for W in Ws]
    return batch, T, Ws, bs


def rel_err(x, r):
    x = np.asarray(x, np.float64)
    r = np.asarray(r, np.float64)
    scale = max(np.abs(r).max(), 1e-300)
    return float(np.abs(x - r).max() / scale)


# ---------------------------------------------------------------- dedup

@pytest.mark.parametrize("name", ["tiny", "c1_f32", "c3_long"])
def test_dedup_matches_numpy_unique(name):
    w = synth.get(name)
    occ = synth.occurrences(synth.make_batch(w))
    d = oracle.dedup(occ, w.n_images)
    u, inv, cnt = np.unique(occ, return_inverse=True, return_counts=True)
    assert d["n_uniq"] == u.size
    np.testing.assert_array_equal(d["uniq"], u)
    np.testing.assert_array_equal(d["inv"], inv.reshape(-1))
    np.testing.assert_array_equal(d["uniq_off"], np.concatenate([[0], np.cumsum(cnt)]))
    np.testing.assert_array_equal(d["occ_perm"], np.argsort(occ, kind="stable"))


def test_dedup_brute_force_dict():
    occ = [7, 2, 7, 7, 0, 2, 9, 0, 7]
    d = oracle.dedup(occ, 10)
    positions = {}
    for k, v in enumerate(occ):
        positions.setdefault(v, []).append(k)
    keys = sorted(positions)
    assert list(d["uniq"]) == keys
    assert list(d["occ_perm"]) == [k for v in keys for k in positions[v]]
    assert list(d["uniq_off"]) == list(np.cumsum([0] + [len(positions[v]) for v in keys]))
    assert [keys[i] for i in d["inv"]] == occ


def test_dedup_invariants_and_edges():
    rng = np.random.default_rng(0)
    occ = rng.integers(0, 50, size=1000).astype(np.int32)
    d = oracle.dedup(occ, 50)
    assert np.all(np.diff(d["uniq"]) > 0)
    np.testing.assert_array_equal(d["uniq"][d["inv"]], occ)
    srt = occ[d["occ_perm"]]
    assert np.all(np.diff(srt) >= 0)
    for u in range(d["n_uniq"]):
        run = d["occ_perm"][d["uniq_off"][u]:d["uniq_off"][u + 1]]
        assert np.all(np.diff(run) > 0)
    e = oracle.dedup(np.zeros(0, np.int32), 5)
    assert e["n_uniq"] == 0 and list(e["uniq_off"]) == [0]
    with pytest.raises(IndexError):
        oracle.dedup([0, 5], 5)
    with pytest.raises(IndexError):
        oracle.dedup([-1], 5)


# ------------------------------------------------------------------ MLP

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_mlp_fwd_matches_torch_linear(dtype):
    batch, T, Ws, bs = small_case(dtype=dtype, dims=(96, 40, 24, 12))
    rows = np.array([3, 0, 39, 17, 17], np.int32)
    f = oracle.mlp_fwd(T, rows, Ws, bs)
    h = T.double()[torch.as_tensor(rows, dtype=torch.long)]
    for l, (W, b) in enumerate(zip(Ws, bs)):
        z = torch.nn.functional.linear(h, W.double(), b.double())
        assert rel_err(f["Z"][l], z.numpy()) < 1e-13
        h = torch.relu(z) if l < len(Ws) - 1 else z
    assert rel_err(f["E"], h.numpy()) < 1e-13


def test_mlp_fwd_closed_form_identity():
    # W = I, b = 0 for two layers: E = ReLU(x) exactly; with final_relu the same.
    x = torch.tensor([[1.5, -2.0, 0.0, 3.25], [-1.0, 4.0, -0.5, 0.125]], dtype=torch.float32)
    I = torch.eye(4)
    z = torch.zeros(4)
    f = oracle.mlp_fwd(x, [0, 1], [I, I], [z, z])
    np.testing.assert_array_equal(f["E"], np.maximum(x.numpy(), 0))
    # a bias shifts the output exactly; the last layer has no activation
    f2 = oracle.mlp_fwd(x, [1], [I, I], [z, torch.full((4,), -10.0)])
    np.testing.assert_array_equal(f2["E"], np.maximum(x.numpy()[1:], 0) - 10.0)
    f3 = oracle.mlp_fwd(x, [1], [I, I], [z, torch.full((4,), -10.0)], final_relu=True)
    np.testing.assert_array_equal(f3["E"], np.zeros((1, 4)))


def test_dedup_then_embed_equals_every_occurrence():
    w = synth.get("tiny")
    batch = synth.make_batch(w)
    occ = synth.occurrences(batch)
    T = synth.table_rows(w, np.arange(w.n_images))
    Ws, bs = synth.make_weights(w)
    d = oracle.dedup(occ, w.n_images)
    e_u = oracle.mlp_fwd(T, d["uniq"], Ws, bs)["E"]
    e_all = oracle.mlp_fwd(T, occ, Ws, bs)["E"]
    np.testing.assert_array_equal(e_u[d["inv"]], e_all)   # bitwise in float64


# ------------------------------------------------------------- pooling

def test_pool_sum_max_match_reduceat():
    batch, T, Ws, bs = small_case(seed=5, B=20)
    occ = np.concatenate([batch["beh_ids"], batch["ad_ids"]])
    d = oracle.dedup(occ, 40)
    E = oracle.mlp_fwd(T, d["uniq"], Ws, bs)["E"]
    seg = batch["seg_off"]
    e_beh = E[d["inv"][:seg[-1]]]
    s = oracle.pool_fwd("sum", seg, d["inv"], E)
    np.testing.assert_allclose(s["U"], np.add.reduceat(e_beh, seg[:-1], axis=0), rtol=1e-14, atol=1e-14)
    np.testing.assert_array_equal(s["A"], E[d["inv"][seg[-1]:]])
    m = oracle.pool_fwd("max", seg, d["inv"], E)
    np.testing.assert_array_equal(m["U"], np.maximum.reduceat(e_beh, seg[:-1], axis=0))
    # first position attaining the max (repeated images inside a sample tie exactly)
    for i in range(seg.size - 1):
        for dd in range(E.shape[1]):
            col = [E[d["inv"][j], dd] for j in range(seg[i], seg[i + 1])]
            assert m["argmax"][i, dd] == seg[i] + int(np.argmax(col))


def test_pool_att_brute_force_and_special_cases():
    batch, T, Ws, bs = small_case(seed=8, B=16)
    occ = np.concatenate([batch["beh_ids"], batch["ad_ids"]])
    d = oracle.dedup(occ, 40)
    E = oracle.mlp_fwd(T, d["uniq"], Ws, bs)["E"]
    seg = batch["seg_off"]
    r = oracle.pool_fwd("att", seg, d["inv"], E)
    for i in range(seg.size - 1):
        e = [E[d["inv"][j]] for j in range(seg[i], seg[i + 1])]
        a = E[d["inv"][seg[-1] + i]]
        s = [float(sum(x * y for x, y in zip(ej, a))) for ej in e]
        m = max(s)
        ex = [np.exp(v - m) for v in s]
        wts = [v / sum(ex) for v in ex]
        u = sum(wj * ej for wj, ej in zip(wts, e))
        assert rel_err(r["U"][i], u) < 1e-13
        assert abs(sum(r["w"][seg[i]:seg[i + 1]]) - 1.0) < 1e-14
    # a = 0 -> the segment mean; one behavior -> u = e; identical e_j -> u = e
    E2 = np.vstack([np.zeros(12), np.arange(12.0), np.arange(12.0)[::-1], np.ones(12)])
    seg2 = np.array([0, 2, 3, 5], np.int32)
    inv2 = np.array([1, 2, 3, 3, 3, 0, 1, 2], np.int32)
    r2 = oracle.pool_fwd("att", seg2, inv2, E2)
    np.testing.assert_allclose(r2["U"][0], (E2[1] + E2[2]) / 2, rtol=0, atol=1e-14)
    np.testing.assert_allclose(r2["U"][1], E2[3], rtol=0, atol=1e-15)
    np.testing.assert_allclose(r2["U"][2], E2[3], rtol=0, atol=1e-15)


def test_pool_bwd_sum_unit_grad_counts_multiplicity():
    w = synth.get("c1_f32")
    batch = synth.make_batch(w)
    occ = synth.occurrences(batch)
    d = oracle.dedup(occ, w.n_images)
    D = w.out_dim
    E = np.zeros((d["n_uniq"], D))
    B = batch["seg_off"].size - 1
    pf = oracle.pool_fwd("sum", batch["seg_off"], d["inv"], E)
    pb = oracle.pool_bwd("sum", batch["seg_off"], d["inv"], d["n_uniq"], E, pf,
                         np.ones((B, D)), np.zeros((B, D)))
    n_beh = batch["seg_off"][-1]
    mult = np.bincount(d["inv"][:n_beh], minlength=d["n_uniq"]).astype(np.float64)
    np.testing.assert_array_equal(pb["dE"], np.repeat(mult[:, None], D, axis=1))


@pytest.mark.parametrize("mode", ["sum", "att", "max"])
def test_pool_bwd_finite_differences(mode):
    batch, T, Ws, bs = small_case(seed=11, B=6, n_ids=15)
    occ = np.concatenate([batch["beh_ids"], batch["ad_ids"]])
    d = oracle.dedup(occ, 15)
    E = oracle.mlp_fwd(T, d["uniq"], Ws, bs)["E"]
    seg = batch["seg_off"]
    gU, gA = batch["g_u"].astype(np.float64), batch["g_a"].astype(np.float64)

    def loss(Ex):
        p = oracle.pool_fwd(mode, seg, d["inv"], Ex)
        return float((gU * p["U"]).sum() + (gA * p["A"]).sum())

    pf = oracle.pool_fwd(mode, seg, d["inv"], E)
    pb = oracle.pool_bwd(mode, seg, d["inv"], d["n_uniq"], E, pf, gU, gA)
    rng = np.random.default_rng(0)
    for _ in range(25):
        u, dd = int(rng.integers(d["n_uniq"])), int(rng.integers(E.shape[1]))
        h = 1e-6
        Ep, Em = E.copy(), E.copy()
        Ep[u, dd] += h
        Em[u, dd] -= h
        fd = (loss(Ep) - loss(Em)) / (2 * h)
        assert abs(fd - pb["dE"][u, dd]) <= 1e-6 * max(1.0, abs(fd)), (u, dd, fd, pb["dE"][u, dd])


def test_att_softmax_gradient_sums_to_zero():
    # sum_j ds_j = 0 per sample (softmax is invariant to a common shift of the
    # logits), and the per-occurrence gradient splits into w_j g + ds_j a.
    batch, T, Ws, bs = small_case(seed=13, B=10)
    occ = np.concatenate([batch["beh_ids"], batch["ad_ids"]])
    d = oracle.dedup(occ, 40)
    E = oracle.mlp_fwd(T, d["uniq"], Ws, bs)["E"]
    seg = batch["seg_off"]
    pf = oracle.pool_fwd("att", seg, d["inv"], E)
    gU = batch["g_u"].astype(np.float64)
    pb = oracle.pool_bwd("att", seg, d["inv"], d["n_uniq"], E, pf, gU, None)
    for i in range(seg.size - 1):
        js = range(seg[i], seg[i + 1])
        u = pf["U"][i]
        c = gU[i] @ u
        ds = [pf["w"][j] * (gU[i] @ E[d["inv"][j]] - c) for j in js]
        assert abs(sum(ds)) < 1e-12
        # ge_j - w_j g = ds_j a  (the rest of the per-occurrence gradient)
        for j, dsj in zip(js, ds):
            np.testing.assert_allclose(pb["ge"][j] - pf["w"][j] * gU[i], dsj * pf["A"][i], atol=1e-13)


# ---------------------------------------------------------- whole step

@pytest.mark.parametrize("mode", ["sum", "max", "att"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_step_matches_torch_autograd_every_occurrence(mode, dtype):
    batch, T, Ws, bs = small_case(seed=21, B=14, dtype=dtype)
    o = oracle.step(batch, 40, T, Ws, bs, mode)
    t = step_autograd(batch, T, Ws, bs, mode)
    assert rel_err(o["pool"]["U"], t["U"]) < 1e-12
    assert rel_err(o["pool"]["A"], t["A"]) < 1e-12
    assert rel_err(o["pool_bwd"]["ge"], t["ge"]) < 1e-12
    for l in range(len(Ws)):
        assert rel_err(o["bwd"]["dW"][l], t["dW"][l]) < 1e-11, l
        assert rel_err(o["bwd"]["db"][l], t["db"][l]) < 1e-11, l


def test_step_tiny_workload_matches_torch_autograd():
    w = synth.get("tiny")
    batch = synth.make_batch(w)
    T = synth.table_rows(w, np.arange(w.n_images))
    Ws, bs = synth.make_weights(w)
    o = oracle.step(batch, w.n_images, T, Ws, bs, "sum")
    t = step_autograd(batch, T, Ws, bs, "sum")
    assert rel_err(o["pool"]["U"], t["U"]) < 1e-12
    for l in range(len(Ws)):
        assert rel_err(o["bwd"]["dW"][l], t["dW"][l]) < 1e-11
        assert rel_err(o["bwd"]["db"][l], t["db"][l]) < 1e-11


def test_final_relu_variant_matches_torch_autograd():
    batch, T, Ws, bs = small_case(seed=23, B=9)
    o = oracle.step(batch, 40, T, Ws, bs, "att", final_relu=True)
    t = step_autograd(batch, T, Ws, bs, "att", final_relu=True)
    assert rel_err(o["pool"]["U"], t["U"]) < 1e-12
    for l in range(len(Ws)):
        assert rel_err(o["bwd"]["dW"][l], t["dW"][l]) < 1e-11


@pytest.mark.parametrize("mode", ["sum", "att"])
def test_weight_gradients_finite_differences(mode):
    batch, T, Ws, bs = small_case(seed=31, B=7, n_ids=20, dims=(32, 16, 8, 12))
    o = oracle.step(batch, 20, T, Ws, bs, mode)
    gU, gA = batch["g_u"].astype(np.float64), batch["g_a"].astype(np.float64)
    W64 = [W.double() for W in Ws]
    b64 = [b.double() for b in bs]

    def loss(Wx, bx):
        # the oracle reads float32 storage: perturb in float64 and feed as
        # float64 -> float32 would round, so evaluate through float64 tables.
        occ = np.concatenate([batch["beh_ids"], batch["ad_ids"]])
        d = oracle.dedup(occ, 20)
        h = T.double()[torch.as_tensor(d["uniq"], dtype=torch.long)]
        for l in range(len(Wx)):
            h = torch.nn.functional.linear(h, Wx[l], bx[l])
            if l < len(Wx) - 1:
                h = torch.relu(h)
        p = oracle.pool_fwd(mode, batch["seg_off"], d["inv"], h.numpy())
        return float((gU * p["U"]).sum() + (gA * p["A"]).sum())

    rng = np.random.default_rng(1)
    for l in range(len(Ws)):
        for _ in range(6):
            o_, i_ = int(rng.integers(W64[l].shape[0])), int(rng.integers(W64[l].shape[1]))
            h = 1e-6
            Wp = [x.clone() for x in W64]
            Wm = [x.clone() for x in W64]
            Wp[l][o_, i_] += h
            Wm[l][o_, i_] -= h
            fd = (loss(Wp, b64) - loss(Wm, b64)) / (2 * h)
            an = o["bwd"]["dW"][l][o_, i_]
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(fd)), (l, o_, i_, fd, an)
        o_ = int(rng.integers(b64[l].shape[0]))
        bp = [x.clone() for x in b64]
        bm = [x.clone() for x in b64]
        bp[l][o_] += 1e-6
        bm[l][o_] -= 1e-6
        fd = (loss(W64, bp) - loss(W64, bm)) / 2e-6
        assert abs(fd - o["bwd"]["db"][l][o_]) <= 1e-6 * max(1.0, abs(fd))


def test_merged_gradient_equals_sum_over_occurrences():
    batch, T, Ws, bs = small_case(seed=41, B=15)
    occ = np.concatenate([batch["beh_ids"], batch["ad_ids"]])
    o = oracle.step(batch, 40, T, Ws, bs, "att")
    # backprop every occurrence separately with its own embedding gradient
    f_all = oracle.mlp_fwd(T, occ, Ws, bs)
    b_all = oracle.mlp_bwd(T, occ, Ws, f_all, o["pool_bwd"]["ge"])
    for l in range(len(Ws)):
        assert rel_err(b_all["dW"][l], o["bwd"]["dW"][l]) < 1e-12
        assert rel_err(b_all["db"][l], o["bwd"]["db"][l]) < 1e-12


def test_oracle_independent_of_thread_count():
    batch, T, Ws, bs = small_case(seed=51, B=30)
    n0 = oracle.num_threads()
    try:
        oracle.set_threads(1)
        a = oracle.step(batch, 40, T, Ws, bs, "att")
        oracle.set_threads(max(n0, 4))
        b = oracle.step(batch, 40, T, Ws, bs, "att")
    finally:
        oracle.set_threads(n0)
    for l in range(len(Ws)):
        np.testing.assert_array_equal(a["bwd"]["dW"][l], b["bwd"]["dW"][l])
    np.testing.assert_array_equal(a["pool"]["U"], b["pool"]["U"])
