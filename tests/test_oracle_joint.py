"""Pins for the joint-step part of the float64 oracle (bags, CTR MLP with
softmax cross-entropy, merged ID-row gradients, sparse Adagrad), each against
something other than the oracle: torch float64 autograd and embedding_bag,
brute-force loops, closed forms of softmax cross-entropy and of Adagrad, and
central finite differences of the oracle's own forward.
"""
import math

import numpy as np
import torch

from oracle import oracle
from paper_1711_06505_amd import synth
from tests.torch_ref import joint_autograd


def rel_err(x, r):
    x = np.asarray(x, np.float64)
    r = np.asarray(r, np.float64)
    return float(np.abs(x - r).max() / max(np.abs(r).max(), 1e-300))


def joint_case(seed=5, B=10, n_img=30, n_rows=(50, 7), dims=(32, 16, 8), hidden=(12, 6), mode_lens=None,
               query_table=None):
    rng = np.random.default_rng(seed)
    lens = rng.integers(1, 7, size=B) if mode_lens is None else np.asarray(mode_lens)
    seg = np.zeros(B + 1, np.int32)
    seg[1:] = np.cumsum(lens)
    n_beh = int(seg[-1])
    beh = rng.integers(0, n_img, size=n_beh).astype(np.int32)
    ad = rng.integers(0, n_img, size=B).astype(np.int32)
    ad[0] = beh[0]
    batch = {"seg_off": seg, "beh_ids": beh, "ad_ids": ad}
    jb = {"beh_ids": [rng.integers(0, N, size=n_beh).astype(np.int32) for N in n_rows],
          "ad_ids": [rng.integers(0, N, size=B).astype(np.int32) for N in n_rows],
          "labels": rng.integers(0, 2, size=B).astype(np.int32)}
    jb["ad_ids"][0][1] = jb["beh_ids"][0][2]          # an ad ID that is also a behavior ID
    T = torch.from_numpy(rng.standard_normal((n_img, dims[0])).astype(np.float32))
    Ws, bs = [], []
    for fi, fo in zip(dims[:-1], dims[1:]):
        lim = math.sqrt(6.0 / (fi + fo))
        Ws.append(torch.from_numpy(rng.uniform(-lim, lim, (fo, fi)).astype(np.float32)))
        bs.append(torch.from_numpy(rng.uniform(-0.1, 0.1, fo).astype(np.float32)))
    tabs = [rng.standard_normal((N, 12)).astype(np.float32) * 0.3 for N in n_rows]
    cd = ((2 if query_table is None else 3) * dims[-1] + 12 * len(n_rows),) + tuple(hidden) + (2,)
    cW, cb = [], []
    for fi, fo in zip(cd[:-1], cd[1:]):
        lim = math.sqrt(6.0 / (fi + fo))
        cW.append(torch.from_numpy(rng.uniform(-lim, lim, (fo, fi)).astype(np.float32)))
        cb.append(torch.from_numpy(rng.uniform(-0.1, 0.1, fo).astype(np.float32)))
    spec = synth.JointSpec(tuple(n_rows), 12, 1.0, tuple(hidden), 2, 0.5, lr=0.01, eps=1e-8)
    return batch, jb, T, Ws, bs, tabs, cW, cb, spec


def oracle_joint(batch, jb, T, Ws, bs, tabs, cW, cb, spec, accum=None, mode="att", query_table=None):
    rows, acc = [], []
    for t, tab in enumerate(tabs):
        u = oracle.dedup(np.concatenate([jb["beh_ids"][t], jb["ad_ids"][t]]), tab.shape[0])["uniq"]
        rows.append(tab[u])
        acc.append(np.zeros((u.size, 12)) if accum is None else accum[t][u])
    return oracle.joint_step(batch, jb, spec, T.shape[0], T, Ws, bs, rows, cW, cb, acc, mode=mode,
                             table_is_compact=False, query_table=query_table)


# ------------------------------------------------------------------ bags

def test_bag_fwd_matches_embedding_bag_and_brute_force():
    rng = np.random.default_rng(1)
    B, N = 9, 40
    lens = np.array([3, 0, 1, 7, 2, 5, 1, 4, 6])
    seg = np.zeros(B + 1, np.int32)
    seg[1:] = np.cumsum(lens)
    idx = rng.integers(0, N, size=int(seg[-1]) + B).astype(np.int32)
    tab = rng.standard_normal((N, 12)).astype(np.float32)
    got = oracle.bag_fwd(seg, idx, tab)
    n_beh = int(seg[-1])
    brute = np.zeros((B, 12))
    for i in range(B):
        for j in range(seg[i], seg[i + 1]):
            brute[i] += tab[idx[j]].astype(np.float64)
        brute[i] += tab[idx[n_beh + i]].astype(np.float64)
    assert np.array_equal(got, brute)
    flat, offs = [], []
    for i in range(B):
        offs.append(len(flat))
        flat += list(idx[seg[i]:seg[i + 1]]) + [idx[n_beh + i]]
    ref = torch.nn.functional.embedding_bag(torch.as_tensor(flat, dtype=torch.int64),
                                            torch.from_numpy(tab).double(), torch.as_tensor(offs), mode="sum")
    assert rel_err(got, ref.numpy()) < 1e-14


def test_bag_fwd_rejects_out_of_range_rows():
    seg = np.array([0, 2], np.int32)
    tab = np.zeros((5, 12), np.float32)
    for bad in (5, -1):
        try:
            oracle.bag_fwd(seg, np.array([0, bad, 1], np.int32), tab)
        except IndexError:
            continue
        raise AssertionError("out-of-range row accepted")


# --------------------------------------------------------------- CTR MLP

def test_ctr_matches_torch_autograd():
    rng = np.random.default_rng(7)
    B, dims = 37, (30, 20, 9, 2)
    X = rng.standard_normal((B, dims[0])) * 0.7
    y = rng.integers(0, 2, size=B).astype(np.int32)
    Ws = [torch.from_numpy(rng.uniform(-0.4, 0.4, (fo, fi)).astype(np.float32)) for fi, fo in zip(dims[:-1], dims[1:])]
    bs = [torch.from_numpy(rng.uniform(-0.1, 0.1, fo).astype(np.float32)) for fo in dims[1:]]
    o = oracle.ctr_fwd_bwd(X, y, Ws, bs)
    Xt = torch.from_numpy(X).requires_grad_()
    Wt = [W.double().requires_grad_() for W in Ws]
    bt = [b.double().requires_grad_() for b in bs]
    z = Xt
    for l in range(3):
        z = torch.nn.functional.linear(z, Wt[l], bt[l])
        if l < 2:
            z = torch.relu(z)
    loss = torch.nn.functional.cross_entropy(z, torch.as_tensor(y, dtype=torch.int64))
    loss.backward()
    assert abs(o["loss"] - float(loss.detach())) < 1e-13
    assert rel_err(o["prob"], torch.softmax(z, 1).detach().numpy()) < 1e-13
    assert rel_err(o["dX"], Xt.grad.numpy()) < 1e-12
    for l in range(3):
        assert rel_err(o["dW"][l], Wt[l].grad.numpy()) < 1e-12
        assert rel_err(o["db"][l], bt[l].grad.numpy()) < 1e-12


def test_ctr_zero_model_closed_form():
    """All weights and biases zero: logits 0, p = 1/2, loss = ln 2; only the
    last bias gets a gradient, sum_i (1/2 - [y_i = c]) / B; nothing reaches X."""
    rng = np.random.default_rng(2)
    B, dims = 16, (10, 6, 2)
    X = rng.standard_normal((B, 10))
    y = rng.integers(0, 2, size=B).astype(np.int32)
    Ws = [torch.zeros(fo, fi) for fi, fo in zip(dims[:-1], dims[1:])]
    bs = [torch.zeros(fo) for fo in dims[1:]]
    o = oracle.ctr_fwd_bwd(X, y, Ws, bs)
    assert abs(o["loss"] - math.log(2.0)) < 1e-15
    assert np.all(o["prob"] == 0.5)
    n1 = int(y.sum())
    assert np.allclose(o["db"][-1], [(0.5 * B - (B - n1)) / B, (0.5 * B - n1) / B], rtol=0, atol=1e-15)
    assert not o["dX"].any() and not o["dW"][0].any() and not o["db"][0].any()


def test_ctr_large_logits_are_stable():
    """Max subtraction: logits of +-800 give finite probabilities and loss."""
    X = np.array([[1.0], [-1.0]])
    Ws = [torch.tensor([[800.0], [-800.0]])]
    bs = [torch.zeros(2)]
    o = oracle.ctr_fwd_bwd(X, np.array([1, 1], np.int32), Ws, bs)
    assert np.isfinite(o["loss"]) and abs(o["loss"] - 800.0) < 1e-9      # (0 + 1600) / 2
    assert np.all(np.isfinite(o["prob"]))


# ----------------------------------------------------- merged row gradients

def test_merged_row_grad_matches_embedding_bag_backward():
    rng = np.random.default_rng(4)
    B, N = 11, 25
    lens = rng.integers(0, 6, size=B)
    seg = np.zeros(B + 1, np.int32)
    seg[1:] = np.cumsum(lens)
    n_beh = int(seg[-1])
    occ = rng.integers(0, N, size=n_beh + B).astype(np.int32)
    dbag = rng.standard_normal((B, 12))
    dd = oracle.dedup(occ, N)
    g = oracle.merged_row_grad(seg, dd["inv"], dd["n_uniq"], dbag)
    tab = torch.zeros((N, 12), dtype=torch.float64, requires_grad=True)
    flat, offs = [], []
    for i in range(B):
        offs.append(len(flat))
        flat += list(occ[seg[i]:seg[i + 1]]) + [occ[n_beh + i]]
    out = torch.nn.functional.embedding_bag(torch.as_tensor(flat, dtype=torch.int64), tab,
                                            torch.as_tensor(offs), mode="sum")
    (out * torch.from_numpy(dbag)).sum().backward()
    dense = tab.grad.numpy()
    assert rel_err(g, dense[dd["uniq"]]) < 1e-14
    untouched = np.setdiff1d(np.arange(N), dd["uniq"])
    assert not dense[untouched].any()


# --------------------------------------------------------------- Adagrad

def test_adagrad_first_step_is_lr_times_sign():
    """From a zero accumulator, one step moves each coordinate by lr * g /
    (|g| + eps): lr * sign(g) up to eps, and nothing where g = 0."""
    rng = np.random.default_rng(9)
    g = rng.standard_normal((6, 12))
    g[2, 3] = 0.0
    rows = rng.standard_normal((6, 12))
    new, acc = oracle.adagrad_rows(g, rows, np.zeros((6, 12)), lr=0.01, eps=1e-8)
    step = rows - new
    assert np.allclose(step, 0.01 * np.sign(g), rtol=0, atol=0.01 * 1e-8 / np.abs(g[g != 0]).min() + 1e-16)
    assert step[2, 3] == 0.0 and acc[2, 3] == 0.0
    assert np.array_equal(acc, g * g)


def test_adagrad_repeated_gradient_follows_harmonic_sqrt_sum():
    """k steps with the same gradient from a zero accumulator (eps = 0): the
    accumulator is m g^2 after step m, so the total move is
    lr * sign(g) * sum_{m=1..k} 1 / sqrt(m)."""
    rng = np.random.default_rng(11)
    g = rng.standard_normal((3, 12))
    rows0 = rng.standard_normal((3, 12))
    rows, acc = rows0.copy(), np.zeros((3, 12))
    k = 7
    for _ in range(k):
        rows, acc = oracle.adagrad_rows(g, rows, acc, lr=0.05, eps=0.0)
    expect = 0.05 * np.sign(g) * sum(1.0 / math.sqrt(m) for m in range(1, k + 1))
    assert np.allclose(rows0 - rows, expect, rtol=1e-13, atol=0)
    assert np.allclose(acc, k * g * g, rtol=1e-14, atol=0)


# ------------------------------------------------------------ whole step

def test_joint_step_matches_torch_autograd():
    batch, jb, T, Ws, bs, tabs, cW, cb, spec = joint_case()
    o = oracle_joint(batch, jb, T, Ws, bs, tabs, cW, cb, spec)
    r = joint_autograd(batch, jb, T, Ws, bs, tabs, cW, cb)
    assert abs(o["ctr"]["loss"] - r["loss"]) < 1e-13
    assert rel_err(o["pool"]["U"], r["U"]) < 1e-12
    for t in range(2):
        assert rel_err(o["bags"][t], r["bags"][t]) < 1e-13
        u = o["id_dedup"][t]["uniq"]
        assert rel_err(o["row_grads"][t], r["id_grad"][t][u]) < 1e-12
    assert rel_err(o["ctr"]["dX"], r["dX"]) < 1e-12
    for l in range(3):
        assert rel_err(o["ctr"]["dW"][l], r["ctr_dW"][l]) < 1e-12
        assert rel_err(o["ctr"]["db"][l], r["ctr_db"][l]) < 1e-12
    for l in range(2):
        assert rel_err(o["bwd"]["dW"][l], r["dW"][l]) < 1e-11
        assert rel_err(o["bwd"]["db"][l], r["db"][l]) < 1e-11


def test_joint_step_sum_pooling_matches_torch_autograd():
    batch, jb, T, Ws, bs, tabs, cW, cb, spec = joint_case(seed=8, B=7)
    o = oracle_joint(batch, jb, T, Ws, bs, tabs, cW, cb, spec, mode="sum")
    r = joint_autograd(batch, jb, T, Ws, bs, tabs, cW, cb, mode="sum")
    assert abs(o["ctr"]["loss"] - r["loss"]) < 1e-13
    for l in range(2):
        assert rel_err(o["bwd"]["dW"][l], r["dW"][l]) < 1e-11


def test_joint_step_row_gradients_by_finite_differences():
    """dLoss/dtable[r][d] by central differences of the oracle's forward
    (bags -> CTR loss) equals the merged row gradient."""
    batch, jb, T, Ws, bs, tabs, cW, cb, spec = joint_case(seed=6, B=8)
    o = oracle_joint(batch, jb, T, Ws, bs, tabs, cW, cb, spec)
    X0 = o["X"]
    D = o["pool"]["U"].shape[1]

    def loss_with(t, r, d, delta):
        tab = tabs[t].astype(np.float64).copy()
        tab[r, d] += delta
        occ = np.concatenate([jb["beh_ids"][t], jb["ad_ids"][t]])
        bag = oracle.bag_fwd(batch["seg_off"], occ, tab)
        X = X0.copy()
        X[:, 2 * D + 12 * t:2 * D + 12 * (t + 1)] = bag
        return oracle.ctr_fwd_bwd(X, jb["labels"], cW, cb)["loss"]

    rng = np.random.default_rng(0)
    for t in range(2):
        u_all = o["id_dedup"][t]["uniq"]
        for _ in range(4):
            ui = int(rng.integers(0, u_all.size))
            d = int(rng.integers(0, 12))
            # the tables are float32: a power-of-two step keeps x +- h exact
            h = 2.0 ** -10
            fd = (loss_with(t, u_all[ui], d, h) - loss_with(t, u_all[ui], d, -h)) / (2 * h)
            g = o["row_grads"][t][ui, d]
            assert abs(fd - g) <= 1e-5 * max(1.0, abs(g)), (t, ui, d, fd, g)


def test_joint_mqap_matches_torch_autograd():
    """MultiQueryAttentivePooling (section 5.2): the second attentive channel
    takes each ad's row of ID table 1 as its query; loss, CTR input and its
    gradient, every ID table's row gradients (the query table's including the
    query gradient of the ad rows) and the image model's gradients against
    torch autograd over the whole chain.  Image embeddings are 12 wide, the
    query's width."""
    batch, jb, T, Ws, bs, tabs, cW, cb, spec = joint_case(seed=21, dims=(32, 16, 12), query_table=1)
    o = oracle_joint(batch, jb, T, Ws, bs, tabs, cW, cb, spec, query_table=1)
    r = joint_autograd(batch, jb, T, Ws, bs, tabs, cW, cb, query_table=1)
    assert o["X"].shape[1] == 3 * 12 + 2 * 12
    assert abs(o["ctr"]["loss"] - r["loss"]) < 1e-13
    assert rel_err(o["X"], r["X"]) < 1e-13
    assert rel_err(o["ctr"]["dX"], r["dX"]) < 1e-12
    for t in range(2):
        u = o["id_dedup"][t]["uniq"]
        assert rel_err(o["row_grads"][t], r["id_grad"][t][u]) < 1e-12
    for l in range(2):
        assert rel_err(o["bwd"]["dW"][l], r["dW"][l]) < 1e-11
        assert rel_err(o["bwd"]["db"][l], r["db"][l]) < 1e-11
    # the query gradient is really there: without it table 1's ad rows differ
    plain = oracle.merged_row_grad(batch["seg_off"], o["id_dedup"][1]["inv"], o["id_dedup"][1]["n_uniq"],
                                   o["dbags"][1])
    assert rel_err(plain, o["row_grads"][1]) > 1e-3


def test_joint_mqap_query_rows_by_finite_differences():
    """dLoss/dtable_q[r][d] by central differences of the oracle's forward
    (the row enters a bag and, for the samples whose ad it is, the query of
    the ID channel) equals the merged row gradient of the query table."""
    batch, jb, T, Ws, bs, tabs, cW, cb, spec = joint_case(seed=22, B=9, dims=(32, 16, 12), query_table=1)
    o = oracle_joint(batch, jb, T, Ws, bs, tabs, cW, cb, spec, query_table=1)
    X0, E = o["X"], o["fwd"]["E"]
    D = 12
    inv_img = o["dedup"]["inv"]
    occ = np.concatenate([jb["beh_ids"][1], jb["ad_ids"][1]])

    def loss_with(r, d, delta):
        tab = tabs[1].astype(np.float64).copy()
        tab[r, d] += delta
        X = X0.copy()
        Q = tab[jb["ad_ids"][1]]
        X[:, D:2 * D] = oracle.pool_query_fwd(batch["seg_off"], inv_img, E, Q)["U"]
        X[:, 3 * D + 12:3 * D + 24] = oracle.bag_fwd(batch["seg_off"], occ, tab)
        return oracle.ctr_fwd_bwd(X, jb["labels"], cW, cb)["loss"]

    u_all = o["id_dedup"][1]["uniq"]
    ads = set(jb["ad_ids"][1].tolist())
    picks = [k for k, r in enumerate(u_all) if r in ads][:3] + [k for k, r in enumerate(u_all) if r not in ads][:1]
    assert len(picks) == 4
    for ui in picks:
        for d in (0, 5, 11):
            h = 2.0 ** -10
            fd = (loss_with(u_all[ui], d, h) - loss_with(u_all[ui], d, -h)) / (2 * h)
            g = o["row_grads"][1][ui, d]
            assert abs(fd - g) <= 1e-5 * max(1.0, abs(g)), (ui, d, fd, g)


def test_joint_step_adagrad_applies_to_touched_rows_only():
    batch, jb, T, Ws, bs, tabs, cW, cb, spec = joint_case(seed=12)
    rng = np.random.default_rng(3)
    accum = [rng.uniform(0.0, 0.5, size=tab.shape) for tab in tabs]
    o = oracle_joint(batch, jb, T, Ws, bs, tabs, cW, cb, spec, accum=accum)
    for t in range(2):
        u = o["id_dedup"][t]["uniq"]
        g = o["row_grads"][t]
        assert np.allclose(o["new_accum"][t], accum[t][u] + g * g, rtol=1e-15, atol=0)
        # the move is against the gradient and never larger than lr
        move = tabs[t][u].astype(np.float64) - o["new_rows"][t]
        assert np.all(move * g >= 0) and np.all(np.abs(move) <= spec.lr + 1e-15)


def test_joint_workloads_are_well_formed():
    for name in ("tiny_joint", "tiny_mqap"):
        w = synth.get(name)
        b = synth.make_batch(w)
        jb = synth.make_joint(w, b)
        n_img = 3 if w.joint.query_table >= 0 else 2
        assert synth.ctr_dims(w)[0] == n_img * w.out_dim + 12 * len(w.joint.id_rows)
        if w.joint.query_table >= 0:
            assert w.joint.id_dim == w.out_dim            # the query meets the image embeddings
        for t, N in enumerate(w.joint.id_rows):
            occ = synth.joint_occurrences(jb, t)
            assert occ.size == int(b["seg_off"][-1]) + w.batch
            assert occ.min() >= 0 and occ.max() < N
        assert set(np.unique(jb["labels"])) <= {0, 1}
    assert synth.ctr_dims("c4_joint") == (60, 200, 80, 2)
