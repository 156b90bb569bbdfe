"""Pins for the oracle's concatenate aggregator (section 5.2), its dense nets
with PReLU (section 7.2) and the pre-rank score of section 6.

Concatenation: float64 torch autograd over every occurrence (no dedup,
per-sample padding and truncation), and the invariant that with Lc at least
the longest behavior list the positions add up to sum pooling (forward) and
a gradient repeated over the positions gives sum pooling's backward.
Dense nets: torch autograd with torch's prelu, slope 0 equal to ReLU, slope 1
collapsing the net into one affine map (a closed form), and the CTR model
with ReLU equal to the oracle's pinned CTR routine.
Pre-rank: torch autograd with torch's logistic loss, the closed form of
linear towers (a bilinear score), and central differences of the loss in
the inputs."""
import numpy as np
import torch

from oracle import oracle

F = torch.nn.functional


def _concat_case(seed=0):
    rng = np.random.default_rng(seed)
    lens = np.array([0, 1, 3, 5, 7, 2, 9, 4])
    B, D, Lc, n_u = lens.size, 5, 5, 11
    seg = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    n_beh = int(seg[-1])
    inv = rng.integers(0, n_u, n_beh + B).astype(np.int32)
    E = rng.standard_normal((n_u, D))
    return seg, inv, E, B, D, Lc, n_u, n_beh, rng


def test_concat_matches_torch_autograd_per_occurrence():
    seg, inv, E, B, D, Lc, n_u, n_beh, rng = _concat_case()
    gU = rng.standard_normal((B, Lc * D))
    gA = rng.standard_normal((B, D))
    Et = torch.tensor(E, requires_grad=True)
    rows = Et[torch.as_tensor(inv, dtype=torch.long)]            # every occurrence
    U = []
    for i in range(B):
        e = rows[seg[i]:seg[i + 1]][:Lc]
        U.append(F.pad(e, (0, 0, 0, Lc - e.shape[0])).reshape(-1))
    U = torch.stack(U)
    A = rows[n_beh:]
    (U * torch.tensor(gU)).sum().add((A * torch.tensor(gA)).sum()).backward()
    f = oracle.pool_concat_fwd(seg, inv, E, Lc)
    assert np.abs(f["U"] - U.detach().numpy()).max() < 1e-15
    assert np.abs(f["A"] - A.detach().numpy()).max() < 1e-15
    dE = oracle.pool_concat_bwd(seg, inv, n_u, D, Lc, gU, gA)
    assert np.abs(dE - Et.grad.numpy()).max() < 1e-13


def test_concat_with_room_for_every_behavior_is_sum_pooling():
    seg, inv, E, B, D, _, n_u, n_beh, rng = _concat_case(1)
    Lc = int(np.diff(seg).max()) + 2
    f = oracle.pool_concat_fwd(seg, inv, E, Lc)
    s = oracle.pool_fwd("sum", seg, inv, E)
    assert np.abs(f["U"].reshape(B, Lc, D).sum(1) - s["U"]).max() < 1e-12
    g = rng.standard_normal((B, D))
    gA = rng.standard_normal((B, D))
    dE = oracle.pool_concat_bwd(seg, inv, n_u, D, Lc, np.tile(g, (1, Lc)), gA)
    ds = oracle.pool_bwd("sum", seg, inv, n_u, E, s, g, gA)["dE"]
    assert np.abs(dE - ds).max() < 1e-12


def _net(rng, dims, prelu=True):
    Ws = [(rng.standard_normal((o, i)) / np.sqrt(i)).astype(np.float32) for i, o in zip(dims[:-1], dims[1:])]
    bs = [(rng.standard_normal(o) * 0.1).astype(np.float32) for o in dims[1:]]
    sl = [rng.uniform(-0.3, 0.6, o).astype(np.float32) for o in dims[1:-1]] if prelu else None
    return Ws, bs, sl


def _torch_net(X, Ws, bs, sl):
    h = X
    Wt = [torch.tensor(W, dtype=torch.float64, requires_grad=True) for W in Ws]
    bt = [torch.tensor(b, dtype=torch.float64, requires_grad=True) for b in bs]
    st = [torch.tensor(s, dtype=torch.float64, requires_grad=True) for s in sl] if sl else []
    for l in range(len(Ws)):
        h = F.linear(h, Wt[l], bt[l])
        if l < len(Ws) - 1:
            h = F.prelu(h, st[l]) if sl else F.relu(h)
    return h, Wt, bt, st


def test_dense_prelu_matches_torch_autograd():
    rng = np.random.default_rng(2)
    dims = [7, 9, 6, 3]
    Ws, bs, sl = _net(rng, dims)
    X = rng.standard_normal((13, 7))
    g = rng.standard_normal((13, 3))
    Xt = torch.tensor(X, requires_grad=True)
    out, Wt, bt, st = _torch_net(Xt, Ws, bs, sl)
    (out * torch.tensor(g)).sum().backward()
    Z = oracle.dense_fwd(X, Ws, bs, sl)
    assert np.abs(Z[-1] - out.detach().numpy()).max() < 1e-13
    r = oracle.dense_bwd(X, Ws, sl, Z, g)
    for l in range(3):
        assert np.abs(r["dW"][l] - Wt[l].grad.numpy()).max() < 1e-12
        assert np.abs(r["db"][l] - bt[l].grad.numpy()).max() < 1e-12
    for l in range(2):
        assert np.abs(r["dslope"][l] - st[l].grad.numpy()).max() < 1e-12
    assert np.abs(r["dX"] - Xt.grad.numpy()).max() < 1e-12


def test_dense_slope_zero_is_relu_and_slope_one_is_affine():
    rng = np.random.default_rng(3)
    dims = [6, 8, 5, 4]
    Ws, bs, _ = _net(rng, dims, prelu=False)
    X = rng.standard_normal((10, 6))
    zero = [np.zeros(d, np.float32) for d in dims[1:-1]]
    one = [np.ones(d, np.float32) for d in dims[1:-1]]
    assert np.array_equal(oracle.dense_fwd(X, Ws, bs, zero)[-1], oracle.dense_fwd(X, Ws, bs, None)[-1])
    # slope 1: the whole net is X M^T + c with M = W2 W1 W0, c = (b0 W1^T + b1) W2^T + b2
    W = [w.astype(np.float64) for w in Ws]
    b = [x.astype(np.float64) for x in bs]
    M = W[2] @ W[1] @ W[0]
    c = (b[0] @ W[1].T + b[1]) @ W[2].T + b[2]
    assert np.abs(oracle.dense_fwd(X, Ws, bs, one)[-1] - (X @ M.T + c)).max() < 1e-12
    g = rng.standard_normal((10, 4))
    r = oracle.dense_bwd(X, Ws, one, oracle.dense_fwd(X, Ws, bs, one), g)
    assert np.abs(r["dX"] - g @ M).max() < 1e-12


def test_ctr_with_relu_equals_the_pinned_ctr_routine():
    rng = np.random.default_rng(4)
    dims = [10, 12, 7, 2]
    Ws, bs, _ = _net(rng, dims, prelu=False)
    X = rng.standard_normal((21, 10))
    y = rng.integers(0, 2, 21)
    a = oracle.ctr_act_fwd_bwd(X, y, Ws, bs, None)
    r = oracle.ctr_fwd_bwd(X, y, Ws, bs)
    assert abs(a["loss"] - r["loss"]) < 1e-14
    assert np.abs(a["prob"] - r["prob"]).max() < 1e-14
    assert np.abs(a["dX"] - r["dX"]).max() < 1e-14
    for l in range(3):
        assert np.abs(a["dW"][l] - r["dW"][l]).max() < 1e-14


def test_ctr_prelu_matches_torch_cross_entropy_with_ignored_labels():
    rng = np.random.default_rng(5)
    dims = [9, 11, 6, 3]
    Ws, bs, sl = _net(rng, dims)
    X = rng.standard_normal((17, 9))
    y = rng.integers(0, 3, 17)
    y[[2, 9]] = [-1, 3]                                        # outside [0, C): ignored
    Xt = torch.tensor(X, requires_grad=True)
    out, Wt, bt, st = _torch_net(Xt, Ws, bs, sl)
    ok = (y >= 0) & (y < 3)
    loss = F.cross_entropy(out[torch.as_tensor(ok)], torch.as_tensor(y[ok]), reduction="sum") / 17
    loss.backward()
    a = oracle.ctr_act_fwd_bwd(X, y, Ws, bs, sl)
    assert abs(a["loss"] - float(loss.detach())) < 1e-14
    assert np.abs(a["dX"] - Xt.grad.numpy()).max() < 1e-14
    for l in range(2):
        assert np.abs(a["dslope"][l] - st[l].grad.numpy()).max() < 1e-13


def test_dssm_matches_torch_logistic_loss():
    rng = np.random.default_rng(6)
    user, ad = _net(rng, [14, 10, 8]), _net(rng, [9, 7, 8])
    Xu, Xa = rng.standard_normal((19, 14)), rng.standard_normal((19, 9))
    y = rng.integers(0, 2, 19)
    y[4] = 7                                                   # not a click label: ignored
    Xut, Xat = torch.tensor(Xu, requires_grad=True), torch.tensor(Xa, requires_grad=True)
    u, Wu, bu, su = _torch_net(Xut, *user)
    a, Wa, ba, sa = _torch_net(Xat, *ad)
    s = (u * a).sum(1)
    ok = torch.as_tensor((y == 0) | (y == 1))
    loss = F.binary_cross_entropy_with_logits(s[ok], torch.as_tensor(y, dtype=torch.float64)[ok],
                                              reduction="sum") / 19
    loss.backward()
    r = oracle.dssm_fwd_bwd(Xu, Xa, y, user, ad)
    assert abs(r["loss"] - float(loss.detach())) < 1e-14
    assert np.abs(r["prob"] - torch.sigmoid(s).detach().numpy()).max() < 1e-15
    assert np.abs(r["user"]["dX"] - Xut.grad.numpy()).max() < 1e-14
    assert np.abs(r["ad"]["dX"] - Xat.grad.numpy()).max() < 1e-14
    for l in range(2):
        assert np.abs(r["user"]["dW"][l] - Wu[l].grad.numpy()).max() < 1e-13
        assert np.abs(r["ad"]["db"][l] - ba[l].grad.numpy()).max() < 1e-13
    assert np.abs(r["user"]["dslope"][0] - su[0].grad.numpy()).max() < 1e-13
    assert np.abs(r["ad"]["dslope"][0] - sa[0].grad.numpy()).max() < 1e-13


def test_dssm_linear_towers_closed_form_and_finite_differences():
    rng = np.random.default_rng(7)
    Wu = (rng.standard_normal((4, 6)) * 0.5).astype(np.float32)
    Wa = (rng.standard_normal((4, 5)) * 0.5).astype(np.float32)
    bu = (rng.standard_normal(4) * 0.1).astype(np.float32)
    ba = (rng.standard_normal(4) * 0.1).astype(np.float32)
    Xu, Xa = rng.standard_normal((8, 6)), rng.standard_normal((8, 5))
    y = rng.integers(0, 2, 8)
    r = oracle.dssm_fwd_bwd(Xu, Xa, y, ([Wu], [bu], None), ([Wa], [ba], None))
    u = Xu @ Wu.T.astype(np.float64) + bu
    a = Xa @ Wa.T.astype(np.float64) + ba
    s = (u * a).sum(1)
    assert np.abs(r["score"] - s).max() < 1e-13
    dS = (1 / (1 + np.exp(-s)) - y) / 8
    assert np.abs(r["user"]["dX"] - dS[:, None] * (a @ Wu.astype(np.float64))).max() < 1e-14
    # central differences of the loss in the inputs (float64 throughout)
    h = 1e-6
    for (X, key) in ((Xu, "user"), (Xa, "ad")):
        for (i, k) in ((0, 0), (3, 2), (7, 4)):
            Xp, Xm = X.copy(), X.copy()
            Xp[i, k] += h
            Xm[i, k] -= h
            args_p = (Xp, Xa) if key == "user" else (Xu, Xp)
            args_m = (Xm, Xa) if key == "user" else (Xu, Xm)
            lp = oracle.dssm_fwd_bwd(*args_p, y, ([Wu], [bu], None), ([Wa], [ba], None))["loss"]
            lm = oracle.dssm_fwd_bwd(*args_m, y, ([Wu], [bu], None), ([Wa], [ba], None))["loss"]
            assert abs((lp - lm) / (2 * h) - r[key]["dX"][i, k]) < 1e-8


def test_dense_with_relu_equals_the_image_model_routine():
    """The ReLU dense net against the oracle's image-model routines (pinned on
    their own against torch), at a size where a float32 upstream gradient and
    every temporary array are large enough to be reused by the allocator if
    the wrapper let them go before the C call."""
    rng = np.random.default_rng(8)
    dims = [512, 128, 64, 12]
    Ws, bs, _ = _net(rng, dims, prelu=False)
    T = torch.from_numpy(rng.standard_normal((1500, 512)).astype(np.float32))
    rows = np.arange(1500, dtype=np.int32)
    dE = rng.standard_normal((1500, 12)).astype(np.float32)
    fo = oracle.mlp_fwd(T, rows, Ws, bs)
    bo = oracle.mlp_bwd(T, rows, Ws, fo, dE)
    X = T.double().numpy()
    Z = oracle.dense_fwd(X, Ws, bs, None)
    for a, b in zip(Z, fo["Z"]):
        assert np.array_equal(a, b)
    r = oracle.dense_bwd(X, Ws, None, Z, dE)
    for l in range(3):
        assert np.abs(r["dW"][l] - bo["dW"][l]).max() <= 1e-12 * np.abs(bo["dW"][l]).max()
        assert np.abs(r["db"][l] - bo["db"][l]).max() <= 1e-12 * np.abs(bo["db"][l]).max()
