"""Pins for the query-attention channel of the float64 oracle (multiple-query
attentive pooling, section 5.2), each against something other than the
oracle: torch float64 autograd of the two-channel pooling (ad image query and
a given query, outputs concatenated), closed forms (a zero query gives the
mean, one behavior gives e, equal rows give e), the oracle's ad-query channel
when the query is the ad embedding, and central differences on the query."""
import numpy as np
import torch

from oracle import oracle


def case(seed=2, B=9, n_u=30, D=12):
    rng = np.random.default_rng(seed)
    lens = rng.integers(1, 9, size=B)
    lens[3] = 0
    seg = np.zeros(B + 1, np.int32)
    seg[1:] = np.cumsum(lens)
    n_beh = int(seg[-1])
    inv = rng.integers(0, n_u, size=n_beh + B).astype(np.int32)
    E = rng.standard_normal((n_u, D))
    Q = rng.standard_normal((B, D))
    gU = rng.standard_normal((B, D))
    gQ = rng.standard_normal((B, D))
    return seg, inv, E, Q, gU, gQ


def rel_err(x, r):
    return float(np.abs(np.asarray(x) - np.asarray(r)).max() / max(np.abs(np.asarray(r)).max(), 1e-300))


def test_two_channels_match_torch_autograd():
    seg, inv, E, Q, gU, gQ = case()
    B = seg.size - 1
    n_beh = int(seg[-1])
    f1 = oracle.pool_fwd("att", seg, inv, E)
    f2 = oracle.pool_query_fwd(seg, inv, E, Q)
    b1 = oracle.pool_bwd("att", seg, inv, E.shape[0], E, f1, gU, np.zeros_like(gU))
    b2 = oracle.pool_query_bwd(seg, inv, E.shape[0], E, Q, f2, gQ)
    Et = torch.from_numpy(E).requires_grad_()
    Qt = torch.from_numpy(Q).requires_grad_()
    outs = []
    for i in range(B):
        e = Et[torch.as_tensor(inv[seg[i]:seg[i + 1]], dtype=torch.int64)]
        a = Et[int(inv[n_beh + i])]
        if e.shape[0] == 0:
            outs.append(torch.zeros(2 * E.shape[1], dtype=torch.float64))
            continue
        u1 = torch.softmax(e @ a, 0) @ e
        u2 = torch.softmax(e @ Qt[i], 0) @ e
        outs.append(torch.cat([u1, u2]))
    out = torch.stack(outs)
    (out * torch.from_numpy(np.concatenate([gU, gQ], 1))).sum().backward()
    D = E.shape[1]
    assert rel_err(f2["U"], out[:, D:].detach().numpy()) < 1e-13
    assert rel_err(b1["dE"] + b2["dE"], Et.grad.numpy()) < 1e-12
    assert rel_err(b2["dQ"], Qt.grad.numpy()) < 1e-12


def test_query_closed_forms():
    seg, inv, E, Q, gU, _ = case(seed=5)
    B = seg.size - 1
    # zero query: uniform weights, the mean of the segment
    f = oracle.pool_query_fwd(seg, inv, E, np.zeros_like(Q))
    for i in range(B):
        idx = inv[seg[i]:seg[i + 1]]
        expect = E[idx].mean(0) if idx.size else np.zeros(E.shape[1])
        assert np.allclose(f["U"][i], expect, rtol=1e-13, atol=1e-15)
    # one behavior: u = e, w = 1, and the query gets no gradient
    one = np.array([0, 1], np.int32)
    inv1 = np.array([4, 2], np.int32)
    f1 = oracle.pool_query_fwd(one, inv1, E, Q[:1])
    assert np.array_equal(f1["U"][0], E[4]) and f1["w"][0] == 1.0
    b1 = oracle.pool_query_bwd(one, inv1, E.shape[0], E, Q[:1], f1, gU[:1])
    assert np.abs(b1["dQ"]).max() < 1e-15
    # equal rows: u = e whatever the query
    same = np.array([0, 5], np.int32)
    inv5 = np.array([7, 7, 7, 7, 7, 0], np.int32)
    assert np.allclose(oracle.pool_query_fwd(same, inv5, E, Q[:1])["U"][0], E[7], rtol=1e-14)


def test_query_equal_to_ad_embedding_is_the_ad_channel():
    seg, inv, E, _, gU, _ = case(seed=8)
    n_beh = int(seg[-1])
    Qad = E[inv[n_beh:]]
    fa = oracle.pool_fwd("att", seg, inv, E)
    fq = oracle.pool_query_fwd(seg, inv, E, Qad)
    assert np.array_equal(fa["U"], fq["U"]) and np.array_equal(fa["w"], fq["w"])
    # ad channel's gradient = the query channel's behaviors + (through the ad) dQ
    ba = oracle.pool_bwd("att", seg, inv, E.shape[0], E, fa, gU, np.zeros_like(gU))
    bq = oracle.pool_query_bwd(seg, inv, E.shape[0], E, Qad, fq, gU)
    through_ad = np.zeros_like(ba["dE"])
    np.add.at(through_ad, inv[n_beh:], bq["dQ"])
    assert rel_err(ba["dE"], bq["dE"] + through_ad) < 1e-12


def test_query_gradient_by_finite_differences_and_ds_sums_to_zero():
    seg, inv, E, Q, gU, _ = case(seed=11)
    f = oracle.pool_query_fwd(seg, inv, E, Q)
    b = oracle.pool_query_bwd(seg, inv, E.shape[0], E, Q, f, gU)

    def L(Qp):
        return float((oracle.pool_query_fwd(seg, inv, E, Qp)["U"] * gU).sum())
    rng = np.random.default_rng(0)
    for _ in range(6):
        i, d = int(rng.integers(0, Q.shape[0])), int(rng.integers(0, Q.shape[1]))
        h = 1e-6
        Qp, Qm = Q.copy(), Q.copy()
        Qp[i, d] += h
        Qm[i, d] -= h
        fd = (L(Qp) - L(Qm)) / (2 * h)
        assert abs(fd - b["dQ"][i, d]) <= 1e-7 * max(1.0, abs(fd))
    # sum_j ds_j = 0: the query gradient of a constant shift along q is zero
    n_beh = int(seg[-1])
    for i in range(seg.size - 1):
        j0, j1 = seg[i], seg[i + 1]
        if j1 == j0:
            continue
        c = gU[i] @ f["U"][i]
        ds = f["w"][j0:j1] * (E[inv[j0:j1]] @ gU[i] - c)
        assert abs(ds.sum()) < 1e-13
