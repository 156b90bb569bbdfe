"""GPU parity of the CTR model with PReLU (section 7.2) and of the pre-rank
model of section 6 (user and ad towers, inner-product score, logistic loss)
through the C ABI against the float64 oracle, at 1e-4 relative.

CTR with PReLU: the worker's 60-200-80-2 net at 4096 and 17 samples, a
3-class 2-layer net, the widest supported net, and a net whose second
hidden layer keeps ReLU (slopes of either sign; their gradients checked).
Pre-rank: towers of 1 to 3 layers with PReLU or ReLU, representation
widths 8 to 64, 1 to 4096 samples, labels outside {0, 1} ignored.  The
pre-rank step end to end on the tiny batch: image path with sum pooling,
towers on [U, user field] and [A, ad field], then the pooling and embedding
backward from the towers' input gradients."""
import numpy as np
import pytest
import torch

from oracle import oracle
from paper_1711_06505_amd import ams, synth
from tests.parity import RTOL, assert_close, f64

pytestmark = pytest.mark.gpu
F32 = RTOL["f32"]


def cuda(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def net_params(rng, dims, prelu):
    """prelu: one flag per hidden layer (True: PReLU slopes, False: ReLU)."""
    Ws, bs, sl = [], [], []
    for l, (fi, fo) in enumerate(zip(dims[:-1], dims[1:])):
        lim = np.sqrt(6.0 / (fi + fo))
        Ws.append(rng.uniform(-lim, lim, (fo, fi)).astype(np.float32))
        bs.append(rng.uniform(-0.1, 0.1, fo).astype(np.float32))
        if l < len(dims) - 2:
            sl.append(rng.uniform(-0.2, 0.5, fo).astype(np.float32) if prelu[l] else None)
    return Ws, bs, sl


def dev_list(xs):
    return None if xs is None else [None if x is None else cuda(x) for x in xs]


def grads_like(Ws, bs, sl):
    dW = [torch.full(W.shape, 7.0, device="cuda") for W in Ws]
    db = [torch.full(b.shape, 7.0, device="cuda") for b in bs]
    ds = [None if s is None else torch.full(s.shape, 7.0, device="cuda") for s in sl]
    return dW, db, ds


def split(X, widths):
    cuts = np.cumsum([0] + list(widths))
    return [cuda(X[:, cuts[i]:cuts[i + 1]].astype(np.float32)) for i in range(len(widths))]


def check_net(name, dW, db, ds, ref):
    for l in range(len(dW)):
        assert_close(dW[l], ref["dW"][l], F32, f"{name} dW{l + 1}")
        assert_close(db[l], ref["db"][l], F32, f"{name} db{l + 1}")
    for l, d in enumerate(ds):
        if d is not None:
            assert_close(d, ref["dslope"][l], F32, f"{name} dslope{l + 1}")


@pytest.mark.parametrize("dims,B,widths,prelu", [
    ((60, 200, 80, 2), 4096, (12, 12, 12, 12, 12), (True, True)),
    ((60, 200, 80, 2), 17, (60,), (True, True)),
    ((30, 40, 3), 33, (30,), (True,)),
    ((128, 256, 256, 8), 50, (64, 64), (True, True)),
    ((68, 32, 16, 2), 64, (16, 16, 12, 12, 12), (True, False)),
])
def test_ctr_prelu_matches_oracle(dims, B, widths, prelu):
    print(f"ctr prelu {dims} B={B} {prelu}", flush=True)
    rng = np.random.default_rng(B + len(dims))
    Ws, bs, sl = net_params(rng, dims, prelu)
    X = (rng.standard_normal((B, dims[0])) * 0.8).astype(np.float32)
    labels = rng.integers(0, dims[-1], B).astype(np.int32)
    labels[:: 13] = -1
    ref = oracle.ctr_act_fwd_bwd(X, labels, Ws, bs, sl)
    fields = split(X, widths)
    dfs = [torch.full_like(f, 7.0) for f in fields]
    dW, db, ds = grads_like(Ws, bs, sl)
    loss = torch.zeros(1, device="cuda")
    prob = torch.zeros((B, dims[-1]), device="cuda")
    net = ams.make_ctr(dims)
    ws = torch.empty(max(ams.ams_ctr_workspace(net, B), 256), dtype=torch.uint8, device="cuda")
    ams.ams_ctr_fwd_bwd(net, fields, cuda(labels), dev_list(Ws), dev_list(bs), loss, prob, dW, db, dfs, ws,
                        slopes=dev_list(sl), dslopes=ds)
    torch.cuda.synchronize()
    assert abs(loss.item() - ref["loss"]) <= F32 * max(1.0, abs(ref["loss"]))
    ok = labels >= 0
    assert_close(prob[torch.from_numpy(ok).cuda()], ref["prob"][ok], F32, "prob")
    assert_close(torch.cat(dfs, 1), ref["dX"], F32, "dX")
    check_net("ctr", dW, db, ds, ref)


def run_dssm(user_dims, ad_dims, uw, aw, Xu, Xa, labels, user, ad):
    B = Xu.shape[0]
    uf, af = split(Xu, uw), split(Xa, aw)
    duf, daf = [torch.full_like(f, 7.0) for f in uf], [torch.full_like(f, 7.0) for f in af]
    gu, ga = grads_like(*user), grads_like(*ad)
    loss = torch.zeros(1, device="cuda")
    prob = torch.zeros(B, device="cuda")
    un, an = ams.make_ctr(user_dims), ams.make_ctr(ad_dims)
    ws = torch.empty(max(ams.ams_dssm_workspace(un, an, B), 256), dtype=torch.uint8, device="cuda")
    ams.ams_dssm_fwd_bwd(un, an, uf, af, cuda(labels), [dev_list(x) for x in user], [dev_list(x) for x in ad],
                         loss, prob, gu, ga, duf, daf, ws)
    torch.cuda.synchronize()
    return loss, prob, gu, ga, torch.cat(duf, 1), torch.cat(daf, 1)


@pytest.mark.parametrize("user_dims,ad_dims,B,prelu", [
    ((36, 64, 32), (24, 48, 32), 4096, True),
    ((36, 64, 32), (24, 32), 17, True),
    ((24, 128, 64, 64), (12, 64), 1, True),
    ((48, 100, 40, 8), (20, 30, 8), 300, False),
])
def test_dssm_matches_oracle(user_dims, ad_dims, B, prelu):
    print(f"dssm {user_dims} {ad_dims} B={B}", flush=True)
    rng = np.random.default_rng(B)
    user = net_params(rng, user_dims, [prelu] * (len(user_dims) - 2))
    ad = net_params(rng, ad_dims, [prelu] * (len(ad_dims) - 2))
    Xu = (rng.standard_normal((B, user_dims[0])) * 0.8).astype(np.float32)
    Xa = (rng.standard_normal((B, ad_dims[0])) * 0.8).astype(np.float32)
    labels = (rng.random(B) < 0.3).astype(np.int32)
    labels[5::11] = 2
    uw = (12,) * (user_dims[0] // 12)
    aw = (12,) * (ad_dims[0] // 12) if ad_dims[0] % 12 == 0 else (ad_dims[0],)
    ref = oracle.dssm_fwd_bwd(Xu, Xa, labels, user, ad)
    loss, prob, gu, ga, dXu, dXa = run_dssm(user_dims, ad_dims, uw, aw, Xu, Xa, labels, user, ad)
    assert abs(loss.item() - ref["loss"]) <= F32 * max(1.0, abs(ref["loss"]))
    assert_close(prob, ref["prob"], F32, "prob")
    assert_close(dXu, ref["user"]["dX"], F32, "user dX")
    assert_close(dXa, ref["ad"]["dX"], F32, "ad dX")
    check_net("user", *gu, ref["user"])
    check_net("ad", *ga, ref["ad"])


def test_prerank_step_end_to_end_tiny():
    """Image path (sum pooling) -> towers -> pooling and embedding backward."""
    w = synth.get("tiny")
    batch = synth.make_batch(w)
    Ws, bs = synth.make_weights(w)
    T = synth.table_full(w, device="cuda")
    n_beh, B, D = int(batch["seg_off"][-1]), w.batch, w.dims[-1]
    st = ams.Step(w.dims, w.dtype, "sum", B, n_beh)
    seg_d = torch.from_numpy(batch["seg_off"].astype(np.int32)).cuda()
    occ = synth.occurrences(batch).astype(np.int32)
    st.dedup(torch.from_numpy(occ).cuda(), w.n_images)
    Wd, bd = [x.cuda() for x in Ws], [x.cuda() for x in bs]
    st.embed_fwd(T, Wd, bd)
    st.pool_fwd(seg_d, n_beh)
    rng = np.random.default_rng(11)
    user_dims, ad_dims = (2 * D, 32, 16), (2 * D, 16)
    user = net_params(rng, user_dims, [True])
    ad = net_params(rng, ad_dims, [])
    xu = (rng.standard_normal((B, D)) * 0.5).astype(np.float32)     # a user-side ID feature
    xa = (rng.standard_normal((B, D)) * 0.5).astype(np.float32)     # an ad-side ID feature
    labels = (rng.random(B) < 0.4).astype(np.int32)
    un, an = ams.make_ctr(user_dims), ams.make_ctr(ad_dims)
    uf, af = [st.U[:B], cuda(xu)], [st.A[:B], cuda(xa)]
    dU, dA = torch.empty((B, D), device="cuda"), torch.empty((B, D), device="cuda")
    dxu, dxa = torch.empty((B, D), device="cuda"), torch.empty((B, D), device="cuda")
    gu, ga = grads_like(*user), grads_like(*ad)
    loss, prob = torch.zeros(1, device="cuda"), torch.zeros(B, device="cuda")
    ws = torch.empty(max(ams.ams_dssm_workspace(un, an, B), 256), dtype=torch.uint8, device="cuda")
    ams.ams_dssm_fwd_bwd(un, an, uf, af, cuda(labels), [dev_list(x) for x in user], [dev_list(x) for x in ad],
                         loss, prob, gu, ga, [dU, dxu], [dA, dxa], ws)
    st.pool_bwd(seg_d, n_beh, dU, dA)
    st.embed_bwd(T, Wd)
    torch.cuda.synchronize()
    # oracle chain on the same batch
    od = oracle.dedup(occ, w.n_images)
    T_u = synth.table_rows(w, od["uniq"])
    rows = np.arange(od["n_uniq"], dtype=np.int32)
    fo = oracle.mlp_fwd(T_u, rows, Ws, bs)
    pf = oracle.pool_fwd("sum", batch["seg_off"], od["inv"], fo["E"])
    ref = oracle.dssm_fwd_bwd(np.concatenate([pf["U"], xu], 1), np.concatenate([pf["A"], xa], 1), labels, user, ad)
    assert abs(loss.item() - ref["loss"]) <= F32 * max(1.0, abs(ref["loss"]))
    assert_close(dU, ref["user"]["dX"][:, :D], F32, "dU")
    assert_close(dA, ref["ad"]["dX"][:, :D], F32, "dA")
    check_net("user", *gu, ref["user"])
    check_net("ad", *ga, ref["ad"])
    pb = oracle.pool_bwd("sum", batch["seg_off"], od["inv"], od["n_uniq"], fo["E"], pf,
                         ref["user"]["dX"][:, :D], ref["ad"]["dX"][:, :D])
    n_u = od["n_uniq"]
    assert_close(st.dE[:n_u], pb["dE"], F32, "dE", rows=True)
    bw = oracle.mlp_bwd(T_u, rows, Ws, fo, pb["dE"])
    for l in range(w.n_layers):
        assert_close(st.dW[l], bw["dW"][l], F32, f"image dW{l + 1}")
        assert_close(st.db[l], bw["db"][l], F32, f"image db{l + 1}")
