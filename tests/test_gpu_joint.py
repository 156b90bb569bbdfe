"""GPU parity of the joint step (worker side of Algorithm 1) through the C ABI
against the float64 oracle: ID bags, merged ID-row gradients, the CTR MLP with
softmax cross-entropy, sparse Adagrad, and whole joint steps (the image path
driven by the CTR model's input gradients) at a small, a mid and the full
joint workload size.  Dedup outputs are compared bit-exactly; floating point
per tests/parity.py (1e-4 for the float32 parts)."""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import oracle
from paper_1711_06505_amd import ams, synth
from tests.parity import RTOL, assert_close, f64, gpu_outputs

pytestmark = pytest.mark.gpu
F32 = RTOL["f32"]


def cuda_i32(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).cuda()


def mid_joint(B=96, query_table=-1):
    base = synth.get("c4_joint")
    return dataclasses.replace(base, name="mid_joint" if query_table < 0 else "mid_mqap", index=21, batch=B,
                               n_images=20_000, stream=-1,
                               joint=dataclasses.replace(base.joint, id_rows=(200_000, 20_000, 500),
                                                         query_table=query_table))


def gpu_dedup(occ_dev, n_ids, n):
    m = max(n, 1)
    d = {k: torch.empty(m, dtype=torch.int32, device="cuda") for k in ("uniq", "inv", "perm")}
    d["off"] = torch.empty(n + 1, dtype=torch.int32, device="cuda")
    d["nu"] = torch.zeros(1, dtype=torch.int32, device="cuda")
    d["st"] = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(ams.ams_dedup_workspace(n, n_ids), 256), dtype=torch.uint8, device="cuda")
    ams.ams_dedup(occ_dev, n_ids, d["uniq"], d["inv"], d["perm"], d["off"], d["nu"], d["st"], ws)
    return d


# ------------------------------------------------------------------ bags

@pytest.mark.parametrize("D", [5, 12, 20, 32])
def test_bag_fwd_shapes_lengths_and_bad_ids(D):
    """Row widths on both kernel instances (vector and scalar loads), empty
    and single-behavior samples, a sample cut at the 64-lane and 512-ID round
    boundaries and one past two rounds; IDs out of range read as zero rows."""
    N = 1000
    rng = np.random.default_rng(D)
    lengths = [0, 1, 63, 64, 600, 1100, 5]
    B = len(lengths)
    seg = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    n_beh = int(seg[-1])
    occ = rng.integers(0, N, size=n_beh + B).astype(np.int32)
    occ[[3, 70, 800, n_beh + 2]] = [N, -1, N + 5, -7]
    tab = rng.standard_normal((N, D)).astype(np.float32)
    bag = torch.full((B, D), float("nan"), device="cuda")
    ams.ams_bag_fwd(cuda_i32(seg), n_beh, cuda_i32(occ), torch.from_numpy(tab).cuda(), bag)
    torch.cuda.synchronize()
    padded = np.concatenate([tab, np.zeros((1, D), np.float32)])       # row N: the zero row
    idx = np.where((occ >= 0) & (occ < N), occ, N)
    assert_close(bag, oracle.bag_fwd(seg, idx, padded), F32, f"bag D={D}", rows=True)


@pytest.mark.parametrize("name", ["tiny_joint", "mid_joint", "c4_joint"])
def test_bag_fwd_and_bwd_match_oracle(name):
    w = mid_joint() if name == "mid_joint" else synth.get(name)
    batch = synth.make_batch(w)
    jb = synth.make_joint(w, batch)
    seg = batch["seg_off"]
    n_beh = int(seg[-1])
    B = w.batch
    rng = np.random.default_rng(1)
    dbag = rng.standard_normal((B, w.joint.id_dim)).astype(np.float32)
    for t, N in enumerate(w.joint.id_rows):
        print(f"bags {name} table {t} ({N} rows)", flush=True)
        occ = synth.joint_occurrences(jb, t)
        od = oracle.dedup(occ, N)
        tab = synth.id_table_full(w, t, device="cuda")
        bag = torch.empty((B, w.joint.id_dim), device="cuda")
        occ_dev = cuda_i32(occ)
        seg_dev = cuda_i32(seg)
        ams.ams_bag_fwd(seg_dev, n_beh, occ_dev, tab, bag)
        rows = synth.id_table_rows(w, t, od["uniq"])
        assert_close(bag, oracle.bag_fwd(seg, od["inv"], rows), F32, f"bag {t}", rows=True)
        # merged row gradients over the GPU's own dedup (checked bit-exact first)
        d = gpu_dedup(occ_dev, N, occ.size)
        torch.cuda.synchronize()
        n_u = int(d["nu"].item())
        assert int(d["st"].item()) == 0 and n_u == od["n_uniq"]
        np.testing.assert_array_equal(d["uniq"][:n_u].cpu().numpy(), od["uniq"])
        np.testing.assert_array_equal(d["inv"][:occ.size].cpu().numpy(), od["inv"])
        grad = torch.empty((occ.size, w.joint.id_dim), device="cuda")
        ws = torch.empty(max(ams.ams_bag_workspace(B, n_beh, w.joint.id_dim, occ.size), 256), dtype=torch.uint8,
                         device="cuda")
        ams.ams_bag_bwd(seg_dev, n_beh, d["inv"], d["perm"], d["off"], d["nu"], occ.size,
                        torch.from_numpy(dbag).cuda(), grad, ws)
        torch.cuda.synchronize()
        ref = oracle.merged_row_grad(seg, od["inv"], od["n_uniq"], dbag)
        assert_close(grad[:n_u], ref, F32, f"row grad {t}", rows=True)
        del tab


# --------------------------------------------------------------- CTR MLP

def gpu_ctr(dims, fields, labels, Ws, bs):
    net = ams.make_ctr(dims)
    B = fields[0].shape[0]
    dev = [torch.from_numpy(np.ascontiguousarray(f, dtype=np.float32)).cuda() for f in fields]
    dfs = [torch.full_like(f, 7.0) for f in dev]
    Wd = [W.cuda() for W in Ws]
    bd = [b.cuda() for b in bs]
    dW = [torch.full_like(W, 7.0) for W in Wd]
    db = [torch.full_like(b, 7.0) for b in bd]
    loss = torch.zeros(1, device="cuda")
    prob = torch.zeros((B, dims[-1]), device="cuda")
    ws = torch.empty(max(ams.ams_ctr_workspace(net, B), 256), dtype=torch.uint8, device="cuda")
    ams.ams_ctr_fwd_bwd(net, dev, cuda_i32(labels), Wd, bd, loss, prob, dW, db, dfs, ws)
    torch.cuda.synchronize()
    return {"loss": float(loss.item()), "prob": f64(prob), "dW": [f64(x) for x in dW], "db": [f64(x) for x in db],
            "dX": np.concatenate([f64(x) for x in dfs], axis=1)}


def ctr_case(dims, B, widths, seed):
    rng = np.random.default_rng(seed)
    X = (rng.standard_normal((B, dims[0])) * 0.8).astype(np.float32)
    labels = (rng.random(B) < 0.3).astype(np.int32)
    Ws, bs = [], []
    for fi, fo in zip(dims[:-1], dims[1:]):
        lim = np.sqrt(6.0 / (fi + fo))
        Ws.append(torch.from_numpy(rng.uniform(-lim, lim, (fo, fi)).astype(np.float32)))
        bs.append(torch.from_numpy(rng.uniform(-0.1, 0.1, fo).astype(np.float32)))
    cuts = np.cumsum([0] + list(widths))
    fields = [X[:, cuts[i]:cuts[i + 1]] for i in range(len(widths))]
    return X, labels, Ws, bs, fields


@pytest.mark.parametrize("dims,B,widths", [
    ((60, 200, 80, 2), 4096, (12, 12, 12, 12, 12)),
    ((60, 200, 80, 2), 17, (12, 12, 12, 12, 12)),
    ((60, 200, 80, 2), 1, (24, 36)),
    ((68, 32, 16, 2), 64, (16, 16, 12, 12, 12)),
    ((30, 40, 3), 33, (30,)),
    ((128, 256, 256, 8), 50, (64, 64)),
])
def test_ctr_fwd_bwd_matches_oracle(dims, B, widths):
    print(f"ctr {dims} B={B}", flush=True)
    X, labels, Ws, bs, fields = ctr_case(dims, B, widths, seed=B + len(dims))
    if dims[-1] > 2:
        labels = np.random.default_rng(0).integers(0, dims[-1], size=B).astype(np.int32)
    g = gpu_ctr(dims, fields, labels, Ws, bs)
    o = oracle.ctr_fwd_bwd(X, labels, Ws, bs)
    assert abs(g["loss"] - o["loss"]) <= F32 * max(1.0, abs(o["loss"]))
    assert_close(g["prob"], o["prob"], F32, "prob")
    assert_close(g["dX"], o["dX"], F32, "dX")
    for l in range(len(Ws)):
        assert_close(g["dW"][l], o["dW"][l], F32, f"dW{l + 1}")
        assert_close(g["db"][l], o["db"][l], F32, f"db{l + 1}")


def test_ctr_ignores_out_of_range_labels():
    dims, B = (60, 200, 80, 2), 40
    X, labels, Ws, bs, fields = ctr_case(dims, B, (60,), seed=3)
    labels[[0, 7]] = [-1, 2]
    g = gpu_ctr(dims, fields, labels, Ws, bs)
    keep = np.ones(B, bool)
    keep[[0, 7]] = False
    o = oracle.ctr_fwd_bwd(X[keep], labels[keep], Ws, bs)
    n = int(keep.sum())
    # the mean is over all B samples; the ignored ones add nothing
    assert abs(g["loss"] - o["loss"] * n / B) <= F32 * max(1.0, o["loss"])
    assert not g["dX"][~keep].any() and not g["prob"][~keep].any()
    assert_close(g["dX"][keep], o["dX"] * n / B, F32, "dX")
    for l in range(3):
        assert_close(g["dW"][l], o["dW"][l] * n / B, F32, f"dW{l + 1}")


# --------------------------------------------------------------- Adagrad

def test_adagrad_rows_matches_oracle_and_leaves_other_rows():
    rng = np.random.default_rng(5)
    N, D, n_u = 5000, 12, 1234
    uniq = np.sort(rng.choice(N, size=n_u, replace=False)).astype(np.int32)
    grad = rng.standard_normal((n_u, D)).astype(np.float32)
    grad[3] = 0.0
    table = rng.standard_normal((N, D)).astype(np.float32)
    accum = rng.uniform(0.0, 2.0, size=(N, D)).astype(np.float32)
    accum[uniq[:10]] = 0.0
    t_dev = torch.from_numpy(table).cuda()
    a_dev = torch.from_numpy(accum).cuda()
    cap = n_u + 100
    g_dev = torch.zeros((cap, D), device="cuda")
    g_dev[:n_u] = torch.from_numpy(grad).cuda()
    u_dev = torch.zeros(cap, dtype=torch.int32, device="cuda")
    u_dev[:n_u] = cuda_i32(uniq)
    nu = torch.tensor([n_u], dtype=torch.int32, device="cuda")
    ams.ams_adagrad_rows(u_dev, nu, cap, g_dev, t_dev, a_dev, 0.01, 1e-8)
    torch.cuda.synchronize()
    new_rows, new_acc = oracle.adagrad_rows(grad, table[uniq], accum[uniq], 0.01, 1e-8)
    tg, ag = t_dev.cpu().numpy(), a_dev.cpu().numpy()
    assert_close(tg[uniq], new_rows, F32, "rows")
    assert_close(ag[uniq], new_acc, F32, "accum")
    other = np.setdiff1d(np.arange(N), uniq)
    np.testing.assert_array_equal(tg[other], table[other])
    np.testing.assert_array_equal(ag[other], accum[other])


# ------------------------------------------------------------- end to end

def run_joint(w, mode="att"):
    batch = synth.make_batch(w)
    jb = synth.make_joint(w, batch)
    Ws, bs = synth.make_weights(w)
    cW, cb = synth.make_ctr_weights(w)
    T = synth.table_full(w, device="cuda")
    tabs = [synth.id_table_full(w, t, device="cuda") for t in range(len(w.joint.id_rows))]
    rng = np.random.default_rng(17)
    accs = [torch.from_numpy(rng.uniform(0.0, 0.1, size=tuple(x.shape)).astype(np.float32)).cuda() for x in tabs]
    n_beh = int(batch["seg_off"][-1])
    tq = w.joint.query_table if w.joint.query_table >= 0 else None
    js = ams.JointStep(w.dims, w.dtype, mode, w.batch, n_beh, w.joint.id_rows, w.joint.id_dim, synth.ctr_dims(w),
                       query_table=tq)
    occ = cuda_i32(synth.occurrences(batch))
    id_occ = [cuda_i32(synth.joint_occurrences(jb, t)) for t in range(len(tabs))]
    # the oracle's inputs: rows of the batch's unique IDs before the update
    od_t = [oracle.dedup(synth.joint_occurrences(jb, t), N) for t, N in enumerate(w.joint.id_rows)]
    rows0 = [tabs[t][torch.from_numpy(od_t[t]["uniq"]).long().cuda()].cpu().numpy() for t in range(len(tabs))]
    acc0 = [accs[t][torch.from_numpy(od_t[t]["uniq"]).long().cuda()].cpu().numpy() for t in range(len(tabs))]
    js.run(occ, w.n_images, T, [x.cuda() for x in Ws], [x.cuda() for x in bs], cuda_i32(batch["seg_off"]),
           id_occ, tabs, accs, cuda_i32(jb["labels"]), [x.cuda() for x in cW], [x.cuda() for x in cb],
           w.joint.lr, w.joint.eps)
    torch.cuda.synchronize()
    g = gpu_outputs(js.img)
    T_u = synth.table_rows(w, g["uniq"], device="cuda").cpu()
    del T
    o = oracle.joint_step(batch, jb, w.joint, w.n_images, T_u, Ws, bs, rows0, cW, cb, acc0, mode=mode,
                          query_table=tq)
    o["_rows0"], o["_acc0"] = rows0, acc0
    return batch, jb, Ws, T_u, js, g, o, tabs, accs, od_t


def compare_image_chained(w, batch, Ws, T_u, g, o, dU, dA):
    """The image path of a joint step.  Forward outputs against the oracle's
    forward; the backward chained: dE against the oracle's attentive-pooling
    backward evaluated on the GPU's own (checked) forward outputs and upstream
    gradients, and the model gradients against the oracle's MLP backward of
    the GPU's dE.  Under the CTR model's upstream gradients the attention term
    of an ad, sum_j w_j (g.e_j - g.u) e_j over up to 500 behaviors, nearly
    cancels, so its value is ill-conditioned in E (fp32 noise of 2e-5 in E has
    moved it by 10%); each stage is checked where it is well-posed."""
    from tests.parity import grad_flip_bounds, relu_flips
    from tests.test_gpu_parity import TAU
    rt = RTOL[w.dtype]
    od = o["dedup"]
    for k in ("uniq", "inv", "occ_perm", "uniq_off"):
        np.testing.assert_array_equal(g[k], od[k], err_msg=k)
    assert g["n_uniq"] == od["n_uniq"] and g["dev_status"] == 0
    fo, pf = o["fwd"], o["pool"]
    assert_close(g["E"], fo["E"], rt, "E", rows=True)
    assert_close(g["U"], pf["U"], rt, "U", rows=True)
    assert_close(g["A"], pf["A"], rt, "A", rows=True)
    assert_close(g["w"], pf["w"], rt, "attention weights")
    gf = {"U": g["U"], "A": g["A"], "w": g["w"], "argmax": np.full(g["U"].shape, -1, np.int32)}
    pb = oracle.pool_bwd("att", batch["seg_off"], od["inv"], od["n_uniq"], g["E"], gf, f64(dU), f64(dA))
    assert_close(g["dE"], pb["dE"], rt, "dE (oracle pooling backward on the GPU's forward)", rows=True)
    bw = oracle.mlp_bwd(T_u, np.arange(od["n_uniq"], dtype=np.int32), Ws, fo, g["dE"])
    flips1 = relu_flips(fo["Z"][0], g["H1"], TAU)
    flips2 = relu_flips(fo["Z"][1], g["H2"], TAU) if w.n_layers == 3 else []
    eW, eb = grad_flip_bounds(w.dims, Ws, T_u, fo, bw, flips1, flips2, None)
    for l in range(w.n_layers):
        assert_close(g["dW"][l], bw["dW"][l], rt, f"dW{l + 1}", extra=eW[l])
        assert_close(g["db"][l], bw["db"][l], rt, f"db{l + 1}", extra=eb[l])


def oracle_chain_from(w, batch, jb, Ws, T_u, o, od_t, E, bags):
    """The oracle's joint step downstream of the first-stage outputs: pooling
    of E (and, with a query table, the query channel with the oracle's
    queries), the CTR model on [U, (U2,) A, bags], the pooling and MLP
    backward, the ID row gradients and their Adagrad step, all in float64 on
    the given E and bags (the MLP backward on the oracle's own forward
    activations)."""
    od = o["dedup"]
    seg = batch["seg_off"]
    mq = "Q" in o
    pf = oracle.pool_fwd("att", seg, od["inv"], E)
    users = [pf["U"]]
    if mq:
        pq = oracle.pool_query_fwd(seg, od["inv"], E, o["Q"])
        users.append(pq["U"])
    X = np.concatenate(users + [pf["A"]] + list(bags), axis=1)
    c = oracle.ctr_fwd_bwd(X, jb["labels"], *synth.make_ctr_weights(w))
    D = w.out_dim
    k = 2 if mq else 1
    dU, dA = c["dX"][:, :D], c["dX"][:, k * D:(k + 1) * D]
    dbags = [c["dX"][:, (k + 1) * D + 12 * t:(k + 1) * D + 12 * (t + 1)] for t in range(len(bags))]
    pb = oracle.pool_bwd("att", seg, od["inv"], od["n_uniq"], E, pf, dU, dA)
    dE = pb["dE"]
    extra = {}
    if mq:
        qb = oracle.pool_query_bwd(seg, od["inv"], od["n_uniq"], E, o["Q"], pq, c["dX"][:, D:2 * D])
        dE = dE + qb["dE"]
        extra = {"U2": pq["U"], "w2": pq["w"], "dU2": c["dX"][:, D:2 * D], "dQ": qb["dQ"]}
    bw = oracle.mlp_bwd(T_u, np.arange(od["n_uniq"], dtype=np.int32), Ws, o["fwd"], dE)
    grads, new_rows, new_acc = [], [], []
    for t in range(len(bags)):
        dad = extra["dQ"] if mq and t == w.joint.query_table else None
        g = oracle.merged_row_grad(seg, od_t[t]["inv"], od_t[t]["n_uniq"], dbags[t], dad)
        r, a = oracle.adagrad_rows(g, o["_rows0"][t], o["_acc0"][t], w.joint.lr, w.joint.eps)
        grads.append(g)
        new_rows.append(r)
        new_acc.append(a)
    return {"U": pf["U"], "A": pf["A"], "w": pf["w"], "ctr": c, "dU": dU, "dA": dA, "dbags": dbags,
            "dE": dE, "dW": bw["dW"], "db": bw["db"], "row_grads": grads, "new_rows": new_rows,
            "new_accum": new_acc, **extra}


def compare_joint_end_to_end(w, batch, jb, Ws, T_u, g, js, o, od_t, tabs, accs):
    """The whole joint step against the whole float64 oracle chain.  E and the
    bags, the first stage, are held to rtol against the oracle's.  Every later
    output X is held to rtol plus twice |X(E_gpu, bags_gpu) - X|, where
    X(E_gpu, bags_gpu) is the oracle's own chain evaluated on the GPU's E and
    bags: the tolerance follows the measured sensitivity of the computation to
    its fp32 inputs (a decision of the CTR model's ReLU near its tie, or a
    long segment's attention term, show up there) instead of assuming it.
    ReLU decisions of the image model near a tie widen its weight gradients'
    tolerance as in compare_step."""
    from tests.parity import assert_close_sensitive, grad_flip_bounds, relu_flips
    from tests.test_gpu_parity import TAU
    rt = RTOL[w.dtype]
    B, n_t = w.batch, len(tabs)
    od = o["dedup"]
    for k in ("uniq", "inv", "occ_perm", "uniq_off"):
        np.testing.assert_array_equal(g[k], od[k], err_msg=k)
    assert g["n_uniq"] == od["n_uniq"] and g["dev_status"] == 0
    assert_close(g["E"], o["fwd"]["E"], rt, "E", rows=True)
    bags_g = [f64(js.bags[t][:B]) for t in range(n_t)]
    for t in range(n_t):
        assert_close(bags_g[t], o["bags"][t], F32, f"bag {t}", rows=True)
    p = oracle_chain_from(w, batch, jb, Ws, T_u, o, od_t, g["E"], bags_g)

    def held(x, ref, pert, name, rtol=rt, extra=None, rows=False):
        return assert_close_sensitive(x, ref, pert, rtol, name, extra=extra, rows=rows)

    held(g["U"], o["pool"]["U"], p["U"], "U", rows=True)
    held(g["A"], o["pool"]["A"], p["A"], "A", rows=True)
    held(g["w"], o["pool"]["w"], p["w"], "attention weights")
    c = o["ctr"]
    assert abs(float(js.loss.item()) - c["loss"]) <= F32 * max(1.0, c["loss"]) + 2 * abs(p["ctr"]["loss"] - c["loss"])
    held(js.prob[:B], c["prob"], p["ctr"]["prob"], "prob", rtol=F32)
    for l in range(len(js.ctr_dW)):
        held(js.ctr_dW[l], c["dW"][l], p["ctr"]["dW"][l], f"ctr dW{l + 1}", rtol=F32)
        held(js.ctr_db[l], c["db"][l], p["ctr"]["db"][l], f"ctr db{l + 1}", rtol=F32)
    held(js.dU[:B], o["dU"], p["dU"], "dU", rtol=F32, rows=True)
    held(js.dA[:B], o["dA"], p["dA"], "dA", rtol=F32, rows=True)
    if "Q" in o:
        np.testing.assert_array_equal(f64(js.Q[:B]), o["Q"])        # a copy of table rows
        held(js.U2[:B], o["query"]["U"], p["U2"], "U2", rows=True)
        held(js.w2[:g["w"].size], o["query"]["w"], p["w2"], "query weights")
        held(js.dU2[:B], o["dU2"], p["dU2"], "dU2", rtol=F32, rows=True)
        held(js.dQ[:B], o["query_bwd"]["dQ"], p["dQ"], "dQ", rtol=F32, rows=True)
    for t in range(n_t):
        n_u = od_t[t]["n_uniq"]
        held(js.dbags[t][:B], o["dbags"][t], p["dbags"][t], f"dbag {t}", rtol=F32, rows=True)
        held(js.row_grad[t][:n_u], o["row_grads"][t], p["row_grads"][t], f"row grad {t}", rtol=F32, rows=True)
        u = torch.from_numpy(od_t[t]["uniq"]).long().cuda()
        held(tabs[t][u], o["new_rows"][t], p["new_rows"][t], f"updated rows {t}", rtol=F32)
        held(accs[t][u], o["new_accum"][t], p["new_accum"][t], f"accumulators {t}", rtol=F32)
    held(g["dE"], o["dE"], p["dE"], "dE", rows=True)
    fo = o["fwd"]
    flips1 = relu_flips(fo["Z"][0], g["H1"], TAU)
    flips2 = relu_flips(fo["Z"][1], g["H2"], TAU) if w.n_layers == 3 else []
    eW, eb = grad_flip_bounds(w.dims, Ws, T_u, fo, o["bwd"], flips1, flips2, None)
    for l in range(w.n_layers):
        held(g["dW"][l], o["bwd"]["dW"][l], p["dW"][l], f"dW{l + 1}", extra=eW[l])
        held(g["db"][l], o["bwd"]["db"][l], p["db"][l], f"db{l + 1}", extra=eb[l])


@pytest.mark.parametrize("name", ["tiny_joint", "mid_joint", "c4_joint"])
def test_joint_step_end_to_end(name):
    from tests.test_gpu_parity import compare_step
    w = mid_joint() if name == "mid_joint" else synth.get(name)
    print(f"joint step {name}", flush=True)
    batch, jb, Ws, T_u, js, g, o, tabs, accs, od_t = run_joint(w)
    # the image path, driven by the CTR model's input gradients: the whole
    # chain against the oracle at the small sizes, chained stage by stage at
    # the full size (see compare_image_chained)
    if name == "c4_joint":
        # the whole chain end to end, then each stage on the GPU's own inputs
        compare_joint_end_to_end(w, batch, jb, Ws, T_u, g, js, o, od_t, tabs, accs)
        compare_image_chained(w, batch, Ws, T_u, g, o, js.dU[:w.batch], js.dA[:w.batch])
    else:
        compare_step(w, "att", batch, Ws, T_u, g, o)
    # the worker side: bags, CTR, ID rows
    B = w.batch
    n_t = len(tabs)
    for t in range(n_t):
        assert int(js.t_status[t].item()) == 0
        n_u = int(js.t_nu[t].item())
        assert n_u == od_t[t]["n_uniq"]
        np.testing.assert_array_equal(js.t_uniq[t][:n_u].cpu().numpy(), od_t[t]["uniq"])
        assert_close(js.bags[t][:B], o["bags"][t], F32, f"bag {t}", rows=True)
    if name != "c4_joint":
        # the whole chain against the oracle
        c, dbags, grads, new_rows, new_acc = o["ctr"], o["dbags"], o["row_grads"], o["new_rows"], o["new_accum"]
        dU, dA = o["dU"], o["dA"]
    else:
        # chained, as the image path: the CTR model on the GPU's own input
        # fields (a hidden unit of one sample sits within the fp32 noise of U
        # and A from its ReLU tie), the row gradients of the GPU's bag
        # gradients, the Adagrad step of the GPU's row gradients
        X = np.concatenate([g["U"], g["A"]] + [f64(js.bags[t][:B]) for t in range(n_t)], axis=1)
        c = oracle.ctr_fwd_bwd(X, jb["labels"], *synth.make_ctr_weights(w))
        D = w.out_dim
        dU, dA = c["dX"][:, :D], c["dX"][:, D:2 * D]
        dbags = [c["dX"][:, 2 * D + 12 * t:2 * D + 12 * (t + 1)] for t in range(n_t)]
        grads, new_rows, new_acc = [], [], []
        for t in range(n_t):
            grads.append(oracle.merged_row_grad(batch["seg_off"], od_t[t]["inv"], od_t[t]["n_uniq"],
                                                f64(js.dbags[t][:B])))
            n_u = od_t[t]["n_uniq"]
            r0, a0 = o["_rows0"][t], o["_acc0"][t]
            nr, na = oracle.adagrad_rows(f64(js.row_grad[t][:n_u]), r0, a0, w.joint.lr, w.joint.eps)
            new_rows.append(nr)
            new_acc.append(na)
    for t in range(n_t):
        n_u = od_t[t]["n_uniq"]
        assert_close(js.dbags[t][:B], dbags[t], F32, f"dbag {t}", rows=True)
        assert_close(js.row_grad[t][:n_u], grads[t], F32, f"row grad {t}", rows=True)
        u = torch.from_numpy(od_t[t]["uniq"]).long().cuda()
        assert_close(tabs[t][u], new_rows[t], F32, f"updated rows {t}")
        assert_close(accs[t][u], new_acc[t], F32, f"accumulators {t}")
    assert abs(float(js.loss.item()) - c["loss"]) <= F32 * max(1.0, c["loss"])
    assert_close(js.prob[:B], c["prob"], F32, "prob")
    assert_close(js.dU[:B], dU, F32, "dU", rows=True)
    assert_close(js.dA[:B], dA, F32, "dA", rows=True)
    for l in range(len(js.ctr_dW)):
        assert_close(js.ctr_dW[l], c["dW"][l], F32, f"ctr dW{l + 1}")
        assert_close(js.ctr_db[l], c["db"][l], F32, f"ctr db{l + 1}")


@pytest.mark.parametrize("name", ["tiny_mqap", "mid_mqap", "c4_mqap"])
def test_mqap_joint_step_end_to_end(name):
    """MultiQueryAttentivePooling in the joint step (section 5.2): a second
    attentive channel with each ad's row of the category-sized ID table as its
    query, both pooled vectors into the CTR model (24-D), dE of both channels
    into the image model's backward and the query gradient into that table's
    rows before their Adagrad step.  The whole chain against the oracle at the
    small sizes; at full size (c4_mqap, 4096 samples) end to end with the
    sensitivity-bounded tolerance of the plain joint step."""
    from tests.test_gpu_parity import compare_step
    w = mid_joint(query_table=2) if name == "mid_mqap" else synth.get(name)
    print(f"mqap joint step {name}", flush=True)
    batch, jb, Ws, T_u, js, g, o, tabs, accs, od_t = run_joint(w)
    B, n_t = w.batch, len(tabs)
    assert js.query_table == 2 and synth.ctr_dims(w)[0] == 3 * w.out_dim + 12 * n_t
    if name == "c4_mqap":
        compare_joint_end_to_end(w, batch, jb, Ws, T_u, g, js, o, od_t, tabs, accs)
        return
    compare_step(w, "att", batch, Ws, T_u, g, o)
    n_beh = int(batch["seg_off"][-1])
    np.testing.assert_array_equal(f64(js.Q[:B]), o["Q"])            # a copy of table rows
    assert_close(js.U2[:B], o["query"]["U"], F32, "U2", rows=True)
    assert_close(js.w2[:n_beh], o["query"]["w"], F32, "query weights")
    c = o["ctr"]
    assert abs(float(js.loss.item()) - c["loss"]) <= F32 * max(1.0, c["loss"])
    assert_close(js.prob[:B], c["prob"], F32, "prob")
    assert_close(js.dU[:B], o["dU"], F32, "dU", rows=True)
    assert_close(js.dU2[:B], o["dU2"], F32, "dU2", rows=True)
    assert_close(js.dA[:B], o["dA"], F32, "dA", rows=True)
    assert_close(js.dQ[:B], o["query_bwd"]["dQ"], F32, "dQ", rows=True)
    for l in range(len(js.ctr_dW)):
        assert_close(js.ctr_dW[l], c["dW"][l], F32, f"ctr dW{l + 1}")
        assert_close(js.ctr_db[l], c["db"][l], F32, f"ctr db{l + 1}")
    for t in range(n_t):
        n_u = od_t[t]["n_uniq"]
        assert int(js.t_status[t].item()) == 0 and int(js.t_nu[t].item()) == n_u
        assert_close(js.bags[t][:B], o["bags"][t], F32, f"bag {t}", rows=True)
        assert_close(js.dbags[t][:B], o["dbags"][t], F32, f"dbag {t}", rows=True)
        assert_close(js.row_grad[t][:n_u], o["row_grads"][t], F32, f"row grad {t}", rows=True)
        u = torch.from_numpy(od_t[t]["uniq"]).long().cuda()
        assert_close(tabs[t][u], o["new_rows"][t], F32, f"updated rows {t}")
        assert_close(accs[t][u], o["new_accum"][t], F32, f"accumulators {t}")


@pytest.mark.parametrize("query", [False, True])
def test_joint_step_is_bitwise_deterministic(query):
    """The joint step twice from the same state (ID tables and accumulators
    restored), with each ID table's work on a side stream of its own beside
    the image path: every output, the updated rows and the accumulators bit for bit;
    also with the query channel (the query table's update then waits for dQ)."""
    w = mid_joint(query_table=2 if query else -1)
    tq = 2 if query else None
    batch = synth.make_batch(w)
    jb = synth.make_joint(w, batch)
    Ws, bs = synth.make_weights(w)
    cW, cb = synth.make_ctr_weights(w)
    T = synth.table_full(w, device="cuda")
    tabs0 = [synth.id_table_full(w, t, device="cuda") for t in range(len(w.joint.id_rows))]
    rng = np.random.default_rng(17)
    accs0 = [torch.from_numpy(rng.uniform(0.0, 0.1, size=tuple(x.shape)).astype(np.float32)).cuda() for x in tabs0]
    n_beh = int(batch["seg_off"][-1])
    occ = cuda_i32(synth.occurrences(batch))
    id_occ = [cuda_i32(synth.joint_occurrences(jb, t)) for t in range(len(tabs0))]
    outs = []
    for _ in range(2):
        js = ams.JointStep(w.dims, w.dtype, "att", w.batch, n_beh, w.joint.id_rows, w.joint.id_dim,
                           synth.ctr_dims(w), query_table=tq)
        tabs, accs = [x.clone() for x in tabs0], [x.clone() for x in accs0]
        js.run(occ, w.n_images, T, [x.cuda() for x in Ws], [x.cuda() for x in bs], cuda_i32(batch["seg_off"]),
               id_occ, tabs, accs, cuda_i32(jb["labels"]), [x.cuda() for x in cW], [x.cuda() for x in cb],
               w.joint.lr, w.joint.eps)
        torch.cuda.synchronize()
        g = gpu_outputs(js.img)
        g.update({"loss": js.loss.cpu().numpy(), "dU": f64(js.dU), "dA": f64(js.dA),
                  "tabs": [x.cpu().numpy() for x in tabs], "accs": [x.cpu().numpy() for x in accs],
                  "ctr_dW": [f64(x) for x in js.ctr_dW], "dbags": [f64(x) for x in js.dbags]})
        if query:
            g.update({"U2": f64(js.U2), "dQ": f64(js.dQ)})
        outs.append(g)
    a, b = outs
    for k in ("E", "U", "A", "dE", "loss", "dU", "dA") + (("U2", "dQ") if query else ()):
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)
    for k in ("dW", "db", "tabs", "accs", "ctr_dW", "dbags"):
        for x, y in zip(a[k], b[k]):
            np.testing.assert_array_equal(x, y, err_msg=k)
