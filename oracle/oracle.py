"""ctypes front end of the float64 CPU oracle (``ams_oracle.c``).

TEST INFRASTRUCTURE ONLY: used by the test suite, the smoke check and the
benchmark's CPU-baseline leg.  It imports nothing from the HIP library or its
Python binding, and the HIP path never imports this module.

Every function takes and returns numpy arrays (torch CPU tensors are accepted
as inputs).  Feature tables and weights may be float32 or bfloat16; bf16 values
are handed to the C code as raw bits and widened exactly to float64 there.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ams_oracle.c")
# AMS_ORACLE_LIB selects another build of the same source (the test that
# runs the oracle under AddressSanitizer/UBSan builds one with sanitize=True)
_LIB_PATH = os.environ.get("AMS_ORACLE_LIB") or os.path.join(_HERE, "libams_oracle.so")

POOL_SUM, POOL_MAX, POOL_ATT = 0, 1, 2
POOL_MODES = {"sum": POOL_SUM, "max": POOL_MAX, "att": POOL_ATT}
F32, BF16 = 0, 1

_lib = None


def build(force: bool = True, sanitize: bool = False, out: str | None = None) -> str:
    """Compile ams_oracle.c with gcc (plain -O2, IEEE semantics, OpenMP).
    sanitize: instrument with AddressSanitizer and UndefinedBehaviorSanitizer
    (every finding fatal); out: where the library goes (default: the one
    this module loads)."""
    path = out or _LIB_PATH
    if not force and os.path.exists(path) and os.path.getmtime(path) >= os.path.getmtime(_SRC):
        return path
    tmp = path + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-Wall", "-Wextra", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"]
    if sanitize:
        cmd[1:1] = ["-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, path)
    return path


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    lib.orc_dedup.argtypes = [P, i64, i32, P, P, P, P, P]
    lib.orc_mlp_fwd.argtypes = [ctypes.c_int, P, ctypes.c_int, P, i64, P, i32, P, P, ctypes.c_int, P, P]
    lib.orc_mlp_bwd.argtypes = [ctypes.c_int, P, ctypes.c_int, P, i64, P, i32, P, ctypes.c_int, P, P, P, P, P]
    lib.orc_pool_fwd.argtypes = [ctypes.c_int, i32, i32, P, i64, P, P, P, P, P, P]
    lib.orc_pool_bwd.argtypes = [ctypes.c_int, i32, i32, P, i64, P, i32, P, P, P, P, P, P, P, P, P, P]
    lib.orc_bag_fwd.argtypes = [i32, i32, P, i64, P, i64, P, P]
    lib.orc_ctr_fwd_bwd.argtypes = [i32, ctypes.c_int, P, P, P, P, P, P, P, P, P, P, P]
    lib.orc_adagrad_rows.argtypes = [i32, i32, P, ctypes.c_double, ctypes.c_double, P, P]
    lib.orc_pool_query_fwd.argtypes = [i32, i32, P, i64, P, P, P, P, P]
    lib.orc_pool_query_bwd.argtypes = [i32, i32, P, i64, P, i32, P, P, P, P, P, P, P]
    lib.orc_adam.argtypes = [i64, P, P, P, P, ctypes.c_double, ctypes.c_double, ctypes.c_double, ctypes.c_double, i64]
    lib.orc_pool_concat_fwd.argtypes = [i32, i32, i32, P, i64, P, P, P, P]
    lib.orc_pool_concat_bwd.argtypes = [i32, i32, i32, P, i64, P, i32, P, P, P]
    lib.orc_dense_fwd.argtypes = [i32, ctypes.c_int, P, P, P, P, P, P]
    lib.orc_dense_bwd.argtypes = [i32, ctypes.c_int, P, P, P, P, P, P, P, P, P, P]
    lib.orc_num_threads.restype = ctypes.c_int
    lib.orc_set_threads.argtypes = [ctypes.c_int]
    _lib = lib
    return lib


def num_threads() -> int:
    return _load().orc_num_threads()


def set_threads(n: int) -> None:
    _load().orc_set_threads(int(n))


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


def _i32(a):
    return np.ascontiguousarray(np.asarray(a), dtype=np.int32)


def _f64(a):
    return np.ascontiguousarray(np.asarray(a), dtype=np.float64)


def _store(x):
    """(array, dtype code) for a float32 or bfloat16 table/weight."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            x = x.detach().cpu().contiguous()
            if x.dtype == torch.bfloat16:
                return x.view(torch.int16).numpy().view(np.uint16), BF16
            return x.to(torch.float32).numpy(), F32
    except ImportError:  # pragma: no cover
        pass
    x = np.ascontiguousarray(x)
    if x.dtype == np.uint16:
        return x, BF16
    return np.ascontiguousarray(x, dtype=np.float32), F32


def _check(rc, what):
    if rc == 2:
        raise IndexError(f"{what}: image ID out of range")
    if rc != 0:
        raise ValueError(f"{what}: bad argument (rc={rc})")


# ------------------------------------------------------------------- dedup

def dedup(ids, n_ids: int) -> dict:
    lib = _load()
    ids = _i32(ids)
    n = ids.size
    uniq = np.zeros(max(n, 1), np.int32)
    inv = np.zeros(max(n, 1), np.int32)
    perm = np.zeros(max(n, 1), np.int32)
    off = np.zeros(n + 1, np.int32)
    nu = np.zeros(1, np.int32)
    _check(lib.orc_dedup(_ptr(ids), n, int(n_ids), _ptr(uniq), _ptr(inv), _ptr(perm), _ptr(off), _ptr(nu)), "dedup")
    k = int(nu[0])
    return {"uniq": uniq[:k].copy(), "inv": inv[:n].copy(), "occ_perm": perm[:n].copy(),
            "uniq_off": off[:k + 1].copy(), "n_uniq": k}


# --------------------------------------------------------------------- MLP

def _weights(Ws):
    arrs, codes = zip(*[_store(W) for W in Ws])
    if len(set(codes)) != 1:
        raise ValueError("mixed weight dtypes")
    return list(arrs), codes[0]


def mlp_fwd(T, rows, Ws, bs, final_relu: bool = False) -> dict:
    """E and per-layer pre-activations Z[l] for unique rows T[rows]."""
    lib = _load()
    Tn, tcode = _store(T)
    Wn, wcode = _weights(Ws)
    if tcode != wcode:
        raise ValueError("table and weights must share a storage dtype")
    dims = [Wn[0].shape[1]] + [W.shape[0] for W in Wn]
    if Tn.ndim != 2 or Tn.shape[1] != dims[0]:
        raise ValueError("table width does not match the first layer")
    rows = _i32(rows)
    n = rows.size
    L = len(Wn)
    bn = [np.ascontiguousarray(b, dtype=np.float32) if not hasattr(b, "numpy") else b.detach().cpu().float().numpy() for b in bs]
    Z = np.zeros(sum(n * d for d in dims[1:]) + 1, np.float64)
    E = np.zeros(max(n * dims[-1], 1), np.float64)
    dims_a = np.array(dims, np.int32)
    Wp = (ctypes.c_void_p * L)(*[W.ctypes.data for W in Wn])
    bp = (ctypes.c_void_p * L)(*[b.ctypes.data for b in bn])
    _check(lib.orc_mlp_fwd(L, _ptr(dims_a), tcode, _ptr(Tn), Tn.shape[0], _ptr(rows), n,
                           Wp, bp, int(final_relu), _ptr(Z), _ptr(E)), "mlp_fwd")
    Zs, o = [], 0
    for d in dims[1:]:
        Zs.append(Z[o:o + n * d].reshape(n, d).copy())
        o += n * d
    return {"E": E[:n * dims[-1]].reshape(n, dims[-1]).copy(), "Z": Zs, "dims": dims}


def mlp_bwd(T, rows, Ws, fwd: dict, dE, final_relu: bool = False) -> dict:
    """dW[l], db[l] (float64) and pre-activation gradients dZ[l]."""
    lib = _load()
    Tn, tcode = _store(T)
    Wn, _ = _weights(Ws)
    dims = fwd["dims"]
    rows = _i32(rows)
    n = rows.size
    L = len(Wn)
    Z = np.concatenate([z.reshape(-1) for z in fwd["Z"]] + [np.zeros(1)])
    dE = _f64(dE).reshape(-1)
    if dE.size != n * dims[-1]:
        raise ValueError("dE shape")
    nW = sum(dims[l] * dims[l + 1] for l in range(L))
    nb = sum(dims[1:])
    dW = np.zeros(nW, np.float64)
    db = np.zeros(nb, np.float64)
    dZ = np.zeros(Z.size, np.float64)
    dims_a = np.array(dims, np.int32)
    Wp = (ctypes.c_void_p * L)(*[W.ctypes.data for W in Wn])
    _check(lib.orc_mlp_bwd(L, _ptr(dims_a), tcode, _ptr(Tn), Tn.shape[0], _ptr(rows), n, Wp,
                           int(final_relu), _ptr(Z), _ptr(dE), _ptr(dW), _ptr(db), _ptr(dZ)), "mlp_bwd")
    dWs, dbs, dZs = [], [], []
    ow = ob = oz = 0
    for l in range(L):
        fi, fo = dims[l], dims[l + 1]
        dWs.append(dW[ow:ow + fi * fo].reshape(fo, fi).copy())
        dbs.append(db[ob:ob + fo].copy())
        dZs.append(dZ[oz:oz + n * fo].reshape(n, fo).copy())
        ow += fi * fo
        ob += fo
        oz += n * fo
    return {"dW": dWs, "db": dbs, "dZ": dZs}


# ----------------------------------------------------------------- pooling

def pool_fwd(mode, seg_off, inv, E, n_beh: int | None = None) -> dict:
    lib = _load()
    m = POOL_MODES[mode] if isinstance(mode, str) else int(mode)
    seg_off = _i32(seg_off)
    inv = _i32(inv)
    E = _f64(E)
    B = seg_off.size - 1
    D = E.shape[1]
    if n_beh is None:
        n_beh = int(seg_off[-1])
    U = np.zeros((B, D), np.float64)
    A = np.zeros((B, D), np.float64)
    am = np.full((B, D), -1, np.int32)
    w = np.zeros(max(n_beh, 1), np.float64)
    _check(lib.orc_pool_fwd(m, B, D, _ptr(seg_off), n_beh, _ptr(inv), _ptr(E), _ptr(U), _ptr(A),
                            _ptr(am), _ptr(w)), "pool_fwd")
    return {"U": U, "A": A, "argmax": am, "w": w[:n_beh].copy()}


def pool_bwd(mode, seg_off, inv, n_uniq: int, E, fwd: dict, gU, gA=None) -> dict:
    lib = _load()
    m = POOL_MODES[mode] if isinstance(mode, str) else int(mode)
    seg_off = _i32(seg_off)
    inv = _i32(inv)
    E = _f64(E)
    B = seg_off.size - 1
    D = E.shape[1]
    n_beh = int(seg_off[-1])
    gU = _f64(gU)
    gA = _f64(gA) if gA is not None else None
    w = np.ascontiguousarray(fwd["w"], np.float64)
    if w.size == 0:
        w = np.zeros(1)
    am = np.ascontiguousarray(fwd["argmax"], np.int32)
    dE = np.zeros((max(n_uniq, 1), D), np.float64)
    ge = np.zeros((n_beh + B, D), np.float64) if n_beh + B > 0 else np.zeros((1, D))
    dA = np.zeros((max(B, 1), D), np.float64)
    U, A = _f64(fwd["U"]), _f64(fwd["A"])      # held: read through raw pointers
    _check(lib.orc_pool_bwd(m, B, D, _ptr(seg_off), n_beh, _ptr(inv), int(n_uniq), _ptr(E),
                            _ptr(U), _ptr(A), _ptr(am), _ptr(w),
                            _ptr(gU), _ptr(gA), _ptr(dE), _ptr(ge), _ptr(dA)), "pool_bwd")
    return {"dE": dE[:n_uniq].copy(), "ge": ge[:n_beh + B].copy(), "dA_att": dA[:B].copy()}


# -------------------------------------------------------------- full step

def step(batch: dict, n_ids: int, T, Ws, bs, mode: str, final_relu: bool = False,
         table_is_compact: bool = False) -> dict:
    """One whole step: dedup -> MLP fwd -> pool fwd -> pool bwd -> MLP bwd.

    T is the full table ([n_ids, F]) or, with table_is_compact, just the rows
    of the batch's unique IDs in ascending ID order (as returned by dedup).
    """
    occ = np.concatenate([_i32(batch["beh_ids"]), _i32(batch["ad_ids"])])
    dd = dedup(occ, n_ids)
    rows = np.arange(dd["n_uniq"], dtype=np.int32) if table_is_compact else dd["uniq"]
    fw = mlp_fwd(T, rows, Ws, bs, final_relu)
    pf = pool_fwd(mode, batch["seg_off"], dd["inv"], fw["E"])
    pb = pool_bwd(mode, batch["seg_off"], dd["inv"], dd["n_uniq"], fw["E"], pf,
                  batch["g_u"], batch.get("g_a"))
    bw = mlp_bwd(T, rows, Ws, fw, pb["dE"], final_relu)
    return {"dedup": dd, "fwd": fw, "pool": pf, "pool_bwd": pb, "bwd": bw}


# ------------------------------------------------- joint step (worker side)

def bag_fwd(seg_off, idx, table) -> np.ndarray:
    """Per sample: sum of table[idx[j]] over its behaviors plus table[idx[n_beh + i]]."""
    lib = _load()
    seg_off = _i32(seg_off)
    idx = _i32(idx)
    tab = np.ascontiguousarray(np.asarray(table.detach().cpu() if hasattr(table, "detach") else table),
                               dtype=np.float32)
    B = seg_off.size - 1
    D = tab.shape[1]
    n_beh = int(seg_off[-1])
    if idx.size != n_beh + B:
        raise ValueError("idx must hold the behaviors then one ad per sample")
    bag = np.zeros((max(B, 1), D), np.float64)
    _check(lib.orc_bag_fwd(B, D, _ptr(seg_off), n_beh, _ptr(idx), tab.shape[0], _ptr(tab), _ptr(bag)),
           "bag_fwd")
    return bag[:B].copy()


def _f32list(xs):
    return [np.ascontiguousarray(np.asarray(x.detach().cpu() if hasattr(x, "detach") else x),
                                 dtype=np.float32) for x in xs]


def ctr_fwd_bwd(X, labels, Ws, bs) -> dict:
    """CTR MLP with softmax cross-entropy (mean over the batch): loss, prob,
    pre-activations Z[l], gradients dW[l], db[l] and dX."""
    lib = _load()
    X = _f64(X)
    labels = _i32(labels)
    Wn, bn = _f32list(Ws), _f32list(bs)
    L = len(Wn)
    dims = [Wn[0].shape[1]] + [W.shape[0] for W in Wn]
    B = X.shape[0]
    if X.shape[1] != dims[0] or labels.size != B:
        raise ValueError("shapes")
    loss = np.zeros(1, np.float64)
    prob = np.zeros((B, dims[-1]), np.float64)
    Z = np.zeros(sum(B * d for d in dims[1:]), np.float64)
    dW = np.zeros(sum(a * b for a, b in zip(dims[:-1], dims[1:])), np.float64)
    db = np.zeros(sum(dims[1:]), np.float64)
    dX = np.zeros_like(X)
    Wp = (ctypes.c_void_p * L)(*[W.ctypes.data for W in Wn])
    bp = (ctypes.c_void_p * L)(*[b.ctypes.data for b in bn])
    dims_a = np.array(dims, np.int32)
    _check(lib.orc_ctr_fwd_bwd(B, L, _ptr(dims_a), Wp, bp, _ptr(X), _ptr(labels), _ptr(loss), _ptr(prob),
                               _ptr(Z), _ptr(dW), _ptr(db), _ptr(dX)), "ctr_fwd_bwd")
    Zs, dWs, dbs = [], [], []
    oz = ow = ob = 0
    for fi, fo in zip(dims[:-1], dims[1:]):
        Zs.append(Z[oz:oz + B * fo].reshape(B, fo).copy())
        dWs.append(dW[ow:ow + fi * fo].reshape(fo, fi).copy())
        dbs.append(db[ob:ob + fo].copy())
        oz += B * fo
        ow += fi * fo
        ob += fo
    return {"loss": float(loss[0]), "prob": prob, "Z": Zs, "dW": dWs, "db": dbs, "dX": dX}


def adagrad_rows(grad, rows, accum, lr: float, eps: float):
    """One sparse Adagrad step of the touched rows (row-compact): returns the
    new rows and accumulators (float64)."""
    lib = _load()
    g = _f64(grad)
    r = _f64(rows).copy()
    a = _f64(accum).copy()
    n, D = g.shape
    _check(lib.orc_adagrad_rows(n, D, _ptr(g), float(lr), float(eps), _ptr(r), _ptr(a)), "adagrad_rows")
    return r, a


def merged_row_grad(seg_off, inv, n_uniq: int, dbag, dad=None) -> np.ndarray:
    """Gradient of every touched row: the sum over its occurrences (ascending)
    of the bag gradient of the sample each belongs to (the SUM aggregator's
    backward with the bag gradient as upstream for behaviors and ad alike).
    dad: a second gradient of each sample's ad row (the ad's ID embedding
    also being the query of an attentive channel, section 5.2), added to
    what the ad occurrence carries."""
    dbag = _f64(dbag)
    D = dbag.shape[1]
    B = dbag.shape[0]
    g_ad = dbag if dad is None else dbag + _f64(dad)
    fwd = {"U": np.zeros((B, D)), "A": np.zeros((B, D)), "w": np.zeros(1), "argmax": np.full((B, D), -1, np.int32)}
    return pool_bwd("sum", seg_off, inv, n_uniq, np.zeros((max(n_uniq, 1), D)), fwd, dbag, g_ad)["dE"]


def joint_step(batch: dict, jb: dict, spec, n_ids: int, T, Ws, bs, id_rows, ctr_Ws, ctr_bs, accum,
               mode: str = "att", table_is_compact: bool = True, query_table=None) -> dict:
    """One joint training step (Algorithm 1: worker iteration, server embed and
    update) in float64.

    batch / jb:  image batch (make_batch) and its ID features (make_joint)
    T:           image feature rows of the batch's unique images (compact, ascending
                 ID) or the whole table
    id_rows[t]:  rows of ID table t for its unique IDs (ascending), float32
    accum[t]:    their Adagrad accumulators
    spec:        the workload's JointSpec (lr, eps)
    query_table: None, or the ID table t_q whose ad row is the query of a
                 second attentive channel (MultiQueryAttentivePooling, section
                 5.2): Q_i = the ad's row of t_q, U2 = pool_query_fwd(E, Q),
                 the CTR input [U, U2, A, bags...]; the backward adds the ID
                 channel's dE to the image channel's and the query gradient
                 dQ_i to the ad occurrence's row gradient in table t_q.
    Returns the image-step pieces (dedup, fwd, pool, pool_bwd, bwd), the ID
    dedups, bags, the CTR forward/backward, the merged row gradients and the
    Adagrad results (new rows and accumulators, float64); with a query table
    also Q, the query channel's forward and backward and dU2.
    """
    occ = np.concatenate([_i32(batch["beh_ids"]), _i32(batch["ad_ids"])])
    dd = dedup(occ, n_ids)
    rows = np.arange(dd["n_uniq"], dtype=np.int32) if table_is_compact else dd["uniq"]
    fw = mlp_fwd(T, rows, Ws, bs)
    pf = pool_fwd(mode, batch["seg_off"], dd["inv"], fw["E"])
    n_t = len(jb["beh_ids"])
    idd, bags = [], []
    for t in range(n_t):
        o_t = np.concatenate([_i32(jb["beh_ids"][t]), _i32(jb["ad_ids"][t])])
        idd.append(dedup(o_t, spec.id_rows[t]))
        bags.append(bag_fwd(batch["seg_off"], idd[t]["inv"], id_rows[t]))
    D = pf["U"].shape[1]
    mq = query_table is not None
    users = [pf["U"]]
    if mq:
        n_beh = int(batch["seg_off"][-1])
        Q = _f64(id_rows[query_table])[idd[query_table]["inv"][n_beh:]]      # each sample's ad row
        pq = pool_query_fwd(batch["seg_off"], dd["inv"], fw["E"], Q)
        users.append(pq["U"])
    X = np.concatenate(users + [pf["A"]] + bags, axis=1)
    cf = ctr_fwd_bwd(X, jb["labels"], ctr_Ws, ctr_bs)
    dU = cf["dX"][:, :D]
    o = D
    if mq:
        dU2 = cf["dX"][:, o:o + D]
        o += D
    dA = cf["dX"][:, o:o + D]
    o += D
    dbags = []
    for t in range(n_t):
        w_t = bags[t].shape[1]
        dbags.append(cf["dX"][:, o:o + w_t])
        o += w_t
    pb = pool_bwd(mode, batch["seg_off"], dd["inv"], dd["n_uniq"], fw["E"], pf, dU, dA)
    dE = pb["dE"]
    if mq:
        qb = pool_query_bwd(batch["seg_off"], dd["inv"], dd["n_uniq"], fw["E"], Q, pq, dU2)
        dE = dE + qb["dE"]
    bw = mlp_bwd(T, rows, Ws, fw, dE)
    grads, new_rows, new_acc = [], [], []
    for t in range(n_t):
        dad = qb["dQ"] if mq and t == query_table else None
        g = merged_row_grad(batch["seg_off"], idd[t]["inv"], idd[t]["n_uniq"], dbags[t], dad)
        grads.append(g)
        r, a = adagrad_rows(g, id_rows[t], accum[t], spec.lr, spec.eps)
        new_rows.append(r)
        new_acc.append(a)
    out = {"dedup": dd, "fwd": fw, "pool": pf, "pool_bwd": pb, "bwd": bw, "id_dedup": idd, "bags": bags,
           "X": X, "ctr": cf, "dU": dU, "dA": dA, "dbags": dbags, "dE": dE, "row_grads": grads,
           "new_rows": new_rows, "new_accum": new_acc}
    if mq:
        out.update({"Q": Q, "query": pq, "query_bwd": qb, "dU2": dU2})
    return out


# ------------------------------------------------- multiple-query attention

def pool_query_fwd(seg_off, inv, E, Q) -> dict:
    """One attentive channel with a per-sample query Q [B x D]."""
    lib = _load()
    seg_off = _i32(seg_off)
    inv = _i32(inv)
    E, Q = _f64(E), _f64(Q)
    B, D = seg_off.size - 1, E.shape[1]
    n_beh = int(seg_off[-1])
    U = np.zeros((max(B, 1), D))
    w = np.zeros(max(n_beh, 1))
    _check(lib.orc_pool_query_fwd(B, D, _ptr(seg_off), n_beh, _ptr(inv), _ptr(E), _ptr(Q), _ptr(U), _ptr(w)),
           "pool_query_fwd")
    return {"U": U[:B].copy(), "w": w[:n_beh].copy()}


def pool_query_bwd(seg_off, inv, n_uniq: int, E, Q, fwd: dict, gU) -> dict:
    """dE (merged per unique image, behaviors only) and dQ of one query channel."""
    lib = _load()
    seg_off = _i32(seg_off)
    inv = _i32(inv)
    E, Q, gU = _f64(E), _f64(Q), _f64(gU)
    B, D = seg_off.size - 1, E.shape[1]
    n_beh = int(seg_off[-1])
    w = np.ascontiguousarray(fwd["w"], np.float64)
    if w.size == 0:
        w = np.zeros(1)
    dE = np.zeros((max(n_uniq, 1), D))
    dQ = np.zeros((max(B, 1), D))
    U = _f64(fwd["U"])                         # held: read through a raw pointer
    _check(lib.orc_pool_query_bwd(B, D, _ptr(seg_off), n_beh, _ptr(inv), int(n_uniq), _ptr(E), _ptr(Q),
                                  _ptr(U), _ptr(w), _ptr(gU), _ptr(dE), _ptr(dQ)), "pool_query_bwd")
    return {"dE": dE[:n_uniq].copy(), "dQ": dQ[:B].copy()}


# ------------------------------------------------------------- dense update

def adam(param, grad, m, v, lr: float, t: int, b1: float = 0.9, b2: float = 0.999, eps: float = 1e-8):
    """One Adam step (t >= 1) in float64; returns new (param, m, v)."""
    lib = _load()
    p, g = _f64(param).copy(), _f64(grad)
    mm, vv = _f64(m).copy(), _f64(v).copy()
    _check(lib.orc_adam(p.size, _ptr(p), _ptr(g), _ptr(mm), _ptr(vv), float(lr), float(b1), float(b2), float(eps),
                        int(t)), "adam")
    return p, mm, vv


def paper_lr(step: int, lr0: float = 1e-3, decay: float = 0.9, every: int = 24000) -> float:
    """Section 7.2: the learning rate starts at 1e-3 and is multiplied by 0.9
    after every 24,000 batches (step counts from 1)."""
    return lr0 * decay ** ((step - 1) // every)


# ------------------------------------------------- concatenate aggregator

def pool_concat_fwd(seg_off, inv, E, Lc: int) -> dict:
    """U [B x Lc*D]: the first Lc behavior embeddings side by side (zero
    padded); A: the ads' embeddings."""
    lib = _load()
    seg_off, inv, E = _i32(seg_off), _i32(inv), _f64(E)
    B, D = seg_off.size - 1, E.shape[1]
    n_beh = int(seg_off[-1])
    U = np.zeros((max(B, 1), Lc * D))
    A = np.zeros((max(B, 1), D))
    _check(lib.orc_pool_concat_fwd(B, D, int(Lc), _ptr(seg_off), n_beh, _ptr(inv), _ptr(E), _ptr(U), _ptr(A)),
           "pool_concat_fwd")
    return {"U": U[:B].copy(), "A": A[:B].copy()}


def pool_concat_bwd(seg_off, inv, n_uniq: int, D: int, Lc: int, gU, gA=None) -> np.ndarray:
    """dE [n_u x D]: each kept position's slice of gU (and gA for the ads),
    merged per unique image in ascending occurrence order."""
    lib = _load()
    seg_off, inv = _i32(seg_off), _i32(inv)
    B = seg_off.size - 1
    n_beh = int(seg_off[-1])
    gU = _f64(gU).reshape(B, Lc * D) if B else np.zeros((1, Lc * D))
    gA = _f64(gA) if gA is not None else None
    dE = np.zeros((max(n_uniq, 1), D))
    _check(lib.orc_pool_concat_bwd(B, D, int(Lc), _ptr(seg_off), n_beh, _ptr(inv), int(n_uniq), _ptr(gU),
                                   _ptr(gA), _ptr(dE)), "pool_concat_bwd")
    return dE[:n_uniq].copy()


# ------------------------------------------- dense nets with PReLU, pre-rank

def _ptr_list(xs):
    return (ctypes.c_void_p * len(xs))(*[None if x is None else x.ctypes.data for x in xs])


def dense_fwd(X, Ws, bs, slopes=None) -> list:
    """Z of every layer of a fully connected net (PReLU with per-channel
    slopes between layers, ReLU where a slope is None, last layer linear)."""
    lib = _load()
    X = _f64(X)
    Wn, bn = _f32list(Ws), _f32list(bs)
    L = len(Wn)
    dims = [Wn[0].shape[1]] + [W.shape[0] for W in Wn]
    sl = [None] * L if slopes is None else [None if s is None else _f32list([s])[0] for s in slopes] + [None]
    B = X.shape[0]
    Z = np.zeros(max(sum(B * d for d in dims[1:]), 1))
    dims_a = np.array(dims, np.int32)          # held: the C call reads it through a raw pointer
    _check(lib.orc_dense_fwd(B, L, _ptr(dims_a), _ptr_list(Wn), _ptr_list(bn), _ptr_list(sl[:L]),
                             _ptr(X), _ptr(Z)), "dense_fwd")
    out, o = [], 0
    for d in dims[1:]:
        out.append(Z[o:o + B * d].reshape(B, d).copy())
        o += B * d
    return out


def dense_bwd(X, Ws, slopes, Z: list, dZL) -> dict:
    """dW, db, dslope (one per hidden layer) and dX of dense_fwd's net."""
    lib = _load()
    X = _f64(X)
    Wn = _f32list(Ws)
    L = len(Wn)
    dims = [Wn[0].shape[1]] + [W.shape[0] for W in Wn]
    sl = [None] * L if slopes is None else [None if s is None else _f32list([s])[0] for s in slopes] + [None]
    B = X.shape[0]
    Zc = np.ascontiguousarray(np.concatenate([np.asarray(z, np.float64).ravel() for z in Z]))
    dW = np.zeros(sum(a * b for a, b in zip(dims[:-1], dims[1:])))
    db = np.zeros(sum(dims[1:]))
    ds = np.zeros(max(sum(dims[1:-1]), 1))
    dX = np.zeros_like(X)
    dims_a, dZL = np.array(dims, np.int32), _f64(dZL)   # held: read through raw pointers
    _check(lib.orc_dense_bwd(B, L, _ptr(dims_a), _ptr_list(Wn), _ptr_list(sl[:L]), _ptr(X),
                             _ptr(Zc), _ptr(dZL), _ptr(dW), _ptr(db), _ptr(ds), _ptr(dX)), "dense_bwd")
    dWs, dbs, dss = [], [], []
    ow = ob = os_ = 0
    for l, (fi, fo) in enumerate(zip(dims[:-1], dims[1:])):
        dWs.append(dW[ow:ow + fi * fo].reshape(fo, fi).copy())
        dbs.append(db[ob:ob + fo].copy())
        ow += fi * fo
        ob += fo
        if l < L - 1:
            dss.append(ds[os_:os_ + fo].copy())
            os_ += fo
    return {"dW": dWs, "db": dbs, "dslope": dss, "dX": dX}


def ctr_act_fwd_bwd(X, labels, Ws, bs, slopes=None) -> dict:
    """The CTR model with PReLU (or ReLU) between layers: softmax over the
    classes, cross-entropy summed over the samples whose label is a class and
    divided by B (others add nothing); its gradients, slopes' included."""
    labels = np.asarray(labels, np.int64)
    Z = dense_fwd(X, Ws, bs, slopes)
    z = Z[-1]
    B, C = z.shape
    m = z.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(z - m).sum(axis=1))
    prob = np.exp(z - lse[:, None])
    ok = (labels >= 0) & (labels < C)
    y = np.where(ok, labels, 0)
    loss = float(np.where(ok, lse - z[np.arange(B), y], 0.0).sum() / B)
    dz = (prob - np.eye(C)[y]) / B
    dz[~ok] = 0.0
    g = dense_bwd(X, Ws, slopes, Z, dz)
    return {"loss": loss, "prob": prob, "Z": Z, **g}


def dssm_fwd_bwd(Xu, Xa, labels, user, ad) -> dict:
    """Pre-rank model of section 6: user tower on Xu, ad tower on Xa (each
    ``(Ws, bs, slopes)``, equal output widths), score s = <u, a>, click
    probability sigmoid(s), logistic loss softplus(s) - y s summed over the
    samples with y in {0, 1} and divided by B; gradients of both towers and
    of both inputs."""
    labels = np.asarray(labels, np.int64)
    Zu = dense_fwd(Xu, *user)
    Za = dense_fwd(Xa, *ad)
    u, a = Zu[-1], Za[-1]
    B = u.shape[0]
    s = (u * a).sum(axis=1)
    prob = 1.0 / (1.0 + np.exp(-s))
    ok = (labels == 0) | (labels == 1)
    y = np.where(ok, labels, 0).astype(np.float64)
    softplus = np.maximum(s, 0.0) + np.log1p(np.exp(-np.abs(s)))
    loss = float(np.where(ok, softplus - y * s, 0.0).sum() / B)
    dS = np.where(ok, (prob - y) / B, 0.0)
    gu = dense_bwd(Xu, user[0], user[2], Zu, dS[:, None] * a)
    ga = dense_bwd(Xa, ad[0], ad[2], Za, dS[:, None] * u)
    return {"loss": loss, "prob": prob, "score": s, "u": u, "a": a, "user": gu, "ad": ga}
