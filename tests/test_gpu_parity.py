"""GPU parity: libams (through its C ABI) against the float64 oracle.

Per call, each entry point gets inputs identical to the oracle's (the oracle's
dedup, embeddings, pooled vectors, saved activations), so every decision is
the same on both sides; end to end, whole steps run through the library and
are compared with decisions checked as in tests/parity.py.  Sizes span several
tiles with ragged tails; the 1024-sample fp32 workload runs at full size in
the same launch configuration the benchmark times.
"""
import dataclasses
import functools

import numpy as np
import pytest
import torch

from oracle import oracle
from paper_1711_06505_amd import ams, synth
from tests.parity import (RTOL, assert_close, device_batch, f64, gpu_outputs, grad_flip_bounds,
                          large_grid_workload, max_flips, relu_flips, run_gpu_step)

pytestmark = pytest.mark.gpu

TAU = 1e-4   # near-tie window for floating-point decisions, relative to the tensor RMS


def mid(dtype="f32", B=96, n_images=20_000, index=11):
    base = synth.get("c1_f32" if dtype == "f32" else "c2_bf16")
    return dataclasses.replace(base, name=f"mid_{dtype}", index=index, batch=B, n_images=n_images,
                               pools=("sum", "max", "att"), stream=-1)


def mid_l2():
    """The mid bf16 batch through a two-layer MLP 4096-256-12 (the
    two-layer instances of the bf16 tails)."""
    return dataclasses.replace(mid("bf16"), name="mid_bf16_l2", dims=(4096, 256, 12))


def named(wname):
    return synth.get("tiny") if wname == "tiny" else mid_l2() if wname == "mid_bf16_l2" else mid(wname[4:])


def cuda_i32(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).cuda()


def gpu_dedup(occ, n_ids):
    occ = np.asarray(occ, np.int32)
    n = occ.size
    ids = cuda_i32(occ) if n else torch.zeros(1, dtype=torch.int32, device="cuda")
    m = max(n, 1)
    out = {k: torch.full((m,), -7, dtype=torch.int32, device="cuda") for k in ("uniq", "inv", "perm")}
    off = torch.full((n + 1,), -7, dtype=torch.int32, device="cuda")
    nu = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    stt = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(ams.ams_dedup_workspace(n, n_ids), 256), dtype=torch.uint8, device="cuda")
    ams.ams_dedup(ids[:n] if n else ids[:0], n_ids, out["uniq"], out["inv"], out["perm"], off, nu, stt, ws)
    torch.cuda.synchronize()
    k = int(nu.item())
    return {"uniq": out["uniq"][:k].cpu().numpy(), "inv": out["inv"][:n].cpu().numpy(),
            "occ_perm": out["perm"][:n].cpu().numpy(), "uniq_off": off[:k + 1].cpu().numpy(),
            "n_uniq": k, "status": int(stt.item())}


def check_dedup(g, o):
    assert g["status"] == 0
    assert g["n_uniq"] == o["n_uniq"]
    for k in ("uniq", "inv", "occ_perm", "uniq_off"):
        np.testing.assert_array_equal(g[k], o[k], err_msg=k)


# ------------------------------------------------------------------ dedup

def test_library_is_the_in_tree_build():
    ams.load()
    maps = open("/proc/self/maps").read()
    assert ams.LIB_PATH in maps


@pytest.mark.parametrize("name", ["tiny", "c1_f32", "c3_long"])
def test_dedup_bit_exact_on_workloads(name):
    w = synth.get(name)
    occ = synth.occurrences(synth.make_batch(w))
    print(f"dedup {name}: n_occ={occ.size}", flush=True)
    check_dedup(gpu_dedup(occ, w.n_images), oracle.dedup(occ, w.n_images))


@pytest.mark.parametrize("n,n_ids,kind", [
    (0, 10, "rand"), (1, 10, "rand"), (1, 1, "rand"), (5000, 1, "rand"), (2047, 300, "rand"),
    (2048, 300, "rand"), (2049, 300, "rand"), (4097, 2 ** 21, "rand"), (10000, 7, "desc"),
    (65537, 2 ** 31 - 1, "rand"), (3000, 2 ** 21, "top"), (40000, 200_000, "same"),
    # larger batches: 2^19 - 1 and 2^19 occurrences, a ragged last tile, all
    # keys equal, descending keys over 24 bits (three passes of 8)
    (2 ** 19 - 1, 2 ** 21, "rand"), (2 ** 19, 2 ** 31 - 1, "rand"), (2 ** 19 + 8193, 300, "rand"),
    (600_000, 200_000, "same"), (2 ** 20, 2 ** 24, "desc"),
    # pass widths: 9 bits in two passes of 5, 18 bits in three of 6, 19 bits
    # in three of 7, 27 bits in four of 7
    (5000, 512, "rand"), (70_000, 2 ** 18, "rand"), (9000, 2 ** 18 + 1, "rand"), (100_000, 2 ** 27, "rand"),
])
def test_dedup_edges(n, n_ids, kind):
    rng = np.random.default_rng(n + n_ids)
    if kind == "rand":
        occ = rng.integers(0, n_ids, size=n)
    elif kind == "desc":
        occ = np.sort(rng.integers(0, n_ids, size=n))[::-1]
    elif kind == "top":
        occ = n_ids - 1 - rng.integers(0, 3, size=n)
    else:
        occ = np.full(n, 123_456)
    occ = occ.astype(np.int32)
    print(f"dedup edge n={n} n_ids={n_ids} {kind}", flush=True)
    check_dedup(gpu_dedup(occ, n_ids), oracle.dedup(occ, n_ids))


@pytest.mark.parametrize("bad", [50, -1, 2 ** 31 - 1])
def test_dedup_flags_out_of_range_ids(bad):
    occ = np.arange(4000, dtype=np.int64) % 50
    occ[1234] = bad
    g = gpu_dedup(occ.astype(np.int32), 50)
    assert g["status"] == 7


# ------------------------------------------------------------ embed fwd

@functools.lru_cache(maxsize=8)
def embed_case(w, seed_k=0):
    batch = synth.make_batch(w, k=seed_k)
    occ = synth.occurrences(batch)
    dd = oracle.dedup(occ, w.n_images)
    Ws, bs = synth.make_weights(w)
    T_u = synth.table_rows(w, dd["uniq"])               # CPU rows for the oracle
    return batch, dd, Ws, bs, T_u


def gpu_embed_fwd(w, T_dev, uniq, Ws, bs, cap=None):
    n_u = len(uniq)
    cap = n_u if cap is None else cap
    mlp = ams.make_mlp(w.dims, w.dtype)
    H = w.dims[1]
    d_uniq = torch.zeros(max(cap, 1), dtype=torch.int32, device="cuda")
    d_uniq[:n_u] = cuda_i32(uniq)
    nu = torch.tensor([n_u], dtype=torch.int32, device="cuda")
    H1 = torch.zeros((max(cap, 1), H), dtype=torch.bfloat16 if w.dtype == "bf16" else torch.float32,
                     device="cuda")
    H2 = torch.zeros((max(cap, 1), w.dims[2]), device="cuda") if w.n_layers == 3 else None
    E = torch.zeros((max(cap, 1), w.out_dim), device="cuda")
    ws = torch.empty(max(ams.ams_embed_workspace(mlp, cap), 256), dtype=torch.uint8, device="cuda")
    ams.ams_embed_fwd(mlp, T_dev, d_uniq, nu, cap, [W.cuda() for W in Ws], [b.cuda() for b in bs],
                      H1, H2, E, ws)
    torch.cuda.synchronize()
    return {"E": f64(E[:n_u]), "H1": f64(H1[:n_u]), "H2": f64(H2[:n_u]) if H2 is not None else None}


@pytest.mark.parametrize("wname", ["tiny", "mid_f32", "mid_bf16", "mid_bf16_l2"])
def test_embed_fwd_matches_oracle(wname):
    w = named(wname)
    batch, dd, Ws, bs, T_u = embed_case(w)
    print(f"embed fwd {wname}: n_u={dd['n_uniq']}", flush=True)
    T_dev = synth.table_rows(w, np.arange(w.n_images), device="cuda")
    g = gpu_embed_fwd(w, T_dev, dd["uniq"], Ws, bs, cap=dd["n_uniq"] + 77)
    o = oracle.mlp_fwd(T_u, np.arange(dd["n_uniq"]), Ws, bs)
    rt = RTOL[w.dtype]
    assert_close(g["E"], o["E"], rt, "E")
    assert_close(g["H1"], np.maximum(o["Z"][0], 0), rt, "H1")
    if w.n_layers == 3:
        assert_close(g["H2"], np.maximum(o["Z"][1], 0), rt, "H2")
    # the bf16 path keeps fp32 accumulation: its forward is far inside 2e-2
    assert_close(g["E"], o["E"], 1e-4, "E (fp32-accumulation accuracy)")


# From this capacity on, the bf16 first layer runs as the row-split kernel
# (each CU a contiguous range of the unique rows); small batches with such a
# capacity leave most CUs a few rows or none, with ragged last tiles.
ROW_SPLIT_CAP = 2 * 256 * 256


@pytest.mark.parametrize("case", ["few_rows", "mid", "c2", "bad_ids"])
def test_embed_fwd_bf16_row_split_matches_oracle(case):
    w = synth.get("c2_bf16") if case == "c2" else mid("bf16")
    batch, dd, Ws, bs, T_u = embed_case(w)
    rows = np.arange(dd["n_uniq"])
    uniq = dd["uniq"].copy()
    if case == "few_rows":                       # fewer rows than CUs
        rows, uniq = rows[:100], uniq[:100]
    T_rows = T_u[rows]
    if case == "bad_ids":                        # out-of-range IDs read as zero rows
        uniq[[3, 700, len(uniq) - 1]] = [w.n_images + 5, -3, w.n_images]
        T_rows = T_rows.clone()
        T_rows[[3, 700, len(uniq) - 1]] = 0
    print(f"row-split embed fwd {case}: n_u={len(uniq)} cap={ROW_SPLIT_CAP + 13}", flush=True)
    T_dev = synth.table_rows(w, np.arange(w.n_images), device="cuda")
    g = gpu_embed_fwd(w, T_dev, uniq, Ws, bs, cap=ROW_SPLIT_CAP + 13)
    o = oracle.mlp_fwd(T_rows, np.arange(len(uniq)), Ws, bs)
    assert_close(g["E"], o["E"], 1e-4, "E")                      # fp32 accumulation
    assert_close(g["H1"], np.maximum(o["Z"][0], 0), RTOL["bf16"], "H1 (bf16 copy)")
    assert_close(g["H2"], np.maximum(o["Z"][1], 0), RTOL["bf16"], "H2")


def test_embed_fwd_out_of_range_row_reads_zero():
    w = synth.get("tiny")
    Ws, bs = synth.make_weights(w)
    T_dev = synth.table_rows(w, np.arange(w.n_images), device="cuda")
    g = gpu_embed_fwd(w, T_dev, np.array([5, w.n_images + 3, -2, 7], np.int32), Ws, bs)
    z = oracle.mlp_fwd(torch.zeros((1, w.in_dim)), [0], Ws, bs)["E"][0]
    assert_close(g["E"][1], z, 1e-5, "zero row")
    assert_close(g["E"][2], z, 1e-5, "negative row")


# ------------------------------------------------------------- pooling

def pool_case(w, mode, seed_k=0):
    batch, dd, Ws, bs, T_u = embed_case(w, seed_k)
    E = oracle.mlp_fwd(T_u, np.arange(dd["n_uniq"]), Ws, bs)["E"].astype(np.float32)  # GPU input
    return batch, dd, E


def gpu_pool(mode, batch, dd, E32, pf_orc=None, unit=False):
    db = device_batch(batch)
    B, n_beh, D = db["B"], db["n_beh"], E32.shape[1]
    n_u = dd["n_uniq"]
    E = torch.from_numpy(E32).cuda()
    inv = cuda_i32(dd["inv"])
    U = torch.zeros((B, D), device="cuda")
    A = torch.zeros((B, D), device="cuda")
    saved = (torch.zeros((B, D), dtype=torch.int32, device="cuda") if mode == "max" else
             torch.zeros(max(n_beh, 1), device="cuda") if mode == "att" else None)
    ams.ams_pool_fwd(mode, db["seg_off"], n_beh, inv, E, U, A, saved)
    torch.cuda.synchronize()
    fwd = {"U": f64(U), "A": f64(A)}
    if mode == "att":
        fwd["w"] = f64(saved[:n_beh])
    if mode == "max":
        fwd["argmax"] = saved.cpu().numpy()
    # backward with the oracle's forward state as input
    if pf_orc is not None:
        U.copy_(torch.from_numpy(pf_orc["U"].astype(np.float32)))
        A.copy_(torch.from_numpy(pf_orc["A"].astype(np.float32)))
        if mode == "att":
            saved[:n_beh].copy_(torch.from_numpy(pf_orc["w"].astype(np.float32)))
        if mode == "max":
            saved.copy_(torch.from_numpy(pf_orc["argmax"]))
    dU, dA = db["dU"], db["dA"]
    if unit:
        dU, dA = torch.ones_like(dU), None
    dE = torch.full((n_u + 5, D), float("nan"), device="cuda")
    nu = torch.tensor([n_u], dtype=torch.int32, device="cuda")
    ws = torch.empty(max(ams.ams_pool_workspace(mode, B, n_beh, D, n_u), 256), dtype=torch.uint8,
                     device="cuda")
    ams.ams_pool_bwd(mode, db["seg_off"], n_beh, inv, cuda_i32(dd["occ_perm"]), cuda_i32(dd["uniq_off"]),
                     nu, n_u, E, U, A, saved, dU, dA, dE, ws)
    torch.cuda.synchronize()
    return fwd, f64(dE[:n_u])


@pytest.mark.parametrize("mode", ["sum", "max", "att"])
@pytest.mark.parametrize("wname", ["tiny", "mid_f32", "c1_f32"])
def test_pool_fwd_bwd_match_oracle(mode, wname):
    w = synth.get(wname) if wname in ("tiny", "c1_f32") else mid("f32")
    batch, dd, E32 = pool_case(w, mode)
    print(f"pool {mode} {wname}: B={batch['seg_off'].size - 1} n_u={dd['n_uniq']}", flush=True)
    pf = oracle.pool_fwd(mode, batch["seg_off"], dd["inv"], E32)
    pb = oracle.pool_bwd(mode, batch["seg_off"], dd["inv"], dd["n_uniq"], E32, pf, batch["g_u"], batch["g_a"])
    fwd, dE = gpu_pool(mode, batch, dd, E32, pf_orc=pf)
    assert_close(fwd["U"], pf["U"], 1e-4, "U")
    np.testing.assert_array_equal(fwd["A"], pf["A"])                 # a copy of E rows
    if mode == "max":
        np.testing.assert_array_equal(fwd["argmax"], pf["argmax"])   # identical inputs: exact
        np.testing.assert_array_equal(fwd["U"], pf["U"])
    if mode == "att":
        assert_close(fwd["w"], pf["w"], 1e-4, "attention weights")
    assert_close(dE, pb["dE"], 1e-4, "dE")


@pytest.mark.parametrize("size", ["c3_long", "large_grid"])
@pytest.mark.parametrize("mode", ["sum", "max", "att"])
def test_pool_long_runs_match_oracle(mode, size):
    """The long-sequence batch (754k behaviors) and the same shapes at 6144
    samples (1.12M occurrences, past the large-grid switch): the hottest
    image's run of the stable order spans over a thousand 64-position
    chunks, so the backward's fix-up adds whole blocks of 512 chunks as block
    sums.  E is seeded random (the embedding model is not under test here)."""
    w = synth.get("c3_long") if size == "c3_long" else large_grid_workload()
    batch = synth.make_batch(w)
    dd = oracle.dedup(synth.occurrences(batch), w.n_images)
    runs = np.diff(dd["uniq_off"])
    assert runs.max() > 2 * 512 * 64                  # a run covering a whole block of chunks
    E32 = (np.random.default_rng(11).standard_normal((dd["n_uniq"], w.out_dim)) * 0.5).astype(np.float32)
    print(f"pool long runs {mode} {size}: n_u={dd['n_uniq']} longest run={runs.max()}", flush=True)
    pf = oracle.pool_fwd(mode, batch["seg_off"], dd["inv"], E32)
    pb = oracle.pool_bwd(mode, batch["seg_off"], dd["inv"], dd["n_uniq"], E32, pf, batch["g_u"], batch["g_a"])
    fwd, dE = gpu_pool(mode, batch, dd, E32, pf_orc=pf)
    assert_close(fwd["U"], pf["U"], 1e-4, "U")
    assert_close(dE, pb["dE"], 1e-4, "dE")


@pytest.mark.parametrize("wname", ["tiny", "c1_f32", "c3_long"])
def test_pool_bwd_sum_unit_gradient_is_exact_multiplicity(wname):
    w = synth.get(wname)
    batch = synth.make_batch(w)
    dd = oracle.dedup(synth.occurrences(batch), w.n_images)
    E32 = np.zeros((dd["n_uniq"], w.out_dim), np.float32)
    _, dE = gpu_pool("sum", batch, dd, E32, unit=True)
    n_beh = batch["seg_off"][-1]
    mult = np.bincount(dd["inv"][:n_beh], minlength=dd["n_uniq"]).astype(np.float64)
    np.testing.assert_array_equal(dE, np.repeat(mult[:, None], w.out_dim, axis=1))


# ------------------------------------------------------------ embed bwd

def run_embed_bwd(w, uniq_np, T_rows, Ws, bs, cap):
    """ams_embed_bwd on the saved activations of the oracle's forward over
    T_rows (the feature rows of uniq_np, zero rows for IDs outside the
    table) against the oracle's backward, at capacity cap."""
    n_u = len(uniq_np)
    fo = oracle.mlp_fwd(T_rows, np.arange(n_u), Ws, bs)
    rng = np.random.default_rng(5)
    dE32 = rng.standard_normal((n_u, w.out_dim)).astype(np.float32)
    bo = oracle.mlp_bwd(T_rows, np.arange(n_u), Ws, fo, dE32)
    T_dev = synth.table_rows(w, np.arange(w.n_images), device="cuda")
    mlp = ams.make_mlp(w.dims, w.dtype)
    h1dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    H1 = torch.zeros((cap, w.dims[1]), dtype=h1dt, device="cuda")
    H1[:n_u] = torch.from_numpy(np.maximum(fo["Z"][0], 0)).to(h1dt).cuda()
    H2 = None
    if w.n_layers == 3:
        H2 = torch.zeros((cap, w.dims[2]), device="cuda")
        H2[:n_u] = torch.from_numpy(np.maximum(fo["Z"][1], 0).astype(np.float32)).cuda()
    dE = torch.zeros((cap, w.out_dim), device="cuda")
    dE[:n_u] = torch.from_numpy(dE32).cuda()
    uniq = torch.zeros(cap, dtype=torch.int32, device="cuda")
    uniq[:n_u] = cuda_i32(uniq_np)
    nu = torch.tensor([n_u], dtype=torch.int32, device="cuda")
    dW = [torch.full((o, i), float("nan"), device="cuda") for i, o in zip(w.dims[:-1], w.dims[1:])]
    db = [torch.full((o,), float("nan"), device="cuda") for o in w.dims[1:]]
    ws = torch.empty(ams.ams_embed_workspace(mlp, cap), dtype=torch.uint8, device="cuda")
    ams.ams_embed_bwd(mlp, T_dev, uniq, nu, cap, [W.cuda() for W in Ws], H1, H2, None, dE, dW, db, ws)
    torch.cuda.synchronize()
    rt = RTOL[w.dtype]
    for l in range(w.n_layers):
        assert_close(dW[l], bo["dW"][l], rt, f"dW{l + 1}")
        assert_close(db[l], bo["db"][l], rt, f"db{l + 1}")


@pytest.mark.parametrize("wname", ["tiny", "mid_f32", "mid_bf16", "mid_bf16_l2"])
def test_embed_bwd_matches_oracle(wname):
    w = named(wname)
    batch, dd, Ws, bs, T_u = embed_case(w)
    print(f"embed bwd {wname}: n_u={dd['n_uniq']}", flush=True)
    run_embed_bwd(w, dd["uniq"], T_u, Ws, bs, dd["n_uniq"] + 40)


@pytest.mark.parametrize("case", ["mid", "few_rows", "bad_ids"])
def test_embed_bwd_bf16_wide_capacity_matches_oracle(case):
    """From a capacity of 2 x 256 x 256 unique slots the bf16 dW1 takes each
    chunk of the unique images in stages of 64 with the feature rows DMA'd
    two stages ahead; mid-size and tiny batches at that capacity give chunks
    of a few stages, a single ragged stage or none."""
    w = mid("bf16")
    batch, dd, Ws, bs, T_u = embed_case(w)
    uniq, T_rows = dd["uniq"].copy(), T_u
    if case == "few_rows":
        uniq, T_rows = uniq[:100], T_u[:100]
    if case == "bad_ids":                        # out-of-range IDs read as zero rows
        bad = [3, 700, len(uniq) - 1]
        uniq[bad] = [w.n_images + 5, -3, w.n_images]
        T_rows = T_rows.clone()
        T_rows[bad] = 0
    print(f"embed bwd wide {case}: n_u={len(uniq)} cap={ROW_SPLIT_CAP + 13}", flush=True)
    run_embed_bwd(w, uniq, T_rows, Ws, bs, ROW_SPLIT_CAP + 13)


# ---------------------------------------------------------- whole step

def step_case(w, mode, T_dev=None):
    batch = synth.make_batch(w)
    Ws, bs = synth.make_weights(w)
    if T_dev is None:
        T_dev = synth.table_full(w, device="cuda")
    st = run_gpu_step(w, batch, T_dev, Ws, bs, mode)
    g = gpu_outputs(st)
    T_u = synth.table_rows(w, g["uniq"], device="cuda").cpu()   # generator rows for the oracle
    o = oracle.step(batch, w.n_images, T_u, Ws, bs, mode, table_is_compact=True)
    return batch, Ws, T_u, g, o


def compare_step(w, mode, batch, Ws, T_u, g, o):
    rt = RTOL[w.dtype]
    od = o["dedup"]
    for k in ("uniq", "inv", "occ_perm", "uniq_off"):
        np.testing.assert_array_equal(g[k], od[k], err_msg=k)
    assert g["n_uniq"] == od["n_uniq"] and g["dev_status"] == 0
    fo, pf, pb, bo = o["fwd"], o["pool"], o["pool_bwd"], o["bwd"]
    assert_close(g["E"], fo["E"], rt, "E", rows=True)
    assert_close(g["U"], pf["U"], rt, "U", rows=True)
    assert_close(g["A"], pf["A"], rt, "A", rows=True)
    dE_delta = None
    if mode == "att":
        assert_close(g["w"], pf["w"], rt, "attention weights")
    if mode == "max":
        bad = max_flips(batch["seg_off"], od["inv"], fo["E"], g["argmax"], pf["argmax"], TAU)
        if len(bad):
            dE_delta = np.zeros_like(fo["E"])
            for i, d in bad:
                for j in (g["argmax"][i, d], pf["argmax"][i, d]):
                    dE_delta[od["inv"][j], d] += abs(batch["g_u"][i, d])
    extra_dE = np.abs(dE_delta) if dE_delta is not None else None
    # (a joint step with a query channel adds that channel's dE: o["dE"])
    assert_close(g["dE"], o.get("dE", pb["dE"]), rt, "dE", extra=extra_dE, rows=True)
    flips1 = relu_flips(fo["Z"][0], g["H1"], TAU)
    flips2 = relu_flips(fo["Z"][1], g["H2"], TAU) if w.n_layers == 3 else []
    eW, eb = grad_flip_bounds(w.dims, Ws, T_u, fo, bo, flips1, flips2, dE_delta)
    print(f"  decisions: relu1 {len(flips1)} relu2 {len(flips2)} "
          f"argmax {0 if dE_delta is None else int((dE_delta > 0).sum())}", flush=True)
    for l in range(w.n_layers):
        assert_close(g["dW"][l], bo["dW"][l], rt, f"dW{l + 1}", extra=eW[l])
        assert_close(g["db"][l], bo["db"][l], rt, f"db{l + 1}", extra=eb[l])


@pytest.mark.parametrize("wname,mode", [
    ("tiny", "sum"), ("tiny", "att"), ("mid_f32", "att"), ("mid_f32", "max"),
    ("mid_bf16", "sum"), ("mid_bf16", "max"), ("mid_bf16", "att"),
])
def test_step_end_to_end(wname, mode):
    w = synth.get("tiny") if wname == "tiny" else mid(wname[4:])
    print(f"step {wname} {mode}", flush=True)
    batch, Ws, T_u, g, o = step_case(w, mode)
    compare_step(w, mode, batch, Ws, T_u, g, o)


def test_step_full_size_fp32_attentive():
    """The benchmarked workload (1024 samples, 200k x 4096 fp32, attentive
    pooling) end to end at full size, grids sized by n_occ as in the bench."""
    w = synth.get("c1_f32")
    print("step c1_f32 att full size", flush=True)
    batch, Ws, T_u, g, o = step_case(w, "att")
    compare_step(w, "att", batch, Ws, T_u, g, o)


@pytest.mark.parametrize("mode", ["att", "max"])
def test_step_full_size_bf16(mode):
    """The bf16 workload (1024 samples, 200k x 4096 bf16 table and weights) end
    to end at full size, grids sized by n_occ as in the bench."""
    w = synth.get("c2_bf16")
    print(f"step c2_bf16 {mode} full size", flush=True)
    batch, Ws, T_u, g, o = step_case(w, mode)
    compare_step(w, mode, batch, Ws, T_u, g, o)


def test_step_full_size_long_sequences():
    """The long-sequence workload (4096 samples of up to 500 behaviors, 2M x
    4096 bf16 table, ~160k unique images, an image repeated ~69k times) end to
    end at full size against the whole float64 oracle step."""
    w = synth.get("c3_long")
    print("step c3_long att full size", flush=True)
    batch, Ws, T_u, g, o = step_case(w, "att")
    compare_step(w, "att", batch, Ws, T_u, g, o)


def test_step_is_bitwise_deterministic():
    w = mid("f32", B=64)
    batch = synth.make_batch(w)
    Ws, bs = synth.make_weights(w)
    T_dev = synth.table_full(w, device="cuda")
    outs = []
    for _ in range(2):
        outs.append(gpu_outputs(run_gpu_step(w, batch, T_dev, Ws, bs, "att")))
    for k in ("E", "U", "dE", "w"):
        np.testing.assert_array_equal(outs[0][k], outs[1][k], err_msg=k)
    for l in range(w.n_layers):
        np.testing.assert_array_equal(outs[0]["dW"][l], outs[1]["dW"][l])
        np.testing.assert_array_equal(outs[0]["db"][l], outs[1]["db"][l])


@pytest.mark.parametrize("mode,cap", [("att", None), ("sum", None), ("att", ROW_SPLIT_CAP)])
def test_bf16_step_is_bitwise_deterministic(mode, cap):
    """The 1024-sample bf16 step twice, on fresh buffers: the stream-K first
    layer (partial tiles added in K order), the split high/low tails and, with
    a capacity past ROW_SPLIT_CAP, the row-split first layer."""
    w = synth.get("c2_bf16")
    batch = synth.make_batch(w)
    Ws, bs = synth.make_weights(w)
    T_dev = synth.table_full(w, device="cuda")
    print(f"bf16 determinism {mode} cap={cap}", flush=True)
    outs = [gpu_outputs(run_gpu_step(w, batch, T_dev, Ws, bs, mode, cap=cap)) for _ in range(2)]
    for k in ("E", "H1", "H2", "U", "A", "dE"):
        np.testing.assert_array_equal(outs[0][k], outs[1][k], err_msg=k)
    for l in range(w.n_layers):
        np.testing.assert_array_equal(outs[0]["dW"][l], outs[1]["dW"][l])
        np.testing.assert_array_equal(outs[0]["db"][l], outs[1]["db"][l])


def test_table_generator_is_device_independent():
    w = synth.get("c2_bf16")
    rows = np.array([0, 1, 77, 199_999, 123_456])
    assert torch.equal(synth.table_rows(w, rows, device="cuda").cpu(), synth.table_rows(w, rows))
