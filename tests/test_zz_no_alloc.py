"""ams_dedup_noalloc, the dedup entry point for callers that cannot allocate
device memory, against ams_dedup (the workspace entry point it shares its
kernels with): bit-identical outputs on calls in a row on the one scratch
array, a large batch first and a smaller one after it, so that anything the
first call left in the scratch would show in the second."""
import numpy as np
import pytest
import torch

from paper_1711_06505_amd import ams, synth

pytestmark = pytest.mark.gpu


def run(ids_np, n_ids, noalloc):
    n = ids_np.size
    ids = torch.from_numpy(np.ascontiguousarray(ids_np, dtype=np.int32)).cuda()
    m = max(n, 1)
    out = {k: torch.full((m,), -7, dtype=torch.int32, device="cuda") for k in ("uniq", "inv", "perm")}
    off = torch.full((n + 1,), -7, dtype=torch.int32, device="cuda")
    nu = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    stt = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    if noalloc:
        ams.ams_dedup_noalloc(ids, n_ids, out["uniq"], out["inv"], out["perm"], off, nu, stt)
    else:
        ws = torch.empty(max(ams.ams_dedup_workspace(n, n_ids), 256), dtype=torch.uint8, device="cuda")
        ams.ams_dedup(ids, n_ids, out["uniq"], out["inv"], out["perm"], off, nu, stt, ws)
    torch.cuda.synchronize()
    k = int(nu.item())
    return {"status": int(stt.item()), "n_uniq": k, "uniq": out["uniq"][:k].cpu().numpy(),
            "inv": out["inv"][:n].cpu().numpy(), "perm": out["perm"][:n].cpu().numpy(),
            "off": off[:k + 1].cpu().numpy()}


def same(a, b):
    assert a["status"] == b["status"] == 0
    assert a["n_uniq"] == b["n_uniq"]
    for k in ("uniq", "inv", "perm", "off"):
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)


def long_batch_ids():
    """The 4096-sample long-behavior batch (lengths up to 500, 2M images)."""
    w = synth.get("c3_long")
    return synth.occurrences(synth.make_batch(w)), w.n_images


def test_noalloc_matches_workspace_dedup_on_calls_in_a_row():
    big, n_big = long_batch_ids()
    assert big.size <= ams.DEDUP_NOALLOC_MAX_OCC
    w = synth.get("tiny")
    small, n_small = synth.occurrences(synth.make_batch(w)), w.n_images
    print(f"no-alloc dedup: {big.size} then {small.size} occurrences", flush=True)
    first = run(big, n_big, noalloc=True)
    second = run(small, n_small, noalloc=True)
    same(first, run(big, n_big, noalloc=False))
    same(second, run(small, n_small, noalloc=False))


def test_noalloc_at_the_capacity_and_empty():
    rng = np.random.default_rng(11)
    n = ams.DEDUP_NOALLOC_MAX_OCC
    ids = rng.integers(0, 2**31 - 1, n, dtype=np.int64).astype(np.int32)   # four radix passes
    ids[::7] = 12345                                                       # one hot ID
    print(f"no-alloc dedup at the capacity: {n} occurrences, 31-bit IDs", flush=True)
    same(run(ids, 2**31 - 1, noalloc=True), run(ids, 2**31 - 1, noalloc=False))
    e = run(np.zeros(0, np.int32), 10, noalloc=True)
    assert e["status"] == 0 and e["n_uniq"] == 0 and e["off"][0] == 0


def test_noalloc_rejects_a_batch_beyond_the_capacity():
    n = ams.DEDUP_NOALLOC_MAX_OCC + 1
    ids = torch.zeros(n, dtype=torch.int32, device="cuda")
    buf = torch.empty(n + 1, dtype=torch.int32, device="cuda")
    one = torch.empty(1, dtype=torch.int32, device="cuda")
    with pytest.raises(ams.AmsError) as e:
        ams.ams_dedup_noalloc(ids, 10, buf, buf, buf, buf, one, one)
    assert e.value.status == 9


def test_noalloc_reports_an_out_of_range_id():
    ids = (np.arange(5000) % 50).astype(np.int32)
    ids[4321] = 77
    r = run(ids, 50, noalloc=True)
    assert r["status"] == 7
    # and the next call on the same scratch is clean again
    same(run(ids % 50, 50, noalloc=True), run(ids % 50, 50, noalloc=False))
