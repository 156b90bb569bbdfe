"""The seeded input generator: reproducibility, distributions, ranges, and
the workload shapes the paper fixes (tests/golden/paper_shapes.json)."""
import json
import os

import numpy as np
import torch

from paper_1711_06505_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_shapes.json")


def test_same_seed_same_bytes():
    for name in ["tiny", "c1_f32"]:
        a = synth.make_batch(name, k=2)
        b = synth.make_batch(name, k=2)
        for key in a:
            np.testing.assert_array_equal(a[key], b[key])
        c = synth.make_batch(name, k=3)
        assert not np.array_equal(a["beh_ids"][:50], c["beh_ids"][:50])


def test_lengths_and_id_ranges():
    t = synth.make_batch("tiny")
    assert np.all(np.diff(t["seg_off"]) == 8) and t["seg_off"][-1] == 512
    c1 = synth.make_batch("c1_f32")
    L = np.diff(c1["seg_off"])
    assert L.min() >= 10 and L.max() <= 100 and abs(L.mean() - 55) < 3
    c3 = synth.make_batch("c3_long")
    L3 = np.diff(c3["seg_off"])
    assert L3.min() >= 1 and L3.max() == 500
    # geometric(1/200) capped at 500 has mean 200 * (1 - (199/200)^500) = 183.6
    assert abs(L3.mean() - 183.6) < 5
    for b, w in [(t, "tiny"), (c1, "c1_f32"), (c3, "c3_long")]:
        occ = synth.occurrences(b)
        assert occ.min() >= 0 and occ.max() < synth.get(w).n_images


def test_zipf_skew_and_dedup_ratio():
    c1 = synth.make_batch("c1_f32")
    occ = synth.occurrences(c1)
    _, cnt = np.unique(occ, return_counts=True)
    ratio = occ.size / cnt.size
    assert 4.0 < ratio < 4.9                # about 4.4 for Zipf(1.1) over 200k
    # the hottest image carries about 1/H_{N,s} of the mass (~13%)
    N, s = 200_000, 1.1
    h = np.sum(np.arange(1, N + 1, dtype=np.float64) ** -s)
    assert abs(cnt.max() / occ.size - 1 / h) < 0.01


def test_table_rows_device_independent_and_chunking():
    w = synth.get("c1_f32")
    rows = np.array([0, 5, 199_999, 12345, 5])
    a = synth.table_rows(w, rows)
    b = synth.table_rows(w, rows, chunk_rows=2)
    assert torch.equal(a, b)
    assert torch.equal(a[1], a[4])
    assert a.dtype == torch.float32 and a.shape == (5, 4096)
    assert float(a.min()) >= 0.0                            # ReLU'd features
    # roughly half zeros, positive part of a unit-variance bell
    assert 0.45 < float((a == 0).float().mean()) < 0.55
    t = synth.table_rows("tiny", np.arange(512))
    assert abs(float(t.mean())) < 0.01 and abs(float(t.std()) - 1.0) < 0.01
    b16 = synth.table_rows("c2_bf16", rows)
    assert b16.dtype == torch.bfloat16
    assert torch.equal(b16, a.to(torch.bfloat16))            # same values, RNE-rounded


def test_weights_glorot_and_bf16_rounding():
    Ws, bs = synth.make_weights("c1_f32")
    assert [tuple(W.shape) for W in Ws] == [(256, 4096), (64, 256), (12, 64)]
    for W in Ws:
        lim = np.sqrt(6.0 / (W.shape[0] + W.shape[1]))
        assert float(W.abs().max()) <= lim
    Wb, _ = synth.make_weights("c2_bf16")
    assert Wb[0].dtype == torch.bfloat16
    assert float(Wb[0].abs().max()) <= np.sqrt(6.0 / 4352) * (1 + 2 ** -8)


def test_workload_shapes_follow_the_paper():
    g = json.load(open(GOLDEN))
    for name in ["c1_f32", "c2_bf16", "c3_long"]:
        w = synth.get(name)
        assert list(w.dims) == g["mlp_widths"]["value"]
        assert w.in_dim == g["feature_dim"]["value"]
        assert w.out_dim == g["embedding_dim"]["value"]
    # 4096-D float -> 12-D float: "over 340 times"
    assert g["feature_dim"]["value"] / g["embedding_dim"]["value"] > g["compression_over"]["value"]
    # per-image byte model: embeddings pulled and their gradients pushed, 12 x fp32
    # each way, for 320k images is the "Image 30M" of Table 2 (within rounding)
    per_image = 2 * g["embedding_dim"]["value"] * 4
    assert abs(per_image * g["images_per_minibatch"]["value"] / g["ams_image_comm_bytes"]["value"] - 1) < 0.05
    # shipping the 4096-D fp32 rows instead is the 5.0G of store-in-server
    raw = g["feature_dim"]["value"] * 4 * g["images_per_minibatch"]["value"]
    assert abs(raw / g["store_in_server_image_comm_bytes"]["value"] - 1) < 0.05
    # 0.12 B images x 4096 fp32 is the 2T server storage total
    assert abs(g["unique_images_total"]["value"] * raw / g["images_per_minibatch"]["value"]
               / g["server_storage_total_bytes"]["value"] - 1) < 0.02
