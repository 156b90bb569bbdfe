"""How sensitive the joint step's float64 chain is to float32-sized changes of
the image embeddings E, measured on the oracle alone (no GPU).

The GPU computes E in float32, so every result downstream of E can differ
from the oracle's by E's rounding carried through the chain.  Here E of the
96-sample joint batch (geometric lengths up to 500, the CTR model and its
upstream gradients) is perturbed by +-2^-23 relative, the size of one float32
rounding, and the chain re-evaluated: pooling, the CTR model, the pooling
backward.  The amplification (largest change relative to the tensor's scale,
divided by 2^-23) stays small for the pooled vectors and every input gradient
of the CTR model (U, A, the bags), and for dE: at this size the attentive
pooling and its backward are well-conditioned, so float32-level noise in E
stays at float32 level downstream.  The full-size GPU check of the joint
step measures the same sensitivity on its own batch (tests/parity.py,
assert_close_sensitive) rather than assuming it.
"""
import dataclasses

import numpy as np
import pytest

from oracle import oracle
from paper_1711_06505_amd import synth

REL = 2.0 ** -23


@pytest.fixture(scope="module")
def chain():
    base = synth.get("c4_joint")
    w = dataclasses.replace(base, name="mid_joint", index=21, batch=96, n_images=20_000, stream=-1,
                            joint=dataclasses.replace(base.joint, id_rows=(200_000, 20_000, 500)))
    batch = synth.make_batch(w)
    jb = synth.make_joint(w, batch)
    dd = oracle.dedup(synth.occurrences(batch), w.n_images)
    T_u = synth.table_rows(w, dd["uniq"])
    Ws, bs = synth.make_weights(w)
    E = oracle.mlp_fwd(T_u, np.arange(dd["n_uniq"]), Ws, bs)["E"]
    cW, cb = synth.make_ctr_weights(w)
    seg, inv = batch["seg_off"], dd["inv"]
    bags = []
    for t in range(len(w.joint.id_rows)):
        idd = oracle.dedup(synth.joint_occurrences(jb, t), w.joint.id_rows[t])
        bags.append(oracle.bag_fwd(seg, idd["inv"], synth.id_table_rows(w, t, idd["uniq"])))
    D = w.out_dim

    def run(Ein):
        pf = oracle.pool_fwd("att", seg, inv, Ein)
        X = np.concatenate([pf["U"], pf["A"]] + bags, axis=1)
        c = oracle.ctr_fwd_bwd(X, jb["labels"], cW, cb)
        dU, dA = c["dX"][:, :D], c["dX"][:, D:2 * D]
        pb = oracle.pool_bwd("att", seg, inv, dd["n_uniq"], Ein, pf, dU, dA)
        return {"U": pf["U"], "dU": dU, "dA": dA, "dbags": c["dX"][:, 2 * D:], "dE": pb["dE"], "Z": c["Z"]}

    return E, run, int(seg[-1])


def amplification(x, y):
    """Largest change relative to max(|x|, rms(x), rms of its row), per REL."""
    rms = np.sqrt(np.mean(x * x))
    scale = np.maximum(np.maximum(np.abs(x), rms), np.sqrt(np.mean(x * x, axis=1, keepdims=True)))
    return float(np.max(np.abs(y - x) / scale)) / REL


def test_joint_chain_is_well_conditioned_in_E(chain):
    E, run, n_beh = chain
    assert n_beh > 10_000                                   # segments up to 500 long
    ref = run(E)
    rng = np.random.default_rng(0)
    worst = {k: 0.0 for k in ("U", "dU", "dA", "dbags", "dE")}
    for _ in range(3):
        out = run(E * (1 + REL * rng.choice([-1.0, 1.0], size=E.shape)))
        for k in worst:
            worst[k] = max(worst[k], amplification(ref[k], out[k]))
    print("amplification of a 2^-23 relative change of E:", {k: round(v, 2) for k, v in worst.items()})
    # float32-level noise in E stays float32-level downstream (measured
    # amplifications are below 10); the float32 tolerance is 1e-4 = 839 x 2^-23
    for k, v in worst.items():
        assert v < 50, (k, v)


def test_ctr_hidden_units_keep_their_side_of_the_tie(chain):
    """No hidden unit of the CTR model changes sign under the perturbation at
    this size: where one would, its sample's input gradients jump by the
    unit's whole contribution, which the sensitivity-bounded GPU check then
    carries in its tolerance."""
    E, run, _ = chain
    ref = run(E)
    rng = np.random.default_rng(1)
    out = run(E * (1 + REL * rng.choice([-1.0, 1.0], size=E.shape)))
    for z0, z1 in zip(ref["Z"][:-1], out["Z"][:-1]):
        assert np.array_equal(z0 > 0, z1 > 0)
