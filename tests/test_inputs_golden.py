"""The seeded generator and the oracle reproduce the stored tiny-workload fixture."""
import hashlib
import json
import os

import numpy as np

import oracle
from paper_2606_20005_amd import inputs

GOLD = os.path.join(os.path.dirname(__file__), "golden", "tiny_oracle.json")


def test_generator_hashes_stable():
    ref = json.load(open(GOLD))
    d = inputs.make("tiny")
    for k, h in ref["sha256"].items():
        assert hashlib.sha256(np.ascontiguousarray(d[k]).tobytes()).hexdigest() == h, k


def test_oracle_reproduces_fixture():
    ref = json.load(open(GOLD))
    d = inputs.make("tiny")
    w = d["w"]
    for causal in (False, True):
        r = ref["causal" if causal else "noncausal"]
        kl, l1, l2, dQ1, dK1, dQ2, dK2 = oracle.backward(d["Q1"], d["K1"], d["Q2"], d["K2"], w.s1, w.s2,
                                                         causal, 0, d["g"])
        np.testing.assert_allclose(kl[0, 0, :16], r["kl_rows_0_16"], rtol=1e-12)
        np.testing.assert_allclose(l1[0, 0, :16], r["lse1_rows_0_16"], rtol=1e-13)
        np.testing.assert_allclose(l2[0, 0, :16], r["lse2_rows_0_16"], rtol=1e-13)
        np.testing.assert_allclose(np.linalg.norm(dQ2), r["dQ2_norm"], rtol=1e-12)
        np.testing.assert_allclose(np.linalg.norm(dK1), r["dK1_norm"], rtol=1e-12)


def test_bf16_rounding_is_round_to_nearest_even():
    x = np.array([1.0, 1.00390625, 1.01171875, -2.5, 3.0e-3, 1.0 + 2**-8, 1.0 + 3 * 2**-8], dtype=np.float32)
    r = inputs.round_bf16(x)
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to even gives 1; 1 + 3*2^-8 rounds up to 1 + 2^-6
    assert r[5] == 1.0 and r[6] == np.float32(1.0 + 2**-6)
    assert np.all(inputs.bf16_bits(r).astype(np.uint32) << 16 == r.view(np.uint32))
    import torch
    t = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(r, t)


def test_workload_structures():
    d = inputs.make("mid", B=1, H=1, n_q=64, n_k=64)
    assert np.array_equal(d["K2"], d["K1"])
    diff = d["Q2"] - d["Q1"]
    assert 0.2 < diff.std() < 0.4
    d = inputs.make("long", H=1, n_q=32, n_k=32)
    for X in (d["Q1"], d["K1"], d["Q2"], d["K2"]):
        big = np.abs(X[..., list(inputs.OUTLIER_CHANNELS)]).mean()
        assert big > 4 * np.abs(X[..., :4]).mean()
