"""The seeded input generator: reproducibility, distributions, bf16 rounding."""
import json
import os

import numpy as np
import torch

import synth


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 100000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, 1e-40, np.inf, -np.inf],
                                 dtype=np.float32)]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = synth.round_to_bf16(x)
    np.testing.assert_array_equal(got, ref)


def test_haar_columns_orthonormal_and_seeded():
    Q = synth.haar_columns(synth.host_rng(0, 3, "U"), 200, 30)
    np.testing.assert_allclose(Q.T @ Q, np.eye(30), atol=1e-12)
    Q2 = synth.haar_columns(synth.host_rng(0, 3, "U"), 200, 30)
    np.testing.assert_array_equal(Q, Q2)
    Q3 = synth.haar_columns(synth.host_rng(0, 4, "U"), 200, 30)
    assert not np.allclose(Q, Q3)


def test_host_matrix_dtypes_and_spectrum():
    W, M, G = synth.host_matrix(0, 2, 64, 96, 64, param_dtype="bf16", grad_dtype="bf16", steps=(0, 1))
    np.testing.assert_array_equal(W, synth.round_to_bf16(W))
    np.testing.assert_array_equal(G[0], synth.round_to_bf16(G[0]))
    np.testing.assert_array_equal(M, M.astype(np.float32).astype(np.float64))
    assert not np.array_equal(G[0], G[1])
    assert abs(W.std() - 0.02) < 0.002
    # signal singular values 1/i sit on top of 0.01-scale noise
    s = np.linalg.svd(G[0], compute_uv=False)
    assert 0.95 < s[0] < 1.2


def test_workload_element_counts():
    counts = [sum(m * n for m, n in wl.shapes) for wl in synth.WORKLOADS]
    assert counts[0] == 917504
    assert abs(counts[1] / 1e9 - 1.812) < 1e-3
    assert abs(counts[2] / 1e9 - 5.436) < 1e-3
    assert abs(counts[3] / 1e9 - 12.080) < 1e-3
    assert abs(counts[4] / 1e9 - 22.649) < 1e-3
    assert len(synth.WORKLOADS[2].shapes) == 160


def test_aux_group_matches_paper_share_and_is_seeded():
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))
    share = gold["muon_routed_fraction"]["value"]
    for w, scale in ((1, "1.3B"), (2, "4B"), (3, "9B"), (4, "15B")):
        wl = synth.WORKLOADS[w]
        aux = synth.aux_numels(w)
        me = sum(m * n for m, n in wl.shapes)
        assert abs(me / (me + sum(aux)) - share[scale]) < 1e-6
        assert min(aux) >= 1 and len(aux) == 4 + len(wl.shapes) + 4 * wl.blocks
    a = synth.host_aux(2, 5, 999, param_dtype="bf16", grad_dtype="bf16", steps=(0, 1))
    b = synth.host_aux(2, 5, 999, param_dtype="bf16", grad_dtype="bf16", steps=(0, 1))
    for k in a:
        assert np.array_equal(a[k], b[k])
    assert not np.array_equal(a["g0"], a["g1"])
    assert np.array_equal(a["p"], synth.round_to_bf16(a["p"]))
    assert np.all(a["v"] > 0)
