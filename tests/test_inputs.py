"""The seeded input generators: determinism, distributions, and the bf16 rounding
they use to store inputs (pinned against torch's own CPU conversion)."""
import numpy as np
import pytest
import torch

from oracle import ssn_oracle as O
from paper_2607_13332_amd import inputs as I


def test_bf16_rounding_matches_torch():
    r = np.random.default_rng(0)
    x = np.concatenate([r.standard_normal(100000).astype(np.float32) * 10.0 ** r.integers(-30, 30, 100000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, 1e-40], np.float32)])
    x = x.astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(I.to_bf16_bits(x), ref)


def test_generators_are_deterministic_and_independent():
    cfg = I.with_tokens(I.MID, 256)
    a = I.codec_inputs_host(cfg)
    b = I.codec_inputs_host(cfg)
    for key in a:
        assert np.array_equal(a[key], b[key]), key
    c = I.codec_inputs_host(I.with_tokens(I.MID, 256, seed=77))
    assert not np.array_equal(a["ids"], c["ids"])
    # changing the noise level changes nothing else
    import dataclasses
    d = I.codec_inputs_host(dataclasses.replace(cfg, noise_std=0.5))
    assert np.array_equal(a["U"], d["U"]) and np.array_equal(a["ids"], d["ids"])


@pytest.mark.parametrize("d,k", [(256, 8), (2048, 32), (4096, 64)])
def test_gaussian_basis_orthonormal(d, k):
    u = I.gaussian_orthonormal_basis(d, k, 1)
    assert np.abs(u.T @ u - np.eye(k)).max() < 1e-12
    ub = O.f64(I.store(u, "bf16"))
    eps = np.linalg.norm(ub.T @ ub - np.eye(k))
    assert 1e-4 < eps < 1e-2        # bf16 storage is only approximately orthonormal


def test_ids_ranges_and_zipf_shape():
    V = 131072
    u = I.token_ids(200000, V, 1)
    assert u.dtype == np.int32 and u.min() >= 0 and u.max() < V
    z = I.token_ids(400000, V, 2, "zipf", 1.1)
    assert z.min() >= 0 and z.max() < V
    counts = np.bincount(z, minlength=V)
    top = np.sort(counts)[::-1]
    # p(r) ~ r^-1.1: rank-1 / rank-10 frequency ratio ~ 10^1.1
    assert 8.0 < top[0] / top[9] < 17.0
    cdf = I.zipf_cdf(V, 1.1)
    assert abs(top[0] / len(z) - cdf[0]) < 0.01
    # unique fraction at N=4096 near the analytic expectation
    z4 = I.token_ids(4096, V, 3, "zipf", 1.1)
    p = np.diff(np.concatenate([[0.0], cdf]))
    expect = np.sum(1 - (1 - p) ** 4096) / 4096
    assert abs(len(np.unique(z4)) / 4096 - expect) < 0.03


def test_hadamard_and_selection_bases():
    h = I.hadamard_basis(256, 8, 0)
    assert np.array_equal(h.T @ h, np.eye(8))
    assert set(np.unique(np.abs(h))) == {1 / 16}
    s = I.selection_basis(100, 7, 0)
    assert np.array_equal(s.T @ s, np.eye(7)) and s.sum() == 7


def test_config_table():
    assert I.TINY.N == 512 and I.MID.N == 8192 and I.STAGE8B.N == 32768
    sw = I.sweep_configs()
    assert len(sw) == 12 and {c.k for c in sw} == {32, 64, 128}
    assert {c.N for c in sw} == {4096, 16384, 65536, 131072}


def test_paper_configs_follow_the_model_cards():
    """The paper-shaped workloads are the shapes the paper prints (fixtures
    in tests/golden cite the passages)."""
    import json
    import math
    import os
    fig = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_figures.json")))
    m8, r8, m1 = fig["model_8b"], fig["rank_8b"], fig["model_1b"]
    p8 = [c for c in I.paper_configs() if c.name.startswith("paper8b")]
    p1 = [c for c in I.paper_configs() if c.name.startswith("paper1b")]
    assert {c.B for c in p8} == {1, 2, 3} and {c.B for c in p1} == {1, 2, 3}
    for c in p8:
        assert (c.d, c.k, c.V, c.S) == (m8["d"], r8["rank"], m8["vocab"], m8["seq_len"])
    for c in p1:
        assert (c.d, c.k, c.V, c.S) == (m1["d"], m1["rank"], m1["vocab"], m1["seq_len"])
    # Llama-style FFN width: 8/3 d times the multiplier, rounded up to 1024
    ffn8 = math.ceil(m8["d"] * 8 / 3 * m8["ffn_multiplier"] / m8["ffn_round"]) * m8["ffn_round"]
    ffn1 = math.ceil(m1["d"] * 8 / 3 * m8["ffn_multiplier"] / m8["ffn_round"]) * m8["ffn_round"]
    assert ffn1 == m1["ffn_inner"]              # the rule reproduces the printed 1B width
    w8, w1 = I.WEIGHTS_PAPER8B, I.WEIGHTS_PAPER1B
    assert (w8.d, w8.k, w8.layers) == (m8["d"], r8["rank"], m8["body_layers"])
    assert tuple(w8.shapes) == ((m8["d"], m8["d"]), (m8["d"], ffn8))
    assert (w1.d, w1.k, w1.layers) == (m1["d"], m1["rank"], m1["body_layers"])
    assert tuple(w1.shapes) == ((m1["d"], m1["d"]), (m1["d"], m1["ffn_inner"]))

