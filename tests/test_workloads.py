"""Host-side checks of the seeded workload generators (no method arithmetic here)."""
import math

import numpy as np
import torch

import oracle
from workloads import gen


def test_tiny_config_shapes_and_determinism():
    spec = gen.config("tiny")
    a = gen.make(spec, 1)
    b = gen.make(spec, 1)
    assert a.queries.shape == (4, 256) and a.queries.dtype == torch.float32
    assert a.keys.shape == (16384, 256)
    assert a.values.dtype == torch.int32 and int(a.values.min()) >= 0 and int(a.values.max()) < 32000
    assert a.p_lm.shape == (4, 32000)
    np.testing.assert_allclose(a.p_lm.double().sum(1).numpy(), 1.0, atol=1e-5)
    assert torch.equal(a.keys, b.keys) and torch.equal(a.queries, b.queries)
    assert torch.equal(a.values, b.values) and torch.equal(a.p_lm, b.p_lm)
    assert a.key_offsets_host.tolist() == [0, 16384] and a.query_offsets_host.tolist() == [0, 4]


def test_bf16_keys_are_rounded_draws_with_the_stated_scale():
    spec = gen.scaled(gen.config("decode_7b"), n_keys=2048)
    w = gen.make(spec, 2)
    assert w.keys.dtype == torch.bfloat16
    std = w.keys.float().std().item()
    assert abs(std - 8.0 / 64.0) < 0.01
    # squared norm of a key is about 64 by construction
    assert abs(w.keys.float().pow(2).sum(1).mean().item() - 64.0) < 1.0


def test_zipf_values_follow_the_bounded_law():
    spec = gen.scaled(gen.config("decode_7b"), n_keys=200000, d=8)
    w = gen.make(spec, 3)
    v = w.values.numpy()
    cdf = gen.zipf_cdf(32000, 1.1)
    p0 = cdf[0]
    assert abs((v == 0).mean() - p0) < 0.01
    assert v.min() >= 0 and v.max() < 32000


def test_ragged_offsets():
    spec = gen.scaled(gen.config("ragged_batch"), d=8, n_keys=("uniform", 100, 400), B=10, S=10)
    w = gen.make(spec, 3)
    sizes = w.keys_per_set()
    assert len(sizes) == 10 and sizes.min() >= 100 and sizes.max() <= 400
    assert w.keys.shape[0] == int(w.key_offsets_host[-1])
    assert w.query_offsets_host.tolist() == list(range(11))


def test_planted_queries_sit_next_to_their_key():
    spec = gen.scaled(gen.config("decode_7b"), n_keys=3000, d=64, B=3, S=1, query_mode="planted")
    w = gen.make(spec, 9)
    q, dt = oracle.host_elements(w.queries)
    k, _ = oracle.host_elements(w.keys)
    d = oracle.sqdist(q, k, dt)
    assert d.argmin(1).tolist() == w.planted_ids.tolist()


def test_projected_queries_have_the_key_scale():
    spec = gen.scaled(gen.config("specverify_static"), n_keys=1024, B=16, d=128, proj_in=512)
    w = gen.make(spec, 6)
    assert w.queries.dtype == torch.float16 and w.queries.shape == (16, 128)
    # entries ~ N(0, (8/sqrt(512))^2 * 512 / 128)
    expect = 8.0 / math.sqrt(512) * math.sqrt(512.0 / 128.0)
    assert abs(w.queries.float().std().item() - expect) / expect < 0.15
