"""The fused select of query batches on long rows (the 128-query matrix-core
distance kernel): each query's threshold comes from a sample of its keys
(the first 512 rows of every eighth 4096-row tile), the distance kernel lists
the keys below it instead of writing the distance matrix, and when a query's
list holds fewer than r or more than its capacity the distance matrix is
written and selected by the wide select instead.

Small integer entries make every distance exact in fp32 (products and sums of
integers below 2^24, accumulated exactly by the matrix cores), so ids and
distances must equal the oracle's bit for bit on the listed path and on both
fallbacks (the sample's keys all far: far too many keys below the threshold;
the sample's keys nearest: fewer than r).
"""
import numpy as np
import pytest
import torch

import oracle
from workloads import gen  # noqa: F401  (keeps the import order of the other GPU modules)

pytestmark = pytest.mark.gpu

knn = pytest.importorskip("paper_2405_19325_amd")

N, D, B, R = 600000, 128, 80, 64
TILE, PIECE, EVERY = 4096, 512, 8  # the distance tiles of d = 128 and the sample's geometry


def _say(msg):
    print(f"[gpu] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    knn.load()
    yield
    torch.cuda.synchronize()


def _sample_rows(n):
    starts = np.arange(0, n, TILE * EVERY)
    return np.concatenate([np.arange(s, min(s + PIECE, n)) for s in starts])


def _store(case, seed):
    rng = np.random.default_rng(seed)
    k = np.zeros((N, D), np.float32)
    k[:, :8] = rng.integers(-30, 31, (N, 8))
    q = np.zeros((B, D), np.float32)
    q[:, :8] = rng.integers(-30, 31, (B, 8))
    sample = _sample_rows(N)
    if case == "sample-far":  # every sampled key far away: the threshold keeps nearly every key
        k[sample, :8] = 120
    elif case == "sample-near":  # the sampled keys are each query's nearest, but too few pass
        k[:, 8] = 100
        k[sample, 8] = 0
    return rng, q, k, sample


@pytest.mark.parametrize("layout", ["row-major", "packed"])
@pytest.mark.parametrize("case", ["listed", "sample-far", "sample-near"])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
def test_fused_select_exact_integers(case, dtype, layout):
    _say(f"fused select: {case}, {dtype}, {layout} keys")
    rng, q, k, _ = _store(case, 120 + len(case))
    vals = rng.integers(0, 1000, N).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(1000), B).astype(np.float32)
    ko, qo = np.array([0, N]), np.array([0, B])
    dev = "cuda"
    tq = torch.as_tensor(q, device=dev).to(dtype).contiguous()
    tk = torch.as_tensor(k, device=dev).to(dtype).contiguous()
    tv, tp = torch.as_tensor(vals, device=dev), torch.as_tensor(p_lm, device=dev)
    tko, tqo = torch.as_tensor(ko, device=dev), torch.as_tensor(qo, device=dev)
    packed = knn.pack_keys(tk) if layout == "packed" else None
    prob = knn.MixtureProblem(tq, tk, tv, tko, tqo, tp, R, 0.01, 0.3, key_offsets_host=ko, query_offsets_host=qo,
                              packed_keys=packed)
    p_m, ids, dists = prob.run()
    torch.cuda.synchronize()
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, R)
    np.testing.assert_array_equal(ids.cpu().numpy(), o_ids)
    np.testing.assert_array_equal(dists.cpu().numpy().astype(np.float64), o_d)
    ref = oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.01, 0.3)
    np.testing.assert_allclose(p_m.cpu().numpy(), ref, rtol=0, atol=1e-5)
    # the same call with precomputed key norms, and the stages one at a time
    norms = knn.key_sqnorms(tk)
    prob2 = knn.MixtureProblem(tq, tk, tv, tko, tqo, tp, R, 0.01, 0.3, key_sqnorms=norms, key_offsets_host=ko,
                               query_offsets_host=qo, packed_keys=packed)
    prob2.run_part("distances")
    prob2.run_part("select")
    torch.cuda.synchronize()
    assert torch.equal(prob2.ids, ids) and torch.equal(prob2.dists, dists)
    del tk, prob, prob2, packed


@pytest.mark.parametrize("layout", ["row-major", "packed"])
def test_fused_nest_step_with_masked_keys(layout):
    """A NEST step (lambda_t, masked keys, decoding outputs) through the fused select: a third of the keys
    masked, among them the exact nearest keys of the first queries."""
    _say("fused select: NEST step with masked keys")
    from oracle import nest

    rng, q, k, _ = _store("listed", 131)
    masked = rng.choice(N, N // 3, replace=False)
    o_ids0, _ = oracle.select(q[:4], k, "f32", np.array([0, N]), np.array([0, 4]), 1)
    masked = np.union1d(masked, o_ids0.ravel())
    words = np.zeros((N + 31) // 32, np.uint32)
    np.bitwise_or.at(words, masked >> 5, (np.uint32(1) << (masked & 31).astype(np.uint32)))
    vals = rng.integers(0, 1000, N).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(1000), B).astype(np.float32)
    ko, qo = np.array([0, N]), np.array([0, B])
    dev = "cuda"
    tq = torch.as_tensor(q, device=dev).to(torch.bfloat16).contiguous()
    tk = torch.as_tensor(k, device=dev).to(torch.bfloat16).contiguous()
    prob = knn.MixtureProblem(tq, tk, torch.as_tensor(vals, device=dev), torch.as_tensor(ko, device=dev),
                              torch.as_tensor(qo, device=dev), torch.as_tensor(p_lm, device=dev), R, 0.01,
                              key_offsets_host=ko, query_offsets_host=qo,
                              packed_keys=knn.pack_keys(tk) if layout == "packed" else None)
    out = prob.run_nest(0.3, 0.1, 0.5, key_mask=knn.mask_words(masked, N, dev))
    torch.cuda.synchronize()
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, R, key_mask=words)
    ids = out["ids"].cpu().numpy()
    assert not np.isin(ids, masked).any()
    np.testing.assert_array_equal(ids, o_ids)
    np.testing.assert_array_equal(out["dists"].cpu().numpy().astype(np.float64), o_d)
    lam = oracle.rrc_lambda(o_d, 0.3, 0.1)
    np.testing.assert_allclose(out["lambdas"].cpu().numpy().astype(np.float64), lam, rtol=0, atol=1e-6)
    ref = oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.01, lam)
    np.testing.assert_allclose(out["p_m"].cpu().numpy(), ref, rtol=0, atol=1e-5)
    want = nest.decode_outputs(out["p_m"].cpu().numpy(), ids, vals, ko, qo, out["lambdas"].cpu().numpy(), 0.5)
    assert out["next_token"].cpu().numpy().tolist() == want["next_token"].tolist()
    assert out["span_key"].cpu().numpy().tolist() == want["span_key"].tolist()
    del tk, prob
