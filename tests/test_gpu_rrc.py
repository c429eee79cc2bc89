"""GPU parity of relative retrieval confidence (paper Section 3.2, eq. rrc):
knn_lm_mixture_rrc and knn_mix_rrc against the oracle's rrc_lambda and its
mixture with one lambda per query, through every select path (split over
workgroups for few queries, one workgroup per query for rows of at most 64K
keys, the wide path for longer rows in fine tiles, and the general path for
the rest: longer rows with r > 2048, or r > 1024)."""
import math

import numpy as np
import pytest
import torch

import oracle
import parity
from workloads import gen

pytestmark = pytest.mark.gpu

knn = pytest.importorskip("paper_2405_19325_amd")

ALPHA, TAU = 0.3, 0.1  # the paper's values (Section 3.2)


def _say(msg):
    print(f"[gpu] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    knn.load()
    yield
    torch.cuda.synchronize()


def _integer_case(n, B, seed):
    """Integer keys (a, b, c, 0), a, b, c in [-6, 6], and queries (0, 0, 0, c_b):
    every distance is the exact integer a^2 + b^2 + c^2 + c_b^2, the nearest key
    sits at 0 or close to it, so d_(1) / d_(r) = (D_(1) + c_b^2) / (D_(r) + c_b^2)
    spreads the queries over the steep part of the sigmoid."""
    rng = np.random.default_rng(seed)
    k = np.zeros((n, 4), np.float32)
    k[:, :3] = rng.integers(-6, 7, (n, 3))
    q = np.zeros((B, 4), np.float32)
    q[:, 3] = np.arange(B) % 6
    V = 997
    vals = rng.integers(0, V, n).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(V), B).astype(np.float32)
    return q, k, vals, p_lm


# (path, n keys, queries, r): the split select needs B * ceil(n / 4096) <= 256,
# the one-workgroup select n <= 65536 and r <= 1024, the wide one rows of more
# than 65536 keys in at least 2 r distance tiles with r <= 2048 (16-row tiles
# here), the general one the rest.
PATHS = [("split", 40000, 6, 1024), ("one-workgroup", 40000, 40, 1024), ("wide-long-row", 70000, 6, 1024),
         ("general-long-row", 70000, 6, 2500), ("general-r2048", 40000, 3, 2048), ("split-r1", 5000, 4, 1)]


@pytest.mark.parametrize("path,n,B,r", PATHS, ids=[p[0] for p in PATHS])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_rrc_exact_integer_inputs(path, n, B, r, dtype):
    _say(f"rrc exact integers: {path} n={n} B={B} r={r} {dtype}")
    q, k, vals, p_lm = _integer_case(n, B, 40 + r)
    ko, qo = np.array([0, n]), np.array([0, B])
    dev = "cuda"
    tq, tk = torch.as_tensor(q, device=dev).to(dtype), torch.as_tensor(k, device=dev).to(dtype)
    prob = knn.MixtureProblem(tq, tk, torch.as_tensor(vals, device=dev), torch.as_tensor(ko, device=dev),
                              torch.as_tensor(qo, device=dev), torch.as_tensor(p_lm, device=dev), r, 0.05,
                              key_offsets_host=ko, query_offsets_host=qo)
    p_m, ids, dists, lam = prob.run_rrc(ALPHA, TAU)
    torch.cuda.synchronize()
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r)
    np.testing.assert_array_equal(ids.cpu().numpy(), o_ids)
    np.testing.assert_array_equal(dists.cpu().numpy().astype(np.float64), o_d)
    o_lam = oracle.rrc_lambda(o_d, ALPHA, TAU)
    np.testing.assert_allclose(lam.cpu().numpy().astype(np.float64), o_lam, rtol=0, atol=1e-6)
    if r > 1:
        assert o_lam.max() - o_lam.min() > 0.2, "the case should spread lambda_t"
    ref = oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.05, o_lam)
    np.testing.assert_allclose(p_m.cpu().numpy(), ref, rtol=0, atol=1e-5)
    # the standalone mixture on the same neighbours, given in reverse order
    rev = torch.flip(ids, dims=[1]).contiguous(), torch.flip(dists, dims=[1]).contiguous()
    p2, lam2 = knn.mix_rrc(rev[0], rev[1], prob.values, prob.key_offsets, prob.query_offsets, prob.p_lm, 0.05,
                           ALPHA, TAU)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(lam2.cpu().numpy(), lam.cpu().numpy())
    np.testing.assert_allclose(p2.cpu().numpy(), ref, rtol=0, atol=1e-5)


def test_rrc_ratio_equal_to_alpha_gives_one_half_exactly():
    """d_(1) = 3 and d_(r) = 10 on exact integers: the fp32 ratio rounds to the
    same float as alpha = 0.3, so lambda_t is exactly 1/2; a second set whose r
    neighbours all sit at distance 0 takes ratio 1."""
    _say("rrc ratio == alpha")
    near = [[1, 1, 1, 0], [2, 0, 0, 0], [2, 1, 0, 0], [2, 1, 1, 0], [2, 1, 1, 1], [2, 2, 0, 0], [3, 0, 0, 0],
            [3, 1, 0, 0]]  # squared norms 3, 4, 5, 6, 7, 8, 9, 10
    far = [[4 + i % 3, i % 5, 0, 0] for i in range(40)]  # squared norms >= 16
    k0 = np.array(near + far, np.float32)
    k1 = np.zeros((30, 4), np.float32)
    k = np.concatenate([k0, k1])
    ko, qo = np.array([0, len(k0), len(k)]), np.array([0, 1, 2])
    q = np.zeros((2, 4), np.float32)
    vals = (np.arange(len(k)) % 7).astype(np.int32)
    p_lm = np.full((2, 7), 1 / 7, np.float32)
    dev = "cuda"
    prob = knn.MixtureProblem(torch.as_tensor(q, device=dev), torch.as_tensor(k, device=dev),
                              torch.as_tensor(vals, device=dev), torch.as_tensor(ko, device=dev),
                              torch.as_tensor(qo, device=dev), torch.as_tensor(p_lm, device=dev), 8, 0.5,
                              key_offsets_host=ko, query_offsets_host=qo)
    _, ids, dists, lam = prob.run_rrc(np.float32(ALPHA), TAU)
    torch.cuda.synchronize()
    assert dists[0].cpu().numpy().tolist() == [3, 4, 5, 6, 7, 8, 9, 10]
    assert lam[0].item() == 0.5
    assert abs(lam[1].item() - 1 / (1 + math.exp(-7.0))) < 1e-6


SYNTH = [
    ("decode-bf16-split", gen.scaled(gen.config("decode_7b"), n_keys=30000, B=2), 51),
    ("ragged-bf16", gen.scaled(gen.config("ragged_batch"), B=12, S=4, n_keys=(1100, 5000, 3333, 2048), r=1024), 52),
    ("batch-f16-mfma", gen.scaled(gen.config("specverify_static"), B=64, S=2, n_keys=(6000, 9000), d=1024,
                                  query_mode="iid"), 53),
    ("decode-bf16-one-workgroup", gen.scaled(gen.config("decode_7b"), n_keys=20000, B=60), 55),
    ("long-row-bf16", gen.scaled(gen.config("decode_7b"), n_keys=80000, B=2, d=512, mu=1 / math.sqrt(512)), 54),
]


@pytest.mark.parametrize("name,spec,seed", SYNTH, ids=[s[0] for s in SYNTH])
def test_rrc_synthetic_workloads(name, spec, seed):
    """Synthetic workloads with alpha at the median of the oracle's ratios, so
    lambda_t sits where the sigmoid is steepest: P2-P6."""
    _say(f"rrc workload {name}")
    w = gen.make(spec, seed, device="cuda")
    ko, qo = w.key_offsets_host, w.query_offsets_host
    ratios = []
    for s in range(len(ko) - 1):
        if qo[s + 1] == qo[s]:
            continue
        kh, dt = oracle.host_elements(w.keys[ko[s]:ko[s + 1]])
        qh, _ = oracle.host_elements(w.queries[qo[s]:qo[s + 1]])
        _, od = oracle.select(qh, kh, dt, np.array([0, len(kh)]), np.array([0, len(qh)]), w.r)
        ratios.extend((od[:, 0] / od[:, -1]).tolist())
    alpha = float(np.median(ratios))
    prob = knn.MixtureProblem(w.queries, w.keys, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu,
                              w.lam, key_offsets_host=ko, query_offsets_host=qo)
    p_m, ids, dists, lam = prob.run_rrc(alpha, TAU)
    torch.cuda.synchronize()
    rep = parity.check_workload(w, p_m, ids, dists, rrc=(alpha, TAU), lambdas=lam)
    _say(f"{name}: alpha={alpha:.4f} lambda_t in [{lam.min().item():.3f}, {lam.max().item():.3f}]: {rep.summary()}")
    assert rep.ok(), rep.failures[:5]


def test_rrc_full_size_decode():
    """The decode workload at full size (64K bf16 keys of width 4096, r = 1024)
    with the paper's alpha and tau."""
    _say("rrc full decode_7b")
    w = gen.make(gen.config("decode_7b"), gen.CONFIG_SEEDS["decode_7b"], device="cuda")
    prob = knn.MixtureProblem(w.queries, w.keys, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu,
                              w.lam, key_offsets_host=w.key_offsets_host, query_offsets_host=w.query_offsets_host)
    p_m, ids, dists, lam = prob.run_rrc(ALPHA, TAU)
    torch.cuda.synchronize()
    rep = parity.check_workload(w, p_m, ids, dists, rrc=(ALPHA, TAU), lambdas=lam)
    _say(f"decode_7b rrc: lambda_t={lam.tolist()}: {rep.summary()}")
    assert rep.ok(), rep.failures[:5]


def test_rrc_rejects_bad_parameters():
    _say("rrc argument checks")
    q, k, vals, p_lm = _integer_case(100, 1, 1)
    dev = "cuda"
    ko, qo = np.array([0, 100]), np.array([0, 1])
    prob = knn.MixtureProblem(torch.as_tensor(q, device=dev), torch.as_tensor(k, device=dev),
                              torch.as_tensor(vals, device=dev), torch.as_tensor(ko, device=dev),
                              torch.as_tensor(qo, device=dev), torch.as_tensor(p_lm, device=dev), 4, 0.5,
                              key_offsets_host=ko, query_offsets_host=qo)
    for alpha, tau in ((0.3, 0.0), (0.3, -1.0), (float("nan"), 0.1), (0.3, float("inf")), (float("inf"), 0.1)):
        with pytest.raises(knn.KnnError):
            prob.run_rrc(alpha, tau)
