"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle (oracle/knn_oracle.c) against something other than
itself: hand-worked closed forms (tests/golden/hand_cases.json), closed-form
invariants of eq. non-parametric and eq. kNN-LM (paper Section 2.2), library
routines (scipy's squared-Euclidean cdist, numpy's stable argsort, scipy's
softmax, numpy / torch element conversions), exact-integer inputs and
metamorphic relations.  A dropped term, a wrong sign, index or operand in the
oracle fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
from scipy.spatial.distance import cdist
from scipy.special import softmax

import oracle

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def _one_set(B, N):
    return np.array([0, N], dtype=np.int64), np.array([0, B], dtype=np.int64)


def _rand_case(rng, B=3, N=200, d=16, V=50, scale=1.0):
    q = (rng.standard_normal((B, d)) * scale).astype(np.float32)
    k = (rng.standard_normal((N, d)) * scale).astype(np.float32)
    vals = rng.integers(0, V, N).astype(np.int32)
    logits = rng.standard_normal((B, V))
    p_lm = softmax(logits, axis=1).astype(np.float32)
    return q, k, vals, p_lm


def _full(q, k, vals, p_lm, r, mu, lam, dtype="f32", want_pknn=False):
    ko, qo = _one_set(q.shape[0], k.shape[0])
    ids, dists = oracle.select(q, k, dtype, ko, qo, r)
    out = oracle.mix(ids, dists, vals, ko, qo, p_lm, mu, lam, want_pknn=want_pknn)
    return ids, dists, out


# ---------------------------------------------------------------- hand cases

def _eval_closed_form(expr: str) -> float:
    return float(eval(expr, {"__builtins__": {}}, {"exp": math.exp, "sqrt": math.sqrt}))


@pytest.mark.parametrize("which", ["H-A", "H-B"])
def test_hand_cases(golden_dir, which):
    doc = json.load(open(os.path.join(golden_dir, "hand_cases.json")))[which]
    q = np.array([doc["query"]], dtype=np.float32)
    k = np.array(doc["keys"], dtype=np.float32)
    vals = np.array(doc["values"], dtype=np.int32)
    p_lm = np.array([doc["p_lm"]], dtype=np.float32)
    for case in doc["cases"]:
        ids, dists, (pm, pk) = _full(q, k, vals, p_lm, case["r"], case["mu"], doc["lam"], want_pknn=True)
        assert ids[0].tolist() == case["expect_ids"], case["name"]
        np.testing.assert_array_equal(dists[0], np.array(case["expect_dists"], dtype=np.float64))
        pknn = np.array([_eval_closed_form(e) for e in case["pknn_expr"]])
        np.testing.assert_allclose(pk[0], pknn, rtol=0, atol=1e-14, err_msg=case["name"])
        p_m = doc["lam"] * p_lm[0].astype(np.float64) + (1 - doc["lam"]) * pknn
        np.testing.assert_allclose(pm[0], p_m, rtol=0, atol=1e-14, err_msg=case["name"])
        # the decimals stored next to the closed forms agree up to p_LM's fp32 rounding
        np.testing.assert_allclose(pm[0], case["p_m"], rtol=0, atol=5e-8)


# ------------------------------------------------------------- closed forms

@pytest.mark.parametrize("lam", [0.0, 0.3, 0.5, 1.0])
def test_pm_sums(lam):
    rng = np.random.default_rng(1)
    q, k, vals, p_lm = _rand_case(rng)
    _, _, pm = _full(q, k, vals, p_lm, 20, 0.25, lam)
    expect = lam * p_lm.astype(np.float64).sum(1) + (1 - lam)
    np.testing.assert_allclose(pm.sum(1), expect, rtol=0, atol=1e-12)


def test_lambda_one_returns_plm_exactly():
    rng = np.random.default_rng(2)
    q, k, vals, p_lm = _rand_case(rng)
    _, _, pm = _full(q, k, vals, p_lm, 17, 0.5, 1.0)
    np.testing.assert_array_equal(pm, p_lm.astype(np.float64))


def test_lambda_zero_returns_pknn():
    rng = np.random.default_rng(3)
    q, k, vals, p_lm = _rand_case(rng)
    _, _, (pm, pk) = _full(q, k, vals, p_lm, 17, 0.5, 0.0, want_pknn=True)
    np.testing.assert_array_equal(pm, pk)
    np.testing.assert_allclose(pk.sum(1), 1.0, atol=1e-12)


def test_r1_is_one_hot_at_nearest_value():
    rng = np.random.default_rng(4)
    q, k, vals, p_lm = _rand_case(rng, B=5)
    ids, _, (pm, pk) = _full(q, k, vals, p_lm, 1, 0.1, 0.3, want_pknn=True)
    nearest = cdist(q.astype(np.float64), k.astype(np.float64), "sqeuclidean").argmin(1)
    for b in range(q.shape[0]):
        assert ids[b, 0] == nearest[b]
        onehot = np.zeros(p_lm.shape[1])
        onehot[vals[nearest[b]]] = 1.0
        np.testing.assert_array_equal(pk[b], onehot)


def test_duplicate_tokens_accumulate():
    rng = np.random.default_rng(5)
    q, k, _, p_lm = _rand_case(rng)
    same = np.full(k.shape[0], 7, dtype=np.int32)
    _, _, (_, pk) = _full(q, k, same, p_lm, 33, 0.7, 0.2, want_pknn=True)
    expect = np.zeros_like(pk)
    expect[:, 7] = 1.0
    np.testing.assert_allclose(pk, expect, atol=1e-14)
    # two neighbours sharing a token: p_kNN(token) is the sum of their weights
    vals = np.arange(k.shape[0], dtype=np.int32) % 50
    ids, dists, (_, pk) = _full(q[:1], k, vals, p_lm[:1], 2, 1.0, 0.0, want_pknn=True)
    vals2 = vals.copy()
    vals2[ids[0, 1]] = vals2[ids[0, 0]]
    _, _, (_, pk2) = _full(q[:1], k, vals2, p_lm[:1], 2, 1.0, 0.0, want_pknn=True)
    t0, t1 = vals[ids[0, 0]], vals[ids[0, 1]]
    assert t0 != t1
    assert pk2[0, t0] == pytest.approx(pk[0, t0] + pk[0, t1], abs=1e-15)
    assert pk2[0, t0] == pytest.approx(1.0, abs=1e-15)


def test_mu_to_zero_gives_counts():
    rng = np.random.default_rng(6)
    q, k, vals, p_lm = _rand_case(rng, V=8)
    r = 40
    ids, _, (_, pk) = _full(q, k, vals, p_lm, r, 1e-30, 0.5, want_pknn=True)
    for b in range(q.shape[0]):
        counts = np.bincount(vals[ids[b]], minlength=8) / r
        np.testing.assert_allclose(pk[b], counts, atol=1e-15)


def test_r_equals_n_is_textbook_softmax_over_all_keys():
    """With every key retrieved, p_kNN is the textbook softmax of -mu*d over all keys,
    scattered onto their tokens (equivalently attention logits mu*(2 q.k - |k|^2))."""
    rng = np.random.default_rng(7)
    q, k, vals, p_lm = _rand_case(rng, B=2, N=64, d=9, V=11)
    mu = 0.37
    _, _, (_, pk) = _full(q, k, vals, p_lm, 64, mu, 0.4, want_pknn=True)
    d = cdist(q.astype(np.float64), k.astype(np.float64), "sqeuclidean")
    w = softmax(-mu * d, axis=1)
    att = softmax(mu * (2 * q.astype(np.float64) @ k.astype(np.float64).T - (k.astype(np.float64) ** 2).sum(1)), axis=1)
    np.testing.assert_allclose(w, att, atol=1e-12)
    for b in range(2):
        expect = np.zeros(11)
        np.add.at(expect, vals, w[b])
        np.testing.assert_allclose(pk[b], expect, atol=1e-12)


# ------------------------------------------------------- distances and order

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_distances_match_library_cdist(seed):
    rng = np.random.default_rng(10 + seed)
    q = rng.standard_normal((4, 37)).astype(np.float32)
    k = rng.standard_normal((300, 37)).astype(np.float32)
    got = oracle.sqdist(q, k, "f32")
    ref = cdist(q.astype(np.float64), k.astype(np.float64), "sqeuclidean")
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-12)


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_topr_matches_stable_argsort(seed):
    rng = np.random.default_rng(20 + seed)
    # small-integer coordinates make many exact ties in distance
    q = rng.integers(-2, 3, (3, 4)).astype(np.float32)
    k = rng.integers(-2, 3, (120, 4)).astype(np.float32)
    r = 30
    ko, qo = _one_set(3, 120)
    ids, dists = oracle.select(q, k, "f32", ko, qo, r)
    d = cdist(q.astype(np.float64), k.astype(np.float64), "sqeuclidean")
    for b in range(3):
        order = np.argsort(d[b], kind="stable")[:r]
        assert ids[b].tolist() == order.tolist()
        np.testing.assert_array_equal(dists[b], d[b, order])


def test_exact_integer_inputs_give_exact_distances():
    rng = np.random.default_rng(30)
    for dtype, conv in (("f32", lambda a: a.astype(np.float32)),
                        ("bf16", lambda a: torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16)),
                        ("f16", lambda a: a.astype(np.float16))):
        qi = rng.integers(-4, 5, (2, 64))
        ki = rng.integers(-4, 5, (500, 64))
        q, k = conv(qi), conv(ki)
        if isinstance(q, torch.Tensor):
            q, _ = oracle.host_elements(q)
            k, _ = oracle.host_elements(k)
        elif dtype == "f16":
            q, k = q.view(np.uint16), k.view(np.uint16)
        got = oracle.sqdist(q, k, dtype)
        exact = ((qi[:, None, :] - ki[None, :, :]) ** 2).sum(-1)
        np.testing.assert_array_equal(got, exact.astype(np.float64))


def test_planted_key_is_rank_one_at_distance_zero():
    rng = np.random.default_rng(31)
    k = rng.standard_normal((400, 24)).astype(np.float32)
    q = k[[123, 7]].copy()
    ko, qo = _one_set(2, 400)
    ids, dists = oracle.select(q, k, "f32", ko, qo, 5)
    assert ids[:, 0].tolist() == [123, 7]
    assert dists[0, 0] == 0.0 and dists[1, 0] == 0.0


def test_metamorphic_permutation_translation_scaling():
    rng = np.random.default_rng(32)
    q = rng.integers(-3, 4, (2, 6)).astype(np.float32)
    k = rng.integers(-3, 4, (90, 6)).astype(np.float32)
    vals = rng.integers(0, 13, 90).astype(np.int32)
    p_lm = softmax(rng.standard_normal((2, 13)), axis=1).astype(np.float32)
    r, mu, lam = 25, 0.3, 0.4
    ids, dists, pm = _full(q, k, vals, p_lm, r, mu, lam)
    # permuting (key, value) rows: same p_M (keys here are distinct rows only up to ties,
    # so compare p_M after breaking no ties: use r such that the r-th distance is not tied)
    perm = rng.permutation(90)
    inv = np.argsort(perm)
    ids_p, dists_p, pm_p = _full(q, k[perm], vals[perm], p_lm, r, mu, lam)
    for b in range(2):
        d_sorted = np.sort(cdist(q[b:b + 1].astype(np.float64), k.astype(np.float64), "sqeuclidean")[0])
        if d_sorted[r - 1] != d_sorted[r]:
            assert sorted(perm[ids_p[b]].tolist()) == sorted(ids[b].tolist())
            np.testing.assert_allclose(pm_p[b], pm[b], atol=1e-15)
        np.testing.assert_array_equal(np.sort(dists_p[b]), np.sort(dists[b]))
    assert inv.shape == perm.shape
    # translating q and every key by one integer vector leaves distances (and all outputs) unchanged
    t = rng.integers(-5, 6, 6).astype(np.float32)
    ids_t, dists_t, pm_t = _full(q + t, k + t, vals, p_lm, r, mu, lam)
    np.testing.assert_array_equal(ids_t, ids)
    np.testing.assert_array_equal(dists_t, dists)
    np.testing.assert_array_equal(pm_t, pm)
    # scaling q, k by c and mu by 1/c^2 leaves p unchanged
    c = 2.0
    ids_s, dists_s, pm_s = _full(q * c, k * c, vals, p_lm, r, mu / c ** 2, lam)
    np.testing.assert_array_equal(ids_s, ids)
    np.testing.assert_array_equal(dists_s, dists * c ** 2)
    np.testing.assert_allclose(pm_s, pm, atol=1e-15)


# ---------------------------------------------------------- key-set structure

def test_ragged_sets_are_independent():
    rng = np.random.default_rng(40)
    d = 12
    sizes = [50, 130, 77]
    qps = [2, 1, 3]
    k = rng.standard_normal((sum(sizes), d)).astype(np.float32)
    q = rng.standard_normal((sum(qps), d)).astype(np.float32)
    vals = rng.integers(0, 30, sum(sizes)).astype(np.int32)
    p_lm = softmax(rng.standard_normal((sum(qps), 30)), axis=1).astype(np.float32)
    ko = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    qo = np.concatenate([[0], np.cumsum(qps)]).astype(np.int64)
    r = 9
    ids, dists = oracle.select(q, k, "f32", ko, qo, r)
    pm = oracle.mix(ids, dists, vals, ko, qo, p_lm, 0.5, 0.3)
    for s in range(3):
        ks = k[ko[s]:ko[s + 1]]
        vs = vals[ko[s]:ko[s + 1]]
        qs = q[qo[s]:qo[s + 1]]
        dd = cdist(qs.astype(np.float64), ks.astype(np.float64), "sqeuclidean")
        ids1, dists1, pm1 = _full(qs, ks, vs, p_lm[qo[s]:qo[s + 1]], r, 0.5, 0.3)
        np.testing.assert_array_equal(ids[qo[s]:qo[s + 1]], ids1)
        np.testing.assert_array_equal(pm[qo[s]:qo[s + 1]], pm1)
        for i, b in enumerate(range(qo[s], qo[s + 1])):
            assert ids[b].tolist() == np.argsort(dd[i], kind="stable")[:r].tolist()


def test_rejects_r_larger_than_set():
    q = np.zeros((1, 2), np.float32)
    k = np.zeros((3, 2), np.float32)
    ko, qo = _one_set(1, 3)
    with pytest.raises(oracle.OracleError):
        oracle.select(q, k, "f32", ko, qo, 4)


def test_rejects_value_out_of_vocab():
    ids = np.array([[0]], np.int32)
    dists = np.array([[1.0]])
    with pytest.raises(oracle.OracleError):
        oracle.mix(ids, dists, np.array([5], np.int32), np.array([0, 1]), np.array([0, 1]),
                   np.full((1, 4), 0.25, np.float32), 1.0, 0.5)


# ------------------------------------------------------------- decoding

def test_bf16_decoding_matches_torch_for_every_pattern():
    pats = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.widen(pats, "bf16")
    ref = torch.from_numpy(pats.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64).numpy()
    nan = np.isnan(ref)
    np.testing.assert_array_equal(np.isnan(got), nan)
    np.testing.assert_array_equal(got[~nan], ref[~nan])


def test_f16_decoding_matches_numpy_for_every_pattern():
    pats = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.widen(pats, "f16")
    ref = pats.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    np.testing.assert_array_equal(np.isnan(got), nan)
    np.testing.assert_array_equal(got[~nan], ref[~nan])


# ------------------------------------------- relative retrieval confidence

ALPHA, TAU = 0.3, 0.1


def test_rrc_hand_cases(golden_dir):
    doc = json.load(open(os.path.join(golden_dir, "rrc_cases.json")))
    h = json.load(open(os.path.join(golden_dir, "hand_cases.json")))["H-A"]
    q = np.array([h["query"]], dtype=np.float32)
    k = np.array(h["keys"], dtype=np.float32)
    vals = np.array(h["values"], dtype=np.int32)
    p_lm = np.array([doc["p_lm"]], dtype=np.float32)
    for case in doc["cases"]:
        ko, qo = _one_set(1, k.shape[0])
        ids, dists = oracle.select(q, k, "f32", ko, qo, case["r"])
        lam = oracle.rrc_lambda(dists, doc["alpha"], doc["tau"])
        want_lam = _eval_closed_form(case["lambda_expr"])
        assert abs(lam[0] - want_lam) <= 1e-15, case["name"]
        pm, pk = oracle.mix(ids, dists, vals, ko, qo, p_lm, case["mu"], lam, want_pknn=True)
        pknn = np.array([_eval_closed_form(e) for e in case["pknn_expr"]])
        np.testing.assert_allclose(pk[0], pknn, rtol=0, atol=1e-14, err_msg=case["name"])
        want = want_lam * p_lm[0].astype(np.float64) + (1 - want_lam) * pknn
        np.testing.assert_allclose(pm[0], want, rtol=0, atol=1e-14, err_msg=case["name"])


def test_rrc_ratio_equal_to_alpha_gives_one_half():
    # 3/10 rounds to the same double as the literal 0.3, so the logit is exactly 0
    lam = oracle.rrc_lambda(np.array([[3.0, 7.0, 10.0], [10.0, 3.0, 5.0]]), ALPHA, TAU)
    assert lam.tolist() == [0.5, 0.5]


def test_rrc_known_sigmoid_values():
    # sigmoid(ln 3) = 3/4 and sigmoid(-ln 3) = 1/4
    for sign, want in ((1, 0.75), (-1, 0.25)):
        ratio = ALPHA + sign * TAU * math.log(3.0)
        lam = oracle.rrc_lambda(np.array([[ratio * 8.0, 8.0]]), ALPHA, TAU)
        assert abs(lam[0] - want) < 1e-15


def test_rrc_symmetry_about_alpha():
    rng = np.random.default_rng(11)
    d = rng.uniform(0.5, 4.0, (64, 16))
    ratio = d.min(1) / d.max(1)
    lam = oracle.rrc_lambda(d, ALPHA, TAU)
    for b in range(0, 64, 7):
        # alpha' = 2*ratio - alpha mirrors the logit: lambda' = 1 - lambda
        mirrored = oracle.rrc_lambda(d[b:b + 1], 2 * ratio[b] - ALPHA, TAU)
        assert abs(mirrored[0] + lam[b] - 1.0) < 1e-12


def test_rrc_limits_and_degenerate_rows():
    # one neighbour, or every neighbour at one distance (0 included): ratio 1
    want = 1.0 / (1.0 + math.exp(-7.0))
    lam = oracle.rrc_lambda(np.array([[2.5, 2.5, 2.5], [0.0, 0.0, 0.0]]), ALPHA, TAU)
    np.testing.assert_allclose(lam, [want, want], rtol=0, atol=1e-15)
    assert abs(oracle.rrc_lambda(np.array([[4.0]]), ALPHA, TAU)[0] - want) < 1e-15
    # an exact match next to a far key: ratio 0
    lam0 = oracle.rrc_lambda(np.array([[0.0, 5.0]]), ALPHA, TAU)
    assert abs(lam0[0] - 1.0 / (1.0 + math.exp(3.0))) < 1e-15
    with pytest.raises(RuntimeError):
        oracle.rrc_lambda(np.array([[-1.0, 2.0]]), ALPHA, TAU)
    with pytest.raises(RuntimeError):
        oracle.rrc_lambda(np.array([[1.0, 2.0]]), ALPHA, 0.0)


def test_rrc_scale_and_order_invariant_and_monotone():
    rng = np.random.default_rng(12)
    d = rng.uniform(0.1, 3.0, (32, 8))
    lam = oracle.rrc_lambda(d, ALPHA, TAU)
    np.testing.assert_allclose(oracle.rrc_lambda(d * 37.0, ALPHA, TAU), lam, rtol=1e-14, atol=0)
    np.testing.assert_array_equal(oracle.rrc_lambda(d[:, ::-1], ALPHA, TAU), lam)
    # moving the nearest neighbour closer lowers the ratio, hence lambda_t
    closer = d.copy()
    closer[np.arange(32), d.argmin(1)] *= 0.5
    assert np.all(oracle.rrc_lambda(closer, ALPHA, TAU) < lam)
    assert np.all((lam > 0) & (lam < 1))


def test_mix_with_per_query_lambdas_matches_rows_of_scalar_mix():
    rng = np.random.default_rng(13)
    q, k, vals, p_lm = _rand_case(rng, B=4, N=120, d=8, V=30)
    ko, qo = _one_set(4, 120)
    ids, dists = oracle.select(q, k, "f32", ko, qo, 10)
    lams = np.array([0.0, 0.25, 0.7, 1.0])
    pm = oracle.mix(ids, dists, vals, ko, qo, p_lm, 0.5, lams)
    for b, lam in enumerate(lams):
        one = oracle.mix(ids, dists, vals, ko, qo, p_lm, 0.5, float(lam))
        np.testing.assert_array_equal(pm[b], one[b])
    np.testing.assert_array_equal(pm[3], p_lm[3].astype(np.float64))
    with pytest.raises(ValueError):
        oracle.mix(ids, dists, vals, ko, qo, p_lm, 0.5, lams[:3])
    with pytest.raises(RuntimeError):
        oracle.mix(ids, dists, vals, ko, qo, p_lm, 0.5, np.array([0.1, 0.2, 1.5, 0.3]))
