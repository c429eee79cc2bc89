"""Pins of the oracle's NEST decoding decisions and key masking (oracle/nest.py,
oracle/knn_oracle.c) against hand-worked cases (tests/golden/verify_cases.json,
tests/golden/rrc_cases.json), brute force on tiny inputs and the properties the
paper's definitions fix (Section 3.3 eq. knn_interpolation and span_expansion,
Section 3.4 eq. rejection, its last paragraph on masking, Algorithm 1)."""
import json
import math
import os

import numpy as np
import pytest
from scipy.spatial.distance import cdist
from scipy.special import softmax

import oracle
from oracle import nest

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


# ------------------------------------------------------ relaxed verification

def _verify_doc(golden_dir):
    return json.load(open(os.path.join(golden_dir, "verify_cases.json")))


@pytest.mark.parametrize("fp32", [False, True])
def test_verify_hand_cases(golden_dir, fp32):
    doc = _verify_doc(golden_dir)
    p = np.array(doc["p_m"], np.float32 if fp32 else np.float64)
    dr = np.array(doc["draft_tokens"])
    out = nest.decode_outputs(p, np.full((len(p), 1), -1, np.int32), np.zeros(4, np.int32), np.array([0, 4]),
                              np.array([0, len(p)]), np.ones(len(p)), 0.5, dr)
    assert out["next_token"].tolist() == doc["next_token"]
    for case in doc["cases"]:
        n_acc, tok = nest.spec_verify(out["p_max"], out["p_draft"], out["next_token"],
                                      np.array(doc["draft_offsets"]), case["gamma"], fp32=fp32)
        assert n_acc.tolist() == case["n_accept"], case
        assert tok.tolist() == case["token"], case


def test_verify_greedy_drafts_are_always_accepted():
    rng = np.random.default_rng(3)
    p = rng.dirichlet(np.ones(50), 40)
    nt = p.argmax(1)
    for gamma in (1.0, 0.7, 0.05):
        n_acc, tok = nest.spec_verify(p.max(1), p[np.arange(40), nt], nt, np.array([0, 10, 25, 40]), gamma)
        assert n_acc.tolist() == [10, 15, 15] and tok.tolist() == [-1, -1, -1]


def test_verify_is_monotone_in_gamma():
    rng = np.random.default_rng(4)
    p = rng.dirichlet(np.full(30, 0.3), 64)
    draft = rng.integers(0, 30, 64)
    offs = np.arange(0, 65, 16)
    prev = None
    for gamma in (1.0, 0.5, 0.2, 0.05, 0.005, 5e-4):
        n_acc, _ = nest.spec_verify(p.max(1), p[np.arange(64), draft], p.argmax(1), offs, gamma)
        if prev is not None:
            assert np.all(n_acc >= prev)
        prev = n_acc
    assert prev.max() > 0


def test_verify_with_uniforms_reads_the_equation_as_a_probability():
    p = np.array([[0.5, 0.3, 0.2, 0.0], [0.5, 0.3, 0.2, 0.0]])
    pm, nt = p.max(1), p.argmax(1)
    # u = 0: accepted whenever p_M(w) > 0; a zero-probability draft is rejected
    n_acc, tok = nest.spec_verify(pm, p[[0, 1], [2, 3]], nt, np.array([0, 2]), 1.0, uniforms=np.zeros(2))
    assert (n_acc.tolist(), tok.tolist()) == ([1], [0])
    # u just below min(1, ratio) accepts, at it rejects: ratio 0.2 / (0.5 * 0.5) = 0.8
    for u, want in ((0.79, 2), (0.8, 0)):
        n_acc, _ = nest.spec_verify(pm, p[[0, 1], [2, 2]], nt, np.array([0, 2]), 0.5, uniforms=np.full(2, u))
        assert n_acc.tolist() == [want]
    # a ratio above 1 is capped: any u < 1 accepts
    n_acc, _ = nest.spec_verify(pm, p[[0, 1], [1, 1]], nt, np.array([0, 2]), 0.1, uniforms=np.full(2, 0.999))
    assert n_acc.tolist() == [2]


def test_verify_fp32_matches_fp64_away_from_the_threshold():
    rng = np.random.default_rng(5)
    p = rng.dirichlet(np.full(100, 0.5), 256).astype(np.float32)
    draft = rng.integers(0, 100, 256)
    pd, pm = p[np.arange(256), draft], p.max(1)
    ratio = pd.astype(np.float64) / (0.05 * pm.astype(np.float64))
    keep = np.abs(ratio - 0.5) > 1e-5
    offs = np.arange(257)  # one-row drafts: one decision each
    a32, _ = nest.spec_verify(pm, pd, p.argmax(1), offs, 0.05, fp32=True)
    a64, _ = nest.spec_verify(pm, pd, p.argmax(1), offs, 0.05)
    assert np.array_equal(a32[keep], a64[keep]) and keep.sum() > 200


# ------------------------------------------------------------ span selection

def test_span_selection_hand_cases(golden_dir):
    doc = json.load(open(os.path.join(golden_dir, "rrc_cases.json")))
    h = json.load(open(os.path.join(golden_dir, "hand_cases.json")))["H-A"]
    q = np.array([h["query"]], np.float32)
    k = np.array(h["keys"], np.float32)
    vals = np.array(h["values"], np.int32)
    p_lm = np.array([doc["p_lm"]], np.float32)
    ko, qo = np.array([0, 3]), np.array([0, 1])
    for case in doc["cases"]:
        ids, d = oracle.select(q, k, "f32", ko, qo, case["r"])
        lam = oracle.rrc_lambda(d, doc["alpha"], doc["tau"])
        pm = oracle.mix(ids, d, vals, ko, qo, p_lm, case["mu"], lam)
        out = nest.decode_outputs(pm, ids, vals, ko, qo, lam, doc["delta"])
        assert out["next_token"][0] == case["next_token"], case["name"]
        assert out["span_key"][0] == case["span_key"], case["name"]
        assert out["use_span"][0] == case["use_span"], case["name"]


def test_span_start_is_the_nearest_neighbour_carrying_the_token():
    rng = np.random.default_rng(6)
    for _ in range(20):
        n, r = 60, 12
        d = rng.integers(0, 5, n).astype(np.float64)  # many equal distances
        vals = rng.integers(0, 4, n).astype(np.int32)
        order = np.lexsort((np.arange(n), d))[:r]  # pi by (distance, id)
        for w in range(5):
            got = nest.span_start(order, vals, w)
            carriers = [i for i in range(n) if i in set(order.tolist()) and vals[i] == w]
            want = min(carriers, key=lambda i: (d[i], i)) if carriers else -1
            assert got == want


def test_use_span_threshold():
    assert nest.use_span(0.5, 0.5, 3) == 1  # lambda_t <= delta: the span
    assert nest.use_span(0.5000001, 0.5, 3) == 0
    assert nest.use_span(0.1, 0.5, -1) == 0  # no start in the store: the token
    assert nest.greedy_token(np.array([0.2, 0.4, 0.4])) == 1


# ------------------------------------------------------------------ masking

def _bits(masked, n):
    words = np.zeros((n + 31) // 32, np.uint32)
    for i in masked:
        words[i >> 5] |= np.uint32(1) << np.uint32(i & 31)
    return words


def test_masked_select_is_select_over_the_unmasked_keys():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((4, 6)).astype(np.float32)
    k = rng.standard_normal((90, 6)).astype(np.float32)
    ko, qo = np.array([0, 40, 90]), np.array([0, 2, 4])
    masked = rng.choice(90, 30, replace=False)
    ids, d = oracle.select(q, k, "f32", ko, qo, 8, key_mask=_bits(masked, 90))
    for b in range(4):
        s = 0 if b < 2 else 1
        keep = [i for i in range(ko[s], ko[s + 1]) if i not in set(masked.tolist())]
        dd = cdist(q[b:b + 1].astype(np.float64), k[keep].astype(np.float64), "sqeuclidean")[0]
        o = np.argsort(dd, kind="stable")[:8]
        assert ids[b].tolist() == [keep[i] - ko[s] for i in o]
        np.testing.assert_allclose(d[b], dd[o], rtol=1e-12, atol=1e-12)
    # an empty mask changes nothing
    ids0, d0 = oracle.select(q, k, "f32", ko, qo, 8)
    ids1, d1 = oracle.select(q, k, "f32", ko, qo, 8, key_mask=np.zeros(3, np.uint32))
    assert np.array_equal(ids0, ids1) and np.array_equal(d0, d1)


def test_masked_select_fills_missing_slots_as_absent():
    rng = np.random.default_rng(8)
    q = rng.standard_normal((1, 4)).astype(np.float32)
    k = rng.standard_normal((20, 4)).astype(np.float32)
    ko, qo = np.array([0, 20]), np.array([0, 1])
    masked = list(range(0, 20, 1))[:15]  # 5 unmasked keys, r = 8
    ids, d = oracle.select(q, k, "f32", ko, qo, 8, key_mask=_bits(masked, 20))
    assert sorted(ids[0, :5].tolist()) == list(range(15, 20))
    assert ids[0, 5:].tolist() == [-1, -1, -1] and np.all(np.isinf(d[0, 5:]))
    # absent neighbours carry no weight: the mixture equals the one over the 5 present
    vals = rng.integers(0, 9, 20).astype(np.int32)
    p_lm = softmax(rng.standard_normal((1, 9)), axis=1).astype(np.float32)
    full = oracle.mix(ids, d, vals, ko, qo, p_lm, 0.7, 0.4)
    part = oracle.mix(ids[:, :5].copy(), d[:, :5].copy(), vals, ko, qo, p_lm, 0.7, 0.4)
    np.testing.assert_allclose(full, part, rtol=0, atol=1e-15)
    # lambda_t ignores them too
    lam_full = oracle.rrc_lambda(d, 0.3, 0.1)
    lam_part = oracle.rrc_lambda(d[:, :5].copy(), 0.3, 0.1)
    assert lam_full[0] == lam_part[0]


def test_everything_masked_leaves_p_lm_weighted_by_lambda():
    rng = np.random.default_rng(9)
    q = rng.standard_normal((1, 4)).astype(np.float32)
    k = rng.standard_normal((10, 4)).astype(np.float32)
    ko, qo = np.array([0, 10]), np.array([0, 1])
    ids, d = oracle.select(q, k, "f32", ko, qo, 4, key_mask=_bits(range(10), 10))
    assert ids.tolist() == [[-1, -1, -1, -1]]
    p_lm = np.full((1, 5), 0.2, np.float32)
    pm = oracle.mix(ids, d, np.zeros(10, np.int32), ko, qo, p_lm, 1.0, 0.25)
    np.testing.assert_array_equal(pm, 0.25 * p_lm.astype(np.float64))
    assert oracle.rrc_lambda(d, 0.3, 0.1)[0] == 1.0 / (1.0 + math.exp(-7.0))
