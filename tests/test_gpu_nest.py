"""GPU parity of a NEST decoding step (knn_nest_step) and of relaxed speculative
verification (knn_spec_verify) against the oracle: key masking (Section 3.4),
the greedy token, span start and span flag (Algorithm 1, Section 3.3) and the
accept/reject decisions (Section 3.4, eq. rejection).

Decisions that floating point takes (an argmax, a ratio against 1/2) are
checked on the GPU's own fp32 p_M rows with the oracle's decision functions,
so both sides decide on the same numbers; the p_M rows themselves are checked
against the fp64 oracle mixture under the usual parity rules."""
import math

import numpy as np
import pytest
import torch

import oracle
import parity
from oracle import nest
from workloads import gen

pytestmark = pytest.mark.gpu

knn = pytest.importorskip("paper_2405_19325_amd")

ALPHA, TAU, DELTA = 0.3, 0.1, 0.5


def _say(msg):
    print(f"[gpu] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    knn.load()
    yield
    torch.cuda.synchronize()


def _bits(masked, n):
    words = np.zeros((n + 31) // 32, np.uint32)
    for i in masked:
        words[i >> 5] |= np.uint32(1) << np.uint32(i & 31)
    return words


def _integer_store(n, B, d, seed):
    """Integer keys (a, b, c, 0, ...), a, b, c in [-6, 6], and queries (0, 0, 0, c_b, 0, ...):
    every distance is an exact integer (as in the RRC tests), so ids and
    distances must match the oracle bit for bit."""
    rng = np.random.default_rng(seed)
    k = np.zeros((n, d), np.float32)
    k[:, :3] = rng.integers(-6, 7, (n, 3))
    q = np.zeros((B, d), np.float32)
    q[:, 3] = np.arange(B) % 6
    V = 997
    vals = rng.integers(0, V, n).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(V), B).astype(np.float32)
    return rng, q, k, vals, p_lm


def _problem(q, k, vals, p_lm, ko, qo, r, mu, dtype):
    dev = "cuda"
    tq, tk = torch.as_tensor(q, device=dev).to(dtype), torch.as_tensor(k, device=dev).to(dtype)
    return knn.MixtureProblem(tq.contiguous(), tk.contiguous(), torch.as_tensor(vals, device=dev),
                              torch.as_tensor(ko, device=dev), torch.as_tensor(qo, device=dev),
                              torch.as_tensor(p_lm, device=dev), r, mu, key_offsets_host=ko, query_offsets_host=qo)


def _check_decisions(out, vals, ko, qo, draft=None):
    """The step's decoding outputs equal the oracle's decisions on the GPU's own p_M rows."""
    pm = out["p_m"].cpu().numpy()
    want = nest.decode_outputs(pm, out["ids"].cpu().numpy(), vals, ko, qo, out["lambdas"].cpu().numpy(), DELTA,
                               None if draft is None else draft.cpu().numpy())
    assert out["next_token"].cpu().numpy().tolist() == want["next_token"].tolist()
    assert np.array_equal(out["p_max"].cpu().numpy(), want["p_max"])
    assert out["span_key"].cpu().numpy().tolist() == want["span_key"].tolist()
    assert out["use_span"].cpu().numpy().tolist() == want["use_span"].tolist()
    if draft is not None:
        assert np.array_equal(out["p_draft"].cpu().numpy(), want["p_draft"])
    return want


# (path, n keys per set, queries, r, d): the split select needs B * ceil(n / 4096)
# <= 256, the one-workgroup select n <= 65536 and r <= 1024, the wide one rows of
# more than 65536 keys in at least 2 r distance tiles with r <= 2048, the general
# one the rest; 16 or more bf16 queries of a set with d % 128 == 0 take the matrix cores.
PATHS = [("split", 40000, 6, 1024, 4), ("one-workgroup", 40000, 40, 1024, 4),
         ("wide-long-row", 70000, 6, 1024, 4), ("general-long-row", 70000, 6, 2500, 4),
         ("general-r2048", 40000, 3, 2048, 4),
         ("matrix-core", 20000, 32, 1024, 128)]


# The matrix cores serve 16-bit keys only, so that path runs in bf16 alone.
MASKED_CASES = [(p, dt) for p in PATHS for dt in (torch.float32, torch.bfloat16)
                if not (p[0] == "matrix-core" and dt == torch.float32)]


@pytest.mark.parametrize("path,n,B,r,d,dtype", [(*p, dt) for p, dt in MASKED_CASES],
                         ids=[f"{p[0]}-{str(dt).split('.')[-1]}" for p, dt in MASKED_CASES])
def test_masked_exact_integer_inputs(path, n, B, r, d, dtype):
    _say(f"masked exact integers: {path} n={n} B={B} r={r} d={d} {dtype}")
    rng, q, k, vals, p_lm = _integer_store(n, B, d, 60 + r + d)
    masked = rng.choice(n, n // 3, replace=False)
    # also mask the exact matches of the first queries, which would be nearest
    masked = np.union1d(masked, np.flatnonzero(np.all(k[:, :3] == 0, axis=1))[:5])
    ko, qo = np.array([0, n]), np.array([0, B])
    prob = _problem(q, k, vals, p_lm, ko, qo, r, 0.05, dtype)
    out = prob.run_nest(ALPHA, TAU, DELTA, key_mask=knn.mask_words(masked, n, "cuda"))
    torch.cuda.synchronize()
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r, key_mask=_bits(masked, n))
    ids = out["ids"].cpu().numpy()
    assert not np.isin(ids, masked).any()
    np.testing.assert_array_equal(ids, o_ids)
    np.testing.assert_array_equal(out["dists"].cpu().numpy().astype(np.float64), o_d)
    o_lam = oracle.rrc_lambda(o_d, ALPHA, TAU)
    np.testing.assert_allclose(out["lambdas"].cpu().numpy().astype(np.float64), o_lam, rtol=0, atol=1e-6)
    ref = oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.05, o_lam)
    np.testing.assert_allclose(out["p_m"].cpu().numpy(), ref, rtol=0, atol=1e-5)
    _check_decisions(out, vals, ko, qo)


@pytest.mark.parametrize("path,B,r", [("split", 2, 64), ("one-workgroup", 300, 64), ("general", 2, 2048)])
def test_fewer_unmasked_keys_than_r(path, B, r):
    """Set 0 keeps r/2 unmasked keys, set 1 none: pi ends in absent slots (id -1,
    distance +inf) that carry no weight, and a query with no neighbour gets
    p_M = lambda_t p_LM with lambda_t = sigmoid((1 - alpha) / tau)."""
    _say(f"fewer unmasked keys than r: {path}")
    n = 3000 if path != "general" else 5000
    rng, q, k, vals, p_lm = _integer_store(2 * n, 2 * B, 4, 70 + B)
    ko, qo = np.array([0, n, 2 * n]), np.array([0, B, 2 * B])
    keep = rng.choice(n, r // 2, replace=False)
    masked = np.concatenate([np.setdiff1d(np.arange(n), keep), np.arange(n, 2 * n)])
    prob = _problem(q, k, vals, p_lm, ko, qo, r, 0.05, torch.float32)
    out = prob.run_nest(ALPHA, TAU, DELTA, key_mask=knn.mask_words(masked, 2 * n, "cuda"))
    torch.cuda.synchronize()
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r, key_mask=_bits(masked, 2 * n))
    ids = out["ids"].cpu().numpy()
    np.testing.assert_array_equal(ids, o_ids)
    assert np.all(ids[:B, r // 2:] == -1) and np.all(ids[B:] == -1)
    assert np.all(np.isinf(out["dists"].cpu().numpy()[:, r // 2:]))
    o_lam = oracle.rrc_lambda(o_d, ALPHA, TAU)
    np.testing.assert_allclose(out["lambdas"].cpu().numpy().astype(np.float64), o_lam, rtol=0, atol=1e-6)
    ref = oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.05, o_lam)
    np.testing.assert_allclose(out["p_m"].cpu().numpy(), ref, rtol=0, atol=1e-5)
    assert out["span_key"].cpu().numpy()[B:].tolist() == [-1] * B
    _check_decisions(out, vals, ko, qo)


@pytest.mark.parametrize("V", [10001, 12288])
def test_rows_written_in_vocabulary_slices(V):
    """The split select's finish writes each row in slices of 4096 entries, one
    workgroup each (here 3), and combines the NEST outputs across them: the
    greedy token lies in a different slice per query, drafts in the first and
    last slice and outside [0, V).  V = 10001 takes the 4-byte mixture, 12288
    the 16-byte one.  Two NEST steps in a row (the row maximum and count start
    again from zero), the RRC step and the fixed-lambda step all match the
    oracle."""
    _say(f"rows in vocabulary slices: V={V}")
    n, B, r, d = 20000, 3, 256, 4
    rng = np.random.default_rng(V)
    k = np.zeros((n, d), np.float32)
    k[:, :3] = rng.integers(-6, 7, (n, 3))
    q = np.zeros((B, d), np.float32)
    q[:, 3] = np.arange(B)
    vals = rng.integers(0, V, n).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(V), B).astype(np.float32)
    for b, w in enumerate([V - 3, 4100, 17]):  # a p_LM peak in the last, middle and first slice
        p_lm[b, w] += 2.0
    p_lm /= p_lm.sum(1, keepdims=True)
    ko, qo = np.array([0, n]), np.array([0, B])
    prob = _problem(q, k, vals, p_lm, ko, qo, r, 0.05, torch.float32)
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r)
    o_lam = oracle.rrc_lambda(o_d, ALPHA, TAU)
    for drafts in ([V - 1, 0, -1], [4096, V, V - 4]):
        draft = torch.as_tensor(np.array(drafts, np.int32), device="cuda")
        for rep in range(2):
            out = prob.run_nest(ALPHA, TAU, DELTA, draft_tokens=draft)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(out["ids"].cpu().numpy(), o_ids)
            np.testing.assert_array_equal(out["dists"].cpu().numpy().astype(np.float64), o_d)
            np.testing.assert_allclose(out["lambdas"].cpu().numpy().astype(np.float64), o_lam, rtol=0, atol=1e-6)
            ref = oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.05, o_lam)
            np.testing.assert_allclose(out["p_m"].cpu().numpy(), ref, rtol=0, atol=1e-5)
            want = _check_decisions(out, vals, ko, qo, draft)
            assert sorted(set((want["next_token"] // 4096).tolist())) == [0, 1, 2], want["next_token"]
    p_m, ids, dists, lam = prob.run_rrc(ALPHA, TAU)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ids.cpu().numpy(), o_ids)
    np.testing.assert_allclose(p_m.cpu().numpy(), oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.05, o_lam),
                               rtol=0, atol=1e-5)
    p_m, ids, dists = prob.run()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ids.cpu().numpy(), o_ids)
    np.testing.assert_allclose(p_m.cpu().numpy(), oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.05, prob.lam),
                               rtol=0, atol=1e-5)


# (path, keys, queries, r): vocabularies larger than one mixture tile (32768
# entries on the one-workgroup select and the unsliced split finish, 8192 on
# the general select), so that rows are written over several tiles.
LARGE_V_PATHS = [("split-sliced", 40000, 2, 256), ("split-unsliced", 40000, 20, 256),
                 ("one-workgroup", 40000, 40, 256), ("general-r2048", 40000, 3, 2048)]


@pytest.mark.parametrize("V", [50257, 65536])
@pytest.mark.parametrize("path,n,B,r", LARGE_V_PATHS, ids=[p[0] for p in LARGE_V_PATHS])
def test_vocabularies_over_several_tiles(path, n, B, r, V):
    """Fixed-lambda, RRC and NEST steps with V = 50257 (4-byte mixture) and
    65536 (16-byte mixture): ids and distances bit for bit (integer distances),
    p_M to the usual bound, the decoding outputs on the GPU's own rows; drafts
    in the first tile, the last one, and outside [0, V)."""
    _say(f"large vocabulary: {path} V={V}")
    rng = np.random.default_rng(V + B)
    d = 4
    k = np.zeros((n, d), np.float32)
    k[:, :3] = rng.integers(-6, 7, (n, 3))
    q = np.zeros((B, d), np.float32)
    q[:, 3] = np.arange(B) % 6
    vals = rng.integers(0, V, n).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(V), B).astype(np.float32)
    ko, qo = np.array([0, n]), np.array([0, B])
    prob = _problem(q, k, vals, p_lm, ko, qo, r, 0.05, torch.float32)
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r)
    p_m, ids, dists = prob.run()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ids.cpu().numpy(), o_ids)
    np.testing.assert_array_equal(dists.cpu().numpy().astype(np.float64), o_d)
    np.testing.assert_allclose(p_m.cpu().numpy(), oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.05, prob.lam),
                               rtol=0, atol=1e-5)
    o_lam = oracle.rrc_lambda(o_d, ALPHA, TAU)
    ref = oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.05, o_lam)
    p_m, ids, dists, lam = prob.run_rrc(ALPHA, TAU)
    torch.cuda.synchronize()
    np.testing.assert_allclose(lam.cpu().numpy().astype(np.float64), o_lam, rtol=0, atol=1e-6)
    np.testing.assert_allclose(p_m.cpu().numpy(), ref, rtol=0, atol=1e-5)
    draft = torch.as_tensor(np.array([[3, V - 2, V, -5][i % 4] for i in range(B)], np.int32), device="cuda")
    out = prob.run_nest(ALPHA, TAU, DELTA, draft_tokens=draft)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out["ids"].cpu().numpy(), o_ids)
    np.testing.assert_allclose(out["p_m"].cpu().numpy(), ref, rtol=0, atol=1e-5)
    _check_decisions(out, vals, ko, qo, draft)


@pytest.mark.parametrize("B", [32, 33])
def test_split_finish_on_both_sides_of_slicing(B):
    """B queries, each on its own set of 4096 keys (split select, one part a
    row): with 32 the finish takes 8 vocabulary slices a row (256 workgroups),
    with 33 one workgroup a row, the parts kernel writing the fixed-lambda
    dense term.  The fixed-lambda, RRC and NEST steps all match the oracle."""
    _say(f"split finish, B={B}")
    spec = gen.scaled(gen.config("ragged_batch"), B=B, S=B, n_keys=4096, d=256, mu=1 / 16, r=256)
    w = gen.make(spec, 90 + B, device="cuda")
    prob = knn.MixtureProblem(w.queries, w.keys, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu,
                              w.lam, key_offsets_host=w.key_offsets_host, query_offsets_host=w.query_offsets_host)
    p_m, ids, dists = prob.run()
    torch.cuda.synchronize()
    rep = parity.check_workload(w, p_m, ids, dists)
    assert rep.ok(), rep.failures[:5]
    alpha = _median_ratio(w)
    p_m, ids, dists, lam = prob.run_rrc(alpha, TAU)
    torch.cuda.synchronize()
    rep = parity.check_workload(w, p_m, ids, dists, rrc=(alpha, TAU), lambdas=lam)
    assert rep.ok(), rep.failures[:5]
    draft = _drafts(w, B)
    out = prob.run_nest(alpha, TAU, DELTA, draft_tokens=draft)
    torch.cuda.synchronize()
    rep = parity.check_workload(w, out["p_m"], out["ids"], out["dists"], rrc=(alpha, TAU), lambdas=out["lambdas"])
    assert rep.ok(), rep.failures[:5]
    _check_decisions(out, w.values.cpu().numpy(), w.key_offsets_host, w.query_offsets_host, draft)


SYNTH = [
    ("decode-bf16-split", gen.scaled(gen.config("decode_7b"), n_keys=30000, B=2), 81),
    ("ragged-bf16", gen.scaled(gen.config("ragged_batch"), B=12, S=4, n_keys=(1100, 5000, 3333, 2048), r=1024), 82),
    ("batch-f16-mfma", gen.scaled(gen.config("specverify_static"), B=64, S=2, n_keys=(6000, 9000), d=1024,
                                  query_mode="iid"), 83),
    ("decode-bf16-one-workgroup", gen.scaled(gen.config("decode_7b"), n_keys=20000, B=60), 84),
    ("long-row-bf16", gen.scaled(gen.config("decode_7b"), n_keys=80000, B=2, d=512, mu=1 / math.sqrt(512)), 85),
]


def _median_ratio(w):
    ko, qo = w.key_offsets_host, w.query_offsets_host
    ratios = []
    for s in range(len(ko) - 1):
        if qo[s + 1] == qo[s]:
            continue
        kh, dt = oracle.host_elements(w.keys[ko[s]:ko[s + 1]])
        qh, _ = oracle.host_elements(w.queries[qo[s]:qo[s + 1]])
        _, od = oracle.select(qh, kh, dt, np.array([0, len(kh)]), np.array([0, len(qh)]), w.r)
        ratios.extend((od[:, 0] / od[:, -1]).tolist())
    return float(np.median(ratios))


def _drafts(w, seed):
    """Draft tokens: the p_LM argmax on even rows (likely accepted), a seeded token on odd rows."""
    rng = np.random.default_rng(seed)
    d = w.p_lm.argmax(1).to(torch.int32).cpu().numpy()
    d[1::2] = rng.integers(0, w.p_lm.shape[1], d[1::2].shape)
    return torch.as_tensor(d, dtype=torch.int32, device="cuda")


@pytest.mark.parametrize("name,spec,seed", SYNTH, ids=[s[0] for s in SYNTH])
def test_nest_step_synthetic_workloads(name, spec, seed):
    """alpha at the median of the oracle's ratios, so lambda_t straddles delta and
    the span flag takes both values; p_M under P2-P6, decisions exact."""
    _say(f"nest step {name}")
    w = gen.make(spec, seed, device="cuda")
    alpha = _median_ratio(w)
    prob = knn.MixtureProblem(w.queries, w.keys, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu,
                              w.lam, key_offsets_host=w.key_offsets_host, query_offsets_host=w.query_offsets_host)
    draft = _drafts(w, seed)
    out = prob.run_nest(alpha, TAU, DELTA, draft_tokens=draft)
    torch.cuda.synchronize()
    rep = parity.check_workload(w, out["p_m"], out["ids"], out["dists"], rrc=(alpha, TAU), lambdas=out["lambdas"])
    _say(f"{name}: {rep.summary()}")
    assert rep.ok(), rep.failures[:5]
    want = _check_decisions(out, w.values.cpu().numpy(), w.key_offsets_host, w.query_offsets_host, draft)
    _say(f"{name}: use_span {int(want['use_span'].sum())}/{len(want['use_span'])}, "
         f"span found {int((want['span_key'] >= 0).sum())}")
    # the same step without decoding outputs: the same neighbours and lambda_t, p_M up to atomics order
    first = {k: v.clone() for k, v in out.items()}
    p_m2, ids2, d2, lam2 = prob.run_rrc(alpha, TAU)
    torch.cuda.synchronize()
    assert torch.equal(ids2, first["ids"]) and torch.equal(d2, first["dists"])
    assert torch.equal(lam2, first["lambdas"])
    torch.testing.assert_close(p_m2, first["p_m"], rtol=0, atol=1e-7)


GRAPH_CASES = {"decode-20k-keys": lambda: gen.scaled(gen.config("decode_7b"), n_keys=20000, B=2),
               "tiny": lambda: gen.config("tiny")}


@pytest.mark.parametrize("case", list(GRAPH_CASES))
def test_steps_replay_from_graphs(case):
    """The fixed-lambda step and the NEST step (split select from group
    minima, finish in vocabulary slices with its cross-slice maximum and
    count, which the distance stage clears, so no memset) captured in HIP graphs: three rounds of
    replays, with eager steps and synchronisations between and every output
    overwritten before each replay, each equal to the eager results: ids,
    distances and decisions exactly, p_M and the p_M values among the outputs
    up to the order of LDS atomics.  The 4-query fp32 workload is the one the
    benchmark also times as graph replays."""
    _say(f"graph replays {case}")
    w = gen.make(GRAPH_CASES[case](), 87, device="cuda")
    prob = knn.MixtureProblem(w.queries, w.keys, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu,
                              w.lam, key_offsets_host=w.key_offsets_host, query_offsets_host=w.query_offsets_host)
    draft = _drafts(w, 87)
    ref_n = {k: v.clone() for k, v in prob.run_nest(ALPHA, TAU, DELTA, draft_tokens=draft).items()}
    ref_f = [t.clone() for t in prob.run()]
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    g_nest, g_fixed = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_nest, stream=side):
        prob.run_nest(ALPHA, TAU, DELTA, draft_tokens=draft)
    with torch.cuda.graph(g_fixed, stream=side):
        prob.run()
    torch.cuda.synchronize()
    exact = ("ids", "dists", "next_token", "span_key", "use_span", "lambdas")

    def poison():  # every output overwritten before a replay, so each replay must write it again
        for t in (prob.p_m, prob.dists, prob.lambdas, prob.p_max, prob.p_draft):
            t.fill_(float("nan"))
        for t in (prob.ids, prob.next_token, prob.span_key, prob.use_span):
            t.fill_(-7)
        torch.cuda.synchronize()

    for rnd in range(3):
        poison()
        g_nest.replay()
        torch.cuda.synchronize()
        got = {"p_m": prob.p_m, "ids": prob.ids, "dists": prob.dists, "lambdas": prob.lambdas,
               "next_token": prob.next_token, "p_max": prob.p_max, "span_key": prob.span_key,
               "use_span": prob.use_span, "p_draft": prob.p_draft}
        for key, want in ref_n.items():
            if key in exact:
                assert torch.equal(got[key], want), (rnd, key)
            else:
                torch.testing.assert_close(got[key], want, rtol=0, atol=1e-7)
        prob.run()  # eager work between replays
        torch.cuda.synchronize()
        poison()
        g_fixed.replay()
        torch.cuda.synchronize()
        assert torch.equal(prob.ids, ref_f[1]) and torch.equal(prob.dists, ref_f[2]), rnd
        torch.testing.assert_close(prob.p_m, ref_f[0], rtol=0, atol=1e-7)
        prob.run_nest(ALPHA, TAU, DELTA, draft_tokens=draft)
        torch.cuda.synchronize()


def test_spec_verify_hand_cases(golden_dir):
    import json
    import os
    doc = json.load(open(os.path.join(golden_dir, "verify_cases.json")))
    p = np.array(doc["p_m"], np.float32)
    dr = np.array(doc["draft_tokens"])
    dev = "cuda"
    p_max = torch.as_tensor(p.max(1), device=dev)
    p_draft = torch.as_tensor(p[np.arange(len(p)), dr], device=dev)
    nt = torch.as_tensor(np.array(doc["next_token"], np.int32), device=dev)
    offs = torch.as_tensor(np.array(doc["draft_offsets"], np.int64), device=dev)
    for case in doc["cases"]:
        n_acc, tok = knn.spec_verify(p_max, p_draft, nt, offs, case["gamma"])
        torch.cuda.synchronize()
        assert n_acc.cpu().tolist() == case["n_accept"], case
        assert tok.cpu().tolist() == case["token"], case


def test_nest_step_and_verify_on_the_speculative_workload():
    """The speculative-verification workload at full size (8 sequences x 16 draft
    positions over their own 64K-key stores, r = 1024): drafts verified on the
    GPU equal the oracle's decisions on the GPU's rows for several gamma and
    with uniforms; p_M parity on sampled rows."""
    _say("nest step + verify: specverify_seq")
    w = gen.make(gen.config("specverify_seq"), gen.CONFIG_SEEDS["specverify_seq"], device="cuda")
    prob = knn.MixtureProblem(w.queries, w.keys, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu,
                              w.lam, key_offsets_host=w.key_offsets_host, query_offsets_host=w.query_offsets_host)
    draft = _drafts(w, 91)
    masked = np.random.default_rng(92).choice(int(w.key_offsets_host[-1]), 5000, replace=False)
    out = prob.run_nest(ALPHA, TAU, DELTA, key_mask=knn.mask_words(masked, int(w.key_offsets_host[-1]), "cuda"),
                        draft_tokens=draft)
    torch.cuda.synchronize()
    ids = out["ids"].cpu().numpy()
    ko = w.key_offsets_host
    for s in range(len(ko) - 1):
        rows = slice(int(w.query_offsets_host[s]), int(w.query_offsets_host[s + 1]))
        local = masked[(masked >= ko[s]) & (masked < ko[s + 1])] - ko[s]
        assert not np.isin(ids[rows], local).any()
    _check_decisions(out, w.values.cpu().numpy(), w.key_offsets_host, w.query_offsets_host, draft)
    offs = torch.as_tensor(w.query_offsets_host, device="cuda")
    u = np.random.default_rng(93).random(w.spec.B).astype(np.float32)
    for gamma, uni in ((1.0, None), (0.05, None), (5e-4, None), (0.05, u)):
        n_acc, tok = knn.spec_verify(out["p_max"], out["p_draft"], out["next_token"], offs, gamma,
                                     None if uni is None else torch.as_tensor(uni, device="cuda"))
        torch.cuda.synchronize()
        w_acc, w_tok = nest.spec_verify(out["p_max"].cpu().numpy(), out["p_draft"].cpu().numpy(),
                                        out["next_token"].cpu().numpy(), w.query_offsets_host, gamma, uni, fp32=True)
        assert n_acc.cpu().numpy().tolist() == w_acc.tolist(), gamma
        assert tok.cpu().numpy().tolist() == w_tok.tolist(), gamma
    # p_M parity on three rows, with the oracle's masked select
    for b in (0, 37, 127):
        s = int(np.searchsorted(w.query_offsets_host, b, side="right") - 1)
        kh, dt = oracle.host_elements(w.keys[ko[s]:ko[s + 1]])
        qh, _ = oracle.host_elements(w.queries[b:b + 1])
        local = masked[(masked >= ko[s]) & (masked < ko[s + 1])] - ko[s]
        o_ids, o_d = oracle.select(qh, kh, dt, np.array([0, len(kh)]), np.array([0, 1]), w.r,
                                   key_mask=_bits(local, len(kh)))
        rep = parity.Report()
        parity.check_query(rep, b, qh, kh, dt, w.values[ko[s]:ko[s + 1]].cpu().numpy(), w.p_lm[b].cpu().numpy(),
                           w.r, w.mu, w.lam, ids[b], out["dists"][b].cpu().numpy(), out["p_m"][b].cpu().numpy(),
                           oracle_ids=o_ids[0], oracle_dists=o_d[0], rrc=(ALPHA, TAU),
                           gpu_lambda=float(out["lambdas"][b]))
        assert rep.ok(), rep.failures[:3]


def test_nest_step_rejects_bad_arguments():
    _say("nest argument checks")
    rng, q, k, vals, p_lm = _integer_store(100, 1, 4, 1)
    prob = _problem(q, k, vals, p_lm, np.array([0, 100]), np.array([0, 1]), 4, 0.5, torch.float32)
    for alpha, tau, delta in ((0.3, 0.0, 0.5), (float("nan"), 0.1, 0.5), (0.3, 0.1, float("inf"))):
        with pytest.raises(knn.KnnError):
            prob.run_nest(alpha, tau, delta)
    z = torch.zeros(1, device="cuda")
    nt = torch.zeros(1, dtype=torch.int32, device="cuda")
    offs = torch.as_tensor([0, 1], device="cuda")
    for gamma in (0.0, 1.5, float("nan")):
        with pytest.raises(knn.KnnError):
            knn.spec_verify(z, z, nt, offs, gamma)


def test_spec_verify_long_and_empty_drafts():
    """Drafts of 0, 1, 63, 64, 65 and 300 rows (one wave reads 64 rows at a time)
    with p_M(draft) = 0.9 max everywhere but at planted rows (0.1 max): row 0 of
    the 1-row draft, the last row of the 64-row draft, row 64 of the 65-row
    draft, rows 130 and 200 of the 300-row draft.  Exact expected counts at
    gamma = 1 and 0.6; with uniforms the GPU's decisions equal the oracle's in
    fp32."""
    _say("spec verify: long and empty drafts")
    rng = np.random.default_rng(94)
    lens = [0, 1, 63, 64, 65, 300]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    n = int(offs[-1])
    p_max = rng.uniform(0.05, 0.9, n).astype(np.float32)
    f = np.full(n, 0.9, np.float32)
    for dft, row in ((1, 0), (3, 63), (4, 64), (5, 130), (5, 200)):
        f[offs[dft] + row] = 0.1
    p_draft = (p_max * f).astype(np.float32)
    nt = rng.integers(0, 32000, n).astype(np.int32)
    u = rng.random(n).astype(np.float32)
    dev = "cuda"
    t = lambda a: torch.as_tensor(a, device=dev)
    want_acc = [0, 0, 63, 63, 64, 130]
    want_tok = [-1, int(nt[offs[1]]), -1, int(nt[offs[3] + 63]), int(nt[offs[4] + 64]), int(nt[offs[5] + 130])]
    for gamma in (1.0, 0.6):
        n_acc, tok = knn.spec_verify(t(p_max), t(p_draft), t(nt), t(offs), gamma)
        torch.cuda.synchronize()
        assert n_acc.cpu().numpy().tolist() == want_acc, gamma
        assert tok.cpu().numpy().tolist() == want_tok, gamma
    for gamma in (1.0, 0.95):
        n_acc, tok = knn.spec_verify(t(p_max), t(p_draft), t(nt), t(offs), gamma, t(u))
        torch.cuda.synchronize()
        w_acc, w_tok = nest.spec_verify(p_max, p_draft, nt, offs, gamma, u, fp32=True)
        assert n_acc.cpu().numpy().tolist() == w_acc.tolist(), gamma
        assert tok.cpu().numpy().tolist() == w_tok.tolist(), gamma
