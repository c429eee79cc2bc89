"""Parity of the HIP path (through the C ABI) against the CPU oracle on the GPU.

Rules P2-P5 are in tests/parity.py.  Cases: the hand-worked cases, exact
integer inputs (every distance exact, so ids, order and distances must match
the oracle bit for bit), every element type and both load paths, ragged key
sets, planted neighbours, degenerate shapes (r = 1, r = N, r = 4096, all keys
equal, empty query groups), lambda = 1, precomputed key norms and the stage
entry points.  The full-size workloads are in test_gpu_full_size.py.
"""
import gc
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import parity
import select_paths
from workloads import gen

pytestmark = pytest.mark.gpu

knn = pytest.importorskip("paper_2405_19325_amd")


def _say(msg):
    print(f"[gpu] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    knn.load()
    yield
    torch.cuda.synchronize()


def _tensor_inputs(q, k, vals, p_lm, ko, qo, dtype):
    dev = "cuda"
    tq = torch.as_tensor(q).to(dev)
    tk = torch.as_tensor(k).to(dev)
    if dtype != torch.float32:
        tq, tk = tq.to(dtype), tk.to(dtype)
    return (tq.contiguous(), tk.contiguous(), torch.as_tensor(vals, dtype=torch.int32, device=dev),
            torch.as_tensor(ko, dtype=torch.int64, device=dev), torch.as_tensor(qo, dtype=torch.int64, device=dev),
            torch.as_tensor(p_lm, dtype=torch.float32, device=dev))


def _run(w, key_sqnorms=None):
    prob = knn.MixtureProblem(w.queries, w.keys, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu,
                              w.lam, key_sqnorms=key_sqnorms, key_offsets_host=w.key_offsets_host,
                              query_offsets_host=w.query_offsets_host)
    out = prob.run()
    torch.cuda.synchronize()
    return out


def _free():
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


# ------------------------------------------------------------------ hand cases

@pytest.mark.parametrize("which", ["H-A", "H-B"])
def test_hand_cases(golden_dir, which):
    doc = json.load(open(os.path.join(golden_dir, "hand_cases.json")))[which]
    for case in doc["cases"]:
        _say(f"hand case {case['name']}")
        tq, tk, tv, tko, tqo, tp = _tensor_inputs([doc["query"]], doc["keys"], doc["values"], [doc["p_lm"]],
                                                  [0, len(doc["keys"])], [0, 1], torch.float32)
        p_m, ids, dists = knn.mixture(tq.float(), tk.float(), tv, tko, tqo, tp, case["r"], case["mu"], doc["lam"])
        torch.cuda.synchronize()
        assert ids[0].tolist() == case["expect_ids"]
        assert dists[0].tolist() == [float(x) for x in case["expect_dists"]]
        pknn = [float(eval(e, {"__builtins__": {}}, {"exp": math.exp, "sqrt": math.sqrt})) for e in case["pknn_expr"]]
        expect = [doc["lam"] * np.float32(p) + (1 - doc["lam"]) * x for p, x in zip(doc["p_lm"], pknn)]
        np.testing.assert_allclose(p_m[0].cpu().numpy(), expect, rtol=0, atol=1e-6)


# ------------------------------------------------------- exact-integer inputs

@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16, torch.float16])
@pytest.mark.parametrize("d,n,r", [(2, 50, 1), (3, 700, 7), (8, 3000, 64), (64, 5000, 1024), (64, 2100, 2100),
                                   (24, 9000, 300)])
def test_exact_integer_inputs_match_bitwise(dtype, d, n, r):
    _say(f"exact integers dtype={dtype} d={d} n={n} r={r}")
    rng = np.random.default_rng(d * 1000 + n)
    B = 3
    q = rng.integers(-4, 5, (B, d)).astype(np.float32)
    k = rng.integers(-4, 5, (n, d)).astype(np.float32)
    vals = rng.integers(0, 1000, n).astype(np.int32)
    p_lm = np.full((B, 1000), 1e-3, np.float32)
    tq, tk, tv, tko, tqo, tp = _tensor_inputs(q, k, vals, p_lm, [0, n], [0, B], dtype)
    p_m, ids, dists = knn.mixture(tq, tk, tv, tko, tqo, tp, r, 0.05, 0.25)
    torch.cuda.synchronize()
    qh, dt = oracle.host_elements(tq)
    kh, _ = oracle.host_elements(tk)
    oids, odists = oracle.select(qh, kh, dt, np.array([0, n]), np.array([0, B]), r)
    np.testing.assert_array_equal(ids.cpu().numpy(), oids)
    np.testing.assert_array_equal(dists.cpu().numpy().astype(np.float64), odists)
    pm_ref = oracle.mix(oids, odists, vals, np.array([0, n]), np.array([0, B]), p_lm, 0.05, 0.25)
    np.testing.assert_allclose(p_m.cpu().numpy(), pm_ref, rtol=0, atol=1e-6)


def test_all_keys_equal_ties_break_by_index():
    _say("all keys equal")
    n, d, r = 5000, 32, 1000
    k = np.ones((n, d), np.float32)
    q = np.zeros((2, d), np.float32)
    vals = (np.arange(n) % 17).astype(np.int32)
    p_lm = np.full((2, 17), 1 / 17, np.float32)
    tq, tk, tv, tko, tqo, tp = _tensor_inputs(q, k, vals, p_lm, [0, n], [0, 2], torch.bfloat16)
    p_m, ids, dists = knn.mixture(tq, tk, tv, tko, tqo, tp, r, 0.1, 0.5)
    torch.cuda.synchronize()
    assert ids.cpu().numpy().tolist() == [list(range(r))] * 2
    assert torch.all(dists == 32.0)
    counts = np.bincount(vals[:r], minlength=17) / r
    expect = np.broadcast_to(0.5 * np.float32(1 / 17) + 0.5 * counts, (2, 17))
    np.testing.assert_allclose(p_m.cpu().numpy(), expect, atol=1e-6)


# ------------------------------------------------------------ small workloads

SMALL = [
    ("tiny-f32", gen.config("tiny"), 1, None),
    ("decode-bf16-small", gen.scaled(gen.config("decode_7b"), n_keys=20000), 2, None),
    ("ragged-bf16", gen.scaled(gen.config("ragged_batch"), B=12, S=7, n_keys=(1100, 5000, 3333, 2048, 2049, 1024, 7777),
                                r=1024), 3, None),
    ("multi-query-f16", gen.scaled(gen.config("specverify_static"), B=24, S=3, n_keys=(6000, 4000, 9000), d=1024,
                                   query_mode="iid"), 6, None),
    ("odd-d-bf16", gen.scaled(gen.config("decode_7b"), d=1000, n_keys=3001, B=2, r=200, mu=1 / math.sqrt(1000)), 7, None),
    ("odd-d-f32", gen.scaled(gen.config("tiny"), d=37, n_keys=2999, B=5, r=33), 8, None),
    ("d8192-bf16", gen.scaled(gen.config("decode_70b"), B=2, S=2, n_keys=6000), 4, None),
    ("r1", gen.scaled(gen.config("decode_7b"), n_keys=5000, r=1), 9, None),
    ("r4096", gen.scaled(gen.config("decode_7b"), n_keys=9000, r=4096, B=2), 10, None),
    ("planted-bf16", gen.scaled(gen.config("decode_7b"), n_keys=30000, B=3, query_mode="planted"), 12, None),
    # 40 queries per set, but d is no multiple of 128: the streaming kernel, 8 queries per workgroup
    ("batch-f16-d1000", gen.scaled(gen.config("specverify_static"), B=80, S=2, n_keys=(3000, 4500), d=1000,
                                   query_mode="iid", mu=1 / math.sqrt(1000)), 14, None),
    ("empty-sets", gen.scaled(gen.config("decode_7b"), B=3, S=5, n_keys=(3000, 2000, 4000, 2500, 1500), d=512,
                              r=256, mu=1 / math.sqrt(512)), 13, [0, 2, 0, 1, 0]),
]


def _make_small(spec, seed, qps):
    if qps is None:
        return gen.make(spec, seed, device="cuda")
    # a workload whose sets own the given numbers of queries (some own none)
    w = gen.make(spec.replace(B=sum(qps), S=len(qps)), seed, device="cuda")
    qo = np.concatenate([[0], np.cumsum(qps)]).astype(np.int64)
    w.query_offsets_host = qo
    w.query_offsets = torch.as_tensor(qo, device="cuda")
    return w


@pytest.mark.parametrize("name,spec,seed,qps", SMALL, ids=[s[0] for s in SMALL])
def test_small_workloads(name, spec, seed, qps):
    _say(f"workload {name}")
    w = _make_small(spec, seed, qps)
    p_m, ids, dists = _run(w)
    rep = parity.check_workload(w, p_m, ids, dists)
    _say(f"{name}: {rep.summary()}")
    assert rep.ok(), rep.failures[:5]
    if spec.query_mode == "planted":
        assert ids[:, 0].cpu().numpy().tolist() == w.planted_ids.tolist()


@pytest.mark.parametrize("B2", [3, 40])
def test_empty_key_sets_without_queries(B2):
    """Key sets of 0 keys own no query (a set that owns one needs r keys): one
    between two sets and one at the end, whose offset is the total.  With 2 +
    B2 queries the rows take the split (B2 = 3) or the one-workgroup select
    (B2 = 40); ids and distances match the oracle bit for bit (integer
    distances), p_M to the usual bound."""
    _say(f"empty key sets, {2 + B2} queries")
    rng = np.random.default_rng(31 + B2)
    n0, n2, d, r = 3000, 2000, 8, 64
    k = np.zeros((n0 + n2, d), np.float32)
    k[:, :3] = rng.integers(-6, 7, (n0 + n2, 3))
    q = np.zeros((2 + B2, d), np.float32)
    q[:, 3] = np.arange(2 + B2) % 5
    V = 1000
    vals = rng.integers(0, V, n0 + n2).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(V), 2 + B2).astype(np.float32)
    ko = np.array([0, n0, n0, n0 + n2, n0 + n2])
    qo = np.array([0, 2, 2, 2 + B2, 2 + B2])
    dev = "cuda"
    prob = knn.MixtureProblem(torch.as_tensor(q, device=dev), torch.as_tensor(k, device=dev),
                              torch.as_tensor(vals, device=dev), torch.as_tensor(ko, device=dev),
                              torch.as_tensor(qo, device=dev), torch.as_tensor(p_lm, device=dev), r, 0.1, 0.4,
                              key_offsets_host=ko, query_offsets_host=qo)
    p_m, ids, dists = prob.run()
    torch.cuda.synchronize()
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r)
    np.testing.assert_array_equal(ids.cpu().numpy(), o_ids)
    np.testing.assert_array_equal(dists.cpu().numpy().astype(np.float64), o_d)
    np.testing.assert_allclose(p_m.cpu().numpy(), oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.1, 0.4),
                               rtol=0, atol=1e-5)


def test_query_equal_to_key_gives_zero_distance():
    _say("q == k")
    spec = gen.scaled(gen.config("decode_7b"), n_keys=8000, B=4)
    w = gen.make(spec, 21, device="cuda")
    picks = [5, 4000, 7999, 123]
    w.queries = w.keys[picks].clone()
    for norms in (None, knn.key_sqnorms(w.keys)):
        p_m, ids, dists = _run(w, key_sqnorms=norms)
        assert ids[:, 0].cpu().tolist() == picks
        assert torch.all(dists[:, 0] == 0.0)


def test_lambda_one_returns_plm_bitwise():
    _say("lambda = 1")
    w = gen.make(gen.scaled(gen.config("decode_7b"), n_keys=6000, B=2, lam=1.0), 22, device="cuda")
    p_m, _, _ = _run(w)
    assert torch.equal(p_m, w.p_lm)


def test_lambda_zero_is_pknn():
    _say("lambda = 0")
    w = gen.make(gen.scaled(gen.config("tiny"), n_keys=3000, lam=0.0), 23, device="cuda")
    p_m, ids, dists = _run(w)
    rep = parity.check_workload(w, p_m, ids, dists)
    assert rep.ok(), rep.failures[:5]


def test_precomputed_norms_give_identical_results():
    _say("precomputed norms")
    w = gen.make(gen.scaled(gen.config("ragged_batch"), B=4, S=4, n_keys=(3000, 5000, 2000, 4096)), 24, device="cuda")
    _, ids0, d0 = _run(w)
    ids0, d0 = ids0.clone(), d0.clone()
    norms = knn.key_sqnorms(w.keys)
    _, ids1, d1 = _run(w, key_sqnorms=norms)
    assert torch.equal(ids0, ids1) and torch.equal(d0, d1)
    ref = w.keys.float().pow(2).sum(1)
    torch.testing.assert_close(norms, ref, rtol=1e-5, atol=1e-5)


# The key-norm pre-pass against the distance kernel's own norms: the distance from a zero query is
# fma(-2, 0, 0 + ||k||^2) = ||k||^2, bit for bit the norm the kernel made on the fly.  At least 262,144 rows
# of at most 4 KB go to the pre-pass's waves in blocks of 64 (row counts off a multiple of 64, and beyond
# 4096 waves x 64 rows so that waves take several blocks); fewer or longer rows stride one at a time, and
# rows off the 16-byte grid take the element kernel.
NORM_CASES = [(65, 64, torch.float32), (1000, 256, torch.float32), (4097, 2048, torch.bfloat16),
              (300001, 1024, torch.float16), (263000, 512, torch.bfloat16), (333, 8192, torch.bfloat16),
              (777, 100, torch.float32), (501, 330, torch.bfloat16)]


@pytest.mark.parametrize("n,d,dtype", NORM_CASES, ids=[f"{c[0]}x{c[1]}-{str(c[2])[6:]}" for c in NORM_CASES])
def test_norm_prepass_equals_on_the_fly_norms(n, d, dtype):
    _say(f"key-norm pre-pass n={n} d={d} {dtype}")
    g = torch.Generator(device="cuda")
    g.manual_seed(n + d)
    keys = torch.randn((n, d), device="cuda", generator=g).to(dtype)
    norms = knn.key_sqnorms(keys)
    zero = torch.zeros((1, d), dtype=dtype, device="cuda")
    ko, qo = np.array([0, n]), np.array([0, 1])
    on_the_fly = knn.distances(zero, keys, torch.as_tensor(ko, device="cuda"), torch.as_tensor(qo, device="cuda"),
                               key_offsets_host=ko, query_offsets_host=qo)
    torch.cuda.synchronize()
    assert torch.equal(norms, on_the_fly[0])
    ref = keys.double().pow(2).sum(1)
    assert ((norms.double() - ref).abs() / ref).max().item() < 1e-5
    del keys, on_the_fly
    _free()


# Rows of 16 chunks per lane (d = 8192 for 16-bit keys, d = 4096 for fp32) stream in two halves that add
# into one sum; d = 4096 bf16 streams whole rows.  Integer coordinates in both halves of every row make every
# distance an exact integer, so ids and distances must equal the oracle's bit for bit, with the key norms
# computed on the fly or given, and with a third of the keys masked (a NEST step).
HALF_ROWS = [("bf16-d8192", torch.bfloat16, 8192), ("f32-d4096", torch.float32, 4096), ("bf16-d4096", torch.bfloat16, 4096)]


@pytest.mark.parametrize("masked", [False, True], ids=["unmasked", "masked"])
@pytest.mark.parametrize("norms", [False, True], ids=["norms-on-the-fly", "norms-given"])
@pytest.mark.parametrize("name,dtype,d", HALF_ROWS, ids=[h[0] for h in HALF_ROWS])
def test_streamed_row_halves_exact_integers(name, dtype, d, norms, masked):
    _say(f"row halves: {name} norms={norms} masked={masked}")
    n, B, r = 5000, 3, 64
    rng = np.random.default_rng(97 + d)
    cols = [0, 1, 2, d // 2 + 3, d - 1000, d - 1]  # both halves of the row (and the last chunk)
    k = np.zeros((n, d), np.float32)
    k[:, cols] = rng.integers(-3, 4, (n, len(cols)))
    q = np.zeros((B, d), np.float32)
    q[:, cols] = rng.integers(-3, 4, (B, len(cols)))
    vals = rng.integers(0, 500, n).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(500), B).astype(np.float32)
    ko, qo = np.array([0, n]), np.array([0, B])
    tq, tk, tv, tko, tqo, tp = _tensor_inputs(q, k, vals, p_lm, ko, qo, dtype)
    kn = knn.key_sqnorms(tk) if norms else None
    prob = knn.MixtureProblem(tq, tk, tv, tko, tqo, tp, r, 0.05, 0.5, key_sqnorms=kn, key_offsets_host=ko,
                              query_offsets_host=qo)
    words = None
    if masked:
        rows = rng.choice(n, n // 3, replace=False)
        words = np.zeros((n + 31) // 32, np.uint32)
        np.bitwise_or.at(words, rows >> 5, (np.uint32(1) << (rows & 31).astype(np.uint32)))
        out = prob.run_nest(0.3, 0.1, 0.5, key_mask=knn.mask_words(rows, n, "cuda"))
        ids, dists = out["ids"], out["dists"]
    else:
        _, ids, dists = prob.run()
    torch.cuda.synchronize()
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r, key_mask=words)
    np.testing.assert_array_equal(ids.cpu().numpy(), o_ids)
    np.testing.assert_array_equal(dists.cpu().numpy().astype(np.float64), o_d)
    if norms:
        np.testing.assert_array_equal(kn.cpu().numpy().astype(np.float64), (k.astype(np.float64) ** 2).sum(1))
    del tk, prob
    _free()


def test_element_path_matches_vector_path_bitwise():
    """A key matrix that is not 16-byte aligned takes the element-load path; the
    accumulation order is the same, so every output bit is the same."""
    _say("element vs vector path")
    w = gen.make(gen.scaled(gen.config("decode_7b"), n_keys=5000, B=2, d=512, mu=1 / math.sqrt(512)), 25, device="cuda")
    _, ids0, d0 = _run(w)
    ids0, d0 = ids0.clone(), d0.clone()
    buf = torch.empty(w.keys.numel() + 1, dtype=w.keys.dtype, device="cuda")
    shifted = buf[1:].view(w.keys.shape)
    shifted.copy_(w.keys)
    assert shifted.data_ptr() % 16 != 0
    w.keys = shifted
    _, ids1, d1 = _run(w)
    assert torch.equal(ids0, ids1) and torch.equal(d0, d1)


def test_stages_equal_whole_call_and_repeat_deterministically():
    _say("stages vs whole call")
    w = gen.make(gen.scaled(gen.config("ragged_batch"), B=6, S=3, n_keys=(4000, 6000, 3000)), 26, device="cuda")
    prob = knn.MixtureProblem(w.queries, w.keys, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu,
                              w.lam, key_offsets_host=w.key_offsets_host, query_offsets_host=w.query_offsets_host)
    prob.run()
    torch.cuda.synchronize()
    ids0, d0, pm0 = prob.ids.clone(), prob.dists.clone(), prob.p_m.clone()
    for parts in (("distances", "select", "mix"), ("distances", "select_mix")):
        prob.ids.zero_()
        prob.p_m.zero_()
        for part in parts:
            prob.run_part(part)
        torch.cuda.synchronize()
        assert torch.equal(ids0, prob.ids) and torch.equal(d0, prob.dists)
        torch.testing.assert_close(pm0, prob.p_m, rtol=0, atol=1e-7)


def test_distance_matrix_entry_point():
    _say("knn_distances")
    w = gen.make(gen.scaled(gen.config("ragged_batch"), B=5, S=2, n_keys=(1000, 1500), d=256, mu=1 / 16), 27,
                 device="cuda")
    D = knn.distances(w.queries, w.keys, w.key_offsets, w.query_offsets, key_offsets_host=w.key_offsets_host,
                      query_offsets_host=w.query_offsets_host).cpu().numpy()
    ko, qo = w.key_offsets_host, w.query_offsets_host
    for s in range(2):
        kh, dt = oracle.host_elements(w.keys[ko[s]:ko[s + 1]])
        qh, _ = oracle.host_elements(w.queries[qo[s]:qo[s + 1]])
        ref = oracle.sqdist(qh, kh, dt)
        got = D[qo[s]:qo[s + 1], :ko[s + 1] - ko[s]]
        np.testing.assert_allclose(got, ref, rtol=1e-5, atol=2e-4)
        assert np.all(np.isnan(D[qo[s]:qo[s + 1], ko[s + 1] - ko[s]:]))


def test_mix_entry_point():
    _say("knn_mix")
    rng = np.random.default_rng(28)
    B, n, r, V = 3, 500, 100, 9000
    ids = np.stack([rng.permutation(n)[:r] for _ in range(B)]).astype(np.int32)
    dists = rng.uniform(10, 20, (B, r)).astype(np.float32)
    vals = rng.integers(0, V, n).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(V), B).astype(np.float32)
    ko, qo = np.array([0, n]), np.array([0, B])
    dev = "cuda"
    out = knn.mix(torch.as_tensor(ids, device=dev), torch.as_tensor(dists, device=dev),
                  torch.as_tensor(vals, device=dev), torch.as_tensor(ko, device=dev), torch.as_tensor(qo, device=dev),
                  torch.as_tensor(p_lm, device=dev), 0.3, 0.4)
    ref = oracle.mix(ids, dists.astype(np.float64), vals, ko, qo, p_lm, 0.3, 0.4)
    np.testing.assert_allclose(out.cpu().numpy(), ref, rtol=0, atol=1e-6)


def test_split_and_one_workgroup_select_agree():
    """The same queries through the split select (few queries: a 64K-key row
    over 16 workgroups) and the one-workgroup select (20 queries): the same
    neighbours and distances bit for bit, p_M within the rounding of the LDS
    atomics.  fp32 keys keep both batches on the streaming distance kernel,
    whose per-query arithmetic does not depend on the batch."""
    _say("split vs one-workgroup select")
    w = gen.make(gen.scaled(gen.config("decode_7b"), B=20, n_keys=65536, d=256, dtype="f32", mu=1 / 16), 29,
                 device="cuda")
    _, ids20, d20 = _run(w)
    p20 = _run(w)[0].clone()
    ids20, d20 = ids20.clone(), d20.clone()
    qo = np.array([0, 3], np.int64)
    prob = knn.MixtureProblem(w.queries[:3].contiguous(), w.keys, w.values, w.key_offsets,
                              torch.as_tensor(qo, device="cuda"), w.p_lm[:3].contiguous(), w.r, w.mu, w.lam,
                              key_offsets_host=w.key_offsets_host, query_offsets_host=qo)
    p3, ids3, d3 = prob.run()
    torch.cuda.synchronize()
    assert torch.equal(ids3, ids20[:3]) and torch.equal(d3, d20[:3])
    torch.testing.assert_close(p3, p20[:3], rtol=0, atol=1e-7)


def _sampled_positions(path, n):
    """Key positions whose distances the sampled threshold of each select path reads."""
    if path in ("parts", "groups"):  # parts kernel: 1024 runs of 4 consecutive keys, one every n / 1024 (at a multiple of 4)
        starts = ((np.arange(1024, dtype=np.int64) * n) >> 10) & ~3
        return (starts[:, None] + np.arange(4)).ravel()
    t = np.arange(1024)
    return (t & 15) * 4096 + 4 * t + ((t >> 4) & 3)  # one-workgroup path: a key per thread's registers


# (path, queries, V) on one 64K-key set of width 16: the split select over 16 workgroups per row, from the
# parts kernel's sample (two queries and a vocabulary too large for the sliced finish) or from the distance
# stage's group minima (one query), and 20 queries (too many parts for one pass of the chip, so one
# workgroup per query).
SAMPLED_PATHS = [("parts", 2, 600001), ("groups", 1, 50), ("one-workgroup", 20, 50)]


def _check_path(path, B, n, d, r, V):
    if path != "one-workgroup":
        assert select_paths.split_path(B, d, 2, 1, n, B, r, V) == path


@pytest.mark.parametrize("path,B,V", SAMPLED_PATHS, ids=[c[0] for c in SAMPLED_PATHS])
def test_adversarial_row_takes_the_streamed_path(path, B, V):
    """Keys at the positions the parts kernel and the one-workgroup select
    sample are far away and every other key sits on the query: their sampled
    threshold then keeps more than the candidate capacity.  On the group
    minima every group holds keys at distance 0, so every minimum is 0 and
    every group is listed, more than the list holds.  Either way the streamed
    path over the whole row takes over, and the answer (ties broken by index)
    is still exact."""
    _say(f"adversarial sample ({path})")
    n, d, r = 65536, 16, 1000
    _check_path(path, B, n, d, r, V)
    sampled = _sampled_positions(path, n)
    k = np.zeros((n, d), np.float32)
    k[sampled] = 3.0
    q = np.zeros((B, d), np.float32)
    vals = (np.arange(n) % 50).astype(np.int32)
    p_lm = np.zeros((B, V), np.float32)
    p_lm[:, :50] = 0.02
    tq, tk, tv, tko, tqo, tp = _tensor_inputs(q, k, vals, p_lm, [0, n], [0, B], torch.bfloat16)
    p_m, ids, dists = knn.mixture(tq, tk, tv, tko, tqo, tp, r, 0.1, 0.5)
    torch.cuda.synchronize()
    expect = np.setdiff1d(np.arange(n), sampled)[:r]
    for b in range(B):
        assert ids[b].cpu().numpy().tolist() == expect.tolist()
    assert torch.all(dists == 0.0)
    # every neighbour is at distance 0: equal weights 1/r on tokens i % 50
    counts = np.bincount(vals[expect], minlength=50).astype(np.float64)
    want = 0.5 * 0.02 + 0.5 * counts / r
    pm = p_m.cpu().numpy()
    np.testing.assert_allclose(pm[:, :50], np.broadcast_to(want, (B, 50)), rtol=0, atol=1e-6)
    assert not pm[:, 50:].any()


FEWER_PATHS = [c for c in SAMPLED_PATHS if c[0] != "groups"]  # at least r groups, hence keys, lie below theirs


@pytest.mark.parametrize("path,B,V", FEWER_PATHS, ids=[c[0] for c in FEWER_PATHS])
def test_sample_keeps_fewer_than_r_takes_the_streamed_path(path, B, V):
    """The keys at the sampled positions are the nearest of the row, at many
    different distances, and every other key is far away: the sampled
    threshold then keeps about a hundred keys, fewer than r, and the streamed
    select over the whole row must take over.  Small integer entries make
    every distance exact, so ids and distances equal the oracle's bit for bit."""
    _say(f"sample keeps fewer than r ({path})")
    n, d, r = 65536, 16, 1000
    _check_path(path, B, n, d, r, V)
    sampled = _sampled_positions(path, n)
    j = np.arange(sampled.size)
    k = np.full((n, d), 100.0, np.float32)
    k[sampled] = 0.0
    k[sampled, 0] = 1 + j % 60
    k[sampled, 1] = j // 60
    q = np.zeros((B, d), np.float32)
    rng = np.random.default_rng(97)
    vals = rng.integers(0, 50, n).astype(np.int32)
    p_lm = np.zeros((B, V), np.float32)
    p_lm[:, :50] = 0.02
    tq, tk, tv, tko, tqo, tp = _tensor_inputs(q, k, vals, p_lm, [0, n], [0, B], torch.bfloat16)
    p_m, ids, dists = knn.mixture(tq, tk, tv, tko, tqo, tp, r, 0.1, 0.5)
    torch.cuda.synchronize()
    qh, dt = oracle.host_elements(tq)
    kh, _ = oracle.host_elements(tk)
    oids, odists = oracle.select(qh, kh, dt, np.array([0, n]), np.array([0, B]), r)
    assert np.isin(oids, sampled).all()  # the answer lies among the samples
    np.testing.assert_array_equal(ids.cpu().numpy(), oids)
    np.testing.assert_array_equal(dists.cpu().numpy().astype(np.float64), odists)
    ref = oracle.mix(oids, odists, vals, np.array([0, n]), np.array([0, B]), p_lm, 0.1, 0.5)
    np.testing.assert_allclose(p_m.cpu().numpy(), ref, rtol=0, atol=1e-5)


# (case, V) over two layouts, each with a mixture whose finish is sliced by 4096-entry pieces of p_M:
# "one-set": 40,000 keys of width 4 and two queries, the split select from the group minima (ten parts per
# row, 16-row distance tiles); "32-sets": 32 sets of 4096 keys with a query each, the split select from the
# parts kernel's sample (64-row distance tiles record no group minima).  V = 10001 takes the mixture's
# scalar path, V = 32000 its 16-byte path.
SPLIT_SLICED = [("threshold", 32000), ("threshold", 10001), ("all-equal", 32000)]


@pytest.mark.parametrize("layout", ["one-set", "32-sets"])
@pytest.mark.parametrize("case,V", SPLIT_SLICED, ids=[f"{c}-V{v}" for c, v in SPLIT_SLICED])
@pytest.mark.parametrize("rrc", [False, True], ids=["fixed-lambda", "rrc"])
def test_split_select_sliced_finish_exact_integers(case, V, rrc, layout):
    """Integer keys (a, b, c, 0) with a, b, c in [-60, 60] give exact distances in many distinct values, so the
    threshold keeps somewhat more than r keys.  With every key equal, the group minima list every group, more
    than the list holds, and the finish falls back to the streamed select; the parts kernel's threshold keeps
    each whole 4096-key row, which the finish still sorts (ties by index).  ids and distances bit for bit
    against the oracle, p_M within 1e-5 (with RRC, lambda_t within 1e-6)."""
    _say(f"split select, sliced finish: {layout}, {case}, V={V}, rrc={rrc}")
    rng = np.random.default_rng(98)
    d = 4
    if layout == "one-set":
        n, B, r = 40000, 2, 1024
        ko, qo = np.array([0, n]), np.array([0, B])
        q = np.zeros((B, d), np.float32)
        q[:, 3] = [2, 5]
        q[1, 0] = 7
    else:
        B, r = 32, 256
        n = 4096 * B
        ko, qo = np.arange(B + 1) * 4096, np.arange(B + 1)
        q = np.zeros((B, d), np.float32)
        q[:, :3] = rng.integers(-30, 31, (B, 3))
        q[:, 3] = np.arange(B) % 5
    sizes = np.diff(ko)
    assert select_paths.split_path(B, d, 4, len(sizes), int(sizes.max()), int(np.diff(qo).max()), r, V) == (
        "groups" if layout == "one-set" else "parts")
    k = np.zeros((n, d), np.float32)
    if case != "all-equal":
        k[:, :3] = rng.integers(-60, 61, (n, 3))
    vals = rng.integers(0, V, n).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(V), B).astype(np.float32)
    tq, tk, tv, tko, tqo, tp = _tensor_inputs(q, k, vals, p_lm, ko, qo, torch.float32)
    prob = knn.MixtureProblem(tq, tk, tv, tko, tqo, tp, r, 0.05, 0.4, key_offsets_host=ko, query_offsets_host=qo)
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r)
    if rrc:
        p_m, ids, dists, lam_t = prob.run_rrc(0.3, 0.1)
        torch.cuda.synchronize()
        lam = oracle.rrc_lambda(o_d, 0.3, 0.1)
        np.testing.assert_allclose(lam_t.cpu().numpy().astype(np.float64), lam, rtol=0, atol=1e-6)
    else:
        p_m, ids, dists = prob.run()
        torch.cuda.synchronize()
        lam = 0.4
    np.testing.assert_array_equal(ids.cpu().numpy(), o_ids)
    np.testing.assert_array_equal(dists.cpu().numpy().astype(np.float64), o_d)
    ref = oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.05, lam)
    np.testing.assert_allclose(p_m.cpu().numpy(), ref, rtol=0, atol=1e-5)


# ------------------------------------------------- matrix-core (query batch) path

MFMA = [
    ("mfma-16q-bf16", gen.scaled(gen.config("specverify_seq"), B=16, S=1, n_keys=5000, d=1024,
                                 mu=1 / 32), 31),
    ("mfma-40q-2sets-f16-d1152", gen.scaled(gen.config("specverify_static"), B=80, S=2, n_keys=(3000, 4500), d=1152,
                                            query_mode="iid", mu=1 / math.sqrt(1152)), 32),
    ("mfma-d128-one-span", gen.scaled(gen.config("specverify_static"), B=32, S=1, n_keys=2900, d=128,
                                      query_mode="iid", mu=1 / math.sqrt(128), r=300), 36),
    ("mfma-130q-bf16-groups", gen.scaled(gen.config("specverify_seq"), B=130, S=1, n_keys=3001, d=256, mu=1 / 16,
                                         r=700), 33),
    ("mfma-ragged-sets", gen.scaled(gen.config("specverify_seq"), B=51, S=3, n_keys=(2048, 1300, 4100), d=512,
                                    mu=1 / math.sqrt(512), r=512), 34),
    ("mfma-d8192", gen.scaled(gen.config("specverify_seq"), B=16, S=1, n_keys=1500, r=256), 35),
]


@pytest.mark.parametrize("name,spec,seed", MFMA, ids=[m[0] for m in MFMA])
def test_matrix_core_workloads(name, spec, seed):
    _say(f"workload {name}")
    w = gen.make(spec, seed, device="cuda")
    p_m, ids, dists = _run(w)
    rep = parity.check_workload(w, p_m, ids, dists)
    _say(f"{name}: {rep.summary()}")
    assert rep.ok(), rep.failures[:5]
    norms = knn.key_sqnorms(w.keys)
    p_m2, ids2, dists2 = _run(w, key_sqnorms=norms)
    rep2 = parity.check_workload(w, p_m2, ids2, dists2)
    assert rep2.ok(), rep2.failures[:5]


# (queries, d): 37 queries take one 64-query group of 128-key passes of 128-element spans; 130 queries take
# two 128-query groups (the second holding 2) of 256-key passes of 64-element spans, and d = 640 gives tiles
# of 1792 rows (7 such passes), the last tile of the row partial.
MFMA_EXACT = [(37, 256), (130, 640)]


@pytest.mark.parametrize("B,d", MFMA_EXACT, ids=[f"{b}q-d{d}" for b, d in MFMA_EXACT])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
def test_matrix_core_exact_integers(dtype, B, d):
    """Integer queries and keys in [-4, 4]: every dot product and norm is exact in fp32, so the matrix-core
    path must give the oracle's ids and distances bit for bit."""
    _say(f"matrix-core exact integers {dtype} B={B} d={d}")
    rng = np.random.default_rng(41 + d)
    n, r = 3000, 300
    q = rng.integers(-4, 5, (B, d)).astype(np.float32)
    k = rng.integers(-4, 5, (n, d)).astype(np.float32)
    vals = rng.integers(0, 500, n).astype(np.int32)
    p_lm = np.full((B, 500), 1 / 500, np.float32)
    tq, tk, tv, tko, tqo, tp = _tensor_inputs(q, k, vals, p_lm, [0, n], [0, B], dtype)
    p_m, ids, dists = knn.mixture(tq, tk, tv, tko, tqo, tp, r, 0.05, 0.25)
    torch.cuda.synchronize()
    qh, dt = oracle.host_elements(tq)
    kh, _ = oracle.host_elements(tk)
    oids, odists = oracle.select(qh, kh, dt, np.array([0, n]), np.array([0, B]), r)
    np.testing.assert_array_equal(ids.cpu().numpy(), oids)
    np.testing.assert_array_equal(dists.cpu().numpy().astype(np.float64), odists)


# ------------------------------------------------ wide select (long rows, fine tiles)

@pytest.mark.parametrize("case", ["threshold", "all-equal-fallback", "masked-nest-step"])
def test_wide_select_exact_integers(case):
    """Rows of 600,000 fp32 keys of width 1024 (256-row distance tiles: 2,344
    tiles, at least 2 r), two queries: the select is cut into parts with a
    threshold from the tile minima.  Integer keys (a, b, c, 0, ...) give exact
    distances, so ids and distances must equal the oracle's bit for bit.  With
    every key equal the threshold keeps the whole row and the finish falls
    back to the streamed select (ties by index); with a third of the keys
    masked (a NEST step) the masked tiles' minima stay out of the threshold."""
    _say(f"wide select: {case}")
    n, d, B, r = 600000, 1024, 2, 1024
    rng = np.random.default_rng(95)
    k = np.zeros((n, d), np.float32)
    if case != "all-equal-fallback":
        k[:, :3] = rng.integers(-6, 7, (n, 3))
    q = np.zeros((B, d), np.float32)
    q[:, 3] = [1, 4]
    vals = rng.integers(0, 300, n).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(300), B).astype(np.float32)
    ko, qo = np.array([0, n]), np.array([0, B])
    tq, tk, tv, tko, tqo, tp = _tensor_inputs(q, k, vals, p_lm, ko, qo, torch.float32)
    if case == "masked-nest-step":
        masked = rng.choice(n, n // 3, replace=False)
        words = np.zeros((n + 31) // 32, np.uint32)
        np.bitwise_or.at(words, masked >> 5, (np.uint32(1) << (masked & 31).astype(np.uint32)))
        prob = knn.MixtureProblem(tq, tk, tv, tko, tqo, tp, r, 0.05, key_offsets_host=ko, query_offsets_host=qo)
        out = prob.run_nest(0.3, 0.1, 0.5, key_mask=knn.mask_words(masked, n, "cuda"))
        torch.cuda.synchronize()
        p_m, ids, dists = out["p_m"], out["ids"], out["dists"]
        o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r, key_mask=words)
        lam = oracle.rrc_lambda(o_d, 0.3, 0.1)
        np.testing.assert_allclose(out["lambdas"].cpu().numpy().astype(np.float64), lam, rtol=0, atol=1e-6)
    else:
        p_m, ids, dists = knn.mixture(tq, tk, tv, tko, tqo, tp, r, 0.05, 0.5)
        torch.cuda.synchronize()
        o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r)
        lam = 0.5
    np.testing.assert_array_equal(ids.cpu().numpy(), o_ids)
    np.testing.assert_array_equal(dists.cpu().numpy().astype(np.float64), o_d)
    ref = oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.05, lam)
    np.testing.assert_allclose(p_m.cpu().numpy(), ref, rtol=0, atol=1e-5)
    del tk
    _free()


def test_wide_select_many_queries_chunked_tile_scan():
    """1,024 queries over one set of 600,000 fp32 keys of width 1024: 2,344
    distance tiles of 256 rows and two select parts per query, so a part lists
    its tiles with keys below the threshold in two chunks of at most 1,024
    tiles and streams only those.  Keys (a, b, c, 0, ...) with a, b, c in
    [-6, 6] and queries (0, 0, 0, c, 0, ...) give exact integer distances;
    the oracle runs on the four leading columns, which give the same values."""
    _say("wide select: 1024 queries, chunked tile scan")
    n, d, B, r = 600000, 1024, 1024, 1024
    rng = np.random.default_rng(96)
    k4 = np.zeros((n, 4), np.float32)
    k4[:, :3] = rng.integers(-6, 7, (n, 3))
    q4 = np.zeros((B, 4), np.float32)
    q4[:, 3] = np.arange(B) % 5
    vals = rng.integers(0, 300, n).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(300), B).astype(np.float32)
    ko, qo = np.array([0, n]), np.array([0, B])
    tk = torch.zeros((n, d), dtype=torch.float32, device="cuda")
    tk[:, :4] = torch.as_tensor(k4, device="cuda")
    tq = torch.zeros((B, d), dtype=torch.float32, device="cuda")
    tq[:, :4] = torch.as_tensor(q4, device="cuda")
    _, _, tv, tko, tqo, tp = _tensor_inputs(q4, k4[:1], vals, p_lm, ko, qo, torch.float32)
    p_m, ids, dists = knn.mixture(tq, tk, tv, tko, tqo, tp, r, 0.05, 0.5)
    torch.cuda.synchronize()
    o_ids, o_d = oracle.select(q4, k4, "f32", ko, qo, r)
    np.testing.assert_array_equal(ids.cpu().numpy(), o_ids)
    np.testing.assert_array_equal(dists.cpu().numpy().astype(np.float64), o_d)
    ref = oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.05, 0.5)
    np.testing.assert_allclose(p_m.cpu().numpy(), ref, rtol=0, atol=1e-5)
    del tk, tq, p_m
    _free()
