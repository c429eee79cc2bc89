"""The split select from group minima (no parts kernel) against the oracle.

With few queries on rows of at most 64 Ki keys served by the streaming
distance kernels in 16- or 32-row tiles, each of a tile's four waves records
the smallest distance of the rows it took (every fourth row of the tile: a
group of 4 or 8 keys).
The finish then takes as threshold the end of the histogram bin holding the
r-th smallest group minimum, lists the groups below it and sorts the keys
below it; a row whose listed groups or keys overflow its buffers falls back
to the streamed select.  Integer keys make every distance exact, so ids and
distances must equal the oracle's bit for bit; p_M is within 1e-5.  Cases:
groups of 4 and 8 keys, rows that end inside a group, whole groups masked,
the nearest keys packed into a few groups, one near key in every group, the
smallest r the rule admits, the fallback, and the same rows through the
parts kernel (a vocabulary too large for the sliced finish).
"""
import numpy as np
import pytest
import torch

import oracle
import select_paths
from oracle import nest

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


def _mask_bits(masked, n):
    words = np.zeros((n + 31) // 32, np.uint32)
    for i in masked:
        words[i >> 5] |= np.uint32(1) << np.uint32(i & 31)
    return words


def _store(sizes, qps, d, V, seed, spread=60):
    """Integer keys (a, b, c, 0, ...) with a, b, c in [-spread, spread] and queries (x, 0, 0, c, 0, ...)."""
    rng = np.random.default_rng(seed)
    n = int(sum(sizes))
    k = np.zeros((n, d), np.float32)
    k[:, :3] = rng.integers(-spread, spread + 1, (n, 3))
    B = int(sum(qps))
    q = np.zeros((B, d), np.float32)
    q[:, 3] = 1 + np.arange(B) % 5
    q[:, 0] = np.arange(B) % 7 - 3
    vals = rng.integers(0, V, n).astype(np.int32)
    p_lm = rng.dirichlet(np.ones(V), B).astype(np.float32)
    ko = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    qo = np.concatenate([[0], np.cumsum(qps)]).astype(np.int64)
    return rng, q, k, vals, p_lm, ko, qo


def _problem(q, k, vals, p_lm, ko, qo, r, mu, lam, dtype):
    dev = "cuda"
    tq, tk = torch.as_tensor(q, device=dev).to(dtype), torch.as_tensor(k, device=dev).to(dtype)
    return knn.MixtureProblem(tq.contiguous(), tk.contiguous(), torch.as_tensor(vals, device=dev),
                              torch.as_tensor(ko, device=dev), torch.as_tensor(qo, device=dev),
                              torch.as_tensor(p_lm, device=dev), r, mu, lam, key_offsets_host=ko,
                              query_offsets_host=qo)


def _path(q, k, ko, qo, r, V, esize):
    sizes, qps = np.diff(ko), np.diff(qo)
    return select_paths.split_path(q.shape[0], k.shape[1], esize, len(sizes), int(sizes.max()), int(qps.max()), r, V)


def _check_select(ids, dists, o_ids, o_d):
    np.testing.assert_array_equal(ids.cpu().numpy(), o_ids)
    np.testing.assert_array_equal(dists.cpu().numpy().astype(np.float64), o_d)


def _check_all_modes(prob, q, k, vals, p_lm, ko, qo, r, mu, lam, masked=None):
    """Fixed lambda, RRC and (with the mask) a NEST step, each against the oracle."""
    n = k.shape[0]
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r)
    p_m, ids, dists = prob.run()
    torch.cuda.synchronize()
    _check_select(ids, dists, o_ids, o_d)
    np.testing.assert_allclose(p_m.cpu().numpy(), oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, mu, lam),
                               rtol=0, atol=1e-5)
    p_m, ids, dists, lam_t = prob.run_rrc(ALPHA, TAU)
    torch.cuda.synchronize()
    _check_select(ids, dists, o_ids, o_d)
    o_lam = oracle.rrc_lambda(o_d, ALPHA, TAU)
    np.testing.assert_allclose(lam_t.cpu().numpy().astype(np.float64), o_lam, rtol=0, atol=1e-6)
    np.testing.assert_allclose(p_m.cpu().numpy(), oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, mu, o_lam),
                               rtol=0, atol=1e-5)
    if masked is None:
        return
    draft = torch.as_tensor(p_lm.argmax(1).astype(np.int32), device="cuda")
    out = prob.run_nest(ALPHA, TAU, DELTA, key_mask=knn.mask_words(masked, n, "cuda"), draft_tokens=draft)
    torch.cuda.synchronize()
    m_ids, m_d = oracle.select(q, k, "f32", ko, qo, r, key_mask=_mask_bits(masked, n))
    _check_select(out["ids"], out["dists"], m_ids, m_d)
    ids = out["ids"].cpu().numpy()  # local key indices of each row's own set
    row_set = np.searchsorted(qo, np.arange(ids.shape[0]), side="right") - 1
    glob = np.where(ids >= 0, ids + ko[row_set][:, None], -1)
    assert not np.isin(glob, masked).any()
    m_lam = oracle.rrc_lambda(m_d, ALPHA, TAU)
    np.testing.assert_allclose(out["p_m"].cpu().numpy(), oracle.mix(m_ids, m_d, vals, ko, qo, p_lm, mu, m_lam),
                               rtol=0, atol=1e-5)
    pm = out["p_m"].cpu().numpy()
    want = nest.decode_outputs(pm, out["ids"].cpu().numpy(), vals, ko, qo, out["lambdas"].cpu().numpy(), DELTA,
                               draft.cpu().numpy())
    for key in ("next_token", "span_key", "use_span"):
        assert out[key].cpu().numpy().tolist() == want[key].tolist(), key
    assert np.array_equal(out["p_max"].cpu().numpy(), want["p_max"])
    assert np.array_equal(out["p_draft"].cpu().numpy(), want["p_draft"])


# (name, key set sizes, queries per set, d, r, V, group rows): rows that end inside a group, two sets of
# different lengths, groups of 8 (32-row tiles) and of 4 (16-row tiles), V on the 16-byte and scalar
# mixture paths.
GROUP_CASES = [
    ("g8-two-sets", (40001, 33333), (2, 1), 16, 1024, 32000, 8),
    ("g4-two-sets", (20001, 17003), (1, 2), 16, 1024, 10001, 4),
    ("g8-r-small", (65536,), (1,), 24, 100, 5000, 8),
    ("g4-r-at-the-limit", (4093,), (3,), 16, 512, 3001, 4),
]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("name,sizes,qps,d,r,V,gr", GROUP_CASES, ids=[c[0] for c in GROUP_CASES])
def test_group_select_exact_integers(name, sizes, qps, d, r, V, gr, dtype):
    _say(f"group-minima select {name} {dtype}")
    esize = 4 if dtype == torch.float32 else 2
    rng, q, k, vals, p_lm, ko, qo = _store(sizes, qps, d, V, 300 + r + d)
    assert _path(q, k, ko, qo, r, V, esize) == "groups"
    assert select_paths.group_rows(q.shape[0], d, esize, len(sizes), max(sizes), max(qps), r) == gr
    n = k.shape[0]
    # a third of the keys and two whole runs of 64 rows (every group in them) masked
    masked = np.union1d(rng.choice(n, n // 3, replace=False), np.r_[128:192, ko[1] - 64:ko[1]])
    prob = _problem(q, k, vals, p_lm, ko, qo, r, 0.05, 0.4, dtype)
    _check_all_modes(prob, q, k, vals, p_lm, ko, qo, r, 0.05, 0.4, masked)


@pytest.mark.parametrize("layout", ["nearest-in-few-groups", "one-near-key-per-group"])
def test_group_select_planted_neighbours(layout):
    """The r nearest keys fill the first r / 8 groups (the threshold then lies among the far groups' minima
    and the finish sorts about twice r keys), or every group holds one near key (only those are listed)."""
    _say(f"group-minima select, {layout}")
    n, d, r, V = 65536, 16, 1024, 32000
    rng, q, k, vals, p_lm, ko, qo = _store((n,), (2,), d, V, 321, spread=40)
    k[:, :3] += 100  # far: every coordinate at least 60 from the query
    if layout == "nearest-in-few-groups":
        near = np.arange(r)
    else:  # rows 32 t + 9 i, i < 4: one in each of the four groups of every 32-row tile
        near = (32 * np.arange(n // 32)[:, None] + 9 * np.arange(4)).ravel()
    k[near, :3] = rng.integers(-20, 21, (near.size, 3))
    assert _path(q, k, ko, qo, r, V, 4) == "groups"
    prob = _problem(q, k, vals, p_lm, ko, qo, r, 0.05, 0.4, torch.float32)
    _check_all_modes(prob, q, k, vals, p_lm, ko, qo, r, 0.05, 0.4)
    if layout == "nearest-in-few-groups":
        assert np.all(prob.ids.cpu().numpy() < r)


def test_group_select_all_keys_equal_falls_back():
    """Every group minimum equal: every group lies below the threshold, the list overflows, and the streamed
    select over the row takes over (ties by index)."""
    _say("group-minima select, all keys equal")
    n, d, r, V = 50000, 16, 1000, 4000
    rng, q, k, vals, p_lm, ko, qo = _store((n,), (2,), d, V, 322)
    k[:] = 0.0
    k[:, 0] = 3.0
    assert _path(q, k, ko, qo, r, V, 4) == "groups"
    prob = _problem(q, k, vals, p_lm, ko, qo, r, 0.05, 0.4, torch.float32)
    _check_all_modes(prob, q, k, vals, p_lm, ko, qo, r, 0.05, 0.4)
    assert prob.ids.cpu().numpy()[0].tolist() == list(range(r))


def test_group_minima_and_parts_kernel_agree():
    """The same rows with a vocabulary too large for the sliced finish: the mixture steps take the parts
    kernel (sampled threshold), the select alone the group minima; both equal the oracle."""
    _say("group minima vs parts kernel")
    sizes, qps, d, r, V = (40001, 33333), (2, 1), 16, 1024, 600001
    rng, q, k, vals, p_lm, ko, qo = _store(sizes, qps, d, V, 323)
    assert _path(q, k, ko, qo, r, V, 4) == "parts"
    assert _path(q, k, ko, qo, r, None, 4) == "groups"
    prob = _problem(q, k, vals, p_lm, ko, qo, r, 0.05, 0.4, torch.float32)
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r)
    prob.run_part("distances")
    prob.run_part("select")
    torch.cuda.synchronize()
    _check_select(prob.ids, prob.dists, o_ids, o_d)
    n = k.shape[0]
    masked = rng.choice(n, n // 4, replace=False)
    _check_all_modes(prob, q, k, vals, p_lm, ko, qo, r, 0.05, 0.4, masked)


@pytest.mark.parametrize("path", ["groups", "parts"])
def test_sliced_finish_sums_are_exact(path):
    """The sliced finish adds each slice's weights as 64-bit fixed-point integers, so its p_M does not
    depend on the order of the atomics: repeated steps give the same bits, also with most neighbours
    sharing a few tokens (Zipf values), and p_M matches the oracle."""
    _say(f"sliced finish, exact sums ({path})")
    if path == "groups":
        sizes, qps, d, r, V = (65536,), (2,), 16, 1024, 32000
    else:  # 64-row tiles (many sets): the parts kernel samples the rows
        sizes, qps, d, r, V = (4096,) * 32, (1,) * 32, 256, 256, 32000
    rng, q, k, vals, p_lm, ko, qo = _store(sizes, qps, d, V, 324)
    vals = np.minimum(rng.zipf(1.1, vals.size) - 1, V - 1).astype(np.int32)
    assert _path(q, k, ko, qo, r, V, 4) == path
    prob = _problem(q, k, vals, p_lm, ko, qo, r, 0.05, 0.4, torch.float32)
    first = [t.clone() for t in prob.run()]
    for _ in range(3):
        again = prob.run()
        torch.cuda.synchronize()
        assert torch.equal(again[0].view(torch.int32), first[0].view(torch.int32)), "p_M bits changed"
        assert torch.equal(again[1], first[1])
    o_ids, o_d = oracle.select(q, k, "f32", ko, qo, r)
    _check_select(first[1], first[2], o_ids, o_d)
    np.testing.assert_allclose(first[0].cpu().numpy(), oracle.mix(o_ids, o_d, vals, ko, qo, p_lm, 0.05, 0.4),
                               rtol=0, atol=1e-5)
