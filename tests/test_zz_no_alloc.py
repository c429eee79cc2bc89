"""knn_lm_mixture_noalloc, whose workspace is the library's static per-GPU
scratch array, against knn_lm_mixture with a caller workspace: three calls in
a row on one GPU (the full single-query decode workload, 20 queries on one
set, then a smaller ragged batch), each equal to the workspace entry point's
neighbours and distances bit for bit and within the p_M tolerance of it, and
to the CPU oracle under rules P2-P5.  A request larger than the array is
rejected before anything is enqueued."""
import numpy as np
import pytest
import torch

import parity
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


CALLS = [
    ("decode_7b full size", gen.config("decode_7b"), 2),
    ("20 queries, one set of 65536 f32 keys, d=256",
     gen.scaled(gen.config("decode_7b"), B=20, n_keys=65536, d=256, dtype="f32", mu=1 / 16), 29),
    ("3 queries on ragged sets of 3000, 4100, 2500 keys",
     gen.scaled(gen.config("decode_7b"), B=3, S=3, n_keys=(3000, 4100, 2500), r=128), 11),
]


def test_noalloc_matches_workspace_entry_point():
    for label, spec, seed in CALLS:
        _say(f"no-alloc entry point: {label}")
        w = gen.make(spec, seed, device="cuda")
        prob = knn.MixtureProblem(w.queries, w.keys, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu,
                                  w.lam, key_offsets_host=w.key_offsets_host,
                                  query_offsets_host=w.query_offsets_host)
        p_ref, ids_ref, d_ref = prob.run()
        B = int(w.query_offsets_host[-1])
        p_m = torch.full((B, w.p_lm.shape[1]), float("nan"), device="cuda")
        ids = torch.full((B, w.r), -7, dtype=torch.int32, device="cuda")
        dists = torch.full((B, w.r), float("nan"), device="cuda")
        knn.mixture_noalloc(w.queries, w.keys, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu, w.lam,
                            p_m, ids, dists, w.key_offsets_host, w.query_offsets_host)
        torch.cuda.synchronize()
        assert torch.equal(ids, ids_ref)
        assert torch.equal(dists, d_ref)
        err = float((p_m.double() - p_ref.double()).abs().max())
        assert err <= parity.PM_TOL, err
        rep = parity.check_workload(w, p_m, ids, dists)
        _say(f"{label}: |p_M - workspace entry point| <= {err:.3g}; oracle: {rep.summary()}")
        assert rep.ok(), rep.failures[:5]
        del w, prob


def test_noalloc_rejects_requests_beyond_the_scratch_array():
    """200 queries on one set of 65536 keys need a 52 MB distance matrix, more than the 32 MiB array."""
    B, n, d = 200, 65536, 64
    dev = "cuda"
    q = torch.zeros((B, d), device=dev)
    k = torch.zeros((n, d), device=dev)
    vals = torch.zeros(n, dtype=torch.int32, device=dev)
    ko = torch.tensor([0, n], device=dev)
    qo = torch.tensor([0, B], device=dev)
    p_lm = torch.full((B, 10), 0.1, device=dev)
    p_m = torch.zeros((B, 10), device=dev)
    ids = torch.zeros((B, 8), dtype=torch.int32, device=dev)
    dists = torch.zeros((B, 8), device=dev)
    with pytest.raises(knn.KnnError) as e:
        knn.mixture_noalloc(q, k, vals, ko, qo, p_lm, 8, 0.1, 0.5, p_m, ids, dists, np.array([0, n]),
                            np.array([0, B]))
    assert e.value.status == 4  # KNN_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert int(ids.abs().sum()) == 0  # nothing was enqueued
