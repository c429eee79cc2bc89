"""The five full-size workloads, in the launch configuration the benchmark
times (the distance stage, then the fused select and mixture), against the CPU
oracle under rules P2-P5 (tests/parity.py).

Every query of decode_7b, ragged_batch, decode_70b and specverify_seq is
compared with the oracle element by element.  The two matrix-core workloads
also run over the packed copy of their keys, which must select the same
neighbours at the same distance bits.  specverify_static (128 queries
on one store of 8,388,608 keys) is compared on all 128 queries too, in four
tests of 32 rows each (rows b with b mod 4 = c), so every 16-query block of the
matrix-core workgroup is covered by every test; the workload, its GPU result
and its keys' host copy are made once for the four.  Properties that hold for
every query (sum of p_M, order, id range) are checked on all rows as well.
"""
import gc
import time

import numpy as np
import pytest
import torch

import oracle
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


def _free():
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _bench_step(w, packed=None):
    """The benchmark's step: the distance stage, then the fused select and mixture (with packed, over
    the packed copy of the keys)."""
    prob = knn.MixtureProblem(w.queries, w.keys, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu,
                              w.lam, key_offsets_host=w.key_offsets_host, query_offsets_host=w.query_offsets_host,
                              packed_keys=packed)
    prob.run_part("distances")
    prob.run_part("select_mix")
    torch.cuda.synchronize()
    return prob


def _same_as_packed(w, prob):
    """The step over the packed copy of the keys selects the same neighbours at the same distance bits."""
    t0 = time.time()
    packed = knn.pack_keys(w.keys)
    pk = _bench_step(w, packed)
    assert torch.equal(pk.ids, prob.ids)
    assert torch.equal(pk.dists.view(torch.int32), prob.dists.view(torch.int32))
    torch.testing.assert_close(pk.p_m, prob.p_m, rtol=0, atol=1e-6)
    _say(f"packed keys: the same neighbours and distances ({time.time() - t0:.1f} s)")
    del packed, pk
    _free()


def _every_query_properties(w, p_m, ids, dists):
    pm64 = p_m.double()
    torch.testing.assert_close(pm64.sum(1), w.lam * w.p_lm.double().sum(1) + (1 - w.lam), rtol=0, atol=1e-5)
    assert torch.all(dists[:, 1:] >= dists[:, :-1])
    assert int(ids.min()) >= 0
    n_of = torch.as_tensor(np.diff(w.key_offsets_host)[w.set_of_query()], device=ids.device)
    assert torch.all(ids.max(1).values < n_of)


@pytest.mark.parametrize("name", ["decode_7b", "ragged_batch", "decode_70b", "specverify_seq"])
def test_full_size_every_query(name):
    _free()
    t0 = time.time()
    _say(f"full workload {name}: generating")
    w = gen.make(gen.config(name), gen.CONFIG_SEEDS[name], device="cuda")
    _say(f"full workload {name}: running")
    prob = _bench_step(w)
    p_m, ids, dists = prob.p_m, prob.ids, prob.dists
    _every_query_properties(w, p_m, ids, dists)
    if name == "specverify_seq":
        _same_as_packed(w, prob)
    B = int(w.query_offsets_host[-1])
    t1 = time.time()
    _say(f"full workload {name}: oracle on all {B} queries, {parity.host_threads()} host threads")
    rep = parity.check_workload(w, p_m, ids, dists)
    _say(f"{name}: {rep.summary()}; oracle check {time.time() - t1:.1f} s, test {time.time() - t0:.1f} s")
    assert rep.queries == B
    assert rep.ok(), rep.failures[:5]
    del w, prob, p_m, ids, dists
    _free()


@pytest.fixture(scope="module")
def static_store():
    """specverify_static run once in the benchmark's launch configuration, with its keys copied to the host."""
    _free()
    t0 = time.time()
    _say("full workload specverify_static: generating")
    w = gen.make(gen.config("specverify_static"), gen.CONFIG_SEEDS["specverify_static"], device="cuda")
    _say("full workload specverify_static: running")
    prob = _bench_step(w)
    _every_query_properties(w, prob.p_m, prob.ids, prob.dists)
    _same_as_packed(w, prob)
    keys_h, dt = oracle.host_elements(w.keys)
    _say(f"specverify_static: step run and keys on the host in {time.time() - t0:.1f} s")
    yield w, prob, (keys_h, dt)
    del w, prob, keys_h
    _free()


@pytest.mark.parametrize("chunk", range(4))
def test_full_size_static_store(static_store, chunk):
    w, prob, host = static_store
    rows = list(range(chunk, int(w.query_offsets_host[-1]), 4))
    t0 = time.time()
    _say(f"specverify_static: oracle on rows {chunk}::4 ({len(rows)} queries, {parity.host_threads()} threads)")
    rep = parity.check_workload(w, prob.p_m, prob.ids, prob.dists, sample=rows, host_keys=lambda s: host)
    _say(f"specverify_static rows {chunk}::4: {rep.summary()}; {time.time() - t0:.1f} s")
    assert rep.queries == len(rows)
    assert rep.ok(), rep.failures[:5]
