"""The packed key layout (knn_pack_keys) and the matrix-core kernels that read it.

The packed copy is unpacked on the host and compared with the row-major keys
element by element (zero rows pad the last block); its stored norms are exact
integer sums on integer keys and agree with fp64 sums on random keys.  The
distance stage over packed keys runs the same MFMA steps in the same k order
as the row-major matrix-core kernel and sums the norms in the same order, so
its distances must equal that kernel's bit for bit -- for every group size
(16, 32, 64, 128 queries), both ring depths, key sets that start inside a
16-row block, and given or stored norms.  The whole step (fixed lambda, RRC,
a NEST step with masked keys) must then select the same neighbours, and a
packed run is also checked against the oracle.
"""
import gc
import math

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


def _free():
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _unpack(packed: torch.Tensor, n: int, d: int):
    """(keys [nblk * 16, d] as uint16, norms [nblk * 16] fp32) from the packed bytes, on the host."""
    nblk = (n + 15) // 16
    raw = packed.cpu().numpy().reshape(nblk, 32 * d + 64)
    frags = raw[:, :32 * d].copy().view(np.uint16).reshape(nblk, d // 32, 4, 16, 8)  # [b, c, g, r, e]
    keys = frags.transpose(0, 3, 1, 2, 4).reshape(nblk * 16, d)  # row 16 b + r, element 32 c + 8 g + e
    norms = raw[:, 32 * d:].copy().view(np.float32).reshape(nblk * 16)
    return keys, norms


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
@pytest.mark.parametrize("n,d", [(16, 128), (1000, 640), (4099, 256)])
def test_pack_layout(dtype, n, d):
    _say(f"pack layout {dtype} n={n} d={d}")
    g = torch.Generator(device="cuda").manual_seed(n + d)
    # integer keys: every norm is an exact integer in fp32
    k = torch.randint(-4, 5, (n, d), generator=g, device="cuda").to(dtype)
    packed = knn.pack_keys(k)
    torch.cuda.synchronize()
    assert packed.numel() == knn.packed_keys_bytes(n, d, dtype) == (n + 15) // 16 * (32 * d + 64)
    keys, norms = _unpack(packed, n, d)
    want = k.view(torch.int16).cpu().numpy().view(np.uint16)
    np.testing.assert_array_equal(keys[:n], want)
    assert not keys[n:].any(), "padding rows must be zero"
    kf = k.float().cpu().numpy().astype(np.float64)
    np.testing.assert_array_equal(norms[:n].astype(np.float64), (kf * kf).sum(1))
    assert not norms[n:].any()
    # random keys: the stored norms are fp32 sums of the same squares
    kr = (torch.randn((n, d), generator=g, device="cuda") * (8 / math.sqrt(d))).to(dtype)
    _, nr = _unpack(knn.pack_keys(kr), n, d)
    ref = (kr.float().cpu().numpy().astype(np.float64) ** 2).sum(1)
    np.testing.assert_allclose(nr[:n].astype(np.float64), ref, rtol=2e-6, atol=0)


# (name, queries per set, key set sizes, d): group sizes 16 (queries from global memory), 32, 64 and 128
# (queries through the LDS ring), deep rings where 64-element steps per pass are a multiple of the ring depth
# and two-set rings otherwise, key sets whose rows start inside a 16-row block.
DIST_CASES = [
    ("16q-d256-deep", 16, (3001,), 256),
    ("16q-d640-shallow", 16, (1500, 2201), 640),
    ("32q-d1024-deep", 32, (2500,), 1024),
    ("64q-3sets-d512", 40, (1000, 1700, 2300), 512),
    ("128q-2groups-d512", 130, (2900,), 512),
    ("128q-d128-shallow", 128, (1031, 777), 128),
    ("128q-d1152-shallow", 96, (2000,), 1152),
]


def _batch(qps, sizes, d, dtype, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    S = len(sizes)
    ko = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    qo = np.arange(S + 1, dtype=np.int64) * qps
    scale = 8 / math.sqrt(d)
    k = (torch.randn((int(ko[-1]), d), generator=g, device="cuda") * scale).to(dtype).contiguous()
    q = (torch.randn((int(qo[-1]), d), generator=g, device="cuda") * scale).to(dtype).contiguous()
    return q, k, ko, qo


def _bits(t):
    return t.view(torch.int32)


@pytest.mark.parametrize("norms", [False, True], ids=["stored-norms", "given-norms"])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
@pytest.mark.parametrize("name,qps,sizes,d", DIST_CASES, ids=[c[0] for c in DIST_CASES])
def test_packed_distances_equal_row_major_bitwise(name, qps, sizes, d, dtype, norms):
    _say(f"packed distances {name} {dtype} norms={'given' if norms else 'stored'}")
    q, k, ko, qo = _batch(qps, sizes, d, dtype, sum(map(ord, name)) + d)
    tko, tqo = torch.as_tensor(ko, device="cuda"), torch.as_tensor(qo, device="cuda")
    kn = knn.key_sqnorms(k) if norms else None
    packed = knn.pack_keys(k)
    ref = knn.distances(q, k, tko, tqo, key_sqnorms=kn, key_offsets_host=ko, query_offsets_host=qo)
    got = knn.distances(q, k, tko, tqo, key_sqnorms=kn, key_offsets_host=ko, query_offsets_host=qo,
                        packed_keys=packed)
    torch.cuda.synchronize()
    assert torch.equal(_bits(got), _bits(ref)), "packed distances differ from the row-major kernel's"
    # and they are the distances: every query against its own set, spot-checked in fp64
    qh = q.double().cpu().numpy()
    kh = k.double().cpu().numpy()
    g = got.cpu().numpy()
    for s in range(len(sizes)):
        for b in (qo[s], qo[s + 1] - 1):
            dd = ((kh[ko[s]:ko[s + 1]] - qh[b]) ** 2).sum(1)
            np.testing.assert_allclose(g[b, :sizes[s]], dd, rtol=1e-5, atol=1e-5 * max(1.0, dd.max()))


MIX_CASES = [
    ("16q-bf16", gen.scaled(gen.config("specverify_seq"), B=32, S=2, n_keys=(3000, 4100), d=1024, mu=1 / 32), 61),
    ("128q-f16", gen.scaled(gen.config("specverify_static"), B=128, S=1, n_keys=9000, d=1024, query_mode="iid",
                            mu=1 / 32), 62),
    ("40q-ragged-bf16", gen.scaled(gen.config("specverify_seq"), B=120, S=3, n_keys=(2049, 1300, 4100), d=512,
                                   mu=1 / math.sqrt(512), r=512), 63),
]


def _problem(w, packed=None, norms=None):
    return knn.MixtureProblem(w.queries, w.keys, w.values, w.key_offsets, w.query_offsets, w.p_lm, w.r, w.mu, w.lam,
                              key_sqnorms=norms, key_offsets_host=w.key_offsets_host,
                              query_offsets_host=w.query_offsets_host, packed_keys=packed)


@pytest.mark.parametrize("name,spec,seed", MIX_CASES, ids=[m[0] for m in MIX_CASES])
def test_packed_steps_match_row_major_and_oracle(name, spec, seed):
    _say(f"packed mixture {name}")
    w = gen.make(spec, seed, device="cuda")
    packed = knn.pack_keys(w.keys)
    a, b = _problem(w), _problem(w, packed)
    # the fixed-lambda step
    pa, ia, da = [t.clone() for t in a.run()]
    pb, ib, db = b.run()
    torch.cuda.synchronize()
    assert torch.equal(ib, ia) and torch.equal(_bits(db), _bits(da))
    torch.testing.assert_close(pb, pa, rtol=0, atol=1e-6)
    rep = parity.check_workload(w, pb, ib, db)
    _say(f"{name} packed: {rep.summary()}")
    assert rep.ok(), rep.failures[:5]
    # lambda_t from relative retrieval confidence
    ra = [t.clone() for t in a.run_rrc(0.3, 0.1)]
    rb = b.run_rrc(0.3, 0.1)
    torch.cuda.synchronize()
    assert torch.equal(rb[1], ra[1]) and torch.equal(_bits(rb[2]), _bits(ra[2]))
    assert torch.equal(rb[3], ra[3])
    # a NEST step with a tenth of the keys masked
    total = int(w.key_offsets_host[-1])
    masked = np.random.default_rng(seed).choice(total, total // 10, replace=False)
    mask = knn.mask_words(masked, total, "cuda")
    draft = w.p_lm.argmax(1).to(torch.int32)
    oa = {k: v.clone() for k, v in a.run_nest(0.3, 0.1, 0.5, key_mask=mask, draft_tokens=draft).items()}
    ob = b.run_nest(0.3, 0.1, 0.5, key_mask=mask, draft_tokens=draft)
    torch.cuda.synchronize()
    for key in ("ids", "next_token", "span_key", "use_span"):
        assert torch.equal(ob[key], oa[key]), key
    assert torch.equal(_bits(ob["dists"]), _bits(oa["dists"]))
    torch.testing.assert_close(ob["p_m"], oa["p_m"], rtol=0, atol=1e-6)
    del w, packed, a, b
    _free()


def test_packed_stages_and_given_norms():
    """The distance stage alone over packed keys with caller norms, then the select: the same as one call."""
    _say("packed stages with given norms")
    w = gen.make(MIX_CASES[1][1], 64, device="cuda")
    packed = knn.pack_keys(w.keys)
    norms = knn.key_sqnorms(w.keys)
    a = _problem(w, packed, norms)
    pa, ia, da = [t.clone() for t in a.run()]
    b = _problem(w, None, norms)
    b.run_part("distances")
    b.run_part("select_mix")
    torch.cuda.synchronize()
    assert torch.equal(b.ids, ia) and torch.equal(_bits(b.dists), _bits(da))
    rep = parity.check_workload(w, pa, ia, da)
    assert rep.ok(), rep.failures[:5]
    del w, packed
    _free()


def test_packed_keys_refused_where_the_matrix_cores_do_not_run():
    """Fewer than 16 queries per set take the streaming kernel, which cannot read packed keys."""
    w = gen.make(gen.scaled(gen.config("decode_7b"), B=2, S=2, n_keys=(3000, 3000), r=64, d=1024), 65,
                 device="cuda")
    packed = knn.pack_keys(w.keys)
    with pytest.raises(knn.KnnError) as e:
        _problem(w, packed).run()
    assert e.value.status == 3  # KNN_ERR_UNSUPPORTED
