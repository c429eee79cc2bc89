"""Host-side checks of the C ABI (no GPU needed): the library loads, exports every
function include/knnlm.h declares, and rejects bad arguments before enqueuing
anything."""
import ctypes
import os

import pytest

from paper_2405_19325_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "knnlm.h")

OK, INVALID, R_EXCEEDS_N, UNSUPPORTED, WORKSPACE, HIP = range(6)


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_exports_every_declared_function(lib):
    names = _lib.header_functions(HEADER)
    assert len(names) >= 9
    for n in names:
        assert hasattr(lib, n), n
        assert n in _lib.SIGNATURES, f"{n} declared in the header but not bound"
    assert set(_lib.SIGNATURES) == set(names)


def test_abi_version_and_status_strings(lib):
    assert lib.knn_abi_version() == 2
    for s in range(6):
        assert lib.knn_status_string(s).decode()
    assert lib.knn_status_string(99).decode() == "unknown status"


# A valid decode-shaped call: B=1, d=4096, V=32000, one set of 65536 keys, r=1024.
BASE = dict(B=1, d=4096, V=32000, S=1, total_keys=65536, min_keys=65536, max_keys=65536, max_queries=1,
            dtype=1, r=1024, mu=1 / 64, lam=0.3)
FAKE = 1 << 20  # a non-null pointer value; validation never dereferences it


def _ws_size(lib, a):
    return lib.knn_lm_mixture_workspace_size(a["B"], a["d"], a["V"], a["S"], a["total_keys"], a["min_keys"],
                                             a["max_keys"], a["max_queries"], a["dtype"], a["r"])


def _validate(lib, ws=FAKE, ws_bytes=None, nulls=(), **over):
    a = dict(BASE, **over)
    if ws_bytes is None:
        ws_bytes = _ws_size(lib, dict(BASE)) + 0
    ptr = {n: (None if n in nulls else FAKE) for n in
           ("queries", "keys", "values", "key_offsets", "query_offsets", "p_lm", "p_m", "ids", "dists")}
    return lib.knn_lm_mixture_validate(ptr["queries"], ptr["keys"], ptr["values"], ptr["key_offsets"],
                                       ptr["query_offsets"], ptr["p_lm"], a["B"], a["d"], a["V"], a["S"],
                                       a["total_keys"], a["min_keys"], a["max_keys"], a["max_queries"], a["dtype"],
                                       a["r"], a["mu"], a["lam"], ptr["p_m"], ptr["ids"], ptr["dists"], ws, ws_bytes)


def test_valid_call_validates(lib):
    assert _ws_size(lib, BASE) > 65536 * 4
    assert _validate(lib) == OK


@pytest.mark.parametrize("over,expect", [
    (dict(r=0), INVALID), (dict(r=-3), INVALID), (dict(B=0), INVALID), (dict(d=0), INVALID),
    (dict(V=0), INVALID), (dict(S=0), INVALID), (dict(dtype=7), INVALID), (dict(mu=0.0), INVALID),
    (dict(mu=-1.0), INVALID), (dict(mu=float("nan")), INVALID), (dict(mu=float("inf")), INVALID),
    (dict(lam=-0.01), INVALID), (dict(lam=1.01), INVALID), (dict(lam=float("nan")), INVALID),
    (dict(min_keys=70000), INVALID), (dict(max_keys=70000), INVALID), (dict(max_queries=2), INVALID),
    (dict(max_queries=0), INVALID), (dict(r=65537), UNSUPPORTED), (dict(r=4097), UNSUPPORTED),
    (dict(min_keys=1000, r=1001), R_EXCEEDS_N), (dict(min_keys=0), R_EXCEEDS_N),
])
def test_rejects_bad_scalars(lib, over, expect):
    assert _validate(lib, **over) == expect


def test_lambda_and_r_edges_accepted(lib):
    assert _validate(lib, lam=0.0) == OK
    assert _validate(lib, lam=1.0) == OK
    assert _validate(lib, r=1) == OK
    assert _validate(lib, r=4096) == OK


@pytest.mark.parametrize("null", ["queries", "keys", "values", "key_offsets", "query_offsets", "p_lm", "p_m", "ids",
                                  "dists"])
def test_rejects_null_pointers(lib, null):
    assert _validate(lib, nulls=(null,)) == INVALID


def test_workspace_checks(lib):
    need = _ws_size(lib, BASE)
    assert _validate(lib, ws=None) == WORKSPACE
    assert _validate(lib, ws_bytes=need - 1) == WORKSPACE
    assert _validate(lib, ws=FAKE + 8) == WORKSPACE  # not 256-byte aligned
    assert _validate(lib, ws_bytes=need) == OK


def test_workspace_size_zero_for_invalid_sizes(lib):
    assert _ws_size(lib, dict(BASE, r=0)) == 0
    assert _ws_size(lib, dict(BASE, min_keys=10)) == 0


def test_entry_points_reject_before_touching_the_device(lib):
    # Invalid arguments return an error code without any HIP call, so these run without a GPU.
    a = BASE
    st = lib.knn_lm_mixture(FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, a["B"], a["d"], a["V"], a["S"],
                            a["total_keys"], a["min_keys"], a["max_keys"], a["max_queries"], a["dtype"], 0, a["mu"],
                            a["lam"], FAKE, FAKE, FAKE, FAKE, 1 << 30, None)
    assert st == INVALID
    st = lib.knn_lm_mixture_part(9, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, a["B"], a["d"], a["V"], a["S"],
                                 a["total_keys"], a["min_keys"], a["max_keys"], a["max_queries"], a["dtype"], 16,
                                 a["mu"], a["lam"], FAKE, FAKE, FAKE, FAKE, 1 << 30, None)
    assert st == INVALID
    assert lib.knn_key_sqnorms(None, 10, 8, 1, FAKE, None) == INVALID
    assert lib.knn_key_sqnorms(FAKE, 10, 0, 1, FAKE, None) == INVALID
    assert lib.knn_mix(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 100, 1, 8, 0.1, 2.0, FAKE, None) == INVALID
    assert lib.knn_mix(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 100, 1, 5000, 0.1, 0.5, FAKE, None) == UNSUPPORTED
    assert lib.knn_distances(FAKE, FAKE, None, FAKE, FAKE, 1, 64, 1, 100, 1, 1, FAKE, 99, None) == INVALID


def test_mixture_part_stage_pointer_rules(lib):
    # The mix stage needs no workspace and no queries/keys; distances needs no outputs.
    a = BASE
    args = lambda part, q, k, ws, pm, ids: lib.knn_lm_mixture_part(
        part, q, k, None, FAKE, FAKE, FAKE, FAKE, a["B"], a["d"], a["V"], a["S"], a["total_keys"], a["min_keys"],
        a["max_keys"], a["max_queries"], a["dtype"], a["r"], float("nan"), a["lam"], pm, ids, ids, ws, 0, None)
    # distances stage with a null workspace: rejected
    assert args(1, FAKE, FAKE, None, None, None) == WORKSPACE
    # select stage with null outputs: rejected
    assert args(2, None, None, FAKE, None, None) == INVALID
    # mix stage: mu = NaN is rejected
    assert args(3, None, None, None, FAKE, FAKE) == INVALID


BF16_PACKED, F16_PACKED, KEYS_PACKED = 0x101, 0x102, 0x100


def test_packed_keys_bytes(lib):
    # blocks of 16 rows, each 32 d bytes of fragments then 16 fp32 norms
    assert lib.knn_packed_keys_bytes(16, 128, 1) == 32 * 128 + 64
    assert lib.knn_packed_keys_bytes(17, 128, 2) == 2 * (32 * 128 + 64)
    assert lib.knn_packed_keys_bytes(8388608, 1024, 2) == 8388608 // 16 * (32 * 1024 + 64)
    assert lib.knn_packed_keys_bytes(1000, 256, BF16_PACKED) == 63 * (32 * 256 + 64)  # the flag is ignored here
    for n, d, t in ((0, 128, 1), (16, 0, 1), (16, 128, 0), (16, 192, 1), (16, 65536 + 128, 1), (16, 128, 7)):
        assert lib.knn_packed_keys_bytes(n, d, t) == 0, (n, d, t)


def test_pack_keys_rejects_before_touching_the_device(lib):
    assert lib.knn_pack_keys(None, 16, 128, 1, FAKE, None) == INVALID
    assert lib.knn_pack_keys(FAKE, 16, 128, 1, None, None) == INVALID
    assert lib.knn_pack_keys(FAKE, 0, 128, 1, FAKE, None) == INVALID
    assert lib.knn_pack_keys(FAKE + 8, 16, 128, 1, FAKE, None) == INVALID  # not 16-byte aligned
    assert lib.knn_pack_keys(FAKE, 16, 128, 0, FAKE, None) == UNSUPPORTED  # fp32
    assert lib.knn_pack_keys(FAKE, 16, 192, 1, FAKE, None) == UNSUPPORTED  # d % 128 != 0


def test_packed_dtype_validation(lib):
    # a batch the matrix cores serve: 128 queries on one set of 65536 keys at d = 1024
    mc = dict(B=128, d=1024, max_queries=128, min_keys=65536, max_keys=65536)
    ws = _ws_size(lib, dict(BASE, **mc))
    assert _validate(lib, ws_bytes=ws, dtype=2, **mc) == OK
    assert _validate(lib, ws_bytes=ws, dtype=F16_PACKED, **mc) == OK
    assert _validate(lib, ws_bytes=ws, dtype=BF16_PACKED, **mc) == OK
    assert _ws_size(lib, dict(BASE, dtype=F16_PACKED, **mc)) == ws
    # fp32 keys cannot be packed; the flag on its own is no element type
    assert _validate(lib, ws_bytes=ws, dtype=KEYS_PACKED, **mc) == INVALID
    # fewer than 16 queries per set (the streaming kernel), or d % 128 != 0: not served packed
    assert _validate(lib, dtype=BF16_PACKED) == UNSUPPORTED
    mc_odd = dict(mc, d=1000)
    assert _validate(lib, ws_bytes=_ws_size(lib, dict(BASE, **mc_odd)), dtype=BF16_PACKED, **mc_odd) == UNSUPPORTED
    # the select and mix stages read no keys: the flag changes nothing there
    a = dict(BASE, **mc)
    st = lib.knn_lm_mixture_part(3, None, None, None, FAKE, FAKE, FAKE, FAKE, a["B"], a["d"], a["V"], a["S"],
                                 a["total_keys"], a["min_keys"], a["max_keys"], a["max_queries"], BF16_PACKED,
                                 a["r"], a["mu"], a["lam"], FAKE, FAKE, FAKE, None, 0, None)
    assert st == OK or st == HIP  # validated; the launch itself needs a GPU
    # knn_distances: packed keys with a streaming-path batch are refused
    assert lib.knn_distances(FAKE, FAKE, None, FAKE, FAKE, 1, 1024, 1, 100, 1, BF16_PACKED, FAKE, 100, None) == \
        UNSUPPORTED
    assert lib.knn_distances(FAKE, FAKE, None, FAKE, FAKE, 16, 1024, 1, 100, 16, KEYS_PACKED, FAKE, 100, None) == \
        INVALID


def test_select_path_rules_match_the_workspace_layout(lib):
    """The tests' restatement of which split rows take the group-minima select
    (tests/select_paths.py) against the library: the workspace holds B * 4 *
    tiles fp32 group minima exactly when it says so."""
    import select_paths

    def ws(**over):
        return _ws_size(lib, dict(BASE, **over))

    # decode shape: 32-row tiles, 8192 groups of 8 rows: on for every r <= 1024
    assert select_paths.group_rows(1, 4096, 2, 1, 65536, 1, 1024) == 8
    # 4096 keys in 16-row tiles: 1024 groups of 4 rows, so r <= 512
    small = dict(total_keys=4096, min_keys=4096, max_keys=4096)
    assert select_paths.tile_rows(4096, 2, 1, 4096) == 16
    assert select_paths.group_rows(1, 4096, 2, 1, 4096, 1, 512) == 4
    assert select_paths.group_rows(1, 4096, 2, 1, 4096, 1, 513) == 0
    assert ws(r=512, **small) - ws(r=513, **small) == 1024 * 4
    # three queries: three rows of minima
    assert ws(B=3, max_queries=3, r=512, **small) - ws(B=3, max_queries=3, r=513, **small) == 3 * 1024 * 4
    # 16 bf16 queries on a set take the matrix cores: no group minima
    assert select_paths.group_rows(16, 4096, 2, 1, 4096, 16, 512) == 0
    assert ws(B=16, max_queries=16, r=512, **small) == ws(B=16, max_queries=16, r=513, **small)
    # fp32 keys of width 16 on 40,000-key rows: 16-row tiles, 10,000 groups of 4
    assert select_paths.tile_rows(16, 4, 1, 40000) == 16
    assert select_paths.group_rows(1, 16, 4, 1, 40000, 1, 1024) == 4
    # 64-row tiles (many sets): the parts kernel samples the rows
    many = dict(B=32, S=32, d=256, total_keys=32 * 4096, min_keys=4096, max_keys=4096, max_queries=1, r=256)
    assert select_paths.tile_rows(256, 2, 32, 4096) == 64
    assert select_paths.split_path(32, 256, 2, 32, 4096, 1, 256, V=32000) == "parts"
    assert ws(**many) == ws(**dict(many, r=255))
