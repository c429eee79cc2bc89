"""Which select path a batch of few queries on short rows takes: the rules of
the library's host code, restated for the tests (pinned against the
workspace size in test_abi_host.py).

Rows of at most 65536 keys with r <= 1024, whose parts (4096 keys each) over
all queries fit in 256 workgroups, take the split select.  When the streaming
distance kernels serve the batch with 16 or 32 key rows per workgroup (each
of its four waves then records the smallest distance of the 4 or 8 rows it
took, every fourth row of the tile), a row holds at least 2 r such groups and the finish runs without a
mixture or in vocabulary slices, the finish reads those group minima and no
parts kernel runs ("groups"); otherwise a parts kernel samples the row first
("parts").
"""


def tile_rows(d: int, esize: int, S: int, max_keys: int) -> int:
    """Key rows per streaming distance workgroup."""
    rpt = min((1 << 20) // (d * esize), 4096)
    rpt = max((rpt + 7) // 8 * 8, 8)
    while rpt > 16 and S * ((max_keys + rpt - 1) // rpt) < 2048:
        rpt = (rpt // 2 + 7) // 8 * 8
    return rpt


def matrix_cores(d: int, esize: int, max_queries: int) -> bool:
    return esize == 2 and d % 128 == 0 and d <= 65536 and max_queries >= 16


def group_rows(B: int, d: int, esize: int, S: int, max_keys: int, max_queries: int, r: int) -> int:
    """Rows per group when the distance stage writes group minima, else 0."""
    if matrix_cores(d, esize, max_queries):
        return 0
    rpt = tile_rows(d, esize, S, max_keys)
    ld = (max_keys + rpt - 1) // rpt * rpt
    if ld > 65536 or r > 1024 or B * ((ld + 4095) // 4096) > 256:
        return 0
    if rpt not in (16, 32):
        return 0
    groups = ld // (rpt // 4)
    return rpt // 4 if 2 * r <= groups <= 16384 else 0


def split_path(B: int, d: int, esize: int, S: int, max_keys: int, max_queries: int, r: int, V=None) -> str:
    """"groups", "parts", "other" (no split select) or "matrix-core" (the split select, if any, samples its
    rows) for a step with a mixture over V tokens (V None: no mixture)."""
    if matrix_cores(d, esize, max_queries):
        return "matrix-core"
    rpt = tile_rows(d, esize, S, max_keys)
    ld = (max_keys + rpt - 1) // rpt * rpt
    if ld > 65536 or r > 1024 or B * ((ld + 4095) // 4096) > 256:
        return "other"
    sliced = V is None or B * ((V + 4095) // 4096) <= 256
    return "groups" if sliced and group_rows(B, d, esize, S, max_keys, max_queries, r) else "parts"
