"""Seeded generators for the kNN-LM mixture workloads.

The paper measures on real corpora encoded by Llama-2-Chat (WikiText-103,
Pile of Law, Wikipedia passages retrieved per query, Section 4 and Appendix A).
None of that data or those weights is available, so synthetic inputs with the
paper's shapes stand in for them:

* keys: the per-input token store built on the fly from the top-b retrieved
  passages (Section 3.1, Algorithm 1), one contiguous block of rows per key set
  (one set per decoding sequence), i.i.d. N(0,1) * key_scale, rounded to the
  key dtype (round to nearest even);
* queries: the LM hidden state q_t, drawn from the same law as the keys
  (fp32 sample, then rounded), or "planted" next to a chosen key;
* values: next-token ids in [0, V), uniform or bounded Zipf(s) by rank;
* p_LM: a softmax of N(0, sigma) logits over the vocabulary, fp32.

Seeds: each named workload has a base seed (CONFIG_SEEDS); the sub-streams are keys +100, queries +200,
values +300, logits +400, offsets +500, projection +600.  Large tensors are
drawn in fixed row blocks, so a workload is a pure function of (spec, seed,
device type).  CPU and GPU generators give different (equally valid) draws.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np
import torch

DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}

# Row block used when drawing keys: bounds the fp32 temporary to 64 Mi elements.
_BLOCK_ELEMS = 1 << 26


@dataclasses.dataclass(frozen=True)
class Spec:
    """Shape and distribution recipe of one workload."""

    name: str
    B: int                      # total queries
    d: int                      # hidden size
    S: int                      # number of key sets
    n_keys: object              # int (every set) | ("uniform", lo, hi) | tuple of ints
    dtype: str                  # "f32" | "bf16" | "f16"
    key_scale: float            # keys ~ N(0,1) * key_scale
    values: str                 # "uniform" | "zipf"
    zipf_s: float
    V: int
    logit_sigma: float
    r: int
    mu: float
    lam: float
    query_mode: str = "iid"     # "iid" | "planted" | "projected"
    planted_noise: float = 0.01  # planted: q = k_j + N(0, (noise*key_scale)^2)
    proj_in: int = 0            # projected: source hidden size
    proj_seed: int = -1         # projected: base seed of the source queries

    def queries_per_set(self) -> List[int]:
        base, extra = divmod(self.B, self.S)
        return [base + (1 if s < extra else 0) for s in range(self.S)]

    def replace(self, **kw) -> "Spec":
        return dataclasses.replace(self, **kw)


@dataclasses.dataclass
class Workload:
    spec: Spec
    seed: int
    queries: torch.Tensor        # [B, d] key dtype
    keys: torch.Tensor           # [total_keys, d] key dtype
    values: torch.Tensor         # [total_keys] int32
    key_offsets: torch.Tensor    # [S+1] int64 (same device as keys)
    query_offsets: torch.Tensor  # [S+1] int64
    p_lm: torch.Tensor           # [B, V] float32
    key_offsets_host: np.ndarray
    query_offsets_host: np.ndarray
    planted_ids: Optional[np.ndarray] = None  # local key index planted per query

    @property
    def r(self) -> int:
        return self.spec.r

    @property
    def mu(self) -> float:
        return self.spec.mu

    @property
    def lam(self) -> float:
        return self.spec.lam

    def keys_per_set(self) -> np.ndarray:
        return np.diff(self.key_offsets_host)

    def set_of_query(self) -> np.ndarray:
        qo = self.query_offsets_host
        out = np.empty(int(qo[-1]), dtype=np.int64)
        for s in range(len(qo) - 1):
            out[qo[s]:qo[s + 1]] = s
        return out


def _gen(device: torch.device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def zipf_cdf(V: int, s: float) -> np.ndarray:
    """CDF of the bounded Zipf law P(rank k) proportional to k^-s, k = 1..V."""
    ranks = np.arange(1, V + 1, dtype=np.float64)
    w = ranks ** (-s)
    c = np.cumsum(w)
    return c / c[-1]


def _draw_normal_rows(n_rows: int, d: int, scale: float, dtype: torch.dtype,
                      device: torch.device, g: torch.Generator) -> torch.Tensor:
    out = torch.empty((n_rows, d), dtype=dtype, device=device)
    rows_per_block = max(1, _BLOCK_ELEMS // max(d, 1))
    for r0 in range(0, n_rows, rows_per_block):
        r1 = min(n_rows, r0 + rows_per_block)
        blk = torch.randn((r1 - r0, d), generator=g, device=device, dtype=torch.float32)
        if scale != 1.0:
            blk.mul_(scale)
        out[r0:r1].copy_(blk)
        del blk
    return out


def _draw_values(n: int, spec: Spec, device: torch.device, g: torch.Generator) -> torch.Tensor:
    if spec.values == "uniform":
        return torch.randint(0, spec.V, (n,), generator=g, device=device, dtype=torch.int64).to(torch.int32)
    if spec.values == "zipf":
        cdf = torch.from_numpy(zipf_cdf(spec.V, spec.zipf_s)).to(device)
        out = torch.empty(n, dtype=torch.int32, device=device)
        blk = 1 << 24
        for i0 in range(0, n, blk):
            i1 = min(n, i0 + blk)
            u = torch.rand(i1 - i0, generator=g, device=device, dtype=torch.float64)
            idx = torch.searchsorted(cdf, u, right=True)
            out[i0:i1] = idx.clamp_(max=spec.V - 1).to(torch.int32)
        return out
    raise ValueError(f"unknown value law {spec.values!r}")


def _set_sizes(spec: Spec, seed: int) -> List[int]:
    nk = spec.n_keys
    if isinstance(nk, int):
        return [nk] * spec.S
    if isinstance(nk, tuple) and len(nk) == 3 and nk[0] == "uniform":
        g = _gen(torch.device("cpu"), seed + 500)
        lo, hi = int(nk[1]), int(nk[2])
        return [int(x) for x in torch.randint(lo, hi + 1, (spec.S,), generator=g)]
    if isinstance(nk, (tuple, list)):
        assert len(nk) == spec.S
        return [int(x) for x in nk]
    raise ValueError(f"bad n_keys {nk!r}")


def make(spec: Spec, seed: int, device="cpu") -> Workload:
    """Draw the workload `spec` with base seed `seed` on `device`."""
    device = torch.device(device)
    dtype = DTYPES[spec.dtype]
    sizes = _set_sizes(spec, seed)
    qps = spec.queries_per_set()
    ko = np.zeros(spec.S + 1, dtype=np.int64)
    ko[1:] = np.cumsum(sizes)
    qo = np.zeros(spec.S + 1, dtype=np.int64)
    qo[1:] = np.cumsum(qps)
    total = int(ko[-1])

    keys = _draw_normal_rows(total, spec.d, spec.key_scale, dtype, device, _gen(device, seed + 100))
    values = _draw_values(total, spec, device, _gen(device, seed + 300))

    planted = None
    if spec.query_mode == "iid":
        queries = _draw_normal_rows(spec.B, spec.d, spec.key_scale, dtype, device, _gen(device, seed + 200))
    elif spec.query_mode == "planted":
        gq = _gen(torch.device("cpu"), seed + 200)
        planted = np.empty(spec.B, dtype=np.int64)
        rows = []
        for s in range(spec.S):
            for _ in range(qps[s]):
                j = int(torch.randint(0, sizes[s], (1,), generator=gq))
                planted[len(rows)] = j
                rows.append(int(ko[s]) + j)
        noise = _draw_normal_rows(spec.B, spec.d, spec.planted_noise * spec.key_scale,
                                  torch.float32, device, _gen(device, seed + 201))
        base = keys[torch.as_tensor(rows, device=device)].to(torch.float32)
        queries = (base + noise).to(dtype)
    elif spec.query_mode == "projected":
        # The queries of a second store are a fixed random projection of the
        # sequence-level queries (an input transformation, not part of the step).
        src = _draw_normal_rows(spec.B, spec.proj_in, 8.0 / math.sqrt(spec.proj_in), torch.bfloat16,
                                device, _gen(device, spec.proj_seed + 200))
        P = _draw_normal_rows(spec.proj_in, spec.d, 1.0 / math.sqrt(spec.d), torch.float32,
                              device, _gen(device, seed + 600))
        queries = (src.to(torch.float32) @ P).to(dtype)
    else:
        raise ValueError(spec.query_mode)

    gl = _gen(device, seed + 400)
    logits = torch.randn((spec.B, spec.V), generator=gl, device=device, dtype=torch.float64) * spec.logit_sigma
    p_lm = torch.softmax(logits, dim=1).to(torch.float32)
    del logits

    return Workload(
        spec=spec, seed=seed, queries=queries.contiguous(), keys=keys, values=values,
        key_offsets=torch.from_numpy(ko).to(device), query_offsets=torch.from_numpy(qo).to(device),
        p_lm=p_lm.contiguous(), key_offsets_host=ko, query_offsets_host=qo, planted_ids=planted,
    )


def _llama(name, B, d, S, n_keys, dtype="bf16", V=32000, r=1024, lam=0.3, **kw) -> Spec:
    return Spec(name=name, B=B, d=d, S=S, n_keys=n_keys, dtype=dtype, key_scale=8.0 / math.sqrt(d),
                values="zipf", zipf_s=1.1, V=V, logit_sigma=2.0, r=r, mu=1.0 / math.sqrt(d), lam=lam, **kw)


CONFIGS = {
    # 4 queries on one shared fp32 store, small enough for the oracle in seconds.
    "tiny": Spec(name="tiny", B=4, d=256, S=1, n_keys=16384, dtype="f32", key_scale=1.0,
                 values="uniform", zipf_s=0.0, V=32000, logit_sigma=1.0, r=64, mu=1.0 / 16, lam=0.5),
    # Llama-2-7B-shaped single-query decode: 64 passages x 1024 tokens.
    "decode_7b": _llama("decode_7b", B=1, d=4096, S=1, n_keys=65536),
    # 64 sequences, each with its own store of 8K..64K keys.
    "ragged_batch": _llama("ragged_batch", B=64, d=4096, S=64, n_keys=("uniform", 8192, 65536)),
    # Llama-2-70B-shaped: 16 queries, each with its own 128-passage store.
    "decode_70b": _llama("decode_70b", B=16, d=8192, S=16, n_keys=131072),
    # Speculative verification: 8 sequences x 16 draft positions on their sequence's store.
    "specverify_seq": _llama("specverify_seq", B=128, d=8192, S=8, n_keys=262144),
    # The same 128 queries projected to 1024 dims against a static shared fp16 store.
    "specverify_static": _llama("specverify_static", B=128, d=1024, S=1, n_keys=8 * 1024 * 1024, dtype="f16",
                                query_mode="projected", proj_in=8192, proj_seed=5),
}

CONFIG_SEEDS = {"tiny": 1, "decode_7b": 2, "ragged_batch": 3, "decode_70b": 4,
                "specverify_seq": 5, "specverify_static": 6}


def config(name: str) -> Spec:
    return CONFIGS[name]


def scaled(spec: Spec, **overrides) -> Spec:
    return spec.replace(**overrides)


def extra_queries(spec: Spec, seed: int, n: int, device="cpu") -> torch.Tensor:
    """n further query rows drawn like the workload's i.i.d. queries (sub-stream +700)."""
    return _draw_normal_rows(n, spec.d, spec.key_scale, DTYPES[spec.dtype], torch.device(device),
                             _gen(torch.device(device), seed + 700))


def second_key_copy(spec: Spec, seed: int, device="cpu") -> torch.Tensor:
    """Another key matrix of the same shape and law (sub-stream +800), used to rotate
    buffers so that repeated timed calls cannot be served from the 256 MB last-level cache."""
    sizes = _set_sizes(spec, seed)
    return _draw_normal_rows(int(sum(sizes)), spec.d, spec.key_scale, DTYPES[spec.dtype], torch.device(device),
                             _gen(torch.device(device), seed + 800))
