"""Parity rules between the HIP path and the CPU oracle (shared by the GPU tests,
the smoke check and the benchmark's sampled check).

P2  neighbour ids: the GPU id set G and the oracle id set O may differ only by
    keys whose oracle distance is within 1e-6 relative of the oracle's r-th
    distance (ties at the boundary; several answers are then correct).
P3  p_M: max |p_M^gpu - p_M^ref| <= 1e-5, where p_M^ref is the oracle mixture
    over the GPU's own id set with the oracle's fp64 distances of those ids
    (so a legitimate boundary swap does not count against p_M).
P4  distances: |d^gpu - d^oracle| <= max(1e-5 * max(1, d^oracle), bound), with
    bound the worst-case fp32 error of the expansion ||q||^2 - 2 q.k + ||k||^2:
    (words per lane + 8) * 2^-23 * (||q||^2 + ||k||^2).  The GPU's order is
    ascending by its own (distance, id).
P5  sum: |sum_w p_M^gpu - (lambda * sum p_LM + (1 - lambda))| <= 1e-5 (fp64 host sum).
P6  (relative retrieval confidence, Section 3.2 eq. rrc) lambda_t: |lambda_t^gpu -
    lambda_t^ref| <= (1 / (4 tau)) * dratio + 1e-6, where lambda_t^ref is the
    oracle's sigmoid((d_(1) / d_(r) - alpha) / tau) over the oracle's fp64
    distances of the GPU's ids, 1 / (4 tau) bounds the sigmoid's slope, and
    dratio = (e_1 + ratio * e_r) / d_(r) is what the P4 tolerances e_1, e_r of
    the first and r-th distance can move the ratio; 1e-6 covers the fp32
    division and sigmoid.  P3 and P5 then take the GPU's lambda_t as lambda.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

import oracle

PM_TOL = 1e-5
TIE_REL = 1e-6
DIST_REL = 1e-5


@dataclass
class Report:
    queries: int = 0
    exact_id_sets: int = 0
    boundary_swaps: int = 0
    max_pm_err: float = 0.0
    max_dist_err_ratio: float = 0.0
    max_sum_err: float = 0.0
    max_lambda_err_ratio: float = 0.0
    failures: List[str] = field(default_factory=list)

    def ok(self) -> bool:
        return not self.failures

    def summary(self) -> str:
        return (f"{self.queries} queries, {self.exact_id_sets} identical id sets, {self.boundary_swaps} boundary "
                f"swaps, max|dp_M|={self.max_pm_err:.3g}, max dist err/tol={self.max_dist_err_ratio:.3g}, "
                f"max|dsum|={self.max_sum_err:.3g}, max lambda_t err/tol={self.max_lambda_err_ratio:.3g}")


def dist_bound(d: int, dtype: str, qq: float, kk: float) -> float:
    per_word = 1 if dtype == "f32" else 2
    words_per_lane = math.ceil(math.ceil(d / per_word) / 64)
    return (words_per_lane + 8) * 2.0 ** -23 * (qq + kk)


def check_query(rep: Report, b: int, q_host: np.ndarray, keys_host: np.ndarray, dtype: str, values_set: np.ndarray,
                p_lm_row: np.ndarray, r: int, mu: float, lam: float, gpu_ids: np.ndarray, gpu_dists: np.ndarray,
                gpu_pm: np.ndarray, oracle_ids: Optional[np.ndarray] = None, oracle_dists: Optional[np.ndarray] = None,
                rrc: Optional[tuple] = None, gpu_lambda: Optional[float] = None):
    """Apply P2-P5 to one query b with its own key set (host element arrays); with
    rrc = (alpha, tau) and the GPU's lambda_t also P6, and P3 / P5 use that lambda_t."""
    n = keys_host.shape[0]
    d = q_host.shape[-1]
    q1 = q_host.reshape(1, d)
    if oracle_ids is None:
        oracle_ids, oracle_dists = oracle.select(q1, keys_host, dtype, np.array([0, n]), np.array([0, 1]), r)
        oracle_ids, oracle_dists = oracle_ids[0], oracle_dists[0]
    rep.queries += 1
    tag = f"query {b}"
    gi = gpu_ids.astype(np.int64)
    if gi.min() < 0 or gi.max() >= n:
        rep.failures.append(f"{tag}: GPU id out of range")
        return
    if len(set(gi.tolist())) != r:
        rep.failures.append(f"{tag}: GPU ids not distinct")
        return
    # oracle fp64 distances of the GPU's ids
    d_or = oracle.sqdist(q1, np.ascontiguousarray(keys_host[gi]), dtype)[0]
    # P2
    G, O = set(gi.tolist()), set(oracle_ids.astype(np.int64).tolist())
    d_r = float(oracle_dists[r - 1])
    sym = G.symmetric_difference(O)
    if not sym:
        rep.exact_id_sets += 1
    else:
        pos = {int(i): j for j, i in enumerate(gi)}
        for i in sym:
            di = d_or[pos[i]] if i in pos else float(oracle_dists[list(oracle_ids).index(i)])
            if abs(di - d_r) > TIE_REL * d_r:
                rep.failures.append(f"{tag}: id {i} (oracle dist {di!r}) differs from the oracle set beyond the "
                                    f"tie window around d_r={d_r!r}")
                break
        rep.boundary_swaps += len(sym) // 2
    # P4 + order
    qq = float(oracle.sqdist(q1, np.zeros_like(q1), dtype)[0, 0])
    kk = oracle.sqdist(np.ascontiguousarray(keys_host[gi]), np.zeros_like(q1), dtype)[:, 0]
    for j in range(r):
        tol = max(DIST_REL * max(1.0, d_or[j]), dist_bound(d, dtype, qq, float(kk[j])))
        err = abs(float(gpu_dists[j]) - d_or[j])
        rep.max_dist_err_ratio = max(rep.max_dist_err_ratio, err / tol)
        if err > tol:
            rep.failures.append(f"{tag}: neighbour {j} id {gi[j]} distance {gpu_dists[j]!r} vs oracle {d_or[j]!r}")
            break
    # P6
    if rrc is not None:
        alpha, tau = rrc
        lam_ref = float(oracle.rrc_lambda(d_or.reshape(1, r), alpha, tau)[0])
        e1 = max(DIST_REL * max(1.0, d_or[0]), dist_bound(d, dtype, qq, float(kk[0])))
        er = max(DIST_REL * max(1.0, d_or[r - 1]), dist_bound(d, dtype, qq, float(kk[r - 1])))
        d1, dr = float(np.min(d_or)), float(np.max(d_or))
        dratio = (e1 + (d1 / dr) * er) / dr if dr > 0 else 0.0
        tol = dratio / (4.0 * tau) + 1e-6
        err = abs(float(gpu_lambda) - lam_ref)
        rep.max_lambda_err_ratio = max(rep.max_lambda_err_ratio, err / tol)
        if err > tol:
            rep.failures.append(f"{tag}: lambda_t {gpu_lambda!r} vs oracle {lam_ref!r} (tol {tol:.3g})")
        lam = float(gpu_lambda)
    gd = gpu_dists.astype(np.float64)
    order_ok = np.all((gd[1:] > gd[:-1]) | ((gd[1:] == gd[:-1]) & (gi[1:] > gi[:-1])))
    if not order_ok:
        rep.failures.append(f"{tag}: GPU neighbours not ascending by (distance, id)")
    # P3
    ids1 = gi.astype(np.int32).reshape(1, r)
    pm_ref = oracle.mix(ids1, d_or.reshape(1, r), values_set, np.array([0, n]), np.array([0, 1]),
                        p_lm_row.reshape(1, -1), mu, lam)[0]
    err = float(np.max(np.abs(gpu_pm.astype(np.float64) - pm_ref)))
    rep.max_pm_err = max(rep.max_pm_err, err)
    if err > PM_TOL:
        rep.failures.append(f"{tag}: max |p_M - ref| = {err:.3g}")
    # P5
    expect = lam * float(p_lm_row.astype(np.float64).sum()) + (1.0 - lam)
    serr = abs(float(gpu_pm.astype(np.float64).sum()) - expect)
    rep.max_sum_err = max(rep.max_sum_err, serr)
    if serr > PM_TOL:
        rep.failures.append(f"{tag}: sum p_M off by {serr:.3g}")


def host_threads() -> int:
    """Host threads the oracle may use here: the cores this process may run on, at most 16."""
    return max(1, min(16, oracle.default_threads()))


def oracle_select_rows(q_rows: np.ndarray, keys_host: np.ndarray, dtype: str, r: int,
                       threads: Optional[int] = None):
    """The oracle's (ids, fp64 dists) of each query row against one key set.

    With several rows, the rows run concurrently, each oracle call on its share
    of the threads (ctypes releases the GIL and the oracle keeps no state
    between calls); with one row, that row's key range is split over all of
    them.  Neither changes the oracle's arithmetic."""
    from concurrent.futures import ThreadPoolExecutor

    threads = threads or host_threads()
    nq = q_rows.shape[0]
    n = keys_host.shape[0]
    workers = max(1, min(threads, nq))
    per = max(1, threads // workers)

    def one(i):
        ids, d = oracle.select(q_rows[i:i + 1], keys_host, dtype, np.array([0, n]), np.array([0, 1]), r,
                               nthreads=per)
        return ids[0], d[0]

    if workers == 1:
        return [one(i) for i in range(nq)]
    with ThreadPoolExecutor(max_workers=workers) as ex:
        return list(ex.map(one, range(nq)))


def check_workload(w, p_m, ids, dists, sample: Optional[List[int]] = None, rrc: Optional[tuple] = None,
                   lambdas=None, host_keys=None) -> Report:
    """P2-P5 on the queries `sample` (all by default) of a workload run on the GPU; with
    rrc = (alpha, tau) and the GPU's per-query lambdas, P6 too.  host_keys(s), if
    given, returns set s's key elements on the host (e.g. from a cache)."""
    rep = Report()
    ko, qo = w.key_offsets_host, w.query_offsets_host
    set_of = w.set_of_query()
    B = int(qo[-1])
    sample = list(range(B)) if sample is None else list(sample)
    ids_h, dists_h = ids.cpu().numpy(), dists.cpu().numpy()
    lam_h = None if lambdas is None else lambdas.cpu().numpy()
    by_set = {}
    for b in sample:
        by_set.setdefault(int(set_of[b]), []).append(b)
    for s, bs in by_set.items():
        if host_keys is not None:
            keys_h, dt = host_keys(s)
        else:
            keys_h, dt = oracle.host_elements(w.keys[ko[s]:ko[s + 1]])
        vals = w.values[ko[s]:ko[s + 1]].cpu().numpy()
        q_rows, _ = oracle.host_elements(w.queries[bs])
        refs = oracle_select_rows(q_rows, keys_h, dt, w.r)
        for j, b in enumerate(bs):
            check_query(rep, b, q_rows[j], keys_h, dt, vals, w.p_lm[b].cpu().numpy(), w.r, w.mu, w.lam, ids_h[b],
                        dists_h[b], p_m[b].cpu().numpy(), oracle_ids=refs[j][0], oracle_dists=refs[j][1], rrc=rrc,
                        gpu_lambda=None if lam_h is None else float(lam_h[b]))
        del keys_h
    return rep
