"""CPU ORACLE for the decoding decisions of one NEST step -- TEST INFRASTRUCTURE ONLY.

Used by the tests, the smoke check and the benchmark's CPU-baseline leg, and by
nothing else; it shares no code with the HIP library.  Plain per-row Python
over numpy arrays, written from the paper:

* greedy next token (Algorithm 1, dynamic span selection): w_t is the token
  with the largest p_M; equal maxima go to the lowest token id.
* span start (Section 3.3, eq. knn_interpolation, max-pooling): among the
  neighbours in pi whose value is w_t, the one with the largest softmax weight,
  i.e. the nearest; equal distances go to the lower key id, which is pi's own
  order.  The paper's p_kNN(w = w_i) is the same for every such neighbour, so
  the pooling is read as over the neighbours' own weights.  No such neighbour:
  -1 (w_t came from p_LM alone and has no continuation in the store).
* span or token (eq. span_expansion): the span when lambda_t <= delta, the
  single token when lambda_t > delta; a span needs a start, so without one the
  token is taken.
* relaxed speculative verification (Section 3.4, eq. rejection, and
  Algorithm 1): draft row i carries p_M(. | prefix, w^(1..i-1)) and the draft
  token w^(i) it checks; ratio_i = p_M(w^(i)) / (gamma * max_w p_M(w)).  With
  no random numbers given, a draft token is accepted while ratio_i > 0.5 (the
  algorithm's threshold); with uniforms u_i given, it is accepted when
  u_i < min(1, ratio_i) (the equation read as a probability).  The first
  rejected row i* ends the draft: i* - first row tokens are accepted and the
  rejected one is replaced by the argmax of its row.  With no rejection every
  draft token is accepted and no replacement is made.

Parity rules: the decisions compare the same floating-point values, so the
tests evaluate them on the GPU's own fp32 p_M rows (fp32=True reproduces the
kernel's fp32 rounding of gamma * max and of the ratio), and check those rows
against the fp64 mixture separately.
"""
from __future__ import annotations

from typing import Optional

import numpy as np


def greedy_token(p_m_row: np.ndarray) -> int:
    """argmax_w p_M(w), the lowest id among equal maxima (Algorithm 1)."""
    return int(np.argmax(p_m_row))  # numpy returns the first maximal entry


def span_start(ids_row: np.ndarray, values_set: np.ndarray, w_t: int) -> int:
    """Key id of the nearest neighbour in pi whose value is w_t, else -1 (eq. knn_interpolation).
    ids_row is pi in ascending (distance, id) order; -1 entries are absent neighbours."""
    for i in ids_row:
        if i >= 0 and int(values_set[i]) == w_t:
            return int(i)
    return -1


def use_span(lambda_t: float, delta: float, start: int) -> int:
    """1 when the step outputs the n-gram from `start` (lambda_t <= delta, eq. span_expansion)."""
    return int(lambda_t <= delta and start >= 0)


def decode_outputs(p_m: np.ndarray, ids: np.ndarray, values: np.ndarray, key_offsets: np.ndarray,
                   query_offsets: np.ndarray, lambdas: np.ndarray, delta: float,
                   draft_tokens: Optional[np.ndarray] = None) -> dict:
    """Per query row: next token, max p_M, p_M of its draft token, span start and the span flag."""
    B = p_m.shape[0]
    out = {"next_token": np.empty(B, np.int32), "p_max": np.empty(B, p_m.dtype),
           "p_draft": np.full(B, np.nan, p_m.dtype), "span_key": np.empty(B, np.int32),
           "use_span": np.empty(B, np.int32)}
    for s in range(len(key_offsets) - 1):
        vals = values[key_offsets[s]:key_offsets[s + 1]]
        for b in range(int(query_offsets[s]), int(query_offsets[s + 1])):
            w = greedy_token(p_m[b])
            out["next_token"][b] = w
            out["p_max"][b] = p_m[b, w]
            if draft_tokens is not None:  # a token outside [0, V) has probability 0
                dt = int(draft_tokens[b])
                out["p_draft"][b] = p_m[b, dt] if 0 <= dt < p_m.shape[1] else 0.0
            k = span_start(ids[b], vals, w)
            out["span_key"][b] = k
            out["use_span"][b] = use_span(float(lambdas[b]), delta, k)
    return out


def accept_ratio(p_draft: float, p_max: float, gamma: float, fp32: bool = False) -> float:
    """p_M(w^(i)) / (gamma * max_w p_M(w)) (eq. rejection, without the min with 1)."""
    if fp32:
        den = np.float32(np.float32(gamma) * np.float32(p_max))
        return float(np.float32(np.float32(p_draft) / den))
    return float(p_draft) / (float(gamma) * float(p_max))


def spec_verify(p_max: np.ndarray, p_draft: np.ndarray, next_token: np.ndarray, draft_offsets: np.ndarray,
                gamma: float, uniforms: Optional[np.ndarray] = None, fp32: bool = False):
    """Per draft (rows draft_offsets[j] .. draft_offsets[j+1]-1): (accepted count, replacement token or -1)."""
    n = len(draft_offsets) - 1
    n_accept = np.empty(n, np.int32)
    token = np.empty(n, np.int32)
    for j in range(n):
        r0, r1 = int(draft_offsets[j]), int(draft_offsets[j + 1])
        n_accept[j], token[j] = r1 - r0, -1
        for i in range(r0, r1):
            ratio = accept_ratio(p_draft[i], p_max[i], gamma, fp32)
            if uniforms is None:
                ok = ratio > 0.5
            else:
                u = np.float32(uniforms[i]) if fp32 else float(uniforms[i])
                ok = u < min(1.0, ratio)
            if not ok:
                n_accept[j], token[j] = i - r0, int(next_token[i])
                break
    return n_accept, token
