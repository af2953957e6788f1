"""Conditional drop-token (COD) training-data processing, sample by sample.

TEST INFRASTRUCTURE (see ``oracle/__init__.py``).

Paper passages followed:
* Sec. 3.2 (mask-token training, eq. 8): subtask k (k = 1..K) predicts the
  k-th next token; its loss term for label x_i conditions on the real tokens
  x_0..x_{i-k} and the mask tokens m_0..m_{k-2}.
* Sec. 3.2 (conditional drop, eqs. 9-11): subtask k keeps N_k' = N * max(r^{k-1},
  r_min) of its N tokens; in total N_COD = sum_k N_k' < N / (1 - r) (before
  the r_min floor).
* Alg. 1 and App. B: per sample and subtask, the retention rate is
  gamma_k = max(r^{k-1}, r_min); only tokens whose whole preceding key/value
  context is retained may be kept; among those, tokens are chosen at random;
  the kept tokens of all subtasks are merged into one sequence with updated
  ids, labels, positions and attention mask.  In the worked example (r = 0.5,
  4 columns) subtask 2 keeps m_{0,1}, m_{0,2}; in subtask 3 only m_{1,2} and
  m_{1,3} have their context (m_{1,1} would need the dropped m_{0,0}) and one
  of them is kept.

Readings where the paper is silent (each one is listed in the design notes):
* A sample of L tokens t_0..t_{L-1} gives n = L - 1 columns per subtask.
  Column j of subtask 1 is the real token t_j; column j of subtask k >= 2 is a
  mask token (the shared mask id) at position j.  Every column j is labelled
  t_{j+1}.  Column (k, j) attends to the real tokens t_0..t_{j-k+1} and to the
  columns (k', j - k + k') for k' = 2..k (the masks before it on its diagonal,
  then itself): the context eq. 8 and the inference pass of eq. 7 give it.
* Column (k, j), k >= 2, is valid iff j >= k - 1 (it has a real token) and
  column (k-1, j-1) is kept (subtask 1 keeps every column).
* Kept count c_k = min(#valid, floor(n * gamma_k + 1/2)), gamma_k from
  repeated float64 multiplication by r, then the max with r_min.
* Random choice: the c_k valid columns with the smallest (key, j), key the top
  24 bits of output j of the SplitMix64 stream seeded with output k of the
  stream seeded with output `sample` of the stream seeded with `seed`.
* Packed order: subtask 1's columns, then each later subtask's kept columns,
  each in column order.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence

import numpy as np

from .sampling import splitmix64_output

MASK64 = (1 << 64) - 1


def cod_key(seed: int, sample: int, k: int, j: int) -> int:
    """24-bit random key of column j of subtask k in sample `sample`."""
    z = splitmix64_output(seed & MASK64, sample)
    z = splitmix64_output(z, k)
    return splitmix64_output(z, j) >> 40


def retention(k: int, r: float, r_min: float) -> float:
    """gamma_k = max(r^(k-1), r_min) (Alg. 1), r^(k-1) by repeated multiplication."""
    g = 1.0
    for _ in range(k - 1):
        g *= float(r)
    return max(g, float(r_min))


def keep_target(n: int, k: int, r: float, r_min: float) -> int:
    """floor(n * gamma_k + 1/2): the number of columns subtask k aims to keep (eq. 11)."""
    return int(np.floor(n * retention(k, r, r_min) + 0.5))


@dataclass
class CodSample:
    ids: List[int]
    labels: List[int]
    pos: List[int]
    section: List[int]      # subtask k (1-based) of each packed token
    column: List[int]       # column j of each packed token
    kept: List[List[int]]   # kept columns of each subtask (1-based index - 1)


def cod_process(tokens: Sequence[int], k_max: int, r: float, r_min: float, mask_id: int, seed: int,
                sample: int) -> CodSample:
    """COD processing of one sample (Alg. 1): select, then pack."""
    t = [int(x) for x in tokens]
    n = len(t) - 1
    if n < 1 or k_max < 1:
        raise ValueError("need at least two tokens and K >= 1")
    kept = [list(range(n))]
    for k in range(2, k_max + 1):
        prev = set(kept[-1])
        valid = [j for j in range(n) if j >= k - 1 and (j - 1) in prev]
        c = min(len(valid), keep_target(n, k, r, r_min))
        ranked = sorted(valid, key=lambda j: (cod_key(seed, sample, k, j), j))
        kept.append(sorted(ranked[:c]))
    out = CodSample([], [], [], [], [], kept)
    for k, cols in enumerate(kept, start=1):
        for j in cols:
            out.ids.append(t[j] if k == 1 else mask_id)
            out.labels.append(t[j + 1])
            out.pos.append(j)
            out.section.append(k)
            out.column.append(j)
    return out


def attends(ka: int, ja: int, kb: int, jb: int) -> bool:
    """Whether packed token (ka, ja) attends to (kb, jb): real tokens
    t_0..t_{ja-ka+1}, and the columns on its diagonal up to itself."""
    if kb == 1:
        return jb <= ja - ka + 1
    return kb <= ka and jb - kb == ja - ka


def attention_mask(s: CodSample) -> np.ndarray:
    """Dense boolean mask of a packed sample (row attends to column)."""
    m = len(s.ids)
    out = np.zeros((m, m), bool)
    for a in range(m):
        for b in range(m):
            out[a, b] = attends(s.section[a], s.column[a], s.section[b], s.column[b])
    return out
