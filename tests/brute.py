"""Brute-force CTC by enumeration of every length-T label string (tiny inputs only).

Independent of the oracle's trellis recursion: alignments are found by applying
the collapse map (merge repeats, then drop blanks; Sec. 3.1) to every string in
C^T, and beam pruning is evaluated by scoring every arc with the best enumerated
alignment that uses it (App. B.3).
"""
from __future__ import annotations

import itertools
import math
from typing import Dict, List, Sequence, Tuple

import numpy as np


def collapse(pi: Sequence[int], blank: int) -> Tuple[int, ...]:
    out = []
    prev = None
    for c in pi:
        if c != prev:
            if c != blank:
                out.append(c)
        prev = c
    return tuple(out)


def valid_alignments(T: int, C: int, y: Sequence[int], blank: int) -> List[Tuple[int, ...]]:
    y = tuple(y)
    return [pi for pi in itertools.product(range(C), repeat=T) if collapse(pi, blank) == y]


def state_path(pi: Sequence[int], blank: int) -> List[int]:
    """Extended-label state of each frame: blank after k emitted labels -> 2k,
    k-th label (1-based) -> 2k-1."""
    states = []
    k = 0
    prev = None
    for c in pi:
        if c == blank:
            states.append(2 * k)
        else:
            if c != prev:
                k += 1
            states.append(2 * k - 1)
        prev = c
    return states


def arcs_of(pi: Sequence[int], blank: int) -> List[tuple]:
    s = state_path(pi, blank)
    arcs = [("start", s[0])]
    for t in range(1, len(s)):
        arcs.append(("tr", t, s[t - 1], s[t]))
    arcs.append(("final", s[-1]))
    return arcs


def brute_ctc(logp: np.ndarray, y: Sequence[int], blank: int, beam: float = math.inf,
              slack: float = 0.0) -> Dict[str, object]:
    """log P over (retained) alignments and occupancies gamma[t, c]."""
    T, C = logp.shape
    aligns = valid_alignments(T, C, y, blank)
    if not aligns:
        return {"logP": -math.inf, "gamma": np.zeros((T, C)), "n_align": 0, "n_kept": 0}
    scores = [float(sum(logp[t, pi[t]] for t in range(T))) for pi in aligns]
    if math.isfinite(beam) and beam >= 0:
        best_through: Dict[tuple, float] = {}
        for pi, sc in zip(aligns, scores):
            for a in arcs_of(pi, blank):
                best_through[a] = max(best_through.get(a, -math.inf), sc)
        best = max(scores)
        kept_arcs = {a for a, v in best_through.items() if v >= best - beam - slack}
        keep = [all(a in kept_arcs for a in arcs_of(pi, blank)) for pi in aligns]
    else:
        keep = [True] * len(aligns)
    ks = [sc for sc, k in zip(scores, keep) if k]
    m = max(ks)
    logP = m + math.log(sum(math.exp(s - m) for s in ks))
    gamma = np.zeros((T, C))
    for pi, sc, k in zip(aligns, scores, keep):
        if k:
            w = math.exp(sc - logP)
            for t in range(T):
                gamma[t, pi[t]] += w
    return {"logP": logP, "gamma": gamma, "n_align": len(aligns), "n_kept": sum(keep),
            "scores": scores}
