"""Plain fp64 CPU oracle of the Pruned CTC head and loss (forward and backward).

TEST INFRASTRUCTURE ONLY: used by tests/, the build entry point's smoke check
and the benchmark's CPU-baseline leg; never by the product path.

What it computes, with the passage each step follows:

* Union subset and relabelling (Sec. 3.2 "Reformulation"; Algorithm 1, union and
  relabel steps; App. B.1 "Forward computation"): the selected classes are blank
  followed by the sorted distinct target labels of the whole batch; each target
  is relabelled by its index in that list.
* Full-vocabulary normaliser lambda_m = log sum_v exp Z_{m,v} with Z = H W^T
  (Eq. "lognorm"), accumulated over vocabulary chunks as Algorithm 1's online
  log-sum-exp does.
* Standard CTC over the extended label sequence (Sec. 3.1, Eq. "ctc"):
  alignments are the length-T label strings that collapse to y (merge repeats,
  then drop blanks).  The recursion over the 2U+1 extended states is the
  textbook one of Graves et al. (2006), in log space.
* Finite-beam pruning (Sec. 3.3, App. B.3 "Alignment pruning"): every trellis
  arc is scored by the best alignment through it; arcs scoring below the best
  alignment minus beta are dropped, and the loss sums over the alignments whose
  arcs are all kept (Eq. "pruned-ctc").
* Loss aggregation (App. B.1 "Loss aggregation"): an utterance is structurally
  alignable iff T_n >= U_n + r_n (r_n = adjacent identical label pairs);
  excluded or nonfinite utterances contribute zero loss and zero gradient.
* Gradient dL/dZ_{m,v} = p_v(m) - gamma_v(m) (Eq. "grad-full"; for a pruned
  lattice held fixed, gamma is the occupancy over retained alignments, Sec. 3.3),
  formed as written in fwd_bwd, and the head gradients dX = dZ W, dW = dZ^T X
  (App. A, end of Step 3).  The recomputed form scatter_U(G) - g p of Eq. "vjp" is
  the separate stage function head_backward.

Everything is float64.  Inputs are taken exactly as the device sees them (bf16
values are exact in float32, and float32 is exact in float64).
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence

import numpy as np

# Status codes shared in meaning (not in code) with the C ABI.
PCTC_OK = 0
PCTC_EINVAL = -1
PCTC_ELABEL = -2
PCTC_ELENGTH = -3

STATUS_OK = 0
STATUS_NOT_ALIGNABLE = 1
STATUS_NONFINITE = 2


def beam_round_tol(E: np.ndarray) -> float:
    """Rounding allowance of the beam rule for one utterance (E [T, S']: per-frame scores).

    The rule of App. B.3 compares the best alignment through an arc with the best alignment
    overall.  Both are sums of T per-frame scores, evaluated here in different orders (the
    forward recursion up to the arc, the backward one after it).  Recursive summation of T
    terms in float64 errs by at most (T - 1) u sum|x| (u = 2^-53), so two evaluations of the
    same path score differ by at most 2 T u A with A = sum_t max_s |E_t(s)|.  Twice that
    (4 T u A) is allowed: it keeps the best alignment's own arcs at beta = 0 and is far below
    any margin the tests use; it is not a tolerance of the method."""
    fin = np.where(np.isfinite(E), np.abs(E), 0.0)
    A = float(fin.max(axis=1).sum()) if fin.size else 0.0
    return 4.0 * E.shape[0] * 2.0 ** -53 * max(A, 1.0)


class OracleError(ValueError):
    def __init__(self, code: int, msg: str):
        super().__init__(msg)
        self.code = code


def beam_enabled(beam: float) -> bool:
    """A finite, non-negative beam prunes; +inf or a negative value keeps all alignments."""
    return bool(np.isfinite(beam) and beam >= 0.0)


def validate(N: int, input_lengths, target_lengths, targets, D: int, V: int, blank: int,
             beam: float) -> None:
    """Argument checks in the order the C ABI applies them."""
    if N < 0 or D <= 0 or V <= 1 or not (0 <= blank < V) or math.isnan(beam):
        raise OracleError(PCTC_EINVAL, "bad sizes, blank or beam")
    T = np.asarray(input_lengths)
    U = np.asarray(target_lengths)
    if T.shape[0] != N or U.shape[0] != N:
        raise OracleError(PCTC_EINVAL, "length arrays do not have N entries")
    if (T <= 0).any() or (U < 0).any():
        raise OracleError(PCTC_ELENGTH, "T_n must be >= 1 and U_n >= 0")
    y = np.asarray(targets)
    if y.shape[0] != int(U.sum()):
        raise OracleError(PCTC_EINVAL, "targets length differs from sum of target lengths")
    if y.size and ((y < 0).any() or (y >= V).any() or (y == blank).any()):
        raise OracleError(PCTC_ELABEL, "label out of range or equal to blank")


# ---------------------------------------------------------------------------------------
# Union subset, remap, relabelled targets (Sec. 3.2; Algorithm 1; App. B.1)
# ---------------------------------------------------------------------------------------

def union_remap(targets, target_lengths, blank: int, V: int) -> Dict[str, np.ndarray]:
    """U = [blank] + sorted(distinct labels); remap[v] = index of v in U or -1; y_rel = remap[y]."""
    distinct = sorted(set(int(v) for v in np.asarray(targets).tolist()))
    u_ids = [int(blank)] + distinct
    remap = np.full(V, -1, dtype=np.int64)
    for j, v in enumerate(u_ids):
        remap[v] = j
    y = np.asarray(targets, dtype=np.int64)
    y_rel = remap[y] if y.size else np.zeros(0, np.int64)
    return {"u_ids": np.array(u_ids, np.int64), "remap": remap, "y_rel": y_rel,
            "K": len(u_ids)}


# ---------------------------------------------------------------------------------------
# Normaliser and selected log-probabilities (Eq. lognorm; Algorithm 1)
# ---------------------------------------------------------------------------------------

def _bias(bias, V: int) -> np.ndarray:
    return np.zeros(V) if bias is None else np.asarray(bias, np.float64)


def log_normalizer(H, W, chunk: int = 4096, bias=None) -> np.ndarray:
    """lambda_m = log sum_v exp(Z_{m,v}), Z = H W^T + 1 b^T (Sec. 2 head (W, b)), combined
    online over vocabulary chunks."""
    H = np.asarray(H, np.float64)
    W = np.asarray(W, np.float64)
    b = _bias(bias, W.shape[0])
    M = H.shape[0]
    run_max = np.full(M, -np.inf)
    run_sum = np.zeros(M)
    for v0 in range(0, W.shape[0], chunk):
        Z = H @ W[v0:v0 + chunk].T + b[v0:v0 + chunk]
        cmax = Z.max(axis=1)
        new_max = np.maximum(run_max, cmax)
        safe = np.where(np.isfinite(new_max), new_max, 0.0)
        with np.errstate(invalid="ignore"):
            run_sum = run_sum * np.exp(run_max - safe) + np.exp(Z - safe[:, None]).sum(axis=1)
        run_max = new_max
    with np.errstate(divide="ignore", invalid="ignore"):
        return np.where(np.isfinite(run_max), run_max + np.log(run_sum), run_max)


def selected_logprobs(H, W, u_ids, lam, bias=None) -> np.ndarray:
    """S = X W_U^T + 1 b_U^T - lambda 1^T: the log-probabilities of the selected classes
    (Algorithm 1)."""
    H = np.asarray(H, np.float64)
    u = np.asarray(u_ids)
    Wu = np.asarray(W, np.float64)[u]
    bu = _bias(bias, np.asarray(W).shape[0])[u]
    return H @ Wu.T + bu - np.asarray(lam, np.float64)[:, None]


# ---------------------------------------------------------------------------------------
# CTC over the extended label sequence, optionally beam-pruned (Sec. 3.1, 3.3; App. B.3)
# ---------------------------------------------------------------------------------------

def extended_labels(y: Sequence[int], blank_col: int):
    """l' = (blank, y_1, blank, ..., y_U, blank) and, per state, whether the skip arc
    s-2 -> s exists (l'_s is a label different from l'_{s-2})."""
    y = [int(v) for v in y]
    ext = [blank_col]
    for v in y:
        ext += [v, blank_col]
    S = len(ext)
    skip_ok = np.zeros(S, bool)
    for s in range(2, S):
        skip_ok[s] = (ext[s] != blank_col) and (ext[s] != ext[s - 2])
    return np.array(ext, np.int64), skip_ok


def _combine(op: str, *xs: np.ndarray) -> np.ndarray:
    """Elementwise max (Viterbi) or log-sum-exp (total probability) with -inf handled."""
    m = xs[0]
    for x in xs[1:]:
        m = np.maximum(m, x)
    if op == "max":
        return m
    fin = np.isfinite(m)
    safe = np.where(fin, m, 0.0)
    acc = np.zeros_like(m)
    for x in xs:
        with np.errstate(invalid="ignore"):
            acc = acc + np.exp(x - safe)
    with np.errstate(divide="ignore", invalid="ignore"):
        return np.where(fin, safe + np.log(acc), m)


def _shift_right(a: np.ndarray, k: int) -> np.ndarray:
    out = np.full_like(a, -np.inf)
    if k < a.shape[-1]:
        out[..., k:] = a[..., :a.shape[-1] - k]
    return out


def _shift_left(a: np.ndarray, k: int, fill) -> np.ndarray:
    out = np.full_like(a, fill)
    if k < a.shape[-1]:
        out[..., :a.shape[-1] - k] = a[..., k:]
    return out


def _recursions(E: np.ndarray, skip_ok: np.ndarray, keep: Dict[str, np.ndarray], op: str):
    """Forward and backward recursions over the trellis with per-arc keep flags.

    E[t, s] is the log-probability of extended state s at frame t (0-based t).
    alpha[t, s]: combined score of partial alignments ending in s at t, including E[t, s].
    beta[t, s]: combined score of continuations from (t, s) to the end, excluding E[t, s].
    Arcs: start -> (0, s); (t-1, s) -> (t, s) "stay"; (t-1, s-1) -> (t, s) "step";
    (t-1, s-2) -> (t, s) "skip" (only where skip_ok); (T-1, s) -> end "final".
    """
    T, S = E.shape
    NEG = -np.inf
    alpha = np.full((T, S), NEG)
    beta = np.full((T, S), NEG)
    alpha[0] = np.where(keep["start"], E[0], NEG)
    for t in range(1, T):
        a = alpha[t - 1]
        stay = np.where(keep["stay"][t], a, NEG)
        step = np.where(keep["step"][t], _shift_right(a, 1), NEG)
        skip = np.where(keep["skip"][t] & skip_ok, _shift_right(a, 2), NEG)
        alpha[t] = E[t] + _combine(op, stay, step, skip)
    beta[T - 1] = np.where(keep["final"], 0.0, NEG)
    for t in range(T - 2, -1, -1):
        nxt = E[t + 1] + beta[t + 1]
        stay = np.where(keep["stay"][t + 1], nxt, NEG)
        step = np.where(_shift_left(keep["step"][t + 1], 1, False), _shift_left(nxt, 1, NEG), NEG)
        skip_arc = _shift_left(keep["skip"][t + 1] & skip_ok, 2, False)
        skip = np.where(skip_arc, _shift_left(nxt, 2, NEG), NEG)
        beta[t] = _combine(op, stay, step, skip)
    final_scores = np.where(keep["final"], alpha[T - 1], NEG)
    total = _combine(op, *[final_scores[s:s + 1] for s in range(S)])[0]
    return alpha, beta, total


def _all_arcs(T: int, S: int) -> Dict[str, np.ndarray]:
    start = np.zeros(S, bool)
    start[0] = True
    if S > 1:
        start[1] = True
    final = np.zeros(S, bool)
    final[S - 1] = True
    if S > 1:
        final[S - 2] = True
    stay = np.ones((T, S), bool)
    step = np.ones((T, S), bool)
    step[:, 0] = False
    skip = np.ones((T, S), bool)
    skip[:, :2] = False
    return {"start": start, "final": final, "stay": stay, "step": step, "skip": skip}


def ctc_utterance(logp: np.ndarray, y: Sequence[int], blank_col: int, beam: float = math.inf,
                  slack: float = 0.0) -> Dict[str, object]:
    """CTC (or beam-pruned CTC) for one utterance.

    logp: [T, C] log-probabilities over some column space; y: labels in that space;
    blank_col: the blank's column.  Returns log P (log of the retained alignment sum),
    per-state occupancies gamma [T, 2U+1], the extended labels, the arc keep flags and,
    when pruning, the signed margin of every arc's decision (through-score minus
    (best - beta); the arc is kept iff its margin >= -(rounding allowance + slack)).

    The paper's rule is slack = 0.  A non-zero slack moves the threshold by that many nats
    (positive keeps more arcs); tests use it only to bracket a device result whose own
    threshold carries a stated tolerance.
    """
    logp = np.asarray(logp, np.float64)
    T = logp.shape[0]
    ext, skip_ok = extended_labels(y, blank_col)
    S = ext.size
    U = len(y)
    r = sum(1 for i in range(1, U) if y[i] == y[i - 1])
    out: Dict[str, object] = {"ext": ext, "skip_ok": skip_ok, "alignable": T >= U + r}
    E = logp[:, ext]
    keep = _all_arcs(T, S)
    margins = None
    if beam_enabled(beam):
        va, vb, vbest = _recursions(E, skip_ok, keep, "max")
        thr = vbest - beam
        allow = beam_round_tol(E) + slack
        margins = {}
        with np.errstate(invalid="ignore"):
            margins["start"] = np.where(keep["start"], E[0] + vb[0] - thr, -np.inf)
            margins["final"] = np.where(keep["final"], va[T - 1] - thr, -np.inf)
            through_in = E[1:] + vb[1:]
            margins["stay"] = np.full((T, S), -np.inf)
            margins["step"] = np.full((T, S), -np.inf)
            margins["skip"] = np.full((T, S), -np.inf)
            if T > 1:
                margins["stay"][1:] = va[:-1] + through_in - thr
                margins["step"][1:] = _shift_right(va[:-1], 1) + through_in - thr
                margins["skip"][1:] = np.where(skip_ok, _shift_right(va[:-1], 2) + through_in - thr,
                                               -np.inf)
        keep = {k: keep[k] & (margins[k] >= -allow) for k in keep}
        out["viterbi_best"] = vbest
    alpha, beta, logP = _recursions(E, skip_ok, keep, "lse")
    with np.errstate(invalid="ignore", over="ignore"):
        gamma = np.exp(alpha + beta - logP) if np.isfinite(logP) else np.zeros((T, S))
    out.update({"logP": logP, "alpha": alpha, "beta": beta, "gamma": gamma, "keep": keep,
                "margins": margins})
    return out


def _offsets(lengths) -> np.ndarray:
    lengths = np.asarray(lengths, np.int64)
    off = np.zeros(lengths.size + 1, np.int64)
    off[1:] = np.cumsum(lengths)
    return off


def ctc_from_scores(S: np.ndarray, y_rel, input_lengths, target_lengths, beam: float = math.inf,
                    slack: float = 0.0, weights=None) -> Dict[str, object]:
    """The alignment stage alone: given per-frame scores S [M, K] over the selected classes
    (blank = column 0) and relabelled targets, return per-utterance losses, statuses, the
    occupancy-derived G = dL/dS (G[m, j] = -gamma over the states labelled j; zero for
    excluded utterances, Algorithm 1 output) and its row sums g."""
    S = np.asarray(S, np.float64)
    M, K = S.shape
    toff = _offsets(input_lengths)
    yoff = _offsets(target_lengths)
    N = len(input_lengths)
    loss_n = np.zeros(N)
    status = np.zeros(N, np.int64)
    G = np.zeros((M, K))
    per_utt: List[Dict[str, object]] = []
    for n in range(N):
        rows = slice(int(toff[n]), int(toff[n + 1]))
        y = [int(v) for v in np.asarray(y_rel)[yoff[n]:yoff[n + 1]]]
        res = ctc_utterance(S[rows], y, 0, beam, slack)
        per_utt.append(res)
        if not res["alignable"]:
            status[n] = STATUS_NOT_ALIGNABLE
            continue
        if not np.isfinite(res["logP"]):
            status[n] = STATUS_NONFINITE
            continue
        loss_n[n] = -res["logP"]
        gam = res["gamma"]
        ext = res["ext"]
        w = 1.0 if weights is None else float(weights[n])
        for s in range(ext.size):
            G[rows, ext[s]] -= w * gam[:, s]
    g = G.sum(axis=1)
    wv = np.ones(N) if weights is None else np.asarray(weights, np.float64)
    return {"loss_n": loss_n, "status": status, "G": G, "g": g, "per_utt": per_utt,
            "loss": float((wv * loss_n).sum())}


def discarded_mass(S: np.ndarray, y_rel, input_lengths, target_lengths, beams,
                   slack: float = 0.0) -> np.ndarray:
    """Discarded posterior mass (App. B.3): delta[b, n] = 1 - exp(-(L_beta,n - L_n)) for each
    beam, the posterior mass (given the transcript) of the alignments the beam drops, from
    the pruned and unpruned losses on the same scores (fp64), evaluated as
    -expm1(-Delta).  NaN for utterances that are not alignable."""
    S = np.asarray(S, np.float64)
    toff = _offsets(input_lengths)
    yoff = _offsets(target_lengths)
    N = len(input_lengths)
    beams = list(beams)
    out = np.full((len(beams), N), np.nan)
    for n in range(N):
        rows = slice(int(toff[n]), int(toff[n + 1]))
        y = [int(v) for v in np.asarray(y_rel)[yoff[n]:yoff[n + 1]]]
        full = ctc_utterance(S[rows], y, 0, math.inf, slack)
        if not full["alignable"] or not np.isfinite(full["logP"]):
            continue
        for b, beam in enumerate(beams):
            pr = ctc_utterance(S[rows], y, 0, beam, slack)
            out[b, n] = -math.expm1(-(full["logP"] - pr["logP"]))
    return out


def head_backward(H, W, lam, G, g, u_ids, chunk: int = 4096, bias=None) -> Dict[str, np.ndarray]:
    """The recomputed backward stage alone (Eq. vjp; Algorithm 1 backward loop):
    dZ[m, v] = scatter_U(G)[m, v] - g_m p_v(m) with p_v(m) = exp(Z[m, v] - lambda_m),
    formed one vocabulary chunk at a time, then dH = dZ W, dW = dZ^T H and db = dZ^T 1
    (the gradients w.r.t. X, W and b by the chain rule, App. A).  A frame with g_m = 0
    belongs to an excluded utterance and contributes nothing."""
    H = np.asarray(H, np.float64)
    W = np.asarray(W, np.float64)
    b = _bias(bias, W.shape[0])
    lam = np.asarray(lam, np.float64)
    G = np.asarray(G, np.float64)
    g = np.asarray(g, np.float64)
    M, D = H.shape
    V = W.shape[0]
    inc = g != 0
    dH = np.zeros((M, D))
    dW = np.zeros((V, D))
    db = np.zeros(V)
    col = {int(v): j for j, v in enumerate(np.asarray(u_ids).tolist())}
    for v0 in range(0, V, chunk):
        v1 = min(V, v0 + chunk)
        Z = H[inc] @ W[v0:v1].T + b[v0:v1]
        dZ = -g[inc, None] * np.exp(Z - lam[inc, None])
        for v in range(v0, v1):
            j = col.get(v)
            if j is not None:
                dZ[:, v - v0] += G[inc, j]
        dH[inc] += dZ @ W[v0:v1]
        dW[v0:v1] = dZ.T @ H[inc]
        db[v0:v1] = dZ.sum(axis=0)
    return {"dH": dH, "dW": dW, "db": db}


def head_backward_rows(H, W, lam, G, g, u_ids, frames, classes, chunk: int = 4096, bias=None) -> Dict[str, np.ndarray]:
    """Selected outputs of the recomputed backward (Eq. vjp), each over its full contraction:
    dH[m] = sum_v dZ[m, v] W[v] for the given frames (every class v) and
    dW[v] = sum_m dZ[m, v] H[m] for the given classes (every frame m), with
    dZ[m, v] = scatter_U(G)[m, v] - g_m exp(Z[m, v] - lambda_m) as in head_backward."""
    H = np.asarray(H, np.float64)
    W = np.asarray(W, np.float64)
    lam = np.asarray(lam, np.float64)
    G = np.asarray(G, np.float64)
    g = np.asarray(g, np.float64)
    frames = np.asarray(frames, np.int64)
    classes = np.asarray(classes, np.int64)
    V = W.shape[0]
    b = _bias(bias, V)
    col = {int(v): j for j, v in enumerate(np.asarray(u_ids).tolist())}

    def dz(rows: np.ndarray, vs: np.ndarray) -> np.ndarray:
        Z = H[rows] @ W[vs].T + b[vs]
        with np.errstate(invalid="ignore", over="ignore"):
            out = -g[rows, None] * np.exp(Z - lam[rows, None])
        for i, v in enumerate(vs.tolist()):
            j = col.get(int(v))
            if j is not None:
                out[:, i] += G[rows, j]
        out[g[rows] == 0] = 0.0
        return out

    dH = np.zeros((frames.size, H.shape[1]))
    for v0 in range(0, V, chunk):
        vs = np.arange(v0, min(V, v0 + chunk))
        dH += dz(frames, vs) @ W[vs]
    inc = np.nonzero(g != 0)[0]
    dzc = dz(inc, classes)
    return {"dH": dH, "dW": dzc.T @ H[inc], "db": dzc.sum(axis=0)}


# ---------------------------------------------------------------------------------------
# Whole path: loss and head gradients by the full-vocabulary definition
# ---------------------------------------------------------------------------------------

def fwd_bwd(H, W, targets, input_lengths, target_lengths, blank: int, beam: float = math.inf,
            chunk: int = 4096, want_grads: bool = True, slack: float = 0.0, bias=None,
            weights=None) -> Dict[str, object]:
    """Loss and gradients of (beam-pruned) CTC on log-softmax(H W^T + 1 b^T) over the full
    vocabulary (Sec. 2 head (W, b); Eqs. lognorm, ctc, pruned-ctc).

    Returns loss = sum_n w_n L_n over alignable utterances with finite loss (w_n = 1 unless
    `weights` is given: a per-utterance loss weight, e.g. one over the target-token count),
    the unweighted loss_n, status, dH [M, D], dW [V, D], db [V] (gradients of that weighted
    sum) and the stages u_ids, remap, y_rel, lam, S, G, g.
    """
    H = np.asarray(H, np.float64)
    W = np.asarray(W, np.float64)
    M, D = H.shape
    V = W.shape[0]
    targets = np.asarray(targets, np.int64)
    N = len(input_lengths)
    validate(N, input_lengths, target_lengths, targets, D, V, blank, beam)
    if int(np.sum(input_lengths)) != M:
        raise OracleError(PCTC_EINVAL, "H rows differ from the sum of input lengths")
    un = union_remap(targets, target_lengths, blank, V)
    b = _bias(bias, V)
    wv = np.ones(N) if weights is None else np.asarray(weights, np.float64)
    lam = log_normalizer(H, W, chunk, bias=b)
    Ssel = selected_logprobs(H, W, un["u_ids"], lam, bias=b)
    toff = _offsets(input_lengths)
    yoff = _offsets(target_lengths)
    loss_n = np.zeros(N)
    status = np.zeros(N, np.int64)
    included = np.zeros(M, bool)
    per_utt = []
    for n in range(N):
        rows = slice(int(toff[n]), int(toff[n + 1]))
        y = [int(v) for v in targets[yoff[n]:yoff[n + 1]]]
        # log p_v(m) on the columns this utterance's alignments can use (Eq. lognorm)
        cols = np.array([blank] + sorted(set(y)), np.int64)
        logp_cols = H[rows] @ W[cols].T + b[cols] - lam[rows, None]
        col_of = {int(v): i for i, v in enumerate(cols)}
        res = ctc_utterance(logp_cols, [col_of[v] for v in y], 0, beam, slack)
        res["cols"] = cols
        per_utt.append(res)
        if not res["alignable"]:
            status[n] = STATUS_NOT_ALIGNABLE
        elif not np.isfinite(res["logP"]):
            status[n] = STATUS_NONFINITE
        else:
            loss_n[n] = -res["logP"]
            included[rows] = True
    # G over the selected classes (the alignment stage's output) and its row sums
    G = np.zeros((M, un["K"]))
    for n in range(N):
        if status[n] != STATUS_OK:
            continue
        rows = slice(int(toff[n]), int(toff[n + 1]))
        res = per_utt[n]
        ext_ids = res["cols"][res["ext"]]
        for s in range(ext_ids.size):
            G[rows, un["remap"][ext_ids[s]]] -= wv[n] * res["gamma"][:, s]
    out = {"loss": float((wv * loss_n).sum()), "loss_n": loss_n, "status": status,
           "u_ids": un["u_ids"], "remap": un["remap"], "y_rel": un["y_rel"], "K": un["K"],
           "lam": lam, "S": Ssel, "G": G, "g": G.sum(axis=1), "per_utt": per_utt,
           "included": included}
    if not want_grads:
        return out
    # Eq. grad-full: dL/dZ[m, v] = w_n (p_v(m) - gamma_v(m)) for a frame m of an included
    # utterance n (zero on the frames of excluded ones), with gamma_v(m) the occupancy of
    # class v at frame m summed over the states labelled v; dense over V, one chunk at a time.
    w_frame = np.zeros(M)
    for n in range(N):
        if status[n] == STATUS_OK:
            w_frame[int(toff[n]):int(toff[n + 1])] = wv[n]
    occ_cols = []   # per included utterance: first frame, its class ids, gamma_v per class
    for n in range(N):
        if status[n] != STATUS_OK:
            continue
        res = per_utt[n]
        ext_ids = res["cols"][res["ext"]]
        classes = np.unique(ext_ids)
        occ = np.zeros((res["gamma"].shape[0], classes.size))
        for s in range(ext_ids.size):
            occ[:, int(np.searchsorted(classes, ext_ids[s]))] += res["gamma"][:, s]
        occ_cols.append((int(toff[n]), classes, occ))
    dH = np.zeros((M, D))
    dW = np.zeros((V, D))
    db = np.zeros(V)
    inc = included
    for v0 in range(0, V, chunk):
        v1 = min(V, v0 + chunk)
        p = np.exp(H[inc] @ W[v0:v1].T + b[v0:v1] - lam[inc, None])
        gam = np.zeros((M, v1 - v0))
        for t0, classes, occ in occ_cols:
            sel = (classes >= v0) & (classes < v1)
            gam[t0:t0 + occ.shape[0], classes[sel] - v0] = occ[:, sel]
        dZ = w_frame[inc, None] * (p - gam[inc])
        dH[inc] += dZ @ W[v0:v1]
        dW[v0:v1] = dZ.T @ H[inc]
        db[v0:v1] = dZ.sum(axis=0)
    out["dH"] = dH
    out["dW"] = dW
    out["db"] = db
    return out


# ---------------------------------------------------------------------------------------
# Grouped logits for unpruned reduced CTC through a stock CTC (Eq. grouped; Prop. 1;
# Eq. offsupport)
# ---------------------------------------------------------------------------------------

def grouped_logprobs(H, W, u_ids, bias=None, chunk: int = 4096) -> Dict[str, np.ndarray]:
    """log softmax of R [M, K+1]: R[:, j] = Z[:, U[j]] and R[:, K] = log sum over the
    complement O of exp Z (the "other class"); the normaliser of R equals lambda, so the
    first K columns are the selected log-probabilities S and the last is log P_O.  The
    complement column is dropped when O is empty.  Also returns lambda."""
    H = np.asarray(H, np.float64)
    W = np.asarray(W, np.float64)
    V = W.shape[0]
    b = _bias(bias, V)
    u = np.asarray(u_ids, np.int64)
    lam = log_normalizer(H, W, chunk, bias=b)
    S = selected_logprobs(H, W, u, lam, bias=b)
    comp = np.setdiff1d(np.arange(V), u)
    if comp.size == 0:
        return {"logp": S, "lam": lam}
    bo = b.copy()
    bo[u] = -np.inf                       # the complement's log-sum-exp
    lam_o = log_normalizer(H, W, chunk, bias=bo)
    return {"logp": np.concatenate([S, (lam_o - lam)[:, None]], axis=1), "lam": lam}


def grouped_gradient(logp, dlogp) -> Dict[str, np.ndarray]:
    """From a gradient w.r.t. log softmax(R) to G = dL/dS and g (Algorithm 1's inputs to the
    recomputed backward).  With c = dlogp[:, K] / P_O and sigma = sum_j dlogp[:, j]:
    dL/dZ_v = dlogp_j - p_v sigma for v = U[j], and p_v (c - sigma) for v in O (Eq.
    offsupport), i.e. scatter_U(G) - g p with G_j = dlogp_j - c p_{U[j]} and g = sigma - c."""
    logp = np.asarray(logp, np.float64)
    dlogp = np.asarray(dlogp, np.float64)
    sigma = dlogp.sum(axis=1)
    K = logp.shape[1] - 1
    with np.errstate(divide="ignore", invalid="ignore"):
        po = np.exp(logp[:, K])
        c = np.where(po > 0, dlogp[:, K] / po, 0.0)
    G = dlogp[:, :K] - c[:, None] * np.exp(logp[:, :K])
    return {"G": G, "g": sigma - c}


def grouped_backward(H, W, lam, logp, dlogp, u_ids, bias=None, chunk: int = 4096) -> Dict[str, np.ndarray]:
    """dH, dW, db from dL/d(log softmax R) (Eq. offsupport, written out): with p_v =
    exp(Z_v - lambda), sigma the row sum of dlogp and P_O = exp(logp[:, K]),
    dL/dZ_v = dlogp_j - sigma p_v for the selected class v = U[j] and
    dL/dZ_v = p_v (dlogp_K / P_O - sigma) for v in the complement; then dH = dZ W,
    dW = dZ^T H, db = dZ^T 1.  logp, dlogp: [M, K + 1], or [M, K] when U is the whole
    vocabulary."""
    H = np.asarray(H, np.float64)
    W = np.asarray(W, np.float64)
    lam = np.asarray(lam, np.float64)
    logp = np.asarray(logp, np.float64)
    dlogp = np.asarray(dlogp, np.float64)
    M, D = H.shape
    V = W.shape[0]
    b = _bias(bias, V)
    u = np.asarray(u_ids, np.int64)
    K = u.size
    sigma = dlogp.sum(axis=1)
    c = np.zeros(M)
    if logp.shape[1] == K + 1:
        po = np.exp(logp[:, K])
        nz = po > 0
        c[nz] = dlogp[nz, K] / po[nz]
    col = np.full(V, -1, np.int64)
    col[u] = np.arange(K)
    dH = np.zeros((M, D))
    dW = np.zeros((V, D))
    db = np.zeros(V)
    for v0 in range(0, V, chunk):
        v1 = min(V, v0 + chunk)
        p = np.exp(H @ W[v0:v1].T + b[v0:v1] - lam[:, None])
        dZ = p * (c - sigma)[:, None]
        for v in range(v0, v1):
            j = col[v]
            if j >= 0:
                dZ[:, v - v0] = dlogp[:, j] - sigma * p[:, v - v0]
        dH += dZ @ W[v0:v1]
        dW[v0:v1] = dZ.T @ H
        db[v0:v1] = dZ.sum(axis=0)
    return {"dH": dH, "dW": dW, "db": db}


# ---------------------------------------------------------------------------------------
# Greedy (best-path) emission head for recognition: framewise argmax over the full
# vocabulary, then the CTC collapse (merge repeated ids, drop blanks; Sec. 3.1)
# ---------------------------------------------------------------------------------------

def ctc_collapse(ids: Sequence[int], blank: int) -> List[int]:
    """The collapse map B of Sec. 3.1: merge consecutive repeats, then remove blanks."""
    out: List[int] = []
    prev = None
    for c in ids:
        c = int(c)
        if c != prev and c != blank:
            out.append(c)
        prev = c
    return out


def greedy_decode(H, W, input_lengths, blank: int, bias=None, chunk: int = 4096) -> Dict[str, object]:
    """Per frame the class with the largest logit H W^T + b (the first such class on ties),
    computed one vocabulary chunk at a time in fp64; per utterance the collapsed sequence.
    Returns ids [M], the top two logits per frame (for tie analysis) and tokens (a list of
    lists)."""
    H = np.asarray(H, np.float64)
    W = np.asarray(W, np.float64)
    b = _bias(bias, W.shape[0])
    M = H.shape[0]
    best = np.full(M, -np.inf)
    second = np.full(M, -np.inf)
    ids = np.zeros(M, np.int64)
    for v0 in range(0, W.shape[0], chunk):
        Z = H @ W[v0:v0 + chunk].T + b[v0:v0 + chunk]
        j = np.argmax(Z, axis=1)
        zmax = Z[np.arange(M), j]
        Z2 = Z.copy()
        Z2[np.arange(M), j] = -np.inf
        z2 = Z2.max(axis=1) if Z.shape[1] > 1 else np.full(M, -np.inf)
        better = zmax > best
        second = np.where(better, np.maximum(best, z2), np.maximum(second, zmax))
        ids = np.where(better, v0 + j, ids)
        best = np.where(better, zmax, best)
    toff = _offsets(input_lengths)
    tokens = [ctc_collapse(ids[toff[n]:toff[n + 1]], blank) for n in range(len(input_lengths))]
    return {"ids": ids, "best": best, "second": second, "tokens": tokens}

