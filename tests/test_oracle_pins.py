"""Pins for the CPU oracle: each check ties it to something other than itself.

* brute-force enumeration of alignments (collapse map of Sec. 3.1);
* closed forms (uniform logits, empty target, unique alignment);
* PyTorch's CPU CTC loss in float64, a library routine for the unpruned case;
* central finite differences of the loss for dH and dW (App. A, Step 3);
* Proposition 1: CTC on the grouped logits R (Eq. "grouped") equals full CTC;
* invariants: occupancies sum to one per frame (App. A, Step 3), dZ rows sum to
  zero, L_beta >= L and |gamma_beta - gamma| <= delta (App. B.3).
"""
import math

import numpy as np
import pytest

import oracle
from oracle import prunedctc_oracle as O
from tests import brute


def _logsoftmax(z):
    z = np.asarray(z, np.float64)
    m = z.max(axis=-1, keepdims=True)
    return z - (m + np.log(np.exp(z - m).sum(axis=-1, keepdims=True)))


# ---------------------------------------------------------------------------------------
# union / remap
# ---------------------------------------------------------------------------------------

def test_union_remap_by_hand():
    # targets of two utterances: [7, 3, 7] and [2, 9]; blank = 5
    u = oracle.union_remap(np.array([7, 3, 7, 2, 9]), np.array([3, 2]), blank=5, V=10)
    assert u["u_ids"].tolist() == [5, 2, 3, 7, 9]
    assert u["K"] == 5
    assert u["remap"].tolist() == [-1, -1, 1, 2, -1, 0, -1, 3, -1, 4]
    assert u["y_rel"].tolist() == [3, 2, 3, 1, 4]


def test_union_remap_empty_targets():
    u = oracle.union_remap(np.zeros(0, np.int64), np.array([0, 0]), blank=0, V=4)
    assert u["u_ids"].tolist() == [0] and u["K"] == 1
    assert u["remap"].tolist() == [0, -1, -1, -1]


# ---------------------------------------------------------------------------------------
# normaliser
# ---------------------------------------------------------------------------------------

def test_lambda_closed_form_zero_head():
    H = np.random.default_rng(1).standard_normal((5, 3))
    W = np.zeros((17, 3))
    np.testing.assert_allclose(oracle.log_normalizer(H, W, chunk=4), np.log(17.0), rtol=0, atol=1e-14)


def test_lambda_shift_invariance_and_mpmath():
    import mpmath
    rng = np.random.default_rng(2)
    H = rng.standard_normal((4, 6))
    W = rng.standard_normal((23, 6)) * 3
    lam = oracle.log_normalizer(H, W, chunk=5)
    # adding a constant feature shifts every logit by c -> lambda shifts by c
    c = 7.25
    H2 = np.concatenate([H, np.ones((4, 1))], axis=1)
    W2 = np.concatenate([W, np.full((23, 1), c)], axis=1)
    np.testing.assert_allclose(oracle.log_normalizer(H2, W2, chunk=3), lam + c, rtol=0, atol=1e-12)
    mpmath.mp.dps = 40
    Z = H @ W.T
    for m in range(4):
        ref = mpmath.log(mpmath.fsum(mpmath.exp(mpmath.mpf(float(z))) for z in Z[m]))
        assert abs(float(ref) - lam[m]) < 1e-12


# ---------------------------------------------------------------------------------------
# unpruned CTC against enumeration and closed forms
# ---------------------------------------------------------------------------------------

CASES = [
    # (T, C, y, blank)
    (1, 3, [], 0), (1, 3, [2], 0), (3, 3, [1, 2], 0), (4, 3, [1, 1], 0),
    (5, 4, [1, 2, 1], 0), (6, 3, [2, 2], 0), (5, 4, [3, 1], 2), (6, 4, [0, 0, 1], 3),
    (4, 3, [1, 1], 0), (3, 3, [1, 1], 0), (2, 3, [1, 1], 0), (6, 4, [], 1), (7, 3, [1, 2, 2], 0),
]


@pytest.mark.parametrize("T,C,y,blank", CASES)
def test_ctc_matches_enumeration(T, C, y, blank):
    rng = np.random.default_rng(T * 100 + C * 10 + len(y))
    logp = _logsoftmax(rng.standard_normal((T, C)) * 2.0)
    ref = brute.brute_ctc(logp, y, blank)
    res = oracle.ctc_utterance(logp, y, blank)
    r = sum(1 for i in range(1, len(y)) if y[i] == y[i - 1])
    assert res["alignable"] == (T >= len(y) + r) == (ref["n_align"] > 0)
    if ref["n_align"] == 0:
        assert res["logP"] == -math.inf
        return
    assert abs(res["logP"] - ref["logP"]) < 1e-12
    gam = np.zeros((T, C))
    for s, c in enumerate(res["ext"]):
        gam[:, c] += res["gamma"][:, s]
    np.testing.assert_allclose(gam, ref["gamma"], rtol=0, atol=1e-12)
    np.testing.assert_allclose(gam.sum(axis=1), 1.0, rtol=0, atol=1e-12)


@pytest.mark.parametrize("T,U,r", [(30, 8, 0), (30, 8, 3), (25, 1, 0), (11, 6, 5), (40, 0, 0), (9, 5, 4)])
def test_uniform_logits_closed_form(T, U, r):
    # With W = 0 every class has p = 1/V, and the count of alignments of U labels with r
    # adjacent repeats into T frames is C(T+U-r, 2U) (2U+1 segments, U+r of them non-empty).
    V = 11
    y = []
    for i in range(U):
        y.append(1 if i == 0 else (y[-1] if i <= r else (y[-1] % (V - 1)) + 1))
    assert sum(1 for i in range(1, U) if y[i] == y[i - 1]) == r
    H = np.ones((T, 2))
    W = np.zeros((V, 2))
    out = oracle.fwd_bwd(H, W, np.array(y), np.array([T]), np.array([U]), blank=0, want_grads=False)
    expect = T * math.log(V) - math.log(math.comb(T + U - r, 2 * U))
    assert abs(out["loss"] - expect) < 1e-9 * max(1.0, expect)


@pytest.mark.parametrize("beam", [math.inf, 0.0])
def test_tight_alignment_closed_form(beam):
    # When T = U + r (r adjacent repeats) the only alignment is the labels with a blank
    # inserted exactly between equal neighbours, so the loss is minus the sum of its
    # log-softmax values and each frame's occupancy is a one-hot of that path's class; a
    # zero beam keeps that path.
    rng = np.random.default_rng(11)
    V, D, blank = 40, 6, 2
    y = [5, 5, 9, 9, 9, 1]
    path = []
    for i, c in enumerate(y):
        if i > 0 and y[i - 1] == c:
            path.append(blank)
        path.append(c)
    T = len(path)
    H = rng.standard_normal((T, D))
    W = rng.standard_normal((V, D))
    z = H @ W.T
    logp = z - (z.max(axis=1, keepdims=True) + np.log(np.exp(z - z.max(axis=1, keepdims=True)).sum(axis=1, keepdims=True)))
    out = oracle.fwd_bwd(H, W, np.array(y), np.array([T]), np.array([len(y)]), blank=blank, beam=beam)
    assert out["status"].tolist() == [0]
    expect = -logp[np.arange(T), path].sum()
    assert abs(out["loss"] - expect) < 1e-10 * expect
    # dZ = p - onehot(path) on every frame, so dW = (p - onehot)^T H
    p = np.exp(logp)
    onehot = np.zeros_like(p)
    onehot[np.arange(T), path] = 1.0
    np.testing.assert_allclose(out["dW"], (p - onehot).T @ H, rtol=0, atol=1e-10)


def test_empty_target_closed_form():
    rng = np.random.default_rng(3)
    H = rng.standard_normal((9, 4))
    W = rng.standard_normal((13, 4))
    blank = 6
    out = oracle.fwd_bwd(H, W, np.zeros(0, np.int64), np.array([9]), np.array([0]), blank=blank)
    logp = _logsoftmax(H @ W.T)
    assert abs(out["loss"] - (-logp[:, blank].sum())) < 1e-11
    # single alignment: gamma is one-hot on blank, so dZ = p - e_blank
    p = np.exp(logp)
    dZ = p.copy()
    dZ[:, blank] -= 1.0
    np.testing.assert_allclose(out["dH"], dZ @ W, atol=1e-12)
    np.testing.assert_allclose(out["dW"], dZ.T @ H, atol=1e-12)


def test_unique_alignment_closed_form():
    # T = U + r: exactly one alignment, labels with a blank between the repeats
    y = [4, 4, 2, 7, 7]
    path = [4, 0, 4, 2, 7, 0, 7]
    rng = np.random.default_rng(4)
    H = rng.standard_normal((7, 5))
    W = rng.standard_normal((9, 5))
    out = oracle.fwd_bwd(H, W, np.array(y), np.array([7]), np.array([5]), blank=0)
    logp = _logsoftmax(H @ W.T)
    assert abs(out["loss"] + sum(logp[t, c] for t, c in enumerate(path))) < 1e-11
    dZ = np.exp(logp)
    for t, c in enumerate(path):
        dZ[t, c] -= 1.0
    np.testing.assert_allclose(out["dH"], dZ @ W, atol=1e-12)


# ---------------------------------------------------------------------------------------
# library cross-check: PyTorch CPU CTC in float64
# ---------------------------------------------------------------------------------------

@pytest.mark.parametrize("seed,blank", [(0, 0), (1, 0), (2, 13), (3, 49)])
def test_against_torch_ctc_loss(seed, blank):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(seed)
    N, V, D = 4, 50, 8
    T = rng.integers(5, 30, size=N)
    U = np.minimum(rng.integers(0, 9, size=N), T // 2)
    ys = []
    for u in U:
        y = rng.integers(0, V - 1, size=u)
        y = np.where(y >= blank, y + 1, y)
        if u > 2:
            y[2] = y[1]  # one adjacent repeat
        ys.append(y)
    targets = np.concatenate(ys)
    H = rng.standard_normal((int(T.sum()), D))
    W = rng.standard_normal((V, D))
    out = oracle.fwd_bwd(H, W, targets, T, U, blank=blank)
    # torch: padded (T, N, C) log-probs, gradient via autograd through log_softmax
    Ht = torch.tensor(H, dtype=torch.float64, requires_grad=True)
    Wt = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    logp = torch.log_softmax(Ht @ Wt.T, dim=1)
    Tm = int(T.max())
    pad = torch.zeros((Tm, N, V), dtype=torch.float64)
    off = np.concatenate([[0], np.cumsum(T)])
    rows = []
    for n in range(N):
        rows.append(torch.nn.functional.pad(logp[off[n]:off[n + 1]], (0, 0, 0, Tm - int(T[n]))))
    pad = torch.stack(rows, dim=1)
    loss = torch.nn.functional.ctc_loss(pad, torch.tensor(targets), torch.tensor(T), torch.tensor(U),
                                        blank=blank, reduction="sum", zero_infinity=True)
    loss.backward()
    assert abs(float(loss.detach()) - out["loss"]) < 1e-9 * max(1.0, abs(out["loss"]))
    np.testing.assert_allclose(out["dH"], Ht.grad.numpy(), rtol=0, atol=1e-9)
    np.testing.assert_allclose(out["dW"], Wt.grad.numpy(), rtol=0, atol=1e-9)


# ---------------------------------------------------------------------------------------
# finite differences of the loss (head gradients, App. A)
# ---------------------------------------------------------------------------------------

@pytest.mark.parametrize("beam", [math.inf, 3.0])
def test_finite_differences(beam):
    rng = np.random.default_rng(5)
    T = np.array([4, 3])
    U = np.array([2, 1])
    targets = np.array([1, 3, 2])
    H = rng.standard_normal((7, 3))
    W = rng.standard_normal((5, 3))
    out = oracle.fwd_bwd(H, W, targets, T, U, blank=0, beam=beam)

    def loss(Hx, Wx):
        return oracle.fwd_bwd(Hx, Wx, targets, T, U, blank=0, beam=beam, want_grads=False)["loss"]

    h = 1e-6
    for (i, j) in [(0, 0), (3, 2), (6, 1), (4, 0)]:
        Hp, Hm = H.copy(), H.copy()
        Hp[i, j] += h
        Hm[i, j] -= h
        fd = (loss(Hp, W) - loss(Hm, W)) / (2 * h)
        assert abs(fd - out["dH"][i, j]) < 1e-6
    for (i, j) in [(0, 0), (1, 2), (3, 1), (4, 2), (2, 0)]:
        Wp, Wm = W.copy(), W.copy()
        Wp[i, j] += h
        Wm[i, j] -= h
        fd = (loss(H, Wp) - loss(H, Wm)) / (2 * h)
        assert abs(fd - out["dW"][i, j]) < 1e-6


# ---------------------------------------------------------------------------------------
# Proposition 1: the grouped formulation (Eq. grouped) gives the same loss and gradient
# ---------------------------------------------------------------------------------------

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_proposition1_grouped_equals_full(seed):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(10 + seed)
    N, V, D = 3, 40, 6
    T = np.array([12, 9, 15])
    U = np.array([3, 4, 5])
    targets = rng.integers(1, 12, size=int(U.sum()))
    H = rng.standard_normal((int(T.sum()), D))
    W = rng.standard_normal((V, D))
    full = oracle.fwd_bwd(H, W, targets, T, U, blank=0)
    u = oracle.union_remap(targets, U, 0, V)
    # grouped logits via torch autograd: R = [Z_U, LSE over the complement]
    Ht = torch.tensor(H, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    Z = Ht @ Wt.T
    comp = [v for v in range(V) if u["remap"][v] < 0]
    R = torch.cat([Z[:, torch.tensor(u["u_ids"])], torch.logsumexp(Z[:, comp], dim=1, keepdim=True)], 1)
    logp_R = torch.log_softmax(R, dim=1)
    off = np.concatenate([[0], np.cumsum(T)])
    yoff = np.concatenate([[0], np.cumsum(U)])
    total = 0.0
    for n in range(N):
        y_rel = u["y_rel"][yoff[n]:yoff[n + 1]].tolist()
        res = oracle.ctc_utterance(logp_R[off[n]:off[n + 1]].detach().numpy(), y_rel, 0)
        total += -res["logP"]
    assert abs(total - full["loss"]) < 1e-10 * abs(full["loss"])
    # gradient of the grouped loss through torch's CTC on R
    Tm = int(T.max())
    pad = torch.stack([torch.nn.functional.pad(logp_R[off[n]:off[n + 1]], (0, 0, 0, Tm - int(T[n])))
                       for n in range(N)], 1)
    l = torch.nn.functional.ctc_loss(pad, torch.tensor(u["y_rel"]), torch.tensor(T), torch.tensor(U),
                                     blank=0, reduction="sum")
    l.backward()
    np.testing.assert_allclose(Ht.grad.numpy(), full["dH"], atol=1e-10)
    np.testing.assert_allclose(Wt.grad.numpy(), full["dW"], atol=1e-10)


# ---------------------------------------------------------------------------------------
# invariants on a mid-size case
# ---------------------------------------------------------------------------------------

def test_invariants_midsize():
    from paper_2609_33645_amd import workloads
    wl = workloads.random_small(7, N=5, T_range=(10, 60), D=16, V=300, dtype="f32", p_repeat=0.2)
    out = oracle.fwd_bwd(wl.H, wl.W, wl.targets, wl.input_lengths, wl.target_lengths, wl.blank,
                         chunk=37)
    inc = out["included"]
    # occupancies sum to one on included frames: g = -1
    np.testing.assert_allclose(out["g"][inc], -1.0, atol=1e-12)
    assert (out["G"] <= 1e-15).all()
    # dZ rows sum to zero: append a zero feature to H and an all-ones column to W;
    # the logits are unchanged and dH[:, -1] = sum_v dZ[m, v]
    ones = np.ones((wl.V, 1))
    H0 = np.concatenate([wl.H, np.zeros((wl.M, 1))], 1)
    out3 = oracle.fwd_bwd(H0, np.concatenate([wl.W, ones], 1), wl.targets, wl.input_lengths,
                          wl.target_lengths, wl.blank, chunk=64)
    np.testing.assert_allclose(out3["dH"][:, -1], 0.0, atol=1e-11)
    # chunk width does not change anything beyond rounding
    out4 = oracle.fwd_bwd(wl.H, wl.W, wl.targets, wl.input_lengths, wl.target_lengths, wl.blank,
                          chunk=4096)
    assert abs(out4["loss"] - out["loss"]) < 1e-10 * abs(out["loss"])
    np.testing.assert_allclose(out4["dW"], out["dW"], atol=1e-12)


def test_excluded_and_nonfinite_utterances():
    rng = np.random.default_rng(8)
    V, D = 20, 4
    T = np.array([3, 6, 5])
    U = np.array([2, 2, 2])
    targets = np.array([4, 4, 1, 2, 3, 5])   # utt 0: "4 4" needs 3 frames -> alignable; make it 2
    T[0] = 2                                  # now T < U + r -> excluded
    H = rng.standard_normal((int(T.sum()), D))
    W = rng.standard_normal((V, D))
    H[2 + 6 + 1, 0] = np.nan                  # NaN in utterance 2
    out = oracle.fwd_bwd(H, W, targets, T, U, blank=0)
    assert out["status"].tolist() == [oracle.STATUS_NOT_ALIGNABLE, oracle.STATUS_OK,
                                      oracle.STATUS_NONFINITE]
    assert out["loss_n"][0] == 0 and out["loss_n"][2] == 0
    assert np.isfinite(out["dW"]).all()
    assert (out["dH"][:2] == 0).all() and (out["dH"][8:] == 0).all()
    # utterance 1 alone gives the same dW
    alone = oracle.fwd_bwd(H[2:8], W, targets[2:4], T[1:2], U[1:2], blank=0)
    np.testing.assert_allclose(out["dW"], alone["dW"], atol=1e-13)
    assert abs(out["loss"] - alone["loss"]) < 1e-12


@pytest.mark.parametrize("bad,code", [
    (dict(targets=np.array([0, 1])), oracle.PCTC_ELABEL),
    (dict(targets=np.array([1, 20])), oracle.PCTC_ELABEL),
    (dict(T=np.array([0, 3])), oracle.PCTC_ELENGTH),
    (dict(U=np.array([-1, 3])), oracle.PCTC_ELENGTH),
    (dict(blank=20), oracle.PCTC_EINVAL),
    (dict(beam=float("nan")), oracle.PCTC_EINVAL),
])
def test_validation_codes(bad, code):
    args = dict(targets=np.array([1, 2]), T=np.array([2, 3]), U=np.array([1, 1]), blank=0, beam=math.inf)
    args.update(bad)
    H = np.zeros((max(1, int(np.sum(np.maximum(args["T"], 0)))), 2))
    with pytest.raises(oracle.OracleError) as e:
        oracle.fwd_bwd(H, np.zeros((20, 2)), args["targets"], args["T"], args["U"], args["blank"],
                       args["beam"])
    assert e.value.code == code


# ---------------------------------------------------------------------------------------
# beam pruning (Sec. 3.3, App. B.3)
# ---------------------------------------------------------------------------------------

BEAM_CASES = [(6, 4, [1, 2, 1], 0), (6, 3, [1, 1], 0), (7, 3, [2, 1], 0), (5, 4, [3], 1), (6, 3, [], 0)]


@pytest.mark.parametrize("T,C,y,blank", BEAM_CASES)
@pytest.mark.parametrize("beam", [0.0, 0.7, 2.0, 5.0, 40.0])
def test_beam_matches_enumeration(T, C, y, blank, beam):
    rng = np.random.default_rng(T * 7 + C + len(y) * 3)
    logp = _logsoftmax(rng.standard_normal((T, C)) * 2.5)
    ref = brute.brute_ctc(logp, y, blank, beam=beam)  # the paper's rule: no slack
    res = oracle.ctc_utterance(logp, y, blank, beam=beam)
    assert abs(res["logP"] - ref["logP"]) < 1e-12
    gam = np.zeros((T, C))
    for s, c in enumerate(res["ext"]):
        gam[:, c] += res["gamma"][:, s]
    np.testing.assert_allclose(gam, ref["gamma"], atol=1e-12)
    # no arc decision sits on the threshold in these cases, except at beta = 0, where the
    # best alignment's own arcs score exactly the best (margin 0 up to rounding) and are kept
    for k, m in res["margins"].items():
        fin = np.isfinite(m)
        near = np.abs(np.asarray(m)[fin]) <= 1e-9
        if beam == 0.0:
            assert np.asarray(res["keep"][k])[fin][near].all(), k
        else:
            assert not near.any(), k


def test_beam_properties():
    from paper_2609_33645_amd import workloads
    wl = workloads.random_small(11, N=4, T_range=(20, 50), D=16, V=200, dtype="f32", p_repeat=0.1,
                                w_std=1.0)
    full = oracle.fwd_bwd(wl.H, wl.W, wl.targets, wl.input_lengths, wl.target_lengths, 0)
    big = oracle.fwd_bwd(wl.H, wl.W, wl.targets, wl.input_lengths, wl.target_lengths, 0, beam=1e6)
    assert abs(big["loss"] - full["loss"]) < 1e-9 * abs(full["loss"])
    np.testing.assert_allclose(big["dW"], full["dW"], atol=1e-12)
    for beam in [0.0, 1.0, 4.0, 10.0]:
        pr = oracle.fwd_bwd(wl.H, wl.W, wl.targets, wl.input_lengths, wl.target_lengths, 0, beam=beam)
        for n in range(wl.N):
            if full["status"][n] != 0:
                continue
            delta_n = pr["loss_n"][n] - full["loss_n"][n]
            assert delta_n >= -1e-9                       # L_beta >= L
            dmass = -math.expm1(-max(delta_n, 0.0))
            rows = slice(int(np.sum(wl.input_lengths[:n])), int(np.sum(wl.input_lengths[:n + 1])))
            diff = np.abs(pr["G"][rows] - full["G"][rows])
            assert diff.max() <= dmass + 1e-9              # |gamma_beta - gamma| <= delta
            assert diff.sum(axis=1).max() <= 2 * dmass + 1e-9


def test_beam_zero_keeps_only_best_path():
    rng = np.random.default_rng(12)
    logp = _logsoftmax(rng.standard_normal((8, 5)) * 3)
    y = [2, 4, 4]
    res = oracle.ctc_utterance(logp, y, 0, beam=0.0)
    ref = brute.brute_ctc(logp, y, 0)
    assert abs(res["logP"] - max(ref["scores"])) < 1e-12
    gam = res["gamma"]
    assert set(np.round(gam, 12).ravel().tolist()) <= {0.0, 1.0}


@pytest.mark.parametrize("gap", [5e-4, -5e-4, 1e-7, -1e-7])
def test_beam_threshold_is_the_papers(gap):
    """App. B.3 keeps an arc iff the best alignment through it is within beta of the best:
    an alignment scoring best - beta - gap is dropped for any gap > 0, however small, and
    kept for gap <= 0.  Two frames, target [1]: alignments (1,1) = 0, (1,-) = -beta - gap
    and (-,1) = -beta + 0.25 written into the scores; the expected sum is enumerated."""
    beta = 2.0
    logp = np.array([[-beta + 0.25, 0.0, -30.0],
                     [-beta - gap, 0.0, -30.0]])
    res = oracle.ctc_utterance(logp, [1], 0, beam=beta)
    ref = brute.brute_ctc(logp, [1], 0, beam=beta)
    kept = [0.0, -beta + 0.25] + ([-beta - gap] if gap <= 0 else [])
    want = math.log(sum(math.exp(x) for x in kept))
    assert abs(ref["logP"] - want) < 1e-14
    assert abs(res["logP"] - want) < 1e-14
    assert ref["n_kept"] == len(kept)


def test_scores_stage_matches_full_path():
    """The alignment stage on the oracle's own S reproduces the full-vocabulary result."""
    from paper_2609_33645_amd import workloads
    wl = workloads.random_small(13, N=3, T_range=(8, 30), D=8, V=120, dtype="f32", p_repeat=0.2)
    full = oracle.fwd_bwd(wl.H, wl.W, wl.targets, wl.input_lengths, wl.target_lengths, 0, beam=3.0)
    st = oracle.ctc_from_scores(full["S"], full["y_rel"], wl.input_lengths, wl.target_lengths, beam=3.0)
    np.testing.assert_allclose(st["loss_n"], full["loss_n"], atol=1e-10)
    np.testing.assert_allclose(st["G"], full["G"], atol=1e-12)


def test_head_backward_stage_matches_full_path():
    """Eq. vjp with the alignment stage's G and g reproduces the full-vocabulary gradient
    (Algorithm 1 backward equals Eq. grad-full when G = -gamma, App. B.1)."""
    from paper_2609_33645_amd import workloads
    wl = workloads.random_small(14, N=4, T_range=(5, 30), D=12, V=150, dtype="f32", p_repeat=0.2)
    wl.input_lengths[1] = 1
    wl.target_lengths[1] = 3          # excluded utterance
    wl.H = wl.H[:int(wl.input_lengths.sum())]
    U = wl.target_lengths
    wl.targets = np.resize(wl.targets, int(U.sum())) % 140 + 1
    full = oracle.fwd_bwd(wl.H, wl.W, wl.targets, wl.input_lengths, U, 0, beam=4.0, chunk=32)
    st = oracle.head_backward(wl.H, wl.W, full["lam"], full["G"], full["g"], full["u_ids"], chunk=50)
    np.testing.assert_allclose(st["dH"], full["dH"], atol=1e-12)
    np.testing.assert_allclose(st["dW"], full["dW"], atol=1e-12)
    assert full["status"][1] == oracle.STATUS_NOT_ALIGNABLE


def test_head_backward_rows_is_gradient_of_surrogate():
    """The sampled backward rows are the gradient of f(H, W) = sum G * Z_U - sum_m g_m lambda_m
    (its derivative w.r.t. Z is scatter_U(G) - g p, Eq. vjp), taken by torch autograd in float64;
    frames with g = 0 are left out of f, and NaN in such a frame must not reach dW."""
    import torch
    rng = np.random.default_rng(21)
    M, D, V, K = 40, 9, 300, 12
    H = rng.standard_normal((M, D))
    W = rng.standard_normal((V, D)) / 3
    u_ids = np.concatenate([[7], np.sort(rng.choice(np.setdiff1d(np.arange(V), [7]), K - 1, replace=False))])
    G = -rng.random((M, K))
    G[5:9] = 0.0                       # an excluded utterance's frames
    g = G.sum(axis=1)
    H[6] = np.nan
    lam = oracle.log_normalizer(H, W, chunk=64)
    frames = np.array([0, 3, 6, 17, M - 1])
    classes = np.array([0, 7, int(u_ids[3]), 150, V - 1])
    got = oracle.head_backward_rows(H, W, lam, G, g, u_ids, frames, classes, chunk=77)
    inc = g != 0
    Ht = torch.tensor(H[inc], dtype=torch.float64, requires_grad=True)
    Wt = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    Z = Ht @ Wt.T
    f = (torch.tensor(G[inc]) * Z[:, torch.tensor(u_ids)]).sum() - (torch.tensor(g[inc]) * torch.logsumexp(Z, 1)).sum()
    f.backward()
    dH = np.zeros((M, D))
    dH[inc] = Ht.grad.numpy()
    np.testing.assert_allclose(got["dH"], dH[frames], atol=1e-11)
    np.testing.assert_allclose(got["dW"], Wt.grad.numpy()[classes], atol=1e-11)
    assert np.all(got["dH"][2] == 0.0) and np.all(np.isfinite(got["dW"]))


# ---------------------------------------------------------------------------------------
# head bias, blank offset and loss weights (Sec. 2 head (W, b); LLM-CTC blank offset;
# token-count normalisation): library and finite-difference cross-checks
# ---------------------------------------------------------------------------------------

@pytest.mark.parametrize("seed,blank", [(0, 0), (1, 17)])
def test_bias_and_weights_against_torch_ctc_loss(seed, blank):
    """Loss sum_n w_n L_n on log_softmax(H W^T + b) and its gradients w.r.t. H, W and b,
    against PyTorch's CPU CTC (reduction 'none', weighted by hand) and autograd in float64."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(100 + seed)
    N, V, D = 4, 40, 6
    T = rng.integers(6, 25, size=N)
    U = np.minimum(rng.integers(1, 7, size=N), T // 2)
    ys = []
    for u in U:
        y = rng.integers(0, V - 1, size=u)
        ys.append(np.where(y >= blank, y + 1, y))
    targets = np.concatenate(ys)
    H = rng.standard_normal((int(T.sum()), D))
    W = rng.standard_normal((V, D)) / 2
    b = rng.standard_normal(V)
    b[blank] += 1.5                      # a blank offset eta
    w = rng.uniform(0.1, 2.0, size=N)
    out = oracle.fwd_bwd(H, W, targets, T, U, blank=blank, bias=b, weights=w)
    Ht = torch.tensor(H, dtype=torch.float64, requires_grad=True)
    Wt = torch.tensor(W, dtype=torch.float64, requires_grad=True)
    bt = torch.tensor(b, dtype=torch.float64, requires_grad=True)
    logp = torch.log_softmax(Ht @ Wt.T + bt, dim=1)
    Tm = int(T.max())
    off = np.concatenate([[0], np.cumsum(T)])
    pad = torch.stack([torch.nn.functional.pad(logp[off[n]:off[n + 1]], (0, 0, 0, Tm - int(T[n])))
                       for n in range(N)], dim=1)
    ln = torch.nn.functional.ctc_loss(pad, torch.tensor(targets), torch.tensor(T), torch.tensor(U),
                                      blank=blank, reduction="none", zero_infinity=True)
    loss = (ln * torch.tensor(w)).sum()
    loss.backward()
    np.testing.assert_allclose(out["loss_n"], ln.detach().numpy(), rtol=1e-10)
    assert abs(float(loss.detach()) - out["loss"]) < 1e-9 * abs(out["loss"])
    np.testing.assert_allclose(out["dH"], Ht.grad.numpy(), rtol=0, atol=1e-9)
    np.testing.assert_allclose(out["dW"], Wt.grad.numpy(), rtol=0, atol=1e-9)
    np.testing.assert_allclose(out["db"], bt.grad.numpy(), rtol=0, atol=1e-9)
    # the blank offset's gradient is the blank entry of db
    assert abs(out["db"][blank] - float(bt.grad[blank])) < 1e-9


@pytest.mark.parametrize("beam", [math.inf, 3.0])
def test_bias_finite_differences(beam):
    """db (and the eta = b[blank] entry) by central differences of the weighted loss,
    unpruned and beam-pruned."""
    rng = np.random.default_rng(7)
    T = np.array([5, 4, 3])
    U = np.array([2, 1, 1])
    targets = np.array([1, 3, 2, 4])
    H = rng.standard_normal((12, 3))
    W = rng.standard_normal((6, 3))
    b = rng.standard_normal(6)
    w = np.array([0.5, 2.0, 1.0])
    out = oracle.fwd_bwd(H, W, targets, T, U, blank=0, beam=beam, bias=b, weights=w)

    def loss(bx):
        return oracle.fwd_bwd(H, W, targets, T, U, blank=0, beam=beam, want_grads=False, bias=bx, weights=w)["loss"]

    h = 1e-6
    for v in range(6):
        bp, bm = b.copy(), b.copy()
        bp[v] += h
        bm[v] -= h
        assert abs((loss(bp) - loss(bm)) / (2 * h) - out["db"][v]) < 1e-6


def test_bias_rows_and_stage_agree():
    """head_backward and head_backward_rows with a bias reproduce the full path's dH, dW, db."""
    from paper_2609_33645_amd import workloads
    wl = workloads.random_small(31, N=3, T_range=(6, 20), D=8, V=90, dtype="f32", p_repeat=0.2)
    b = np.random.default_rng(3).standard_normal(90)
    w = np.array([1.0, 0.25, 3.0])
    full = oracle.fwd_bwd(wl.H, wl.W, wl.targets, wl.input_lengths, wl.target_lengths, 0, beam=4.0, bias=b,
                          weights=w, chunk=17)
    st = oracle.head_backward(wl.H, wl.W, full["lam"], full["G"], full["g"], full["u_ids"], chunk=40, bias=b)
    for k in ("dH", "dW", "db"):
        np.testing.assert_allclose(st[k], full[k], atol=1e-12)
    fr = np.array([0, 5, int(wl.M) - 1])
    cl = np.array([0, 3, 50, 89])
    rows = oracle.head_backward_rows(wl.H, wl.W, full["lam"], full["G"], full["g"], full["u_ids"], fr, cl, bias=b)
    np.testing.assert_allclose(rows["dH"], full["dH"][fr], atol=1e-12)
    np.testing.assert_allclose(rows["dW"], full["dW"][cl], atol=1e-12)
    np.testing.assert_allclose(rows["db"], full["db"][cl], atol=1e-12)


# ---------------------------------------------------------------------------------------
# discarded posterior mass (App. B.3)
# ---------------------------------------------------------------------------------------

@pytest.mark.parametrize("seed,beam", [(0, 0.5), (1, 1.5), (2, 3.0), (3, 0.0)])
def test_discarded_mass_by_enumeration(seed, beam):
    """delta = 1 - (retained alignment sum) / (all-alignment sum), with both sums taken by
    brute-force enumeration of alignments and the arc rule applied per enumerated arc."""
    rng = np.random.default_rng(300 + seed)
    T, C = 5, 3
    y = [1, 2] if seed % 2 == 0 else [2]
    logp = np.log(rng.dirichlet(np.ones(C), size=T))
    aligns = brute.valid_alignments(T, C, y, 0)
    scores = np.array([sum(logp[t, pi[t]] for t in range(T)) for pi in aligns])
    best_through = {}
    for pi, sc in zip(aligns, scores):
        for a in brute.arcs_of(pi, 0):
            best_through[a] = max(best_through.get(a, -math.inf), sc)
    kept = {a for a, v in best_through.items() if v >= scores.max() - beam}
    keep = np.array([all(a in kept for a in brute.arcs_of(pi, 0)) for pi in aligns])
    want = 1.0 - np.exp(scores[keep]).sum() / np.exp(scores).sum()
    got = oracle.discarded_mass(logp, np.array(y), [T], [len(y)], [beam])
    assert abs(got[0, 0] - want) < 1e-12
    assert -1e-15 <= got[0, 0] <= 1.0


def test_discarded_mass_limits():
    """delta = 0 without pruning (infinite beam), the occupancy bound of App. B.3
    |gamma_beta - gamma| <= delta holds, and a not-alignable utterance gives NaN."""
    from paper_2609_33645_amd import workloads
    S = workloads.random_scores(9, 30, 6).astype(np.float64)
    T, U = [20, 10], [4, 7]
    y = np.array([1, 2, 3, 1, 2, 2, 2, 2, 2, 2, 2], np.int64)
    d = oracle.discarded_mass(S, y, T, U, [math.inf, 2.0, 6.0])
    assert d[0, 0] == 0.0 and np.isnan(d[:, 1]).all()   # 7 labels with 6 repeats need 13 frames
    assert 0.0 <= d[2, 0] <= d[1, 0] <= 1.0
    full = oracle.ctc_utterance(S[:20], [1, 2, 3, 1], 0)
    pr = oracle.ctc_utterance(S[:20], [1, 2, 3, 1], 0, beam=2.0)
    assert np.abs(pr["gamma"] - full["gamma"]).max() <= d[1, 0] + 1e-12


# ---------------------------------------------------------------------------------------
# greedy emission head (framewise argmax, CTC collapse)
# ---------------------------------------------------------------------------------------

def test_ctc_collapse_examples():
    """The collapse map of Sec. 3.1 on written-out strings (blank = '-')."""
    enc = {"-": 0, "a": 1, "b": 2, "c": 3}

    def col(sx):
        return "".join("-abc"[i] for i in oracle.ctc_collapse([enc[ch] for ch in sx], 0))
    assert col("aa-ab-") == "aab"
    assert col("--a--") == "a"
    assert col("abc") == "abc"
    assert col("aaaa") == "a"
    assert col("a-a") == "aa"
    assert col("----") == ""
    assert col("") == ""
    # every alignment of a target collapses to it (brute-force enumeration)
    for pi in brute.valid_alignments(4, 3, [1, 1], 0):
        assert oracle.ctc_collapse(pi, 0) == [1, 1]


def test_greedy_decode_against_torch_argmax():
    """Framewise argmax equals torch.argmax of the dense logits (first index on ties),
    across chunk widths, with a bias; ties are broken toward the smaller class id."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(12)
    H = rng.standard_normal((37, 5))
    W = rng.standard_normal((301, 5))
    b = rng.standard_normal(301)
    W[200] = W[17]
    b[200] = b[17]                           # duplicate class: exact ties between 17 and 200
    Z = torch.tensor(H) @ torch.tensor(W).T + torch.tensor(b)
    want = torch.argmax(Z, dim=1).numpy()
    for chunk in (7, 64, 4096):
        got = oracle.greedy_decode(H, W, [20, 17], blank=3, bias=b, chunk=chunk)
        np.testing.assert_array_equal(got["ids"], want)
        assert np.all(got["ids"] != 200)
        srt = np.sort(Z.numpy(), axis=1)
        np.testing.assert_allclose(got["best"], srt[:, -1], atol=1e-12)
        np.testing.assert_allclose(got["second"], srt[:, -2], atol=1e-12)
    assert got["tokens"][0] == oracle.ctc_collapse(want[:20], 3)


# ---------------------------------------------------------------------------------------
# grouped-logit export for a stock CTC (Eq. grouped, Prop. 1, Eq. offsupport)
# ---------------------------------------------------------------------------------------

@pytest.mark.parametrize("seed,leaf_grad", [(0, True), (1, False), (2, True)])
def test_grouped_export_through_torch_ctc(seed, leaf_grad):
    """The exported log softmax(R) matches torch's log_softmax of R built by autograd; torch's
    CTC on it gives the full loss; the gradient w.r.t. the exported log-probabilities, taken
    back through grouped_gradient and the recomputed backward, gives the autograd dH, dW and db.
    leaf_grad: the exported tensor is a leaf (torch's CTC then returns p - gamma, its
    convention) or the output of torch's log_softmax (true gradient -gamma)."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(50 + seed)
    N, V, D = 3, 40, 6
    T = np.array([12, 9, 15])
    U = np.array([3, 4, 5])
    targets = rng.integers(1, 12, size=int(U.sum()))
    H = rng.standard_normal((int(T.sum()), D))
    W = rng.standard_normal((V, D))
    b = rng.standard_normal(V)
    full = oracle.fwd_bwd(H, W, targets, T, U, blank=0, bias=b)
    u = oracle.union_remap(targets, U, 0, V)
    ex = oracle.grouped_logprobs(H, W, u["u_ids"], bias=b, chunk=13)
    Ht = torch.tensor(H, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    Z = Ht @ Wt.T + bt
    comp = [v for v in range(V) if u["remap"][v] < 0]
    R = torch.cat([Z[:, torch.tensor(u["u_ids"])], torch.logsumexp(Z[:, comp], dim=1, keepdim=True)], 1)
    np.testing.assert_allclose(ex["logp"], torch.log_softmax(R, 1).detach().numpy(), atol=1e-12)
    np.testing.assert_allclose(ex["lam"], full["lam"], atol=1e-12)
    off = np.concatenate([[0], np.cumsum(T)])
    Tm = int(T.max())
    lp = torch.tensor(ex["logp"], requires_grad=True) if leaf_grad else torch.log_softmax(R, 1)
    if not leaf_grad:
        lp.retain_grad()
    pad = torch.stack([torch.nn.functional.pad(lp[off[n]:off[n + 1]], (0, 0, 0, Tm - int(T[n]))) for n in range(N)], 1)
    loss = torch.nn.functional.ctc_loss(pad, torch.tensor(u["y_rel"]), torch.tensor(T), torch.tensor(U), blank=0,
                                        reduction="sum")
    assert abs(float(loss) - full["loss"]) < 1e-10 * abs(full["loss"])
    loss.backward()
    gg = oracle.grouped_gradient(ex["logp"], lp.grad.numpy())
    back = oracle.head_backward(H, W, ex["lam"], gg["G"], gg["g"], u["u_ids"], bias=b)
    np.testing.assert_allclose(back["dH"], full["dH"], atol=1e-10)
    np.testing.assert_allclose(back["dW"], full["dW"], atol=1e-10)
    np.testing.assert_allclose(back["db"], full["db"], atol=1e-10)
    direct = oracle.grouped_backward(H, W, ex["lam"], ex["logp"], lp.grad.numpy(), u["u_ids"], bias=b, chunk=11)
    for k in ("dH", "dW", "db"):
        np.testing.assert_allclose(direct[k], full[k], atol=1e-10)
    if not leaf_grad:
        np.testing.assert_allclose(direct["dW"], Wt.grad.numpy(), atol=1e-10)
        np.testing.assert_allclose(back["dH"], Ht.grad.numpy(), atol=1e-10)
        np.testing.assert_allclose(back["db"], bt.grad.numpy(), atol=1e-10)


def test_grouped_export_invariants():
    """Rows of exp(log softmax R) sum to one; the complement column is log(1 - sum_U p);
    a union covering the whole vocabulary leaves no complement column and G = dlogp, g = sigma."""
    rng = np.random.default_rng(77)
    M, V, D = 20, 9, 4
    H = rng.standard_normal((M, D))
    W = rng.standard_normal((V, D))
    u_ids = np.array([0, 2, 5, 7])
    ex = oracle.grouped_logprobs(H, W, u_ids, chunk=4)
    np.testing.assert_allclose(np.exp(ex["logp"]).sum(1), 1.0, atol=1e-13)
    np.testing.assert_allclose(ex["logp"][:, -1], np.log1p(-np.exp(ex["logp"][:, :-1]).sum(1)), atol=1e-12)
    full = oracle.grouped_logprobs(H, W, np.arange(V))
    assert full["logp"].shape == (M, V)
    dl = rng.standard_normal((M, V))
    gg = oracle.grouped_gradient(np.concatenate([full["logp"], np.full((M, 1), -np.inf)], 1),
                                 np.concatenate([dl, np.zeros((M, 1))], 1))
    np.testing.assert_allclose(gg["G"], dl, atol=0)
    np.testing.assert_allclose(gg["g"], dl.sum(1), atol=1e-13)


def test_grouped_backward_whole_vocabulary_autograd():
    """U = the whole vocabulary (no complement column) and a linear loss sum(dl * logp) whose
    row sums vanish (the case where g = 0 for every frame): the written-out backward matches
    torch autograd through log_softmax of the permuted logits."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(78)
    M, V, D = 15, 7, 5
    H = rng.standard_normal((M, D))
    W = rng.standard_normal((V, D))
    b = rng.standard_normal(V)
    perm = rng.permutation(V)
    dl = rng.standard_normal((M, V))
    dl -= dl.mean(axis=1, keepdims=True)
    ex = oracle.grouped_logprobs(H, W, perm, bias=b)
    Ht = torch.tensor(H, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    lp = torch.log_softmax((Ht @ Wt.T + bt)[:, torch.tensor(perm)], dim=1)
    (lp * torch.tensor(dl)).sum().backward()
    direct = oracle.grouped_backward(H, W, ex["lam"], ex["logp"], dl, perm, bias=b, chunk=3)
    np.testing.assert_allclose(direct["dH"], Ht.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(direct["dW"], Wt.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(direct["db"], bt.grad.numpy(), atol=1e-12)
