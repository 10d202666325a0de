"""Parity at the full sizes of the paper's head workloads, in the launch configuration the
benchmark times (one pruned_ctc_fwd_bwd call, default vocabulary chunk).

The oracle computes, in float64, everything that a full-size problem allows: the union,
lambda for every frame, S, the alignment stage for every utterance (losses, statuses,
G, g), and the backward outputs of a sample of frames (dH rows, each over all V classes)
and of classes (dW rows, each over all M frames).  Bars: union bit-exact; loss relative
error <= 2e-3 and gradient cosine >= 0.999 (bf16 path), with tighter checks recording the
accuracy actually reached.  The lattice stage is also run on the oracle's S: its kept-arc
mask must match the oracle's decision on every arc whose fp64 margin is further than
1e-2 nats from the threshold (nearer arcs may go either way in float32).

A vocabulary sweep at fixed targets checks that the library's device memory does not
grow with V beyond the 4-byte-per-class remap table.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2609_33645_amd import workloads
from tests.gpu_util import KERNEL_BAND, ambiguous_arcs, beam_bracket, cosine, loss_rel, rel_err, say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_33645_amd import prunedctc
    prunedctc.lib()
    yield
    torch.cuda.empty_cache()


def _samples(wl, rng, u_ids):
    """Frames: first and last of every utterance plus random ones; classes: blank, union
    members, non-members, the last class."""
    off = np.concatenate([[0], np.cumsum(wl.input_lengths)])
    frames = set()
    for n in range(wl.N):
        frames.update([int(off[n]), int(off[n + 1]) - 1])
    frames.update(rng.choice(wl.M, size=min(wl.M, 8), replace=False).tolist())
    frames = np.array(sorted(frames), np.int64)
    mem = rng.choice(np.asarray(u_ids[1:]), size=min(12, len(u_ids) - 1), replace=False)
    others = rng.choice(wl.V, size=12, replace=False)
    classes = np.unique(np.concatenate([[wl.blank, wl.V - 1], mem, others])).astype(np.int64)
    return frames, classes


def _mask_check(res_utt, mk, T, Sp, band=1e-2):
    """Arc bits as in the lattice stage (start/stay bit0, step bit1, skip bit2, final bit3);
    returns (arcs compared, arcs disagreeing) among arcs with |margin| > band."""
    mg = res_utt["margins"]
    stay = mg["stay"].copy()
    stay[0] = mg["start"]
    planes = [(stay, 0), (mg["step"], 1), (mg["skip"], 2)]
    fin = np.full((T, Sp), -np.inf)
    fin[T - 1] = mg["final"]
    planes.append((fin, 3))
    compared = bad = 0
    for m, bit in planes:
        sure = np.isfinite(m) & (np.abs(m) > band)
        got = ((mk >> bit) & 1).astype(bool)
        want = m >= 0
        compared += int(sure.sum())
        bad += int((sure & (got != want)).sum())
        # arcs outside the trellis (margin -inf) are never kept
        assert not np.any(got & np.isneginf(m))
    return compared, bad


# Every workload at every beam it is specified with (Qwen3-32B: the beam sweep {8, 16, 64}),
# plus the K-stress variant and the encoder memory shape in fp32.
FULL = [("zipformer_m", 16.0), ("zipformer_m", math.inf), ("qwen3_0p6b", 32.0), ("qwen3_8b", 32.0),
        ("qwen3_8b", math.inf), ("qwen3_32b", 8.0), ("qwen3_32b", 16.0), ("qwen3_32b", 64.0),
        ("qwen3_8b_kstress", 32.0), ("e1_zipformer_f32", math.inf)]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,beam", FULL)
def test_full_size_parity(name, beam):
    import torch
    from paper_2609_33645_amd import prunedctc
    wl = workloads.NAMED[name](0, beam=beam)
    say(f"full-size {name} beam={beam}: N={wl.N} M={wl.M} D={wl.D} V={wl.V} U={int(wl.target_lengths.sum())}")
    H, W, y = to_dev(wl)
    out = prunedctc.pruned_ctc_fwd_bwd(H, W, y, wl.input_lengths, wl.target_lengths, wl.blank, wl.beam)
    torch.cuda.synchronize()
    say("  gpu path done")
    un = prunedctc.union_remap(y, wl.blank, wl.V)
    st = prunedctc.lse_select(H, W, un["u_ids"])
    lam_gpu = st["lam"].cpu().numpy()
    S_gpu = st["S"].cpu().numpy()
    say("  gpu stages done")

    W64 = wl.W.astype(np.float64)
    H64 = wl.H.astype(np.float64)
    ref_un = oracle.union_remap(wl.targets, wl.target_lengths, wl.blank, wl.V)
    assert un["K"] == ref_un["K"]
    np.testing.assert_array_equal(un["u_ids"].cpu().numpy(), ref_un["u_ids"])
    np.testing.assert_array_equal(un["remap"].cpu().numpy(), ref_un["remap"])
    np.testing.assert_array_equal(un["y_rel"].cpu().numpy(), ref_un["y_rel"])
    lam = oracle.log_normalizer(H64, W64)
    say("  oracle lambda done")
    S = oracle.selected_logprobs(H64, W64, ref_un["u_ids"], lam)
    assert np.abs(lam_gpu - lam).max() < 5e-5
    assert np.abs(S_gpu - S).max() < 5e-5
    dp = oracle.ctc_from_scores(S, ref_un["y_rel"], wl.input_lengths, wl.target_lengths, beam)
    say("  oracle lattice done")

    status = out["status"].cpu().numpy()
    np.testing.assert_array_equal(status, dp["status"])
    ln = out["loss_per_utt"].cpu().numpy()
    assert loss_rel(float(out["loss"].item()), dp["loss"]) <= 2e-3
    assert np.abs(ln - dp["loss_n"]).max() / np.abs(dp["loss_n"]).max() <= 2e-3
    if math.isfinite(beam):
        # arcs within the kernel's tolerance band of the threshold may be decided either way
        # by the device: its losses must lie between the oracle's with those arcs all kept and
        # all dropped (the paper's rule lies between the two as well)
        dp["S"], dp["y_rel"] = S, ref_un["y_rel"]
        lo, hi = beam_bracket(dp, wl.input_lengths, wl.target_lengths, beam)
        width = np.abs(lo["loss_n"] - hi["loss_n"]) / np.abs(dp["loss_n"]).clip(1.0)
        say(f"  {ambiguous_arcs(dp)} arcs within {KERNEL_BAND} nats of the threshold; "
            f"relative loss bracket {width.max():.3g}")
        tol = 1e-5 * np.abs(dp["loss_n"])
        assert np.all(ln >= np.minimum(lo["loss_n"], hi["loss_n"]) - tol)
        assert np.all(ln <= np.maximum(lo["loss_n"], hi["loss_n"]) + tol)
    if not math.isfinite(beam) or width.max() <= 1e-7:
        np.testing.assert_allclose(ln, dp["loss_n"], rtol=1e-5)      # achieved accuracy

    rng = np.random.default_rng(7)
    frames, classes = _samples(wl, rng, ref_un["u_ids"])
    rows = oracle.head_backward_rows(H64, W64, lam, dp["G"], dp["g"], ref_un["u_ids"], frames, classes)
    say(f"  oracle sampled backward done ({frames.size} frames, {classes.size} classes)")
    dH_s = out["dH"][torch.from_numpy(frames).cuda()].cpu().numpy()
    dW_s = out["dW"][torch.from_numpy(classes).cuda()].cpu().numpy()
    assert cosine(dH_s, rows["dH"]) >= 0.999 and cosine(dW_s, rows["dW"]) >= 0.999
    assert cosine(dH_s, rows["dH"]) >= 0.99999 and cosine(dW_s, rows["dW"]) >= 0.99999
    assert rel_err(dH_s, rows["dH"]) < 1e-2 and rel_err(dW_s, rows["dW"]) < 1e-2
    for i in range(frames.size):       # row by row, so that no frame is drowned by the others
        assert cosine(dH_s[i], rows["dH"][i]) >= 0.999, f"frame {frames[i]}"

    if math.isfinite(beam):
        res = prunedctc.ctc_dp(torch.from_numpy(S.astype(np.float32)).cuda(),
                               torch.from_numpy(ref_un["y_rel"].astype(np.int32)).cuda(),
                               wl.input_lengths, wl.target_lengths, beam=beam, want_mask=True)
        mask = res["mask"].cpu().numpy()
        base = compared = bad = 0
        for n in range(wl.N):
            Tn, Sp = int(wl.input_lengths[n]), 2 * int(wl.target_lengths[n]) + 1
            mk = mask[base:base + Tn * Sp].reshape(Tn, Sp)
            base += Tn * Sp
            if dp["status"][n] == 0:
                c, b = _mask_check(dp["per_utt"][n], mk, Tn, Sp)
                compared += c
                bad += b
        say(f"  mask: {compared} arcs compared, {bad} disagree")
        assert compared > 0 and bad == 0
    del out, H, W, y
    torch.cuda.empty_cache()


@pytest.mark.timeout(300)
def test_workspace_flat_in_vocabulary():
    """Device memory the call adds above its inputs and preallocated gradients grows with V
    only by the remap table (4 bytes per class), for V from 10,000 to 180,000."""
    import torch
    from paper_2609_33645_amd import prunedctc
    base_wl = workloads.zipformer_m(3, beam=16.0, V=10_000)
    rng = np.random.default_rng(5)
    H = torch.from_numpy(base_wl.H).cuda().to(torch.bfloat16)
    y = torch.from_numpy(base_wl.targets).cuda()
    M, D = base_wl.M, base_wl.D
    dH = torch.empty((M, D), dtype=torch.float32, device="cuda")
    extra = {}
    for V in (10_000, 50_000, 100_000, 151_936, 180_000):
        W = torch.from_numpy(workloads.round_to_bf16(rng.standard_normal((V, D), dtype=np.float32) / math.sqrt(D)))
        W = W.cuda().to(torch.bfloat16)
        dW = torch.empty((V, D), dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        base = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        out = prunedctc.pruned_ctc_fwd_bwd(H, W, y, base_wl.input_lengths, base_wl.target_lengths, 0, 16.0,
                                           dH_out=dH, dW_out=dW)
        torch.cuda.synchronize()
        assert int(out["status"].ne(0).sum().item()) == 0
        extra[V] = torch.cuda.max_memory_allocated() - base - 4 * V
        say(f"  V={V}: peak above inputs and gradients {(extra[V] + 4 * V) / 2**20:.1f} MiB")
        del out, W, dW
    vals = np.array(list(extra.values()))
    assert vals.max() - vals.min() <= 1 << 20, extra


@pytest.mark.timeout(900)
def test_full_size_bias_weights_db():
    """Zipformer-M-sized head with a bias (blank offset included), token-count loss weights
    and db, in the benchmark's launch configuration; sampled outputs as above."""
    import torch
    from paper_2609_33645_amd import prunedctc
    wl = workloads.zipformer_m(1, beam=16.0)
    rng = np.random.default_rng(11)
    b = (0.5 * rng.standard_normal(wl.V)).astype(np.float32)
    b[wl.blank] += 3.0
    w = np.full(wl.N, 1.0 / float(wl.target_lengths.sum()), np.float32)
    say(f"full-size bias/weights zipformer_m: N={wl.N} M={wl.M} V={wl.V}")
    H, W, y = to_dev(wl)
    out = prunedctc.pruned_ctc_fwd_bwd(H, W, y, wl.input_lengths, wl.target_lengths, wl.blank, wl.beam,
                                       bias=torch.from_numpy(b).cuda(), utt_weight=torch.from_numpy(w).cuda(),
                                       want_db=True)
    torch.cuda.synchronize()
    W64 = wl.W.astype(np.float64)
    H64 = wl.H.astype(np.float64)
    b64 = b.astype(np.float64)
    un = oracle.union_remap(wl.targets, wl.target_lengths, wl.blank, wl.V)
    lam = oracle.log_normalizer(H64, W64, bias=b64)
    S = oracle.selected_logprobs(H64, W64, un["u_ids"], lam, bias=b64)
    dp = oracle.ctc_from_scores(S, un["y_rel"], wl.input_lengths, wl.target_lengths, wl.beam,
                                weights=w.astype(np.float64))
    say("  oracle forward done")
    np.testing.assert_array_equal(out["status"].cpu().numpy(), dp["status"])
    assert loss_rel(float(out["loss"].item()), dp["loss"]) <= 1e-5
    np.testing.assert_allclose(out["loss_per_utt"].cpu().numpy(), dp["loss_n"], rtol=1e-5)
    frames, classes = _samples(wl, rng, un["u_ids"])
    rows = oracle.head_backward_rows(H64, W64, lam, dp["G"], dp["g"], un["u_ids"], frames, classes, bias=b64)
    dH_s = out["dH"][torch.from_numpy(frames).cuda()].cpu().numpy()
    dW_s = out["dW"][torch.from_numpy(classes).cuda()].cpu().numpy()
    db_s = out["db"][torch.from_numpy(classes).cuda()].cpu().numpy()
    say(f"  cos dH={cosine(dH_s, rows['dH']):.7f} dW={cosine(dW_s, rows['dW']):.7f} db={cosine(db_s, rows['db']):.7f}")
    assert cosine(dH_s, rows["dH"]) >= 0.99999 and cosine(dW_s, rows["dW"]) >= 0.99999
    assert cosine(db_s, rows["db"]) >= 0.999
    # d eta = db[blank]
    bi = int(np.nonzero(classes == wl.blank)[0][0])
    assert abs(db_s[bi] - rows["db"][bi]) <= 1e-3 * abs(rows["db"][bi])
    del out, H, W, y
    torch.cuda.empty_cache()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["zipformer_m", "qwen3_8b"])
def test_full_size_greedy(name):
    """Greedy emission head at full size; the oracle recomputes a sample of frames over the
    full vocabulary."""
    import torch
    from paper_2609_33645_amd import prunedctc
    from tests.test_gpu_parity import _check_greedy
    wl = workloads.NAMED[name](2)
    say(f"full-size greedy {name}: M={wl.M} D={wl.D} V={wl.V}")
    H, W, _ = to_dev(wl)
    got = prunedctc.greedy_decode(H, W, wl.input_lengths, wl.blank)
    rng = np.random.default_rng(4)
    frames = np.sort(rng.choice(wl.M, size=64, replace=False))
    H64, W64 = wl.H.astype(np.float64), wl.W.astype(np.float64)
    ref = oracle.greedy_decode(H64[frames], W64, [frames.size], wl.blank)
    _check_greedy(wl, H64, W64, np.zeros(wl.V), got, ref, frames=frames)
    del H, W
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
def test_full_size_grouped_export():
    """The grouped export at the zipformer_m size feeding torch's own CTC on the GPU: sampled
    exported rows against the oracle's, every row a distribution, the stock loss against the
    oracle's full-vocabulary loss, and sampled gradient rows (Prop. 1) against the oracle's."""
    import torch
    from paper_2609_33645_amd import prunedctc
    wl = workloads.NAMED["zipformer_m"](0, beam=math.inf)
    say(f"full-size grouped export: N={wl.N} M={wl.M} D={wl.D} V={wl.V}")
    H, W, y = to_dev(wl)
    un = prunedctc.union_remap(y, wl.blank, wl.V)
    K = un["K"]
    uid = un["u_ids"][:K].contiguous()
    Hg = H.clone().requires_grad_(True)
    Wg = W.clone().requires_grad_(True)
    lp = prunedctc.grouped_head(Hg, Wg, uid)
    off = np.concatenate([[0], np.cumsum(wl.input_lengths)])
    Tm = int(wl.input_lengths.max())
    pad = torch.stack([torch.nn.functional.pad(lp[off[n]:off[n + 1]], (0, 0, 0, Tm - int(wl.input_lengths[n])))
                       for n in range(wl.N)], 1)
    loss = torch.nn.functional.ctc_loss(pad, un["y_rel"].long(), torch.as_tensor(wl.input_lengths, dtype=torch.long),
                                        torch.as_tensor(wl.target_lengths, dtype=torch.long), blank=0,
                                        reduction="sum")
    loss.backward()
    torch.cuda.synchronize()
    logp = lp.detach().cpu().numpy()
    say(f"  gpu path done (K={K})")
    rowsum = np.exp(logp.astype(np.float64)).sum(axis=1)
    assert np.abs(rowsum - 1.0).max() < 1e-5

    W64 = wl.W.astype(np.float64)
    H64 = wl.H.astype(np.float64)
    ref_un = oracle.union_remap(wl.targets, wl.target_lengths, wl.blank, wl.V)
    np.testing.assert_array_equal(uid.cpu().numpy(), ref_un["u_ids"])
    rng = np.random.default_rng(11)
    frames, classes = _samples(wl, rng, ref_un["u_ids"])
    ex = oracle.grouped_logprobs(H64[frames], W64, ref_un["u_ids"])
    say(f"  sampled export max err {np.abs(logp[frames] - ex['logp']).max():.3g}")
    assert np.abs(logp[frames] - ex["logp"]).max() < 5e-5

    lam = oracle.log_normalizer(H64, W64)
    S = oracle.selected_logprobs(H64, W64, ref_un["u_ids"], lam)
    dp = oracle.ctc_from_scores(S, ref_un["y_rel"], wl.input_lengths, wl.target_lengths, math.inf)
    assert (dp["status"] == 0).all()
    lr = loss_rel(float(loss.item()), dp["loss"])
    say(f"  stock CTC loss gpu={float(loss.item()):.9g} oracle={dp['loss']:.9g} rel={lr:.3g}")
    assert lr <= 2e-3
    rows = oracle.head_backward_rows(H64, W64, lam, dp["G"], dp["g"], ref_un["u_ids"], frames, classes)
    dH_s = Hg.grad.float()[torch.from_numpy(frames).cuda()].cpu().numpy()
    dW_s = Wg.grad.float()[torch.from_numpy(classes).cuda()].cpu().numpy()
    cH, cW = cosine(dH_s, rows["dH"]), cosine(dW_s, rows["dW"])
    say(f"  sampled gradients cos dH={cH:.7f} dW={cW:.7f}")
    assert cH >= 0.999 and cW >= 0.999
    del lp, pad, loss, Hg, Wg, H, W, y
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
def test_e3_memory_shape_frozen_head():
    """The LLM benchmark's memory shape (107 utterances, M = 11,458, D = 4096, V = 151,936,
    head frozen: no dW).  Utterance losses and dH rows depend only on their own utterance, so
    ten utterances spread over the batch are checked against the oracle run on those alone."""
    import torch
    from paper_2609_33645_amd import prunedctc
    wl = workloads.NAMED["e3_qwen3_8b"](0)
    say(f"e3 shape: N={wl.N} M={wl.M} D={wl.D} V={wl.V} U={int(wl.target_lengths.sum())}")
    H, W, y = to_dev(wl)
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    out = prunedctc.pruned_ctc_fwd_bwd(H, W, y, wl.input_lengths, wl.target_lengths, wl.blank, wl.beam,
                                       want_dW=False)
    torch.cuda.synchronize()
    peak = (torch.cuda.max_memory_allocated() - base) / 2**20
    say(f"  peak above inputs {peak:.1f} MiB (workspace {out['workspace_bytes'] / 2**20:.1f} MiB)")
    assert out["dW"] is None
    assert (out["status"].cpu().numpy() == 0).all()
    pick = np.linspace(0, wl.N - 1, 10).round().astype(np.int64)
    toff = np.concatenate([[0], np.cumsum(wl.input_lengths)])
    yoff = np.concatenate([[0], np.cumsum(wl.target_lengths)])
    fr = np.concatenate([np.arange(toff[n], toff[n + 1]) for n in pick])
    T2, U2 = wl.input_lengths[pick], wl.target_lengths[pick]
    y2 = np.concatenate([wl.targets[yoff[n]:yoff[n + 1]] for n in pick])
    ref = oracle.fwd_bwd(wl.H[fr].astype(np.float64), wl.W.astype(np.float64), y2, T2, U2, wl.blank, wl.beam)
    ln = out["loss_per_utt"].cpu().numpy()[pick]
    say(f"  utterances {pick.tolist()}: losses gpu={ln.tolist()} oracle={ref['loss_n'].tolist()}")
    np.testing.assert_allclose(ln, ref["loss_n"], rtol=1e-5)
    dH = out["dH"][torch.from_numpy(fr).cuda()].cpu().numpy()
    c = cosine(dH, ref["dH"])
    say(f"  dH rows of those utterances: cos={c:.7f} rel={rel_err(dH, ref['dH']):.3g}")
    assert c >= 0.99999
    for i, n in enumerate(pick):       # utterance by utterance
        rows = slice(int(np.sum(T2[:i])), int(np.sum(T2[:i + 1])))
        assert cosine(dH[rows], ref["dH"][rows]) >= 0.99999, f"utterance {n}"
    del out, H, W, y
    torch.cuda.empty_cache()
