"""The allocation-free entry point (pruned_ctc_fwd_bwd_noalloc: the library's static per-device
scratch instead of a caller workspace) against the workspace entry point
(pruned_ctc_fwd_bwd_ex) on the same inputs, through the C ABI.

Two calls in a row share the scratch, the second on a smaller batch (the first call's
contents are still there).  Bars: statuses exact; bf16 loss relative error <= 2e-3 and
gradient cosine >= 0.999 (with tighter checks of the accuracy reached); fp32 loss relative
error <= 1e-5 and gradient max-abs relative error <= 1e-4.  A batch the scratch cannot hold
is refused before any work is queued.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2609_33645_amd import workloads
from tests.gpu_util import cosine, loss_rel, rel_err, say, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_33645_amd import prunedctc
    prunedctc.lib()
    yield


def _outputs(N, M, D, V, want_db):
    """Output buffers for the allocation-free call, filled with NaN so that anything left
    unwritten shows."""
    import torch
    f = dict(device="cuda")
    out = {"loss": torch.full((1,), math.nan, dtype=torch.float64, **f),
           "loss_per_utt": torch.full((N,), math.nan, dtype=torch.float64, **f),
           "status": torch.full((N,), -7, dtype=torch.int32, **f),
           "dH": torch.full((M, D), math.nan, dtype=torch.float32, **f),
           "dW": torch.full((V, D), math.nan, dtype=torch.float32, **f)}
    if want_db:
        out["db"] = torch.full((V,), math.nan, dtype=torch.float32, **f)
    return out


def _compare(name, got, want, fp32):
    got = got.cpu().numpy()
    want = want.cpu().numpy()
    assert np.isfinite(got).all(), name
    if fp32:
        assert rel_err(got, want) <= 1e-4, name
    else:
        c = cosine(got, want)
        say(f"  {name}: cos={c:.8f} rel={rel_err(got, want):.3g}")
        assert c >= 0.999 and c >= 0.99999, name


def _run_pair(wl, bias=None, weights=None, want_db=False):
    """One call through each entry point on the same inputs; returns the allocation-free
    call's outputs after checking them against the workspace entry point's."""
    import torch
    from paper_2609_33645_amd import prunedctc
    H, W, y = to_dev(wl)
    b = None if bias is None else torch.from_numpy(bias).cuda()
    w = None if weights is None else torch.from_numpy(weights).cuda()
    ref = prunedctc.pruned_ctc_fwd_bwd(H, W, y, wl.input_lengths, wl.target_lengths, wl.blank, wl.beam, bias=b,
                                       utt_weight=w, want_db=want_db)
    out = prunedctc.pruned_ctc_fwd_bwd_noalloc(H, W, y, wl.input_lengths, wl.target_lengths,
                                               _outputs(wl.N, wl.M, wl.D, wl.V, want_db), blank=wl.blank,
                                               beam=wl.beam, bias=b, utt_weight=w)
    torch.cuda.synchronize()
    fp32 = wl.dtype == "f32"
    np.testing.assert_array_equal(out["status"].cpu().numpy(), ref["status"].cpu().numpy())
    lr = loss_rel(float(out["loss"].item()), float(ref["loss"].item()))
    say(f"  loss no-alloc={float(out['loss'].item()):.10g} workspace={float(ref['loss'].item()):.10g} rel={lr:.3g}")
    assert lr <= (1e-5 if fp32 else 2e-3) and lr <= 1e-5
    np.testing.assert_allclose(out["loss_per_utt"].cpu().numpy(), ref["loss_per_utt"].cpu().numpy(), rtol=1e-5)
    for k in ("dH", "dW") + (("db",) if want_db else ()):
        _compare(k, out[k], ref[k], fp32)
    return out


def test_noalloc_two_calls_match_workspace_entry():
    """A larger then a smaller batch (bias, loss weights and db on the first), both against
    the workspace entry point; the smaller one also against the oracle."""
    wl1 = workloads.random_small(201, N=6, T_range=(60, 240), D=256, V=20_000, dtype="bf16", p_repeat=0.1,
                                 beam=16.0, w_std=0.5 * math.sqrt(128 / 256))
    rng = np.random.default_rng(201)
    bias = (0.5 * rng.standard_normal(wl1.V)).astype(np.float32)
    weights = rng.uniform(0.5, 1.5, size=wl1.N).astype(np.float32)
    say(f"no-alloc call 1: N={wl1.N} M={wl1.M} D={wl1.D} V={wl1.V}")
    _run_pair(wl1, bias=bias, weights=weights, want_db=True)
    wl2 = workloads.random_small(202, N=3, T_range=(10, 70), D=256, V=20_000, dtype="bf16", p_repeat=0.1,
                                 beam=math.inf, w_std=0.5 * math.sqrt(128 / 256))
    say(f"no-alloc call 2: N={wl2.N} M={wl2.M} (smaller)")
    out = _run_pair(wl2)
    ref = oracle.fwd_bwd(wl2.H, wl2.W, wl2.targets, wl2.input_lengths, wl2.target_lengths, wl2.blank, wl2.beam)
    assert loss_rel(float(out["loss"].item()), ref["loss"]) <= 1e-5
    assert cosine(out["dH"].cpu().numpy(), ref["dH"]) >= 0.99999
    assert cosine(out["dW"].cpu().numpy(), ref["dW"]) >= 0.99999


def test_noalloc_fp32_then_smaller():
    """The fp32 path, a larger then a smaller batch."""
    for seed, N, Tr in ((203, 5, (40, 160)), (204, 2, (5, 30))):
        wl = workloads.random_small(seed, N=N, T_range=Tr, D=136, V=3000, dtype="f32", p_repeat=0.1, beam=math.inf,
                                    w_std=0.5)
        say(f"no-alloc fp32: N={wl.N} M={wl.M}")
        _run_pair(wl)


@pytest.mark.timeout(300)
def test_noalloc_full_size_zipformer_m():
    """The benchmark's workload: the scratch cannot hold the default 60,160-column backward
    chunk, so the call takes the widest chunk that fits; results match the workspace entry
    point's (default chunk) to the stated bars."""
    from paper_2609_33645_amd import prunedctc
    wl = workloads.zipformer_m(0, beam=16.0)
    say(f"no-alloc full size zipformer_m: M={wl.M} V={wl.V}; scratch {prunedctc.noalloc_scratch_bytes() >> 20} MiB")
    assert prunedctc.workspace_size(1, wl.input_lengths, wl.target_lengths, wl.D, wl.V, wl.beam) > \
        prunedctc.noalloc_scratch_bytes()
    _run_pair(wl)


def test_noalloc_refuses_oversized_batch():
    """The 107-utterance D = 4096 shape needs more scratch than the array holds even at the
    narrowest chunk, and an explicit chunk too wide for it is refused too: PCTC_EWORKSPACE,
    before any work (the outputs keep their NaN fill)."""
    import torch
    from paper_2609_33645_amd import prunedctc
    T = np.full(107, 107, np.int32)
    U = np.full(107, 25, np.int32)
    M, D, V = int(T.sum()), 4096, 151_936
    H = torch.zeros((M, D), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros((V, D), dtype=torch.bfloat16, device="cuda")
    y = torch.ones(int(U.sum()), dtype=torch.int32, device="cuda")
    out = _outputs(107, M, D, V, False)
    with pytest.raises(prunedctc.PrunedCTCError) as e:
        prunedctc.pruned_ctc_fwd_bwd_noalloc(H, W, y, T, U, out, beam=32.0)
    assert e.value.code == -4
    assert math.isnan(float(out["loss"].item()))
    zwl = workloads.zipformer_m(0, beam=16.0)
    Hz, Wz, yz = to_dev(zwl)
    with pytest.raises(prunedctc.PrunedCTCError) as e:
        prunedctc.pruned_ctc_fwd_bwd_noalloc(Hz, Wz, yz, zwl.input_lengths, zwl.target_lengths,
                                             _outputs(zwl.N, zwl.M, zwl.D, zwl.V, False), beam=16.0,
                                             chunk=65536)
    assert e.value.code == -4
