"""Alignment-beam sweep by discarded posterior mass (App. B.3 "Discarded posterior mass").

For each beam, delta_n is the posterior mass (given the transcript) of the alignments the
beam drops; a batch meets the criterion when max_n delta_n <= 1e-11, and the required beam
is the smallest tested beam that meets it.  Everything runs on the GPU through the C ABI:
union and relabelling, the full-vocabulary normaliser and S, then the discarded mass.

    python -m paper_2609_33645_amd.beam_sweep [--workload qwen3_8b] [--seed 0]
"""
from __future__ import annotations

import argparse
import json
import math
import sys
from typing import Dict, Sequence

import numpy as np

DEFAULT_BEAMS = (8.0, 10.0, 16.0, 25.0, 32.0, 50.0, 64.0, 75.0, 100.0)
CRITERION = 1e-11


def beam_sweep(H, W, targets, input_lengths, target_lengths, blank: int = 0,
               beams: Sequence[float] = DEFAULT_BEAMS, criterion: float = CRITERION) -> Dict[str, object]:
    """H [M, D], W [V, D] device tensors (bf16 or fp32), targets device int32; lengths on the
    host.  Returns per-beam maximum delta, the count of utterances above the criterion, the
    required beam (None if no tested beam meets it) and the full delta matrix."""
    from . import prunedctc
    un = prunedctc.union_remap(targets, blank, int(W.shape[0]))
    sel = prunedctc.lse_select(H, W, un["u_ids"])
    delta = prunedctc.discarded_mass(sel["S"], un["y_rel"], input_lengths, target_lengths, beams)
    d = delta.cpu().numpy()
    rows = []
    required = None
    for b, beam in enumerate(beams):
        ok = ~np.isnan(d[b])
        mx = float(np.max(d[b][ok])) if ok.any() else float("nan")
        above = int(np.sum(d[b][ok] > criterion))
        rows.append({"beam": float(beam), "max_delta": mx, "above": above, "utterances": int(ok.sum())})
        if required is None and above == 0:
            required = float(beam)
    return {"rows": rows, "required_beam": required, "criterion": criterion, "delta": d}


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="qwen3_8b")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--beams", default=",".join(str(b) for b in DEFAULT_BEAMS))
    a = ap.parse_args(argv)
    import torch
    from . import workloads
    wl = workloads.NAMED[a.workload](a.seed)
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    H = torch.from_numpy(wl.H).cuda().to(dt)
    W = torch.from_numpy(wl.W).cuda().to(dt)
    y = torch.from_numpy(wl.targets).cuda()
    beams = [float(x) for x in a.beams.split(",")]
    res = beam_sweep(H, W, y, wl.input_lengths, wl.target_lengths, wl.blank, beams)
    for r in res["rows"]:
        print(f"{a.workload} seed={a.seed} beam={r['beam']:6.1f}  max delta={r['max_delta']:.3e}  "
              f"above {CRITERION:g}: {r['above']}/{r['utterances']}", flush=True)
    print(json.dumps({"workload": a.workload, "seed": a.seed, "required_beam": res["required_beam"],
                      "rows": res["rows"]}), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
