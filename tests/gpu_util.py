"""Helpers for the GPU parity tests: move seeded workloads to the device, error metrics."""
from __future__ import annotations

import sys

import numpy as np


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(wl):
    import torch
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    H = torch.from_numpy(np.ascontiguousarray(wl.H, np.float32)).to("cuda").to(dt)
    W = torch.from_numpy(np.ascontiguousarray(wl.W, np.float32)).to("cuda").to(dt)
    y = torch.from_numpy(np.ascontiguousarray(wl.targets, np.int32)).to("cuda")
    return H, W, y


def rel_err(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-300))


def cosine(a, b) -> float:
    a = np.asarray(a, np.float64).ravel()
    b = np.asarray(b, np.float64).ravel()
    na, nb = np.linalg.norm(a), np.linalg.norm(b)
    if na == 0 and nb == 0:
        return 1.0
    return float(a @ b / (na * nb))


def loss_rel(a: float, b: float) -> float:
    return abs(a - b) / max(abs(b), 1e-300)


def run_gpu(wl, chunk=0, want_dH=True, want_dW=True):
    from paper_2609_33645_amd import prunedctc
    H, W, y = to_dev(wl)
    out = prunedctc.pruned_ctc_fwd_bwd(H, W, y, wl.input_lengths, wl.target_lengths, wl.blank, wl.beam,
                                       chunk=chunk, want_dH=want_dH, want_dW=want_dW)
    res = {"loss": float(out["loss"].item()), "loss_n": out["loss_per_utt"].cpu().numpy(),
           "status": out["status"].cpu().numpy()}
    if want_dH:
        res["dH"] = out["dH"].cpu().numpy()
    if want_dW:
        res["dW"] = out["dW"].cpu().numpy()
    res["workspace_bytes"] = out["workspace_bytes"]
    return res
