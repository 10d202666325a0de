"""Python binding of libprunedctc.so (C ABI in include/prunedctc.h).

Argument marshalling only: every step of the computation runs in the library's HIP
kernels.  PyTorch supplies device memory (outputs and workspace come from its caching
allocator) and the current stream.  If the library has not been built, every call
raises ``PrunedCTCError``; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Dict, Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libprunedctc.so")

PCTC_F32, PCTC_BF16 = 0, 1
STATUS = {0: "ok", -1: "invalid argument", -2: "bad label", -3: "bad length", -4: "workspace too small",
          -5: "HIP error", -6: "target too long"}
UTT_OK, UTT_NOT_ALIGNABLE, UTT_NONFINITE = 0, 1, 2
MAX_TARGET = 1023


class PrunedCTCError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(msg)
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """Load the HIP library once.  torch is imported first so that the library binds to
    the HIP runtime torch already loaded."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise PrunedCTCError(-5, f"HIP library not built: {LIB_PATH} is missing "
                                 f"(run: python -m paper_2609_33645_amd.build)")
    L = ctypes.CDLL(LIB_PATH)
    c_i32, c_f, c_p, c_sz = ctypes.c_int32, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t
    i32p = ctypes.POINTER(ctypes.c_int32)
    L.pctc_workspace_size.argtypes = [c_i32, c_i32, i32p, i32p, c_i32, c_i32, c_f, c_i32]
    L.pctc_workspace_size.restype = c_sz
    L.pctc_workspace_size_ex.argtypes = [c_i32, c_i32, i32p, i32p, c_i32, c_i32, c_f, c_i32, c_i32]
    L.pctc_workspace_size_ex.restype = c_sz
    L.pctc_normaliser_chunk_columns.argtypes = [c_i32, c_i32, i32p, i32p, c_i32, c_i32, c_f, c_i32, c_i32]
    L.pctc_normaliser_chunk_columns.restype = c_i32
    L.pruned_ctc_fwd_bwd.argtypes = [c_i32, c_p, c_i32, c_p, c_i32, c_p, i32p, i32p, c_i32, c_i32, c_f, c_i32,
                                     c_p, c_p, c_p, c_p, c_p, c_p, c_sz, c_p]
    L.pruned_ctc_fwd_bwd.restype = c_i32
    L.pruned_ctc_fwd_bwd_ex.argtypes = [c_i32, c_p, c_i32, c_p, c_p, c_i32, c_p, i32p, i32p, c_i32, c_i32, c_f, c_i32,
                                        c_p, c_p, c_p, c_p, c_p, c_p, c_p, c_p, c_sz, c_p]
    L.pruned_ctc_fwd_bwd_ex.restype = c_i32
    L.pctc_noalloc_scratch_bytes.argtypes = []
    L.pctc_noalloc_scratch_bytes.restype = c_sz
    L.pruned_ctc_fwd_bwd_noalloc.argtypes = [c_i32, c_p, c_i32, c_p, c_p, c_i32, c_p, i32p, i32p, c_i32, c_i32, c_f,
                                             c_i32, c_p, c_p, c_p, c_p, c_p, c_p, c_p, c_p]
    L.pruned_ctc_fwd_bwd_noalloc.restype = c_i32
    L.pctc_status_string.argtypes = [c_i32]
    L.pctc_status_string.restype = ctypes.c_char_p
    L.pctc_last_error.argtypes = []
    L.pctc_last_error.restype = ctypes.c_char_p
    L.pctc_union_scratch_bytes.argtypes = [c_i32]
    L.pctc_union_scratch_bytes.restype = c_sz
    L.pctc_union_remap.argtypes = [c_p, c_i32, c_i32, c_i32, c_p, c_p, c_p, c_p, c_p, c_p, c_p]
    L.pctc_union_remap.restype = c_i32
    L.pctc_lse_scratch_bytes.argtypes = [c_i32, c_i32]
    L.pctc_lse_scratch_bytes.restype = c_sz
    L.pctc_lse_select.argtypes = [c_i32, c_p, c_i32, c_i32, c_p, c_i32, c_p, c_p, c_i32, c_p, c_p, c_i32, c_p, c_p]
    L.pctc_lse_select.restype = c_i32
    L.pctc_dp_scratch_bytes.argtypes = [c_i32, i32p, i32p, c_f]
    L.pctc_dp_scratch_bytes.restype = c_sz
    L.pctc_ctc_dp.argtypes = [c_p, c_i32, c_i32, c_p, i32p, i32p, c_i32, c_f, c_p, c_p, c_p, c_p, c_p, c_p, c_p]
    L.pctc_ctc_dp.restype = c_i32
    L.pctc_greedy_workspace_size.argtypes = [c_i32, c_i32, c_i32]
    L.pctc_greedy_workspace_size.restype = c_sz
    L.pctc_greedy_decode.argtypes = [c_i32, c_p, c_i32, c_p, c_p, c_i32, i32p, c_i32, c_i32, c_p, c_p, c_p, c_p, c_sz,
                                     c_p]
    L.pctc_greedy_decode.restype = c_i32
    L.pctc_discarded_mass_scratch_bytes.argtypes = [c_i32, i32p, i32p]
    L.pctc_discarded_mass_scratch_bytes.restype = c_sz
    L.pctc_discarded_mass.argtypes = [c_p, c_i32, c_i32, c_p, i32p, i32p, c_i32, ctypes.POINTER(ctypes.c_float), c_i32,
                                      c_p, c_p, c_p]
    L.pctc_discarded_mass.restype = c_i32
    L.pctc_bwd_scratch_bytes.argtypes = [c_i32, c_i32, c_i32, c_i32, c_i32, c_i32]
    L.pctc_bwd_scratch_bytes.restype = c_sz
    L.pctc_bwd_chunk.argtypes = [c_i32, c_i32, c_i32, c_i32, c_i32]
    L.pctc_bwd_chunk.restype = c_i32
    L.pctc_head_bwd.argtypes = [c_i32, c_p, c_i32, c_i32, c_p, c_i32, c_p, c_p, c_i32, c_p, c_p, c_i32, c_p, c_p,
                                c_p, c_p]
    L.pctc_head_bwd.restype = c_i32
    L.pctc_grouped_workspace_size.argtypes = [c_i32, c_i32, c_i32, c_i32, c_i32, c_i32]
    L.pctc_grouped_workspace_size.restype = c_sz
    L.pctc_grouped_logprobs.argtypes = [c_i32, c_p, c_i32, c_i32, c_p, c_p, c_i32, c_p, c_i32, c_p, c_p, c_p, c_sz, c_p]
    L.pctc_grouped_logprobs.restype = c_i32
    L.pctc_grouped_backward.argtypes = [c_i32, c_p, c_i32, c_i32, c_p, c_p, c_i32, c_p, c_i32, c_p, c_p, c_p, c_i32,
                                        c_p, c_p, c_p, c_p, c_sz, c_p]
    L.pctc_grouped_backward.restype = c_i32
    L.pctc_prof_enable.argtypes = [c_i32]
    L.pctc_prof_select.argtypes = [ctypes.c_char_p]
    L.pctc_prof_reset.argtypes = []
    L.pctc_prof_count.argtypes = []
    L.pctc_prof_count.restype = c_i32
    L.pctc_prof_get.argtypes = [c_i32, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_double),
                                ctypes.POINTER(ctypes.c_int64)]
    L.pctc_prof_get.restype = c_i32
    _lib = L
    return L


def _check(code: int, what: str) -> None:
    if code != 0:
        L = lib()
        detail = L.pctc_last_error().decode() if code == -5 else ""
        raise PrunedCTCError(code, f"{what}: {L.pctc_status_string(code).decode()} {detail}".strip())


def _host_i32(x) -> np.ndarray:
    if isinstance(x, torch.Tensor):
        x = x.detach().cpu().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32))


def _i32p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return PCTC_BF16
    if t.dtype == torch.float32:
        return PCTC_F32
    raise PrunedCTCError(-1, f"unsupported dtype {t.dtype}")


def _workspace(nbytes: int, device) -> torch.Tensor:
    ws = torch.empty(max(int(nbytes), 256) + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off:off + max(int(nbytes), 256)]


def _bias_vector(bias: torch.Tensor, V: int, dev) -> torch.Tensor:
    if bias.numel() != V:
        raise PrunedCTCError(-1, f"bias must hold V = {V} values, got {bias.numel()}")
    return bias.reshape(V).to(device=dev, dtype=torch.float32).contiguous()


WS_NO_DW = 1  # workspace for calls without dW (frozen head)


def workspace_size(dtype: int, input_lengths, target_lengths, D: int, V: int, beam: float, chunk: int = 0,
                   want_dW: bool = True) -> int:
    T = _host_i32(input_lengths)
    U = _host_i32(target_lengths)
    return int(lib().pctc_workspace_size_ex(dtype, T.size, _i32p(T), _i32p(U), D, V, float(beam), chunk,
                                            0 if want_dW else WS_NO_DW))


def normaliser_chunk_columns(dtype: int, input_lengths, target_lengths, D: int, V: int, beam: float, chunk: int = 0,
                             want_dW: bool = True) -> int:
    """Vocabulary columns of the first backward chunk that the normaliser of a fused call writes
    itself (0: every chunk is recomputed); see pctc_normaliser_chunk_columns."""
    T = _host_i32(input_lengths)
    U = _host_i32(target_lengths)
    return int(lib().pctc_normaliser_chunk_columns(dtype, T.size, _i32p(T), _i32p(U), D, V, float(beam), chunk,
                                                   0 if want_dW else WS_NO_DW))


def bwd_chunk(dtype: int, M: int, D: int, V: int, chunk: int = 0) -> int:
    """Vocabulary columns per backward step used for this problem (0 chunk = the default)."""
    return int(lib().pctc_bwd_chunk(int(dtype), int(M), int(D), int(V), int(chunk)))


def _grad_buffer(t: Optional[torch.Tensor], shape, dev) -> torch.Tensor:
    if t is None:
        return torch.empty(shape, dtype=torch.float32, device=dev)
    if t.dtype != torch.float32 or tuple(t.shape) != tuple(shape) or not t.is_contiguous() or t.device != dev:
        raise PrunedCTCError(-1, f"gradient buffer must be contiguous float32 {tuple(shape)} on {dev}")
    return t


def pruned_ctc_fwd_bwd(H: torch.Tensor, W: torch.Tensor, targets: torch.Tensor, input_lengths: Sequence[int],
                       target_lengths: Sequence[int], blank: int = 0, beam: float = math.inf, chunk: int = 0,
                       want_dH: bool = True, want_dW: bool = True, workspace: Optional[torch.Tensor] = None,
                       stream=None, dH_out: Optional[torch.Tensor] = None,
                       dW_out: Optional[torch.Tensor] = None, bias: Optional[torch.Tensor] = None,
                       utt_weight: Optional[torch.Tensor] = None, want_db: bool = False) -> Dict[str, torch.Tensor]:
    """Loss and head gradients of Pruned CTC.  H [M, D] and W [V, D] are device tensors of
    the same dtype (bfloat16 or float32); targets is a device int32 tensor; the length
    arrays are host sequences.  Returns loss (float64 [1]), loss_per_utt, status, dH, dW
    and, with want_db, db.  dH_out / dW_out: optional preallocated float32 [M, D] / [V, D]
    gradient buffers.  bias: optional float32 [V] head bias (logits H W^T + b; a blank
    offset eta is added to bias[blank], and its gradient is db[blank]).  utt_weight:
    optional float32 [N] loss weights (loss = sum_n w_n L_n; loss_per_utt stays
    unweighted)."""
    L = lib()
    dt = _dtype_code(H)
    if W.dtype != H.dtype:
        raise PrunedCTCError(-1, "H and W must have the same dtype")
    if not (H.is_cuda and W.is_cuda and targets.is_cuda):
        raise PrunedCTCError(-1, "H, W and targets must be device tensors")
    H = H.contiguous()
    W = W.contiguous()
    targets = targets.to(torch.int32).contiguous()
    T = _host_i32(input_lengths)
    U = _host_i32(target_lengths)
    N = int(T.size)
    M, D = int(H.shape[0]), int(H.shape[1])
    V = int(W.shape[0])
    if W.shape[1] != D:
        raise PrunedCTCError(-1, "H and W widths differ")
    if int(T.sum()) != M:
        raise PrunedCTCError(-1, "sum of input lengths differs from the rows of H")
    if int(U.sum()) != int(targets.numel()):
        raise PrunedCTCError(-1, "sum of target lengths differs from the number of targets")
    dev = H.device
    nbytes = int(L.pctc_workspace_size_ex(dt, N, _i32p(T), _i32p(U), D, V, float(beam), chunk,
                                          0 if want_dW else WS_NO_DW))
    if nbytes == 0:
        code = -6 if (U > MAX_TARGET).any() else (-3 if ((T < 1).any() or (U < 0).any()) else -1)
        _check(code, "pruned_ctc_fwd_bwd")
    ws = workspace if workspace is not None else _workspace(nbytes, dev)
    # the library writes all three on success: one uninitialised allocation, split in views
    n1 = max(N, 1)
    small = torch.empty(8 + 8 * n1 + 4 * n1, dtype=torch.uint8, device=dev)
    loss = small[:8].view(torch.float64)
    loss_n = small[8:8 + 8 * n1].view(torch.float64)
    status = small[8 + 8 * n1:].view(torch.int32)
    dH = _grad_buffer(dH_out, (M, D), dev) if want_dH else None
    dW = _grad_buffer(dW_out, (V, D), dev) if want_dW else None
    db = torch.empty(V, dtype=torch.float32, device=dev) if want_db else None
    if bias is not None:
        bias = _bias_vector(bias, V, dev)
    if utt_weight is not None:
        utt_weight = utt_weight.to(device=dev, dtype=torch.float32).contiguous()
        if utt_weight.numel() != N:
            raise PrunedCTCError(-1, "utt_weight must have N entries")
    if bias is None and utt_weight is None and db is None:
        code = L.pruned_ctc_fwd_bwd(dt, _ptr(H), D, _ptr(W), V, _ptr(targets), _i32p(T), _i32p(U), N, int(blank),
                                    float(beam), int(chunk), _ptr(loss), _ptr(loss_n), _ptr(status), _ptr(dH),
                                    _ptr(dW), ctypes.c_void_p(ws.data_ptr()), ctypes.c_size_t(ws.numel()),
                                    _stream(stream))
    else:
        code = L.pruned_ctc_fwd_bwd_ex(dt, _ptr(H), D, _ptr(W), _ptr(bias), V, _ptr(targets), _i32p(T), _i32p(U), N,
                                       int(blank), float(beam), int(chunk), _ptr(utt_weight), _ptr(loss), _ptr(loss_n),
                                       _ptr(status), _ptr(dH), _ptr(dW), _ptr(db), ctypes.c_void_p(ws.data_ptr()),
                                       ctypes.c_size_t(ws.numel()), _stream(stream))
    _check(code, "pruned_ctc_fwd_bwd")
    return {"loss": loss, "loss_per_utt": loss_n[:N], "status": status[:N], "dH": dH, "dW": dW, "db": db,
            "workspace_bytes": nbytes}


def noalloc_scratch_bytes() -> int:
    """Size of the allocation-free entry point's per-device scratch array."""
    return int(lib().pctc_noalloc_scratch_bytes())


def pruned_ctc_fwd_bwd_noalloc(H: torch.Tensor, W: torch.Tensor, targets: torch.Tensor,
                               input_lengths: Sequence[int], target_lengths: Sequence[int], out: Dict[str, torch.Tensor],
                               blank: int = 0, beam: float = math.inf, chunk: int = 0,
                               bias: Optional[torch.Tensor] = None, utt_weight: Optional[torch.Tensor] = None,
                               stream=None) -> Dict[str, torch.Tensor]:
    """The fused call through pruned_ctc_fwd_bwd_noalloc: the library uses its own static
    scratch, and every output is a caller buffer passed in `out` (allocated beforehand):
    loss (float64 [1]), loss_per_utt (float64 [N]) and status (int32 [N]) or absent, and
    dH (float32 [M, D]), dW (float32 [V, D]), db (float32 [V]) or absent.  H, W, targets,
    bias and utt_weight must already be contiguous device tensors of the right dtypes (no
    conversion or copy is made here).  Returns `out`."""
    L = lib()
    dt = _dtype_code(H)
    T = _host_i32(input_lengths)
    U = _host_i32(target_lengths)
    N = int(T.size)
    for name, t in (("H", H), ("W", W), ("targets", targets), ("bias", bias), ("utt_weight", utt_weight)):
        if t is not None and not (t.is_cuda and t.is_contiguous()):
            raise PrunedCTCError(-1, f"{name} must be a contiguous device tensor")
    if targets.dtype != torch.int32 or W.dtype != H.dtype:
        raise PrunedCTCError(-1, "targets must be int32 and W of H's dtype")
    if bias is not None and bias.dtype != torch.float32 or utt_weight is not None and utt_weight.dtype != torch.float32:
        raise PrunedCTCError(-1, "bias and utt_weight must be float32")
    code = L.pruned_ctc_fwd_bwd_noalloc(dt, _ptr(H), int(H.shape[1]), _ptr(W), _ptr(bias), int(W.shape[0]),
                                        _ptr(targets), _i32p(T), _i32p(U), N, int(blank), float(beam), int(chunk),
                                        _ptr(utt_weight), _ptr(out["loss"]), _ptr(out.get("loss_per_utt")),
                                        _ptr(out.get("status")), _ptr(out.get("dH")), _ptr(out.get("dW")),
                                        _ptr(out.get("db")), _stream(stream))
    _check(code, "pruned_ctc_fwd_bwd_noalloc")
    return out


# ---- stage entry points ------------------------------------------------------------------

def union_remap(targets: torch.Tensor, blank: int, V: int, stream=None) -> Dict[str, torch.Tensor]:
    L = lib()
    targets = targets.to(torch.int32).contiguous()
    dev = targets.device
    Y = int(targets.numel())
    remap = torch.empty(V, dtype=torch.int32, device=dev)
    u_ids = torch.empty(1 + Y, dtype=torch.int32, device=dev)
    y_rel = torch.empty(max(Y, 1), dtype=torch.int32, device=dev)
    K = torch.zeros(1, dtype=torch.int32, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    scratch = _workspace(int(L.pctc_union_scratch_bytes(int(V))), dev)
    code = L.pctc_union_remap(_ptr(targets), Y, int(blank), int(V), _ptr(remap), _ptr(u_ids), _ptr(y_rel), _ptr(K),
                              _ptr(err), ctypes.c_void_p(scratch.data_ptr()), _stream(stream))
    _check(code, "pctc_union_remap")
    k = int(K.item())
    return {"remap": remap, "u_ids": u_ids[:k], "y_rel": y_rel[:Y], "K": k}


def lse_select(H: torch.Tensor, W: torch.Tensor, u_ids: Optional[torch.Tensor] = None,
               stream=None) -> Dict[str, torch.Tensor]:
    """lambda [M] (float64) and, given the union u_ids, S [M, K] (float32)."""
    L = lib()
    dt = _dtype_code(H)
    H = H.contiguous()
    W = W.contiguous()
    M, D = int(H.shape[0]), int(H.shape[1])
    V = int(W.shape[0])
    dev = H.device
    lam = torch.empty(max(M, 1), dtype=torch.float64, device=dev)
    scratch = _workspace(int(L.pctc_lse_scratch_bytes(M, D)), dev)
    S = Kdev = None
    K = 1
    ldS = 1
    if u_ids is not None:
        u_ids = u_ids.to(torch.int32).contiguous()
        K = int(u_ids.numel())
        ldS = ((K + 3) // 4) * 4
        S = torch.zeros((max(M, 1), ldS), dtype=torch.float32, device=dev)
        Kdev = torch.tensor([K], dtype=torch.int32, device=dev)
    code = L.pctc_lse_select(dt, _ptr(H), M, D, _ptr(W), V, _ptr(u_ids), _ptr(Kdev), K, _ptr(lam), _ptr(S), ldS,
                             ctypes.c_void_p(scratch.data_ptr()), _stream(stream))
    _check(code, "pctc_lse_select")
    out = {"lam": lam[:M]}
    if S is not None:
        out["S"] = S[:M, :K]
    return out


def ctc_dp(S: torch.Tensor, y_rel: torch.Tensor, input_lengths, target_lengths, beam: float = math.inf,
           want_mask: bool = False, stream=None) -> Dict[str, torch.Tensor]:
    """Alignment stage on given selected-class scores S [M, K] (column 0 = blank)."""
    L = lib()
    T = _host_i32(input_lengths)
    U = _host_i32(target_lengths)
    N = int(T.size)
    M, K = int(S.shape[0]), int(S.shape[1])
    dev = S.device
    ldS = ((K + 3) // 4) * 4
    Sp = torch.zeros((max(M, 1), ldS), dtype=torch.float32, device=dev)
    Sp[:M, :K] = S.to(torch.float32)
    y_rel = y_rel.to(torch.int32).contiguous()
    G = torch.empty((max(M, 1), ldS), dtype=torch.float32, device=dev)
    g = torch.empty(max(M, 1), dtype=torch.float32, device=dev)
    loss_n = torch.zeros(max(N, 1), dtype=torch.float64, device=dev)
    status = torch.zeros(max(N, 1), dtype=torch.int32, device=dev)
    lattice = int(np.sum(T.astype(np.int64) * (2 * U.astype(np.int64) + 1)))
    mask = torch.zeros(max(lattice, 1), dtype=torch.uint8, device=dev) if want_mask else None
    nbytes = int(L.pctc_dp_scratch_bytes(N, _i32p(T), _i32p(U), float(beam)))
    scratch = _workspace(nbytes, dev)
    code = L.pctc_ctc_dp(_ptr(Sp), ldS, K, _ptr(y_rel), _i32p(T), _i32p(U), N, float(beam), _ptr(loss_n),
                         _ptr(status), _ptr(G), _ptr(g), _ptr(mask), ctypes.c_void_p(scratch.data_ptr()),
                         _stream(stream))
    _check(code, "pctc_ctc_dp")
    out = {"loss_per_utt": loss_n[:N], "status": status[:N], "G": G[:M, :K], "g": g[:M]}
    if mask is not None:
        out["mask"] = mask[:lattice]
    return out


def greedy_decode(H: torch.Tensor, W: torch.Tensor, input_lengths, blank: int = 0,
                  bias: Optional[torch.Tensor] = None, stream=None, to_host: bool = True) -> Dict[str, object]:
    """Framewise full-vocabulary argmax ids [M] and the collapsed token sequence of each
    utterance (a list of lists, only when to_host), plus the device buffers (tokens of
    utterance n at the offset of its first frame)."""
    L = lib()
    dt = _dtype_code(H)
    H = H.contiguous()
    W = W.contiguous()
    T = _host_i32(input_lengths)
    N = int(T.size)
    M, D = int(H.shape[0]), int(H.shape[1])
    V = int(W.shape[0])
    if int(T.sum()) != M:
        raise PrunedCTCError(-1, "sum of input lengths differs from the rows of H")
    dev = H.device
    if bias is not None:
        bias = _bias_vector(bias, V, dev)
    ids = torch.empty(max(M, 1), dtype=torch.int32, device=dev)
    tokens = torch.empty(max(M, 1), dtype=torch.int32, device=dev)
    lengths = torch.empty(max(N, 1), dtype=torch.int32, device=dev)
    ws = _workspace(int(L.pctc_greedy_workspace_size(N, M, D)), dev)
    code = L.pctc_greedy_decode(dt, _ptr(H), D, _ptr(W), _ptr(bias), V, _i32p(T), N, int(blank), _ptr(ids),
                                _ptr(tokens), _ptr(lengths), ctypes.c_void_p(ws.data_ptr()), ctypes.c_size_t(ws.numel()),
                                _stream(stream))
    _check(code, "pctc_greedy_decode")
    if not to_host:
        return {"ids": ids[:M], "tokens_dev": tokens[:M], "token_lengths": lengths[:N]}
    off = np.concatenate([[0], np.cumsum(T)]).astype(np.int64)
    tk = tokens.cpu().numpy()
    ln = lengths.cpu().numpy()[:N]
    seqs = [tk[off[n]:off[n] + ln[n]].tolist() for n in range(N)]
    return {"ids": ids[:M], "tokens": seqs, "token_lengths": lengths[:N]}


def discarded_mass(S: torch.Tensor, y_rel: torch.Tensor, input_lengths, target_lengths, beams: Sequence[float],
                   stream=None) -> torch.Tensor:
    """Discarded posterior mass delta [len(beams), N] (float64) of every utterance at every
    beam, on given selected-class scores S [M, K] (column 0 = blank)."""
    L = lib()
    T = _host_i32(input_lengths)
    U = _host_i32(target_lengths)
    N = int(T.size)
    M, K = int(S.shape[0]), int(S.shape[1])
    dev = S.device
    if S.dtype == torch.float32 and S.is_contiguous() and K % 4 == 0 and M > 0:
        ldS, Sp = K, S                     # already in the library's layout
    else:
        ldS = ((K + 3) // 4) * 4
        Sp = torch.zeros((max(M, 1), ldS), dtype=torch.float32, device=dev)
        Sp[:M, :K] = S.to(torch.float32)
    y_rel = y_rel.to(torch.int32).contiguous()
    b = np.ascontiguousarray(np.asarray(beams, np.float32))
    delta = torch.empty((max(len(b), 1), max(N, 1)), dtype=torch.float64, device=dev)
    nbytes = int(L.pctc_discarded_mass_scratch_bytes(N, _i32p(T), _i32p(U)))
    scratch = _workspace(nbytes, dev)
    code = L.pctc_discarded_mass(_ptr(Sp), ldS, K, _ptr(y_rel), _i32p(T), _i32p(U), N,
                                 b.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), int(b.size), _ptr(delta),
                                 ctypes.c_void_p(scratch.data_ptr()), _stream(stream))
    _check(code, "pctc_discarded_mass")
    return delta[:len(b), :N]


def head_bwd(H: torch.Tensor, W: torch.Tensor, lam: torch.Tensor, G: torch.Tensor, g: torch.Tensor,
             remap: torch.Tensor, chunk: int = 0, want_dH: bool = True, want_dW: bool = True,
             stream=None) -> Dict[str, torch.Tensor]:
    L = lib()
    dt = _dtype_code(H)
    H = H.contiguous()
    W = W.contiguous()
    M, D = int(H.shape[0]), int(H.shape[1])
    V = int(W.shape[0])
    dev = H.device
    G = G.to(torch.float32).contiguous()
    ldG = int(G.shape[1])
    dH = torch.empty((M, D), dtype=torch.float32, device=dev) if want_dH else None
    dW = torch.empty((V, D), dtype=torch.float32, device=dev) if want_dW else None
    scratch = _workspace(int(L.pctc_bwd_scratch_bytes(dt, M, D, V, ldG, int(chunk))), dev)
    code = L.pctc_head_bwd(dt, _ptr(H), M, D, _ptr(W), V, _ptr(lam.to(torch.float64).contiguous()), _ptr(G), ldG,
                           _ptr(g.to(torch.float32).contiguous()), _ptr(remap.to(torch.int32).contiguous()),
                           int(chunk), _ptr(dH), _ptr(dW), ctypes.c_void_p(scratch.data_ptr()), _stream(stream))
    _check(code, "pctc_head_bwd")
    return {"dH": dH, "dW": dW}


# ---- grouped logits for a stock CTC -------------------------------------------------------

def grouped_logprobs(H: torch.Tensor, W: torch.Tensor, u_ids: torch.Tensor, bias: Optional[torch.Tensor] = None,
                     stream=None) -> Dict[str, torch.Tensor]:
    """log softmax of the grouped logits [M, K + 1] (float32: the K selected classes, then
    the merged "other" class) and the full normaliser lam [M] (float64)."""
    L = lib()
    dt = _dtype_code(H)
    H = H.contiguous()
    W = W.contiguous()
    M, D = int(H.shape[0]), int(H.shape[1])
    V = int(W.shape[0])
    dev = H.device
    u_ids = u_ids.to(device=dev, dtype=torch.int32).contiguous()
    K = int(u_ids.numel())
    if bias is not None:
        bias = _bias_vector(bias, V, dev)
    logp = torch.empty((M, K + 1), dtype=torch.float32, device=dev)
    lam = torch.empty(max(M, 1), dtype=torch.float64, device=dev)
    nbytes = int(L.pctc_grouped_workspace_size(dt, M, D, V, K, 0))
    if nbytes == 0:
        raise PrunedCTCError(-1, "pctc_grouped_workspace_size: invalid arguments")
    ws = _workspace(nbytes, dev)
    code = L.pctc_grouped_logprobs(dt, _ptr(H), M, D, _ptr(W), _ptr(bias), V, _ptr(u_ids), K, _ptr(logp), _ptr(lam),
                                   ctypes.c_void_p(ws.data_ptr()), ctypes.c_size_t(ws.numel()), _stream(stream))
    _check(code, "pctc_grouped_logprobs")
    return {"logp": logp, "lam": lam[:M]}


def grouped_backward(H: torch.Tensor, W: torch.Tensor, u_ids: torch.Tensor, logp: torch.Tensor, lam: torch.Tensor,
                     dlogp: torch.Tensor, bias: Optional[torch.Tensor] = None, chunk: int = 0,
                     want_dH: bool = True, want_dW: bool = True, want_db: bool = False,
                     stream=None) -> Dict[str, Optional[torch.Tensor]]:
    """dH, dW (and db) from the gradient of a loss w.r.t. the exported grouped log-probabilities."""
    L = lib()
    dt = _dtype_code(H)
    H = H.contiguous()
    W = W.contiguous()
    M, D = int(H.shape[0]), int(H.shape[1])
    V = int(W.shape[0])
    dev = H.device
    u_ids = u_ids.to(device=dev, dtype=torch.int32).contiguous()
    K = int(u_ids.numel())
    if tuple(logp.shape) != (M, K + 1) or tuple(dlogp.shape) != (M, K + 1):
        raise PrunedCTCError(-1, f"logp and dlogp must be [{M}, {K + 1}]")
    if bias is not None:
        bias = _bias_vector(bias, V, dev)
    logp = logp.to(torch.float32).contiguous()
    dlogp = dlogp.to(torch.float32).contiguous()
    lam = lam.to(torch.float64).contiguous()
    dH = torch.empty((M, D), dtype=torch.float32, device=dev) if want_dH else None
    dW = torch.empty((V, D), dtype=torch.float32, device=dev) if want_dW else None
    db = torch.empty(V, dtype=torch.float32, device=dev) if want_db else None
    nbytes = int(L.pctc_grouped_workspace_size(dt, M, D, V, K, int(chunk)))
    if nbytes == 0:
        raise PrunedCTCError(-1, "pctc_grouped_workspace_size: invalid arguments")
    ws = _workspace(nbytes, dev)
    code = L.pctc_grouped_backward(dt, _ptr(H), M, D, _ptr(W), _ptr(bias), V, _ptr(u_ids), K, _ptr(logp), _ptr(lam),
                                   _ptr(dlogp), int(chunk), _ptr(dH), _ptr(dW), _ptr(db),
                                   ctypes.c_void_p(ws.data_ptr()), ctypes.c_size_t(ws.numel()), _stream(stream))
    _check(code, "pctc_grouped_backward")
    return {"dH": dH, "dW": dW, "db": db}


class GroupedHead(torch.autograd.Function):
    """Autograd wrapper: grouped log-probabilities [M, K + 1] of the head H W^T (+ b), for a
    stock CTC loss over K + 1 classes.  The backward runs the library's recomputed backward;
    gradients are returned in the dtypes of H, W and b."""

    @staticmethod
    def forward(ctx, H, W, bias, u_ids):
        out = grouped_logprobs(H.detach(), W.detach(), u_ids, None if bias is None else bias.detach())
        ctx.save_for_backward(H, W, bias, u_ids, out["logp"], out["lam"])
        return out["logp"]

    @staticmethod
    def backward(ctx, dlogp):
        H, W, bias, u_ids, logp, lam = ctx.saved_tensors
        need = ctx.needs_input_grad
        r = grouped_backward(H.detach(), W.detach(), u_ids, logp, lam, dlogp,
                             bias=None if bias is None else bias.detach(), want_dH=need[0], want_dW=need[1],
                             want_db=bias is not None and need[2])
        dH = r["dH"].to(H.dtype) if r["dH"] is not None else None
        dW = r["dW"].to(W.dtype) if r["dW"] is not None else None
        db = r["db"].to(bias.dtype) if r["db"] is not None else None
        return dH, dW, db, None


def grouped_head(H: torch.Tensor, W: torch.Tensor, u_ids: torch.Tensor, bias: Optional[torch.Tensor] = None):
    return GroupedHead.apply(H, W, bias, u_ids)


# ---- kernel timing -----------------------------------------------------------------------

def prof_enable(on: bool = True) -> None:
    lib().pctc_prof_enable(1 if on else 0)


def prof_select(name: Optional[str] = None) -> None:
    """Time only the kernels called `name` (None: all of them)."""
    lib().pctc_prof_select(name.encode() if name else None)


def prof_reset() -> None:
    lib().pctc_prof_reset()


def prof_read() -> Dict[str, Dict[str, float]]:
    L = lib()
    out = {}
    for i in range(L.pctc_prof_count()):
        name = ctypes.c_char_p()
        ms = ctypes.c_double()
        n = ctypes.c_int64()
        if L.pctc_prof_get(i, ctypes.byref(name), ctypes.byref(ms), ctypes.byref(n)):
            out[name.value.decode()] = {"total_ms": ms.value, "launches": int(n.value)}
    return out
