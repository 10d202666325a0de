"""The C-ABI library loads and exports every function include/prunedctc.h declares
(no compute calls: runs without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "prunedctc.h")
LIB = os.path.join(ROOT, "paper_2609_33645_amd", "libprunedctc.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w\s\*]*?\b([a-z_][a-z0-9_]*)\s*\(", text, flags=re.M)
    return sorted(set(n for n in names if n.startswith(("pctc_", "pruned_ctc"))))


def test_header_declares_entry_points():
    names = declared_functions()
    for must in ["pruned_ctc_fwd_bwd", "pctc_workspace_size", "pctc_union_remap", "pctc_lse_select", "pctc_ctc_dp",
                 "pctc_head_bwd", "pctc_status_string", "pctc_prof_enable"]:
        assert must in names


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_library_exports_every_declared_symbol():
    import torch  # noqa: F401  (binds the library to torch's HIP runtime)
    lib = ctypes.CDLL(LIB)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_host_side_validation_without_gpu():
    """Argument checks and workspace sizing are host code: they run without a device."""
    import numpy as np
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB)
    lib.pctc_workspace_size.restype = ctypes.c_size_t
    i32p = ctypes.POINTER(ctypes.c_int32)
    lib.pctc_workspace_size.argtypes = [ctypes.c_int32, ctypes.c_int32, i32p, i32p, ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_float, ctypes.c_int32]
    T = np.array([300, 200], np.int32)
    U = np.array([50, 40], np.int32)
    p = lambda a: a.ctypes.data_as(i32p)  # noqa: E731
    ws = [lib.pctc_workspace_size(1, 2, p(T), p(U), 512, V, 16.0, 0) for V in (10_000, 100_000, 180_000)]
    assert all(w > 0 for w in ws)
    # only V-entry tables grow with V: the remap (4 bytes per class) and the union's
    # membership bitmap and block counts (1/8 + 1/512 bytes per class), each 256-byte aligned
    assert ws[2] - ws[0] <= (4 + 1 / 8 + 1 / 512) * (180_000 - 10_000) + 3 * 256
    assert lib.pctc_workspace_size(1, 2, p(T), p(U), 500, 1000, 16.0, 0) == 0      # D % 8 != 0
    assert lib.pctc_workspace_size(1, 2, p(T), p(U), 1 << 20, 1000, 16.0, 0) > 0   # D = PCTC_MAX_DIM
    assert lib.pctc_workspace_size(1, 2, p(T), p(U), (1 << 20) + 8, 1000, 16.0, 0) == 0  # D too wide
    assert lib.pctc_workspace_size(1, 2, p(T), p(U), 512, 1000, float("nan"), 0) == 0
    U2 = np.array([50, 2000], np.int32)
    assert lib.pctc_workspace_size(1, 2, p(T), p(U2), 512, 1000, 16.0, 0) == 0   # target too long
    lib.pctc_status_string.restype = ctypes.c_char_p
    assert lib.pctc_status_string(-2).decode().startswith("target label")


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_host_side_sizing_rules():
    """Scratch sizes of the stage entry points and the backward's chunk choice (host code)."""
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB)
    sz, i32 = ctypes.c_size_t, ctypes.c_int32
    lib.pctc_lse_scratch_bytes.restype = sz
    lib.pctc_lse_scratch_bytes.argtypes = [i32, i32]
    lib.pctc_greedy_workspace_size.restype = sz
    lib.pctc_greedy_workspace_size.argtypes = [i32, i32, i32]
    lib.pctc_bwd_chunk.restype = i32
    lib.pctc_bwd_chunk.argtypes = [i32, i32, i32, i32, i32]
    lib.pctc_bwd_scratch_bytes.restype = sz
    lib.pctc_bwd_scratch_bytes.argtypes = [i32, i32, i32, i32, i32, i32]
    up = lambda x: (x + 255) // 256 * 256  # noqa: E731
    # normaliser scratch: 8-byte (max, sum) pairs for 256 vocabulary partitions per frame, 1024
    # for D >= 2048, then lambda's hi/lo pair per frame; no V argument at all
    for M in (1, 4215, 11458):
        assert lib.pctc_lse_scratch_bytes(M, 512) == up(256 * M * 8) + up(M * 8)
        assert lib.pctc_lse_scratch_bytes(M, 2048) == up(1024 * M * 8) + up(M * 8)
    assert lib.pctc_lse_scratch_bytes(-1, 512) == 0 and lib.pctc_lse_scratch_bytes(10, 0) == 0
    assert lib.pctc_greedy_workspace_size(16, 4215, 4096) > lib.pctc_greedy_workspace_size(16, 4215, 512) > 0
    assert lib.pctc_greedy_workspace_size(16, 4215, 0) == 0
    # default chunk: the fewest equal chunks (multiples of 256) whose bf16 gradient fits ~512 MiB;
    # narrow bf16 heads (D < 2048) round to whole normaliser partitions (2048 columns), so that
    # the normaliser can write the first chunk's gradient rows
    for M, V in ((4215, 180_000), (2567, 151_936), (11458, 151_936), (16000, 180_000), (64, 1000)):
        for D, align in ((512, 2048), (4096, 256)):
            c = lib.pctc_bwd_chunk(1, M, D, V, 0)
            assert c > 0 and c % align == 0
            cap = min(65536, (512 * 2**20 // (2 * M)) // 256 * 256)
            assert c <= cap
            n = -(-V // c)
            assert c - -(-V // n) < align or n == 1   # equal chunks, rounded up to whole tiles/partitions
        c = lib.pctc_bwd_chunk(0, M, 512, V, 0)     # fp32: whole tiles
        assert c % 256 == 0 and c - -(-V // -(-V // c)) < 256
    assert lib.pctc_bwd_chunk(1, 4215, 512, 180_000, 0) == 61440
    assert lib.pctc_bwd_chunk(1, 2567, 4096, 151_936, 0) == 50688
    assert lib.pctc_bwd_chunk(1, 4215, 512, 180_000, 1024) == 1024
    # an explicit chunk wider than the vocabulary is cut to V rounded up to whole tiles
    assert lib.pctc_bwd_chunk(1, 4215, 512, 1000, 65536) == 1024
    assert lib.pctc_bwd_chunk(0, 4215, 512, 3000, 1 << 20) == 3072
    assert lib.pctc_bwd_chunk(1, 4215, 512, 3072, 3072) == 3072
    # the backward's scratch does not grow with V
    b = [lib.pctc_bwd_scratch_bytes(1, 4215, 512, V, 384, 0) for V in (100_000, 180_000, 400_000)]
    assert b[0] > 0 and b[0] == b[1] == b[2]


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_normaliser_chunk_columns():
    """Host rule for the first backward chunk that the normaliser writes itself (bf16, D a
    multiple of 128, chunk a whole number of normaliser partitions: 2048 columns for D < 2048,
    256 for wider heads, and the selected logits and partial pairs lodged past those rows
    within 64 MiB of extra memory)."""
    import numpy as np
    from paper_2609_33645_amd import prunedctc as pc

    rng = np.random.default_rng(0)
    Tz = rng.integers(150, 376, size=16).astype(np.int32)       # Zipformer-M-like batch
    Tq = rng.integers(500, 751, size=4).astype(np.int32)        # Qwen3-8B-like batch
    Te = np.full(107, 107, np.int32)                            # 107 utterances (LLM memory shape)

    def cols(dtype, T, D, V, chunk=0, want_dW=True, u=6):
        return pc.normaliser_chunk_columns(dtype, T, T // u, D, V, float("inf"), chunk, want_dW)
    assert cols(1, Tz, 512, 180_000) == pc.bwd_chunk(1, int(Tz.sum()), 512, 180_000) == 61440
    assert cols(0, Tz, 512, 180_000) == 0                       # fp32: every chunk recomputed
    assert cols(1, Tz, 512, 180_000, chunk=4096) == 4096 and cols(1, Tz, 512, 180_000, chunk=4352) == 0
    assert cols(1, Tq, 4096, 151_936, u=4) == pc.bwd_chunk(1, int(Tq.sum()), 4096, 151_936) == 50688
    assert cols(1, Te, 4096, 151_936, want_dW=False, u=4) == 0  # off: lodging would add > 64 MiB
    assert cols(1, Tz[:3], 136, 5000) == 0                      # D not a multiple of 128
    assert cols(1, Tz[:3], 128, 5000) == 5000                   # one chunk: the whole vocabulary
    bad = np.array([0], np.int32)
    assert pc.normaliser_chunk_columns(1, bad, bad, 128, 5000, 0.0) == 0   # invalid lengths


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_zero_frame_sizing():
    """Every size query accepts a batch without frames (N = 0 or M = 0) and returns a usable
    size: the bf16 union part once divided by a zero frame-slice length there."""
    import numpy as np
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB)
    sz, i32, f32 = ctypes.c_size_t, ctypes.c_int32, ctypes.c_float
    i32p = ctypes.POINTER(ctypes.c_int32)
    lib.pctc_workspace_size.restype = sz
    lib.pctc_workspace_size.argtypes = [i32, i32, i32p, i32p, i32, i32, f32, i32]
    lib.pctc_dp_scratch_bytes.restype = sz
    lib.pctc_dp_scratch_bytes.argtypes = [i32, i32p, i32p, f32]
    lib.pctc_discarded_mass_scratch_bytes.restype = sz
    lib.pctc_discarded_mass_scratch_bytes.argtypes = [i32, i32p, i32p]
    lib.pctc_lse_scratch_bytes.restype = sz
    lib.pctc_lse_scratch_bytes.argtypes = [i32, i32]
    lib.pctc_greedy_workspace_size.restype = sz
    lib.pctc_greedy_workspace_size.argtypes = [i32, i32, i32]
    lib.pctc_bwd_scratch_bytes.restype = sz
    lib.pctc_bwd_scratch_bytes.argtypes = [i32, i32, i32, i32, i32, i32]
    lib.pctc_grouped_workspace_size.restype = sz
    lib.pctc_grouped_workspace_size.argtypes = [i32, i32, i32, i32, i32, i32]
    T = np.zeros(0, np.int32)
    U = np.zeros(0, np.int32)
    p = lambda a: a.ctypes.data_as(i32p)  # noqa: E731
    for dt in (0, 1):
        for D, V in ((8, 2), (64, 300), (512, 180_000), (4096, 151_936)):
            for beam in (0.0, 16.0, float("inf")):
                assert lib.pctc_workspace_size(dt, 0, p(T), p(U), D, V, beam, 0) > 0, (dt, D, V, beam)
        assert lib.pctc_bwd_scratch_bytes(dt, 0, 512, 180_000, 8, 0) > 0
        assert lib.pctc_grouped_workspace_size(dt, 0, 512, 180_000, 100, 0) > 0
    for beam in (16.0, float("inf")):
        assert lib.pctc_dp_scratch_bytes(0, p(T), p(U), beam) > 0
    assert lib.pctc_discarded_mass_scratch_bytes(0, p(T), p(U)) > 0
    for D in (512, 4096):
        assert lib.pctc_lse_scratch_bytes(0, D) > 0
        assert lib.pctc_greedy_workspace_size(0, 0, D) > 0


@pytest.mark.skipif(not os.path.exists(LIB), reason="library not built")
def test_misaligned_head_pointers_rejected_on_host():
    """H and W are read in 16-byte pieces: a pointer off that alignment is PCTC_EINVAL, returned
    before any device work (the pointers here are never dereferenced)."""
    import numpy as np
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB)
    i32, f32, vp, sz = ctypes.c_int32, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t
    i32p = ctypes.POINTER(ctypes.c_int32)
    lib.pruned_ctc_fwd_bwd.restype = i32
    lib.pruned_ctc_fwd_bwd.argtypes = [i32, vp, i32, vp, i32, vp, i32p, i32p, i32, i32, f32, i32, vp, vp, vp, vp, vp,
                                       vp, sz, vp]
    T = np.array([30, 20], np.int32)
    U = np.array([5, 4], np.int32)
    p = lambda a: a.ctypes.data_as(i32p)  # noqa: E731
    ok, off = 0x7f0000000000, 0x7f0000000008  # aligned and 8-byte-offset stand-ins
    for H, W in ((off, ok), (ok, off)):
        rc = lib.pruned_ctc_fwd_bwd(1, H, 64, W, 100, ok, p(T), p(U), 2, 0, 16.0, 0, ok, None, None, None, None,
                                    ok, 1 << 30, None)
        assert rc == -1, (hex(H), hex(W), rc)
