"""The C-ABI library loads on the CPU and exports every function the headers declare."""
import ctypes
import os
import re

import pytest


def declared_functions(repo_root):
    names = set()
    for h in ("metro.h", "metro_ops.h", "metro_sched.h"):
        text = open(os.path.join(repo_root, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(metro_[a-z_0-9]+)\s*\(", text))
    return sorted(names)


def test_headers_declare_the_entry_points(repo_root):
    names = declared_functions(repo_root)
    for must in ("metro_create_model", "metro_prefill_chunk", "metro_decode_step", "metro_seq_fork",
                 "metro_op_gemm", "metro_sched_next", "metro_sched_ack"):
        assert must in names


def test_library_exports_every_declared_symbol(repo_root):
    path = os.path.join(repo_root, "paper_2411_03519_amd", "libmetro.so")
    if not os.path.exists(path):
        pytest.skip("libmetro.so not built (run __graft_entry__.build())")
    lib = ctypes.CDLL(path)
    missing = [n for n in declared_functions(repo_root) if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_reports_abi_and_errors_without_gpu(repo_root):
    path = os.path.join(repo_root, "paper_2411_03519_amd", "libmetro.so")
    if not os.path.exists(path):
        pytest.skip("libmetro.so not built")
    from paper_2411_03519_amd import metro
    assert metro.lib.metro_abi_version() == metro.ABI_VERSION == 2
    assert metro.lib.metro_status_name(-3) == b"METRO_E_NOPAGES"
    # configuration errors are found before any HIP call
    bad = metro.Config(n_layers=2, d_model=200, n_heads=4, n_kv_heads=2, head_dim=64, ffn_dim=688, vocab=4096,
                       rope_base=1e4, rms_eps=1e-5, page_size=16, max_batch=4, max_tokens=64, max_context=64,
                       max_seqs=4, kv_pool_bytes=0)
    h = ctypes.c_void_p()
    assert metro.lib.metro_create_model(ctypes.byref(bad), 0, ctypes.byref(h)) == -1
    assert b"d_model" in metro.lib.metro_last_error()
    assert metro.lib.metro_seq_open(None, ctypes.byref(ctypes.c_int64())) == -1


# Llama-3-8B (d 4096, QKV 6144, gate/up 2 x 14336, down K 14336) and 70B (d 8192,
# gate/up 2 x 28672) products; compute units counted as 256 (no device here).
PLAN_CASES = [
    # M, N, Kp, epilogue, workspace -> kind, k slices, tail split
    (25, 6144, 4096, 0, True, "decode", 2, 1),          # decode QKV: too few blocks, K split
    (25, 28672, 4096, 2, True, "decode", 1, 1),         # SwiGLU never splits K
    (64, 4096, 14336, 1, False, "decode", 1, 1),        # no workspace, no split
    (65, 4096, 4096, 1, False, "tile128x128", 1, 1),    # past 64 rows: tiled
    (1000, 6144, 4096, 0, False, "tile128x128", 1, 1),  # narrow up to 1000 rows
    (1001, 6144, 4096, 0, False, "tile256x256", 1, 1),
    (128, 28672, 4096, 2, True, "tile128x128", 1, 1),   # wide, 224 tiles <= CUs
    (192, 28672, 4096, 2, True, "tile256x128", 1, 1),   # 448 128 x 128 tiles > CUs, 224 256 x 128
    (128, 57344, 8192, 2, True, "tile256x128", 1, 1),   # 70B gate/up: 448 128-wide tiles > CUs
    (200, 28672, 4096, 2, True, "tile256x128", 1, 1),   # 224 256 x 128 tiles <= CUs
    (300, 28672, 4096, 2, True, "tile256x256", 1, 1),
    (80, 4096, 4096, 1, True, "tile128x128", 8, 1),    # 32 tiles x 8 slices: one round of 256 CUs
    (80, 6144, 4096, 0, True, "tile128x128", 4, 1),    # 48 tiles: 8 slices would need two rounds
    (200, 4096, 4096, 1, True, "tile128x128", 4, 1),   # 64 tiles x 4; 4 * 4 * 200 <= 4096
    (256, 4096, 4096, 1, True, "tile128x128", 4, 1),
    (300, 4096, 4096, 1, True, "tile128x128", 2, 1),   # 96 tiles: 4 slices would need two rounds
    (200, 4096, 14336, 1, True, "tile128x128", 4, 1),  # 8B down
    (128, 8192, 28672, 1, True, "tile128x128", 4, 1),  # 70B down
    (128, 10240, 8192, 0, True, "tile256x128", 4, 1),  # 70B QKV: 80 x 2 of 128 x 128 -> 40 x 4 of 256 x 128
    (200, 10240, 8192, 0, True, "tile128x128", 1, 1),  # past 128 rows narrow products keep 128 x 128 tiles
    (600, 4096, 14336, 1, True, "tile128x128", 1, 1),  # 8B down at an agent-trace batch
    (5376, 4096, 14336, 1, True, "tile256x256", 1, 2),  # 336 tiles: last 80 cut in 2 k slices
    (5376, 4096, 14336, 1, False, "tile256x256", 1, 1),
    (12800, 28672, 4096, 2, True, "tile256x256", 1, 1), # last round 224 of 256 CUs: no split
]


@pytest.mark.parametrize("M,N,Kp,epi,ws,kind,ks,tail", PLAN_CASES)
def test_gemm_plan_rules(repo_root, M, N, Kp, epi, ws, kind, ks, tail):
    if not os.path.exists(os.path.join(repo_root, "paper_2411_03519_amd", "libmetro.so")):
        pytest.skip("libmetro.so not built")
    from paper_2411_03519_amd import metro
    got = metro.op_gemm_plan(M, N, Kp, epi, ws)
    assert got[0] == kind
    if kind == "decode" and ks > 1:
        assert got[1] > 1  # the exact slice count follows the block count
    else:
        assert got[1] == ks
    assert got[2] == tail


def test_gemm_plan_rejects_bad_shapes(repo_root):
    if not os.path.exists(os.path.join(repo_root, "paper_2411_03519_amd", "libmetro.so")):
        pytest.skip("libmetro.so not built")
    from paper_2411_03519_amd import metro
    for args in ((0, 4096, 4096, 0), (64, 4016, 4096, 0), (64, 4096, 4000, 0), (64, 4096, 4096, 7)):
        with pytest.raises(metro.MetroError):
            metro.op_gemm_plan(*args)


def test_gemm_rejects_misaligned_operands_before_any_launch(repo_root):
    """Alignment and stride are checked on the host (E_INVAL) before any device
    work, so this runs without a GPU: the pointers are never dereferenced."""
    if not os.path.exists(os.path.join(repo_root, "paper_2411_03519_amd", "libmetro.so")):
        pytest.skip("libmetro.so not built")
    from paper_2411_03519_amd import metro
    lib = metro.lib
    P = ctypes.c_void_p
    base = 1 << 20  # stand-in device addresses, 16-byte aligned
    cases = [(base + 2, 4096, base, base), (base, 4100, base, base), (base, 4096, base + 8, base),
             (base, 4096, base, base + 4)]
    for X, ldx, W, out in cases:
        st = lib.metro_op_gemm(P(X), ldx, P(W), 4096, 64, 4096, 0, P(out), None, 4096, None, None)
        assert st == -1, (X, ldx, W, out)
        assert b"aligned" in lib.metro_last_error()


def test_rmsnorm_and_attention_reject_misaligned_buffers(repo_root):
    if not os.path.exists(os.path.join(repo_root, "paper_2411_03519_amd", "libmetro.so")):
        pytest.skip("libmetro.so not built")
    from paper_2411_03519_amd import metro
    lib = metro.lib
    P = ctypes.c_void_p
    base = 1 << 20
    assert lib.metro_op_rmsnorm(P(base + 8), P(base), ctypes.c_float(1e-5), P(base), 4, 256, None) == -1
    assert b"aligned" in lib.metro_last_error()
    ctx = (ctypes.c_int32 * 1)(16)
    bt = (ctypes.c_int32 * 1)(0)
    for q, kv, out in ((base + 8, base, base), (base, base + 4, base), (base, base, base + 2)):
        assert lib.metro_op_attn_decode(P(q), P(kv), 1, 4, 2, 64, 1, ctx, bt, P(out), None) == -1
        assert b"aligned" in lib.metro_last_error()
