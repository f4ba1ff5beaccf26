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
    assert metro.lib.metro_abi_version() == 1
    assert metro.lib.metro_status_name(-3) == b"METRO_E_NOPAGES"
    # configuration errors are found before any HIP call
    bad = metro.Config(n_layers=2, d_model=200, n_heads=4, n_kv_heads=2, head_dim=64, ffn_dim=688, vocab=4096,
                       rope_base=1e4, rms_eps=1e-5, page_size=16, max_batch=4, max_tokens=64, max_context=64,
                       max_seqs=4, kv_pool_bytes=0)
    h = ctypes.c_void_p()
    assert metro.lib.metro_create_model(ctypes.byref(bad), 0, ctypes.byref(h)) == -1
    assert b"d_model" in metro.lib.metro_last_error()
    assert metro.lib.metro_seq_open(None, ctypes.byref(ctypes.c_int64())) == -1
