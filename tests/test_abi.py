"""The C ABI without a GPU: the library loads, exports every symbol the header
declares, and rejects bad arguments before touching the device."""

import ctypes
import os
import re

import pytest

import paper_2607_00712_amd as ispa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ispa.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ispa_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(ispa.LIB_PATH):
        pytest.fail("libispa.so missing: build it with python -m paper_2607_00712_amd.build first")
    return ispa.lib()


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) >= 10, names
    for n in names:
        assert hasattr(L, n), f"{n} declared in include/ispa.h but not exported"
    assert set(names) == set(ispa._SIGNATURES), "binding signatures and header disagree"


def test_status_strings(L):
    for code in (0, -1, -2, -3, -4, -5, -6):
        assert ispa.status_string(code).startswith("ISPA")
    assert "unknown" in ispa.status_string(7)
    assert L.ispa_abi_version() == 104


def _attn(L, **kw):
    args = dict(q=16, k=32, v=48, cache_len=256, window=64, sink=0, n_q=64, heads=2, hd=64, scale=0.0,
                out=64, lse=128, out_local=0, lse_local=0)
    args.update(kw)
    p = lambda v: ctypes.c_void_p(v) if v else ctypes.c_void_p(0)
    # pointers are fake (never dereferenced): validation must fail first
    return L.ispa_attn_chunk(p(args["q"]), p(args["k"]), p(args["v"]), args["cache_len"], args["window"],
                             args["sink"], args["n_q"], args["heads"], args["hd"], args["scale"], p(args["out"]),
                             p(args["lse"]), p(args["out_local"]), p(args["lse_local"]), p(0))


def test_attention_argument_errors(L):
    E, U = ispa.ISPA_ERR_INVALID_ARG, ispa.ISPA_ERR_UNSUPPORTED
    assert _attn(L, hd=96) == U
    assert _attn(L, hd=32) == U
    assert _attn(L, q=0) == E
    assert _attn(L, out=0) == E
    assert _attn(L, k=33) == E                 # misaligned
    assert _attn(L, out_local=72) == E         # misaligned
    assert _attn(L, lse=130) == E              # misaligned float
    assert _attn(L, lse_local=256) == E        # lse_local without out_local
    assert _attn(L, window=0) == E
    assert _attn(L, sink=-1) == E
    assert _attn(L, cache_len=63) == E         # fewer keys than queries
    assert _attn(L, n_q=0, cache_len=0) == E
    assert _attn(L, heads=0) == E
    assert _attn(L, scale=float("nan")) == E
    assert _attn(L, scale=float("inf")) == E


def test_noalloc_argument_errors(L):
    # invalid arguments are rejected before the scratch is looked up
    E, U = ispa.ISPA_ERR_INVALID_ARG, ispa.ISPA_ERR_UNSUPPORTED
    p = ctypes.c_void_p
    call = lambda hd=64, k=32, out=64, window=64: L.ispa_attn_chunk_noalloc(
        p(16), p(k), p(48), 256, window, 0, 64, 2, hd, 0.0, p(out), p(128), p(0), p(0), p(0))
    assert call(hd=96) == U
    assert call(k=33) == E
    assert call(out=0) == E
    assert call(window=0) == E
    hdr = open(HEADER).read()
    m = re.search(r"#define ISPA_STATIC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", hdr)
    assert m and int(m.group(1)) << int(m.group(2)) == ispa.ISPA_STATIC_SCRATCH_BYTES


def test_workspace_sizes(L):
    assert L.ispa_stats_workspace_bytes(0, 8, 1) == 0
    assert L.ispa_stats_workspace_bytes(12, 8, 1) == 0      # not a multiple of 8
    assert L.ispa_stats_workspace_bytes(8, 8, 0) == 0
    assert L.ispa_stats_workspace_bytes(16392, 8, 1) == 0
    d, m = 1536, 4680
    b = L.ispa_stats_workspace_bytes(d, d, m)
    # G, C, L in fp32 plus bf16 X and R staging, each 256-byte aligned
    assert b >= 3 * d * d * 4 + 2 * m * d * 2
    assert b % 256 == 0


def test_stats_handle_errors(L):
    h = ctypes.c_void_p(0)
    assert L.ispa_stats_create(None, ctypes.c_void_p(256), 1 << 20, 8, 8, 1, None) == ispa.ISPA_ERR_INVALID_ARG
    assert L.ispa_stats_create(ctypes.byref(h), ctypes.c_void_p(0), 1 << 20, 8, 8, 1, None) == ispa.ISPA_ERR_INVALID_ARG
    assert L.ispa_stats_create(ctypes.byref(h), ctypes.c_void_p(128), 1 << 20, 8, 8, 1, None) == ispa.ISPA_ERR_INVALID_ARG
    assert L.ispa_stats_create(ctypes.byref(h), ctypes.c_void_p(256), 16, 8, 8, 1, None) == ispa.ISPA_ERR_STATE
    assert not h.value
    assert L.ispa_stats_reset(None) == ispa.ISPA_ERR_STATE
    assert L.ispa_stats_destroy(None) == ispa.ISPA_ERR_STATE
    assert L.ispa_accum_stats(None, None, 0, None, None, 0, 1) == ispa.ISPA_ERR_STATE
    assert L.ispa_solve_modulation(None, ctypes.c_float(1e-3), None, None) == ispa.ISPA_ERR_STATE
    assert L.ispa_stats_views(None, None, None, None, None) == ispa.ISPA_ERR_STATE


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(ispa, "_lib", None)
    monkeypatch.setattr(ispa, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        ispa.lib()


def test_product_never_imports_oracle():
    pkg = os.path.join(ROOT, "paper_2607_00712_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".cpp", ".hip", ".h")):
                src = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in src.replace("the oracle", ""), f"{f} mentions the oracle"


def test_select_layers_against_oracle(L):
    # host-only entry point: compared with the oracle's stable ranking
    import numpy as np
    import oracle
    rng = np.random.default_rng(7)
    for n in (1, 5, 30, 40):
        eps = rng.integers(0, 6, size=n).astype(np.float64) * 0.25   # many ties
        for k in (0, 1, n // 2, n):
            assert ispa.select_layers(eps, k) == list(oracle.select_layers(eps, k))
    # NaN sorts after every number
    assert ispa.select_layers([float("nan"), 2.0, -1.0, float("inf")], 4) == [2, 1, 3, 0]
    E = ispa.ISPA_ERR_INVALID_ARG
    arr = (ctypes.c_double * 3)(1.0, 2.0, 3.0)
    out = (ctypes.c_int32 * 4)()
    assert L.ispa_select_layers(arr, 3, 4, out) == E
    assert L.ispa_select_layers(arr, 3, -1, out) == E
    assert L.ispa_select_layers(None, 3, 1, out) == E


def test_absorption_argument_errors(L):
    E, U = ispa.ISPA_ERR_INVALID_ARG, ispa.ISPA_ERR_UNSUPPORTED
    p = lambda v: ctypes.c_void_p(v)
    assert L.ispa_inject_modulation(p(256), 7, 0, p(4096), 4, 4, p(0)) == U
    assert L.ispa_inject_modulation(p(0), 0, 0, p(4096), 4, 4, p(0)) == E
    assert L.ispa_inject_modulation(p(256), 0, 0, p(4096), 0, 4, p(0)) == E
    assert L.ispa_inject_modulation(p(4096), 0, 0, p(4096), 4, 4, p(0)) == E      # overlap
    assert L.ispa_kv_evict(p(16), p(32), 10, 3, 0, 12, p(64), p(128), None, p(0)) == E   # hidden % 8
    assert L.ispa_kv_evict(p(16), p(32), 0, 3, 0, 16, p(64), p(128), None, p(0)) == E
    assert L.ispa_kv_evict(p(16), p(32), 10, 3, 0, 16, p(16), p(128), None, p(0)) == E  # ring == cache
    assert L.ispa_kv_ring_append(p(16), p(32), 0, 0, 0, p(64), p(128), 4, 16, p(0)) == E  # window 0
    assert L.ispa_kv_ring_append(p(16), p(32), 0, 4, -1, p(64), p(128), 4, 16, p(0)) == E
    # projection and its W8A8 form: the host checks reject before any launch
    assert L.ispa_project(p(256), p(512), 4, 48, 8, p(4096), 0, p(0)) == E             # d_in % 32
    assert L.ispa_project(p(256), p(512), 4, 32, 8, p(4096), 5, p(0)) == U
    assert L.ispa_project(p(256), p(512), 4, 32, 8, p(256), 1, p(0)) == E              # y overlaps a
    assert L.ispa_quantize_rows(p(256), 3, 4, 16, p(4096), p(8192), p(0)) == U
    assert L.ispa_quantize_rows(p(256), 0, 4, 12, p(4096), p(8192), p(0)) == E         # cols % 8
    assert L.ispa_quantize_rows(p(264), 0, 4, 16, p(4096), p(8192), p(0)) == E         # x alignment
    assert L.ispa_quantize_rows(p(256), 0, 4, 16, p(264), p(8192), p(0)) == E          # q overlaps x
    assert L.ispa_quantize_rows(p(256), 0, 4, 16, p(4096), p(4100), p(0)) == E         # scale overlaps q
    assert L.ispa_project_w8a8(p(256), p(1024), p(2048), p(3072), 4, 96, 8, p(8192), 1, p(0)) == E  # d_in % 64
    assert L.ispa_project_w8a8(p(256), p(1024), p(2048), p(3072), 4, 64, 8, p(8192), 2, p(0)) == U
    assert L.ispa_project_w8a8(p(256), p(1024), p(2048), p(3072), 4, 64, 8, p(2048), 1, p(0)) == E  # y over q_w
    assert L.ispa_project_w8a8(p(256), p(1024), p(2048), p(3072), 0, 64, 8, p(8192), 1, p(0)) == E  # no rows
    assert L.ispa_project_w8a8(p(256), p(1024), p(2048), p(3072), 4, 65600, 8, p(1 << 40), 1, p(0)) == E


def test_async_solve_argument_errors(L):
    # checked before anything is enqueued (no handle: state error; bad pointers)
    p = lambda v: ctypes.c_void_p(v)
    assert L.ispa_solve_modulation_async(None, 1e-3, p(256), None, None) == ispa.ISPA_ERR_STATE


def test_batch_solve_argument_errors(L):
    # checked before anything is enqueued: no handle array, a count out of range,
    # a null handle in the array
    p = lambda v: ctypes.c_void_p(v)
    hs = (ctypes.c_void_p * 2)(None, None)
    assert L.ispa_solve_modulation_batch(None, 1, 1e-3, p(256), None, None) == ispa.ISPA_ERR_INVALID_ARG
    assert L.ispa_solve_modulation_batch(hs, 0, 1e-3, p(256), None, None) == ispa.ISPA_ERR_INVALID_ARG
    assert L.ispa_solve_modulation_batch(hs, 4097, 1e-3, p(256), None, None) == ispa.ISPA_ERR_INVALID_ARG
    assert L.ispa_solve_modulation_batch(hs, 2, 1e-3, p(256), None, None) == ispa.ISPA_ERR_STATE
