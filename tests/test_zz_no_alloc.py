"""ispa_attn_chunk_noalloc (the variant whose split partials live in the
library's fixed per-GPU device scratch) against ispa_attn_chunk_ws with a
caller workspace, called through the C ABI on the same seeded inputs: the
outputs must be bitwise equal, over consecutive calls that reuse the scratch
with a smaller problem second."""

import ctypes

import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2607_00712_amd as ispa
from parity_util import assert_attn, assert_lse, f64

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _nan_outputs(n_q, hidden, heads, dual):
    mk = lambda *s: torch.full(s, float("nan"), dtype=torch.float32, device=DEV)
    outs = [mk(n_q, hidden), mk(heads, n_q)]
    if dual:
        outs += [mk(n_q, hidden), mk(heads, n_q)]
    return outs


def _call_noalloc(q, k, v, N, w, sink, heads, outs):
    """Raw C-ABI call; returns the status."""
    L = ispa.lib()
    n_q, hidden = q.shape
    p = lambda t: ctypes.c_void_p(t.data_ptr() if t is not None else 0)
    dual = len(outs) == 4
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return L.ispa_attn_chunk_noalloc(p(q), p(k), p(v), N, w, sink, n_q, heads, hidden // heads, 0.0,
                                     p(outs[0]), p(outs[1]), p(outs[2] if dual else None),
                                     p(outs[3] if dual else None), stream)


def _check_case(wid, n_q, N, w, sink, heads, hd, dual, expect_split, oracle_rows=None):
    print(f"[noalloc] wid={wid} n_q={n_q} N={N} w={w} s={sink} H={heads} d={hd} dual={dual}", flush=True)
    L = ispa.lib()
    need = L.ispa_attn_workspace_bytes(N, w, sink, n_q, heads, hd, int(dual), 0)
    assert (need > 0) == expect_split, need
    assert need <= ispa.ISPA_STATIC_SCRATCH_BYTES
    q, k, v = synth.chunk_qkv(wid, 0, 0, n_q, N, heads * hd, DEV)
    outs = _nan_outputs(n_q, heads * hd, heads, dual)
    assert _call_noalloc(q, k, v, N, w, sink, heads, outs) == ispa.ISPA_OK
    torch.cuda.synchronize()
    ref = _nan_outputs(n_q, heads * hd, heads, dual)
    ispa.attn_chunk(q, k, v, N, w, heads, sink_len=sink, dual=dual, out=ref[0], lse=ref[1],
                    out_local=ref[2] if dual else None, lse_local=ref[3] if dual else None, segments=0)
    torch.cuda.synchronize()
    for name, a, b in zip(("out", "lse", "out_local", "lse_local"), outs, ref):
        assert not torch.isnan(a).any(), f"{name}: unwritten output"
        assert torch.equal(a, b), f"{name}: noalloc and workspace outputs differ"
    if oracle_rows is not None:
        sel = np.asarray(oracle_rows)
        r = oracle.chunk_attention(f64(q), f64(k[:N]), f64(v[:N]), N, w, heads, sink_len=sink,
                                   branches=("full", "local") if dual else ("local",), query_rows=sel)
        first = "full" if dual else "local"
        assert_attn(f64(outs[0])[sel], r[first][0], first)
        assert_lse(f64(outs[1])[:, sel], r[first][1], first + " lse")
        if dual:
            assert_attn(f64(outs[2])[sel], r["local"][0], "local")
            assert_lse(f64(outs[3])[:, sel], r["local"][1], "local lse")


def test_noalloc_two_calls_second_smaller():
    # a 1.3B-shaped dual-stream chunk with 10 heads x 128 (4680 queries, 7
    # chunks of cache, window of 2 chunks): 190 work items, split over the
    # chip, 129 MiB of partials
    _check_case(10, 4680, 32760, 9360, 0, 10, 128, True, True)
    # then a smaller split problem on the same scratch (head_dim 64, sink):
    # stale partials of the first call must not leak into it
    _check_case(12, 1000, 32760, 9360, 4680, 4, 64, True, True, oracle_rows=[0, 255, 256, 511, 999])


def test_noalloc_single_stream_and_unsplit():
    # single-stream split, then a problem too small to split (no scratch use)
    _check_case(13, 700, 30000, 26000, 64, 3, 128, False, True)
    _check_case(1, 64, 256, 64, 64, 2, 64, True, False, oracle_rows=[0, 31, 63])


def test_noalloc_rejects_plans_beyond_scratch():
    # 14 heads x 128 at 4680 queries: 266 work items, a split of three pieces
    # per segment needs 192 MiB of partials; nothing is enqueued
    n_q, N, w, heads, hd = 4680, 24576, 9360, 14, 128
    L = ispa.lib()
    need = L.ispa_attn_workspace_bytes(N, w, 0, n_q, heads, hd, 1, 0)
    print(f"[noalloc] over-limit plan needs {need} bytes", flush=True)
    assert need > ispa.ISPA_STATIC_SCRATCH_BYTES
    q, k, v = synth.chunk_qkv(14, 0, 0, n_q, N, heads * hd, DEV)
    outs = _nan_outputs(n_q, heads * hd, heads, True)
    assert _call_noalloc(q, k, v, N, w, 0, heads, outs) == ispa.ISPA_ERR_SCRATCH
    torch.cuda.synchronize()
    assert all(torch.isnan(t).all() for t in outs)
    assert "scratch" in ispa.status_string(ispa.ISPA_ERR_SCRATCH)
    with pytest.raises(ispa.IspaError) as e:
        ispa.attn_chunk_noalloc(q, k, v, N, w, heads, out=outs[0], lse=outs[1], out_local=outs[2],
                                lse_local=outs[3])
    assert e.value.status == ispa.ISPA_ERR_SCRATCH
