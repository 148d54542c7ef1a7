"""GPU parity of ispa_attn_chunk against the oracle on identical seeded bf16
inputs (through the C ABI via the ctypes binding)."""

import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2607_00712_amd as ispa
from parity_util import assert_attn, assert_lse, f64

pytestmark = pytest.mark.gpu

DEV = "cuda"


def run_and_check(n_q, cache_len, window, sink, heads, hd, dual, wid, capacity=None, q_scale=1.0,
                  rows=None, segments=0):
    print(f"[attn] n_q={n_q} N={cache_len} w={window} s={sink} H={heads} d={hd} dual={dual} "
          f"wid={wid} segments={segments}", flush=True)
    q, k, v = synth.chunk_qkv(wid, 0, 0, n_q, cache_len, heads * hd, DEV, q_scale=q_scale,
                              capacity=capacity)
    res = ispa.attn_chunk(q, k, v, cache_len, window, heads, sink_len=sink, dual=dual, segments=segments)
    torch.cuda.synchronize()
    if rows is None:
        qn, sel = f64(q), None
    else:
        sel = np.asarray(rows)
        qn = f64(q)
    ref = oracle.chunk_attention(qn, f64(k[:cache_len]), f64(v[:cache_len]), cache_len, window, heads,
                                 sink_len=sink, branches=("full", "local") if dual else ("local",),
                                 query_rows=sel)
    pick = (lambda t: f64(t)) if sel is None else (lambda t: f64(t)[sel])
    pick_lse = (lambda t: f64(t)) if sel is None else (lambda t: f64(t)[:, sel])
    errs = {}
    if dual:
        out, lse, out_l, lse_l = res
        errs["full"] = assert_attn(pick(out), ref["full"][0], "full")
        assert_lse(pick_lse(lse), ref["full"][1], "full lse")
        errs["local"] = assert_attn(pick(out_l), ref["local"][0], "local")
        assert_lse(pick_lse(lse_l), ref["local"][1], "local lse")
    else:
        out, lse = res
        errs["local"] = assert_attn(pick(out), ref["local"][0], "single")
        assert_lse(pick_lse(lse), ref["local"][1], "single lse")
    return res, errs


# the tiny single-layer workload: 2 heads x 64, chunk of 64 queries, 4 chunks of cache,
# window of one chunk, with and without a one-chunk sink
@pytest.mark.parametrize("sink", [0, 64])
@pytest.mark.parametrize("dual", [False, True])
def test_tiny_layer(sink, dual):
    run_and_check(64, 256, 64, sink, 2, 64, dual, wid=1)


@pytest.mark.parametrize("case", [
    # n_q, N, w, s, H, d, dual
    (100, 333, 97, 13, 3, 128, True),     # ragged everywhere
    (300, 1000, 200, 0, 2, 128, True),    # several query and key tiles
    (129, 129, 64, 0, 1, 128, True),      # N == n_q, one query past a tile
    (64, 640, 1, 0, 2, 64, True),         # single visible key
    (64, 640, 64, 700, 2, 64, True),      # sink covers the cache
    (40, 4000, 130, 1, 4, 64, True),      # one sink key, long history
    (257, 1500, 1500, 0, 2, 128, False),  # F-Layer: window = cache
    (96, 700, 5000, 0, 2, 128, True),     # window beyond the cache: hist empty
    (33, 200, 70, 70, 1, 64, False),      # L-Layer with sink, single stream
])
def test_ragged_and_degenerate(case):
    n_q, N, w, s, H, d, dual = case
    res, _ = run_and_check(n_q, N, w, s, H, d, dual, wid=2)
    if dual and (N <= w + min(s, N)):
        out, lse, out_l, lse_l = res
        # no history: the two streams are the same numbers
        assert torch.equal(out, out_l) and torch.equal(lse, lse_l)


def test_rows_beyond_cache_len_are_not_read():
    # rows past cache_len hold 1e4 values; any read would wreck parity
    run_and_check(128, 777, 256, 64, 2, 128, True, wid=3, capacity=1024)


def test_sharp_softmax():
    run_and_check(128, 1024, 300, 0, 2, 128, True, wid=4, q_scale=4.0)


def test_without_lse_outputs():
    q, k, v = synth.chunk_qkv(5, 0, 0, 64, 300, 256, DEV)
    out, lse = ispa.attn_chunk(q, k, v, 300, 100, 2, need_lse=False)
    assert lse is None
    out2, _ = ispa.attn_chunk(q, k, v, 300, 100, 2)
    torch.cuda.synchronize()
    assert torch.equal(out, out2)


@pytest.mark.parametrize("shape", [(64, 300, 100, 0), (200, 900, 300, 10), (700, 1100, 400, 0)])
def test_deterministic(shape):
    # repeated launches are bit-identical (the two waves sharing a SIMD make
    # any missing wait on an MFMA result show up as run-to-run differences)
    n_q, N, w, s = shape
    q, k, v = synth.chunk_qkv(6, 0, 0, n_q, N, 256, DEV)
    first = ispa.attn_chunk(q, k, v, N, w, 2, sink_len=s, dual=True)
    for i in range(8):
        again = ispa.attn_chunk(q, k, v, N, w, 2, sink_len=s, dual=True, need_lse=(i % 2 == 0))
        torch.cuda.synchronize()
        for x, y in zip(first, again):
            if y is not None:
                assert torch.equal(x, y), f"launch {i + 1} differs"


# the work split over the chip: runs of (work item, key tile) units that end
# inside a work item leave partial results merged with Eq. 11-12
@pytest.mark.parametrize("case", [
    # n_q, N, w, s, H, d, dual, segments
    (300, 1000, 200, 0, 2, 128, True, 3),      # pieces across items and the local boundary
    (100, 333, 97, 13, 3, 128, True, 5),       # sink + window + history, ragged
    (257, 1500, 1500, 0, 2, 128, False, 7),    # F-Layer, single stream
    (600, 3000, 1000, 64, 2, 64, True, 11),    # d = 64
    (64, 640, 64, 0, 2, 64, True, 20),         # one tile per run
    (520, 2000, 300, 1, 1, 128, True, 2),      # fewer runs than work items
    (300, 4000, 500, 3, 2, 128, True, 64),     # ~16 pieces per item, merged four at a time
])
def test_split_parity(case):
    n_q, N, w, s, H, d, dual, seg = case
    run_and_check(n_q, N, w, s, H, d, dual, wid=12, segments=seg)


@pytest.mark.parametrize("merge_kernel", ["0", "1"])
def test_split_completion_paths(merge_kernel, monkeypatch):
    # head_dim 128 completes split work items inside the attention kernel (the
    # last piece of an item merges, its own part from registers when the item
    # has two pieces); ISPA_ATTN_MERGE_KERNEL=1 leaves them to the merge kernel
    monkeypatch.setenv("ISPA_ATTN_MERGE_KERNEL", merge_kernel)
    run_and_check(300, 1000, 200, 0, 2, 128, True, wid=14, segments=5)     # two and three pieces per item
    run_and_check(700, 2600, 900, 0, 3, 128, True, wid=15, segments=16)   # local set split inside pieces


def test_split_matches_unsplit_and_is_deterministic():
    q, k, v = synth.chunk_qkv(13, 0, 0, 500, 2200, 256, DEV)
    ref = ispa.attn_chunk(q, k, v, 2200, 700, 2, sink_len=5, dual=True, segments=-1)
    a = ispa.attn_chunk(q, k, v, 2200, 700, 2, sink_len=5, dual=True, segments=9)
    b = ispa.attn_chunk(q, k, v, 2200, 700, 2, sink_len=5, dual=True, segments=9)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    # the runs restart the softmax reference, so the bf16 rounding of the
    # weights differs from the unsplit pass: agreement is within the parity
    # tolerances, not bitwise
    for x, y in zip(a[::2], ref[::2]):
        assert_attn(f64(x), f64(y), "split vs unsplit")
    for x, y in zip(a[1::2], ref[1::2]):
        assert_lse(f64(x), f64(y), "split vs unsplit lse")


def test_automatic_split_choice():
    # 12 heads x 19 query blocks = 228 work items fill 89% of 256 compute units:
    # whole items (the launch is power-limited, so the idle units cost little);
    # 10 heads = 190 items fill 74%: split over the chip
    L = ispa.lib()
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    if n_cu == 256:
        assert L.ispa_attn_workspace_bytes(32760, 9360, 0, 4680, 12, 128, 1, 0) == 0
        assert L.ispa_attn_workspace_bytes(32760, 9360, 0, 4680, 10, 128, 1, 0) > 0
    assert L.ispa_attn_workspace_bytes(32760, 9360, 0, 4680, 10, 128, 1, -1) == 0


# the paper's literal decomposable form (Eq. 9-12): local and history branches
# as separate calls, fused by the LSE merge
@pytest.mark.parametrize("case", [(300, 1000, 200, 0, 2, 128), (130, 900, 64, 7, 3, 64), (96, 700, 5000, 0, 2, 128)])
def test_decomposable_branches_and_merge(case):
    n_q, N, w, s, H, d = case
    q, k, v = synth.chunk_qkv(14, 0, 0, n_q, N, H * d, DEV)
    s1, lo = min(s, N), max(N - w, 0)
    o_loc, l_loc = ispa.attn_chunk(q, k, v, N, w, H, sink_len=s)
    hist = [(s1, lo)] if lo > s1 else []
    o_hist, l_hist = ispa.attn_ranges(q, k, v, hist, H)
    o_full, l_full = ispa.attn_merge(o_loc, l_loc, o_hist, l_hist)
    torch.cuda.synchronize()
    ref = oracle.chunk_attention(f64(q), f64(k[:N]), f64(v[:N]), N, w, H, sink_len=s,
                                 branches=("full", "hist"))
    assert_attn(f64(o_full), ref["full"][0], "merged full")
    assert_lse(f64(l_full), ref["full"][1], "merged full lse")
    if hist:
        assert_attn(f64(o_hist), ref["hist"][0], "hist")
        assert_lse(f64(l_hist), ref["hist"][1], "hist lse")
    else:
        assert torch.all(o_hist == 0) and torch.all(torch.isneginf(l_hist))
        assert torch.equal(o_full, o_loc) and torch.equal(l_full, l_loc)


def test_merge_kernel_against_oracle():
    g = torch.Generator().manual_seed(15)
    n_q, H, d = 77, 3, 64
    oa = torch.randn(n_q, H * d, generator=g)
    ob = torch.randn(n_q, H * d, generator=g)
    la = torch.randn(H, n_q, generator=g) * 20
    lb = torch.randn(H, n_q, generator=g) * 20
    la[0, :5] = -float("inf")                 # one branch empty
    lb[1, 3:9] = -float("inf")
    la[2, 10:12] = -float("inf")              # both empty
    lb[2, 10:12] = -float("inf")
    out, lse = ispa.attn_merge(oa.to(DEV), la.to(DEV), ob.to(DEV), lb.to(DEV))
    torch.cuda.synchronize()
    o_ref = np.zeros((n_q, H * d))
    l_ref = np.zeros((H, n_q))
    for h in range(H):
        cols = slice(h * d, (h + 1) * d)
        o_ref[:, cols], l_ref[h] = oracle.lse_merge(f64(oa)[:, cols], f64(la)[h], f64(ob)[:, cols], f64(lb)[h])
    np.testing.assert_allclose(f64(out), o_ref, rtol=2e-6, atol=2e-6)
    fin = np.isfinite(l_ref)
    np.testing.assert_allclose(f64(lse)[fin], l_ref[fin], rtol=0, atol=1e-5)
    assert np.all(np.isneginf(f64(lse)[~fin]))


def test_binding_rejects_bad_tensors():
    q, k, v = synth.chunk_qkv(7, 0, 0, 64, 256, 128, DEV)
    with pytest.raises(TypeError):
        ispa.attn_chunk(q.float(), k, v, 256, 64, 2)
    with pytest.raises(ValueError):
        ispa.attn_chunk(q, k, v, 300, 64, 2)
    with pytest.raises(ispa.IspaError):
        ispa.attn_chunk(q, k, v, 256, 0, 2)


# full-size shapes: sampled query rows checked one by one against the oracle
SAMPLE_ROWS = [0, 1, 31, 32, 127, 128, 129, 1000, 2047, 2048, 4095, 4096, 4600, 4679]
# plus one row inside every 256-query block (each block is one work item, and
# every piece of a split work item covers all of its rows)
BLOCK_ROWS = sorted(set(SAMPLE_ROWS) | {min(4679, 256 * b + (37 * b + 5) % 256) for b in range(19)})


def test_wan13b_chunk_all_rows():
    # 12 heads x 128, chunk of 4680 queries, 7 chunks of cache, window of 2
    # chunks: every query row of every head against the oracle
    run_and_check(4680, 32760, 9360, 0, 12, 128, True, wid=10)


def test_wan13b_chunk_sink_sampled():
    # the same chunk with a one-chunk sink (the paper's local set of Eq. 7)
    run_and_check(4680, 32760, 9360, 4680, 12, 128, True, wid=10, rows=BLOCK_ROWS)


def test_wan13b_chunk_split_sampled():
    # the same chunk split over 256 runs (the automatic choice for fills of the
    # chip below 85%), each work item completed inside the kernel
    run_and_check(4680, 32760, 9360, 0, 12, 128, True, wid=10, rows=BLOCK_ROWS, segments=256)


def test_14b_chunk_sampled_heads():
    # 40 heads x 128, 21 chunks of cache; the oracle checks 4 of the 40 heads
    n_q, N, w, H, d = 4680, 98280, 9360, 40, 128
    print(f"[attn] 14B-shaped n_q={n_q} N={N} w={w}", flush=True)
    q, k, v = synth.chunk_qkv(11, 0, 0, n_q, N, H * d, DEV)
    out, lse, out_l, lse_l = ispa.attn_chunk(q, k, v, N, w, H, dual=True)
    torch.cuda.synchronize()
    for h in (0, 13, 26, 39):
        cols = slice(h * d, (h + 1) * d)
        ref = oracle.chunk_attention(f64(q[:, cols]), f64(k[:, cols]), f64(v[:, cols]), N, w, 1,
                                     branches=("full", "local"), query_rows=BLOCK_ROWS)
        assert_attn(f64(out[:, cols])[BLOCK_ROWS], ref["full"][0], f"head {h} full")
        assert_attn(f64(out_l[:, cols])[BLOCK_ROWS], ref["local"][0], f"head {h} local")
        assert_lse(f64(lse[h])[BLOCK_ROWS], ref["full"][1][0], f"head {h} lse")
        assert_lse(f64(lse_l[h])[BLOCK_ROWS], ref["local"][1][0], f"head {h} local lse")
