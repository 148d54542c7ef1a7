"""GPU parity of ispa_accum_stats (discrepancy + Gram) against the oracle."""

import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2607_00712_amd as ispa
from parity_util import assert_gram, f64, lower_sym

pytestmark = pytest.mark.gpu

DEV = "cuda"


def oracle_stats(blocks, d_in, d_out):
    st = oracle.Stats(d_in, d_out)
    rs = []
    for x, yf, yl in blocks:
        # the ABI rounds an fp32 x to bf16 before it enters the statistics
        X = oracle.bf16_round(f64(x).astype(np.float32)) if x.dtype == torch.float32 else f64(x)
        rs.append(st.accumulate(X, f64(yf).astype(np.float32), f64(yl).astype(np.float32)))
    S = sum((r * r).sum(axis=0) for r in rs)
    return st, S


def check(stats, blocks, d_in, d_out):
    torch.cuda.synchronize()
    G, C, s, n = stats.views()
    ref, S = oracle_stats(blocks, d_in, d_out)
    eg, ec = assert_gram(f64(G), f64(C), ref.G, ref.C, S)
    assert n == ref.n
    assert abs(float(s.item()) - ref.s) <= 1e-6 * max(ref.s, 1e-300)
    return eg, ec


def rand_block(wid, i, rows, d_in, d_out, xdt, ydt, x_is_ylocal=False):
    yf = synth.normal((rows, d_out), synth.seed_of(wid, i, synth.Y_FULL), DEV, dtype=ydt)
    yl = synth.normal((rows, d_out), synth.seed_of(wid, i, synth.Y_LOCAL), DEV, dtype=ydt)
    if x_is_ylocal:
        return yl, yf, yl
    x = synth.normal((rows, d_in), synth.seed_of(wid, i, synth.X), DEV, dtype=xdt)
    return x, yf, yl


def test_residual_bits_exact():
    """X = I makes C = R exactly: checks the bf16 rounding of y_full - y_local
    bit for bit (products by 1 and additions of 0 are exact in fp32)."""
    d = 64
    eye = torch.eye(d, dtype=torch.bfloat16, device=DEV)
    base = synth.normal((d, d), synth.seed_of(20, 0, synth.Y_FULL), DEV, dtype=torch.float32)
    # y_local close to y_full so the difference exercises the rounding
    yl = (base + 1e-3 * synth.normal((d, d), synth.seed_of(20, 0, synth.Y_LOCAL), DEV,
                                     dtype=torch.float32)).contiguous()
    st = ispa.Stats(d, d, max_rows=d, device=DEV)
    st.accum(eye, base, yl)
    torch.cuda.synchronize()
    _, C, s, _ = st.views()
    R = oracle.residual(f64(base).astype(np.float32), f64(yl).astype(np.float32))
    assert np.array_equal(f64(C), R)
    assert float(s.item()) == pytest.approx(float((R * R).sum()), rel=1e-6)


@pytest.mark.parametrize("xdt,ydt,alias", [
    (torch.bfloat16, torch.float32, False),
    (torch.float32, torch.float32, False),
    (torch.float32, torch.float32, True),     # x is y_local (the warmup chain)
    (torch.bfloat16, torch.bfloat16, False),
])
def test_dtypes(xdt, ydt, alias):
    d_in = d_out = 128
    blocks = [rand_block(21, i, 64, d_in, d_out, xdt, ydt, alias) for i in range(2)]
    st = ispa.Stats(d_in, d_out, max_rows=64, device=DEV)
    for b in blocks:
        st.accum(*b)
    check(st, blocks, d_in, d_out)


def test_ragged_shapes_and_staging():
    # d not a multiple of the 128 tile, rows not a multiple of 32, rows > max_rows
    d_in, d_out = 72, 40
    blocks = [rand_block(22, i, r, d_in, d_out, torch.bfloat16, torch.float32)
              for i, r in enumerate((333, 1, 95))]
    st = ispa.Stats(d_in, d_out, max_rows=100, device=DEV)
    for b in blocks:
        st.accum(*b)
    check(st, blocks, d_in, d_out)


def test_zero_rows_and_reset():
    d = 64
    st = ispa.Stats(d, d, max_rows=32, device=DEV)
    x, yf, yl = rand_block(23, 0, 50, d, d, torch.bfloat16, torch.float32)
    st.accum(x, yf, yl)
    st.reset()
    st.accum(x[:0], yf[:0], yl[:0])
    torch.cuda.synchronize()
    G, C, s, n = st.views()
    assert n == 0 and not torch.any(G) and not torch.any(C) and float(s.item()) == 0.0
    st.accum(x, yf, yl)
    check(st, [(x, yf, yl)], d, d)


def test_wan13b_warmup_chunk():
    # one warmup chunk of the 1.3B shape: 4680 rows, d = 1536, x = y_local (fp32)
    d = 1536
    print("[stats] 4680 x 1536", flush=True)
    blocks = [rand_block(24, 0, 4680, d, d, torch.float32, torch.float32, True)]
    st = ispa.Stats(d, d, max_rows=4680, device=DEV)
    st.accum(*blocks[0])
    check(st, blocks, d, d)


def test_warmup_bitwise_reproducible():
    """Two identical 4-chunk warmups at the 1.3B width (d = 1536: fewer Gram
    tiles than CUs, so the rows are split and the halves meet in the
    workspace) give bitwise equal G, C, s and, through the solve, dW and eps."""
    d = 1536
    print("[stats] bitwise rerun 4 x 4680 x 1536", flush=True)
    blocks = [rand_block(25, i, 4680, d, d, torch.float32, torch.float32, True) for i in range(4)]
    runs = []
    for _ in range(2):
        st = ispa.Stats(d, d, max_rows=4680, device=DEV)
        for b in blocks:
            st.accum(*b)
        dw, eps = st.solve(1e-3)
        G, C, s, n = st.views()
        torch.cuda.synchronize()
        runs.append((G.clone(), C.clone(), float(s.item()), dw.clone(), eps))
    (Ga, Ca, sa, dwa, ea), (Gb, Cb, sb, dwb, eb) = runs
    assert torch.equal(torch.tril(Ga), torch.tril(Gb))
    assert torch.equal(Ca, Cb)
    assert sa == sb
    assert torch.equal(dwa, dwb)
    assert ea == eb


@pytest.mark.parametrize("d_in,d_out,chunks", [(5120, 2560, (777, 1, 64)), (4096, 4096, (1000,)),
                                                (5120, 5120, (777, 33)), (1536, 1536, (4680, 100)),
                                                (1024, 512, (777, 300, 5))])
def test_gram_256_tiles(d_in, d_out, chunks):
    """Widths that are multiples of 256 take the hand-scheduled Gram kernel: G
    and C against the oracle over ragged chunks (a last 32-row stage part
    empty, a one-row chunk), and a second run bitwise equal to the first. At
    5120 x 5120 (610 tiles on 256 compute units) the last 98 tiles are
    computed as two row pieces each (a 33-row chunk: pieces of one row stage
    each). With fewer tiles than compute units (1536: 57 tiles; 1024 x 512: 18)
    every tile is cut into 4 or 8 row pieces, added in piece order after the
    launch; chunks too short for pieces of 4 stages take the C++ kernel."""
    print(f"[stats] 256-tile Gram {d_in} x {d_out}, chunks {chunks}", flush=True)
    blocks = [rand_block(26, i, r, d_in, d_out, torch.bfloat16, torch.float32) for i, r in enumerate(chunks)]
    runs = []
    for _ in range(2):
        st = ispa.Stats(d_in, d_out, max_rows=max(chunks), device=DEV)
        for b in blocks:
            st.accum(*b)
        torch.cuda.synchronize()
        G, C, s, n = st.views()
        runs.append((G.clone(), C.clone(), float(s.item())))
    check(st, blocks, d_in, d_out)
    (Ga, Ca, sa), (Gb, Cb, sb) = runs
    assert torch.equal(torch.tril(Ga), torch.tril(Gb)) and torch.equal(Ca, Cb) and sa == sb
