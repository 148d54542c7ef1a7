"""GPU parity of the W8A8 linear layer (Sec. 4 pairs the method with int8
linear layers) against the oracle on identical seeded inputs, through the C
ABI via the ctypes binding: the per-row quantiser and the int8 projection
are bitwise equal to the oracle (the integer product is exact and every fp32
step is one IEEE operation on both sides)."""

import numpy as np
import pytest
import torch

import oracle
import paper_2607_00712_amd as ispa

pytestmark = pytest.mark.gpu

DEV = "cuda"


def f32_bits(t):
    return t.detach().cpu().contiguous().view(torch.int32).numpy()


def bf16_bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy()


def rows_input(rows, cols, dtype, seed):
    """Rows of very different magnitudes, one all-zero row, one row of exact
    ties (absmax 127, so scale 1 and x / scale = x)."""
    g = torch.Generator().manual_seed(seed)
    mag = torch.exp(torch.empty((rows, 1)).uniform_(-12.0, 8.0, generator=g))
    x = torch.randn((rows, cols), generator=g) * mag
    if rows > 2:
        x[1] = 0.0
        ties = torch.arange(cols, dtype=torch.float32) % 9 - 4.0 + 0.5
        ties[0] = 127.0
        x[2] = ties
    return x.to(dtype)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("shape", [(1, 8), (3, 24), (37, 200), (301, 1536), (9, 5120)])
def test_quantize_rows_bitwise(dtype, shape):
    rows, cols = shape
    x = rows_input(rows, cols, dtype, rows * 31 + cols)
    print(f"quantize_rows {dtype} {shape}", flush=True)
    q, s = ispa.quantize_rows(x.to(DEV))
    torch.cuda.synchronize()
    want_q, want_s = oracle.quantize_rows(x.float().numpy())
    assert np.array_equal(q.cpu().numpy(), want_q)
    assert np.array_equal(s.cpu().numpy().view(np.int32), want_s.view(np.int32))


def codes(rows, cols, g):
    return torch.randint(-127, 128, (rows, cols), generator=g, dtype=torch.int8)


def scales(n, g):
    return torch.exp(torch.empty(n).uniform_(-9.0, 1.0, generator=g)).float()


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("shape", [(1, 64, 1), (300, 192, 200), (513, 1536, 384), (257, 320, 131),
                                   (40, 128, 1000), (700, 384, 512), (2560, 128, 5120), (4200, 256, 4096)])
def test_project_w8a8_bitwise(shape, out_dtype):
    n, d_in, d_out = shape
    g = torch.Generator().manual_seed(n * 3 + d_in + d_out)
    qa, qw = codes(n, d_in, g), codes(d_out, d_in, g)
    sa, sw = scales(n, g), scales(d_out, g)
    print(f"project_w8a8 {shape} {out_dtype}", flush=True)
    y = ispa.project_w8a8(qa.to(DEV), sa.to(DEV), qw.to(DEV), sw.to(DEV), out_dtype=out_dtype)
    torch.cuda.synchronize()
    want = oracle.project_w8a8(qa.numpy(), sa.numpy(), qw.numpy(), sw.numpy())
    if out_dtype == torch.float32:
        assert np.array_equal(f32_bits(y), want.view(np.int32))
    else:
        assert np.array_equal(bf16_bits(y), bf16_bits(torch.from_numpy(want).to(torch.bfloat16)))


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_w8a8_fast_kernel_matches_legacy(out_dtype, monkeypatch):
    # the hand-scheduled kernel (widths that are multiples of 256; whole tiles
    # and 128-column halves) and the C++ kernel (ISPA_PROJ_LEGACY=1) are both
    # exact in int32 and dequantise in the same order: bit for bit equal
    n, d_in, d_out = 4200, 512, 4096
    g = torch.Generator().manual_seed(42)
    qa, qw = codes(n, d_in, g).to(DEV), codes(d_out, d_in, g).to(DEV)
    sa, sw = scales(n, g).to(DEV), scales(d_out, g).to(DEV)
    monkeypatch.setenv("ISPA_PROJ_LEGACY", "0")
    y_fast = ispa.project_w8a8(qa, sa, qw, sw, out_dtype=out_dtype)
    monkeypatch.setenv("ISPA_PROJ_LEGACY", "1")
    y_old = ispa.project_w8a8(qa, sa, qw, sw, out_dtype=out_dtype)
    monkeypatch.delenv("ISPA_PROJ_LEGACY")
    torch.cuda.synchronize()
    bits = f32_bits if out_dtype == torch.float32 else bf16_bits
    assert np.array_equal(bits(y_fast), bits(y_old))


def test_extreme_codes_accumulate_exactly():
    # every product is +-127^2 and d_in = 65536 reaches the largest sum the
    # int32 accumulator has to hold (1.06e9)
    n, d_in, d_out = 3, 65536, 5
    qa = torch.full((n, d_in), 127, dtype=torch.int8)
    qa[1] = -127
    qa[2, ::2] = -127
    qw = torch.full((d_out, d_in), 127, dtype=torch.int8)
    qw[3] = -127
    one_a, one_w = torch.ones(n), torch.ones(d_out)
    y = ispa.project_w8a8(qa.to(DEV), one_a.to(DEV), qw.to(DEV), one_w.to(DEV))
    torch.cuda.synchronize()
    want = oracle.project_w8a8(qa.numpy(), one_a.numpy(), qw.numpy(), one_w.numpy())
    assert np.array_equal(f32_bits(y), want.view(np.int32))
    assert want[0, 0] == np.float32(65536 * 127 * 127)


def test_w8a8_chain_and_error_bound():
    # quantise a bf16 activation and a bf16 linear weight on the GPU, then the
    # int8 projection: bitwise equal to the oracle's chain, and within the
    # quantisation error bound of the exact product of the unquantised inputs
    n, d_in, d_out = 700, 1536, 640
    g = torch.Generator().manual_seed(8)
    a = torch.randn((n, d_in), generator=g).to(torch.bfloat16)
    w = (torch.randn((d_out, d_in), generator=g) / d_in ** 0.5).to(torch.bfloat16)
    qa, sa = ispa.quantize_rows(a.to(DEV))
    qw, sw = ispa.quantize_rows(w.to(DEV))
    y = ispa.project_w8a8(qa, sa, qw, sw)
    torch.cuda.synchronize()
    oqa, osa = oracle.quantize_rows(a.float().numpy())
    oqw, osw = oracle.quantize_rows(w.float().numpy())
    want = oracle.project_w8a8(oqa, osa, oqw, osw)
    assert np.array_equal(f32_bits(y), want.view(np.int32))
    # |a.w - a^.w^| <= sum_k |a_k| dw + |w^_k| da with da = s_a / 2, dw = s_w / 2,
    # plus the three fp32 roundings of the dequantisation (acc, * s_a, * s_w)
    A, W = a.double().numpy(), w.double().numpy()
    exact = A @ W.T
    wq = oracle.dequantize_rows(oqw, osw).astype(np.float64)
    bound = (np.abs(A).sum(1)[:, None] * (osw[None, :] / 2) + (osa[:, None] / 2) * np.abs(wq).sum(1)[None, :])
    bound = bound + 2.0 ** -22 * np.abs(want.astype(np.float64))
    err = np.abs(y.cpu().double().numpy() - exact)
    assert np.all(err <= bound)


@pytest.mark.parametrize("shape", [(4680, 1536, 1536), (4680, 5120, 5120), (4000, 128, 4000)])
def test_w8a8_full_size_sampled_rows(shape):
    # the chunk's output projection at the sizes of the two workloads (4680 query
    # rows, hidden d; 128 x 128 and 256 x 128 tiles), and a shape of 256 x 256
    # tiles: the oracle recomputes 24 sampled rows exactly
    n, d_in, d_out = shape
    g = torch.Generator().manual_seed(d_out)
    qa, qw = codes(n, d_in, g), codes(d_out, d_in, g)
    sa, sw = scales(n, g), scales(d_out, g)
    print(f"project_w8a8 full size {shape}", flush=True)
    y = ispa.project_w8a8(qa.to(DEV), sa.to(DEV), qw.to(DEV), sw.to(DEV))
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(d_out).choice(n, 24, replace=False))
    rows[-1] = n - 1
    want = oracle.project_w8a8(qa.numpy()[rows], sa.numpy()[rows], qw.numpy(), sw.numpy())
    assert np.array_equal(f32_bits(y)[rows], want.view(np.int32))
