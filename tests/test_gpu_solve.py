"""GPU parity of ispa_solve_modulation (Cholesky + triangular solves, fp32)
and of the whole warmup chain against the oracle."""

import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2607_00712_amd as ispa
from parity_util import DW_TOL, assert_attn, assert_gram, f64, lower_sym, rel_fro

pytestmark = pytest.mark.gpu

DEV = "cuda"


def rows(wid, i, n, d, dtype=torch.bfloat16):
    return synth.normal((n, d), synth.seed_of(wid, i, synth.X), DEV, dtype=dtype)


@pytest.mark.parametrize("d_in,d_out,n", [(200, 72, 700), (600, 136, 1300), (776, 328, 1600), (1288, 64, 2000)])
def test_solve_matches_oracle_ragged(d_in, d_out, n):
    # d not a multiple of the 64-wide panel (776: three 256-blocks and a ragged
    # fourth of 8 rows); 600 and 1288 give three and six 256-blocks, so the
    # sweeps' pairs of blocks end on a ragged pair and on a ragged single;
    # rows > d so G is well conditioned
    lam = 0.5
    x = rows(30, 0, n, d_in)
    yf = synth.normal((n, d_out), synth.seed_of(30, 0, synth.Y_FULL), DEV, dtype=torch.float32)
    yl = synth.normal((n, d_out), synth.seed_of(30, 0, synth.Y_LOCAL), DEV, dtype=torch.float32)
    st = ispa.Stats(d_in, d_out, max_rows=n, device=DEV)
    st.accum(x, yf, yl)
    dw, eps = st.solve(lam)
    ref = oracle.Stats(d_in, d_out)
    ref.accumulate(f64(x), f64(yf).astype(np.float32), f64(yl).astype(np.float32))
    dw_ref = oracle.solve_modulation(ref.G, ref.C, lam)
    assert rel_fro(f64(dw), dw_ref) <= DW_TOL
    eps_ref = oracle.feasibility(ref.s, dw_ref, ref.C, lam)
    assert abs(eps - eps_ref) <= 1e-4 * ref.s
    # G and C are left intact: a second solve with another lambda works
    dw2, _ = st.solve(2 * lam)
    assert rel_fro(f64(dw2), oracle.solve_modulation(ref.G, ref.C, 2 * lam)) <= DW_TOL


def test_not_spd_reported():
    d, n = 64, 80
    x = rows(31, 0, n, d)
    x[:, 5] = 0          # a zero column makes the pivot exactly zero when lambda = 0
    y = synth.normal((n, d), synth.seed_of(31, 0, synth.Y_FULL), DEV, dtype=torch.float32)
    st = ispa.Stats(d, d, max_rows=n, device=DEV)
    st.accum(x, y, torch.zeros_like(y))
    with pytest.raises(ispa.NotSPDError):
        st.solve(0.0)
    dw, _ = st.solve(1e-3)   # regularised: fine again
    assert torch.all(torch.isfinite(dw))


def test_planted_solution():
    # R = X B exactly in bf16 (small integers): dW recovers B as lambda -> 0
    d_in, d_out, n = 64, 32, 512
    g = torch.Generator(device="cpu").manual_seed(32)
    xi = torch.randint(-2, 3, (n, d_in), generator=g).to(torch.bfloat16)
    B = torch.randint(-2, 3, (d_in, d_out), generator=g).float()
    t = (xi.float() @ B)
    st = ispa.Stats(d_in, d_out, max_rows=n, device=DEV)
    st.accum(xi.to(DEV), t.to(DEV), torch.zeros_like(t, device=DEV))
    dw, eps = st.solve(1e-6)
    assert np.max(np.abs(f64(dw) - B.double().numpy())) < 1e-3
    assert abs(eps) < 1e-6 * float((t.double() ** 2).sum())


@pytest.mark.parametrize("d_in,d_out,n", [(1536, 256, 4680), (5120, 256, 8192)])
def test_eps_near_a_fit(d_in, d_out, n):
    # The layer ranking of Sec. 3.3 keeps the layers whose eps is much smaller
    # than s, where eps = s - <dW, C> - lambda ||dW||^2 (Eq. 6) cancels about
    # three digits. R = X B plus noise of 1e-3 of its energy puts eps / s near
    # (1 - d_in / n) 1e-3; eps must still agree with the oracle's to 1% of eps
    # (G is well conditioned at n > d_in, so the fp32 solve's relative error
    # of about 1e-6 moves eps by about 1e-3 of itself). 5120 takes the
    # look-ahead factorisation and the two-stream sweeps.
    lam = 0.5
    x = rows(41, 0, n, d_in)
    b = synth.normal((d_in, d_out), synth.seed_of(41, 1, synth.X), DEV, dtype=torch.float32,
                     scale=d_in ** -0.5)
    noise = synth.normal((n, d_out), synth.seed_of(41, 0, synth.Y_FULL), DEV, dtype=torch.float32,
                         scale=0.032)
    yf = x.float() @ b + noise
    yl = torch.zeros_like(yf)
    st = ispa.Stats(d_in, d_out, max_rows=n, device=DEV)
    st.accum(x, yf, yl)
    dw, eps = st.solve(lam)
    ref = oracle.Stats(d_in, d_out)
    ref.accumulate(f64(x), f64(yf).astype(np.float32), f64(yl).astype(np.float32))
    dw_ref = oracle.solve_modulation(ref.G, ref.C, lam)
    eps_ref = oracle.feasibility(ref.s, dw_ref, ref.C, lam)
    assert 1e-4 * ref.s < eps_ref < 2e-3 * ref.s, (eps_ref, ref.s)
    assert rel_fro(f64(dw), dw_ref) <= DW_TOL
    assert abs(eps - eps_ref) <= 1e-2 * eps_ref, (eps, eps_ref)


def tiny_chain(sink):
    """The tiny single-layer workload end to end: 2 warmup chunks of 64
    queries against a 256-key cache, local window of one chunk, lambda 1e-3."""
    H, d, n_q, N, w, lam = 2, 64, 64, 256, 64, 1e-3
    D = H * d
    st = ispa.Stats(D, D, max_rows=n_q, device=DEV)
    ref = oracle.Stats(D, D)
    for chunk in range(2):
        q, k, v = synth.chunk_qkv(33, 0, chunk, n_q, N, D, DEV)
        out, _, out_l, _ = ispa.attn_chunk(q, k, v, N, w, H, sink_len=sink, dual=True)
        st.accum(out_l, out, out_l)           # X = A_loc, y_full = A_full, y_local = A_loc
        torch.cuda.synchronize()
        o = oracle.chunk_attention(f64(q), f64(k), f64(v), N, w, H, sink_len=sink, branches=("full", "local"))
        assert_attn(f64(out), o["full"][0], "full")
        assert_attn(f64(out_l), o["local"][0], "local")
        # the oracle's statistics take the GPU's attention outputs as given, so the
        # comparison below isolates the statistics and the solve
        xo = oracle.bf16_round(f64(out_l).astype(np.float32))
        ref.accumulate(xo, f64(out).astype(np.float32), f64(out_l).astype(np.float32))
    dw, eps = st.solve(lam)
    dw_ref = oracle.solve_modulation(ref.G, ref.C, lam)
    G, C, s, n = st.views()
    return f64(dw), dw_ref, eps, oracle.feasibility(ref.s, dw_ref, ref.C, lam), ref


@pytest.mark.parametrize("sink", [0, 64])
def test_tiny_chain(sink):
    dw, dw_ref, eps, eps_ref, ref = tiny_chain(sink)
    e = rel_fro(dw, dw_ref)
    print(f"[solve] tiny chain sink={sink} rel err {e:.3e}", flush=True)
    assert e <= DW_TOL
    assert abs(eps - eps_ref) <= 1e-3 * ref.s


def test_wan13b_solve():
    # d = 1536 with 4 warmup chunks of 4680 rows (bf16 X, fp32 y)
    d, lam = 1536, 1e-3
    print("[solve] 1536 x 1536 from 18720 rows", flush=True)
    st = ispa.Stats(d, d, max_rows=4680, device=DEV)
    ref = oracle.Stats(d, d)
    for i in range(4):
        x = rows(34, i, 4680, d)
        yf = synth.normal((4680, d), synth.seed_of(34, i, synth.Y_FULL), DEV, dtype=torch.float32)
        yl = synth.normal((4680, d), synth.seed_of(34, i, synth.Y_LOCAL), DEV, dtype=torch.float32)
        st.accum(x, yf, yl)
        ref.accumulate(f64(x), f64(yf).astype(np.float32), f64(yl).astype(np.float32))
    dw, eps = st.solve(lam)
    dw_ref = oracle.solve_modulation(ref.G, ref.C, lam)
    e = rel_fro(f64(dw), dw_ref)
    print(f"[solve] 1536 rel err {e:.3e}", flush=True)
    assert e <= DW_TOL


def test_async_solve_matches_sync():
    # the variant that does not wait: the same dW bit for bit, the same eps in
    # device memory, and the status word instead of the NOT_SPD error
    d, n = 776, 1600
    x = rows(33, 0, n, d)
    yf = synth.normal((n, d), synth.seed_of(33, 0, synth.Y_FULL), DEV, dtype=torch.float32)
    yl = synth.normal((n, d), synth.seed_of(33, 0, synth.Y_LOCAL), DEV, dtype=torch.float32)
    st = ispa.Stats(d, d, max_rows=n, device=DEV)
    st.accum(x, yf, yl)
    dw_sync, eps_sync = st.solve(0.25)
    dw_async, eps_dev, status_dev = st.solve_async(0.25)
    torch.cuda.synchronize()
    assert torch.equal(dw_sync.view(torch.int32), dw_async.view(torch.int32))
    assert int(status_dev.item()) == 0
    assert float(eps_dev.item()) == eps_sync
    # a zero column with lambda = 0: status 1 and no exception
    x0 = rows(34, 0, 80, 64)
    x0[:, 5] = 0
    y0 = synth.normal((80, 64), synth.seed_of(34, 0, synth.Y_FULL), DEV, dtype=torch.float32)
    st0 = ispa.Stats(64, 64, max_rows=80, device=DEV)
    st0.accum(x0, y0, torch.zeros_like(y0))
    _, _, status0 = st0.solve_async(0.0)
    torch.cuda.synchronize()
    assert int(status0.item()) == 1
    with pytest.raises(ispa.NotSPDError):
        st0.solve(0.0)


def _fill_batch(sb, wid, n):
    """Accumulate different seeded rows into every layer of a StatsBatch."""
    refs = []
    for i, st in enumerate(sb.layers):
        x = rows(wid, i, n, sb.d_in)
        yf = synth.normal((n, sb.d_out), synth.seed_of(wid, i, synth.Y_FULL), DEV, dtype=torch.float32)
        yl = synth.normal((n, sb.d_out), synth.seed_of(wid, i, synth.Y_LOCAL), DEV, dtype=torch.float32)
        st.accum(x, yf, yl)
        refs.append((x, yf, yl))
    return refs


@pytest.mark.parametrize("d_in,d_out,n,layers", [(200, 72, 700, 3), (600, 136, 1300, 2), (776, 328, 1600, 4)])
def test_batch_solve_matches_single(d_in, d_out, n, layers):
    # the batched solve runs every layer's arithmetic unchanged: dW and eps bit
    # for bit those of the single-layer solve, and within the oracle's bound
    lam = 0.5
    print(f"[solve] batch of {layers} at d_in={d_in} d_out={d_out}", flush=True)
    sb = ispa.StatsBatch(layers, d_in, d_out, max_rows=n, device=DEV)
    refs = _fill_batch(sb, 35, n)
    dw_b, eps_b, status_b = sb.solve(lam)
    torch.cuda.synchronize()
    assert status_b.tolist() == [0] * layers
    for i, st in enumerate(sb.layers):
        dw_1, eps_1, status_1 = st.solve_async(lam)
        torch.cuda.synchronize()
        assert int(status_1.item()) == 0
        assert torch.equal(dw_b[i].view(torch.int32), dw_1.view(torch.int32)), f"layer {i}: dW differs"
        assert float(eps_b[i].item()) == float(eps_1.item()), f"layer {i}: eps differs"
        x, yf, yl = refs[i]
        ref = oracle.Stats(d_in, d_out)
        ref.accumulate(f64(x), f64(yf).astype(np.float32), f64(yl).astype(np.float32))
        dw_ref = oracle.solve_modulation(ref.G, ref.C, lam)
        assert rel_fro(f64(dw_b[i]), dw_ref) <= DW_TOL
        assert abs(float(eps_b[i].item()) - oracle.feasibility(ref.s, dw_ref, ref.C, lam)) <= 1e-4 * ref.s
    # every layer's G and C are left intact: solving again gives the same bits
    dw_again, _, _ = sb.solve(lam)
    torch.cuda.synchronize()
    assert torch.equal(dw_again.view(torch.int32), dw_b.view(torch.int32))


def test_batch_eps_ranks_near_fits():
    # three layers whose R is X B plus noise of 1e-2, 1e-3 and 3e-3 of its
    # energy (d_in = 1536): each layer's eps within 1% of the oracle's, and the
    # lowest-eps selection of Sec. 3.3 orders them as the oracle does
    lam, d_in, d_out, n = 0.5, 1536, 256, 4680
    scales = (0.1, 0.032, 0.056)
    print(f"[solve] near-fit batch of {len(scales)} at d_in={d_in}", flush=True)
    sb = ispa.StatsBatch(len(scales), d_in, d_out, max_rows=n, device=DEV)
    eps_ref = []
    for i, (st, sc) in enumerate(zip(sb.layers, scales)):
        x = rows(42, i, n, d_in)
        b = synth.normal((d_in, d_out), synth.seed_of(42, i, synth.X, 1), DEV, dtype=torch.float32,
                         scale=d_in ** -0.5)
        noise = synth.normal((n, d_out), synth.seed_of(42, i, synth.Y_FULL), DEV, dtype=torch.float32,
                             scale=sc)
        yf = x.float() @ b + noise
        yl = torch.zeros_like(yf)
        st.accum(x, yf, yl)
        ref = oracle.Stats(d_in, d_out)
        ref.accumulate(f64(x), f64(yf).astype(np.float32), f64(yl).astype(np.float32))
        eps_ref.append(oracle.feasibility(ref.s, oracle.solve_modulation(ref.G, ref.C, lam), ref.C, lam))
    _, eps_b, status_b = sb.solve(lam)
    torch.cuda.synchronize()
    assert status_b.tolist() == [0] * len(scales)
    eps = [float(e) for e in eps_b.tolist()]
    for i in range(len(scales)):
        assert abs(eps[i] - eps_ref[i]) <= 1e-2 * eps_ref[i], (i, eps[i], eps_ref[i])
    assert oracle.select_layers(eps, 2).tolist() == oracle.select_layers(eps_ref, 2).tolist() == [1, 2]


def test_batch_solve_reports_each_layer():
    # a zero column with lambda = 0 makes only layer 1 fail; the others solve
    d, n = 64, 80
    sb = ispa.StatsBatch(3, d, d, max_rows=n, device=DEV)
    for i, st in enumerate(sb.layers):
        x = rows(36, i, n, d)
        if i == 1:
            x[:, 5] = 0
        y = synth.normal((n, d), synth.seed_of(36, i, synth.Y_FULL), DEV, dtype=torch.float32)
        st.accum(x, y, torch.zeros_like(y))
    dw, eps, status = sb.solve(0.0)
    torch.cuda.synchronize()
    assert status.tolist() == [0, 1, 0]
    for i in (0, 2):
        dw_1, eps_1, _ = sb.layers[i].solve_async(0.0)
        torch.cuda.synchronize()
        assert torch.equal(dw[i].view(torch.int32), dw_1.view(torch.int32))


def test_batch_solve_wan13b_size():
    # 4 layers of d = 1536 (the per-layer systems of the 1.3B absorption) from
    # 4680 rows each plus lambda: bit for bit the single-layer solve
    d, n, layers, lam = 1536, 4680, 4, 1e-1
    print("[solve] batch of 4 at 1536", flush=True)
    sb = ispa.StatsBatch(layers, d, d, max_rows=n, device=DEV)
    _fill_batch(sb, 37, n)
    dw_b, eps_b, status_b = sb.solve(lam)
    torch.cuda.synchronize()
    assert status_b.tolist() == [0] * layers
    for i in (0, 3):
        dw_1, eps_1, _ = sb.layers[i].solve_async(lam)
        torch.cuda.synchronize()
        assert torch.equal(dw_b[i].view(torch.int32), dw_1.view(torch.int32))
        assert float(eps_b[i].item()) == float(eps_1.item())


def test_batch_matches_single_with_look_ahead():
    # d = 3072 (48 panels): the single-layer factorisation takes its look-ahead
    # form (panel groups applied by extra workgroups of later panel launches),
    # the batch defers every super-panel to launches of its own; every panel's
    # product is subtracted on its own in panel order either way, so dW and
    # eps agree bit for bit
    d, d_out, n, layers, lam = 3072, 256, 4000, 2, 1e-1
    print("[solve] batch of 2 at 3072", flush=True)
    sb = ispa.StatsBatch(layers, d, d_out, max_rows=n, device=DEV)
    _fill_batch(sb, 38, n)
    dw_b, eps_b, status_b = sb.solve(lam)
    torch.cuda.synchronize()
    assert status_b.tolist() == [0] * layers
    for i in range(layers):
        dw_1, eps_1, _ = sb.layers[i].solve_async(lam)
        torch.cuda.synchronize()
        assert torch.equal(dw_b[i].view(torch.int32), dw_1.view(torch.int32))
        assert float(eps_b[i].item()) == float(eps_1.item())


@pytest.mark.parametrize("d", [200, 776, 1288, 2560, 3000])
def test_look_ahead_factorisation_is_bitwise(d, monkeypatch):
    # the look-ahead form against one launch per panel applied everywhere, at
    # sizes where the schedule's bands end ragged or the form is not the
    # default (ISPA_SOLVE_LOOKAHEAD forces it): the same bits
    d_out, n, lam = 64, 4000, 1e-1
    print(f"[solve] look-ahead on / off at d={d}", flush=True)
    st = ispa.Stats(d, d_out, max_rows=n, device=DEV)
    x = rows(39, 0, n, d)
    yf = synth.normal((n, d_out), synth.seed_of(39, 0, synth.Y_FULL), DEV, dtype=torch.float32)
    yl = synth.normal((n, d_out), synth.seed_of(39, 0, synth.Y_LOCAL), DEV, dtype=torch.float32)
    st.accum(x, yf, yl)
    out = {}
    for v in ("0", "1"):
        monkeypatch.setenv("ISPA_SOLVE_LOOKAHEAD", v)
        dw, eps, status = st.solve_async(lam)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        out[v] = (dw.clone(), float(eps.item()))
    assert torch.equal(out["0"][0].view(torch.int32), out["1"][0].view(torch.int32))
    assert out["0"][1] == out["1"][1]


@pytest.mark.parametrize("d,d_out", [(776, 328), (1288, 200), (600, 136), (304, 64)])
def test_sweeps_on_two_streams_are_bitwise(d, d_out, monkeypatch):
    # the sweeps split the right-hand side's columns in two halves on two
    # streams (d_out >= 128; 64 stays on one): the same bits as one stream
    n, lam = 2000, 1e-2
    print(f"[solve] sweeps on one / two streams at d={d} d_out={d_out}", flush=True)
    st = ispa.Stats(d, d_out, max_rows=n, device=DEV)
    x = rows(40, 0, n, d)
    yf = synth.normal((n, d_out), synth.seed_of(40, 0, synth.Y_FULL), DEV, dtype=torch.float32)
    yl = synth.normal((n, d_out), synth.seed_of(40, 0, synth.Y_LOCAL), DEV, dtype=torch.float32)
    st.accum(x, yf, yl)
    out = {}
    for v in ("0", "1"):
        monkeypatch.setenv("ISPA_SOLVE_TWO_STREAMS", v)
        dw, eps, status = st.solve_async(lam)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        out[v] = (dw.clone(), float(eps.item()))
    assert torch.equal(out["0"][0].view(torch.int32), out["1"][0].view(torch.int32))
    assert out["0"][1] == out["1"][1]


@pytest.mark.timeout(900)
def test_14b_absorption():
    # the 14B layer's absorption: G (5120 x 5120) and C from 4 warmup chunks of
    # 4680 rows (bf16 X, fp32 y_full / y_local), then dW and eps; G and C on
    # the Cauchy-Schwarz scale, dW within 1e-3 of the fp64 oracle
    d, n, lam = 5120, 4680, 1e-3
    print("[solve] 14B absorption: 5120 x 5120 from 4 x 4680 rows", flush=True)
    st = ispa.Stats(d, d, max_rows=n, device=DEV)
    ref = oracle.Stats(d, d)
    s_cols = np.zeros(d)
    for i in range(4):
        x = rows(38, i, n, d)
        yf = synth.normal((n, d), synth.seed_of(38, i, synth.Y_FULL), DEV, dtype=torch.float32)
        yl = synth.normal((n, d), synth.seed_of(38, i, synth.Y_LOCAL), DEV, dtype=torch.float32)
        st.accum(x, yf, yl)
        r = ref.accumulate(f64(x), f64(yf).astype(np.float32), f64(yl).astype(np.float32))
        s_cols += np.sum(r * r, axis=0)
        del x, yf, yl, r
    G, C, S, n_rows = st.views()
    torch.cuda.synchronize()
    assert n_rows == 4 * n
    eg, ec = assert_gram(f64(G), f64(C), ref.G, ref.C, s_cols)
    print(f"[solve] 14B Gram err {eg:.2e} / {ec:.2e}", flush=True)
    dw, eps = st.solve(lam)
    dw_ref = oracle.solve_modulation(ref.G, ref.C, lam)
    e = rel_fro(f64(dw), dw_ref)
    print(f"[solve] 14B dW rel err {e:.3e}", flush=True)
    assert e <= DW_TOL
    assert abs(eps - oracle.feasibility(ref.s, dw_ref, ref.C, lam)) <= 1e-4 * ref.s


def test_eps_small_relative_to_s():
    """A layer whose discrepancy is almost in the span of its inputs (R = X B
    plus 3 % noise, eps / s ~ 1e-3): the layers the ranking of Sec. 3.3 keeps
    are of this kind, and eps is then a small difference of large terms."""
    d_in, d_out, n, lam = 1536, 128, 4680, 1e-3
    print("[solve] eps << s at d = 1536", flush=True)
    x = rows(36, 0, n, d_in)
    g = torch.Generator(device="cpu").manual_seed(36)
    B = (torch.randn(d_in, d_out, generator=g, dtype=torch.float64) / np.sqrt(d_in)).to(DEV)
    noise = torch.randn(n, d_out, generator=g, dtype=torch.float64).to(DEV)
    yf = (x.double() @ B + 0.03 * noise).float()
    st = ispa.Stats(d_in, d_out, max_rows=n, device=DEV)
    st.accum(x, yf, torch.zeros_like(yf))
    dw, eps = st.solve(lam)
    ref = oracle.Stats(d_in, d_out)
    r = ref.accumulate(f64(x), f64(yf).astype(np.float32), np.zeros((n, d_out), dtype=np.float32))
    dw_ref = oracle.solve_modulation(ref.G, ref.C, lam)
    assert rel_fro(f64(dw), dw_ref) <= DW_TOL
    eps_ref = oracle.feasibility(ref.s, dw_ref, ref.C, lam)
    # the closed form against the direct residual of the same dW (Eq. 6)
    assert eps_ref == pytest.approx(oracle.feasibility_direct(f64(x), r, dw_ref), rel=1e-6)
    assert 1e-4 < eps_ref / ref.s < 1e-2
    assert abs(eps - eps_ref) <= 0.02 * eps_ref, (eps, eps_ref, ref.s)
