"""Pins that tie the oracle to the paper and to mathematics, not to itself.

Each ``pin_*`` takes the implementation under test as arguments so that
``test_oracle.py`` runs it against the real oracle and
``test_oracle_mutations.py`` runs it against copies with planted mistakes
(every planted mistake must make at least one pin fail).
"""

import json
import math
import os

import numpy as np
import torch

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def rng(seed):
    return np.random.default_rng(seed)


def bf16_values(a):
    """float64 copy of the bf16 rounding of ``a`` (torch's conversion)."""
    return torch.from_numpy(np.asarray(a, dtype=np.float32)).to(torch.bfloat16).to(torch.float64).numpy()


# ---------------------------------------------------------------- attention

def brute_attention(q, k, v, cache_len, window, sink, n_heads, scale):
    """Pure-Python softmax attention over the key sets of Sec. 3.4, Eq. 7-8.

    Written with scalar loops and math.exp, for tiny inputs only. A key j of
    the cache is local when it is a sink key (j < sink) or among the
    ``window`` most recent keys (j >= cache_len - window).
    """
    n_q, hd = q.shape
    d = hd // n_heads
    res = {}
    for name in ("full", "local", "hist"):
        o = [[0.0] * hd for _ in range(n_q)]
        lse = [[-math.inf] * n_q for _ in range(n_heads)]
        for h in range(n_heads):
            for i in range(n_q):
                keys = []
                for j in range(cache_len):
                    is_local = j < sink or j >= cache_len - window
                    if name == "full" or (name == "local") == is_local:
                        keys.append(j)
                if not keys:
                    continue
                logits = []
                for j in keys:
                    acc = 0.0
                    for c in range(d):
                        acc += float(q[i, h * d + c]) * float(k[j, h * d + c])
                    logits.append(acc * scale)
                mx = max(logits)
                z = sum(math.exp(x - mx) for x in logits)
                lse[h][i] = mx + math.log(z)
                for c in range(d):
                    o[i][h * d + c] = sum(math.exp(x - mx) / z * float(v[j, h * d + c])
                                          for x, j in zip(logits, keys))
        res[name] = (np.array(o), np.array(lse))
    return res


def pin_attention_brute_force(chunk_attention):
    """Tiny shapes, every (window, sink) regime, against the scalar loops."""
    r = rng(1)
    for (n_q, n, w, s, h, d) in [(3, 7, 3, 2, 2, 4), (2, 9, 2, 0, 1, 8), (4, 6, 6, 0, 2, 4),
                                 (1, 5, 1, 1, 1, 3), (3, 8, 3, 5, 1, 4), (2, 4, 9, 9, 2, 2)]:
        q = r.standard_normal((n_q, h * d))
        k = r.standard_normal((n, h * d))
        v = r.standard_normal((n, h * d))
        scale = 1.0 / math.sqrt(d)
        got = chunk_attention(q, k, v, n, w, h, sink_len=s)
        ref = brute_attention(q, k, v, n, w, s, h, scale)
        for name in ("full", "local", "hist"):
            np.testing.assert_allclose(got[name][0], ref[name][0], rtol=0, atol=1e-12)
            np.testing.assert_array_equal(np.isneginf(got[name][1]), np.isneginf(ref[name][1]))
            fin = np.isfinite(ref[name][1])
            np.testing.assert_allclose(got[name][1][fin], ref[name][1][fin], rtol=0, atol=1e-12)


def pin_attention_vs_sdpa(chunk_attention):
    """Library routine: torch SDPA in float64 with an explicit boolean mask."""
    r = rng(2)
    n_q, n, w, s, h, d = 16, 40, 12, 4, 3, 16
    q = r.standard_normal((n_q, h * d))
    k = r.standard_normal((n, h * d))
    v = r.standard_normal((n, h * d))
    got = chunk_attention(q, k, v, n, w, h, sink_len=s)
    j = np.arange(n)
    local_mask = (j < s) | (j >= n - w)
    for name, mask in (("full", np.ones(n, bool)), ("local", local_mask)):
        qt = torch.from_numpy(q).view(n_q, h, d).transpose(0, 1)
        kt = torch.from_numpy(k).view(n, h, d).transpose(0, 1)
        vt = torch.from_numpy(v).view(n, h, d).transpose(0, 1)
        m = torch.from_numpy(np.broadcast_to(mask, (n_q, n)).copy())
        ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=m)
        ref = ref.transpose(0, 1).reshape(n_q, h * d).numpy()
        np.testing.assert_allclose(got[name][0], ref, rtol=0, atol=1e-12)


def pin_softmax_rows_sum_to_one(attend):
    r = rng(3)
    q = 3.0 * r.standard_normal((33, 16))
    k = r.standard_normal((50, 16))
    v = r.standard_normal((50, 16))
    keys = np.arange(5, 45)
    _, _, p = attend(q, k, v, keys, 0.25, return_probs=True)
    assert np.all(p >= 0)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-12)


def pin_local_equals_full_when_window_covers(chunk_attention):
    r = rng(4)
    n_q, n, h, d = 8, 24, 2, 8
    q = r.standard_normal((n_q, h * d))
    k = r.standard_normal((n, h * d))
    v = r.standard_normal((n, h * d))
    for (w, s) in [(24, 0), (30, 0), (16, 8), (20, 10)]:
        got = chunk_attention(q, k, v, n, w, h, sink_len=s)
        assert np.array_equal(got["local"][0], got["full"][0])
        assert np.array_equal(got["local"][1], got["full"][1])
        assert np.all(np.isneginf(got["hist"][1])) and not np.any(got["hist"][0])


def pin_single_visible_key(chunk_attention):
    """window = 1, no sink: every query sees only the newest key."""
    r = rng(5)
    n_q, n, h, d = 4, 12, 2, 8
    q = r.standard_normal((n_q, h * d))
    k = r.standard_normal((n, h * d))
    v = r.standard_normal((n, h * d))
    got = chunk_attention(q, k, v, n, 1, h, sink_len=0)
    o, lse = got["local"]
    for hh in range(h):
        cols = slice(hh * d, (hh + 1) * d)
        np.testing.assert_allclose(o[:, cols], np.broadcast_to(v[n - 1, cols], (n_q, d)), rtol=0, atol=1e-15)
        np.testing.assert_allclose(lse[hh], q[:, cols] @ k[n - 1, cols] / math.sqrt(d), rtol=0, atol=1e-13)


def pin_zero_query_gives_mean(chunk_attention):
    """Q = 0: all logits are 0, so o is the mean of the visible values and
    LSE = ln |V|."""
    r = rng(6)
    n_q, n, w, s, h, d = 3, 20, 6, 3, 2, 4
    q = np.zeros((n_q, h * d))
    k = r.standard_normal((n, h * d))
    v = r.standard_normal((n, h * d))
    got = chunk_attention(q, k, v, n, w, h, sink_len=s)
    j = np.arange(n)
    loc = (j < s) | (j >= n - w)
    for name, sel in (("full", np.ones(n, bool)), ("local", loc), ("hist", ~loc)):
        np.testing.assert_allclose(got[name][0], np.broadcast_to(v[sel].mean(axis=0), (n_q, h * d)),
                                   rtol=0, atol=1e-14)
        np.testing.assert_allclose(got[name][1], math.log(sel.sum()), rtol=0, atol=1e-14)


def pin_dominant_logit(chunk_attention):
    """One key aligned with the query 60 logits above the rest: o ~ v_j."""
    r = rng(7)
    n, h, d = 16, 1, 8
    q = r.standard_normal((1, d))
    q /= np.linalg.norm(q)
    k = 0.01 * r.standard_normal((n, d))
    k[9] = q[0] * 60.0 * math.sqrt(d)
    v = r.standard_normal((n, d))
    o, _ = chunk_attention(q, k, v, n, n, h)["full"]
    np.testing.assert_allclose(o[0], v[9], rtol=0, atol=1e-15)


def pin_key_permutation_invariance(attend):
    r = rng(8)
    q = r.standard_normal((6, 8))
    k = r.standard_normal((30, 8))
    v = r.standard_normal((30, 8))
    keys = np.array([0, 1, 2, 17, 18, 19, 20, 29])
    o1, l1 = attend(q, k, v, keys, 0.3)
    perm = r.permutation(30)
    inv = np.empty_like(perm)
    inv[perm] = np.arange(30)
    o2, l2 = attend(q, k[perm], v[perm], inv[keys][::-1], 0.3)
    np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-13)
    np.testing.assert_allclose(l1, l2, rtol=0, atol=1e-13)


def pin_visible_sets(visible_key_sets):
    """Sec. 3.4, Eq. 7-8 on hand-listed examples."""
    cases = {
        (10, 3, 2): ([0, 1, 7, 8, 9], [2, 3, 4, 5, 6]),
        (10, 3, 0): ([7, 8, 9], [0, 1, 2, 3, 4, 5, 6]),
        (5, 9, 0): ([0, 1, 2, 3, 4], []),
        (6, 2, 4): ([0, 1, 2, 3, 4, 5], []),
        (6, 1, 5): ([0, 1, 2, 3, 4, 5], []),
        (7, 1, 1): ([0, 6], [1, 2, 3, 4, 5]),
    }
    for (n, w, s), (loc, hist) in cases.items():
        a, b = visible_key_sets(n, w, s)
        assert list(a) == loc and list(b) == hist, (n, w, s, list(a), list(b))


def pin_merge_identity(chunk_attention, lse_merge):
    """Eq. 11-12 applied to the local and history branches gives full."""
    r = rng(9)
    n_q, n, w, s, h, d = 24, 200, 50, 20, 2, 16
    q = 2.0 * r.standard_normal((n_q, h * d))
    k = r.standard_normal((n, h * d))
    v = r.standard_normal((n, h * d))
    got = chunk_attention(q, k, v, n, w, h, sink_len=s)
    for hh in range(h):
        cols = slice(hh * d, (hh + 1) * d)
        o, lse = lse_merge(got["local"][0][:, cols], got["local"][1][hh],
                           got["hist"][0][:, cols], got["hist"][1][hh])
        np.testing.assert_allclose(o, got["full"][0][:, cols], rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse, got["full"][1][hh], rtol=0, atol=1e-12)
    # an empty branch leaves the other one untouched (Eq. 11-12 with -inf)
    oa = r.standard_normal((3, 4))
    la = r.standard_normal(3)
    o, lse = lse_merge(oa, la, np.zeros((3, 4)), np.full(3, -np.inf))
    np.testing.assert_allclose(o, oa, rtol=0, atol=1e-15)
    np.testing.assert_allclose(lse, la, rtol=0, atol=1e-15)


# ---------------------------------------------------------------- absorb

def pin_bf16_round_matches_torch(bf16_round):
    """Library routine: torch's float32 -> bfloat16 conversion (RNE)."""
    r = rng(10)
    x = np.concatenate([
        r.standard_normal(20000).astype(np.float32) * np.float32(10.0) ** r.integers(-30, 30, 20000).astype(np.float32),
        # exact ties: bit 15 set and bits 0..14 clear, both parities of bit 16
        (np.arange(1, 4001, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
        np.array([0.0, -0.0, np.inf, -np.inf, 1e-40, -1e-40, 3.3895e38, -3.3895e38], dtype=np.float32),
    ]).astype(np.float32)
    got = bf16_round(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32))
    assert np.isnan(bf16_round(np.array([np.nan], np.float32)))[0]


def pin_residual_rounding(residual):
    """R = bf16(fp32(y_full) - fp32(y_local)), against torch's ops."""
    r = rng(11)
    yf = r.standard_normal((64, 40)).astype(np.float32)
    yl = (yf + np.float32(1e-3) * r.standard_normal((64, 40)).astype(np.float32)).astype(np.float32)
    got = residual(yf, yl)
    ref = (torch.from_numpy(yf) - torch.from_numpy(yl)).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(got, ref)
    assert not np.any(residual(yf, yf))


def pin_stats_chunking_and_psd(Stats):
    r = rng(12)
    x = bf16_values(r.standard_normal((90, 12)))
    yf = r.standard_normal((90, 5)).astype(np.float32)
    yl = r.standard_normal((90, 5)).astype(np.float32)
    a = Stats(12, 5)
    a.accumulate(x, yf, yl)
    b = Stats(12, 5)
    for i0 in (0, 31, 64):
        i1 = {0: 31, 31: 64, 64: 90}[i0]
        b.accumulate(x[i0:i1], yf[i0:i1], yl[i0:i1])
    np.testing.assert_allclose(a.G, b.G, rtol=1e-13, atol=1e-12)
    np.testing.assert_allclose(a.C, b.C, rtol=1e-13, atol=1e-12)
    assert abs(a.s - b.s) <= 1e-12 * a.s and a.n == b.n == 90
    assert np.array_equal(a.G, a.G.T)
    assert np.linalg.eigvalsh(a.G).min() > -1e-10
    # the literal sum of per-row outer products (Sec. 3.2, last paragraph)
    rr = (torch.from_numpy(yf) - torch.from_numpy(yl)).to(torch.bfloat16).double().numpy()
    g = np.zeros((12, 12))
    c = np.zeros((12, 5))
    for t in range(90):
        g += np.outer(x[t], x[t])
        c += np.outer(x[t], rr[t])
    np.testing.assert_allclose(a.G, g, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(a.C, c, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(a.s, float(np.sum(rr * rr)), rtol=1e-12)
    z = Stats(12, 5)
    z.accumulate(x, yf, yf)
    assert not np.any(z.C) and z.s == 0.0


def pin_solve_scalar_hand_example(solve_modulation):
    """D_in = D_out = 1, x = (1, 2), r = (2, 3), lam = 1:
    dW = (1*2 + 2*3) / (1 + 4 + 1) = 8/6."""
    G = np.array([[1.0 * 1 + 2.0 * 2]])
    C = np.array([[1.0 * 2 + 2.0 * 3]])
    dw = solve_modulation(G, C, 1.0)
    assert abs(dw[0, 0] - 4.0 / 3.0) < 1e-15


def pin_solve_normal_equations(Stats, solve_modulation, lstsq_modulation, residual):
    """Residual of (G + lam I) dW = C, and the QR/SVD brute force of Eq. 4."""
    r = rng(13)
    for (m, d_in, d_out, lam) in [(50, 8, 3, 1e-3), (40, 16, 16, 0.5), (12, 20, 4, 1e-2)]:
        x = bf16_values(r.standard_normal((m, d_in)))
        yf = r.standard_normal((m, d_out)).astype(np.float32)
        yl = r.standard_normal((m, d_out)).astype(np.float32)
        st = Stats(d_in, d_out)
        st.accumulate(x, yf, yl)
        dw = solve_modulation(st.G, st.C, lam)
        res = (st.G + lam * np.eye(d_in)) @ dw - st.C
        assert np.linalg.norm(res) <= 1e-12 * np.linalg.norm(st.C)
        ref = lstsq_modulation(x, residual(yf, yl), lam)
        assert np.linalg.norm(dw - ref) <= 1e-9 * np.linalg.norm(ref)


def pin_solve_planted(Stats, solve_modulation):
    """R = X B with lam -> 0 recovers B; y_full - y_local carries the sign."""
    r = rng(14)
    m, d_in, d_out = 64, 10, 6
    x = bf16_values(r.standard_normal((m, d_in)))
    B = r.standard_normal((d_in, d_out))
    target = bf16_values(x @ B)           # exactly representable residual
    st = Stats(d_in, d_out)
    st.accumulate(x, target.astype(np.float32), np.zeros((m, d_out), np.float32))
    dw = solve_modulation(st.G, st.C, 1e-12)
    Bhat = np.linalg.lstsq(x, target, rcond=None)[0]
    np.testing.assert_allclose(dw, Bhat, rtol=0, atol=1e-8)
    np.testing.assert_allclose(dw, B, rtol=0, atol=0.05)


def pin_solve_orthonormal(solve_modulation):
    """X^T X = I gives dW = X^T R / (1 + lam)."""
    r = rng(15)
    x, _ = np.linalg.qr(r.standard_normal((30, 7)))
    R = r.standard_normal((30, 4))
    for lam in (0.0, 1e-3, 0.5, 3.0):
        dw = solve_modulation(x.T @ x, x.T @ R, lam)
        np.testing.assert_allclose(dw, x.T @ R / (1.0 + lam), rtol=0, atol=1e-12)
    big = 1e9
    dw = solve_modulation(x.T @ x, x.T @ R, big)
    np.testing.assert_allclose(big * dw, x.T @ R, rtol=1e-7, atol=1e-9)


def pin_not_spd(solve_modulation, NotSPD):
    """lam = 0 with fewer rows than columns: singular, must be reported."""
    r = rng(16)
    x = r.standard_normal((3, 6))
    G = x.T @ x
    G[5, 5] = -1.0          # make it indefinite so the factorisation must fail
    try:
        solve_modulation(G, np.ones((6, 2)), 0.0)
    except NotSPD:
        return
    raise AssertionError("indefinite system not reported")


def pin_feasibility(Stats, solve_modulation, feasibility, feasibility_direct, residual):
    r = rng(17)
    m, d_in, d_out, lam = 80, 9, 5, 0.01
    x = bf16_values(r.standard_normal((m, d_in)))
    yf = r.standard_normal((m, d_out)).astype(np.float32)
    yl = r.standard_normal((m, d_out)).astype(np.float32)
    st = Stats(d_in, d_out)
    st.accumulate(x, yf, yl)
    dw = solve_modulation(st.G, st.C, lam)
    e1 = feasibility(st.s, dw, st.C, lam)
    e2 = feasibility_direct(x, residual(yf, yl), dw)
    assert abs(e1 - e2) <= 1e-10 * e2 and e2 > 0
    # a residual inside the span of X is absorbed completely (lam -> 0)
    # small integers keep X B exactly representable in bf16
    xi = r.integers(-2, 3, (m, d_in)).astype(np.float64)
    B = r.integers(-2, 3, (d_in, d_out)).astype(np.float64)
    t = (xi @ B).astype(np.float32)
    st2 = Stats(d_in, d_out)
    st2.accumulate(xi, t, np.zeros_like(t))
    dw2 = solve_modulation(st2.G, st2.C, 1e-12)
    np.testing.assert_allclose(dw2, B, rtol=0, atol=1e-9)
    assert feasibility_direct(xi, residual(t, np.zeros_like(t)), dw2) < 1e-18 * st2.s
    assert abs(feasibility(st2.s, dw2, st2.C, 1e-12)) < 1e-9 * st2.s


def pin_select_layers(select_layers):
    eps = np.array([3.0, 1.0, 2.0, 1.0, 0.5, 9.0])
    assert list(select_layers(eps, 3)) == [4, 1, 3]
    assert list(select_layers(eps, 0)) == []
    assert list(select_layers(eps, 6)) == [4, 1, 3, 2, 0, 5]


def pin_inject(inject, bf16_round):
    # hand example: W_new = W + dW (Sec. 3.3), in both storage orders
    W = np.array([[1.0, 2.0], [3.0, 4.0]], dtype=np.float32)
    dW = np.array([[0.5, -1.0], [0.25, 0.0]], dtype=np.float32)
    want = np.array([[1.5, 1.0], [3.25, 4.0]], dtype=np.float32)
    assert np.array_equal(inject(W, dW), want)
    assert np.array_equal(inject(W.T.copy(), dW, transposed=True), want.T)
    # a non-square weight: [D_in, D_out] = [2, 3], transposed [3, 2]
    W2 = np.arange(6, dtype=np.float32).reshape(2, 3)
    d2 = np.full((2, 3), 0.5, dtype=np.float32)
    d2[1, 2] = -2.0
    assert np.array_equal(inject(W2, d2), W2 + d2)
    assert np.array_equal(inject(W2.T.copy(), d2, transposed=True), (W2 + d2).T)
    try:
        inject(W2, d2, transposed=True)
        raise AssertionError("shape mismatch not rejected")
    except ValueError:
        pass
    # bf16 weight: the fp32 sum rounded to nearest even bf16 (spacing 2^-7 at 1)
    one = np.ones((1, 1), dtype=np.float32)
    assert bf16_round(inject(one, np.full((1, 1), 2.0 ** -9, np.float32)))[0, 0] == 1.0
    assert bf16_round(inject(one, np.full((1, 1), 3 * 2.0 ** -9, np.float32)))[0, 0] == 1.0 + 2.0 ** -7


def pin_project(project):
    # hand example, both weight layouts
    a = np.array([[1.0, 2.0, 0.5]])
    w = np.array([[1.0, 0.0], [0.0, 1.0], [2.0, -2.0]])        # [D_in = 3, D_out = 2]
    assert np.array_equal(project(a, w), np.array([[2.0, 1.0]]))
    assert np.array_equal(project(a, w.T.copy(), transposed=True), np.array([[2.0, 1.0]]))
    # identity weight, and agreement with an explicit triple loop
    rng = np.random.default_rng(3)
    x = rng.standard_normal((5, 4))
    assert np.array_equal(project(x, np.eye(4)), x)
    m = rng.standard_normal((4, 3))
    loop = np.array([[sum(x[i, k] * m[k, j] for k in range(4)) for j in range(3)] for i in range(5)])
    assert np.allclose(project(x, m), loop, rtol=1e-14, atol=1e-14)
    assert np.allclose(project(x, m.T.copy(), transposed=True), loop, rtol=1e-14, atol=1e-14)


def pin_quantize_rows(quantize_rows, dequantize_rows):
    q, s = quantize_rows(np.array([[1.0, -2.0, 0.5, 127.0]], np.float32))
    assert list(q[0]) == [1, -2, 0, 127] and s[0] == 1.0          # 0.5 rounds to even 0
    q, s = quantize_rows(np.array([[2.5, 3.5, -2.5, 127.0]], np.float32))
    assert list(q[0]) == [2, 4, -2, 127]                           # half to even, both signs
    q, s = quantize_rows(np.array([[-254.0, 1.0], [0.0, 0.0]], np.float32))
    assert list(q[0]) == [-127, 0] and s[0] == 2.0                 # 1 / 2 = 0.5 -> 0
    assert list(q[1]) == [0, 0] and s[1] == 1.0                    # all-zero row
    # every code within half a step of its value, and the absmax maps to +-127
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((6, 50)) * rng.uniform(0.01, 100, (6, 1))).astype(np.float32)
    q, s = quantize_rows(x)
    err = np.abs(dequantize_rows(q, s).astype(np.float64) - x)
    assert np.all(err <= 0.5 * s[:, None] * (1 + 1e-6))
    assert np.all(np.max(np.abs(q.astype(np.int32)), axis=1) == 127)


def pin_project_w8a8(project_w8a8):
    qa = np.array([[1, -2, 3], [127, 0, -127]], np.int8)
    qw = np.array([[1, 1, 1], [2, 0, -1]], np.int8)               # [d_out = 2, d_in = 3]
    sa = np.array([1.0, 0.5], np.float32)
    sw = np.array([2.0, 0.25], np.float32)
    want = np.array([[2 * 2.0, -1 * 0.25], [0 * 0.5 * 2.0, 381 * 0.5 * 0.25]], np.float32)
    assert np.array_equal(project_w8a8(qa, sa, qw, sw), want)
    # a loop over the codes
    rng = np.random.default_rng(6)
    a = rng.integers(-127, 128, (4, 9)).astype(np.int8)
    w = rng.integers(-127, 128, (3, 9)).astype(np.int8)
    one = np.ones(4, np.float32), np.ones(3, np.float32)
    loop = [[sum(int(a[i, k]) * int(w[j, k]) for k in range(9)) for j in range(3)] for i in range(4)]
    assert np.array_equal(project_w8a8(a, one[0], w, one[1]), np.array(loop, np.float32))


def pin_evict_local(evict_local):
    rows = np.arange(10, dtype=np.float32)[:, None] * np.ones((1, 4), np.float32)
    k, v = evict_local(rows, -rows, 10, 3, 2)
    assert list(k[:, 0]) == [0, 1, 7, 8, 9] and list(v[:, 0]) == [0, -1, -7, -8, -9]
    k, v = evict_local(rows, -rows, 5, 3, 4)       # sink and window meet: all rows
    assert list(k[:, 0]) == [0, 1, 2, 3, 4]
    k, v = evict_local(rows, -rows, 8, 100, 0)     # window beyond the cache
    assert list(k[:, 0]) == list(range(8))
    k, v = evict_local(rows, -rows, 10, 1, 0)      # the last key only
    assert list(k[:, 0]) == [9]


def pin_local_history(LocalHistory):
    lab = lambda a, b: np.arange(a, b, dtype=np.float32)[:, None] * np.ones((1, 2), np.float32)
    h = LocalHistory(lab(0, 6), -lab(0, 6), 6, 4, 1)
    k, v = h.rows()
    assert list(k[:, 0]) == [0, 2, 3, 4, 5]
    h.append(lab(6, 9), -lab(6, 9))                # rows 6..8 arrive
    k, v = h.rows()
    assert list(k[:, 0]) == [0, 5, 6, 7, 8] and list(v[:, 0]) == [0, -5, -6, -7, -8]
    h.append(lab(9, 15), -lab(9, 15))              # more than the window at once
    k, _ = h.rows()
    assert list(k[:, 0]) == [0, 11, 12, 13, 14]


# ---------------------------------------------------------------- budget

def _frac(s):
    a, b = s.split("/")
    return int(a) / int(b)


def pin_kv_table(kv_retained_fraction):
    g = load_golden("kv_retained.json")
    tol = g["printed_precision_percent"] + 1e-9
    for row in g["rows"]:
        got = 100.0 * kv_retained_fraction(row["x"], _frac(row["local_to_full"]))
        assert abs(got - row["kv_percent"]) <= tol, (row, got)


def pin_layer_budget(n_local_layers):
    # K = xN (table captions): 30 layers at 1.3B, 40 layers at 14B
    assert [n_local_layers(30, x) for x in (0.3, 0.4, 0.5)] == [9, 12, 15]
    assert [n_local_layers(40, x) for x in (0.3, 0.4, 0.5)] == [12, 16, 20]


def pin_hyperparams():
    g = load_golden("hyperparams.json")
    assert g["lambda"] == 0.001 and g["t_warm_latent_frames"] == 12
    assert g["t_warm_latent_frames"] // 3 == 4
