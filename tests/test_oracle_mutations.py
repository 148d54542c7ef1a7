"""Plant plausible mistakes in copies of the oracle (CPU only) and check that
the pins catch every one of them: a dropped term, a wrong sign, an index off
by one, a transposed or swapped operand, a wrong rounding."""

import importlib
import inspect
import types

import pytest

import oracle_pins as P


def mutant(module_name, old, new):
    src = inspect.getsource(importlib.import_module(module_name))
    assert src.count(old) >= 1, f"mutation anchor not found: {old!r}"
    mod = types.ModuleType(module_name + "_mutant")
    exec(compile(src.replace(old, new, 1), module_name + "_mutant", "exec"), mod.__dict__)
    return mod


def attention_pins(m):
    return [
        lambda: P.pin_visible_sets(m.visible_key_sets),
        lambda: P.pin_attention_brute_force(m.chunk_attention),
        lambda: P.pin_attention_vs_sdpa(m.chunk_attention),
        lambda: P.pin_softmax_rows_sum_to_one(m.attend),
        lambda: P.pin_local_equals_full_when_window_covers(m.chunk_attention),
        lambda: P.pin_single_visible_key(m.chunk_attention),
        lambda: P.pin_zero_query_gives_mean(m.chunk_attention),
        lambda: P.pin_dominant_logit(m.chunk_attention),
        lambda: P.pin_key_permutation_invariance(m.attend),
        lambda: P.pin_merge_identity(m.chunk_attention, m.lse_merge),
    ]


def absorb_pins(m):
    return [
        lambda: P.pin_bf16_round_matches_torch(m.bf16_round),
        lambda: P.pin_residual_rounding(m.residual),
        lambda: P.pin_stats_chunking_and_psd(m.Stats),
        lambda: P.pin_solve_scalar_hand_example(m.solve_modulation),
        lambda: P.pin_solve_normal_equations(m.Stats, m.solve_modulation, m.lstsq_modulation, m.residual),
        lambda: P.pin_solve_planted(m.Stats, m.solve_modulation),
        lambda: P.pin_solve_orthonormal(m.solve_modulation),
        lambda: P.pin_not_spd(m.solve_modulation, m.NotSPD),
        lambda: P.pin_feasibility(m.Stats, m.solve_modulation, m.feasibility, m.feasibility_direct, m.residual),
        lambda: P.pin_select_layers(m.select_layers),
        lambda: P.pin_inject(m.inject, m.bf16_round),
        lambda: P.pin_project(m.project),
    ]


def w8a8_pins(m):
    return [lambda: P.pin_quantize_rows(m.quantize_rows, m.dequantize_rows),
            lambda: P.pin_project_w8a8(m.project_w8a8)]


def kvcache_pins(m):
    return [lambda: P.pin_evict_local(m.evict_local),
            lambda: P.pin_local_history(m.LocalHistory)]


def budget_pins(m):
    return [lambda: P.pin_kv_table(m.kv_retained_fraction),
            lambda: P.pin_layer_budget(m.n_local_layers)]


MUTATIONS = [
    # attention
    ("oracle.attention", "s = (q[r0:r1] @ ks.T) * scale", "s = (q[r0:r1] @ ks.T)", attention_pins),
    ("oracle.attention", "p = e / l", "p = e / e.sum(axis=0, keepdims=True)", attention_pins),
    ("oracle.attention", "o[r0:r1] = p @ vs", "o[r0:r1] = p @ ks", attention_pins),
    ("oracle.attention", "lse[r0:r1] = m[:, 0] + np.log(l[:, 0])", "lse[r0:r1] = np.log(l[:, 0])", attention_pins),
    ("oracle.attention", "in_local[max(n - w, 0):] = True", "in_local[max(n - w + 1, 0):] = True", attention_pins),
    ("oracle.attention", "in_local[: min(s, n)] = True", "pass", attention_pins),
    ("oracle.attention", "wb = np.where(both_empty, 0.0, np.exp(lse_b - lse_safe))",
     "wb = np.where(both_empty, 0.0, np.exp(lse_safe - lse_b))", attention_pins),
    ("oracle.attention", "e = np.exp(s - m)", "e = np.exp(s - m.mean())", attention_pins),
    # absorb
    ("oracle.absorb", "rounded = ((u + 0x7FFF + lsb) & 0xFFFF0000)", "rounded = ((u) & 0xFFFF0000)", absorb_pins),
    ("oracle.absorb", "rounded = ((u + 0x7FFF + lsb) & 0xFFFF0000)", "rounded = ((u + 0x8000) & 0xFFFF0000)", absorb_pins),
    ("oracle.absorb", "np.asarray(y_full, dtype=np.float32) - np.asarray(y_local, dtype=np.float32)",
     "np.asarray(y_local, dtype=np.float32) - np.asarray(y_full, dtype=np.float32)", absorb_pins),
    ("oracle.absorb", "return bf16_round(d).astype(np.float64)", "return d.astype(np.float64)", absorb_pins),
    ("oracle.absorb", "self.C += x.T @ r", "self.C += x.T @ np.asarray(y_full, dtype=np.float64)", absorb_pins),
    ("oracle.absorb", "self.G += x.T @ x", "self.G += x @ x.T if x.shape[0] == x.shape[1] else x.T @ x * 1.0001", absorb_pins),
    ("oracle.absorb", "a = G + float(lam) * np.eye(G.shape[0])", "a = G", absorb_pins),
    ("oracle.absorb", "a = G + float(lam) * np.eye(G.shape[0])", "a = G + 2.0 * float(lam) * np.eye(G.shape[0])", absorb_pins),
    ("oracle.absorb", "return float(s) - float(np.sum(dW * C)) - float(lam) * float(np.sum(dW * dW))",
     "return float(s) - float(np.sum(dW * C))", absorb_pins),
    ("oracle.absorb", "return float(s) - float(np.sum(dW * C)) - float(lam) * float(np.sum(dW * dW))",
     "return float(s) + float(np.sum(dW * C)) - float(lam) * float(np.sum(dW * dW))", absorb_pins),
    ("oracle.absorb", "key=lambda i: (eps[i], i)", "key=lambda i: (-eps[i], i)", absorb_pins),
    ("oracle.absorb", "self.s += float(np.sum(r * r))", "self.s += float(np.sum(np.abs(r)))", absorb_pins),
    ("oracle.absorb", "        d = d.T", "        pass", absorb_pins),
    ("oracle.absorb", "return (W + d).astype(np.float32)", "return (W - d).astype(np.float32)", absorb_pins),
    ("oracle.absorb", "return a @ (w.T if transposed else w)", "return a @ (w if transposed else w.T)", absorb_pins),
    # w8a8
    ("oracle.w8a8", "q = np.rint((x / scale[:, None]).astype(np.float32))",
     "q = np.floor((x / scale[:, None]).astype(np.float32) + 0.5)", w8a8_pins),
    ("oracle.w8a8", "(amax / np.float32(127.0))", "(amax / np.float32(128.0))", w8a8_pins),
    ("oracle.w8a8", "acc = np.asarray(qa, dtype=np.int64) @ np.asarray(qw, dtype=np.int64).T",
     "acc = np.asarray(qa, dtype=np.int64) @ np.asarray(qw, dtype=np.int64).T[:, ::-1]", w8a8_pins),
    ("oracle.w8a8", "y = acc.astype(np.float32) * np.asarray(sa, dtype=np.float32)[:, None]",
     "y = acc.astype(np.float32)", w8a8_pins),
    # kvcache
    ("oracle.kvcache", "return k[local], v[local]", "return k[local], k[local]", kvcache_pins),
    ("oracle.kvcache", "k = np.concatenate(self.k, axis=0)", "k = self.k[-1]", kvcache_pins),
    ("oracle.kvcache", "return evict_local(k, v, k.shape[0], self.window, self.sink)",
     "return evict_local(k, v, k.shape[0], self.window + 1, self.sink)", kvcache_pins),
    # budget
    ("oracle.budget", "return (1.0 - x) * 1.0 + x * r", "return 1.0 - x * r", budget_pins),
    ("oracle.budget", "return int(round(float(x) * int(n_layers)))",
     "return int(round((1.0 - float(x)) * int(n_layers)))", budget_pins),
]


@pytest.mark.parametrize("module_name,old,new,pins", MUTATIONS,
                         ids=[f"{m[0].split('.')[-1]}-{i}" for i, m in enumerate(MUTATIONS)])
def test_planted_mistake_is_caught(module_name, old, new, pins):
    m = mutant(module_name, old, new)
    caught = 0
    for pin in pins(m):
        try:
            pin()
        except Exception:
            caught += 1
    assert caught >= 1, f"no pin caught the mutation {old!r} -> {new!r}"


def test_unmutated_copies_pass():
    for name, pins in (("oracle.attention", attention_pins), ("oracle.absorb", absorb_pins),
                       ("oracle.kvcache", kvcache_pins), ("oracle.w8a8", w8a8_pins),
                       ("oracle.budget", budget_pins)):
        m = mutant(name, "\"\"\"", "\"\"\"")
        for pin in pins(m):
            pin()
