"""Comparison helpers for the GPU parity tests. Tolerances:

* attention output: max |O_gpu - O_ref| <= 2e-2 * RMS(O_ref) per output tensor
  (bf16 operands and P rounded to bf16 before P.V, fp32 accumulation);
* LSE: |LSE_gpu - LSE_ref| <= 2e-3 absolute (fp32 scores of bf16 inputs);
* Gram: |G_gpu - G_ref|_ij <= 1e-4 sqrt(G_ii G_jj) and
        |C_gpu - C_ref|_ij <= 1e-4 sqrt(G_ii S_jj), S_jj = sum_k R_kj^2
  (the Cauchy-Schwarz scale of each entry);
* dW: ||dW_gpu - dW_ref||_F / ||dW_ref||_F <= 1e-3.
"""

import numpy as np
import torch

ATTN_TOL = 2e-2
LSE_TOL = 1e-3
GRAM_TOL = 1e-4
DW_TOL = 1e-3


def f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def attn_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    rms = float(np.sqrt(np.mean(ref * ref)))
    return float(np.max(np.abs(got - ref))) / rms


def assert_attn(got, ref, what=""):
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    e = attn_err(got, ref)
    assert e <= ATTN_TOL, f"{what}: max err / RMS = {e:.3e} > {ATTN_TOL}"
    return e


def assert_lse(got, ref, what=""):
    d = float(np.max(np.abs(np.asarray(got, dtype=np.float64) - ref)))
    assert d <= LSE_TOL, f"{what}: LSE max abs err {d:.3e} > {LSE_TOL}"
    return d


def lower_sym(G):
    """Symmetric matrix from the lower triangle of G."""
    L = np.tril(G)
    return L + np.tril(G, -1).T


def assert_gram(G_gpu, C_gpu, G_ref, C_ref, S_ref_cols):
    G = lower_sym(G_gpu)
    dg = np.sqrt(np.maximum(np.diag(G_ref), 0.0))
    scale_g = np.outer(dg, dg)
    scale_c = np.outer(dg, np.sqrt(np.maximum(S_ref_cols, 0.0)))
    eg = np.abs(G - G_ref) / np.maximum(scale_g, 1e-30)
    ec = np.abs(C_gpu - C_ref) / np.maximum(scale_c, 1e-30)
    eg[scale_g == 0] = np.abs(G - G_ref)[scale_g == 0]
    ec[scale_c == 0] = np.abs(C_gpu - C_ref)[scale_c == 0]
    assert eg.max() <= GRAM_TOL, f"G err {eg.max():.3e}"
    assert ec.max() <= GRAM_TOL, f"C err {ec.max():.3e}"
    return float(eg.max()), float(ec.max())


def rel_fro(got, ref):
    return float(np.linalg.norm(got - ref) / np.linalg.norm(ref))
