"""Oracle: layer absorption by closed-form least squares (test infrastructure).

Definitions followed (arXiv 2607.00712):

* Sec. 3.2, Eq. 4: minimise ||A_loc (W + dW) - A_full W||^2 + lam ||dW||^2,
  read as squared Frobenius norms (ridge regression).
* Sec. 3.2, the line after Eq. 4: residual R = (A_full - A_loc) W.
* Sec. 3.2, Eq. 5: dW = (A_loc^T A_loc + lam I)^-1 A_loc^T R.
* Sec. 3.2, Eq. 6: feasibility score eps = ||A_loc (W + dW) - A_full W||_F^2.
* Sec. 3.2, last paragraph: the method only sums A_loc^T A_loc and A_loc^T R
  over the warmup rows and solves one D x D system at the end of warmup.
* Sec. 3.3: layers are ranked by eps ascending and the K lowest become
  L-Layers; each of them takes W_new = W + dW in place and from then on
  projects its local attention output with it: Y = A_loc W_new (Sec. 3.1
  step 3).

Readings where the paper is silent:

* X denotes the rows of A_loc that are fed to the statistics (one row per
  token of every warmup chunk, heads concatenated), already in bf16.
* The residual is taken from two outputs y_full and y_local of the caller's
  choice (post-projection A*W for the paper's dW directly, or the attention
  outputs themselves, in which case the paper's dW is the result times W).
  It is formed as bf16_rne(fp32(y_full) - fp32(y_local)); this rounding is
  part of the operation's definition, so the oracle performs it too, and
  then works in float64.
* lam is added to the summed Gram matrix (no division by the row count).
* "Matrix inversion" is carried out as a Cholesky solve of the SPD system;
  a non-positive pivot (possible only when lam = 0) is reported as NotSPD.
* Ties in the ranking are broken by layer index (stable ascending sort).
* W is stored either as in Eq. 4 ([D_in, D_out], rows are input features) or
  transposed ([D_out, D_in], the usual linear-layer weight); a bf16 weight is
  updated as bf16_rne(fp32(W) + dW), an fp32 weight as fp32(W) + dW (one IEEE
  float32 addition per element).
"""

import numpy as np
import scipy.linalg


class NotSPD(ArithmeticError):
    """G + lam I is not (numerically) symmetric positive definite."""


def bf16_round(x):
    """Round float32 values to the nearest bfloat16, ties to even.

    bfloat16 keeps the top 16 bits of an IEEE-754 binary32 word. Rounding to
    nearest-even adds 0x7FFF plus the lowest kept bit to the word before
    truncating. NaN stays NaN (quiet). Returns float32 values that are exactly
    representable in bfloat16.
    """
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    rounded = ((u + 0x7FFF + lsb) & 0xFFFF0000).astype(np.uint32)
    nan = np.isnan(x)
    quiet = ((u.astype(np.uint32) | 0x00400000) & 0xFFFF0000).astype(np.uint32)
    rounded = np.where(nan, quiet, rounded)
    return rounded.view(np.float32).reshape(x.shape)


def residual(y_full, y_local):
    """R = bf16_rne(fp32(y_full) - fp32(y_local)) as float64 (Sec. 3.2).

    The subtraction is one IEEE float32 operation per element; the result is
    then rounded once to bfloat16.
    """
    d = np.asarray(y_full, dtype=np.float32) - np.asarray(y_local, dtype=np.float32)
    return bf16_round(d).astype(np.float64)


class Stats:
    """Sufficient statistics summed over warmup rows (Sec. 3.2, last paragraph).

    G = sum X^T X  (d_in x d_in), C = sum X^T R (d_in x d_out),
    s = sum ||R||_F^2, n = number of rows.
    """

    def __init__(self, d_in, d_out):
        self.d_in = int(d_in)
        self.d_out = int(d_out)
        self.G = np.zeros((self.d_in, self.d_in), dtype=np.float64)
        self.C = np.zeros((self.d_in, self.d_out), dtype=np.float64)
        self.s = 0.0
        self.n = 0

    def accumulate(self, x, y_full, y_local):
        """Add one block of rows: x [rows, d_in]; y_* [rows, d_out]."""
        x = np.asarray(x, dtype=np.float64)
        r = residual(y_full, y_local)
        if x.shape[0] != r.shape[0] or x.shape[1] != self.d_in or r.shape[1] != self.d_out:
            raise ValueError("shape mismatch")
        self.G += x.T @ x
        self.C += x.T @ r
        self.s += float(np.sum(r * r))
        self.n += x.shape[0]
        return r


def solve_modulation(G, C, lam):
    """dW = (G + lam I)^-1 C by Cholesky factorisation (Sec. 3.2, Eq. 5)."""
    G = np.asarray(G, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    a = G + float(lam) * np.eye(G.shape[0])
    try:
        factor = scipy.linalg.cho_factor(a, lower=True, check_finite=True)
    except np.linalg.LinAlgError as exc:
        raise NotSPD(str(exc)) from exc
    return scipy.linalg.cho_solve(factor, C, check_finite=True)


def lstsq_modulation(x, r, lam):
    """Direct minimiser of Eq. 4 (brute force for small sizes).

    Stacks the ridge problem as an ordinary least-squares problem
    [X; sqrt(lam) I] dW ~ [R; 0] and solves it with an orthogonal
    factorisation (numpy.linalg.lstsq), never forming X^T X.
    """
    x = np.asarray(x, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    d_in = x.shape[1]
    a = np.vstack([x, np.sqrt(float(lam)) * np.eye(d_in)])
    b = np.vstack([r, np.zeros((d_in, r.shape[1]))])
    sol, *_ = np.linalg.lstsq(a, b, rcond=None)
    return sol


def feasibility(s, dW, C, lam):
    """eps of Eq. 6 from the summed statistics.

    With X(W + dW) - A_full W = X dW - R and (G + lam I) dW = C:
    eps = ||X dW - R||^2 = s - tr(dW^T C) - lam ||dW||_F^2.
    """
    dW = np.asarray(dW, dtype=np.float64)
    C = np.asarray(C, dtype=np.float64)
    return float(s) - float(np.sum(dW * C)) - float(lam) * float(np.sum(dW * dW))


def feasibility_direct(x, r, dW):
    """eps of Eq. 6 evaluated from the rows themselves: ||X dW - R||_F^2."""
    e = np.asarray(x, dtype=np.float64) @ np.asarray(dW, dtype=np.float64) - np.asarray(r, dtype=np.float64)
    return float(np.sum(e * e))


def select_layers(eps, k):
    """Indices of the k layers with the lowest eps (Sec. 3.3), ascending.

    Ties are broken by layer index.
    """
    eps = np.asarray(eps, dtype=np.float64)
    order = sorted(range(eps.size), key=lambda i: (eps[i], i))
    return np.asarray(order[: int(k)], dtype=np.int64)


def inject(W, dW, transposed=False):
    """W_new = W + dW for an L-Layer's output projection (Sec. 3.3).

    ``W`` is float32 holding the weight's values (bf16 values for a bf16
    weight); ``dW`` is [D_in, D_out] as solved by Eq. 5. With ``transposed``
    the weight is [D_out, D_in] and receives dW^T. Returns the float32 sum
    (the caller rounds to bf16 with bf16_round for a bf16 weight).
    """
    W = np.asarray(W, dtype=np.float32)
    d = np.asarray(dW, dtype=np.float32)
    if transposed:
        d = d.T
    if W.shape != d.shape:
        raise ValueError("weight and dW shapes differ")
    return (W + d).astype(np.float32)


def project(a, w, transposed=False):
    """The output projection Y = A W of Eq. 4 (Sec. 3.1 step 3 with W_new).

    ``a`` [n, D_in]; ``w`` [D_in, D_out], or with ``transposed`` the
    linear-layer weight [D_out, D_in] (Y = A W^T). float64.
    """
    a = np.asarray(a, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    return a @ (w.T if transposed else w)
