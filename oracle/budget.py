"""Oracle: KV-cache accounting for an L-Layer budget (test infrastructure).

Sec. 4 (Tables 1 and 2) labels each variant ISPA-x with K = xN of the N
layers turned into L-Layers, and prints the fraction of the KV cache kept.
The paper does not state how that fraction is computed. Reading: every
layer holds the same number of keys per cached frame; an
F-Layer keeps the full cache and an L-Layer keeps a fixed local part of it,
a fraction ``r`` of the full cache. The kept fraction is then

    ((N - K) * full + K * r * full) / (N * full) = 1 - x (1 - r).

With r = 1/12, 1/9 and 1/6 this reproduces all nine printed values; those
values are the pin (tests/golden/kv_retained.json).
"""


def n_local_layers(n_layers, x):
    """K = x N layers become L-Layers (Sec. 4 table captions), rounded."""
    return int(round(float(x) * int(n_layers)))


def kv_retained_fraction(x, local_to_full):
    """Fraction of the all-F-Layer KV cache kept when a fraction x of the
    layers keep only ``local_to_full`` of their cache."""
    x = float(x)
    r = float(local_to_full)
    return (1.0 - x) * 1.0 + x * r
