"""The launch schedule of a single layer's look-ahead Cholesky factorisation,
checked on the host through the C ABI (no device): every 64 x 64 block on or
below the diagonal receives each earlier panel once, in panel order, after
that panel was factored, no launch writes a block twice, and each launch finds
its panel column complete (Sec. 3.2, Eq. 5: the factorisation of G + lambda I).
The check walks the same workgroup decode the kernel runs."""

import pytest

import paper_2607_00712_amd as ispa


@pytest.mark.parametrize("n_cu", [256, 304, 64, 8, 1])
def test_lookahead_schedule_is_valid_at_every_size(n_cu):
    L = ispa.lib()
    bad = [n for n in range(1, 128) if L.ispa_solve_lookahead_check(n, n_cu) != 0]
    assert bad == [], f"schedule invalid for {bad[:5]} panels on {n_cu} compute units"


def test_lookahead_check_rejects_sizes_out_of_range():
    L = ispa.lib()
    assert L.ispa_solve_lookahead_check(0, 256) == -1
    assert L.ispa_solve_lookahead_check(128, 256) == -1
    assert L.ispa_solve_lookahead_check(80, 0) == -1
