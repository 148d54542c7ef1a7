"""Plain, slow, obviously-correct CPU oracle for the ISPA hot path.

THIS PACKAGE IS TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import or call it. The product
path (``paper_2607_00712_amd``) never imports it and shares no code with it:
no kernels, helpers, tables or constants. Both sides receive the same seeded
inputs from ``synth``, which holds none of the method's arithmetic.

Everything here is fp64 numpy/scipy unless a step is defined by a rounding
(bf16 inputs, the bf16 residual), and each function cites the passage of the
paper (arXiv 2607.00712, "Instance-Specific Parametric Absorption") it
follows:

* ``attention``  -- chunk attention over an explicit key set (Sec. 2, Eq. 3;
  Sec. 3.4, Eq. 7-10) and the log-sum-exp fusion (Eq. 11-12).
* ``absorb``     -- residual, sufficient statistics, closed-form ridge solve,
  feasibility score, layer ranking and the weight update (Sec. 3.2, Eq. 4-6;
  Sec. 3.3).
* ``kvcache``    -- what an L-Layer's cache holds after the permanent
  eviction (Sec. 3.3; the local set of Eq. 7 as chunks keep arriving).
* ``w8a8``       -- int8 quantisation of the linear layers (Sec. 4, Fig. 7).
* ``budget``     -- KV-cache accounting for a given L-Layer budget
  (Sec. 4, Table 1/2 "KVCache" column; K = xN).

Pins that tie each function to something other than itself live in
``tests/test_oracle.py``; the values the paper prints live in
``tests/golden/``.
"""

from .attention import (
    visible_key_sets,
    attend,
    chunk_attention,
    lse_merge,
)
from .absorb import (
    NotSPD,
    bf16_round,
    residual,
    Stats,
    solve_modulation,
    lstsq_modulation,
    feasibility,
    feasibility_direct,
    select_layers,
    inject,
    project,
)
from .kvcache import evict_local, LocalHistory
from .w8a8 import quantize_rows, dequantize_rows, project_w8a8
from .budget import kv_retained_fraction, n_local_layers

__all__ = [
    "visible_key_sets",
    "attend",
    "chunk_attention",
    "lse_merge",
    "NotSPD",
    "bf16_round",
    "residual",
    "Stats",
    "solve_modulation",
    "lstsq_modulation",
    "feasibility",
    "feasibility_direct",
    "select_layers",
    "inject",
    "project",
    "evict_local",
    "LocalHistory",
    "quantize_rows",
    "dequantize_rows",
    "project_w8a8",
    "kv_retained_fraction",
    "n_local_layers",
]
