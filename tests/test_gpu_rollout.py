"""Parity along the 60-chunk streaming rollout at the 1.3B shape (12 heads x
128, chunks of 4680 queries, L-Layer window of 2 chunks, no sink).

One F-Layer and one L-Layer are built chunk by chunk from the rollout's draws,
exactly as the benchmark builds them: the F-Layer appends every chunk to its
cache and attends to all of it (4680 n keys at chunk n, 280800 at chunk 60);
the L-Layer evicts its cache to the local set at the first chunk and then
appends each chunk to its ring (Sec. 3.3). At chunks 1, 2, 3, 30 and 60,
sampled query rows of three heads are checked one by one against the oracle,
which attends over the whole key sequence with the key sets of Eq. 7.
"""

import pytest
import torch

import oracle
import synth
import paper_2607_00712_amd as ispa
from parity_util import assert_attn, assert_lse, f64

pytestmark = pytest.mark.gpu

DEV = "cuda"
ROWS = [0, 1, 255, 256, 2047, 4095, 4096, 4679]
SPOT = (1, 2, 3, 30, 60)
F_LAYER, L_LAYER = 0, 15


def test_rollout_spot_chunks():
    H, d, n_q, win, chunks = 12, 128, 4680, 9360, 60
    D = H * d
    cap = n_q * chunks
    kc = {layer: torch.empty((cap, D), dtype=torch.bfloat16, device=DEV) for layer in (F_LAYER, L_LAYER)}
    vc = {layer: torch.empty((cap, D), dtype=torch.bfloat16, device=DEV) for layer in (F_LAYER, L_LAYER)}
    local = None
    for n in range(1, chunks + 1):
        N = n_q * n
        qs = {}
        for layer in (F_LAYER, L_LAYER):
            q, kn, vn = synth.rollout_chunk(layer, n, n_q, D, DEV)
            qs[layer] = q
            kc[layer][N - n_q:N].copy_(kn)
            vc[layer][N - n_q:N].copy_(vn)
            if layer == L_LAYER:
                if local is None:
                    local = ispa.LocalKV(kc[layer], vc[layer], N, win)
                else:
                    local.append(kn, vn)
        if n not in SPOT:
            continue
        print(f"[rollout] chunk {n}: F-Layer over {N} keys, L-Layer over {local.rows} ring rows", flush=True)
        out_f, lse_f = ispa.attn_chunk(qs[F_LAYER], kc[F_LAYER], vc[F_LAYER], N, N, H)
        r = local.rows
        assert r == min(N, win)
        out_l, lse_l = ispa.attn_chunk(qs[L_LAYER], local.k, local.v, r, r, H)
        torch.cuda.synchronize()
        for h in (0, 5, 11):
            cols = slice(h * d, (h + 1) * d)
            ref_f = oracle.chunk_attention(f64(qs[F_LAYER][:, cols]), f64(kc[F_LAYER][:N, cols]),
                                           f64(vc[F_LAYER][:N, cols]), N, N, 1, branches=("full",),
                                           query_rows=ROWS)
            assert_attn(f64(out_f[:, cols])[ROWS], ref_f["full"][0], f"chunk {n} F-Layer head {h}")
            assert_lse(f64(lse_f[h])[ROWS], ref_f["full"][1][0], f"chunk {n} F-Layer head {h} lse")
            ref_l = oracle.chunk_attention(f64(qs[L_LAYER][:, cols]), f64(kc[L_LAYER][:N, cols]),
                                           f64(vc[L_LAYER][:N, cols]), N, win, 1, branches=("local",),
                                           query_rows=ROWS)
            assert_attn(f64(out_l[:, cols])[ROWS], ref_l["local"][0], f"chunk {n} L-Layer head {h}")
            assert_lse(f64(lse_l[h])[ROWS], ref_l["local"][1][0], f"chunk {n} L-Layer head {h} lse")
