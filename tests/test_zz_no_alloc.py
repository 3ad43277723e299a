"""sc_attention_noalloc (attention with the library's own scratch, for
callers that cannot allocate) against sc_attention on the same inputs.

Two calls in a row on one GPU, the second on a smaller input, so the second
runs over the scratch the first left behind: the Wan-shaped progressive
diagonal (912 work units, its last 144 cut into key-range pieces whose
partials live in the scratch; fewer pieces than sc_attention may use), then
the same diagonal with one latent frame per chunk (336 units; its last 80
cut into fewer pieces).  Each output must match sc_attention's
within the bf16 attention tolerances (max 2e-2, mean 2e-3, relative
Frobenius 1e-2 per head: only the summation order may differ) and the oracle
on sampled rows; a plan that needs no pieces must match bit for bit.
"""
import dataclasses

import numpy as np
import pytest

import paper_2609_22283_amd as sc
from synth.configs import SMALL, WAN, cfg4_prog

from gpu_cases import AttnCase, bf16_gates, from_device, sample_rows, torch_mod

pytestmark = pytest.mark.gpu


def _noalloc(case):
    torch = torch_mod()
    o = torch.full_like(case.q_dev, float("nan"))
    sc.sc_attention_noalloc(case.plan, case.cache, case.layer, case.q_dev, o, case.scale)
    torch.cuda.synchronize()
    out = from_device(o)
    n = case.geo.tokens_per_chunk
    return {i: out[i * n:(i + 1) * n] for i in range(len(case.pack))}


def test_noalloc_matches_attention_on_two_calls():
    assert sc.sc_attention_noalloc_scratch_bytes() == 64 << 20
    one_frame = dataclasses.replace(WAN, frames_per_chunk=1)
    wl = cfg4_prog(False)
    for geo, seed in ((WAN, 41), (one_frame, 42)):
        case = AttnCase(geo, sc.SC_DTYPE_BF16, wl.policy, wl.pack, wl.resident, seed=seed)
        assert sc.sc_attention_workspace_bytes(case.plan, case.cache) > 0   # the split is taken
        ref = case.run()
        got = _noalloc(case)
        rows = sample_rows(geo.tokens_per_chunk, 24, seed=seed)
        for i, node in enumerate(wl.pack):
            assert np.all(np.isfinite(got[i])), f"{wl.name} node {node}"
            bf16_gates(got[i], ref[i], f"{wl.name} node {node}: no-alloc vs sc_attention")
            bf16_gates(got[i][rows], case.oracle(i, rows=rows), f"{wl.name} node {node}: vs oracle")


def test_noalloc_without_pieces_is_bitwise():
    """A plan too short to cut (two nodes of 3 and 4 small chunks, 15-20 key
    tiles): the same launch as sc_attention."""
    case = AttnCase(SMALL, sc.SC_DTYPE_BF16, "prog", [(2, 1), (3, 2)], [(0, 0), (1, 0)], seed=43)
    assert sc.sc_attention_workspace_bytes(case.plan, case.cache) == 0
    ref = case.run()
    got = _noalloc(case)
    for i in range(len(case.pack)):
        np.testing.assert_array_equal(got[i], ref[i])


def test_noalloc_rejects_a_stale_plan():
    case = AttnCase(SMALL, sc.SC_DTYPE_BF16, "prog", [(6, 1), (7, 2)], [(c, 0) for c in range(6)], seed=44)
    case.cache.release((0, 0))
    torch = torch_mod()
    with pytest.raises(sc.ScError) as e:
        sc.sc_attention_noalloc(case.plan, case.cache, 0, case.q_dev, torch.empty_like(case.q_dev), case.scale)
    assert e.value.code == sc.SC_ESTALE
