"""Oracle pins against hand-worked values (CPU only).

* ``golden/block_worked_example.txt``: a DiT block at hidden 4 with
  few-entry, non-symmetric weights, every intermediate listed (written by
  ``golden/make_block_worked_example.py`` with scalar arithmetic, independent
  of the oracle).  It fixes the use of each piece of the block reading inside
  the block: the pre-attention and pre-MLP RMSNorms, the tanh GELU between
  the MLP projections, the residual additions, the attention over the
  chunk's own tokens, and RoPE on q and k with a non-unit frequency.
* ``golden/rope_angles.txt``: the angle by which single channel pairs turn
  at given (t, h, w) positions for the Wan split 44 / 42 / 42, theta 10000,
  pairs 0, 1, 2 and the last of each axis -- the frequency table
  pos * theta^(-2 i / d_a) and the pair-to-axis assignment.
* ``golden/input_times_k4.txt``: the four denoising input times as the
  paper's training configuration table prints them, per level, for the
  sampler's schedule in the oracle and in bench.py's workloads.
"""
import math
import os

import numpy as np
import pytest

from oracle.block import BlockShape, block_forward, project_kv, project_q, rmsnorm
from oracle.policy import policy, select
from oracle.rope import rope

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _read_block_golden():
    vals = {}
    with open(os.path.join(GOLDEN, "block_worked_example.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            head, nums = line.split(":")
            case, step, tok = head.split()
            vals.setdefault(case, {}).setdefault(step, {})[int(tok)] = np.array(
                [float(v) for v in nums.split()])
    return vals


def _weights():
    w_q = np.eye(4)
    w_q[0, 1] = 0.5
    w_k = np.diag([1.0, -1.0, 1.0, 1.0])
    w_v = np.array([[0, 1, 0, 0], [0, 0, 1, 0], [0, 0, 0, 1], [1, 0, 0, 0]], dtype=np.float64)
    return {"w_qkv": np.concatenate([w_q, w_k, w_v]),
            "w_o": 0.5 * np.eye(4) + 0.25 * np.eye(4, k=1) * (np.arange(4) == 2)[:, None],
            "w_up": np.array([[1, 0, 0, 0], [0, 0, 0, 1]], dtype=np.float64),
            "w_down": np.array([[1, 0], [0, 1], [1, 1], [0, -1]], dtype=np.float64)}


@pytest.mark.parametrize("case", ["one_token", "two_tokens"])
def test_block_worked_example(case):
    g = _read_block_golden()[case]
    n = len(g["x"])
    shp = BlockShape(hidden=4, heads=1, head_dim=4, mlp=2, frames_per_chunk=1, grid_h=1, grid_w=n,
                     rope_dims=(0, 0, 4), theta=16.0)
    x = np.stack([g["x"][t] for t in range(n)])
    w = _weights()
    want = lambda step: np.stack([g[step][t] for t in range(n)])
    np.testing.assert_allclose(rmsnorm(x), want("h"), rtol=1e-14, atol=1e-15)
    q = project_q(x, 0, w["w_qkv"], shp)[:, 0, :]
    k, v = project_kv(x, 0, w["w_qkv"], shp)
    np.testing.assert_allclose(q, want("q"), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(k[:, 0, :], want("k"), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(v[:, 0, :], want("v"), rtol=1e-13, atol=1e-15)
    sel = select(policy("clean", 4, 0), [(0, 4)])
    y, new_kv = block_forward(sel, lambda i: x, w, None, shp)
    np.testing.assert_allclose(y[0], want("y"), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(new_kv[0][0][:, 0, :], want("k"), rtol=1e-13, atol=1e-15)


def test_block_worked_example_has_teeth():
    """The worked example separates the block from its near misses: ReLU
    for GELU, a missing pre-MLP RMSNorm, or a missing residual change y by
    far more than the comparison tolerance."""
    g = _read_block_golden()["one_token"]
    y = g["y"][0]
    x1, h2, u = g["x1"][0], g["h2"][0], g["u"][0]
    w = _weights()
    relu = x1 + w["w_down"] @ np.maximum(u, 0.0)
    no_norm = x1 + w["w_down"] @ np.array([0.5 * a * (1 + math.tanh(math.sqrt(2 / math.pi) * (a + 0.044715 * a ** 3)))
                                            for a in w["w_up"] @ x1])
    no_resid = w["w_down"] @ g["g"][0]
    for near in (relu, no_norm, no_resid):
        assert np.abs(near - y).max() > 1e-3            # the comparison tolerance is 1e-13
    assert u[0] > 0 > u[1]                                 # GELU sees both signs
    assert not np.allclose(h2, x1)


def _read_rope_golden():
    rows = []
    with open(os.path.join(GOLDEN, "rope_angles.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            t, h, w, a, i, p, ang = line.split()
            rows.append(((int(t), int(h), int(w)), int(a), int(i), int(p), float(ang)))
    return rows


def test_rope_pair_angles_match_the_hand_table():
    rows = _read_rope_golden()
    assert len(rows) == 24
    for pos, a, i, p, ang in rows:
        x = np.zeros((1, 1, 128))
        x[0, 0, 2 * p] = 1.0                               # the pair's real unit vector
        y = rope(x, np.array([pos]), (44, 42, 42), 10000.0)[0, 0]
        got = math.atan2(y[2 * p + 1], y[2 * p]) % (2 * math.pi)
        diff = (got - ang) % (2 * math.pi)
        assert min(diff, 2 * math.pi - diff) < 1e-9, (pos, a, i, got, ang)
        others = np.delete(y, [2 * p, 2 * p + 1])
        assert np.all(others == 0.0)                       # a rotation stays in its pair


def test_input_times_match_paper_table():
    """t_j of levels 0..4: the oracle's schedule and bench.py's, exactly."""
    from fractions import Fraction

    import bench
    from oracle.pipeline import T_SCHEDULE_K4

    want = {}
    with open(os.path.join(GOLDEN, "input_times_k4.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            level, num, den = (int(v) for v in line.split())
            want[level] = Fraction(num, den)
    assert sorted(want) == [0, 1, 2, 3, 4]
    for sched in (T_SCHEDULE_K4, bench.T_SCHEDULE_K4):
        assert len(sched) == 5
        for level, t in want.items():
            assert sched[level] == float(t), (level, sched[level], t)
