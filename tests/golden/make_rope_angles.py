"""Writes rope_angles.txt: rotation angles of single RoPE channel pairs.

The 3D RoPE reading of the Wan-shaped workload: head_dim 128 split into
44 / 42 / 42 channels for the (t, h, w) axes, interleaved pairs, pair i of
axis a turned by pos_a * theta^(-2 i / d_a) with theta = 10000.  Pair i of
axis a is channel pair p = (sum of the earlier axes' d / 2) + i.  Scalar
arithmetic with Python's ``math`` only; angles are reduced to [0, 2 pi).

Run:  python tests/golden/make_rope_angles.py
"""
import math
import os

DIMS = (44, 42, 42)
THETA = 10000.0
POSITIONS = [(7, 13, 29), (20, 1, 51)]


def main():
    lines = [
        "# 3D RoPE, head_dim 128 = 44 (t) + 42 (h) + 42 (w) channels, theta 10000;",
        "# pair i of axis a is turned by pos_a * 10000^(-2 i / d_a), reduced to [0, 2 pi).",
        "# Written by tests/golden/make_rope_angles.py (scalar arithmetic only).",
        "# Example: 10000^(-2/44) = exp(-ln(10000) / 22) = 0.6579332246575682, so pair 1",
        "# of the time axis at t = 7 turns by 7 * 0.65793... = 4.6055 rad.",
        "# Lines: t h w axis i pair angle",
    ]
    for pos in POSITIONS:
        off = 0
        for a, d in enumerate(DIMS):
            for i in sorted({0, 1, 2, d // 2 - 1}):
                ang = math.fmod(pos[a] * THETA ** (-2.0 * i / d), 2.0 * math.pi)
                lines.append(f"{pos[0]} {pos[1]} {pos[2]} {a} {i} {off + i} {ang:.17g}")
            off += d // 2
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "rope_angles.txt")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {path}")


if __name__ == "__main__":
    main()
