"""Writes block_worked_example.txt: a DiT block worked by hand at hidden 4.

Independent of every other module in this repository: scalar arithmetic with
Python's ``math`` only, one step of the block reading at a time, on weights
chosen so that each intermediate can be checked with a pocket calculator
(matrices of a few nonzero entries, none symmetric where a
transposed projection could hide).  The block reading it follows:

    h  = RMSNorm(x)              x / sqrt(mean(x^2) + 1e-6), unit gain
    q, k, v = h Wq^T, h Wk^T, h Wv^T          (one head of 4 channels)
    q, k rotated by RoPE: channel pairs (0,1) and (2,3) both on the width
         axis (dims 0/0/4), pair i turned by  w * theta^(-2 i / 4),  theta 16,
         so pair 0 turns by w and pair 1 by w / 4
    o  = softmax(q k^T / sqrt(4)) v      over the chunk's own tokens
    x' = x + o Wo^T
    y  = x' + GELU_tanh(RMSNorm(x') Wup^T) Wdown^T,
         GELU_tanh(u) = u/2 (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3)))

Run:  python tests/golden/make_block_worked_example.py
"""
import math
import os

EPS = 1e-6
THETA = 16.0

W_Q = [[1, 0.5, 0, 0], [0, 1, 0, 0], [0, 0, 1, 0], [0, 0, 0, 1]]
W_K = [[1, 0, 0, 0], [0, -1, 0, 0], [0, 0, 1, 0], [0, 0, 0, 1]]
W_V = [[0, 1, 0, 0], [0, 0, 1, 0], [0, 0, 0, 1], [1, 0, 0, 0]]
W_O = [[0.5, 0, 0, 0], [0, 0.5, 0, 0], [0, 0, 0.5, 0.25], [0, 0, 0, 0.5]]
W_UP = [[1, 0, 0, 0], [0, 0, 0, 1]]
W_DOWN = [[1, 0], [0, 1], [1, 1], [0, -1]]

CASES = {
    # one token (grid 1 x 1): attention over a single key returns its value
    "one_token": [[0.5, -1.0, 1.5, -2.0]],
    # two tokens of one frame (grid 1 x 2, widths 0 and 1)
    "two_tokens": [[1.0, 0.5, -0.5, 2.0], [-1.5, 1.0, 0.25, 0.5]],
}


def rmsnorm(v):
    r = math.sqrt(sum(a * a for a in v) / len(v) + EPS)
    return [a / r for a in v]


def apply(W, v):  # W in [out, in] layout: (v W^T)[r] = sum_c W[r][c] v[c]
    return [sum(W[r][c] * v[c] for c in range(len(v))) for r in range(len(W))]


def rotate(v, w):
    out = list(v)
    for p in range(2):
        ang = w * THETA ** (-2.0 * p / 4.0)
        c, s = math.cos(ang), math.sin(ang)
        out[2 * p] = v[2 * p] * c - v[2 * p + 1] * s
        out[2 * p + 1] = v[2 * p] * s + v[2 * p + 1] * c
    return out


def gelu(u):
    return 0.5 * u * (1.0 + math.tanh(math.sqrt(2.0 / math.pi) * (u + 0.044715 * u ** 3)))


def block(xs):
    hs = [rmsnorm(x) for x in xs]
    qs = [rotate(apply(W_Q, h), w) for w, h in enumerate(hs)]
    ks = [rotate(apply(W_K, h), w) for w, h in enumerate(hs)]
    vs = [apply(W_V, h) for h in hs]
    steps = {"h": hs, "q": qs, "k": ks, "v": vs, "o": [], "x1": [], "h2": [], "u": [], "g": [], "y": []}
    for i, x in enumerate(xs):
        s = [sum(a * b for a, b in zip(qs[i], k)) / 2.0 for k in ks]
        m = max(s)
        e = [math.exp(a - m) for a in s]
        z = sum(e)
        o = [sum(e[j] / z * vs[j][d] for j in range(len(xs))) for d in range(4)]
        x1 = [a + b for a, b in zip(x, apply(W_O, o))]
        h2 = rmsnorm(x1)
        u = apply(W_UP, h2)
        g = [gelu(a) for a in u]
        y = [a + b for a, b in zip(x1, apply(W_DOWN, g))]
        for name, val in (("o", o), ("x1", x1), ("h2", h2), ("u", u), ("g", g), ("y", y)):
            steps[name].append(val)
    return steps


def main():
    lines = [
        "# DiT block worked at hidden 4 (one head of 4 channels, MLP width 2),",
        "# written by tests/golden/make_block_worked_example.py with scalar",
        "# arithmetic only (no other module of this repository).  One node, chunk 0,",
        "# one latent frame, no history (W = 0); RoPE dims (0, 0, 4), theta 16;",
        "# RMSNorm eps 1e-6.  Weights in [out, in] layout:",
        "#   Wq = I plus 0.5 at row 0, column 1;  Wk = diag(1, -1, 1, 1);",
        "#   Wv rows (0,1,0,0), (0,0,1,0), (0,0,0,1), (1,0,0,0) (v = (h1, h2, h3, h0));",
        "#   Wo = I / 2 plus 0.25 at row 2, column 3;  Wup rows (1,0,0,0), (0,0,0,1);  Wdown rows (1,0), (0,1), (1,1), (0,-1).",
        "# Steps per token: h = RMSNorm(x); q = RoPE(h Wq^T); k = RoPE(h Wk^T); v = h Wv^T;",
        "# o = softmax(q k^T / 2) v; x1 = x + o Wo^T; h2 = RMSNorm(x1); u = h2 Wup^T;",
        "# g = GELU_tanh(u); y = x1 + g Wdown^T.  Token n of the chunk sits at width n,",
        "# so token 1's pair 0 turns by 1 rad and its pair 1 by 16^(-1/2) = 1/4 rad.",
        "# Lines: case name step token : values",
    ]
    for name, xs in CASES.items():
        steps = block(xs)
        for t, x in enumerate(xs):
            lines.append(f"{name} x {t} : " + " ".join(repr(float(a)) for a in x))
        for step in ("h", "q", "k", "v", "o", "x1", "h2", "u", "g", "y"):
            for t, val in enumerate(steps[step]):
                lines.append(f"{name} {step} {t} : " + " ".join(f"{a:.17g}" for a in val))
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "block_worked_example.txt")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {path}")


if __name__ == "__main__":
    main()
