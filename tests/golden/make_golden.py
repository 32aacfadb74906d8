"""Writes tests/golden/case3_masks.txt from oracle/ only: Case-III keep masks
(Sec. 3.1; generator, counter layout and exact threshold as read in R5) for a
few (seed, step, stream, rate) cases, one row of 0/1 per time step, and the
first four 64-bit words of each case in hex.  The paper prints no worked
example of the computation, so this file is a frozen draw: a change to the
generator or its counter layout shows up as a mismatch.

    python -m tests.golden.make_golden
"""
import os

from oracle import masks as om

CASES = [  # seed, step, stream, T, K, p
    (12345, 3, 6, 4, 40, 0.5),
    (1, 0, 0, 3, 17, 0.3),
    (2**63 + 7, 11, 4, 2, 9, 0.9),
]

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "case3_masks.txt")


def render():
    lines = ["# Case-III keep masks (Sec. 3.1; generator reading R5), written by",
             "# tests/golden/make_golden.py from oracle/masks.py.",
             "# case: seed step stream T K p; then words: first 4 uniform words of t = 0 (hex);",
             "# then T rows of K bits (1 = kept)."]
    for seed, step, stream, T, K, p in CASES:
        lines.append(f"case {seed} {step} {stream} {T} {K} {p!r}")
        u = om.uniform_words(seed, step, stream, T, K)
        lines.append("words " + " ".join(f"{int(w):016x}" for w in u[0, :4]))
        m = om.keep_mask(seed, step, stream, T, K, p)
        for t in range(T):
            lines.append("".join(str(int(v)) for v in m[t]))
    return "\n".join(lines) + "\n"


if __name__ == "__main__":
    with open(OUT, "w") as f:
        f.write(render())
    print("wrote", OUT)
