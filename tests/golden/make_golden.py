"""Write tests/golden/worked_examples.json from oracle/exact.py only.

Each case is a tiny token whose eq. (5) codes are computed in exact rational
arithmetic (the sqrt(b) of the normalized rotation cancels in z/delta), so the
stored codes and the stored r*A/q are exact.  Inputs are chosen by hand to pin
specific behaviours; the comment of each case says which.
Run:  python tests/golden/make_golden.py
"""
import json
import os
import sys
from fractions import Fraction

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)
from oracle import exact  # noqa: E402

CASES = [
    # (what it pins, x, b, bits, r as (num, den))
    ("b=4 Sylvester order and signs: H4 [1,2,3,4] = [10,-2,-4,0]", [1, 2, 3, 4], 4, 4, (1, 1)),
    ("b=1 is plain per-token RTN", [0.5, -1.25, 3.0, -2.0], 1, 4, (1, 1)),
    ("two blocks of b=2, absmax taken over the whole token", [1, 1, 4, -4, 0.5, 0.25, -3, 1], 2, 4, (1, 1)),
    ("exact ties round half to even: A=14, ratios k+1/2", [14, 5, 3, 1, -5, -3, -1, 9], 1, 4, (1, 1)),
    ("ties at INT4 with A = 14 after the transform", [7, 7, 1.5, -0.5], 2, 4, (1, 1)),
    ("INT8 codes, b=8", [1, -2, 3, -4, 5, -6, 7, -8], 8, 8, (1, 1)),
    ("clip ratio r=1/2 saturates at +-q", [1, 2, 3, 4, 0, 0, 0, 1], 4, 4, (1, 2)),
    ("zero token gives codes 0 and delta 0", [0, 0, 0, 0], 4, 4, (1, 1)),
    ("negative absmax element maps to -q", [-9, 1, 2, 0.5], 2, 4, (1, 1)),
    ("b=16 single block", [float(i % 5) - 2 for i in range(16)], 16, 4, (1, 1)),
]


def main():
    out = []
    for what, x, b, bits, (rn, rd) in CASES:
        codes, rA_over_q, ratios = exact.quantize_token(x, b, bits, Fraction(rn, rd))
        out.append({
            "pins": what, "x": x, "b": b, "bits": bits, "r": [rn, rd],
            "codes": codes,
            "rA_over_q": [rA_over_q.numerator, rA_over_q.denominator],
            "ratios": [[t.numerator, t.denominator] for t in ratios],
        })
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "worked_examples.json")
    with open(path, "w") as f:
        json.dump({"source": "exact rational eq. (5) with the Sylvester H_b of Sec. III-C "
                             "(oracle/exact.py); written by tests/golden/make_golden.py",
                   "cases": out}, f, indent=1)
    print(path)


if __name__ == "__main__":
    main()
