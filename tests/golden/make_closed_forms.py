"""Write closed_forms.json: exact expected values derived by hand, in rationals.

Uses only ``fractions``; calls neither the oracle nor the GPU path.

1. Selection with all-zero keys (Alg. 2 "sparsify", cumulative attention
   weight of Sec. 3.4).  Every logit is 0, so observation row i (position
   L-W+i) spreads weight 1/(L-W+i+1) uniformly over keys 0..L-W+i, and each
   of the G heads of a KV head adds the same amount.  All prefix scores are
   equal, so the lowest-position tie rule keeps prefix positions 0..B-W-1.
2. Greedy acceptance (Eq. 3, Alg. 2): hand-made logit rows with ties; the
   greedy token is the lowest index among equal maxima.
"""
import json
import os
from fractions import Fraction


def zero_key_scores(L, W, G):
    raw = [Fraction(0)] * L
    for i in range(W):
        p = L - W + i
        for t in range(p + 1):
            raw[t] += Fraction(G, p + 1)
    return raw


def main():
    L, W, G, B = 12, 3, 2, 7
    raw = zero_key_scores(L, W, G)
    sel = list(range(B - W)) + list(range(L - W, L))
    accept = {
        "gamma": 3,
        "logits": [[0.5, 2.0, 2.0, -1.0], [3.0, 1.0, 3.0, 3.0], [0.0, -0.0, -2.0, -5.0], [1.0, 1.0, 1.0, 4.0]],
        "draft": [1, 0, 1],
        "argmax": [1, 0, 0, 3],
        "accept": 2,
        "bonus": 0,
    }
    data = {
        "select_zero_keys": {"L": L, "W": W, "G": G, "B": B,
                             "raw_num_den": [[f.numerator, f.denominator] for f in raw], "idx": sel},
        "accept_worked": accept,
    }
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "closed_forms.json"), "w") as f:
        json.dump(data, f, indent=1)


if __name__ == "__main__":
    main()
