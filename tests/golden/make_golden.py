"""Write the exact rational fixture used by the oracle pins.

Calls only ``oracle.exact`` (rational arithmetic, no rounding).  The inputs are
fixed dyadic rationals; the outputs are stored as exact fraction strings.
Run from the repository root:  python tests/golden/make_golden.py
"""
import json
import os
import sys
from fractions import Fraction as Fr

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
from oracle import exact  # noqa: E402

INPUTS = {
    "q": [["1/2", "-1/4", "3/4"], ["0", "1", "-1/2"], ["1/8", "1/8", "-3/4"], ["-1", "1/2", "0"],
          ["3/8", "-5/8", "1/4"]],
    "k": [["1/4", "3/4", "-1/2"], ["-1/2", "0", "1/2"], ["3/4", "-1/4", "1/8"], ["0", "1/2", "1/2"],
          ["-3/8", "1/4", "5/8"]],
    "v": [["1", "-1/2"], ["1/4", "3/4"], ["-3/4", "1/8"], ["1/2", "1/2"], ["-1/8", "-1"]],
    "beta": ["1/2", "3/4", "1/8", "1", "5/8"],
    "lam": ["1/4", "0", "1", "1/2", "7/8"],
    "alpha": ["1", "3/4", "1/2", "7/8", "1/4"],
    "S0": [["1/4", "0", "-1/2"], ["1/8", "1/2", "0"]],
}


def main():
    conv = lambda a: [[Fr(x) for x in row] for row in a]
    o, S = exact.dense_product(conv(INPUTS["q"]), conv(INPUTS["k"]), conv(INPUTS["v"]),
                               [Fr(x) for x in INPUTS["beta"]], [Fr(x) for x in INPUTS["lam"]],
                               [Fr(x) for x in INPUTS["alpha"]], conv(INPUTS["S0"]))
    out = {
        "what": "Q-Delta recurrence (Sec. 3.3, Eq. (qdelta_decay)), T=5, d_k=3, d_v=2, exact rationals",
        "inputs": INPUTS,
        "o": [[str(x) for x in row] for row in o],
        "S_final": [[str(x) for x in row] for row in S],
    }
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "exact_T5_dk3_dv2.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(path)


if __name__ == "__main__":
    main()
