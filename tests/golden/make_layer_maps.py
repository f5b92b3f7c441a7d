"""Writes layer_maps.txt: the target->source layer maps of the two
cross-family workloads, enumerated with exact rational arithmetic
(fractions.Fraction), independently of the integer formulas the input
generator uses.

* Qwen2.5-1.5B (28 layers) -> Gemma-2-2B (26 layers): target layer l reads
  source layer round(l * 27/25).
* Llama3.1-70B (80 layers) -> Qwen2.5-7B (28 layers): target layer l mixes the
  3 consecutive source layers starting at floor(l * 80/28).
"""
import math
import os
from fractions import Fraction


def main():
    rows = []
    m3 = []
    for l in range(26):
        q = Fraction(27 * l, 25)
        lo = math.floor(q)
        assert q - lo != Fraction(1, 2), "tie"
        m3.append(lo + (1 if q - lo > Fraction(1, 2) else 0))
    rows.append("qwen1.5b_to_gemma2b " + " ".join(map(str, m3)))
    m5 = [math.floor(Fraction(80 * l, 28)) for l in range(28)]
    rows.append("llama70b_to_qwen7b_window_start " + " ".join(map(str, m5)))
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "layer_maps.txt")
    with open(path, "w") as f:
        f.write("# written by make_layer_maps.py (exact rational arithmetic)\n")
        f.write("\n".join(rows) + "\n")


if __name__ == "__main__":
    main()
