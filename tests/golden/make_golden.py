"""Writes the stored plan fixtures of tests/golden/ using the oracle only.

Run from the repository root:  python tests/golden/make_golden.py
"""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import plan  # noqa: E402


def main():
    lengths = plan.balanced_plan(131072, 16, 128)
    with open(os.path.join(HERE, "balanced_plan_131072x16_align128.txt"), "w") as f:
        f.write("# Latency-balanced chunk lengths for S=131072, M=16, boundaries on multiples of 128.\n")
        f.write("# Balancing goal: equal causal attention work L_c (P_c + L_c/2) per chunk, i.e. the\n")
        f.write("# attention term of Eq. (1) (Section 3.2) evened out as Section 4.2 intends; boundary\n")
        f.write("# c = S sqrt(c/M) rounded to the nearest multiple of 128.  Written by make_golden.py.\n")
        f.write(" ".join(str(n) for n in lengths) + "\n")


if __name__ == "__main__":
    main()
