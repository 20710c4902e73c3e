"""Writes the stored expected values under tests/golden/ (calls only oracle/).

primes.txt: for each parameter set used by the workloads (log2 N, L, K), the
L+K primes the oracle selects (largest 50-bit primes = 1 mod 2N, descending).
tests/test_oracle_pins.py checks them by trial division and maximality.
"""
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
from oracle import ckks  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))

if __name__ == "__main__":
    with open(os.path.join(HERE, "primes.txt"), "w") as f:
        f.write("# logN L K primes(hex) -- written by tests/golden/make_golden.py\n")
        for logn, L, K in [(13, 3, 1), (15, 8, 2), (16, 12, 3)]:
            ps = ckks.find_primes(logn, L + K)
            f.write(f"{logn} {L} {K} " + " ".join(hex(p) for p in ps) + "\n")
