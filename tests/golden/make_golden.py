"""Write tests/golden/hash_vectors.txt from the CPU oracle alone.

The vectors freeze the oracle's chained prefix hash (a definition of this
library: the paper reuses LMCache's lookup and prints no hash values).  Rerun
only when the hash definition itself changes, and say why in the commit.

    python tests/golden/make_golden.py
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
import oracle  # noqa: E402


def cases():
    rng = np.random.default_rng(20260)
    yield "empty", [], 0
    yield "fifteen_tokens_no_block", list(range(15)), 0
    yield "sixteen_zeros", [0] * 16, 0
    yield "zero_to_fifteen", list(range(16)), 0
    yield "zero_to_fifteen_seed1", list(range(16)), 1
    yield "ramp_33_seed_max", list(range(100, 133)), (1 << 64) - 1
    yield "max_id_64", [31999] * 64, 0
    yield "negative_words", [-1, -2, 0x7FFFFFFF, -0x80000000] * 4, 0
    yield "random_256", [int(t) for t in rng.integers(0, 32000, 256)], 0x5EED
    yield "random_300_seed", [int(t) for t in rng.integers(0, 32000, 300)], 42


def main():
    out = os.path.join(HERE, "hash_vectors.txt")
    with open(out, "w") as f:
        f.write("# Chained prefix hash golden vectors, written by make_golden.py from the oracle.\n")
        f.write("# h_{-1} = seed; h_b = M(h_{b-1} ^ d_b ^ 0x9E3779B97F4A7C15);\n")
        f.write("# d_b = sum_j M(uint32(tok[16b+j]) + ((j+1) << 32)); M = SplitMix64 finalizer.\n")
        for name, toks, seed in cases():
            t = np.array(toks, np.int64).astype(np.int32)
            h = oracle.hash_prefix(t, np.array([0, t.size], np.int64), seed)
            f.write(f"case={name}\n")
            f.write(f"seed={seed:#x}\n")
            f.write("tokens=" + " ".join(str(int(x)) for x in t) + "\n")
            f.write("hashes=" + " ".join(f"{int(x):016x}" for x in h) + "\n\n")
    print("wrote", out)


if __name__ == "__main__":
    main()
