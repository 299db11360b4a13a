"""Writes the stored block-key vectors from the oracle alone.

Run from the repository root:  python tests/golden/make_golden.py
Each line: name, token count, the tokens, then the chained key of every full
block (hex).  The token streams are seeded and synthetic.
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle.prefix_ref import block_digests, chain_keys  # noqa: E402


def cases():
    rng = np.random.default_rng(20250711)
    yield "zeros32", np.zeros(32, np.int32)
    yield "iota48", np.arange(48, dtype=np.int32)
    yield "neg16", -np.arange(1, 17, dtype=np.int32)          # read as u32 words
    yield "extremes16", np.array([0, -1, 2**31 - 1, -2**31] * 4, dtype=np.int32)
    yield "partial40", rng.integers(0, 32000, 40).astype(np.int32)
    for i in range(4):
        n = int(rng.integers(16, 200))
        yield f"rand{i}_{n}", rng.integers(0, 32000, n).astype(np.int32)


def main():
    out = os.path.join(HERE, "chain_keys.txt")
    with open(out, "w") as f:
        f.write("# name n tokens... | digest(hex)... | key(hex)...  (written by make_golden.py)\n")
        for name, toks in cases():
            d = [f"{int(x):016x}" for x in block_digests(toks).tolist()]
            k = [f"{x:016x}" for x in chain_keys(toks)]
            f.write(f"{name} {len(toks)} {' '.join(str(int(t)) for t in toks)} | "
                    f"{' '.join(d)} | {' '.join(k)}\n")
    print("wrote", out)


if __name__ == "__main__":
    main()
