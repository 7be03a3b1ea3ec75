"""Writes pch64_vectors.txt: PCH64 keys of seeded token sequences.

Calls only the oracle.  Token ids span the full int32 range so that the
uint32 reinterpretation and the mod-2^32 factor wrap are both exercised.
Run from the repository root:  python tests/golden/make_golden.py
"""
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
import oracle  # noqa: E402

CASES = [(0, 11, 16), (1, 12, 47), (7, 13, 160), (63, 14, 100), (4294967295, 15, 64)]

out = os.path.join(os.path.dirname(os.path.abspath(__file__)), "pch64_vectors.txt")
with open(out, "w") as f:
    f.write("# ns seed n_tokens key_0 key_1 ... (hex); tokens = PCG64(seed).integers(-2^31, 2^31, n)\n")
    for ns, seed, L in CASES:
        toks = np.random.Generator(np.random.PCG64(seed)).integers(-2**31, 2**31, L, dtype=np.int64).astype(np.int32)
        keys = oracle.hash_request(toks, ns)
        f.write(f"{ns} {seed} {L} " + " ".join(f"{int(k):016x}" for k in keys) + "\n")
print("wrote", out)
