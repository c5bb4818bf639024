"""Writes the known-answer vectors of the garbling hash and PRG
(hash_kat.txt, prg_kat.txt) from the CPU oracle alone.

    python tests/golden/make_hash_kat.py

The paper fixes no hash (Sec. 2.3 projection gates), so these values are the
oracle's; tests/test_oracle_spec.py checks each of them against a second
statement of the construction on libcrypto's AES, and the GPU tests check the
library's hash against them.  Inputs are drawn from a fixed seed and cover
output modulus 2 (one AES block), odd and power-of-two moduli (two blocks),
labels of 4 to 6 packed words, gadget ids with the top bit set and tweaks at
and above 2^32, 2^62 and 2^63.
"""

from __future__ import annotations

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import oracle as O  # noqa: E402

PAIRS = [(2, 37), (37, 2), (3, 5), (5, 3), (11, 13), (17, 19), (37, 31), (2, 3), (4, 16), (32, 167),
         (167, 32), (97, 251), (251, 97), (128, 7), (8, 19), (2, 2)]
TAUS = [0, 1, 77, 2 ** 31 - 1, 2 ** 32, 2 ** 32 + 5, 3 * 2 ** 40 + 11, 2 ** 62 - 1, 2 ** 62, 2 ** 63 + 3]
GIDS = [0, 3, 0x80000001, 0xFFFFFFFF]


def hash_lines():
    rng = np.random.default_rng(20250617)
    lines = []
    for q, m in PAIRS:
        for tau in TAUS[: 4 if (q, m) != (3, 5) else len(TAUS)] + [TAUS[4], TAUS[8], TAUS[9]]:
            gid = GIDS[int(rng.integers(0, len(GIDS)))]
            res = rng.integers(0, q, size=O.lam(q)).astype(np.uint32)
            words = O.pk32_pack(q, res)
            out = O.pk32_pack(m, O.hash_label(q, m, res, gid, tau))
            lines.append(f"{q} {m} {gid:#010x} {tau} " + ",".join(f"{int(w):08x}" for w in words) + " "
                         + ",".join(f"{int(w):08x}" for w in out))
    return sorted(set(lines), key=lines.index)


def prg_lines():
    lines = []
    for seed in (0, 3, 2 ** 40 + 7, 2 ** 64 - 1):
        for stream in (1, 2):
            for idx in (0, 1, 2 ** 31 - 1, 2 ** 31, 2 ** 32 + 3, 2 ** 62 + 9, 2 ** 63 + 1):
                V = O.prg_value(seed, stream, idx)
                lines.append(f"{seed} {stream} {idx} " + ",".join(f"{int(v):08x}" for v in V))
    return lines


def main():
    head = ("# {what}: written by tests/golden/make_hash_kat.py from the CPU oracle.\n"
            "# The paper fixes no hash or PRG (Sec. 2.3); see tests/rspec.py for the construction.\n")
    with open(os.path.join(HERE, "hash_kat.txt"), "w") as f:
        f.write(head.format(what="projection-gate hash H_m(A, tau)"))
        f.write("# q m gadget_id tau PK32(A) words (hex, word 0 first) PK32(H) words\n")
        f.write("\n".join(hash_lines()) + "\n")
    with open(os.path.join(HERE, "prg_kat.txt"), "w") as f:
        f.write(head.format(what="garbler PRG rho(stream, idx)"))
        f.write("# seed stream idx V as 8 little-endian 32-bit limbs (hex, limb 0 first)\n")
        f.write("\n".join(prg_lines()) + "\n")


if __name__ == "__main__":
    main()
