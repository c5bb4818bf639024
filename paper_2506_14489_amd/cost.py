"""Work model of one scaling-gadget instance, used to report throughput
against hardware roofs.

Per gadget (structure of the gate list in include/redash.h):
  * algorithmic HBM bytes: the k input labels and k output labels (packed
    words) plus, per projection gate q -> m, one W_m-word row, read with
    probability (q-1)/q because the colour-0 row is implicit (row reduction);
  * AES-128 blocks: two per gate, one when the output modulus is 2;
  * algorithmic 32-bit integer (vector ALU) operations of the table
    formulation:
      - per AES block: 10 rounds x 16 lookups, each an index extraction and
        one XOR (the 16 XORs of a round combine 4 table words and the round
        key per column; the table reads themselves are LDS reads, counted
        separately below), + 4 initial key XORs = 324, plus 12 XORs for the
        tweak and the feed-forward;
      - per gate: W_q + 1 for folding the input label and sigma;
      - per output word (m > 2): 8 limb multiply-adds of 4 operations each;
      - per output residue (m > 2): 14 (digit split 3, row add 3, free
        operation 5, field extract and insert 3); per word for m = 2: 3;
  * LDS table reads: 160 4-byte lookups per AES block (T-table AES).
"""

from __future__ import annotations

AES_OPS_PER_BLOCK = 10 * 16 * 2 + 4 + 12
AES_LOOKUPS_PER_BLOCK = 10 * 16
LIMB_OPS_PER_WORD = 8 * 4
OPS_PER_RESIDUE = 14


def lam(m: int) -> int:
    """Residues per label: least lambda with m^lambda >= 2^128."""
    v, lam_ = 1, 0
    while v < (1 << 128):
        v *= m
        lam_ += 1
    return lam_


def words(m: int) -> int:
    b = (m - 1).bit_length()
    g = 32 // b
    return -(-lam(m) // g)


def gates(moduli, scale_idx):
    """(q, m) per gate in gate order."""
    S = sorted(scale_idx)
    R = [i for i in range(len(moduli)) if i not in S]
    out = []
    for a, si in enumerate(S):
        for dst in S[a + 1:] + R:
            out.append((moduli[si], moduli[dst]))
    for b, ri in enumerate(R):
        for dst in R[b + 1:] + S:
            out.append((moduli[ri], moduli[dst]))
    return out


def bytes_per_gadget(moduli, scale_idx) -> float:
    labels = 2 * sum(4 * words(m) for m in moduli)
    rows = sum((q - 1) / q * 4 * words(m) for (q, m) in gates(moduli, scale_idx))
    return labels + rows


def aes_blocks_per_gadget(moduli, scale_idx) -> int:
    return sum(1 if m == 2 else 2 for (_q, m) in gates(moduli, scale_idx))


def ops_per_gadget(moduli, scale_idx) -> int:
    total = 0
    for (q, m) in gates(moduli, scale_idx):
        total += (1 if m == 2 else 2) * AES_OPS_PER_BLOCK + words(q) + 1
        if m == 2:
            total += 3 * words(m)
        else:
            total += LIMB_OPS_PER_WORD * words(m) + OPS_PER_RESIDUE * lam(m)
    return total


def lds_bytes_per_gadget(moduli, scale_idx) -> int:
    """Bytes of AES round-table reads per gadget (4-byte lookups)."""
    return 4 * AES_LOOKUPS_PER_BLOCK * aes_blocks_per_gadget(moduli, scale_idx)


def table_bytes_per_gadget(moduli, scale_idx) -> int:
    return sum((q - 1) * 4 * words(m) for (q, m) in gates(moduli, scale_idx))


# ---------------------------------------------------------------------------
# Garbler (offline phase), per gadget instance:
#   * AES-128 blocks: 2 per modulus for the input zero-label (PRG), and per
#     gate q -> m one hash of each of the q input values (2 blocks, or 1 when
#     m = 2);
#   * HBM bytes written: the garbled rows, (q-1) W_m words per gate, plus
#     the input and output zero-labels;
#   * 32-bit vector-ALU operations: the AES work, per hash the fold and
#     sigma (W_q + 1), per hashed value the pad (32 per output word for the
#     limb multiply-adds when m > 2, 3 per word when m = 2) and the row or
#     zero-label residues (OPS_PER_RESIDUE each), per value the step
#     A_v -> A_v + R_q of the input label (3 per input residue), and per
#     modulus the zero-label digits (32 per word + 3 per residue).
# ---------------------------------------------------------------------------
def garble_aes_blocks_per_gadget(moduli, scale_idx) -> int:
    return 2 * len(moduli) + sum(q * (1 if m == 2 else 2) for (q, m) in gates(moduli, scale_idx))


def garble_bytes_per_gadget(moduli, scale_idx) -> int:
    return table_bytes_per_gadget(moduli, scale_idx) + 2 * sum(4 * words(m) for m in moduli)


def garble_ops_per_gadget(moduli, scale_idx) -> int:
    total = 2 * len(moduli) * AES_OPS_PER_BLOCK
    total += sum(LIMB_OPS_PER_WORD * words(m) + 3 * lam(m) for m in moduli)
    for (q, m) in gates(moduli, scale_idx):
        per_value = (1 if m == 2 else 2) * AES_OPS_PER_BLOCK + words(q) + 1 + 3 * lam(q)
        if m == 2:
            per_value += 3 * words(m)
        else:
            per_value += LIMB_OPS_PER_WORD * words(m) + OPS_PER_RESIDUE * lam(m)
        total += q * per_value
    return total


# ---------------------------------------------------------------------------
# Garbled linear layer (Y = sum w X on every residue), per output activation:
#   * int8 matrix-core operations: 2 per multiply-add, c_in kh kw of them for
#     each residue of each of the k labels: 2 c_in kh kw sum_m lambda_m;
#   * algorithmic HBM bytes per launch: the input labels read once and the
#     output labels written once, 4 sum_m W_m bytes per activation each (the
#     prepared weights, under 0.5 MB for a 3x3x64x64 layer, are left out).
# ---------------------------------------------------------------------------
def linear_ops_per_output(moduli, c_in: int, kh: int, kw: int) -> int:
    return 2 * c_in * kh * kw * sum(lam(m) for m in moduli)


def linear_bytes(moduli, n_in: int, n_out: int) -> int:
    return 4 * sum(words(m) for m in moduli) * (n_in + n_out)
