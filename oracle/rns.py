"""Value-level residue arithmetic of the ReDASH scaling gadget.

TEST INFRASTRUCTURE (oracle).  Only ``tests/``, ``__graft_entry__.smoke()``
and ``bench.py``'s CPU-baseline leg may import this module.  The product
path (the HIP library and its binding) never does.

Everything here is plain Python on Python integers and follows the paper's
definitions one step at a time:

* residue number system, cardinality and CPM           -- Sec. 2.2
* associated mixed-radix system                         -- Sec. 2.2
* signed encoding into Z_P                              -- Sec. 2.4
* scaling y = floor(x / s) as a remainder-zero division -- Sec. 3.2
* per-residue exact division by a base modulus          -- Sec. 3.2 (display eq.)
* generalized base extension via RNS->MRS conversion    -- Sec. 3.3, Eq. (rns_to_mrs)
* the four-step scaling gadget (ShiftUp, scale, BE,
  ShiftDown)                                            -- Sec. 3.4, Table 1
* extension by several moduli (scale by a product)      -- Sec. 3.4 (closing paragraph)

Readings where the paper is silent or misprinted are marked "READING" and
listed in the design notes of the repository.
"""

from __future__ import annotations

from dataclasses import dataclass


# ---------------------------------------------------------------------------
# Sec. 2.2 -- number systems
# ---------------------------------------------------------------------------

def is_prime(n: int) -> bool:
    if n < 2:
        return False
    d = 2
    while d * d <= n:
        if n % d == 0:
            return False
        d += 1
    return True


def first_primes(k: int) -> list[int]:
    """The first k primes; their product is the k-th CPM (Sec. 2.2)."""
    out, n = [], 2
    while len(out) < k:
        if is_prime(n):
            out.append(n)
        n += 1
    return out


def cardinality(base) -> int:
    """P_k = prod p_i (Sec. 2.2)."""
    P = 1
    for m in base:
        P *= m
    return P


def inv_mod(a: int, m: int) -> int:
    """Multiplicative inverse of a modulo m, found by exhaustive search."""
    a %= m
    for x in range(1, m):
        if (a * x) % m == 1:
            return x
    raise ValueError(f"{a} has no inverse mod {m}")


def rns(x: int, base) -> list[int]:
    """x -> ([x]_1, ..., [x]_k) with [x]_i = x mod p_i (Sec. 2.2)."""
    return [x % m for m in base]


def crt(residues, base) -> int:
    """The unique y in [0, P) with y = r_i (mod p_i), found by building y one
    modulus at a time and searching the single free coefficient."""
    y, M = 0, 1
    for r, m in zip(residues, base):
        for t in range(m):
            if (y + t * M) % m == r % m:
                y += t * M
                break
        else:  # pragma: no cover - coprime base always succeeds
            raise ValueError("base not pairwise coprime")
        M *= m
    return y


def mrs_digits(y: int, radices) -> list[int]:
    """Digits of the associated mixed-radix system (Sec. 2.2):
    y = d_1 + d_2 r_1 + d_3 r_1 r_2 + ..., with 0 <= d_i < r_i."""
    out = []
    for r in radices:
        out.append(y % r)
        y //= r
    if y:
        raise ValueError("value exceeds the MRS cardinality")
    return out


def mrs_value(digits, radices) -> int:
    y, w = 0, 1
    for d, r in zip(digits, radices):
        y += d * w
        w *= r
    return y


# ---------------------------------------------------------------------------
# Sec. 2.4 -- signed encoding
# ---------------------------------------------------------------------------

def signed_encode(x: int, P: int) -> int:
    """Positives to the lower half of Z_P, negatives to the upper half."""
    return x % P


def signed_decode(v: int, P: int) -> int:
    """Inverse of the signed encoding.  READING: the representable range is
    [-floor(P/2), ceil(P/2) - 1]; for the paper's P=5 example this gives
    (0,1,2,-2,-1) and for Table 1's P=6 it maps 3 to -3."""
    v %= P
    half_up = (P + 1) // 2
    return v if v < half_up else v - P


# ---------------------------------------------------------------------------
# Sec. 3.2 -- scaling by a base modulus (per-residue exact division)
# ---------------------------------------------------------------------------

def scale_residues(res, base, q_idx):
    """[y]_i = ([x]_i - [x]_q) * p_q^{-1} mod p_i for every i != q.

    The slot of the divisor itself is not defined by this equation; it is
    returned as 0, matching the paper's y' = ([y]_1, ..., [y]_{k-1}, 0)."""
    q = base[q_idx]
    d = res[q_idx]
    out = []
    for i, m in enumerate(base):
        if i == q_idx:
            out.append(0)
        else:
            out.append(((res[i] - d) * inv_mod(q, m)) % m)
    return out


# ---------------------------------------------------------------------------
# Sec. 3.3 -- generalized base extension
# ---------------------------------------------------------------------------

def be_recursion(y_prime, base):
    """Eq. (rns_to_mrs): z_1 = y', z_i[j] = (z_{i-1}[j] - z_{i-1}[i-1]) p_{i-1}^{-1} mod p_j,
    d_i = z_i[i].  Returns (digits d_1..d_k, list of z vectors z_1..z_k).
    Indices here are 0-based: z[0] is the paper's z_1."""
    k = len(base)
    z = [list(y_prime)]
    for i in range(1, k):
        prev = z[-1]
        p = base[i - 1]
        cur = []
        for j in range(k):
            if j < i:
                cur.append(None)  # not defined by the recursion
            else:
                cur.append(((prev[j] - prev[i - 1]) * inv_mod(p, base[j])) % base[j])
        z.append(cur)
    digits = [z[i][i] for i in range(k)]
    return digits, z


def be_missing_residue_printed(y_prime, base):
    """The missing residue exactly as printed after Eq. (rns_to_mrs):
    [y]_k = -(prod_{i<k} p_i)^{-1} * [z_{k-1}]_k mod p_k.
    Kept only so that a test can document that it disagrees with Table 1."""
    k = len(base)
    _, z = be_recursion(y_prime, base)
    pk = base[-1]
    Pk1 = cardinality(base[:-1])
    return (-inv_mod(Pk1, pk) * z[k - 2][k - 1]) % pk


def be_missing_residue(y_prime, base):
    """READING of the missing-residue formula: since y < P_{k-1} its top MRS
    digit is zero, so [y]_k = sum_{i<k} d_i * prod_{l<i} p_l mod p_k, with the
    digits d_i from Eq. (rns_to_mrs) over the first k-1 moduli.  This is the
    form that reproduces Table 1."""
    digits, _ = be_recursion(y_prime, base)
    pk = base[-1]
    acc, w = 0, 1
    for i in range(len(base) - 1):
        acc += digits[i] * w
        w *= base[i]
    return acc % pk


# ---------------------------------------------------------------------------
# Sec. 3.4 -- the generalized scaling gadget, value level
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class Gate:
    """One projection gate of the gadget: digit wire ``src`` (modulus q) is
    projected into Z_m of wire ``dst`` and combined there by a free operation.
    kind 'sub': L_dst <- coeff * (L_dst - E)   (coeff = q^{-1} mod m)
    kind 'acc': Acc_dst <- Acc_dst + coeff * E (coeff = MRS weight mod m)"""
    phase: str
    src: int
    dst: int
    kind: str
    coeff: int


def split_base(base, scale_idx):
    S = sorted(scale_idx)
    R = [i for i in range(len(base)) if i not in S]
    return S, R


def gate_list(base, scale_idx):
    """Gate order of the gadget (READING: scaling moduli S ascending, then the
    remaining moduli R ascending).

    Phase A divides by every modulus of S in turn (Sec. 3.2, applied once per
    factor of s as allowed by the closing paragraph of Sec. 3.4): the digit
    wire S[a] is projected onto every later S wire and every R wire.

    Phase B is the generalized base extension of Sec. 3.3 over R: digit wire
    R[b] is projected onto every later R wire (the MRS recursion, which only
    needs the z-entries that feed later digits, as Sec. 3.3 prunes them) and
    onto every S wire, where the digits are recombined with their MRS
    weights prod_{b'<b} R[b'] (the corrected missing-residue formula)."""
    S, R = split_base(base, scale_idx)
    gates = []
    for a, si in enumerate(S):
        q = base[si]
        for dst in S[a + 1:] + R:
            gates.append(Gate("A", si, dst, "sub", inv_mod(q, base[dst])))
    for b, ri in enumerate(R):
        q = base[ri]
        for dst in R[b + 1:]:
            gates.append(Gate("B", ri, dst, "sub", inv_mod(q, base[dst])))
        for dst in S:
            w = 1
            for rb in R[:b]:
                w *= base[rb]
            gates.append(Gate("B", ri, dst, "acc", w % base[dst]))
    return gates


def shift_constants(base, scale_idx):
    """ShiftUp by P/2 and ShiftDown by P/(2s) (Sec. 3.4).  READING where they
    are not integers (odd P; a 2^l modulus scaled by, the bases of Sec. 4):
    ShiftUp by U = floor(P/2) and ShiftDown by floor(U/s).  The gadget then
    returns floor((x + (U mod s)) / s), equal to floor(x/s) whenever P/(2s)
    is an integer."""
    P = cardinality(base)
    s = cardinality([base[i] for i in scale_idx])
    return P // 2, (P // 2) // s


def rounding_offset(base, scale_idx) -> int:
    """r = floor(P/2) mod s: the gadget computes floor((x + r)/s) (0 when
    P/(2s) is an integer)."""
    s = cardinality([base[i] for i in scale_idx])
    return (cardinality(base) // 2) % s


def gadget_trace(base, scale_idx, x: int):
    """Run the gadget on plaintext residues and record every intermediate.

    Returns a dict with
      x_up      : the shifted input value x + P/2 (an integer in [0, P))
      gates     : gate_list(...)
      digit     : per gate, the value v in Z_q carried by the source wire
      slots     : G+1 lists of the k slot values: slots[g] is the state gate
                  g sees, slots[G] the final state.  During Phase A slot i
                  carries the current residue of wire i; when Phase B starts
                  the S slots are reset to the accumulator value 0 and the R
                  slots continue as the working copies T of the BE recursion
      out_R     : residues of wire R after Phase A (gadget outputs on R)
      out       : k output residues of floor(x_up/s) (before ShiftDown)
      y         : the decoded signed result after ShiftDown
    """
    P = cardinality(base)
    half, down = shift_constants(base, scale_idx)
    S, R = split_base(base, scale_idx)
    gates = gate_list(base, scale_idx)
    x_up = (signed_encode(x, P) + half) % P
    slot = rns(x_up, base)
    slots = []
    digit = []
    out_R = None
    for gate in gates:
        if gate.phase == "B" and out_R is None:
            out_R = {i: slot[i] for i in R}
            for i in S:
                slot[i] = 0
        slots.append(list(slot))  # the state this gate sees
        v = slot[gate.src]
        digit.append(v)
        m = base[gate.dst]
        if gate.kind == "sub":
            slot[gate.dst] = (gate.coeff * (slot[gate.dst] - v)) % m
        else:
            slot[gate.dst] = (slot[gate.dst] + gate.coeff * v) % m
    slots.append(list(slot))  # final state
    if out_R is None:  # no Phase B (cannot happen for valid params)
        out_R = {i: slot[i] for i in R}
    out = [out_R[i] if i in out_R else slot[i] for i in range(len(base))]
    y_unsigned = (crt(out, base) - down) % P
    return {
        "x_up": x_up,
        "gates": gates,
        "digit": digit,
        "slots": slots,
        "out_R": out_R,
        "out": out,
        "y": signed_decode(y_unsigned, P),
    }


def plain_scale(x: int, base, scale_idx) -> int:
    """floor((x + r)/s), r = rounding_offset(base, scale_idx) (floor(x/s) when
    P/(2s) is an integer), computed through the gadget's residue steps."""
    return gadget_trace(base, scale_idx, x)["y"]


# ---------------------------------------------------------------------------
# Ciphertext counts (Sec. 3.3 cost statement; projection-gate sizes Sec. 2.3)
# ---------------------------------------------------------------------------

def ciphertext_counts(base, scale_idx, row_reduction=True):
    """Ciphertexts per gadget instance, split into Phase A and Phase B.
    A projection gate with input modulus q has q ciphertexts, or q-1 with row
    reduction (Sec. 2.3)."""
    a = b = 0
    for gate in gate_list(base, scale_idx):
        q = base[gate.src]
        n = q - 1 if row_reduction else q
        if gate.phase == "A":
            a += n
        else:
            b += n
    return a, b


def be_cost_formula(moduli_in_paper_order) -> int:
    """sum_{i=1}^{k-1} sum_{j=i}^{k-1} p_j for a BE over the listed moduli
    p_1..p_{k-1} (Sec. 3.3)."""
    p = list(moduli_in_paper_order)
    n = len(p)
    return sum(p[j] for i in range(n) for j in range(i, n))
