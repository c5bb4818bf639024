"""Helpers shared by the GPU tests: running the HIP pipeline through the
binding, and gathering the words of selected gadgets out of device buffers so
that they can be compared with the oracle gadget by gadget.

Nothing here computes any of the method's arithmetic; layouts are the ones
documented in include/redash.h.
"""

from __future__ import annotations

import numpy as np
import torch

from paper_2506_14489_amd import binding as B


def label_layout(moduli):
    """(woff, W) per modulus index: word offsets of a gadget's k labels."""
    out, off = [], 0
    for m in moduli:
        W = B.label_words_of(m)
        out.append((off, W))
        off += W
    return out, off


def gate_list_sizes(oracle_gates, moduli):
    """(q, W_dst) per gate from the oracle's gate list."""
    return [(moduli[src], B.label_words_of(moduli[dst])) for (src, dst, *_r) in oracle_gates]


def label_index(moduli, n: int, gadgets: np.ndarray) -> np.ndarray:
    """Indices of the words of the given gadgets in a LabelTensor with stride n,
    ordered modulus by modulus, word by word, gadget by gadget, i.e. the order
    of a LabelTensor with stride len(gadgets)."""
    lay, _ = label_layout(moduli)
    idx = []
    for (woff, W) in lay:
        for w in range(W):
            idx.append((woff + w) * n + gadgets)
    return np.concatenate(idx).astype(np.int64)


def table_index(gates_qw, n: int, gadgets: np.ndarray) -> np.ndarray:
    """Indices of all rows of the given gadgets, in the order of a table with
    stride len(gadgets)."""
    idx, base = [], 0
    for (q, W) in gates_qw:
        per = (q - 1) * W
        cols = np.arange(per, dtype=np.int64)
        idx.append((base + gadgets[:, None].astype(np.int64) * per + cols[None, :]).reshape(-1))
        base += n * per
    return np.concatenate(idx)


def gather(t: torch.Tensor, idx: np.ndarray) -> np.ndarray:
    """t[idx] copied to the host as uint32."""
    sel = t.index_select(0, torch.from_numpy(idx).to(t.device))
    return sel.cpu().numpy().view(np.uint32)


def to_u32(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint32)


def to_dev(a: np.ndarray, device="cuda") -> torch.Tensor:
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def gpu_pipeline(params, x: np.ndarray, device="cuda"):
    """Garble, encode, evaluate and decode on the GPU.  Returns the Buffers."""
    buf = B.Buffers(params, device)
    B.redash_garble_scale(params, buf.offsets, buf.in_zero, buf.out_zero, buf.tables, buf.work)
    xd = torch.from_numpy(np.ascontiguousarray(x, dtype=np.int64)).to(device)
    B.redash_encode(params, xd, buf.in_zero, buf.offsets, buf.in_labels)
    B.redash_eval_scale(params, buf.in_labels, buf.tables, buf.out_labels, buf.work)
    B.redash_decode(params, buf.out_labels, buf.out_zero, buf.offsets, buf.y, buf.bad)
    torch.cuda.synchronize()
    return buf
