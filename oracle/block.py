"""Float64 oracle of the stitched pre-LN transformer block.

TEST INFRASTRUCTURE ONLY (see ``oracle/subkernels.py``).

Def. 1 (Section 3) splits a compiled model into generated sub-kernels and
fixed library calls; Gate 3 (Section 4.4) checks the re-stitched model end to
end against a float64 reference.  This module is that reference for one
pre-LN block whose sub-kernels are the fused classes of this library and
whose GEMMs stand for the library calls:

    a    = LN1(x)
    qkv  = a @ Wqkv + bqkv            -> q | k | v, each split into heads
    P_h  = softmax(q_h k_h^T / sqrt(d) + causal)
    o    = concat_h(P_h v_h)
    att  = o @ Wo + bo
    h1   = x + att ;  m = LN2(h1)
    g    = GELU_erf(m @ W1 + b1)
    d    = g @ W2 + b2
    out  = h1 + d

Readings (paper silent): pre-LN GPT-style order; q, k and v occupy columns
[0, H), [H, 2H), [2H, 3H) of qkv, each head-major (head h owns columns
h*dh .. h*dh+dh-1 of its third); the softmax scale is 1/sqrt(dh).

The computation runs per sequence (attention never crosses sequences), so
memory stays bounded and a subset of sequences is an exact sample.
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, Optional

import numpy as np

from .subkernels import gelu_erf, layernorm_residual, row_softmax

__all__ = ["block_forward_sequence", "block_forward"]

STAGES = ("a", "qkv", "scores", "probs", "o", "att", "h1", "m", "u", "g", "d", "out")


def block_forward_sequence(x, p: Dict[str, np.ndarray], heads: int, eps: float,
                           keep: Iterable[str] = STAGES) -> Dict[str, np.ndarray]:
    """One sequence x [seq, hidden] (float64) through the block.

    ``p`` holds float64 parameters w_qkv [H,3H], b_qkv [3H], w_o [H,H],
    b_o [H], w_1 [H,F], b_1 [F], w_2 [F,H], b_2 [H], ln1_gamma, ln1_beta,
    ln2_gamma, ln2_beta [H].  Returns the requested intermediates; "scores"
    are the scaled, unmasked logits [heads, seq, seq] and "probs" the causal
    softmax [heads, seq, seq].
    """
    keep = set(keep)
    x = np.asarray(x, dtype=np.float64)
    s, hid = x.shape
    dh = hid // heads
    out: Dict[str, np.ndarray] = {}

    a, _ = layernorm_residual(x, None, p["ln1_gamma"], p["ln1_beta"], eps)
    qkv = a @ p["w_qkv"] + p["b_qkv"][None, :]
    q = qkv[:, 0 * hid:1 * hid]
    k = qkv[:, 1 * hid:2 * hid]
    v = qkv[:, 2 * hid:3 * hid]
    o = np.empty((s, hid), dtype=np.float64)
    scale = 1.0 / math.sqrt(dh)
    scores = np.empty((heads, s, s)) if "scores" in keep else None
    probs = np.empty((heads, s, s)) if "probs" in keep else None
    for h in range(heads):
        cols = slice(h * dh, (h + 1) * dh)
        sc = q[:, cols] @ k[:, cols].T
        pr = row_softmax(sc, None, scale, causal_q_len=s)
        o[:, cols] = pr @ v[:, cols]
        if scores is not None:
            scores[h] = sc * scale
        if probs is not None:
            probs[h] = pr
    att = o @ p["w_o"] + p["b_o"][None, :]
    m, h1 = layernorm_residual(att, x, p["ln2_gamma"], p["ln2_beta"], eps)
    u = m @ p["w_1"]
    g = gelu_erf(u + p["b_1"][None, :])
    d = g @ p["w_2"] + p["b_2"][None, :]
    y = h1 + d

    for name, val in (("a", a), ("qkv", qkv), ("scores", scores), ("probs", probs),
                      ("o", o), ("att", att), ("h1", h1), ("m", m), ("u", u),
                      ("g", g), ("d", d), ("out", y)):
        if name in keep:
            out[name] = val
    return out


def block_forward(x, p: Dict[str, np.ndarray], heads: int, eps: float,
                  sequences: Optional[Iterable[int]] = None,
                  keep: Iterable[str] = ("out",)) -> Dict[str, np.ndarray]:
    """x [batch, seq, hidden]; runs the listed sequences (default all) and
    stacks each requested intermediate along a leading sequence axis."""
    x = np.asarray(x, dtype=np.float64)
    seqs = list(range(x.shape[0])) if sequences is None else list(sequences)
    keep = tuple(keep)
    parts = [block_forward_sequence(x[b], p, heads, eps, keep) for b in seqs]
    return {k: np.stack([pt[k] for pt in parts]) for k in keep}
