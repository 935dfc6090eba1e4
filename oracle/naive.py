"""CPU float64 oracle for one attention layer's forward and backward pass.

TEST INFRASTRUCTURE ONLY. This module is the slow, plain definition that the
HIP library is checked against. Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import it; the library and its Python binding
never do, and nothing here is shared with the GPU path.

What is computed (per batch-head, all in float64)
-------------------------------------------------
The paper names the arrays of the naive path (Q, K, V, the n x n attention
matrix A, Out, and the gradients GQ, GK, GV with the score gradient GS) and
contrasts two realisations of the same result: a naive one that writes A to
memory and reads it back, and a fused one that consumes A as soon as it is
produced (Fig. fig:concept, section sec:dnf-onf-machines; Paper II,
section sec:paper2-cpu, "Algorithm 1" reading A from memory versus the fused
"Algorithm 2"). The paper does not print the attention formula itself; it
verifies its kernels against PyTorch autograd (abstract; section
sec:methodology, "Kernels benchmarked") and points to FlashAttention as the
same kernel (section sec:related-work). The reading used here is therefore
the standard scaled softmax attention, with loss l = <O, dO>_F:

    S  = s * Q K^T                          (n x n, explicit)
    S_ij = -inf for j > i                   (causal mask, diagonal kept)
    P  = softmax_rows(S);  L_i = log sum_j exp(S_ij)   (natural log)
    O  = P V
    dV = P^T dO
    dP = dO V^T
    D_i = sum_j P_ij dP_ij                  (the backward's row pre-pass)
    dS = P * (dP - D 1^T)                   (GS in the paper's naming)
    dQ = s * dS K;   dK = s * dS^T Q

Parity is pinned by the CPU tests (finite differences of l, closed forms,
row invariants, a metamorphic shift, and an independent autograd derivation),
not by anything the paper prints: the paper prints no attention values.
"""
from __future__ import annotations

from typing import Dict, Iterable, Optional

import numpy as np

__all__ = ["scores", "forward_head", "backward_head", "attention_head",
           "attention", "attention_forward", "rows_forward_dq", "max_rel_err",
           "row_invariants"]


def scores(q: np.ndarray, k: np.ndarray, scale: float, causal: bool) -> np.ndarray:
    """S = s Q K^T with the causal mask applied (key j <= query i kept).

    The attention matrix of the naive path, materialised in full (Paper I,
    section sec:paper1, Table tab:paper1-dram counts it as an n x n array).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    S = scale * (q @ k.T)
    if causal:
        n_q, n_k = S.shape
        masked = np.triu(np.ones((n_q, n_k), dtype=bool), k=1)
        S[masked] = -np.inf
    return S


def forward_head(q, k, v, scale: float, causal: bool):
    """Naive forward of one head: returns (S, P, O, L).

    Row softmax with its maximum subtracted for range only (the quotient is
    unchanged); L is the natural-log log-sum-exp of the scaled, masked row.
    """
    S = scores(q, k, scale, causal)
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    Z = E.sum(axis=1, keepdims=True)
    P = E / Z
    L = (m + np.log(Z))[:, 0]
    O = P @ np.asarray(v, dtype=np.float64)
    return S, P, O, L


def backward_head(q, k, v, do, P, scale: float):
    """Naive backward of one head from the stored P (the path that reads A
    back from memory, Paper II section sec:paper2-cpu): returns
    (dQ, dK, dV, dS, Dvec)."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    dV = P.T @ do
    dP = do @ v.T
    Dvec = (P * dP).sum(axis=1)
    dS = P * (dP - Dvec[:, None])
    dQ = scale * (dS @ k)
    dK = scale * (dS.T @ q)
    return dQ, dK, dV, dS, Dvec


def attention_head(q, k, v, do, scale: float, causal: bool, keep: bool = False) -> Dict[str, np.ndarray]:
    """Forward then backward of one head. With keep=True the n x n S, P, dS
    are returned too (for the invariant tests)."""
    S, P, O, L = forward_head(q, k, v, scale, causal)
    dQ, dK, dV, dS, Dvec = backward_head(q, k, v, do, P, scale)
    out = {"O": O, "L": L, "dQ": dQ, "dK": dK, "dV": dV, "D": Dvec}
    if keep:
        out.update({"S": S, "P": P, "dS": dS})
    return out


def _heads(B: int, H: int, heads: Optional[Iterable]):
    if heads is None:
        return [(b, h) for b in range(B) for h in range(H)]
    return list(heads)


def attention(q, k, v, do, scale: float, causal: bool, heads=None) -> Dict[str, np.ndarray]:
    """Forward+backward over [B, H, n, d] inputs, head by head.

    ``heads`` optionally lists (b, h) pairs; outputs then have a leading axis
    over those pairs ([len(heads), n, d] and [len(heads), n])."""
    B, H, n, d = q.shape
    hs = _heads(B, H, heads)
    res = {key: [] for key in ("O", "L", "dQ", "dK", "dV")}
    for (b, h) in hs:
        r = attention_head(q[b, h], k[b, h], v[b, h], do[b, h], scale, causal)
        for key in res:
            res[key].append(r[key])
    out = {key: np.stack(val) for key, val in res.items()}
    if heads is None:
        out = {key: val.reshape((B, H) + val.shape[1:]) for key, val in out.items()}
    return out


def attention_forward(q, k, v, scale: float, causal: bool, heads=None) -> Dict[str, np.ndarray]:
    """Forward only (O, L) over [B, H, n, d] inputs, head by head."""
    B, H, n, d = q.shape
    hs = _heads(B, H, heads)
    Os, Ls = [], []
    for (b, h) in hs:
        _, _, O, L = forward_head(q[b, h], k[b, h], v[b, h], scale, causal)
        Os.append(O)
        Ls.append(L)
    O, L = np.stack(Os), np.stack(Ls)
    if heads is None:
        O, L = O.reshape(B, H, n, d), L.reshape(B, H, n)
    return {"O": O, "L": L}


def rows_forward_dq(q, k, v, do, rows, scale: float, causal: bool) -> Dict[str, np.ndarray]:
    """O, L and dQ of selected query rows of one head.

    Each of these depends only on its own row of S and P (a row of dS needs
    only its own D_i), so a row subset is the same definition restricted to
    those rows; used to sample very long sequences.
    """
    rows = np.asarray(rows)
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    S = scale * (q[rows] @ k.T)
    if causal:
        cols = np.arange(k.shape[0])[None, :]
        S[cols > rows[:, None]] = -np.inf
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    Z = E.sum(axis=1, keepdims=True)
    P = E / Z
    L = (m + np.log(Z))[:, 0]
    O = P @ v
    dP = do[rows] @ v.T
    Dvec = (P * dP).sum(axis=1)
    dS = P * (dP - Dvec[:, None])
    dQ = scale * (dS @ k)
    return {"O": O, "L": L, "dQ": dQ}


def row_invariants(P: np.ndarray, dS: np.ndarray):
    """Largest |sum_j P_ij - 1| and largest |sum_j dS_ij| / sum_j |dS_ij|.

    Softmax rows sum to one, and each row of dS sums to zero because
    sum_j P_ij (dP_ij - D_i) = D_i - D_i.
    """
    p_err = np.abs(P.sum(axis=1) - 1.0).max()
    denom = np.maximum(np.abs(dS).sum(axis=1), np.finfo(np.float64).tiny)
    ds_err = (np.abs(dS.sum(axis=1)) / denom).max()
    return float(p_err), float(ds_err)


def max_rel_err(x, ref) -> float:
    """max_i |x_i - ref_i| / max_i |ref_i| over a whole tensor, in float64."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.abs(ref).max()
    if den == 0.0:
        return float(np.abs(x - ref).max())
    return float(np.abs(x - ref).max() / den)
