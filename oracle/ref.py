"""CPU oracle for SALT's batched centroid + residual LoRA apply.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in ``oracle/``.
The product path (``libsalt`` and its Python binding) never does, and it shares
no code with this file: no kernels, headers, helpers, tables or constants.

What it computes, and where the paper fixes it
----------------------------------------------
* Sec. 3.1 (centroid-residual decomposition): an adapter update is the sum of a
  shared centroid and a per-user residual, ``dW_i = Wbar + delta_i``, with the
  residual itself a low-rank product of rank <= 2 (the only part that is swapped).
* Sec. 3.3 (multi-tenant serving): the served weight of request i is
  ``W_base + gamma * Wbar + delta_i``; gamma is a discrete per-request scale of
  the centroid term only, and the frontend groups requests by (centroid, gamma).
* Sec. 1 (LoRA): an update is the product of an (in x r) factor A and an
  (r x out) factor B.

With the base GEMM excluded (``y`` arrives holding ``x W_base``), the served
delta for token t with centroid c_t and residual slot u_t is

    y_t <- y_t + gamma_t * (x_t A_{c_t}) B_{c_t} + (x_t A_{u_t}) B_{u_t}

(row-vector convention, A is in x r and B is r x out).  Adapters are handed in
the storage layout of the boundary: A transposed, ``At[r][in]``, and ``B[r][out]``.
Everything here is float64 numpy, one token at a time; ``y`` is left unrounded.

Sec. 3.3 also lets a node fold one scaled centroid into its base weight at
start-up (``fuse_centroid``: ``W_base + gamma * A_c B_c``) and then add only the
residual per request.

Where the paper is silent this oracle reads it as follows: A is in x r and B is
r x out for row vectors (y += x A B); gamma scales only the centroid term; the
segment order is (centroid, slot, token) ascending with -1 first; an id of -1
means the term is absent.
"""
from __future__ import annotations

from typing import Dict, Mapping, Optional, Sequence, Tuple

import numpy as np


# --------------------------------------------------------------------------
# input decoding
# --------------------------------------------------------------------------
def decode(a: np.ndarray, dtype: str) -> np.ndarray:
    """Widen a storage array to float64 exactly.

    ``dtype == "f32"``: float32 values.  ``dtype == "bf16"``: uint16 bfloat16 bit
    patterns; a bfloat16 is the upper half of a float32, so the value is the
    float32 whose bits are ``pattern << 16``."""
    a = np.asarray(a)
    if dtype == "f32":
        return a.astype(np.float64)
    if dtype == "bf16":
        if a.dtype != np.uint16:
            raise TypeError("bf16 storage must be uint16 bit patterns")
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    raise ValueError(dtype)


# --------------------------------------------------------------------------
# O1: the segment plan (Sec. 3.3: requests grouped by their assigned centroid)
# --------------------------------------------------------------------------
def plan(tok_c: np.ndarray, tok_u: np.ndarray) -> Dict[str, np.ndarray]:
    """Canonical grouping of a batch's tokens.

    Sec. 3.3 has the serving frontend group requests that share a centroid; the
    residual of each user is a separate small adapter.  The plan orders tokens
    by (centroid id, residual slot, token index) ascending, -1 ("no centroid" /
    "no residual") first.  Because the token index is part of the key the order
    is total, so exactly one plan is correct.

    Returns
      perm     [T]        token index at each sorted position
      seg_off  [n_seg+1]  sorted-position starts of maximal runs of equal (c, u), then T
      seg_c    [n_seg]    centroid id of each run
      seg_u    [n_seg]    residual slot of each run
      grp_off  [n_grp+1]  segment indices where the centroid id changes, then n_seg
    """
    c = np.asarray(tok_c, dtype=np.int64)
    u = np.asarray(tok_u, dtype=np.int64)
    T = c.shape[0]
    t = np.arange(T, dtype=np.int64)
    perm = np.lexsort((t, u, c))          # last key is the primary key
    cs, us = c[perm], u[perm]
    if T == 0:
        z = np.zeros(0, np.int32)
        return dict(perm=z, seg_off=np.zeros(1, np.int32), seg_c=z, seg_u=z,
                    grp_off=np.zeros(1, np.int32))
    new_seg = np.ones(T, dtype=bool)
    new_seg[1:] = (cs[1:] != cs[:-1]) | (us[1:] != us[:-1])
    seg_start = np.flatnonzero(new_seg)
    seg_off = np.append(seg_start, T)
    seg_c = cs[seg_start]
    seg_u = us[seg_start]
    n_seg = seg_start.shape[0]
    new_grp = np.ones(n_seg, dtype=bool)
    new_grp[1:] = seg_c[1:] != seg_c[:-1]
    grp_off = np.append(np.flatnonzero(new_grp), n_seg)
    i32 = lambda a: np.asarray(a, dtype=np.int32)
    return dict(perm=i32(perm), seg_off=i32(seg_off), seg_c=i32(seg_c), seg_u=i32(seg_u),
                grp_off=i32(grp_off))


# --------------------------------------------------------------------------
# O2: the apply (Sec. 3.1 decomposition, Sec. 3.3 served weight)
# --------------------------------------------------------------------------
def apply(x: np.ndarray, y0: np.ndarray,
          cent_at: np.ndarray, cent_b: np.ndarray,
          residuals: Mapping[int, Tuple[np.ndarray, np.ndarray]],
          tok_c: np.ndarray, tok_u: np.ndarray,
          gamma: Optional[np.ndarray] = None,
          rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """Served output rows, float64, unrounded.

    x          [T][in]          activations (float64)
    y0         [T][out]         y on entry (float64)
    cent_at    [C][r_c][in]     centroid A, transposed (float64)
    cent_b     [C][r_c][out]    centroid B (float64)
    residuals  slot -> (At [r][in], B [r][out]) (float64); rank 0 allowed
    tok_c      [T] centroid id or -1 (no centroid term)
    tok_u      [T] residual slot or -1 (no residual term)
    gamma      [T] centroid scale (Sec. 3.3), None meaning 1 for every token
    rows       token indices to compute (default: all); the result has one row
               per requested token, in the order given

    For token t:  d = 0;  if c_t >= 0:  d += gamma_t * ((x_t @ A_c) @ B_c);
    if u_t >= 0:  d += (x_t @ A_u) @ B_u;  out_t = y0_t + d.
    """
    T = x.shape[0]
    if rows is None:
        rows = range(T)
    out = []
    for t in rows:
        xt = x[t]
        d = np.zeros(y0.shape[1], dtype=np.float64)
        c = int(tok_c[t])
        if c >= 0:
            g = 1.0 if gamma is None else float(gamma[t])
            A = cent_at[c].T                 # in x r_c
            B = cent_b[c]                    # r_c x out
            d += g * ((xt @ A) @ B)
        u = int(tok_u[t])
        if u >= 0:
            at_u, b_u = residuals[u]
            if at_u.shape[0] > 0:
                d += (xt @ at_u.T) @ b_u
        out.append(y0[t] + d)
    if not out:
        return np.zeros((0, y0.shape[1]), dtype=np.float64)
    return np.stack(out)


# --------------------------------------------------------------------------
# O3: a centroid fused into the base weight (Sec. 3.3, high-frequency domains)
# --------------------------------------------------------------------------
def fuse_centroid(w: np.ndarray, at: np.ndarray, b: np.ndarray, gamma: float) -> np.ndarray:
    """Base weight with the scaled centroid folded in, float64, unrounded.

    w      [in][out]   base weight (float64), row-vector convention y = x @ w
    at     [r][in]     the centroid's A, transposed (float64)
    b      [r][out]    the centroid's B (float64)
    gamma  the centroid scale of the node's domain

    Sec. 3.3 serves W_base + gamma * Wbar + delta_i; a node that fuses Wbar keeps
    W_base + gamma * Wbar as its weight and adds only delta_i per request.  With
    Wbar = A B (Sec. 1, A in x r, B r x out) the fused weight is
    ``w + gamma * (A @ B)``."""
    return w + float(gamma) * (at.T @ b)


# --------------------------------------------------------------------------
# O4: the alignment penalty / matrix cosine of two updates (Sec. 3.1, Eq. 2)
# --------------------------------------------------------------------------
def update_terms(at1: np.ndarray, b1: np.ndarray, at2: np.ndarray, b2: np.ndarray) -> Tuple[float, float, float]:
    """(Tr(dW1^T dW2), ||dW1||_F^2, ||dW2||_F^2), float64, from the dense updates.

    dW_k = A_k B_k is formed explicitly (in x out) from the storage factors
    At_k [r_k][in] and B_k [r_k][out]; Tr(X^T Y) is the sum of the elementwise
    product of X and Y."""
    dw1 = at1.T @ b1
    dw2 = at2.T @ b2
    return float(np.sum(dw1 * dw2)), float(np.sum(dw1 * dw1)), float(np.sum(dw2 * dw2))


def align_loss(inner: float, norm1_sq: float, norm2_sq: float, eps: float = 1e-8) -> float:
    """Eq. 2: 1 - Tr(dW1^T dW2) / (||dW1||_F ||dW2||_F + eps), eps = 1e-8 (Sec. 3.1)."""
    return 1.0 - inner / (np.sqrt(norm1_sq) * np.sqrt(norm2_sq) + eps)


# --------------------------------------------------------------------------
# O5: centroid routing (Sec. 3.2, the two-stage activation profiling filter)
# --------------------------------------------------------------------------
def route_decide(z_n_min: float, z_r: Sequence[float], tau_n: float, tau_r: float) -> Tuple[int, bool, bool]:
    """(k*, out_of_distribution, blended) from the two stages' deviations.

    Stage 1 rejects the data when the smallest norm deviation exceeds tau_N.
    Stage 2 picks the centroid with the smallest ratio deviation; if even that
    one exceeds tau_R the task is treated as blended and also falls back.
    k* = -1 means the fallback (standard LoRA)."""
    if z_n_min > tau_n:
        return -1, True, False
    best = min(range(len(z_r)), key=lambda k: (z_r[k], k))
    if z_r[best] > tau_r:
        return -1, False, True
    return best, False, False


def route(n: Sequence[float], mu_n: Sequence[float], sigma_n: Sequence[float],
          mu_r: Sequence[float], sigma_r: Sequence[float], tau_n: float = 2.0,
          tau_r: float = 2.0) -> Dict[str, object]:
    """Sec. 3.2 on per-centroid displacement norms N_k and their Phase 1
    calibration (mu, sigma): Z_N,k = |N_k - mu_N,k| / sigma_N,k; the dominance
    ratio R_k = N_k / ((1 / (K - 1)) sum_{j != k} N_j); Z_R,k = |R_k - mu_R,k| /
    sigma_R,k; then ``route_decide``.  Plain Python floats."""
    K = len(n)
    z_n = [abs(n[k] - mu_n[k]) / sigma_n[k] for k in range(K)]
    z_r = []
    for k in range(K):
        others = sum(n[j] for j in range(K) if j != k) / (K - 1)
        z_r.append(abs(n[k] / others - mu_r[k]) / sigma_r[k])
    k_star, ood, blended = route_decide(min(z_n), z_r, tau_n, tau_r)
    return {"k_star": k_star, "ood": ood, "blended": blended, "z_n": z_n, "z_r": z_r}


# --------------------------------------------------------------------------
# swap footprint (Table 1 and the appendix tables, Memory (MB) columns)
# --------------------------------------------------------------------------
def adapter_bytes(rank: int, shapes: Sequence[Tuple[int, int]], n_layers: int = 1,
                  esize: int = 2) -> int:
    """Bytes of one rank-``rank`` LoRA adapter over the given (in, out) targets.

    Each target holds A (in x r) and B (r x out), so ``r * (in + out)`` parameters;
    summed over the targets of a layer and over layers, times the element size.
    The paper's Memory (MB) columns (swap size of a residual or LoRA, pinned size
    of an r=16 centroid) are this count in bytes / 1e6 at 2 bytes per parameter."""
    per_layer = sum(int(i) + int(o) for i, o in shapes)
    return int(rank) * per_layer * int(n_layers) * int(esize)
