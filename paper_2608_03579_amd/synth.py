"""Seeded synthetic workloads for the batched centroid + residual LoRA apply.

This module draws random inputs and lays them out in the byte formats the
``libsalt`` boundary takes (``include/salt.h``). It holds none of the method's
arithmetic: no contraction, no grouping, no plan. Both the CPU oracle (via the
tests) and the GPU path consume what it returns, so neither side can hide a
mistake behind a shared helper.

Workload shapes follow the paper's serving setting (Sec. 3.3, multi-tenant
serving with a pinned centroid and swapped residuals; Sec. 4.4 and the appendix
throughput tables for Llama-3.2-3B; appendix A.2 for "all linear layers" as
LoRA targets). The paper's own traces and datasets are not used; seeded draws of
the same shapes stand in for them.

Random streams: every tensor is drawn from its own
``numpy.random.SeedSequence([2608, 3579, cfg, seed, kind, ...])`` so a single
table, user or slot can be regenerated on its own (needed for the 196-table
prefill workload, whose activations do not fit in host memory at once).

Storage forms
-------------
* ``dtype == "f32"``: ``numpy.float32`` arrays.
* ``dtype == "bf16"``: ``numpy.uint16`` arrays holding bfloat16 bit patterns,
  rounded to nearest-even from a float32 draw.

Layouts (all row-major, rank-major adapters, matching ``salt.h``)
-----------------------------------------------------------------
* centroid table: ``At[C][r_c][in]`` (A transposed) and ``B[C][r_c][out]``.
* residual of one user for one table: ``At[r][in]``, ``B[r][out]``.
* residual blob of one user (what one swap moves): for each table in order,
  ``At[r][in]`` followed by ``B[r][out]``; ``r * sum(in + out)`` elements.
* activations ``x[T][in]``, outputs ``y[T][out]``.
* maps ``tok_c[T]``, ``tok_u[T]`` (int32, -1 = term absent), ``gamma[T]``
  (float32) or ``None`` for gamma = 1.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

SEED_ROOT = (2608, 3579)

# stream kinds (part of the SeedSequence entropy)
_K_MAP, _K_CENT, _K_RES, _K_X, _K_Y0, _K_GAMMA, _K_SEGLEN, _K_W = range(8)

ADAPTER_STD = 0.02   # A, B ~ N(0, 0.02^2)
BASE_STD = 0.02      # base weight entries ~ N(0, 0.02^2) (a centroid is folded into it)
GAMMA_BINS = (0.6, 0.8, 1.0)   # discrete centroid scales, Sec. 3.3

# Decoder-layer projection shapes (in -> out). "All linear layers" are the LoRA
# targets for Llama-family models (appendix A.2).
LLAMA32_3B = dict(hidden=3072, kv=1024, inter=8192, layers=28)
LLAMA31_8B = dict(hidden=4096, kv=1024, inter=14336, layers=32)


def decoder_projections(hidden: int, kv: int, inter: int) -> List[Tuple[str, int, int]]:
    """The seven linear projections of one Llama decoder layer as (name, in, out)."""
    return [
        ("q_proj", hidden, hidden),
        ("k_proj", hidden, kv),
        ("v_proj", hidden, kv),
        ("o_proj", hidden, hidden),
        ("gate_proj", hidden, inter),
        ("up_proj", hidden, inter),
        ("down_proj", inter, hidden),
    ]


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([*SEED_ROOT, *[int(k) for k in key]]))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Encode float32 values as bfloat16 bit patterns, round-to-nearest-even.

    Input encoding only (the draws are finite, so no NaN handling is needed)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    bias = 0x7FFF + ((u >> 16) & 1)
    return ((u + bias) >> 16).astype(np.uint16)


def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    return (rng.standard_normal(size=shape, dtype=np.float32) * np.float32(std)).astype(np.float32)


def segment_lengths(rng: np.random.Generator, n_users: int, lo: int, hi: int, total: int) -> np.ndarray:
    """Per-user prefill lengths: L_i ~ U{lo..hi}, rescaled to integers summing to ``total``.

    Rescale rule: n_i = max(1, floor(L_i * total / sum L)); the shortfall is handed
    out one token at a time by largest fractional part (ties to the lower index);
    any excess (from the max(1, .) floor) is taken from the largest n_i (ties to
    the lower index)."""
    L = rng.integers(lo, hi + 1, size=n_users).astype(np.int64)
    f = L * total / L.sum()
    n = np.maximum(1, np.floor(f).astype(np.int64))
    frac = f - np.floor(f)
    short = total - int(n.sum())
    if short > 0:
        order = sorted(range(n_users), key=lambda i: (-frac[i], i))
        for k in range(short):
            n[order[k % n_users]] += 1
    while int(n.sum()) > total:
        i = int(np.argmax(n))   # argmax returns the lowest index among ties
        n[i] -= 1
    assert int(n.sum()) == total and n.min() >= 1
    return n


def truncated_zipf_pmf(s: float, n: int) -> np.ndarray:
    """P(k) proportional to k^-s for k = 1..n (user k maps to slot k-1)."""
    w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    return w / w.sum()


@dataclasses.dataclass
class Workload:
    """One seeded instance of a serving batch plus its adapter tables.

    Only the maps and the slot ranks are materialised eagerly; adapter tables,
    residual blobs and activations are drawn on demand, per table or per user."""

    cfg: int
    seed: int
    name: str
    dtype: str                               # "f32" | "bf16"
    tables: List[Tuple[str, int, int]]       # (name, in, out), in call order
    n_centroids: int
    r_c: int
    n_slots: int
    r_u_max: int
    slot_rank: np.ndarray                    # int32 [n_slots]; rank a loaded slot holds
    tok_c: np.ndarray                        # int32 [T]
    tok_u: np.ndarray                        # int32 [T]
    gamma: Optional[np.ndarray]              # float32 [T] or None (= 1)
    y0_kind: str = "zero"                    # "zero" | "normal" | "int"
    exact: bool = False                      # integer-valued variant (exact in any order)
    user_of_slot: Optional[np.ndarray] = None
    meta: Dict = dataclasses.field(default_factory=dict)
    _blob_cache: Dict = dataclasses.field(default_factory=dict, repr=False)

    # ---- sizes -----------------------------------------------------------
    @property
    def T(self) -> int:
        return int(self.tok_c.shape[0])

    @property
    def esize(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def storage(self):
        return np.float32 if self.dtype == "f32" else np.uint16

    def referenced_slots(self) -> np.ndarray:
        u = self.tok_u[self.tok_u >= 0]
        return np.unique(u).astype(np.int32)

    def table_prefix(self) -> List[int]:
        """Element offset of each table inside a rank-1 residual blob (sum of in+out before it)."""
        out, acc = [], 0
        for _, i, o in self.tables:
            out.append(acc)
            acc += i + o
        return out

    def blob_elems(self, r: int) -> int:
        return r * sum(i + o for _, i, o in self.tables)

    # ---- draws -------------------------------------------------------------
    def _encode(self, a: np.ndarray) -> np.ndarray:
        if self.dtype == "f32":
            return np.ascontiguousarray(a, dtype=np.float32)
        return f32_to_bf16_bits(a)

    def _adapter(self, rng: np.random.Generator, shape) -> np.ndarray:
        if not self.exact:
            return self._encode(_normal(rng, shape, ADAPTER_STD))
        return self._encode(rng.integers(-1, 2, size=shape).astype(np.float32))

    def _adapter_at(self, rng: np.random.Generator, r: int, n_in: int) -> np.ndarray:
        """A transposed, [r][in]. Exact variant: at most 3 nonzeros in {-1, +1} per rank row."""
        if not self.exact:
            return self._encode(_normal(rng, (r, n_in), ADAPTER_STD))
        a = np.zeros((r, n_in), dtype=np.float32)
        for j in range(r):
            nnz = int(rng.integers(0, 4))
            cols = rng.choice(n_in, size=nnz, replace=False)
            a[j, cols] = rng.choice(np.array([-1.0, 1.0], dtype=np.float32), size=nnz)
        return self._encode(a)

    def centroids(self, table: int) -> Tuple[np.ndarray, np.ndarray]:
        """(At [C][r_c][in], B [C][r_c][out]) of one table, storage form."""
        _, n_in, n_out = self.tables[table]
        C, r = self.n_centroids, self.r_c
        rng = _rng(self.cfg, self.seed, _K_CENT, table)
        at = np.stack([self._adapter_at(rng, r, n_in) for _ in range(C)]) if C else \
            np.zeros((0, r, n_in), self.storage)
        b = np.stack([self._adapter(rng, (r, n_out)) for _ in range(C)]) if C else \
            np.zeros((0, r, n_out), self.storage)
        return at.reshape(C, r, n_in), b.reshape(C, r, n_out)

    def residual_blob(self, slot: int, gen: int = 0) -> np.ndarray:
        """Packed residual of the user in ``slot`` (all tables), storage form, 1-D.

        ``gen`` selects a fresh draw for a slot that is swapped to a new user."""
        key = (slot, gen)
        if key in self._blob_cache:
            return self._blob_cache[key]
        r = int(self.slot_rank[slot])
        rng = _rng(self.cfg, self.seed, _K_RES, slot, gen)
        parts = []
        for _, n_in, n_out in self.tables:
            parts.append(self._adapter_at(rng, r, n_in).reshape(-1))
            parts.append(self._adapter(rng, (r, n_out)).reshape(-1))
        blob = np.concatenate(parts) if parts else np.zeros(0, self.storage)
        blob = np.ascontiguousarray(blob)
        if len(self._blob_cache) < 4096:
            self._blob_cache[key] = blob
        return blob

    def residual(self, slot: int, table: int, gen: int = 0) -> Tuple[np.ndarray, np.ndarray]:
        """(At [r][in], B [r][out]) of one user for one table, cut out of the blob."""
        r = int(self.slot_rank[slot])
        blob = self.residual_blob(slot, gen)
        off = r * self.table_prefix()[table]
        _, n_in, n_out = self.tables[table]
        at = blob[off: off + r * n_in].reshape(r, n_in)
        b = blob[off + r * n_in: off + r * (n_in + n_out)].reshape(r, n_out)
        return at, b

    def x(self, table: int, rows: Optional[Sequence[int]] = None) -> np.ndarray:
        _, n_in, _ = self.tables[table]
        rng = _rng(self.cfg, self.seed, _K_X, table)
        if self.exact:
            a = rng.integers(-1, 2, size=(self.T, n_in)).astype(np.float32)
        else:
            a = rng.standard_normal(size=(self.T, n_in), dtype=np.float32)
        if rows is not None:
            a = a[np.asarray(rows)]
        return self._encode(a)

    def base_weight(self, table: int, ldw: Optional[int] = None) -> np.ndarray:
        """Base weight of one table, [in][ldw] storage form (ldw >= out; the
        columns past out are drawn too and must come back unchanged from a fuse).
        Exact variant: integers in [-8, 8]."""
        _, n_in, n_out = self.tables[table]
        ldw = n_out if ldw is None else int(ldw)
        rng = _rng(self.cfg, self.seed, _K_W, table)
        if self.exact:
            a = rng.integers(-8, 9, size=(n_in, ldw)).astype(np.float32)
        else:
            a = _normal(rng, (n_in, ldw), BASE_STD)
        return self._encode(a)

    def y0(self, table: int, rows: Optional[Sequence[int]] = None) -> np.ndarray:
        _, _, n_out = self.tables[table]
        if self.y0_kind == "zero":
            a = np.zeros((self.T, n_out), dtype=np.float32)
        else:
            rng = _rng(self.cfg, self.seed, _K_Y0, table)
            if self.y0_kind == "int":
                a = rng.integers(-8, 9, size=(self.T, n_out)).astype(np.float32)
            else:
                a = rng.standard_normal(size=(self.T, n_out), dtype=np.float32)
        if rows is not None:
            a = a[np.asarray(rows)]
        return self._encode(a)


class ConcatTail(Workload):
    """A workload whose slots in ``concat`` (slot -> (centroid c, base slot)) hold
    long-tail concatenated adapters: per table, the rows of centroid c followed
    by the rows of the residual drawn for the base slot (At stacked over At, B
    over B; rank r_c + rank of the base slot).  Array stacking only."""

    def residual_blob(self, slot: int, gen: int = 0) -> np.ndarray:
        cat_map = getattr(self, "concat", {})
        if slot not in cat_map:
            return super().residual_blob(slot, gen)
        c, base = cat_map[slot]
        parts = []
        for t in range(len(self.tables)):
            cat, cb = self.centroids(t)
            at_u, b_u = self.residual(base, t, gen)
            parts.append(np.concatenate([cat[c], at_u]).reshape(-1))
            parts.append(np.concatenate([cb[c], b_u]).reshape(-1))
        return np.ascontiguousarray(np.concatenate(parts))


def long_tail(w: Workload, tail_from: int) -> "ConcatTail":
    """The batch of ``w`` with the users of slots >= tail_from (the rare end of a
    Zipf draw) served by concatenated adapters: each such user gets a new slot
    (n_slots + its slot) of rank r_c + r_u and its tokens no centroid (c = -1).
    Sec. 3.3's long tail next to the centroid + residual head."""
    tail = w.tok_u >= tail_from
    tok_c = np.where(tail, -1, w.tok_c).astype(np.int32)
    tok_u = np.where(tail, w.n_slots + w.tok_u, w.tok_u).astype(np.int32)
    slot_rank = np.concatenate([w.slot_rank, w.r_c + w.slot_rank]).astype(np.int32)
    concat = {}
    for t in np.nonzero(tail)[0]:
        concat[int(tok_u[t])] = (int(w.tok_c[t]), int(w.tok_u[t]))
    out = ConcatTail(cfg=w.cfg, seed=w.seed, name=w.name + " (long tail concatenated)", dtype=w.dtype,
                     tables=w.tables, n_centroids=w.n_centroids, r_c=w.r_c, n_slots=2 * w.n_slots,
                     r_u_max=int(slot_rank[np.unique(tok_u[tok_u >= 0])].max()), slot_rank=slot_rank,
                     tok_c=tok_c, tok_u=tok_u, gamma=None if w.gamma is None else w.gamma.copy(),
                     y0_kind=w.y0_kind, exact=w.exact, meta=dict(w.meta, tail_from=tail_from))
    out.concat = concat
    return out


def _gamma_per_user(cfg: int, seed: int, n_users: int) -> np.ndarray:
    rng = _rng(cfg, seed, _K_GAMMA)
    return np.asarray(GAMMA_BINS, dtype=np.float32)[rng.integers(0, len(GAMMA_BINS), size=n_users)]


def make(cfg: int, seed: int = 0, *, y0: str = "zero", gamma: str = "one", exact: bool = False,
         baseline: bool = False, T: Optional[int] = None, layers: Optional[int] = None) -> Workload:
    """Build workload ``cfg`` (1..5) for ``seed``.

    Config recipes (one GPU, synthetic, seeded):

    1. Tiny, fp32: one 256->256 table, 4 centroids r=8, 16 residual slots r=2,
       64 tokens, each token's (centroid, residual) pair uniform over the 64 pairs.
    2. Llama-3.2-3B q_proj (3072->3072), bf16 decode: 64 tokens, one per user,
       64 residual slots r=2 (users in a random slot order), 4 centroids r=32, the
       centroid of each user uniform.
    3. Llama-3.2-3B, every projection of 28 layers (196 tables), bf16 prefill of
       8192 tokens in 256 contiguous user segments with lengths ~U{1..512}
       rescaled to sum 8192, 8 centroids r=64, residuals r=1.
    4. Llama-3.1-8B one layer (7 tables), bf16 decode of 256 tokens over 1024
       resident slots r=2, 16 centroids r=32; 256 distinct users, one token each;
       ``meta['swap_slots']`` lists 32 batch slots that are swapped to new users
       (residual generation 1) just before the step.
    5. Llama-3.2-3B one layer (7 tables), bf16, 512 tokens whose users are i.i.d.
       truncated Zipf(1.1) over 2000 users (scattered order), residual rank per user
       1 or 2 with probability 1/2, 8 centroids r=64.  ``baseline=True`` gives the
       comparison run: no centroid (C=0) and an independent rank-16 LoRA per user.

    Variants: ``y0`` in {"zero", "normal", "int"}; ``gamma`` in {"one", "bins"}
    (per-user gamma from {0.6, 0.8, 1.0}); ``exact`` draws integer-valued inputs
    (x, B in {-1, 0, 1}; at most 3 nonzeros +-1 per rank row of A; y0 integer)
    whose every partial sum is exact in fp32 and whose outputs are exact in
    bf16; ``T`` and ``layers`` shrink configs 3-5 for quick runs.
    """
    rng = _rng(cfg, seed, _K_MAP)
    meta: Dict = {}
    if cfg == 1:
        tables = [("tiny", 256, 256)]
        C, rc, S, ru, dt = 4, 8, 16, 2, "f32"
        Tn = T or 64
        tok_c = rng.integers(0, C, size=Tn).astype(np.int32)
        tok_u = rng.integers(0, S, size=Tn).astype(np.int32)
        slot_rank = np.full(S, ru, np.int32)
        user_of_tok = tok_u.copy()
        n_users = S
    elif cfg == 2:
        tables = [("q_proj", 3072, 3072)]
        C, rc, S, ru, dt = 4, 32, 64, 2, "bf16"
        Tn = T or 64
        users = rng.permutation(S)[:Tn].astype(np.int32)
        c_of_user = rng.integers(0, C, size=S).astype(np.int32)
        tok_u = users
        tok_c = c_of_user[users]
        slot_rank = np.full(S, ru, np.int32)
        user_of_tok = tok_u.copy()
        n_users = S
    elif cfg == 3:
        L = layers if layers is not None else LLAMA32_3B["layers"]
        proj = decoder_projections(LLAMA32_3B["hidden"], LLAMA32_3B["kv"], LLAMA32_3B["inter"])
        tables = [(f"l{l}.{n}", i, o) for l in range(L) for (n, i, o) in proj]
        C, rc, S, ru, dt = 8, 64, 256, 1, "bf16"
        Tn = T or 8192
        lens = segment_lengths(_rng(cfg, seed, _K_SEGLEN), S, 1, 512, Tn) if Tn >= S else \
            np.ones(Tn, np.int64)
        n_users = len(lens)
        c_of_user = rng.integers(0, C, size=S).astype(np.int32)
        tok_u = np.repeat(np.arange(n_users, dtype=np.int32), lens)
        tok_c = c_of_user[tok_u]
        slot_rank = np.full(S, ru, np.int32)
        user_of_tok = tok_u.copy()
        meta["seg_lens"] = lens
        n_users = S
    elif cfg == 4:
        L = layers if layers is not None else 1
        proj = decoder_projections(LLAMA31_8B["hidden"], LLAMA31_8B["kv"], LLAMA31_8B["inter"])
        tables = [(f"l{l}.{n}", i, o) for l in range(L) for (n, i, o) in proj]
        C, rc, S, ru, dt = 16, 32, 1024, 2, "bf16"
        Tn = T or 256
        c_of_user = rng.integers(0, C, size=S).astype(np.int32)
        tok_u = rng.choice(S, size=Tn, replace=False).astype(np.int32)
        tok_c = c_of_user[tok_u]
        slot_rank = np.full(S, ru, np.int32)
        meta["swap_slots"] = np.sort(rng.choice(tok_u, size=min(32, Tn), replace=False)).astype(np.int32)
        user_of_tok = tok_u.copy()
        n_users = S
    elif cfg == 5:
        proj = decoder_projections(LLAMA32_3B["hidden"], LLAMA32_3B["kv"], LLAMA32_3B["inter"])
        L = layers if layers is not None else 1
        tables = [(f"l{l}.{n}", i, o) for l in range(L) for (n, i, o) in proj]
        S, dt = 2000, "bf16"
        Tn = T or 512
        pmf = truncated_zipf_pmf(1.1, S)
        tok_u = rng.choice(S, size=Tn, p=pmf).astype(np.int32)
        rank_of_user = rng.integers(1, 3, size=S).astype(np.int32)
        c_of_user = rng.integers(0, 8, size=S).astype(np.int32)
        if baseline:
            C, rc, ru = 0, 0, 16
            slot_rank = np.full(S, 16, np.int32)
            tok_c = np.full(Tn, -1, np.int32)
        else:
            C, rc, ru = 8, 64, 2
            slot_rank = rank_of_user
            tok_c = c_of_user[tok_u]
        user_of_tok = tok_u.copy()
        n_users = S
        meta["baseline"] = baseline
    else:
        raise ValueError(f"unknown config {cfg}")

    g = None
    if gamma == "bins":
        g = _gamma_per_user(cfg, seed, n_users)[user_of_tok].astype(np.float32)
    elif gamma != "one":
        raise ValueError(gamma)
    if exact:
        y0 = "int" if y0 != "zero" else "zero"
        if g is not None:
            raise ValueError("the exact variant keeps gamma = 1")
    name = {1: "tiny fp32 256x256", 2: "llama3.2-3b q_proj decode T=64",
            3: "llama3.2-3b 28-layer prefill T=8192", 4: "llama3.1-8b decode T=256 (1024 slots)",
            5: "llama3.2-3b zipf multi-tenant T=512"}[cfg]
    if baseline:
        name += " (rank-16 LoRA baseline)"
    return Workload(cfg=cfg, seed=seed, name=name, dtype=dt, tables=tables, n_centroids=C, r_c=rc,
                    n_slots=S, r_u_max=ru, slot_rank=slot_rank.astype(np.int32),
                    tok_c=np.ascontiguousarray(tok_c, np.int32), tok_u=np.ascontiguousarray(tok_u, np.int32),
                    gamma=g, y0_kind=y0, exact=exact, user_of_slot=None, meta=meta)
