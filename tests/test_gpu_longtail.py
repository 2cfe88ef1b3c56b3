"""GPU parity of long-tail concatenated adapters (Sec. 3.3: for rare tasks the
scaled centroid and the residual are concatenated offline into one adapter of
rank r_c + r_u, e.g. 17 / 33 / 65, served by standard heterogeneous batching).

Such an adapter sits in a residual slot of rank r_c + r_u and its tokens carry
no centroid (c = -1); it shares the batch with centroid + residual tokens.
Residual ranks above 16 run in chunks of 16 ranks per shrink block.  Every
output is compared with the CPU oracle; in addition a user served both ways
(centroid c + its rank-r_u residual, and its concatenated adapter with c = -1)
must get the same output within the tolerance (the concatenation identity of
Sec. 3.3, on the GPU).
"""
import numpy as np
import pytest

import oracle
from paper_2608_03579_amd import synth
from tests.gpu_harness import TOL_F32, TOL_BF16, Run, close_enough

pytestmark = pytest.mark.gpu


def _announce(name):
    print(f"\n[gpu case] {name}", flush=True)


def _workload(seed, tables, C, r_c, T, n_reg, n_tail, dtype="bf16", r_u_hi=2):
    """n_reg regular users (slot k: rank 1..r_u_hi, centroid drawn), n_tail users served
    by concatenated adapters (slot n_reg + k: rank r_c + rank of slot k, the
    centroid and residual of regular user k); tokens drawn over all of them."""
    rng = np.random.default_rng(np.random.SeedSequence([2608, 3579, 77, seed]))
    n_slots = n_reg + n_tail
    slot_rank = np.zeros(n_slots, np.int32)
    slot_rank[:n_reg] = rng.integers(1, r_u_hi + 1, size=n_reg)
    user_c = rng.integers(0, C, size=n_reg).astype(np.int32)
    for k in range(n_tail):
        slot_rank[n_reg + k] = r_c + slot_rank[k]
    # every user gets at least one token; the rest at random
    users = np.concatenate([np.arange(n_slots), rng.integers(0, n_slots, size=T - n_slots)])
    rng.shuffle(users)
    tok_u = users.astype(np.int32)
    tok_c = np.where(users < n_reg, user_c[np.minimum(users, n_reg - 1)], -1).astype(np.int32)
    w = synth.ConcatTail(cfg=8, seed=seed, name="long-tail", dtype=dtype, tables=tables, n_centroids=C, r_c=r_c,
                 n_slots=n_slots, r_u_max=int(slot_rank.max()), slot_rank=slot_rank, tok_c=tok_c, tok_u=tok_u,
                 gamma=None, y0_kind="normal")
    w.concat = {n_reg + k: (int(user_c[k]), k) for k in range(n_tail)}
    return w


def _check(run, tol):
    w = run.w
    p = run.plan.download(run.stream)
    want = oracle.plan(run.maps[0], run.maps[1])
    for k in want:
        assert np.array_equal(p[k], want[k]), k
    for t in range(len(w.tables)):
        got = oracle.decode(run.apply(t), w.dtype)
        assert run.plan.errors(run.stream) == 0
        ok, worst, nbad = close_enough(got, run.oracle_table(t), tol)
        assert ok, f"table {t}: {nbad} out of tolerance, worst {worst:.3f}x"


def _both_ways(run, n_reg, n_tail):
    """Tokens of regular user k (centroid + residual) and of its concatenated twin
    (slot n_reg + k, no centroid) with the same x row get the same output."""
    w = run.w
    T = 2 * n_tail
    tok_c = np.concatenate([[w.concat[n_reg + k][0] for k in range(n_tail)], np.full(n_tail, -1)]).astype(np.int32)
    tok_u = np.concatenate([np.arange(n_tail), n_reg + np.arange(n_tail)]).astype(np.int32)
    run.set_and_build(tok_c, tok_u, None)
    for t in range(len(w.tables)):
        x = w.x(t)[np.concatenate([np.arange(n_tail), np.arange(n_tail)])]
        y0 = w.y0(t)[np.concatenate([np.arange(n_tail), np.arange(n_tail)])]
        got = oracle.decode(run.apply(t, x=x, y0=y0), w.dtype)
        ok, worst, nbad = close_enough(got[n_tail:], got[:n_tail], TOL_BF16 if w.dtype == "bf16" else TOL_F32)
        assert ok, f"table {t}: concatenated twin differs ({nbad}, worst {worst:.3f}x)"
        assert T == got.shape[0]


CASES = [
    # seed, tables, C, r_c, T, n_reg, n_tail, dtype
    (0, [("a", 520, 776), ("q", 3072, 3072)], 4, 16, 64, 24, 16, "bf16"),      # r = 17 / 18: two chunks
    (1, [("a", 776, 1032), ("k", 3072, 1024)], 4, 32, 128, 40, 24, "bf16"),   # r = 33 / 34
    (2, [("q", 3072, 3072), ("d", 8192, 3072)], 8, 64, 96, 32, 32, "bf16"),    # r = 65 / 66: five chunks
    (3, [("a", 1024, 264)], 2, 64, 512, 120, 60, "bf16"),                      # larger batch, 32-token tiles
    (4, [("tiny", 256, 256), ("a", 264, 520)], 4, 8, 64, 24, 16, "f32"),      # fp32, r = 9 / 10
]


@pytest.mark.parametrize("seed,tables,C,r_c,T,n_reg,n_tail,dtype", CASES)
def test_long_tail_mixed_batch(seed, tables, C, r_c, T, n_reg, n_tail, dtype):
    _announce(f"long tail r_c={r_c} T={T} {dtype}")
    w = _workload(seed, tables, C, r_c, T, n_reg, n_tail, dtype)
    run = Run(w)
    try:
        run.set_and_build()
        _check(run, TOL_BF16 if dtype == "bf16" else TOL_F32)
        _both_ways(run, n_reg, n_tail)
    finally:
        run.close()
