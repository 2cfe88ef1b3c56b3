"""Several plans of one context rotated through back-to-back batches with no host
synchronisation between them (Sec. 3.3: a server groups and serves one tenant
mix after another), the sequence ``bench.py`` runs.

Per step k, plan k mod 4 gets new maps (a different batch, sometimes a
different size), is built and applied to every table of the workload in one
salt_apply_batch into fresh y buffers, all on one stream.  Only after the last
step is the stream synchronised; then every step's outputs are compared with the
oracle on that step's maps, and every plan must report no device plan error.
"""
import numpy as np
import pytest

import oracle
from paper_2608_03579_amd import synth
from tests.gpu_harness import TOL_BF16, Run, close_enough, to_dev

pytestmark = pytest.mark.gpu


def _announce(name):
    print(f"\n[gpu case] {name}", flush=True)


def _step_maps(w, k):
    """Maps of step k over the slots and centroids loaded for w: a seeded
    shuffle of w's tokens, cut to a size that varies with k."""
    rng = np.random.default_rng(np.random.SeedSequence([2608, 3579, 99, w.cfg, k]))
    order = rng.permutation(w.T)
    sizes = (w.T, w.T, max(1, w.T // 3), w.T, max(1, (2 * w.T) // 3), 1)
    T = sizes[k % len(sizes)]
    tok_c = w.tok_c[order][:T].copy()
    tok_u = w.tok_u[order][:T].copy()
    if k % 5 == 3:                                   # some tokens without a centroid or a residual
        tok_c[rng.random(T) < 0.2] = -1
        tok_u[rng.random(T) < 0.2] = -1
    return tok_c.astype(np.int32), tok_u.astype(np.int32), order[:T]


@pytest.mark.parametrize("cfg,steps", [(2, 16), (4, 12), (5, 10)])
def test_rotating_plans_back_to_back(cfg, steps):
    _announce(f"cfg{cfg}: 4 plans rotated over {steps} steps without host sync")
    w = synth.make(cfg, 0)
    run = Run(w)
    n_plans = 4
    plans = [run.plan] + [run.ctx.plan() for _ in range(n_plans - 1)]
    tables = list(range(len(w.tables)))
    try:
        xs = [to_dev(w.x(t)) for t in tables]
        steps_io = []
        for k in range(steps):
            tok_c, tok_u, rows = _step_maps(w, k)
            T = len(tok_c)
            # x rows of this step: the shuffled tokens' rows, so each token keeps its own x
            xk = [to_dev(np.ascontiguousarray(w.x(t)[rows])) for t in tables]
            yk = [to_dev(np.ascontiguousarray(w.y0(t)[rows])) for t in tables]
            steps_io.append((tok_c, tok_u, rows, xk, yk))
        for k, (tok_c, tok_u, rows, xk, yk) in enumerate(steps_io):
            p = plans[k % n_plans]
            p.set_maps(tok_c, tok_u, None, run.stream)
            p.build(run.stream)
            run.ctx.apply_batch(tables, p, [d.ptr for d in xk], [d.ptr for d in yk], run.stream)
        run._stream.synchronize()
        for p in plans:
            assert p.errors(run.stream) == 0
        for k, (tok_c, tok_u, rows, xk, yk) in enumerate(steps_io):
            run.maps = (tok_c, tok_u, None)
            for j, t in enumerate(tables):
                got = oracle.decode(yk[j].to_host(), w.dtype)
                ref = _oracle_rows(run, t, rows)
                ok, worst, nbad = close_enough(got, ref, TOL_BF16)
                assert ok, f"step {k} table {t}: {nbad} out of tolerance, worst {worst:.3f}x"
        # the last maps of each plan are what it downloads
        for i, p in enumerate(plans):
            last = max(k for k in range(steps) if k % n_plans == i)
            got = p.download(run.stream)
            want = oracle.plan(steps_io[last][0], steps_io[last][1])
            for key in want:
                assert np.array_equal(got[key], want[key]), (i, key)
        for _, _, _, xk, yk in steps_io:
            for d in xk + yk:
                d.free()
        for d in xs:
            d.free()
    finally:
        for p in plans[1:]:
            p.close()
        run.close()


def _oracle_rows(run, table, rows):
    """The oracle on a step's batch: token i of the step is token rows[i] of the
    workload (its x and y0 rows) under the step's maps."""
    w = run.w
    d = w.dtype
    tok_c, tok_u, _ = run.maps
    x = oracle.decode(w.x(table), d)[rows]
    y0 = oracle.decode(w.y0(table), d)[rows]
    cat, cb = (oracle.decode(a, d) for a in w.centroids(table))
    res = {int(s): tuple(oracle.decode(a, d) for a in w.residual(int(s), table)) for s in np.unique(tok_u[tok_u >= 0])}
    return oracle.apply(x, y0, cat, cb, res, tok_c, tok_u, None)
