"""salt_apply_batch_noalloc (split-K partials in the library's static device
scratch, no allocation) against salt_apply_batch on the same plans and inputs,
through the C ABI: y must be bit-identical (same kernels, same K split), and
within the benchmark spec's bound of the oracle.  Two calls in a row on one stream,
the second on a smaller batch (the scratch keeps the first call's contents,
which the second must not see), then a launch whose partials cannot fit the
scratch, which must be refused before anything is enqueued.
"""
import numpy as np
import pytest

import oracle
from paper_2608_03579_amd import synth
from tests.gpu_harness import TOL_BF16, Run, close_enough, to_dev

pytestmark = pytest.mark.gpu


def _announce(name):
    print(f"\n[gpu case] {name}", flush=True)


def _both(run, tables, rows):
    """y of salt_apply_batch and of salt_apply_batch_noalloc for the plan's
    current maps (token i of the batch is workload row rows[i])."""
    w = run.w
    xs = [to_dev(np.ascontiguousarray(w.x(t)[rows])) for t in tables]
    out = []
    for noalloc in (False, True):
        ys = [to_dev(np.ascontiguousarray(w.y0(t)[rows])) for t in tables]
        f = run.ctx.apply_batch_noalloc if noalloc else run.ctx.apply_batch
        f(tables, run.plan, [d.ptr for d in xs], [d.ptr for d in ys], run.stream)
        run._stream.synchronize()
        out.append([d.to_host() for d in ys])
        for d in ys:
            d.free()
    for d in xs:
        d.free()
    return out


def _oracle(run, table, rows):
    w, d = run.w, run.w.dtype
    tok_c, tok_u, _ = run.maps
    x = oracle.decode(w.x(table), d)[rows]
    y0 = oracle.decode(w.y0(table), d)[rows]
    cat, cb = (oracle.decode(a, d) for a in w.centroids(table))
    res = {int(s): tuple(oracle.decode(a, d) for a in w.residual(int(s), table)) for s in np.unique(tok_u[tok_u >= 0])}
    return oracle.apply(x, y0, cat, cb, res, tok_c, tok_u, None)


def test_noalloc_matches_apply_batch_twice_then_smaller():
    _announce("salt_apply_batch_noalloc vs salt_apply_batch: zipf layer T=512, then T=200")
    w = synth.make(5, 0)
    run = Run(w)
    tables = list(range(len(w.tables)))
    try:
        for T in (w.T, 200):
            rows = np.arange(T)
            tok_c, tok_u = w.tok_c[:T].copy(), w.tok_u[:T].copy()
            run.plan.set_maps(tok_c, tok_u, None, run.stream)
            run.plan.build(run.stream)
            run.maps = (tok_c, tok_u, None)
            ref_y, na_y = _both(run, tables, rows)
            for t, a, b in zip(tables, ref_y, na_y):
                assert np.array_equal(a, b), f"T={T} table {t}: noalloc differs from salt_apply_batch"
                ok, worst, nbad = close_enough(oracle.decode(b, w.dtype), _oracle(run, t, rows), TOL_BF16)
                assert ok, f"T={T} table {t}: {nbad} out of tolerance, worst {worst:.3f}x"
            assert run.plan.errors(run.stream) == 0
    finally:
        run.close()


def test_noalloc_refuses_partials_beyond_the_scratch():
    """16 tables of 8192 tokens at r_c = 128 + r_u = 16 (144 ranks): even one K
    range per table needs 16 x 8192 x 144 floats, more than the 16 Mi floats of
    the scratch; salt_apply_batch on the same plan still runs."""
    _announce("salt_apply_batch_noalloc: partials beyond the scratch are refused")
    from paper_2608_03579_amd import salt
    tables = [(64, 64)] * 16
    T = 8192
    ctx = salt.Context("bf16", tables, 1, 128, 4, 16, T)
    try:
        rng = np.random.default_rng(5)
        bits = lambda shape: synth.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * 0.05)
        for t in range(16):
            ctx.pin_centroids(t, bits((1, 128, 64)), bits((1, 128, 64)))
        ctx.load_residual(0, 16, bits(ctx.residual_bytes(16) // 2))
        ctx.wait_loads()
        from tests.gpu_harness import hipmod
        stream = hipmod().Stream()
        plan = ctx.plan()
        tok_c = np.zeros(T, np.int32)
        tok_u = np.zeros(T, np.int32)
        plan.set_maps(tok_c, tok_u, None, stream.h)
        plan.build(stream.h)
        xs = [to_dev(np.zeros((T, 64), np.uint16)) for _ in range(16)]
        ys = [to_dev(np.zeros((T, 64), np.uint16)) for _ in range(16)]
        st = ctx.apply_batch_noalloc_status(list(range(16)), plan, [d.ptr for d in xs], [d.ptr for d in ys], stream.h)
        assert st == salt.ERR_OUT_OF_RANGE, st
        assert "static scratch" in salt.lib.salt_last_error(ctx.h).decode()
        ctx.apply_batch(list(range(16)), plan, [d.ptr for d in xs], [d.ptr for d in ys], stream.h)
        stream.synchronize()
        for d in xs + ys:
            d.free()
        plan.close()
        stream.destroy()
    finally:
        ctx.close()
