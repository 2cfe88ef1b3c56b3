"""GPU edge cases, error paths and swap ordering of the libsalt C ABI.

Every case prints its name before touching the GPU.  Expected values come from
the CPU oracle on the same seeded inputs.
"""
import numpy as np
import pytest

import oracle
from paper_2608_03579_amd import synth
from tests.gpu_harness import TOL_F32, TOL_BF16, Run, close_enough

pytestmark = pytest.mark.gpu


def _announce(name):
    print(f"\n[gpu case] {name}", flush=True)


def _tol(w):
    return TOL_F32 if w.dtype == "f32" else TOL_BF16


def _check(run, table=0, rows=None):
    got = oracle.decode(run.apply(table), run.w.dtype)
    ref = run.oracle_table(table, rows)
    if rows is not None:
        got = got[np.asarray(rows)]
    ok, worst, nbad = close_enough(got, ref, _tol(run.w))
    assert ok, f"{nbad} elements out of tolerance, worst {worst:.3f}x"


def _plan_matches(run):
    p = run.plan.download(run.stream)
    want = oracle.plan(run.maps[0], run.maps[1])
    for k in want:
        assert np.array_equal(p[k], want[k]), k
    assert run.plan.errors(run.stream) == 0


@pytest.mark.parametrize("cfg", [1, 2])
def test_term_absent_cases(cfg):
    """c = -1 (residual only), u = -1 (centroid only), both -1 (y untouched)."""
    _announce(f"absent terms cfg={cfg}")
    w = synth.make(cfg, 5, y0="normal")
    run = Run(w)
    try:
        T = w.T
        rng = np.random.default_rng(9)
        cases = {
            "no centroid": (np.full(T, -1, np.int32), w.tok_u),
            "no residual": (w.tok_c, np.full(T, -1, np.int32)),
            "neither": (np.full(T, -1, np.int32), np.full(T, -1, np.int32)),
            "mixed": (np.where(rng.random(T) < 0.3, -1, w.tok_c).astype(np.int32),
                      np.where(rng.random(T) < 0.3, -1, w.tok_u).astype(np.int32)),
        }
        for name, (tc, tu) in cases.items():
            run.set_and_build(tc, tu)
            _plan_matches(run)
            _check(run)
        # both absent: bit-identical y
        run.set_and_build(cases["neither"][0], cases["neither"][1])
        assert np.array_equal(run.apply(0), w.y0(0))
    finally:
        run.close()


def test_ragged_and_degenerate_batches():
    _announce("ragged batch sizes, T = 0 and T = 1, one big centroid group")
    w = synth.make(2, 6, y0="normal")
    run = Run(w)
    try:
        for k, T in enumerate((1, 5, 17, 33, 63)):
            run.set_and_build(w.tok_c[:T], w.tok_u[:T])
            if k % 2 == 0:
                _plan_matches(run)
            got = oracle.decode(run.apply(0), w.dtype)[:T]
            if k % 2 == 1:
                _plan_matches(run)
            ref = run.oracle_table(0, rows=list(range(T)))
            assert close_enough(got, ref, TOL_BF16)[0], T
            # rows past T are untouched
            assert np.array_equal(run.apply(0)[T:], w.y0(0)[T:])
        # one centroid for everyone: a group spanning several tiles
        run.set_and_build(np.zeros(w.T, np.int32), w.tok_u)
        _plan_matches(run)
        _check(run)
        # empty batch: plan is empty, apply is a no-op
        run.set_and_build(np.zeros(0, np.int32), np.zeros(0, np.int32))
        p = run.plan.download(run.stream)
        assert p["perm"].size == 0 and p["seg_off"].tolist() == [0] and p["grp_off"].tolist() == [0]
        assert np.array_equal(run.apply(0), w.y0(0))
    finally:
        run.close()


def test_rank_zero_and_mixed_rank_slots():
    _announce("rank-0 slots and ranks 1/2 in one batch")
    w = synth.make(5, 2, layers=1, T=160)
    run = Run(w)
    try:
        # empty the residual term of a few referenced slots
        slots = w.referenced_slots()[:5]
        for s in slots:
            run.ctx.load_residual(int(s), 0, None)
            run.w.slot_rank[int(s)] = 0
        run.ctx.wait_loads()
        run.set_and_build()
        _plan_matches(run)
        for t in (0, 6):
            _check(run, t)
    finally:
        run.close()


def test_repeated_applies_and_rebuilds():
    """Many applies of one plan (its partials buffer reused each time), then
    rebuilds with batches of a different tiling."""
    _announce("40 applies on one plan, then rebuilds")
    w = synth.make(2, 7)
    run = Run(w)
    try:
        run.set_and_build()
        x = w.x(0)
        from tests.gpu_harness import to_dev
        xd, yd = to_dev(x), to_dev(w.y0(0))
        for _ in range(40):
            run.ctx.apply(0, run.plan, xd.ptr, yd.ptr, run.stream)
        run._stream.synchronize()
        got = oracle.decode(yd.to_host(), w.dtype)
        one = run.oracle_table(0) - oracle.decode(w.y0(0), w.dtype)
        ref = oracle.decode(w.y0(0), w.dtype) + 40 * one
        # 40 bf16 roundings of the running y: allow 40x the per-step bound
        assert np.all(np.abs(got - ref) <= 40 * TOL_BF16 * (1 + np.abs(ref)))
        for seed in (8, 9):
            w2 = synth.make(2, seed)
            run.set_and_build(w2.tok_c, w2.tok_u)
            _plan_matches(run)
            _check(run)
    finally:
        run.close()


def test_api_errors_change_no_state():
    from paper_2608_03579_amd import salt
    _announce("api error paths")
    w = synth.make(2, 1)
    run = Run(w)
    try:
        ctx, plan = run.ctx, run.plan
        T = w.T
        st = plan.set_maps_status
        assert st(np.full(T, 4, np.int32), w.tok_u) == salt.ERR_OUT_OF_RANGE           # c >= C
        assert st(w.tok_c, np.full(T, 64, np.int32)) == salt.ERR_OUT_OF_RANGE          # u >= n_slots
        assert st(np.full(T, -2, np.int32), w.tok_u) == salt.ERR_OUT_OF_RANGE
        assert st(np.zeros(T + 1, np.int32), np.zeros(T + 1, np.int32)) == salt.ERR_OUT_OF_RANGE   # > max_tokens
        g = np.ones(T, np.float32)
        g[3] = np.nan
        assert st(w.tok_c, w.tok_u, g) == salt.ERR_INVALID_ARG
        # residual loads: range, size, pageable memory
        nb = ctx.residual_bytes(2)
        blob = np.zeros(nb, np.uint8)
        assert ctx.load_residual_ptr(64, 2, blob.ctypes.data, nb) == salt.ERR_OUT_OF_RANGE
        assert ctx.load_residual_ptr(0, 3, blob.ctypes.data, nb) == salt.ERR_OUT_OF_RANGE
        assert ctx.load_residual_ptr(0, 2, blob.ctypes.data, nb - 2) == salt.ERR_INVALID_ARG
        assert ctx.load_residual_ptr(0, 2, blob.ctypes.data, nb) == salt.ERR_NOT_PINNED
        # the calls above changed nothing: the real batch still applies correctly
        run.set_and_build()
        _check(run)
        # apply: table out of range
        from tests.gpu_harness import to_dev
        xd, yd = to_dev(w.x(0)), to_dev(w.y0(0))
        assert ctx.apply_status(1, plan, xd.ptr, yd.ptr, run.stream) == salt.ERR_OUT_OF_RANGE
        # a slot of the plan reloaded with another rank: the plan is stale
        s0 = int(w.tok_u[0])
        ctx.load_residual(s0, 1, np.zeros(ctx.residual_bytes(1) // 2, np.uint16))
        ctx.wait_loads()
        assert ctx.apply_status(0, plan, xd.ptr, yd.ptr, run.stream) == salt.ERR_BAD_STATE
        # never-loaded slot
        fresh = salt.Context(w.dtype, [(3072, 3072)], 4, 32, 8, 2, 16)
        p2 = fresh.plan()
        assert p2.set_maps_status(np.zeros(2, np.int32), np.array([0, 1], np.int32)) == salt.ERR_SLOT_EMPTY
        # centroids of the table never pinned
        fresh.load_residual(0, 2, np.zeros(fresh.residual_bytes(2) // 2, np.uint16))
        fresh.wait_loads()
        p2.set_maps(np.zeros(2, np.int32), np.zeros(2, np.int32))
        p2.build()
        assert fresh.apply_status(0, p2, xd.ptr, yd.ptr, 0) == salt.ERR_BAD_STATE
        p2.close()
        fresh.close()
    finally:
        run.close()


def test_swap_is_ordered_after_inflight_apply():
    """Reloading a slot right after an apply is enqueued must not change what
    that apply reads; the next apply sees the new residual."""
    _announce("swap ordering against an in-flight apply")
    w = synth.make(4, 3)
    run = Run(w)
    try:
        run.set_and_build()
        from tests.gpu_harness import to_dev
        t = 4                                            # gate_proj 4096 -> 14336
        xd, y1 = to_dev(w.x(t)), to_dev(w.y0(t))
        run.ctx.apply(t, run.plan, xd.ptr, y1.ptr, run.stream)
        swapped = [int(s) for s in w.meta["swap_slots"]]
        for s in swapped:
            run.load(s, 1)                               # enqueued behind the apply's reads
        y2 = to_dev(w.y0(t))
        run.ctx.apply(t, run.plan, xd.ptr, y2.ptr, run.stream)
        run._stream.synchronize()
        run.ctx.wait_loads()
        got1 = oracle.decode(y1.to_host(), w.dtype)
        got2 = oracle.decode(y2.to_host(), w.dtype)
        ref2 = run.oracle_table(t)                       # gen 1 for the swapped slots
        for s in swapped:
            run.gen[s] = 0
        ref1 = run.oracle_table(t)
        assert close_enough(got1, ref1, TOL_BF16)[0]
        assert close_enough(got2, ref2, TOL_BF16)[0]
        assert not close_enough(got1, ref2, TOL_BF16)[0]
    finally:
        run.close()


def test_swap_waits_for_applies_of_replaced_maps_and_other_streams():
    """The reader event of a plan's applies is recorded lazily: when the plan's
    maps are replaced, when the plan moves to another stream, or when a slot it
    references is swapped.  Each of those must still order a later swap behind
    the applies that read the slot."""
    _announce("swap ordering: replaced maps, second stream")
    from paper_2608_03579_amd import hip
    from tests.gpu_harness import to_dev
    w = synth.make(4, 3)
    run = Run(w)
    try:
        run.set_and_build()
        t = 4
        swapped = [int(s) for s in w.meta["swap_slots"]]
        xd = to_dev(w.x(t))
        # (1) apply, then new maps without the swapped slots, then the swap
        y1 = to_dev(w.y0(t))
        run.ctx.apply(t, run.plan, xd.ptr, y1.ptr, run.stream)
        keep = ~np.isin(w.tok_u, swapped)
        tok_u2 = np.where(keep, w.tok_u, -1).astype(np.int32)
        run.plan.set_maps(w.tok_c, tok_u2, w.gamma, run.stream)
        for s in swapped:
            run.load(s, 1)
        run._stream.synchronize()
        run.ctx.wait_loads()
        got1 = oracle.decode(y1.to_host(), w.dtype)
        for s in swapped:
            run.gen[s] = 0
        ref1 = run.oracle_table(t)
        assert close_enough(got1, ref1, TOL_BF16)[0], "swap overtook an apply of the replaced maps"
        # (2) the plan applied on a second stream, then the swap back to generation 0
        run.plan.set_maps(w.tok_c, w.tok_u, w.gamma, run.stream)
        run.plan.build(run.stream)
        for s in swapped:
            run.gen[s] = 1
        other = hip.Stream()
        run._stream.synchronize()
        y2, y3 = to_dev(w.y0(t)), to_dev(w.y0(t))
        run.ctx.apply(t, run.plan, xd.ptr, y2.ptr, run.stream)
        run._stream.synchronize()                    # applies of one plan are ordered
        run.ctx.apply(t, run.plan, xd.ptr, y3.ptr, other.h)
        for s in swapped:
            run.load(s, 0)
        run._stream.synchronize()
        other.synchronize()
        run.ctx.wait_loads()
        for s in swapped:
            run.gen[s] = 1                           # what both applies read (run.load set 0)
        ref_gen1 = run.oracle_table(t)
        assert close_enough(oracle.decode(y2.to_host(), w.dtype), ref_gen1, TOL_BF16)[0]
        assert close_enough(oracle.decode(y3.to_host(), w.dtype), ref_gen1, TOL_BF16)[0]
        other.destroy()
    finally:
        run.close()


def test_prefill_full_size_sampled():
    """28-layer Llama-3.2-3B prefill at full size (196 tables, T = 8192), the
    shapes and launch configuration bench.py times; sampled tables and rows."""
    _announce("cfg3 full size: 196 tables, T=8192, sampled tables/rows")
    w = synth.make(3, 0)
    run = Run(w)
    try:
        run.set_and_build()
        _plan_matches(run)
        rng = np.random.default_rng(3)
        seg = np.cumsum(w.meta["seg_lens"])
        rows = sorted(set(rng.choice(w.T, 96, replace=False).tolist()) | {0, w.T - 1} |
                      set((seg[:20] - 1).tolist()))
        for t in (0, 1, 4, 6, 97, 195):
            _check(run, t, rows=rows)
    finally:
        run.close()


def test_timed_batch_matches_batch_and_times_both_kernels():
    """salt_apply_batch_timed runs the same apply (bit-identical: the partial sums
    are added in a fixed order); its four events bracket the shrink and the
    expand kernels."""
    _announce("salt_apply_batch_timed on three zipf tables")
    from paper_2608_03579_amd import hip, salt
    from tests.gpu_harness import to_dev
    w = synth.make(5, 11, y0="normal")
    run = Run(w)
    try:
        run.set_and_build()
        tables = [0, 4, 6]
        want = run.apply_batch(tables)
        xd = [to_dev(w.x(t)) for t in tables]
        yd = [to_dev(w.y0(t)) for t in tables]
        ev = [hip.Event() for _ in range(4)]
        run.ctx.apply_batch_timed(tables, run.plan, [d.ptr for d in xd], [d.ptr for d in yd], run.stream,
                                  [e.h for e in ev])
        run._stream.synchronize()
        for d, y in zip(yd, want):
            assert np.array_equal(d.to_host(), y)
        shrink_ms, expand_ms = ev[0].elapsed_ms(ev[1]), ev[2].elapsed_ms(ev[3])
        assert 0.0 < shrink_ms < 100.0 and 0.0 < expand_ms < 100.0, (shrink_ms, expand_ms)
        assert ev[1].elapsed_ms(ev[2]) >= 0.0                  # the expand starts after the shrink ends
        nul = salt.C.c_void_p * 4
        st = salt.lib.salt_apply_batch_timed(run.ctx.h, 1, salt._i32p(np.zeros(1, np.int32)), run.plan.h,
                                             run.ctx._ptrs([xd[0].ptr]), run.ctx._ptrs([yd[0].ptr]), run.stream,
                                             nul(ev[0].h, None, ev[2].h, ev[3].h))
        assert st == salt.ERR_INVALID_ARG
        for e in ev:
            e.destroy()
    finally:
        run.close()


def test_repeated_applies_are_bit_identical():
    """The split-K partials are summed in a fixed order: the same call on equal
    inputs gives equal bytes, apply after apply.  The K split depends on the
    tables that share a launch, so a table applied alone and inside a batch agree
    within the tolerance, not necessarily bit for bit."""
    _announce("bit-identical repeats: q_proj decode, zipf layer")
    for cfg, tables in ((2, [0]), (5, [0, 1, 2, 3, 4, 5, 6])):
        w = synth.make(cfg, 12, y0="normal")
        run = Run(w)
        try:
            run.set_and_build()
            first = run.apply_batch(tables)
            for _ in range(3):
                for a, b in zip(first, run.apply_batch(tables)):
                    assert np.array_equal(a, b)
            for t, y in zip(tables, first):
                alone = run.apply(t)
                assert np.array_equal(alone, run.apply(t))
                assert close_enough(oracle.decode(alone, w.dtype), oracle.decode(y, w.dtype), TOL_BF16)[0]
        finally:
            run.close()


def test_plan_used_across_streams():
    """Set maps and build on one stream, then apply on another without any host
    synchronisation: the library orders the plan's work across streams."""
    _announce("plan built on stream 1, applied on stream 2")
    from paper_2608_03579_amd import hip
    from tests.gpu_harness import to_dev
    w = synth.make(5, 13)
    run = Run(w)
    try:
        s2 = hip.Stream()
        xd, yd = to_dev(w.x(4)), to_dev(w.y0(4))
        for rep in range(3):
            run.plan.set_maps(w.tok_c, w.tok_u, w.gamma, run.stream)
            run.plan.build(run.stream)
            run.maps = (w.tok_c, w.tok_u, w.gamma)
            yd.upload(w.y0(4))
            run.ctx.apply(4, run.plan, xd.ptr, yd.ptr, s2.h)
            s2.synchronize()
            got = oracle.decode(yd.to_host(), w.dtype)
            assert close_enough(got, run.oracle_table(4), TOL_BF16)[0], rep
        # and the other way round: build on stream 2, apply on stream 1
        run.plan.set_maps(w.tok_c, w.tok_u, w.gamma, s2.h)
        run.plan.build(s2.h)
        yd.upload(w.y0(4))
        run.ctx.apply(4, run.plan, xd.ptr, yd.ptr, run.stream)
        run._stream.synchronize()
        assert close_enough(oracle.decode(yd.to_host(), w.dtype), run.oracle_table(4), TOL_BF16)[0]
        _plan_matches(run)
        s2.destroy()
    finally:
        run.close()


def test_apply_map_one_shot():
    """salt_apply_map: the context's own plan, built and applied on host maps,
    batch after batch of different sizes."""
    _announce("salt_apply_map")
    from paper_2608_03579_amd import salt
    from tests.gpu_harness import to_dev
    w = synth.make(2, 14, y0="normal")
    run = Run(w)
    try:
        for T in (64, 17, 1, 64):
            xd, yd = to_dev(w.x(0)), to_dev(w.y0(0))
            run.ctx.apply_map(0, w.tok_c[:T], w.tok_u[:T], None, xd.ptr, yd.ptr, run.stream)
            run._stream.synchronize()
            got = oracle.decode(yd.to_host(), w.dtype)
            run.maps = (w.tok_c[:T], w.tok_u[:T], None)
            ref = run.oracle_table(0, rows=list(range(T)))
            assert close_enough(got[:T], ref, TOL_BF16)[0], T
            assert np.array_equal(yd.to_host()[T:], w.y0(0)[T:])
        assert run.ctx.apply_map_status(1, w.tok_c, w.tok_u, None, xd.ptr, yd.ptr, run.stream) == \
            salt.ERR_OUT_OF_RANGE
        assert run.ctx.apply_map_status(0, np.full(w.T, 9, np.int32), w.tok_u, None, xd.ptr, yd.ptr,
                                        run.stream) == salt.ERR_OUT_OF_RANGE
    finally:
        run.close()


def test_batched_swaps():
    """salt_load_residuals: 32 swaps in one call, validated as a whole, ordered
    behind the applies that read the old residuals."""
    _announce("salt_load_residuals: 32 rank-2 swaps of the 8B decode batch")
    from paper_2608_03579_amd import salt
    from tests.gpu_harness import to_dev
    w = synth.make(4, 3)
    run = Run(w)
    try:
        run.set_and_build()
        t = 6
        xd, y1 = to_dev(w.x(t)), to_dev(w.y0(t))
        run.ctx.apply(t, run.plan, xd.ptr, y1.ptr, run.stream)
        swapped = [int(s) for s in w.meta["swap_slots"]]
        nb = run.ctx.residual_bytes(2)
        bufs = [salt.HostBuffer(nb) for _ in swapped]
        for b, s in zip(bufs, swapped):
            b.view(np.uint16)[:] = w.residual_blob(s, 1)
        # an invalid entry fails the whole call and changes nothing
        bad = list(swapped)
        bad[5] = 1 << 20
        assert run.ctx.load_residuals_ptr(bad, [2] * 32, [b.ptr for b in bufs], [nb] * 32) == salt.ERR_OUT_OF_RANGE
        assert run.ctx.load_residuals_ptr(swapped, [2] * 32, [b.ptr for b in bufs], [nb] * 31 + [nb - 2]) == \
            salt.ERR_INVALID_ARG
        assert run.ctx.load_residuals_ptr(swapped, [2] * 32, [b.ptr for b in bufs], [nb] * 32) == salt.OK
        for s in swapped:
            run.gen[s] = 1
        y2 = to_dev(w.y0(t))
        run.ctx.apply(t, run.plan, xd.ptr, y2.ptr, run.stream)
        run._stream.synchronize()
        run.ctx.wait_loads()
        ref_new = run.oracle_table(t)
        assert close_enough(oracle.decode(y2.to_host(), w.dtype), ref_new, TOL_BF16)[0]
        for s in swapped:
            run.gen[s] = 0
        assert close_enough(oracle.decode(y1.to_host(), w.dtype), run.oracle_table(t), TOL_BF16)[0]
        for b in bufs:
            b.free()
    finally:
        run.close()


def test_swap_paths_many_blobs_and_a_repeated_slot():
    """salt_load_residuals past one gather launch (100 blobs from salt_host_alloc
    memory: launches of 64 and 36), then a call that lists a slot twice (ordered
    DMA copies: the last blob wins); after each, an apply that reads the swapped
    slots is compared with the oracle."""
    _announce("salt_load_residuals: 100 gathered swaps, then a slot listed twice")
    from paper_2608_03579_amd import salt
    from tests.gpu_harness import to_dev
    w = synth.make(4, 5)
    run = Run(w)
    bufs = []
    try:
        run.set_and_build()
        slots = [int(s) for s in w.referenced_slots() if int(w.slot_rank[s]) == 2][:100]
        assert len(slots) == 100
        nb = run.ctx.residual_bytes(2)
        bufs = [salt.HostBuffer(nb) for _ in slots]
        for b, s in zip(bufs, slots):
            b.view(np.uint16)[:] = w.residual_blob(s, 1)
        assert run.ctx.load_residuals_ptr(slots, [2] * 100, [b.ptr for b in bufs], [nb] * 100) == salt.OK
        for s in slots:
            run.gen[s] = 1
        t = 2
        xd = to_dev(w.x(t))

        def check():
            y = to_dev(w.y0(t))
            run.ctx.apply(t, run.plan, xd.ptr, y.ptr, run.stream)
            run._stream.synchronize()
            run.ctx.wait_loads()
            ok, worst, nbad = close_enough(oracle.decode(y.to_host(), w.dtype), run.oracle_table(t), TOL_BF16)
            assert ok, f"{nbad} out of tolerance, worst {worst:.3f}x"

        check()
        s0 = slots[0]
        b2, b3 = salt.HostBuffer(nb), salt.HostBuffer(nb)
        bufs += [b2, b3]
        b2.view(np.uint16)[:] = w.residual_blob(s0, 2)
        b3.view(np.uint16)[:] = w.residual_blob(s0, 3)
        assert run.ctx.load_residuals_ptr([s0, slots[1], s0], [2, 2, 2], [b2.ptr, bufs[1].ptr, b3.ptr],
                                          [nb] * 3) == salt.OK
        run.gen[s0] = 3
        check()
    finally:
        run.close()
        for b in bufs:
            b.free()


def test_plan_tiling_reports_the_launch_structure():
    """salt_plan_tiling: every apply is two launches; decode batches with short
    centroid groups take 16-token tiles, fp32 16, the Zipf batch 32 and the
    8192-token prefill 128; the tile count matches the centroid groups."""
    _announce("salt_plan_tiling")
    for cfg, kw, want in ((2, {}, (16, 2)), (1, {}, (16, 2)), (4, {}, (16, 2)), (5, {}, (32, 2)),
                          (3, {"layers": 1}, (128, 2))):
        w = synth.make(cfg, 0, **kw)
        run = Run(w, pin_tables=[])
        try:
            run.plan.set_maps(w.tok_c, w.tok_u, w.gamma, run.stream)
            m, n_tiles, launches = run.plan.tiling()
            assert (m, launches) == want, (cfg, m, launches)
            counts = np.bincount(w.tok_c + 1)
            assert n_tiles == int(sum((c + m - 1) // m for c in counts if c)), (cfg, n_tiles)
        finally:
            run.close()
