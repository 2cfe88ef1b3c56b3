"""The two ways an apply sums its split-K partials.

Default: fp32 device atomics in arrival order.  SALT_DETERMINISTIC: a fixed-order
sum, which makes y bit-reproducible.  Both must meet the oracle bound; the
deterministic mode must also give identical bytes on repeated applies, and the
integer-valued variants must be bit-exact in either mode.
"""
import numpy as np
import pytest

import oracle
from paper_2608_03579_amd import synth
from tests.gpu_harness import TOL_F32, TOL_NORTH_STAR, Run, close_enough

pytestmark = pytest.mark.gpu


def _announce(name):
    print(f"\n[gpu case] {name}", flush=True)


def _tol(w):
    return TOL_F32 if w.dtype == "f32" else TOL_NORTH_STAR


CASES = [
    ("tiny fp32", lambda: synth.make(1, 0, y0="normal"), [0], None),
    ("q_proj decode", lambda: synth.make(2, 0, y0="normal"), [0], None),
    ("zipf T=512", lambda: synth.make(5, 1), [0, 4, 6], None),
    ("prefill 1 layer T=2048", lambda: synth.make(3, 1, layers=1, T=2048), [0, 6],
     list(range(0, 2048, 5)) + [2047]),
]


@pytest.mark.parametrize("name,make,tables,rows", CASES, ids=[c[0] for c in CASES])
def test_deterministic_mode_parity_and_reproducibility(name, make, tables, rows):
    _announce(f"deterministic mode: {name}")
    w = make()
    run = Run(w, deterministic=True)
    try:
        run.set_and_build()
        for t in tables:
            first = run.apply(t)
            assert run.plan.errors(run.stream) == 0
            got = oracle.decode(first, w.dtype)
            ref = run.oracle_table(t, rows)
            if rows is not None:
                got = got[np.asarray(rows)]
            ok, worst, nbad = close_enough(got, ref, _tol(w))
            assert ok, f"table {t}: {nbad} out of tolerance, worst {worst:.3f}x"
            for _ in range(2):
                assert np.array_equal(run.apply(t), first), f"table {t}: not bit-reproducible"
    finally:
        run.close()


def test_modes_agree_and_integer_inputs_are_exact_in_both():
    _announce("atomic vs deterministic sums, exact-integer q_proj")
    w = synth.make(2, 5, exact=True, y0="int")
    outs = []
    for det in (False, True):
        run = Run(w, deterministic=det)
        try:
            run.set_and_build()
            y = oracle.decode(run.apply(0), w.dtype)
            assert run.plan.errors(run.stream) == 0
            assert np.array_equal(y, run.oracle_table(0)), f"deterministic={det}"
            outs.append(y)
        finally:
            run.close()
    assert np.array_equal(outs[0], outs[1])


def test_atomic_mode_alternating_tables_and_rebuilds():
    """Atomic sums alternate between two v buffers, one cleared per apply: a run
    of applies over tables with different K splits, then a rebuild with a new
    batch, must stay exact on integer inputs."""
    _announce("atomic mode: 21 applies over 7 tables, rebuild, 7 more")
    w = synth.make(5, 2, exact=True, y0="int", T=160)
    run = Run(w)
    try:
        run.set_and_build()
        for k in range(21):
            t = (3 * k) % 7
            y = oracle.decode(run.apply(t), w.dtype)
            assert np.array_equal(y, run.oracle_table(t)), (k, t)
        tc = np.roll(w.tok_c, 17)
        tu = np.roll(w.tok_u, 5)
        run.set_and_build(tc, tu)
        for t in range(7):
            y = oracle.decode(run.apply(t), w.dtype)
            assert np.array_equal(y, run.oracle_table(t)), t
        assert run.plan.errors(run.stream) == 0
    finally:
        run.close()
