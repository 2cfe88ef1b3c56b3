"""GPU parity: libsalt (through the C ABI) against the fp64 CPU oracle.

Plans must match the oracle bit for bit.  Outputs must satisfy
|y - ref| <= 1e-2 * (1 + |ref|) element-wise for bf16 (fp32 accumulation), and
1e-5 * (1 + |ref|) for the fp32 Tiny workload; the integer-valued variants must be
bit-exact.  Multi-table workloads are applied both table by table (salt_apply)
and as one salt_apply_batch over a decoder layer's seven tables, the call the
bench times.  Every case prints its name before the GPU work starts.
"""
import numpy as np
import pytest

import oracle
from paper_2608_03579_amd import synth
from tests.gpu_harness import TOL_F32, TOL_BF16, Run, close_enough

pytestmark = pytest.mark.gpu


def _tol(w):
    return TOL_F32 if w.dtype == "f32" else TOL_BF16


def _check_plan(run):
    p = run.plan.download(run.stream)
    want = oracle.plan(run.maps[0], run.maps[1])
    for k in ("perm", "seg_off", "seg_c", "seg_u", "grp_off"):
        assert np.array_equal(p[k], want[k]), (k, p[k][:16], want[k][:16])
    assert run.plan.errors(run.stream) == 0, "device plan disagrees with the host's tiles"


def _compare(run, table, got, rows=None, exact=False):
    got = oracle.decode(got, run.w.dtype)
    ref = run.oracle_table(table, rows)
    if rows is not None:
        got = got[np.asarray(rows)]
    if exact:
        assert np.array_equal(got, ref), f"table {table}: {np.sum(got != ref)} exact mismatches"
        return
    ok, worst, nbad = close_enough(got, ref, _tol(run.w))
    assert ok, f"table {table}: {nbad} elements out of tolerance, worst {worst:.3f}x the bound"


def _check_table(run, table, rows=None, exact=False):
    _compare(run, table, run.apply(table), rows, exact)


def _check_batch(run, tables, rows=None, exact=False):
    for t, y in zip(tables, run.apply_batch(tables)):
        _compare(run, t, y, rows, exact)


def _announce(name):
    print(f"\n[gpu case] {name}", flush=True)


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("y0", ["zero", "normal"])
def test_tiny_fp32(seed, y0):
    _announce(f"tiny fp32 seed={seed} y0={y0}")
    run = Run(synth.make(1, seed, y0=y0))
    try:
        run.set_and_build()
        _check_plan(run)
        _check_table(run, 0)
    finally:
        run.close()


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_llama32_qproj_decode(seed):
    _announce(f"cfg2 q_proj decode seed={seed}")
    run = Run(synth.make(2, seed, y0="normal" if seed == 1 else "zero"))
    try:
        run.set_and_build()
        if seed == 2:
            _check_table(run, 0)         # apply before the plan is read back
            _check_plan(run)
        else:
            _check_plan(run)
            _check_table(run, 0)
    finally:
        run.close()


@pytest.mark.parametrize("cfg", [1, 2, 5])
def test_exact_integer_bit_exact(cfg):
    _announce(f"exact integer cfg={cfg}")
    w = synth.make(cfg, 3, exact=True, y0="int")
    run = Run(w)
    try:
        run.set_and_build()
        _check_plan(run)
        for t in range(len(w.tables)):
            _check_table(run, t, exact=True)
        if len(w.tables) > 1:
            _check_batch(run, list(range(len(w.tables))), exact=True)
    finally:
        run.close()


def test_gamma_bins():
    _announce("gamma bins cfg1 + cfg2 + cfg5")
    for cfg in (1, 2, 5):
        run = Run(synth.make(cfg, 4, gamma="bins"))
        try:
            run.set_and_build()
            _check_table(run, 0)
            if cfg == 5:
                _check_batch(run, [0, 4, 6])
        finally:
            run.close()


def test_llama31_decode_with_swaps():
    _announce("cfg4 llama3.1-8b decode T=256 with 32 swapped residuals")
    w = synth.make(4, 0)
    run = Run(w)
    try:
        for s in w.meta["swap_slots"]:
            run.load(int(s), 1)
        run.set_and_build()
        _check_batch(run, list(range(len(w.tables))))
        for t in (0, 6):
            _check_table(run, t)
        _check_plan(run)
    finally:
        run.close()


@pytest.mark.parametrize("baseline", [False, True])
def test_zipf_multitenant(baseline):
    _announce(f"cfg5 zipf T=512 baseline={baseline}")
    w = synth.make(5, 0, baseline=baseline)
    run = Run(w)
    try:
        run.set_and_build()
        _check_plan(run)
        _check_batch(run, list(range(len(w.tables))))
        _check_table(run, 3)
    finally:
        run.close()


def test_prefill_reduced():
    _announce("cfg3 prefill 1 layer, T=2048")
    w = synth.make(3, 0, layers=1, T=2048)
    run = Run(w)
    try:
        run.set_and_build()
        _check_plan(run)
        rows = list(range(0, w.T, 7)) + [w.T - 1]
        _check_batch(run, list(range(len(w.tables))), rows=rows)
    finally:
        run.close()


def test_prefill_full_layer_sampled():
    """One Llama-3.2-3B layer at the prefill's full size (T = 8192, 8 centroids of
    rank 64, 256 users of rank 1) in the launch configuration the bench times:
    128-token expand tiles over 64-token shrink tiles, one salt_apply_batch of the
    layer's 7 tables.  The plan is compared whole; outputs on sampled rows (every
    61st token and the last), which the oracle computes one by one."""
    _announce("cfg3 prefill, one layer at T=8192, salt_apply_batch of 7 tables, sampled rows")
    w = synth.make(3, 0, layers=1)
    assert w.T == 8192
    run = Run(w)
    try:
        run.set_and_build()
        m, _, launches = run.plan.tiling()
        assert (m, launches) == (128, 2)
        _check_plan(run)
        rows = list(range(0, w.T, 61)) + [w.T - 1]
        _check_batch(run, list(range(len(w.tables))), rows=rows)
    finally:
        run.close()

