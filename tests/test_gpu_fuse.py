"""GPU parity of salt_fuse_centroid (Sec. 3.3: a high-frequency domain's scaled
centroid folded into the base weight at node start-up).

The GPU result is rne(W + gamma * A_c B_c) with an fp32 contraction; the oracle
gives the exact float64 value.  Bound per element: one bf16 rounding of the
result (2^-8 |ref| covers it with the fp32 sum's own error on top) plus the fp32
accumulation error, 2^-16 (|W| + |gamma| sum_r |A_ir B_ro|) (r_c fp32 terms).  A dropped, negated
or transposed centroid term moves W by about 10 % of its size here (W ~ N(0, 0.02^2),
r_c >= 8), far outside that bound.  Integer inputs must come back bit-exact.
Columns past out_dim (ldw > out) must come back unchanged.
"""
import numpy as np
import pytest

import oracle
from paper_2608_03579_amd import synth
from tests.gpu_harness import fuse_within_bound, hipmod, to_dev

pytestmark = pytest.mark.gpu


def _announce(name):
    print(f"\n[gpu case] {name}", flush=True)


def _workload(tables, C, r_c, dtype="bf16", exact=False, seed=0):
    one = np.zeros(1, np.int32)
    return synth.Workload(cfg=6, seed=seed, name="fuse", dtype=dtype, tables=tables, n_centroids=C, r_c=r_c,
                          n_slots=1, r_u_max=0, slot_rank=np.zeros(1, np.int32), tok_c=one - 1, tok_u=one - 1,
                          gamma=None, exact=exact)


def _ctx(w):
    from paper_2608_03579_amd import salt
    ctx = salt.Context(w.dtype, [(i, o) for _, i, o in w.tables], w.n_centroids, w.r_c, 1, 0, 1)
    for t in range(len(w.tables)):
        at, b = w.centroids(t)
        ctx.pin_centroids(t, at, b)
    return ctx


def _fuse_on_gpu(ctx, w, t, c, gamma, ldw, w_host=None):
    hip = hipmod()
    wh = w.base_weight(t, ldw) if w_host is None else w_host
    wd = to_dev(wh)
    s = hip.Stream()
    ctx.fuse_centroid(t, c, gamma, wd.ptr, ldw, s.h)
    s.synchronize()
    got = wd.to_host()
    wd.free()
    return wh, got


def _check(w, t, c, gamma, ldw, wh, got):
    _, n_in, n_out = w.tables[t]
    at, b = w.centroids(t)
    A = oracle.decode(at[c], w.dtype)
    B = oracle.decode(b[c], w.dtype)
    W0 = oracle.decode(wh, w.dtype)
    ref = oracle.fuse_centroid(W0[:, :n_out], A, B, gamma)
    g = oracle.decode(got, w.dtype)
    if w.exact:
        assert np.array_equal(g[:, :n_out], ref), f"{np.sum(g[:, :n_out] != ref)} exact mismatches"
    else:
        ok, worst, nbad = fuse_within_bound(g[:, :n_out], ref, W0[:, :n_out], A, B, gamma, w.dtype)
        assert ok, f"{nbad} elements out of bound, worst {worst:.3f}x"
    assert np.array_equal(got[:, n_out:], wh[:, n_out:]), "columns past out_dim changed"


CASES = [
    # tables, C, r_c, dtype
    ([("a", 520, 776), ("b", 1024, 384)], 2, 32, "bf16"),
    ([("q", 3072, 3072)], 2, 64, "bf16"),
    ([("a", 776, 1032), ("b", 64, 136)], 3, 8, "bf16"),
    ([("a", 1024, 520)], 1, 128, "bf16"),
    ([("a", 264, 200)], 2, 96, "bf16"),
    ([("tiny", 256, 256), ("a", 520, 776)], 2, 8, "f32"),
    ([("a", 520, 392)], 2, 40, "f32"),
]


@pytest.mark.parametrize("tables,C,r_c,dtype", CASES)
@pytest.mark.parametrize("gamma", [1.0, 0.6, -0.8])
def test_fuse_parity(tables, C, r_c, dtype, gamma):
    _announce(f"fuse {dtype} r_c={r_c} tables={tables} gamma={gamma}")
    w = _workload(tables, C, r_c, dtype)
    ctx = _ctx(w)
    try:
        for t, (_, _, n_out) in enumerate(tables):
            for c in range(C):
                ldw = n_out if (t + c) % 2 == 0 else n_out + 24
                wh, got = _fuse_on_gpu(ctx, w, t, c, gamma, ldw)
                _check(w, t, c, gamma, ldw, wh, got)
    finally:
        ctx.close()


def test_fuse_integer_inputs_bit_exact():
    _announce("fuse integer inputs")
    tables = [("a", 520, 1032), ("b", 3072, 776)]
    w = _workload(tables, 2, 64, "bf16", exact=True)
    ctx = _ctx(w)
    try:
        for t in range(2):
            for c in range(2):
                wh, got = _fuse_on_gpu(ctx, w, t, c, 1.0, tables[t][2])
                _check(w, t, c, 1.0, tables[t][2], wh, got)
    finally:
        ctx.close()


def test_fuse_then_unfuse_returns_near_the_base():
    """gamma then -gamma: two roundings away from W at most."""
    _announce("fuse and unfuse")
    tables = [("a", 520, 776)]
    w = _workload(tables, 2, 32, "bf16")
    ctx = _ctx(w)
    try:
        wh, once = _fuse_on_gpu(ctx, w, 0, 1, 0.8, 776)
        _, back = _fuse_on_gpu(ctx, w, 0, 1, -0.8, 776, w_host=once)
        W0 = oracle.decode(wh, "bf16")
        err = np.abs(oracle.decode(back, "bf16") - W0)
        assert np.all(err <= 2.0 ** -7 * (np.abs(W0) + 0.01)), float(err.max())
    finally:
        ctx.close()


def test_fuse_errors_change_nothing():
    _announce("fuse error paths")
    from paper_2608_03579_amd import salt
    tables = [("a", 520, 776), ("b", 256, 264)]
    w = _workload(tables, 2, 32, "bf16")
    ctx = salt.Context("bf16", [(i, o) for _, i, o in tables], 2, 32, 1, 0, 1)
    hip = hipmod()
    wh = w.base_weight(0)
    wd = to_dev(wh)
    try:
        at, b = w.centroids(0)
        ctx.pin_centroids(0, at[:1], b[:1], c0=0)            # centroid 1 of table 0 never pinned
        assert ctx.fuse_centroid_status(0, 1, 1.0, wd.ptr, 776) == salt.ERR_BAD_STATE
        assert ctx.fuse_centroid_status(0, 2, 1.0, wd.ptr, 776) == salt.ERR_OUT_OF_RANGE
        assert ctx.fuse_centroid_status(0, -1, 1.0, wd.ptr, 776) == salt.ERR_OUT_OF_RANGE
        assert ctx.fuse_centroid_status(2, 0, 1.0, wd.ptr, 776) == salt.ERR_OUT_OF_RANGE
        assert ctx.fuse_centroid_status(0, 0, 1.0, 0, 776) == salt.ERR_INVALID_ARG
        assert ctx.fuse_centroid_status(0, 0, 1.0, wd.ptr + 2, 776) == salt.ERR_INVALID_ARG
        assert ctx.fuse_centroid_status(0, 0, 1.0, wd.ptr, 770) == salt.ERR_INVALID_ARG    # ldw < out
        assert ctx.fuse_centroid_status(0, 0, 1.0, wd.ptr, 780) == salt.ERR_INVALID_ARG    # ldw % 8
        assert ctx.fuse_centroid_status(0, 0, float("nan"), wd.ptr, 776) == salt.ERR_INVALID_ARG
        hip.synchronize()
        assert np.array_equal(wd.to_host(), wh), "a refused call wrote W"
        assert ctx.fuse_centroid_status(0, 0, 1.0, wd.ptr, 776) == salt.OK
    finally:
        wd.free()
        ctx.close()
