"""GPU parity of salt_adapter_gram (Sec. 3.1 Eq. 2 / Sec. 4.5: the matrix cosine of
two low-rank updates, computed from r x r Gram products of their factors).

Expected values: the oracle forms the dense updates dW = A B in float64.  Bound
per term: a Gram entry is a sum of K <= 16384 exact products (bf16) taken as 16
MFMA steps of 32 per 512-chunk and at most 32 fp32 atomic adds across chunks, so
its error is below (16 + 32) 2^-24 < 2^-18 of sum_k |x_k y_k|; a term (a sum of
products of two Grams) is then within 2^-17 T_abs, where T_abs is the same term
from absolute values; the test allows 2^-16 T_abs.  Adapters are built so that a
dropped, transposed or mis-paired Gram moves a term by more than that (the
second adapter holds the first one's rows, reversed, plus a few of its own).  Integer factors give exact Grams
(every sum below 2^24) and must match bit for bit.
"""
import numpy as np
import pytest

import oracle
from paper_2608_03579_amd import synth
from tests.gpu_harness import hipmod, to_dev

pytestmark = pytest.mark.gpu


def _announce(name):
    print(f"\n[gpu case] {name}", flush=True)


def _workload(tables, ranks, dtype="bf16", exact=False):
    n = len(ranks)
    z = np.zeros(1, np.int32)
    return synth.Workload(cfg=7, seed=0, name="gram", dtype=dtype, tables=tables, n_centroids=0, r_c=0,
                          n_slots=n, r_u_max=max(ranks), slot_rank=np.asarray(ranks, np.int32), tok_c=z - 1,
                          tok_u=z - 1, gamma=None, exact=exact)


def _split(w, blob, r):
    """Per-table (At, B) of a blob of rank r (array slicing only)."""
    out, off = [], 0
    for _, n_in, n_out in w.tables:
        at = blob[off: off + r * n_in].reshape(r, n_in)
        b = blob[off + r * n_in: off + r * (n_in + n_out)].reshape(r, n_out)
        out.append((at, b))
        off += r * (n_in + n_out)
    return out


def _stack(w, parts):
    """A blob from per-table (At, B) pairs (array concatenation only)."""
    return np.ascontiguousarray(np.concatenate([np.concatenate([at.reshape(-1), b.reshape(-1)]) for at, b in parts]))


def _related(w, r1, r_extra):
    """Adapter 1 = slot 0 (rank r1); adapter 2 = adapter 1's rows in reverse order followed
    by slot 1's (rank r1 + r_extra), so dW2 = dW1 + dW_extra while the cross Grams are
    not symmetric."""
    p1 = _split(w, w.residual_blob(0), r1)
    px = _split(w, w.residual_blob(1), r_extra)
    p2 = [(np.concatenate([a1[::-1], ax]), np.concatenate([b1[::-1], bx])) for (a1, b1), (ax, bx) in zip(p1, px)]
    return _stack(w, p1), r1, _stack(w, p2), r1 + r_extra


def _check(w, blob1, r1, blob2, r2, got):
    d = w.dtype
    p1 = _split(w, blob1, r1)
    p2 = _split(w, blob2, r2)
    for t, ((at1, b1), (at2, b2)) in enumerate(zip(p1, p2)):
        A1, B1, A2, B2 = (oracle.decode(x, d) for x in (at1, b1, at2, b2))
        ref = np.array(oracle.update_terms(A1, B1, A2, B2))
        if w.exact:
            assert np.array_equal(got[t], ref), (t, got[t], ref)
            continue
        t_abs = np.array(oracle.update_terms(np.abs(A1), np.abs(B1), np.abs(A2), np.abs(B2)))
        t_abs[1] = oracle.update_terms(np.abs(A1), np.abs(B1), np.abs(A1), np.abs(B1))[0]
        t_abs[2] = oracle.update_terms(np.abs(A2), np.abs(B2), np.abs(A2), np.abs(B2))[0]
        err = np.abs(got[t] - ref)
        assert np.all(err <= 2.0 ** -16 * t_abs), (t, got[t], ref, err / t_abs)
        # the loss of Eq. 2 from the GPU terms, next to the oracle's
        l_gpu = oracle.align_loss(*got[t])
        l_ref = oracle.align_loss(*ref)
        assert abs(l_gpu - l_ref) <= 1e-3, (t, l_gpu, l_ref)


def _ctx(w):
    from paper_2608_03579_amd import salt
    return salt.Context(w.dtype, [(i, o) for _, i, o in w.tables], 0, 0, 1, 0, 1)


CASES = [
    # tables, r1, r_extra, dtype
    ([("a", 520, 776), ("b", 3072, 1024), ("c", 264, 8200)], 16, 2, "bf16"),
    ([("q", 3072, 3072), ("down", 8192, 3072)], 2, 14, "bf16"),
    ([("a", 1032, 136)], 64, 1, "bf16"),
    ([("a", 776, 520)], 100, 40, "bf16"),
    ([("tiny", 256, 256), ("a", 520, 776)], 8, 8, "f32"),
]


@pytest.mark.parametrize("tables,r1,r_extra,dtype", CASES)
def test_gram_parity(tables, r1, r_extra, dtype):
    _announce(f"adapter gram {dtype} r1={r1} extra={r_extra} tables={tables}")
    w = _workload(tables, [r1, r_extra], dtype)
    b1, r1_, b2, r2 = _related(w, r1, r_extra)
    ctx = _ctx(w)
    d1, d2 = to_dev(b1), to_dev(b2)
    try:
        got = ctx.adapter_gram(d1.ptr, r1_, d2.ptr, r2)
        _check(w, b1, r1_, b2, r2, got)
        # the symmetric call swaps the norms and keeps the cross term
        back = ctx.adapter_gram(d2.ptr, r2, d1.ptr, r1_)
        _check(w, b2, r2, b1, r1_, back)
    finally:
        d1.free(); d2.free()
        ctx.close()


def test_gram_integer_factors_bit_exact():
    _announce("adapter gram, integer factors")
    tables = [("a", 520, 776), ("b", 3072, 1032)]
    w = _workload(tables, [16, 4], "bf16", exact=True)
    b1, r1, b2, r2 = _related(w, 16, 4)
    ctx = _ctx(w)
    d1, d2 = to_dev(b1), to_dev(b2)
    try:
        _check(w, b1, r1, b2, r2, ctx.adapter_gram(d1.ptr, r1, d2.ptr, r2))
    finally:
        d1.free(); d2.free()
        ctx.close()


def test_gram_scratch_grown_and_reused():
    """Calls on one context: ranks 4 / 6, then 48 / 64 (the context's scratch
    grows), then 4 / 6 again (it is reused); each result against the oracle."""
    _announce("adapter gram: one context, scratch grown and reused")
    tables = [("a", 520, 776), ("b", 3072, 1024)]
    runs = [_workload(tables, [4, 2], "bf16"), _workload(tables, [48, 16], "bf16"), _workload(tables, [4, 2], "bf16")]
    ctx = _ctx(runs[0])
    try:
        for w, (r1, extra) in zip(runs, ((4, 2), (48, 16), (4, 2))):
            b1, r1_, b2, r2 = _related(w, r1, extra)
            d1, d2 = to_dev(b1), to_dev(b2)
            try:
                _check(w, b1, r1_, b2, r2, ctx.adapter_gram(d1.ptr, r1_, d2.ptr, r2))
            finally:
                d1.free(); d2.free()
    finally:
        ctx.close()


def test_gram_errors():
    _announce("adapter gram error paths")
    from paper_2608_03579_amd import salt
    w = _workload([("a", 256, 264)], [2, 2])
    ctx = _ctx(w)
    d = to_dev(w.residual_blob(0))
    try:
        assert ctx.adapter_gram_status(d.ptr, 0, d.ptr, 2) == salt.ERR_OUT_OF_RANGE
        assert ctx.adapter_gram_status(d.ptr, 2, d.ptr, 257) == salt.ERR_OUT_OF_RANGE
        assert ctx.adapter_gram_status(0, 2, d.ptr, 2) == salt.ERR_INVALID_ARG
        assert ctx.adapter_gram_status(d.ptr + 4, 2, d.ptr, 2) == salt.ERR_INVALID_ARG
        assert ctx.adapter_gram_status(d.ptr, 2, d.ptr, 2) == salt.OK
    finally:
        d.free()
        ctx.close()
