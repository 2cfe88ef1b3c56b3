"""The kernel and runtime sources of libsalt, compiled for the CPU under
AddressSanitizer (tests/cpu_build.py), against the fp64 oracle: every global and
LDS access of the shrink / expand / plan kernels is checked by the sanitizer, and
the outputs must meet the same bounds as on the GPU (bf16 1e-2 * (1 + |ref|),
fp32 1e-5 * (1 + |ref|), integer inputs bit-exact).  The cases cover each tile
size (16 / 32 / 64 / 128 tokens, LDS-staged or not), fp32, residual ranks 0 / 1 / 2 / 16,
no centroid, and long-tail concatenated adapters (ranks 17 / 18 and 33 / 34, the
latter on LDS-staged 64-token tiles)."""
import numpy as np
import pytest

import oracle
from paper_2608_03579_amd import synth
from tests import cpu_build
from tests.test_gpu_longtail import _workload as longtail_workload
from tests.test_gpu_tiles import RAGGED, _workload as tile_workload

pytestmark = pytest.mark.skipif(not cpu_build.available(), reason="needs the ROCm host clang")


def _check(w, tmp_path, want_m, exact=False, n_cu=256):
    tables = list(range(len(w.tables)))
    shapes = [(i, o) for _, i, o in w.tables]
    cents = [w.centroids(t) for t in tables] if w.n_centroids else []
    loads = [(int(s), int(w.slot_rank[s]), w.residual_blob(int(s)) if w.slot_rank[s] else None)
             for s in w.referenced_slots()]
    b = cpu_build.Batch(w.tok_c, w.tok_u, w.gamma, tables, [w.x(t) for t in tables], [w.y0(t) for t in tables])
    r = cpu_build.run(w.dtype, shapes, w.n_centroids, w.r_c, w.n_slots, w.r_u_max, max(1, w.T), cents, loads,
                      [b], str(tmp_path), n_cu=n_cu)[0]
    assert r["status"] == (0, 0, 0, 0) and r["n_errors"] == 0, r["status"]
    assert r["tile_tokens"] == want_m
    want = oracle.plan(w.tok_c, w.tok_u)
    for k in want:
        assert np.array_equal(r[k], want[k]), k
    d = w.dtype
    for j, t in enumerate(tables):
        if w.n_centroids:
            cat, cb = (oracle.decode(a, d) for a in w.centroids(t))
        else:
            cat, cb = np.zeros((0, 0, shapes[t][0])), np.zeros((0, 0, shapes[t][1]))
        res = {int(s): tuple(oracle.decode(a, d) for a in w.residual(int(s), t)) for s in w.referenced_slots()}
        ref = oracle.apply(oracle.decode(w.x(t), d), oracle.decode(w.y0(t), d), cat, cb, res, w.tok_c, w.tok_u,
                           w.gamma)
        got = oracle.decode(r["ys"][j], d)
        if exact:
            assert np.array_equal(got, ref), f"table {t}: {np.sum(got != ref)} mismatches"
        tol = (1e-5 if d == "f32" else 1e-2) * (1 + np.abs(ref))
        assert np.all(np.abs(got - ref) <= tol), f"table {t}: worst {float((np.abs(got - ref) / tol).max()):.3f}x"


def test_qproj_decode_bf16(tmp_path):
    _check(synth.make(2, 0, y0="normal"), tmp_path, 16)


def test_m32_staged_integer_bit_exact(tmp_path):
    _check(tile_workload(4, RAGGED, 8, 64, 256, 80, (1, 2), exact=True), tmp_path, 32, exact=True)


def test_m64_no_centroid_rank16(tmp_path):
    _check(tile_workload(3, RAGGED, 0, 0, 300, 40, (1, 16)), tmp_path, 64)


def test_fp32_rank2(tmp_path):
    _check(tile_workload(6, [("a", 264, 136), ("b", 520, 1032)], 4, 8, 96, 30, (2,), dtype="f32"), tmp_path, 16)


def test_long_tail_rank17(tmp_path):
    _check(longtail_workload(0, [("a", 520, 776)], 4, 16, 64, 24, 16, "bf16"), tmp_path, 16)


def test_long_tail_rank33_staged_64_token_tiles(tmp_path):
    """Long-tail ranks past 16 read v inside the column loop while 64-token tiles
    stage B_c in LDS: the two must not share LDS."""
    _check(longtail_workload(3, [("a", 264, 136), ("b", 136, 520)], 2, 32, 512, 8, 8, "bf16"), tmp_path, 64)


def test_expand_blocks_walk_many_tiles(tmp_path):
    """A device of one compute unit: the expand runs a handful of blocks, each
    walking the block-chunks of many tiles and tables in turn (integer inputs,
    bit-exact)."""
    _check(tile_workload(4, RAGGED, 8, 64, 256, 80, (1, 2), exact=True), tmp_path, 32, exact=True, n_cu=1)


def test_m128_tiles_eight_wave_blocks(tmp_path):
    """128-token tiles: blocks of 8 waves share one staged centroid operand."""
    _check(tile_workload(12, RAGGED, 2, 64, 1024, 40, (1,), exact=True), tmp_path, 128, exact=True)
