"""The parity gate |y - ref| <= 1e-2 (1 + |ref|) must reject plausible wrong
outputs at the workloads' own scales (CPU only, oracle-generated mutants).

Each mutant is what a kernel with one planted mistake would produce, rounded
to bf16 like a real output; the correct output rounded the same way must pass.
"""
import numpy as np
import pytest

import oracle
from paper_2608_03579_amd import synth
from tests.gpu_harness import TOL_BF16, close_enough


def to_bf16_values(a):
    return oracle.decode(synth.f32_to_bf16_bits(a.astype(np.float32)), "bf16")


def outputs(w, table, tok_c, tok_u, gamma, drop_residual=False, rows=None):
    d = w.dtype
    x = oracle.decode(w.x(table), d)
    y0 = oracle.decode(w.y0(table), d)
    cat, cb = (oracle.decode(a, d) for a in w.centroids(table))
    res = {}
    for s in set(int(u) for u in tok_u if u >= 0):
        at, b = (oracle.decode(a, d) for a in w.residual(s, table))
        res[s] = (at * 0, b * 0) if drop_residual else (at, b)
    return oracle.apply(x, y0, cat, cb, res, tok_c, tok_u, gamma, rows=rows)


CASES = [(2, {}), (4, dict(T=64)), (5, dict(T=96)), (2, dict(gamma="bins"))]


@pytest.mark.parametrize("cfg,kw", CASES)
def test_gate_rejects_planted_mistakes(cfg, kw):
    w = synth.make(cfg, 0, **kw)
    t = 0
    rows = list(range(min(w.T, 48)))
    ref = outputs(w, t, w.tok_c, w.tok_u, w.gamma, rows=rows)
    assert close_enough(to_bf16_values(ref), ref, TOL_BF16)[0]
    C, S = w.n_centroids, w.n_slots
    mutants = {
        "y unchanged": oracle.decode(w.y0(t), w.dtype)[rows],
        "residual dropped": outputs(w, t, w.tok_c, w.tok_u, w.gamma, drop_residual=True, rows=rows),
        "centroid off by one": outputs(w, t, (w.tok_c + 1) % C, w.tok_u, w.gamma, rows=rows),
        "centroid dropped": outputs(w, t, np.full_like(w.tok_c, -1), w.tok_u, w.gamma, rows=rows),
    }
    # a slot off by one only matters where the neighbouring slot is loaded
    tu = w.tok_u.copy()
    ref_slots = set(w.referenced_slots().tolist())
    nxt = np.array([(u + 1) % S for u in tu])
    ok = np.array([n in ref_slots and w.slot_rank[n] == w.slot_rank[u] for u, n in zip(tu, nxt)])
    if ok.any():
        tu[ok] = nxt[ok]
        mutants["slot off by one"] = outputs(w, t, w.tok_c, tu, w.gamma, rows=rows)
    if w.gamma is not None:
        mutants["gamma ignored"] = outputs(w, t, w.tok_c, w.tok_u, None, rows=rows)
    for name, m in mutants.items():
        passed, worst, nbad = close_enough(to_bf16_values(m), ref, TOL_BF16)
        assert not passed, f"cfg {cfg}: the gate accepts '{name}' (worst {worst:.2f}x)"


# ---------------------------------------------------------------------------
# the fused-weight bound (salt_fuse_centroid parity) against planted mistakes
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("kind", ["dropped", "negated", "gamma_ignored", "other_centroid", "b_rank_reversed"])
def test_fuse_bound_rejects_planted_mistakes(kind):
    from tests.gpu_harness import fuse_within_bound
    tables = [("a", 264, 200)]
    one = np.zeros(1, np.int32)
    w = synth.Workload(cfg=6, seed=0, name="fuse", dtype="bf16", tables=tables, n_centroids=2, r_c=32,
                       n_slots=1, r_u_max=0, slot_rank=one, tok_c=one - 1, tok_u=one - 1, gamma=None)
    at, b = (oracle.decode(a, "bf16") for a in w.centroids(0))
    W0 = oracle.decode(w.base_weight(0), "bf16")
    gamma = 0.6
    ref = oracle.fuse_centroid(W0, at[0], b[0], gamma)
    good = to_bf16_values(ref)
    assert fuse_within_bound(good, ref, W0, at[0], b[0], gamma, "bf16")[0]
    bad = {"dropped": W0,
           "negated": oracle.fuse_centroid(W0, at[0], b[0], -gamma),
           "gamma_ignored": oracle.fuse_centroid(W0, at[0], b[0], 1.0),
           "other_centroid": oracle.fuse_centroid(W0, at[1], b[1], gamma),
           "b_rank_reversed": oracle.fuse_centroid(W0, at[0], b[0][::-1], gamma)}[kind]
    assert not fuse_within_bound(to_bf16_values(bad), ref, W0, at[0], b[0], gamma, "bf16")[0], kind


# ---------------------------------------------------------------------------
# the adapter-Gram bound (salt_adapter_gram parity) against planted mistakes
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("kind", ["b_gram_transposed", "second_adapter_truncated", "norm_not_squared",
                                  "cross_with_own_b", "sign"])
def test_gram_bound_rejects_planted_mistakes(kind):
    rng = np.random.default_rng(5)
    r, rx, n_in, n_out = 8, 2, 520, 776
    to = lambda a: oracle.decode(synth.f32_to_bf16_bits((a * 0.02).astype(np.float32)), "bf16")
    A1, B1 = to(rng.standard_normal((r, n_in))), to(rng.standard_normal((r, n_out)))
    Ax, Bx = to(rng.standard_normal((rx, n_in))), to(rng.standard_normal((rx, n_out)))
    A2, B2 = np.concatenate([A1[::-1], Ax]), np.concatenate([B1[::-1], Bx])   # dW2 = dW1 + dWx
    ref = np.array(oracle.update_terms(A1, B1, A2, B2))
    t_abs = np.array([oracle.update_terms(np.abs(A1), np.abs(B1), np.abs(A2), np.abs(B2))[0],
                      oracle.update_terms(np.abs(A1), np.abs(B1), np.abs(A1), np.abs(B1))[0],
                      oracle.update_terms(np.abs(A2), np.abs(B2), np.abs(A2), np.abs(B2))[0]])
    ga = A1 @ A2.T                                    # Gram of the At rows (r x (r + rx))
    gb = B1 @ B2.T
    bad = ref.copy()
    if kind == "b_gram_transposed":
        bad[0] = np.sum(ga[:, :r] * gb[:, :r].T) + np.sum(ga[:, r:] * gb[:, r:])   # r x r block transposed
    elif kind == "second_adapter_truncated":
        bad[0] = oracle.update_terms(A1, B1, A2[:r], B2[:r])[0]                    # extra rows of adapter 2 lost
    elif kind == "norm_not_squared":
        bad[1] = np.sqrt(ref[1])
    elif kind == "cross_with_own_b":
        bad[0] = np.sum(ga[:, :r] * (B1 @ B1.T)[:, ::-1])                          # B side of the cross term from adapter 1
    else:
        bad[0] = -ref[0]
    assert not np.all(np.abs(bad - ref) <= 2.0 ** -16 * t_abs), kind
