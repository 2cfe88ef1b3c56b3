"""salt_route (Sec. 3.2 centroid routing) is host-only: the library's decision and
statistics against the oracle's on random inputs and on the paper's routing
table, and its argument checks.  CPU only."""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2608_03579_amd import salt

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("seed", range(20))
def test_route_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    K = int(rng.integers(2, 9))
    n = rng.uniform(0.1, 5.0, K)
    mu_n = n + rng.normal(0.0, 1.0, K) * rng.uniform(0.1, 2.0)
    sigma_n = rng.uniform(0.2, 1.5, K)
    mu_r = rng.uniform(0.3, 2.5, K)
    sigma_r = rng.uniform(0.1, 1.0, K)
    tau_n, tau_r = float(rng.choice([0.5, 2.0, 4.0])), float(rng.choice([0.5, 2.0, 4.0]))
    st, got = salt.route(n, mu_n, sigma_n, mu_r, sigma_r, tau_n, tau_r)
    assert st == salt.OK
    want = oracle.route(n.tolist(), mu_n.tolist(), sigma_n.tolist(), mu_r.tolist(), sigma_r.tolist(), tau_n, tau_r)
    np.testing.assert_allclose(got["z_n"], want["z_n"], rtol=1e-12)
    assert got["k_star"] == want["k_star"] and got["ood"] == want["ood"] and got["blended"] == want["blended"]
    if not want["ood"]:
        np.testing.assert_allclose(got["z_r"], want["z_r"], rtol=1e-12)


def test_route_library_decision_on_paper_table():
    """Inputs built so that the library's statistics equal the printed deviations
    (N = 1 for both centroids, so R_k = 1; mu_N and mu_R offset by the printed Z
    values, sigma = 1): the library must reach the printed routing."""
    g = json.load(open(os.path.join(GOLDEN, "paper_routing_table.json")))
    for row in g["rows"]:
        n = np.array([1.0, 1.0])                         # R_k = 1 for both centroids
        mu_n = n + np.array([row["z_n_min"], row["z_n_min"] + 0.5])
        st, got = salt.route(n, mu_n, [1.0, 1.0], 1.0 + np.array(row["z_r"]), [1.0, 1.0], g["tau_n"], g["tau_r"])
        assert st == salt.OK
        routed = "OOD" if got["ood"] else ("blended" if got["blended"] else g["centroids"][got["k_star"]])
        assert routed == row["routed"], row
        assert abs(got["z_n_min"] - row["z_n_min"]) < 1e-12


def test_route_rejects_bad_arguments():
    ok = dict(n=[1.0, 2.0], mu_n=[1.0, 2.0], sigma_n=[1.0, 1.0], mu_r=[1.0, 1.0], sigma_r=[1.0, 1.0])
    assert salt.route(**ok)[0] == salt.OK
    assert salt.route([1.0], [1.0], [1.0], [1.0], [1.0])[0] == salt.ERR_INVALID_ARG           # K < 2
    assert salt.route([1.0, 2.0], [1.0, 2.0], [0.0, 1.0], [1.0, 1.0], [1.0, 1.0])[0] == salt.ERR_INVALID_ARG
    assert salt.route([1.0, 2.0], [1.0, 2.0], [1.0, 1.0], [1.0, 1.0], [-1.0, 1.0])[0] == salt.ERR_INVALID_ARG
    assert salt.route([-1.0, 2.0], [1.0, 2.0], [1.0, 1.0], [1.0, 1.0], [1.0, 1.0])[0] == salt.ERR_INVALID_ARG
    assert salt.route([float("nan"), 2.0], [1.0, 2.0], [1.0, 1.0], [1.0, 1.0], [1.0, 1.0])[0] == salt.ERR_INVALID_ARG
    assert salt.route([1.0, 0.0], [1.0, 2.0], [1.0, 1.0], [1.0, 1.0], [1.0, 1.0])[0] == salt.ERR_INVALID_ARG  # others 0
    assert salt.route(**ok, tau_n=float("inf"))[0] == salt.ERR_INVALID_ARG
