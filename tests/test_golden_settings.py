"""Pins from values the paper prints (tests/golden/paper_settings.json): the
hyper-parameters of the paper-mode workload, the scale rule sigma_k =
sigma sqrt(d / d_k) = sqrt(K) sigma (Eq. 11) evaluated by the workload code
and by the oracle's perturbation (E||sigma_k P_k eps||^2 = d sigma^2, Eq. 10),
and the bf16 byte count the backup sizes in the design use (2P / 2^30)."""
import json
import math
import os

import numpy as np

import synthetic as S

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "paper_settings.json")


def _golden():
    return json.load(open(GOLDEN))


def test_paper_mode_workload_uses_the_printed_settings():
    g = _golden()["es_copes"]
    W = S.workload("p0")
    assert (W.n, W.K, W.n // W.K) == (g["N"], g["K"], g["N_k"])
    assert W.sigma == g["sigma"] and W.alpha == g["alpha"]
    assert W.scale_mode == S.SCALE_ALPHA_OVER_N                      # alpha / N_k (Eq. 13)
    assert W.norm_mode == S.NORM_Z                                  # joint z-score (Eq. 12)


def test_sigma_k_rule_matches_the_printed_value():
    g = _golden()["es_copes"]
    d = 8 * 1000003
    W = S.Workload("t", d, S.BF16, g["K"], S.PART_CONTIGUOUS, S.equal_bounds(d, g["K"]), 0, [1], [1],
                   "uniform", 0, S.NORM_Z, sigma=g["sigma"], alpha=g["alpha"])
    for k in range(g["K"]):
        assert W.sigma_k(k) == np.float32(g["sigma_k"])              # sqrt(K) sigma for equal subspaces
    for K, nk in zip(_golden()["k_ablation"]["K"], (40, 20, 10, 5)):
        assert _golden()["k_ablation"]["N"] // K == nk
        assert math.isclose(g["sigma"] * math.sqrt(K), g["sigma"] * math.sqrt(d / (d // K)), rel_tol=1e-12)


def test_subspace_perturbation_energy_equals_full_space(orc):
    """Eq. 10-11: a subspace perturbation with sigma_k has the energy d sigma^2
    of a full-space one.  Checked on the oracle's noise with the printed
    sigma and K (one subspace of d / K positions, many seeds)."""
    g = _golden()["es_copes"]
    d, K = 1 << 16, g["K"]
    dk = d // K
    sk = np.float32(g["sigma_k"])
    energies = []
    for seed in range(1, 41):
        w = np.zeros(dk, dtype=np.float32)
        orc.perturb(w, 0, dk, sk, seed, 1)
        energies.append(float(np.sum(w.astype(np.float64) ** 2)))
    mean = np.mean(energies)
    target = d * g["sigma"] ** 2
    se = target * math.sqrt(2.0 / dk) / math.sqrt(len(energies))
    assert abs(mean - target) < 5 * se


def test_bf16_bytes_per_parameter():
    m = _golden()["memory"]
    assert round(2 * m["params"] / 2 ** 30, 2) == m["bf16_weights_GB"]
