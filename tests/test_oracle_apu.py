"""Pins of the efficiency helpers against the worked numbers the paper prints."""

import json
import math
import os

import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "apu_printed.json")
with open(GOLDEN) as _f:
    G = json.load(_f)


def _printed_as(v, digits):
    """The values the paper could print for v: it rounds some figures and truncates others
    (0.8576 is printed 0.86 in Sec. 2.3, 0.7852 is printed 0.78 in Sec. 5)."""
    scale = 10 ** digits
    return {round(math.floor(v * scale + 0.5) / scale, digits), round(math.floor(v * scale) / scale, digits)}


@pytest.mark.parametrize("e", G["sd_aal"], ids=lambda e: e["cite"])
def test_sd_aal(e):
    assert e["printed"] in _printed_as(oracle.sd_aal(e["alpha"], e["gamma"]), e["digits"])


@pytest.mark.parametrize("e", G["sd_apu"], ids=lambda e: e["cite"])
def test_sd_apu(e):
    aal = oracle.sd_aal(e["alpha"], e["gamma"])
    v = oracle.apu(e["gamma"], e["density"], 1.0, aal)
    assert e["printed"] in _printed_as(v, e["digits"])


def test_sd_best_gamma():
    e = G["sd_best_gamma"]
    vals = {g: oracle.apu(g, e["density"], 1.0, oracle.sd_aal(e["alpha"], g)) for g in range(1, e["search_max"] + 1)}
    assert min(vals, key=vals.get) == e["best_gamma"]


@pytest.mark.parametrize("e", G["apu"], ids=lambda e: e["cite"])
def test_apu(e):
    v = oracle.apu(e["n_sparse"], e["density"], 1.0, e["n_aal"])
    assert e["printed"] in _printed_as(v, e["digits"])


@pytest.mark.parametrize("e", G["effective_density"], ids=lambda e: e["cite"])
def test_effective_density(e):
    v = oracle.effective_density(e["period"], e["density"], e["n_aal"])
    assert e["printed"] in _printed_as(v, e["digits"])
    # The period form equals the n_sparse form with n_sparse = period - 1.
    assert abs(v - oracle.apu(e["period"] - 1, e["density"], 1.0, e["n_aal"])) < 1e-15


def test_sd_aal_limits():
    assert oracle.sd_aal(0.0, 5) == 1.0
    assert oracle.sd_aal(1.0, 5) == 6.0
