"""The paper's parameter values (Example 4.1, Table "lpn-tradeoff") against
the parameter sets and the oracle's client-cost formula (CPU only)."""
import json
import os

import pytest

from oracle.protocol import client_cost_per_row
from synthetic_inputs import (PARAMS_PAPER_D1, PARAMS_PAPER_D2_SPARSE, PARAMS_PAPER_D2_T80,
                              PARAMS_PAPER_D3_SPARSE, PARAMS_PAPER_D3_T80, ProtocolParams)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")


@pytest.fixture(scope="module")
def golden():
    with open(GOLDEN) as f:
        return json.load(f)


def test_lwe_level(golden):
    r1 = golden["lwe_rank_lambda140"]["value"]
    sigma = golden["lwe_sigma_lambda140"]["value"]
    for p in (PARAMS_PAPER_D1, PARAMS_PAPER_D2_T80, PARAMS_PAPER_D3_T80):
        assert p.ranks[0] == r1
        assert p.noise.kind == "dgauss" and p.noise.sigma == sigma
    assert PARAMS_PAPER_D2_SPARSE.ranks[0] == r1 and PARAMS_PAPER_D3_SPARSE.ranks[0] == r1


def test_lpn_levels(golden):
    levels = golden["lpn_levels"]["value"]           # [[r_2, t_2], [r_3, t_3]]
    p = PARAMS_PAPER_D3_T80
    assert [list(x) for x in zip(p.ranks[1:], p.lpn_weights)] == levels
    assert list(PARAMS_PAPER_D3_SPARSE.ranks[1:]) == [r for r, _ in levels]
    q = PARAMS_PAPER_D2_T80
    assert [list(x) for x in zip(q.ranks[1:], q.lpn_weights)] == levels[:1]


def test_client_cost_table(golden):
    """r_d + sum t_i per (m + n) l: 1536 (LWE only), 1104 (+ LPN-1), 812 (+ LPN-2)."""
    cost = golden["client_compute_per_row"]["value"]
    assert client_cost_per_row(PARAMS_PAPER_D1) == cost["lwe_only"]
    assert client_cost_per_row(PARAMS_PAPER_D2_T80) == cost["lpn1"]
    assert client_cost_per_row(PARAMS_PAPER_D3_T80) == cost["lpn2"]
    with pytest.raises(ValueError):
        client_cost_per_row(ProtocolParams(ranks=(16, 8)))
