"""Pins for the Appendix E cost model against the numbers the paper prints (Tables 9 and 10)."""
import json
import os

import pytest

from oracle import cost
from paper_2609_36590_amd import synth

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "app_e_cost.json")))


def _r(x, nd):
    return round(x, nd)


def test_qwen3_1p7b_parameter_counts():
    g = GOLD["qwen3_1p7b"]
    c = synth.C2_28L
    assert _r(cost.attention_params(c) / 1e6, 2) == g["attention_params_M"]
    assert _r(cost.mlp_params(c) / 1e6, 2) == g["mlp_params_M"]
    assert _r(cost.layer_params(c) / 1e6, 2) == g["layer_params_M"]
    assert _r(c.n_layers * cost.layer_params(c) / 1e9, 3) == g["all_layers_params_B"]
    assert _r(cost.embedding_params(c) / 1e6, 1) == g["embedding_params_M"]
    # The paper prints 1.721B although its own parts (1.409B + 311.2M) sum to 1.7204B; the
    # exact count 1,720,451,072 is within 0.05% of the printed figure.
    assert abs(cost.full_params(c) / 1e9 - g["full_params_B"]) / g["full_params_B"] < 5e-4


def test_table9_drafting_cost():
    g = GOLD["table9"]
    c = synth.C2_28L
    # The paper adds its rounded components (50.33M per layer, 311.2M head, 1721M total).
    layer_M = _r(cost.layer_params(c) / 1e6, 2)
    head_M = _r(cost.embedding_params(c) / 1e6, 1)
    total_M = 1721.0
    assert _r(2 * layer_M + head_M, 1) == g["seed_draft_weights_M"]
    assert _r((2 * layer_M + head_M) / total_M, 3) == g["seed_draft_cost"]
    # LayerSkip's early-exit draft is "8 layers + head"; its verify recomputes 20 layers + head
    assert _r(8 * layer_M + head_M, 1) == g["layerskip_draft_weights_M"]
    assert _r((8 * layer_M + head_M) / total_M, 3) == g["layerskip_draft_cost"]
    assert _r((20 * layer_M + head_M) / total_M, 3) == g["layerskip_verify_cost"]
    # exact counts agree with the printed ones to 0.05%
    assert abs(cost.draft_weights(c) / 1e6 - g["seed_draft_weights_M"]) < 5e-4 * g["seed_draft_weights_M"]
    assert _r(cost.draft_cost(c), 3) == g["seed_draft_cost"]
    assert _r(cost.draft_cost(c, n_dec=8), 3) == g["layerskip_draft_cost"]
    assert _r(cost.draft_cost(c, n_dec=20), 3) == g["layerskip_verify_cost"]


def test_qwen3_4b_drafting_cost():
    g = GOLD["qwen3_4b"]
    c = synth.C3_4B
    assert round(cost.layer_params(c) / 1e6) == g["layer_params_M"]
    assert round(cost.embedding_params(c) / 1e6) == g["embedding_params_M"]
    assert _r(cost.draft_cost(c), 3) == g["draft_cost"]


@pytest.mark.parametrize("row", GOLD["table10"]["rows"], ids=lambda r: r["method"])
def test_table10_throughput_prediction(row):
    t = GOLD["table10"]
    # the paper rounds each printed intermediate (T_unit to 2 decimals, T to 0.1 ms, n to 2)
    T_unit = _r(cost.round_cost(t["d"], row["c_draft"], row["c_verify"]), 2)
    assert T_unit == row["T_unit"]
    # one unit = one AR forward pass = 1/37.9 s (printed as 26.4 ms)
    unit_ms = 1000.0 / t["ar_tokens_per_s"]
    assert _r(unit_ms, 1) == t["unit_ms"]
    T_ms = _r(T_unit * unit_ms, 1)
    assert T_ms == row["T_ms"]
    n = _r(cost.tokens_per_round(t["d"], row["rate"]), 2)
    assert n == row["n"]
    assert _r(cost.predicted_throughput(T_ms, n), 1) == row["predicted"]
