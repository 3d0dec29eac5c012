"""The byte model used for roofline fractions, pinned to the paper's Table 1
(KV memory per request, Sec. 3.2) and to closed forms of the model shapes."""
import json
import os

import pytest

from paper_2512_22420_amd import roofline as R
from paper_2512_22420_amd import workload as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "kv_cache_per_request.json")


def test_kv_bytes_reproduce_table1():
    g = json.load(open(GOLDEN))
    for name, m in g["models"].items():
        per_tok = R.kv_bytes_per_token(m["n_layers"], m["n_kv_heads"], m["head_dim"], m["elt_bytes"])
        for row in g["rows"]:
            assert per_tok * row["context"] / 2 ** 20 == row[name]


def test_qwen_shape_matches_table1_model():
    # the Qwen2.5-7B-shaped workload has the KV geometry of the Table 1 7B model
    s = W.QWEN7B
    assert R.kv_bytes_per_token(s.n_layers, s.n_kv_heads, s.head_dim) * 1024 / 2 ** 20 == 56


def test_layer_parameter_counts():
    assert R.layer_params(W.LLAMA8B_LAYER) == 218_103_808
    assert R.layer_params(W.QWEN7B) == 233_046_016
    assert W.LLAMA8B_LAYER.vocab * W.LLAMA8B_LAYER.d_model == 525_336_576


def test_step_model_small_batch_point():
    m = R.step_model(W.LLAMA8B_LAYER, 1, 0, [1024])
    assert m["M"] == 1
    assert m["weight_bytes"] == 2 * (218_103_808 + 525_336_576)
    assert m["kv_bytes"] == 1024 * 4096
    # HBM-bound at M=1: ~186.6 us at 8 TB/s
    assert m["t_roof_s"] == pytest.approx(186.6e-6, rel=2e-3)
