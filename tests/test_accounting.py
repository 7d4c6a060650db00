import json
import os

from paper_2511_06077_amd import accounting

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_mac_counts.json")


def test_transformer_mac_counts_reproduce_the_paper():
    g = json.load(open(GOLDEN))
    for L, gmacs in g["transformer_gmacs"].items():
        got = accounting.transformer_macs_per_sample(float(L), g["d_model"], g["n_layers"]) / 1e9
        assert abs(got - gmacs) < 0.005, (L, got, gmacs)


def test_stage_costs_headline_shape():
    c = accounting.stage_costs([10240] * 128, [32] * 128, 256, 4)
    assert abs(c["proj"]["flop"] - 1.374e12) / 1.374e12 < 1e-3
    assert abs(c["attn"]["flop"] - 1.718e11) / 1.718e11 < 1e-3
    assert abs(c["attn"]["bytes"] - 5.369e9) / 5.369e9 < 1e-3
