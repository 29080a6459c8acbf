"""Figures the paper states about its setup (Sec. 4.1), stored with their citations in
tests/golden/paper_sec4_1.json, against the synthetic workloads' shapes: the number of
speculative heads, the size of the added Clover modules, the size of the 7B target."""
import json
import os

import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_sec4_1.json")


def _counts(name):
    cfg = synth.get_config(name)
    total = clover = 0
    for n, shape in synth.weight_specs(cfg):
        k = 1
        for x in shape:
            k *= x
        total += k
        if n.startswith(("ab.", "ad", "head")):  # Augmenting Block, Attention Decoder, head MLPs
            clover += k
    return cfg, total, clover


def test_seven_b_workload_has_the_papers_head_count_and_sizes():
    g = json.load(open(GOLDEN))
    cfg, total, clover = _counts("llama7b_b1")
    assert cfg.n_spec_heads == g["speculative_heads"]["value"]
    paper = g["trainable_parameters"]["baichuan_small_7b"]
    assert paper / 2 <= clover <= paper * 2, clover
    target = total - clover
    assert abs(target - g["target_model_parameters"]["baichuan_small"]) / 7e9 < 0.1, target


def test_large_workload_clover_modules_are_of_the_papers_magnitude():
    g = json.load(open(GOLDEN))
    _, _, clover = _counts("large_gqa_b1")
    paper = g["trainable_parameters"]["baichuan_large_100b"]
    assert paper / 2 <= clover <= paper * 2, clover
