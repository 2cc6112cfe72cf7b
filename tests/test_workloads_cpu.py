"""The synthetic workload tables against the paper's values kept in tests/golden."""
import json
import os

import workloads

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "paper_constants.json")


def test_qwen3_block0_shapes_match_the_papers_table():
    gold = json.load(open(GOLDEN))["qwen3_block_shapes"]
    for model, shapes in workloads.QWEN3_BLOCK0.items():
        assert [[h, w] for _, h, w in shapes] == gold[model], model
        assert [n for n, _, _ in shapes] == ["q_proj", "k_proj", "v_proj", "o_proj", "gate_proj", "up_proj",
                                             "down_proj"]
