"""Tile counts of the tiling operator against numbers the paper prints."""
import json
import os

import oracle

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def _tiles(shapes, T, blocks):
    return blocks * sum(oracle.tile_count(H, W, T) for H, W in shapes)


def test_qwen3_tile_totals_match_paper():
    ch = GOLD["cross_layer_chunking"]
    shapes = GOLD["qwen3_block_shapes"]
    blocks = GOLD["qwen3_1p7b_blocks"]["blocks"]
    assert _tiles(shapes["1.7B"], ch["T"], blocks) == ch["1.7B_total_tiles"]
    # The paper gives no block count for 0.6B; 1680 tiles at 60 per block is 28 blocks.
    per_block = sum(oracle.tile_count(H, W, ch["T"]) for H, W in shapes["0.6B"])
    assert per_block * 28 == ch["0.6B_total_tiles"]
