"""Pin of the oracle's mapper-size bookkeeping against the sizes the paper
prints (Appendix D, Table tab:mapper_sizes)."""

import json
import os

from oracle import kvx_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "mapper_sizes.json")


def test_cross_head_sizes_match_printed_table():
    rows = json.load(open(GOLDEN))["rows"]
    for r in rows:
        n = O.mapper_params(L_t=r["L_t"], H_t=8, k=r["k"], H_s=8, d_s=128, d_t=128)
        assert abs(n / 1e9 - r["params_B"]) <= 0.0051, r
        gib = n * 4 / 2**30
        assert abs(gib - r["storage_GB"]) <= 0.5 + 1e-9, (r, gib)


def test_per_head_form_is_the_block_diagonal_restriction():
    """Per-head W [k*d, d] has 1/H_s of the cross-head W's input features."""
    cross = O.mapper_params(64, 8, 4, 8, 128, 128)
    per_head = O.mapper_params(64, 8, 4, 1, 128, 128)
    assert cross == 8 * per_head
    assert per_head == 2 * 64 * 8 * 512 * 128      # 67.1 M for the 14B->32B shape at k=4
