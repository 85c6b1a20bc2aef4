"""Pins for the oracle's rotary position ids (hand-derived fixture + invariants)."""
import os

import numpy as np
import pytest

from oracle import positions as P

GOLD = os.path.join(os.path.dirname(__file__), "golden", "positions_small.txt")


def _load_cases():
    cases, cur = [], None
    for line in open(GOLD):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        f = line.split()
        if f[0] == "case":
            total, nb = int(f[2]), int(f[3])
            vals = list(map(int, f[4:]))
            blocks = [tuple(vals[4 * i:4 * i + 4]) for i in range(nb)]
            cur = {"name": f[1], "total": total, "blocks": blocks, "rows": []}
            cases.append(cur)
        else:
            cur["rows"].append(tuple(map(int, f)))
    return cases


@pytest.mark.parametrize("case", _load_cases(), ids=lambda c: c["name"])
def test_golden_positions(case):
    pos = P.target_positions(case["total"], case["blocks"])
    assert len(case["rows"]) == case["total"]
    for i, pt, ph, pw in case["rows"]:
        assert tuple(pos[:, i]) == (pt, ph, pw), i


def test_text_only_is_flat():
    assert np.array_equal(P.target_positions(50, []), P.flat_positions(50))


def test_adjacent_patches_differ_in_one_axis():
    # Sec. 4.2: patches adjacent along w differ only in p_W; along h only in p_H.
    pos = P.target_positions(3 * 4 * 5 + 7, [(7, 3, 4, 5)])
    s = 7
    for t in range(3):
        for h in range(4):
            for w in range(4):
                i = s + (t * 4 + h) * 5 + w
                d = pos[:, i + 1] - pos[:, i]
                assert tuple(d) == (0, 0, 1)
            if h < 3:
                i = s + (t * 4 + h) * 5
                d = pos[:, i + 5] - pos[:, i]
                assert tuple(d) == (0, 1, 0)


def test_blocks_validated():
    with pytest.raises(ValueError):
        P.target_positions(10, [(8, 1, 2, 2)])
    with pytest.raises(ValueError):
        P.target_positions(20, [(0, 1, 2, 2), (3, 1, 1, 2)])
