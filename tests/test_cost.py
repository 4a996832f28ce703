"""The MAC counter reproduces the paper's Table 1 (tests/golden/table1_la_macs.txt)."""

import os

import pytest

from paper_2609_32114_amd import cost

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "table1_la_macs.txt")


def _rows():
    for line in open(GOLDEN):
        line = line.strip()
        if line and not line.startswith("#"):
            t, g = line.split()
            yield int(t), float(g)


@pytest.mark.parametrize("tokens,gmac", list(_rows()))
def test_mac_count_matches_table1(tokens, gmac):
    macs = cost.macs_per_token_head(64, 128, 128) * tokens * 16
    assert round(macs / 1e9, 2) == gmac


def test_bytes_workload_gdn_T4096_H16():
    # 16 heads x 128 x 2 B x (q, k, v, o) + 16 x (4 + 4) B per token, plus a 1 MiB final state
    b = cost.algorithmic_bytes(4096, 1, 16, 16, 128, 128, 2, kda=False, with_s0=False)
    assert b == 4096 * 16512 + 16 * 128 * 128 * 4
