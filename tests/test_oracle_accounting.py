"""Pins of the oracle's bit accounting against figures the paper prints."""

import json
import math
import os

from oracle import accounting


def _golden(golden_dir):
    with open(os.path.join(golden_dir, "paper_accounting.json")) as f:
        return json.load(f)


def test_trit_information(golden_dir):
    g = _golden(golden_dir)["trit_bits"]
    assert round(accounting.TRIT_BITS, g["digits"]) == g["value"]


def test_two_plane_fraction_from_mask_table(golden_dir):
    gold = _golden(golden_dir)
    orders = gold["mask_orders"]["value"]
    cov = gold["mask_coverage_pct"]["value"]
    assert abs(sum(cov) - 100.1) < 1e-9            # the printed coverages round to 100.1%
    f2_pct = sum(c for c, o in zip(cov, orders) if o == 2)
    assert abs(f2_pct - gold["two_plane_pct"]["value"]) < 1e-9


def test_effective_bits_match_paper(golden_dir):
    gold = _golden(golden_dir)
    f2 = gold["two_plane_pct"]["value"] / 100.0
    e = gold["effective_bits"]
    assert round(accounting.b_eff(f2), e["digits"]) == e["value"]
    assert accounting.b_eff(0.0) == accounting.TRIT_BITS
    assert abs(accounting.b_eff(0.10) - 1.1 * math.log2(3)) < 1e-15


def test_stored_bytes_closed_form():
    # 1024 x 4096, one plane: 26 code bytes + 2 scale bytes per 128 weights.
    assert accounting.packed_bytes(1024, 4096, 0) == 1024 * 32 * 28
    assert accounting.stored_bits_per_weight(1024, 4096, 0) == 1.75
    assert accounting.gemv_bytes(1024, 4096, 0) == 927_744
    # q 4096 x 4096 with 10% two-plane groups (13,107 records of 32 bytes).
    assert accounting.gemv_bytes(4096, 4096, 13_107) == 4_122_212
