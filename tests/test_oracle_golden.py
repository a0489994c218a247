"""The oracle against its stored expected values (CPU only).

``tests/golden/tiny_stage_oracle.txt`` holds float64 oracle results for a
two-layer tiny stage (prefill of two prompts, then a decode step), written by
``tests/golden/make_golden.py`` from the oracle alone. Recomputing them here
catches any later change to the oracle's arithmetic; a deliberate change
(with its justification) regenerates the file.
"""

from __future__ import annotations

import os

import numpy as np

from tests.golden import make_golden as G

PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "tiny_stage_oracle.txt")


def _read():
    blocks, name = {}, None
    for line in open(PATH):
        if line.startswith("#"):
            continue
        if line.startswith("["):
            name = line[1:line.index("]")]
            blocks[name] = []
            continue
        blocks[name].append([float(v) for v in line.split()])
    return {k: np.array(v) for k, v in blocks.items()}


def test_stored_values_are_the_oracle_of_today():
    g = _read()
    y_pf, y_dc = G.tiny_case()
    np.testing.assert_allclose(y_pf[list(G.FULL_PREFILL_ROWS)], g["prefill_rows_0_20_21_29"],
                               rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(np.stack([y_pf.sum(1), (y_pf * y_pf).sum(1)], 1),
                               g["prefill_row_sum_and_sumsq"], rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(y_dc, g["decode"], rtol=1e-12, atol=1e-13)


def test_stored_file_shape_and_header():
    text = open(PATH).read()
    assert "oracle/stage_oracle.py" in text and "make_golden.py" in text
    g = _read()
    assert g["prefill_rows_0_20_21_29"].shape == (4, 256)
    assert g["prefill_row_sum_and_sumsq"].shape == (30, 2)
    assert g["decode"].shape == (2, 256)
