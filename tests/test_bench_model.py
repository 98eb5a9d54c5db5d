"""Host-side checks of the benchmark's byte model (no GPU)."""
import random

import pytest
import torch

import bench


def _kernel_span_loads(nks, span, seg_len=128):
    """Rows the training kernel loads into its word-row span, counted by walking its steps one by one:
    per work unit the first centre's 2*span slots that lie in the document, then per later centre the
    previous centre's row and, when it exists, the row span positions past the new centre."""
    total = 0
    for nk in nks:
        for j0 in range(0, nk, seg_len):
            j1 = min(nk, j0 + seg_len)
            for q in range(2 * span):
                pos = j0 - span + q if q < span else j0 + 1 + q - span
                total += 0 <= pos < nk
            for j in range(j0, j1 - 1):
                total += 1 + (j + 1 + span < nk)
    return total


@pytest.mark.parametrize("span", [1, 2, 5])
def test_span_rows_matches_a_step_by_step_count(span):
    rng = random.Random(span)
    nks = [rng.choice([0, 2, 3, 5, 7, 127, 128, 129, 255, 256, 300, 451, 1000]) for _ in range(300)]
    assert bench.span_rows(torch, torch.tensor(nks), span) == _kernel_span_loads(nks, span)


def test_span_rows_one_long_document():
    # one document of 1000 kept words, span 5, work units of 128: every unit but the first starts with
    # 10 rows, every later centre brings 2 rows except the last 5 of the document (no row ahead)
    n = bench.span_rows(torch, torch.tensor([1000]), 5)
    assert n == _kernel_span_loads([1000], 5)
    assert 2 * 1000 - 20 < n < 2 * 1000 + 8 * 10
