"""Write the stored expected values under tests/golden/ (test code only).

Every value here is computed by the CPU oracle (``oracle/stage_oracle.py``)
in float64 from the seeded input generators; nothing comes from the HIP path.
The paper prints no worked example of a decoder layer, so these files anchor
the oracle's own results: ``tests/test_oracle_golden.py`` recomputes them and
fails if a later change to the oracle's arithmetic moves any value. The
oracle itself is pinned to closed forms, invariants and library layers by
``tests/test_oracle_pins.py``.

Run from the repository root:  python -m tests.golden.make_golden
"""

from __future__ import annotations

import os

import numpy as np

from oracle import stage_oracle as O
from paper_2606_18600_amd import synth
from tests.helpers import ocfg, seqs_from

HERE = os.path.dirname(os.path.abspath(__file__))

# Two decoder layers of the tiny shape (hidden 256, 4 query / 2 kv heads,
# head_dim 64, ffn 704), global layers 0 and 1, weights from the seeded
# generator: a prefill of two prompts (21 and 9 tokens, shuffled 16-token
# blocks), then one decode step of both sequences.
SEED = 2606
PROMPTS = (21, 9)


def tiny_case():
    shape = synth.TINY
    cfg = ocfg(shape)
    layers = [synth.host_layer_weights(shape, SEED, l) for l in range(2)]
    totals = [p + 1 for p in PROMPTS]
    nb = sum((t + 15) // 16 for t in totals) + 2
    bt = synth.make_block_tables(totals, max((t + 15) // 16 for t in totals),
                                 synth.BlockAllocator(nb, SEED))
    kv = O.new_kv_cache(cfg, 2, nb)
    x_pf = synth.hidden_states(SEED, 1, sum(PROMPTS), shape.hidden, np.float64)
    y_pf = O.stage_forward(cfg, layers, x_pf, seqs_from([0, 0], PROMPTS, bt), kv)
    x_dc = synth.hidden_states(SEED, 2, len(PROMPTS), shape.hidden, np.float64)
    y_dc = O.stage_forward(cfg, layers, x_dc, seqs_from(PROMPTS, [1, 1], bt), kv)
    return y_pf, y_dc


HEADER = """# Expected stage outputs of the float64 oracle (oracle/stage_oracle.py):
# tiny shape (hidden 256, n_q 4, n_kv 2, head_dim 64, ffn 704, eps 1e-5,
# rope theta 5e5), global layers [0, 2), seed {seed}; prefill of prompts
# {prompts} (rows in batch order), then one decode step of both sequences.
# The layer is the pre-norm block of the paper's served models (Sec. 7) with
# the operations of Table 2; readings of the paper as in the oracle.
# Written by tests/golden/make_golden.py (calls only oracle/ and the seeded
# input generators). Values at 17 significant digits: the first and last row
# of each prompt and both decode rows in full, and for every prefill row its
# sum and its sum of squares.
"""

FULL_PREFILL_ROWS = (0, 20, 21, 29)  # first / last row of each prompt


def write(path, name, rows):
    with open(path, "a") as f:
        f.write(f"[{name}] {rows.shape[0]} x {rows.shape[1]}\n")
        for r in rows:
            f.write(" ".join(f"{v:.17g}" for v in r) + "\n")


def main():
    path = os.path.join(HERE, "tiny_stage_oracle.txt")
    y_pf, y_dc = tiny_case()
    with open(path, "w") as f:
        f.write(HEADER.format(seed=SEED, prompts=list(PROMPTS)))
    write(path, "prefill_rows_0_20_21_29", y_pf[list(FULL_PREFILL_ROWS)])
    write(path, "prefill_row_sum_and_sumsq", np.stack([y_pf.sum(1), (y_pf * y_pf).sum(1)], 1))
    write(path, "decode", y_dc)
    print(f"wrote {path}")


if __name__ == "__main__":
    main()
