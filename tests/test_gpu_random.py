"""Seeded random configurations against the fp64 oracle.

Shapes, masks and document layouts are drawn from a fixed seed so that the
cases land on both sides of the launchers' choices (persistent or one block
per workgroup, grids smaller or larger than the item count) and on ragged
tails; each case compares the forward and backward of three sampled (b, h)
slices element by element (slices are independent, so this is exact parity
for them).
"""
import numpy as np
import pytest

import synth
from paper_2405_13226_amd import dd

from parity import check_case

pytestmark = pytest.mark.gpu


def _cases(n=40, seed=2405):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        D = int(rng.choice([64, 128]))
        L = int(rng.choice([int(rng.integers(1, 160)), int(rng.integers(160, 1200)),
                            int(rng.integers(1200, 2600))]))
        B = int(rng.integers(1, 40))
        H = int(rng.integers(1, 9))
        causal = bool(rng.random() < 0.8)
        cu = None
        if rng.random() < 0.4 and B * L >= 2:
            lens = synth.lognormal_doc_lengths(int(rng.integers(1 << 30)), total_tokens=B * L,
                                               median=float(rng.choice([40, 150, 600])),
                                               sigma=1.0)
            cu = dd.chunk_doclens(lens, B * L)
        bh = sorted({(int(rng.integers(B)), int(rng.integers(H))) for _ in range(3)})
        out.append((i, B, L, H, D, causal, cu, bh))
    return out


@pytest.mark.parametrize("case", _cases(), ids=lambda c: f"case{c[0]}")
def test_random_configuration(cuda, case):
    i, B, L, H, D, causal, cu, bh = case
    check_case(B, L, H, D, causal=causal, cu=cu, seed=100 + i, bh=bh,
               tag=f"random {i}: B={B} L={L} H={H} D={D} causal={int(causal)} "
                   f"docs={None if cu is None else len(cu) - 1}")
