"""The attention calls inside a captured HIP graph.

The library allocates nothing, synchronises nothing and issues no memset on
the caller's stream, so a forward + backward can be captured once and
replayed.  Each replay is checked bit for bit against the eager result, with
eager work of the program itself and a device synchronisation between the
replays.  Rows of 700 tokens take the persistent kernels (several work items
per workgroup), rows of 200 tokens at D=64 the one-kernel backward; the
document-masked cases pass offsets prepared outside the capture (their
host-to-device copy is not a graph operation).
"""
import pytest
import torch

import synth
import paper_2405_13226_amd as dd
from paper_2405_13226_amd.attention import DocLens

from parity import log, to_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("D,docs,L", [(64, False, 700), (128, False, 700), (64, True, 700),
                                      (128, True, 700), (64, False, 200), (64, True, 200)])
def test_graph_replay_matches_eager(cuda, D, docs, L):
    B, H = 2, 2
    x = {n: to_dev(a, cuda) for n, a in synth.attention_inputs(B, L, H, D, seed=40 + D).items()}
    offs = [0, 150, 600, 700, 1100, 1400] if L == 700 else [0, 30, 170, 200, 290, 400]
    cu = DocLens(offs, B * L, cuda) if docs else None
    log(f"graph case D={D} docs={docs} L={L}")

    def step():
        o, lse = dd.forward(x["q"], x["k"], x["v"], cu_doclens=cu)
        return (o, lse) + tuple(dd.backward(x["q"], x["k"], x["v"], o, lse, x["do"],
                                            cu_doclens=cu))

    ref = [t.clone() for t in step()]
    torch.cuda.synchronize(cuda)

    side = torch.cuda.Stream(cuda)
    side.wait_stream(torch.cuda.current_stream(cuda))
    with torch.cuda.stream(side):
        step()  # warm-up on the capture stream
    torch.cuda.current_stream(cuda).wait_stream(side)
    torch.cuda.synchronize(cuda)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        out = step()
    torch.cuda.synchronize(cuda)

    other = {n: to_dev(a, cuda) for n, a in synth.attention_inputs(1, 300, 1, D, seed=7).items()}
    for rep in range(3):
        for t in out:
            t.zero_()
        graph.replay()
        torch.cuda.synchronize(cuda)
        for name, a, b in zip(("o", "lse", "dq", "dk", "dv"), out, ref):
            assert torch.equal(a, b), f"replay {rep}: {name} differs from the eager result"
        # eager work of the program between replays
        o2, lse2 = dd.forward(other["q"], other["k"], other["v"])
        dd.backward(other["q"], other["k"], other["v"], o2, lse2, other["do"])
        torch.cuda.synchronize(cuda)
