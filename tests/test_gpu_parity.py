"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Small cases compare every element; the full 65,536-token buckets compare all
rows of sampled (b, h) pairs, which is exact parity for those pairs because
pairs are independent.  Tolerances are in tests/parity.py.
"""
import numpy as np
import pytest

import synth
from paper_2405_13226_amd import dd

from parity import assert_ok, check_case, compare, gpu_run, log

pytestmark = pytest.mark.gpu


def test_tiny_config_full_parity(cuda):
    # B=4 sequences x L=256, H=4, D=64, causal: every output element.
    _, _, res = check_case(4, 256, 4, 64, causal=True, seed=0, tag="tiny")
    assert res["o_maxabs"] <= 1e-2


@pytest.mark.parametrize("B,L,H,D,causal", [
    (1, 1, 1, 64, True), (3, 1, 2, 128, True), (2, 7, 3, 64, True), (1, 100, 2, 128, True),
    (2, 129, 1, 64, True), (1, 300, 2, 128, True), (2, 64, 2, 64, False),
    (1, 200, 1, 128, False), (1, 513, 1, 64, True), (2, 384, 2, 128, True)])
def test_ragged_shapes(cuda, B, L, H, D, causal):
    check_case(B, L, H, D, causal=causal, seed=B * 1000 + L)


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("causal", [True, False])
def test_document_masked_chunks(cuda, D, causal):
    # Concat-and-chunk rows of 512 with short and row-crossing documents.
    B, L, H = 3, 512, 2
    lens = synth.lognormal_doc_lengths(5, total_tokens=B * L, median=150, sigma=1.0)
    cu = dd.chunk_doclens(lens, B * L)
    check_case(B, L, H, D, causal=causal, cu=cu, seed=D + causal)


# Short rows take the persistent forms of the forward, dK/dV and (D = 64) dQ
# kernels, where a workgroup walks several blocks back to back.  Grids:
# forward 768 (D = 64) / 512 (D = 128) workgroups, dK/dV 512 / 256, dQ 512
# (D = 64).  48 x 3 slices of
# L = 700 hold 6 query blocks and 6 key blocks each (864 of each), so the last
# slices fall in a workgroup's second (or later) item; the last block of every
# slice holds 60 rows (ragged).  The choice follows the row length, so the
# document-masked case takes the same persistent forms.
PERSIST_CASES = {128: (48, [(0, 0), (15, 1), (31, 0), (40, 2), (47, 2)]),
                 64: (48, [(0, 0), (15, 1), (31, 0), (40, 2), (47, 2)])}


@pytest.mark.parametrize("D", [64, 128])
def test_persistent_kernels_several_items_per_workgroup(cuda, D):
    B, bh = PERSIST_CASES[D]
    check_case(B, 700, 3, D, causal=True, seed=11, bh=bh, tag=f"persistent D={D}")


@pytest.mark.parametrize("D", [64, 128])
def test_persistent_kernels_non_causal(cuda, D):
    # Without the causal mask every block spans its whole row.
    B, bh = PERSIST_CASES[D]
    check_case(B, 700, 3, D, causal=False, seed=13, bh=bh, tag=f"persistent D={D}, non-causal")


@pytest.mark.parametrize("D", [64, 128])
def test_persistent_kernels_document_masked(cuda, D):
    (B, bh), L, H = PERSIST_CASES[D], 700, 3
    lens = synth.lognormal_doc_lengths(2, total_tokens=B * L, median=300, sigma=0.8)
    cu = dd.chunk_doclens(lens, B * L)
    check_case(B, L, H, D, causal=True, cu=cu, seed=12, bh=bh,
               tag=f"persistent D={D}, documents")


# Rows of 129..256 tokens at D = 64 take the persistent one-kernel backward:
# 256 workgroups (one per CU) walk the slices b*H + h, a workgroup's next
# slice 256 further on, its inputs staged tile by tile during the previous
# slice.  200 x 3 slices give two or three slices per workgroup; the sampled
# slices 0, 256, 300, 512 and 599 are first, second and third slices of
# their workgroups.  L = 200 leaves a ragged last query tile.
SHORT_PERSIST_BH = [(0, 0), (85, 1), (100, 0), (170, 2), (199, 2)]


@pytest.mark.parametrize("L", [200, 256])
@pytest.mark.parametrize("mode", ["causal", "full", "docs"])
def test_short_rows_persistent_several_slices(cuda, L, mode):
    B, H = 200, 3
    cu = None
    if mode == "docs":
        lens = synth.lognormal_doc_lengths(L, total_tokens=B * L, median=L / 3, sigma=0.8)
        cu = dd.chunk_doclens(lens, B * L)
    check_case(B, L, H, 64, causal=mode != "full", cu=cu, seed=500 + L, bh=SHORT_PERSIST_BH,
               tag=f"persistent one-kernel backward L={L} {mode}")


# Persistent forward and dQ (D=64) whose items span a single key tile: rows
# of at most 64 tokens, or a ragged last query block that starts a document
# (documents of `doc` tokens).  Many items per workgroup, so the next item's
# rows are staged in LDS while the current item's only tile runs.
@pytest.mark.parametrize("B,L,H,doc", [(128, 48, 8, None), (64, 130, 8, 2), (16, 520, 8, 8)])
def test_persistent_one_tile_items(cuda, B, L, H, doc):
    cu = None if doc is None else dd.chunk_doclens([doc] * (B * L // doc), B * L)
    bh = [(0, 0), (B // 2, H - 1), (B - 1, 3)]
    check_case(B, L, H, 64, causal=True, cu=cu, seed=700 + L, bh=bh,
               tag=f"persistent one-tile items B={B} L={L} doc={doc}")


@pytest.mark.parametrize("B,L,D,causal", [(2, 700, 64, True), (2, 700, 128, False),
                                         (1, 2100, 64, True), (1, 2100, 128, True)])
def test_large_scores_forward(cuda, B, L, D, causal):
    # Q and K times 8 (exact in bf16): the scaled scores in log2 units reach
    # several hundred, far outside exp2's fp32 range, so each tile's running
    # maximum must be the true maximum of its rows (a smaller one overflows
    # the probabilities, a larger one underflows their sum).  L = 700 takes
    # the persistent forward, L = 2100 one block per workgroup.
    H = 2
    inputs = synth.attention_inputs(B, L, H, D, seed=21 + D, with_grad=False)
    for n in ("q", "k"):
        inputs[n] = synth.bf16_bits_from_f32(synth.f32_from_bf16_bits(inputs[n]) * 8.0)
    log(f"case large scores B={B} L={L} D={D} causal={int(causal)}")
    out = gpu_run(inputs, causal, None, "cuda:0", backward=False)
    for n, t in out.items():
        assert bool(np.isfinite(t.float().cpu().numpy()).all()), f"{n} has non-finite values"
    bh = [(b, h) for b in range(B) for h in range(H)]
    res = compare(inputs, out, causal, None, bh, backward=False, tag="large scores")
    assert_ok(res, backward=False)


def test_single_token_documents(cuda):
    B, L, H, D = 1, 130, 1, 64
    cu = np.arange(0, B * L + 1)
    check_case(B, L, H, D, cu=cu, seed=3)


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("L", [256, 512, 1024, 2048, 4096, 8192])
def test_full_step_buckets_sampled(cuda, L, D):
    # A 65,536-token step: B = 65536 / L sequences, H = 16, in the launch
    # configuration the benchmark times (every bucket of both head-dim
    # sweeps: persistent and one-block forms, the one-kernel short-row
    # backward at D = 64, L = 256).
    B, H = 65536 // L, 16
    bh = [(0, 0), (B - 1, H - 1), (B // 2, 7)]
    check_case(B, L, H, D, causal=True, seed=0, bh=bh, tag=f"bucket L={L} D={D}")


def test_concat_chunk_step_sampled(cuda):
    # 8 chunks x 8192 tokens of log-normal documents, document-masked.
    B, L, H, D = 8, 8192, 16, 64
    lens = synth.lognormal_doc_lengths(0)
    cu = dd.chunk_doclens(lens, B * L)
    check_case(B, L, H, D, causal=True, cu=cu, seed=0, bh=[(0, 0), (5, 9), (7, 15)],
               tag="chunk 8x8192 masked")


def test_packed_dd_step_real_shape(cuda):
    # A whole DD step in one document-masked launch, at the shape the
    # benchmark times: the binary pieces (256..8192 tokens) of a 65,536-token
    # step of log-normal documents (seed 0) packed into one row, H = 16,
    # D = 64.  Pieces never attend to each other, so each sampled piece of
    # the packed outputs must equal the oracle run on that piece alone (a DD
    # sequence of its length): the longest pieces, a middle one and the two
    # shortest, on two heads.
    H, D = 16, 64
    packed = dd.pack_step(synth.lognormal_doc_lengths(0), min_len=256, max_len=8192)
    cu, L = packed.cu_doclens, packed.tokens
    log(f"packed DD step: {len(cu) - 1} pieces, {L} tokens")
    assert len(cu) - 1 >= 50 and L > 50000
    inputs = synth.attention_inputs(1, L, H, D, seed=0, with_grad=True)
    out = gpu_run(inputs, True, cu, "cuda:0")
    lens = np.diff(cu)
    order = np.argsort(lens, kind="stable")
    picks = sorted({int(order[-1]), int(order[-2]), int(order[len(order) // 2]),
                    int(order[0]), int(order[1])})
    for i in picks:
        lo, hi = int(cu[i]), int(cu[i + 1])
        piece = {n: x[:, lo:hi] for n, x in inputs.items()}
        piece_out = {n: t[:, lo:hi] for n, t in out.items()}
        res = compare(piece, piece_out, True, None, [(0, 0), (0, 11)],
                      tag=f"packed piece {i}: tokens {lo}..{hi - 1} (length {hi - lo})")
        assert_ok(res)


def test_longest_bucket_sampled(cuda):
    B, L, H, D = 4, 16384, 16, 128
    check_case(B, L, H, D, causal=True, seed=0, bh=[(3, 15)], tag="bucket L=16384 D=128")
    log("done")


# D = 64 rows of at most 256 tokens (without RoPE) take the one-kernel
# backward, with a row capacity of 64, 128 or 256 tokens; each capacity is
# covered at and around its edges, with the causal mask, without it, and
# with documents.
@pytest.mark.parametrize("L", [1, 31, 64, 65, 100, 128, 129, 255, 256])
@pytest.mark.parametrize("mode", ["causal", "full", "docs"])
def test_short_rows_one_kernel_backward(cuda, L, mode):
    B, H = 3, 2
    cu = None
    if mode == "docs":
        lens = synth.lognormal_doc_lengths(L, total_tokens=B * L, median=max(L / 3, 1.0),
                                           sigma=0.8)
        cu = dd.chunk_doclens(lens, B * L)
    check_case(B, L, H, 64, causal=mode != "full", cu=cu, seed=300 + L,
               tag=f"one-kernel backward L={L} {mode}")
