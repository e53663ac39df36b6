"""The whole path captured in a HIP graph (torch.cuda.CUDAGraph over the library's launches).

The library's calls enqueue kernels only (no allocation, memset or synchronisation), so a step can be
captured once and replayed.  Each replay follows eager work on the same outputs (they are overwritten
with NaN by torch fills) and must reproduce the eager step bit for bit: the kernels use no atomics.
The eager step is itself checked against the oracle on sampled rows, so the replays are too.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_15592_amd as estp
import synth
from paper_2608_15592_amd.path import alloc_buffers
from synth import inputs as I
from tests._util import dev, host

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("workload,overrides", [
    ("qwen", {"n_prompts": 3, "seq_len": 300, "V": 20000}),
    ("ragged", {"n_prompts": 12, "ragged_max": 700, "V": 5000}),
], ids=["qwen-shaped-3x300", "ragged-12-prompts"])
def test_path_replays_in_a_hip_graph(workload, overrides):
    w = synth.get_workload(workload, **overrides)
    inp = I.make_inputs(w, 7)
    n_tok, B = int(inp["n_tok"]), len(inp["lengths"])
    max_len = int(inp["lengths"].max())
    Hdn, K = w.head
    X, W, Q, Kk = (dev(inp[k]) for k in ("X", "W", "Q", "K"))
    cu = dev(inp["cu_seqlens"])
    head = tuple(dev(inp[k]) for k in ("W1", "b1", "W2", "b2")) + (dev(inp["centres"]) if K > 1 else None,)
    bufs = alloc_buffers(n_tok, B, max_len, w.d, w.V, w.L, w.Hq, w.Hkv, w.dh, Hdn, K, X.device)

    def step():
        return estp.run_path(X, W, Q, Kk, cu, max_len, 0.5, 0.5, 1.0, "none", head=head, bufs=bufs)

    eager = {k: v.clone() for k, v in step().items() if isinstance(v, torch.Tensor)}
    torch.cuda.synchronize()
    rows = np.array(sorted({0, n_tok // 2, n_tok - 1}))
    ref_H = oracle.token_entropy(inp["X"][rows], inp["W"])
    assert np.abs(host(eager["H"])[rows] - ref_H).max() <= 2e-3

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up off the default stream, as torch asks before capture
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = step()
    torch.cuda.synchronize()
    outs = {k: v for k, v in out.items() if isinstance(v, torch.Tensor)}
    assert outs.keys() == eager.keys()
    for rep in range(3):
        for t in outs.values():  # eager work on the outputs between replays
            t.fill_(float("nan") if t.is_floating_point() else -1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, ref in eager.items():
            assert torch.equal(outs[k], ref), f"replay {rep}: {k} differs from the eager step"


def test_noalloc_entropy_replays_in_a_hip_graph():
    # estp_token_entropy_noalloc is for callers that cannot allocate, such as code under graph
    # capture: captured once with no workspace, replayed after eager calls that overwrite its
    # scratch with another problem's partial states; each replay equals the workspace entry point
    g = np.random.default_rng(5)
    n, d, V = 3000, 512, 30000
    X = dev(I.f32_to_bf16_bits((g.standard_normal((n, d)) / 1.0).astype(np.float32)))
    W = dev(I.f32_to_bf16_bits((g.standard_normal((V, d)) * 0.02).astype(np.float32)))
    X2 = dev(I.f32_to_bf16_bits(g.standard_normal((700, d)).astype(np.float32)))
    am_ref = torch.empty(n, dtype=torch.int32, device="cuda")
    H_ref = estp.token_entropy(X, W, vocab_argmax=am_ref)
    H = torch.empty(n, device="cuda")
    am = torch.empty(n, dtype=torch.int32, device="cuda")
    H2 = torch.empty(700, device="cuda")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        estp.token_entropy_noalloc(X, W, H, vocab_argmax=am)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        estp.token_entropy_noalloc(X, W, H, vocab_argmax=am)
    torch.cuda.synchronize()
    for rep in range(3):
        H.fill_(float("nan"))
        am.fill_(-1)
        estp.token_entropy_noalloc(X2, W, H2)  # eager call on the same scratch, another problem
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(H, H_ref), f"replay {rep}: H"
        assert torch.equal(am, am_ref), f"replay {rep}: argmax"
