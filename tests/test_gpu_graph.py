"""The resident stack enqueues kernel launches only (no allocation, memset or
host synchronisation), so a caller can capture a whole forward in one HIP
graph and replay it.  Each replay must reproduce the eager result bit for
bit; replays are separated by eager work and synchronisations."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from tests.gpu_util import dev, dev_u16, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ql():
    import paper_2608_30877_amd as ql

    return ql


def _layers(seed, d, dff, n):
    mk = lambda l, i, rows, k: O.quantize_pack(synth.weights_f32(synth.matrix_seed(seed, l, i), rows, k))
    out = []
    for l in range(n):
        layer = {"qkv": mk(l, 0, 3 * d, d), "out": mk(l, 1, d, d), "up": mk(l, 2, dff, d),
                 "down": mk(l, 3, d, dff)}
        out.append({k: (dev(q), dev_u16(s)) for k, (q, s) in layer.items()})
    return out


@pytest.mark.parametrize("M,attn", [(8, None), (200, None), (256, "uniform"), (240, "ragged")])
def test_stack_graph_replay_matches_eager(ql, M, attn):
    d, dff, n = 256, 1024, 4
    say(f"graph replay M={M} attn={attn}")
    layers = _layers(70, d, dff, n)
    arr = ql.make_layers(layers)
    if attn == "uniform":
        cfg = (2, 64, 40)
    elif attn == "ragged":
        lengths = [100, 3, 77, 60]
        cu = torch.tensor(np.concatenate([[0], np.cumsum(lengths)]), dtype=torch.int32,
                          device="cuda")
        cfg = (2, cu, max(lengths), 32768)
    else:
        cfg = None
    h0 = dev(synth.residual_f32(70 + M, M, d))
    ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
    h = h0.clone()
    # eager reference (also warms up the library on this stream)
    ref = h0.clone()
    ql.stack_forward(arr, ref, dff, ws, attn=cfg)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        h.copy_(h0)
        ql.stack_forward(arr, h, dff, ws, attn=cfg)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        ql.stack_forward(arr, h, dff, ws, attn=cfg)
    for rep in range(3):
        h.copy_(h0)                       # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(h, ref), f"replay {rep} differs from the eager forward"
    # eager again after the replays: unchanged
    h2 = h0.clone()
    ql.stack_forward(arr, h2, dff, ws, attn=cfg)
    torch.cuda.synchronize()
    assert torch.equal(h2, ref)
    del g


@pytest.mark.parametrize("M", [2048, 8])
def test_qlinear_forward_graph_replay_matches_eager(ql, M):
    """qlinear_forward allocates nothing and never synchronises, so it can be
    captured: M = 2048 (the MFMA kernel on x as stored) and M = 8 (the
    small-batch kernel), K = 12288, N = 36864, each replay bit-equal to the
    eager call."""
    K, N = 12288, 36864
    say(f"graph replay of qlinear_forward M={M}")
    x = dev_u16(synth.activations_bf16(synth.SEED_QKV, M, K, outlier_frac=0.01))
    qw = synth.random_packed_bytes_cuda(71, N, K)
    sc = synth.random_scales_f16_cuda(71, N, K // 128)
    ref = ql.forward(x, qw, sc)
    torch.cuda.synchronize()
    y = torch.empty_like(ref)
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        ql.forward(x, qw, sc, out=y)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        ql.forward(x, qw, sc, out=y)
    for rep in range(3):
        y.zero_()                          # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref), f"replay {rep} differs from the eager call"
    del g
