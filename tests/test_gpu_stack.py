"""GPU parity of the linear stack (qlayer_stack_forward) against the oracle.

Small-width stacks are compared end to end; the 175B-width block is compared
on sampled tokens (tokens never mix in this stack, so the oracle can compute a
few rows of the full-width block exactly); the zero-scale invariant is checked
over all 96 layers at full width.
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from tests.gpu_util import bf16_as_f64, dev, dev_u16, host_u16, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ql():
    import paper_2608_30877_amd as ql

    return ql


def _packed_layer_oracle(seed, layer, d, dff):
    """Weights N(0, 0.02) packed by the oracle (host, small widths)."""
    mk = lambda i, n, k: O.quantize_pack(synth.weights_f32(synth.matrix_seed(seed, layer, i), n, k))
    return {"qkv": mk(0, 3 * d, d), "out": mk(1, d, d), "up": mk(2, dff, d), "down": mk(3, d, dff)}


def _packed_layer_direct(seed, layer, d, dff):
    """Packed weights drawn directly: uniform code bytes and scales in the
    range N(0, 0.02) weights give (full widths, no host packing needed)."""
    def mk(i, n, k):
        s = synth.matrix_seed(seed, layer, i)
        return synth.random_packed_bytes(s, n, k), synth.random_scales_f16(s, n, k // 128)
    return {"qkv": mk(0, 3 * d, d), "out": mk(1, d, d), "up": mk(2, dff, d), "down": mk(3, d, dff)}


def _to_dev(layer):
    return {k: (dev(q), dev_u16(s)) for k, (q, s) in layer.items()}


def _run(ql, dev_layers, h0, dff, n_layers=None):
    M, d = h0.shape
    ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
    arr = ql.make_layers(dev_layers)
    h = dev(h0)
    ql.stack_forward(arr, h, dff, ws, n_layers=n_layers)
    torch.cuda.synchronize()
    return h, ws


@pytest.mark.parametrize("M", [8, 16, 24, 64, 200])
def test_small_stack_end_to_end(ql, M):
    """4 blocks at d = 256, d_ff = 1024 (small-batch kernel for M <= 16, MFMA
    kernel with 32-, 64- and 128-row tiles above)."""
    d, dff, L = 256, 1024, 4
    say(f"stack M={M} d={d} L={L}")
    layers = [_packed_layer_oracle(40, l, d, dff) for l in range(L)]
    h0 = synth.residual_f32(40 + M, M, d)
    h, _ = _run(ql, [_to_dev(x) for x in layers], h0, dff)
    ref = h0
    for x in layers:
        ref = O.stack_layer(ref, x)
    got = h.cpu().numpy()
    err = O.rel_fro(got.astype(np.float64) - h0, ref.astype(np.float64) - h0)
    say(f"  end-to-end rel err of the residual update: {err:.3e}")
    assert err <= 5e-3


@pytest.mark.parametrize("M", [8, 24, 64])
def test_small_stack_intermediates(ql, M):
    """One block: the workspace's qkv and u buffers against the oracle's."""
    d, dff = 256, 1024
    layer = _packed_layer_oracle(41, 0, d, dff)
    h0 = synth.residual_f32(41 + M, M, d)
    h, ws = _run(ql, [_to_dev(layer)], h0, dff)
    _, mid = O.stack_layer(h0, layer, keep=True)
    qoff, uoff = ql.stack_workspace_offsets(M, d, dff)
    qkv = host_u16(ws[qoff:qoff + M * 3 * d * 2].view(torch.int16)).reshape(M, 3 * d)
    u = host_u16(ws[uoff:uoff + M * dff * 2].view(torch.int16)).reshape(M, dff)
    if M > 16:
        # the MFMA path keeps u in its operand layout: element e of every
        # 8-element chunk sits at position 2 * (e % 4) + e // 4
        c = np.arange(dff)
        u = u[:, (c & ~7) + 2 * (c & 3) + ((c & 7) >> 2)]
    assert O.rel_fro(bf16_as_f64(qkv), bf16_as_f64(mid["qkv"])) <= 5e-3
    assert O.rel_fro(bf16_as_f64(u), bf16_as_f64(mid["u"])) <= 5e-3


def test_zero_scales_keep_residual_small(ql):
    d, dff, M = 256, 1024, 40
    z = lambda n, k: (synth.random_packed_bytes(n + k, n, k), synth.const_f16_bits(n, k // 128, 0))
    layer = {"qkv": z(3 * d, d), "out": z(d, d), "up": z(dff, d), "down": z(d, dff)}
    h0 = synth.residual_f32(5, M, d)
    h, _ = _run(ql, [_to_dev(layer)] * 6, h0, dff)
    np.testing.assert_array_equal(h.cpu().numpy(), h0)


def test_zero_scales_keep_residual_full_96_layers(ql):
    """175B shape, M = 4096 tokens (8 pairs x 512), 96 blocks whose scales are
    all zero: the residual stream leaves the stack bit for bit unchanged."""
    d, dff, M, L = 12288, 49152, 4096, 96
    say("stack zero-scale 96 layers full width")
    g = torch.Generator("cuda").manual_seed(3)
    mk = lambda n, k: (torch.randint(0, 256, (n, k // 2), dtype=torch.uint8, device="cuda",
                                     generator=g),
                       torch.zeros((n, k // 128), dtype=torch.int16, device="cuda"))
    layer = {"qkv": mk(3 * d, d), "out": mk(d, d), "up": mk(dff, d), "down": mk(d, dff)}
    h0 = synth.residual_f32(6, M, d)
    h, _ = _run(ql, [layer] * L, h0, dff)
    assert torch.equal(h.cpu(), torch.from_numpy(h0))


def test_full_width_two_blocks_sampled_tokens(ql):
    """Two 175B-width blocks (layers 0 and 1 of the seeded stack) at
    M = 4096: 16 sampled tokens against the oracle run through both blocks
    from the same seeded input (tokens never mix in this stack, so the
    oracle's rows are exact), checked after each block."""
    d, dff, M = 12288, 49152, 4096
    say("stack full-width blocks 0 and 1")
    layers = [_packed_layer_direct(synth.SEED_STACK, l, d, dff) for l in range(2)]
    dev_layers = [_to_dev(x) for x in layers]
    h0 = synth.residual_f32(synth.SEED_STACK, M, d)
    rows = np.sort(np.random.default_rng(8).choice(M, 16, replace=False))
    h1, _ = _run(ql, dev_layers[:1], h0, dff)
    got1 = h1.cpu().numpy()[rows].astype(np.float64)
    del h1
    h2, _ = _run(ql, dev_layers, h0, dff)
    got2 = h2.cpu().numpy()[rows].astype(np.float64)
    del h2, dev_layers
    say("  oracle on sampled tokens, block 0")
    ref1 = O.stack_layer(h0[rows], layers[0])
    err1 = O.rel_fro(got1 - h0[rows], ref1.astype(np.float64) - h0[rows])
    say(f"  block 0: rel err of the residual update {err1:.3e}")
    assert err1 <= 5e-3
    say("  oracle on sampled tokens, block 1")
    ref2 = O.stack_layer(ref1, layers[1]).astype(np.float64)
    err2 = O.rel_fro(got2 - h0[rows], ref2 - h0[rows])
    say(f"  blocks 0-1: rel err of the residual update {err2:.3e}")
    assert err2 <= 5e-3
