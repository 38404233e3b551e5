"""GPU tests of the host-streamed stack (qlayer_stack_forward_streamed): the
weights stay in page-locked host memory and are copied block by block into
two device slots while the previous block computes.  The kernels and their
inputs are the resident stack's, so the results must be identical bit for
bit; the oracle parity of those kernels is covered by the resident tests."""
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


def _layer_np(seed, l, d, dff, packed_by_oracle=True):
    shapes = {"qkv": (3 * d, d), "out": (d, d), "up": (dff, d), "down": (d, dff)}
    out = {}
    for i, (name, (n, k)) in enumerate(shapes.items()):
        s = synth.matrix_seed(seed, l, i)
        if packed_by_oracle:
            out[name] = O.quantize_pack(synth.weights_f32(s, n, k))
        else:
            out[name] = (synth.random_packed_bytes(s, n, k), synth.random_scales_f16(s, n, k // 128))
    return out


def _on_device(layer):
    return {k: (dev(q), dev_u16(s)) for k, (q, s) in layer.items()}


def _pinned(layer):
    """Page-locked host copies (new pinned tensors, no registration)."""
    return {k: (torch.from_numpy(q).pin_memory(),
                torch.from_numpy(np.ascontiguousarray(s).view(np.int16)).pin_memory())
            for k, (q, s) in layer.items()}


def _run_both(ql, layers_np, h0, dff, attn=None):
    M, d = h0.shape
    dev_layers = [_on_device(x) for x in layers_np]
    host_layers = [_pinned(x) for x in layers_np]
    ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
    slots = torch.empty(2 * ql.stack_slot_bytes(d, dff), dtype=torch.uint8, device="cuda")
    a = dev(h0)
    ql.stack_forward(ql.make_layers(dev_layers), a, dff, ws, attn=attn)
    b = dev(h0)
    cs = torch.cuda.Stream()
    host_arr = ql.make_layers(host_layers)
    ql.stack_forward_streamed(host_arr, b, dff, ws, slots, cs, attn=attn)
    torch.cuda.synchronize()
    return a, b


@pytest.mark.parametrize("M", [8, 64, 300])
def test_streamed_equals_resident(ql, M):
    d, dff, L = 256, 1024, 6
    say(f"streamed stack M={M}")
    layers = [_layer_np(60, l, d, dff) for l in range(L)]
    h0 = synth.residual_f32(60 + M, M, d)
    a, b = _run_both(ql, layers, h0, dff)
    assert torch.equal(a, b)
    # and the result is the oracle's (end to end, as for the resident stack)
    if M == 64:
        ref = h0
        for x in layers:
            ref = O.stack_layer(ref, x)
        err = O.rel_fro(b.cpu().numpy().astype(np.float64) - h0, ref.astype(np.float64) - h0)
        assert err <= 5e-3


def test_streamed_with_attention_equals_resident(ql):
    d, dff, L, M = 256, 1024, 5, 256
    layers = [_layer_np(61, l, d, dff) for l in range(L)]
    h0 = synth.residual_f32(61, M, d)
    a, b = _run_both(ql, layers, h0, dff, attn=(2, 128, 100))
    assert torch.equal(a, b)


def test_streamed_larger_blocks_equal_resident(ql):
    """d = 1024, d_ff = 4096 (3.4 MB of weights per block), 8 blocks, 1024
    tokens: copies long enough to overlap the previous block's compute."""
    d, dff, L, M = 1024, 4096, 8, 1024
    say("streamed stack, larger blocks")
    layers = [_layer_np(62, l, d, dff, packed_by_oracle=False) for l in range(L)]
    h0 = synth.residual_f32(62, M, d)
    a, b = _run_both(ql, layers, h0, dff)
    assert torch.equal(a, b)


def test_streamed_back_to_back_calls(ql):
    """Two calls in a row on the same slots and stream with different
    weights, enqueued with no synchronisation between them (the second
    call's first copies must wait for the first call's last blocks): each
    equals its resident result, computed beforehand."""
    d, dff, M, L = 256, 1024, 40, 3
    ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
    slots = torch.empty(2 * ql.stack_slot_bytes(d, dff), dtype=torch.uint8, device="cuda")
    cs = torch.cuda.Stream()
    cases = []
    for seed in (63, 64):
        layers = [_layer_np(seed, l, d, dff) for l in range(L)]
        h0 = synth.residual_f32(seed, M, d)
        ref = dev(h0)
        ql.stack_forward(ql.make_layers([_on_device(x) for x in layers]), ref, dff, ws)
        cases.append((layers, h0, ref))
    torch.cuda.synchronize()
    keep, outs = [], []
    for layers, h0, ref in cases:
        host = [_pinned(x) for x in layers]
        keep.append(host)
        b = dev(h0)
        outs.append((ref, b))
    torch.cuda.synchronize()   # inputs in place; nothing below synchronises
    for (layers, h0, ref), host, (_, b) in zip(cases, keep, outs):
        ql.stack_forward_streamed(ql.make_layers(host), b, dff, ws, slots, cs)
    torch.cuda.synchronize()
    for ref, b in outs:
        assert torch.equal(ref, b)


def test_streamed_refuses_pageable_host_memory(ql):
    d, dff, M = 256, 1024, 8
    layer = _layer_np(65, 0, d, dff)
    pageable = {k: (torch.from_numpy(q), torch.from_numpy(np.ascontiguousarray(s).view(np.int16)))
                for k, (q, s) in layer.items()}
    ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
    slots = torch.empty(2 * ql.stack_slot_bytes(d, dff), dtype=torch.uint8, device="cuda")
    h = dev(synth.residual_f32(65, M, d))
    with pytest.raises(ql.QLError) as e:
        ql.stack_forward_streamed(ql.make_layers([pageable]), h, dff, ws, slots,
                                  torch.cuda.Stream())
    assert e.value.code == 1
