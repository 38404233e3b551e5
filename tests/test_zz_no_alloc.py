"""qlayer_stack_forward_noalloc (the stack with its workspace in the
library's fixed device scratch) against qlayer_stack_forward with a caller
workspace, through the C ABI: the same kernels on the same inputs, so the
residual streams must agree bit for bit.  Two calls in a row, the second
with a smaller batch (the scratch keeps the first call's contents), and a
batch too large for the scratch, which is refused before anything runs."""
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


def _layers(d, dff, n):
    out = []
    for l in range(n):
        mk = lambda i, rows, k: O.quantize_pack(
            synth.weights_f32(synth.matrix_seed(90, l, i), rows, k))
        layer = {"qkv": mk(0, 3 * d, d), "out": mk(1, d, d), "up": mk(2, dff, d),
                 "down": mk(3, d, dff)}
        out.append({k: (dev(q), dev_u16(s)) for k, (q, s) in layer.items()})
    return out


def test_noalloc_matches_caller_workspace_twice(ql):
    d, dff, n = 256, 1024, 3
    layers = _layers(d, dff, n)
    arr = ql.make_layers(layers)
    for M in (300, 40, 8):          # MFMA path, then smaller batches, then small-batch kernel
        say(f"noalloc stack M={M}")
        h0 = dev(synth.residual_f32(91 + M, M, d))
        ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
        ref = h0.clone()
        ql.stack_forward(arr, ref, dff, ws)
        got = h0.clone()
        ql.stack_forward_noalloc(arr, got, dff)
        torch.cuda.synchronize()
        assert torch.equal(got, ref), f"M={M}"


def test_noalloc_full_width_small_batch(ql):
    """175B width, M = 64 tokens (fits the 128 MiB scratch), one block."""
    d, dff, M = 12288, 49152, 64
    say("noalloc stack full width M=64")
    g = torch.Generator("cuda").manual_seed(92)
    mk = lambda rows, k: (torch.randint(0, 256, (rows, k // 2), dtype=torch.uint8, device="cuda",
                                        generator=g),
                          synth.random_scales_f16_cuda(rows + k, rows, k // 128))
    layer = {"qkv": mk(3 * d, d), "out": mk(d, d), "up": mk(dff, d), "down": mk(d, dff)}
    arr = ql.make_layers([layer])
    h0 = dev(synth.residual_f32(92, M, d))
    ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
    ref = h0.clone()
    ql.stack_forward(arr, ref, dff, ws)
    got = h0.clone()
    ql.stack_forward_noalloc(arr, got, dff)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)


def test_noalloc_refuses_batches_beyond_the_scratch(ql):
    d, dff = 12288, 49152
    cap = ql.stack_scratch_capacity()
    assert cap == 128 << 20
    M = 598                          # the first batch whose workspace exceeds 128 MiB
    assert ql.stack_workspace_bytes(M, d, dff) > cap >= ql.stack_workspace_bytes(M - 1, d, dff)
    h = torch.zeros((M, d), dtype=torch.float32, device="cuda")
    p = torch.zeros(16, dtype=torch.uint8, device="cuda")
    fake = {k: (p, p.view(torch.int16)) for k in ("qkv", "out", "up", "down")}
    with pytest.raises(ql.QLError) as e:
        ql.stack_forward_noalloc(ql.make_layers([fake]), h, dff)
    assert e.value.code == 7
    torch.cuda.synchronize()
    assert not h.any()               # nothing ran
