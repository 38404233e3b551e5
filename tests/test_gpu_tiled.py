"""GPU tests of the tiled code layout (QL_LAYOUT_TILED in include/qlinear.h).

The conversion entry points are checked byte for byte against the host
definition in tests/layout_ref.py.  The layout changes where the kernels read
the codes from, not the arithmetic, so every forward path on tiled codes must
reproduce the same path on row-major codes bit for bit: the small-batch
kernel at each of its widths, the MFMA kernel with 32-, 64- and 128-row tiles
on both operand forms and every epilogue, the >2^31-byte launch split, and
the stack entry points (resident, with attention, host-streamed, allocation-
free).  One exact-arithmetic case per kernel also goes to the oracle directly.
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from tests.gpu_util import dev, dev_u16, host_u16, say
from tests.layout_ref import tile_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ql():
    import paper_2608_30877_amd as ql

    return ql


def _bits(t):
    return t.view(torch.int32 if t.dtype == torch.float32 else torch.int16)


# ------------------------------------------------------------------ conversion

@pytest.mark.parametrize("N,K", [(16, 128), (48, 384), (4112, 1024), (12288, 12288)])
def test_tile_untile_bit_exact(ql, N, K):
    say(f"tile N={N} K={K}")
    qw = synth.random_packed_bytes(40 + N % 7, N, K)
    t = ql.tile_codes(dev(qw))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(t.cpu().numpy().reshape(-1), tile_np(qw))
    back = ql.untile_codes(t)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(back.cpu().numpy(), qw)


# ------------------------------------------------------------------ single projections

def _forward_pair(ql, M, N, K, epi, with_ws, seed):
    """The same projection on row-major and on tiled codes."""
    x = dev_u16(synth.activations_bf16(seed, M, K))
    qw = synth.random_packed_bytes_cuda(seed + 1, N, K)
    sc = synth.random_scales_f16_cuda(seed + 2, N, K // 128)
    qt = ql.tile_codes(qw)
    ws = None
    if with_ws and ql.workspace_bytes(M, K) > 0:
        ws = torch.empty(ql.workspace_bytes(M, K), dtype=torch.uint8, device="cuda")
    outs = []
    for q, tiled in ((qw, False), (qt, True)):
        if epi == ql.EPI_RESID_F32:
            out = torch.from_numpy(synth.residual_f32(seed + 3, M, N)).cuda()
        else:
            out = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
        ql.forward_ex(x, q, sc, out, epi, ws, tiled=tiled)
        outs.append(out)
    torch.cuda.synchronize()
    return outs


# small-batch kernel: 6-fragment (N = 49152, 24560 ragged), 3-fragment with
# pair tiles (36864), eight waves (12288 x 49152), 4-fragment (12304), one group
GEMV_SHAPES = [(1, 49152, 12288), (8, 36864, 12288), (8, 12288, 49152), (16, 24560, 384),
               (5, 12304, 640), (3, 12288, 128)]


@pytest.mark.parametrize("M,N,K", GEMV_SHAPES)
@pytest.mark.parametrize("epi", [0, 1, 2])
def test_small_batch_tiled_equals_rows(ql, M, N, K, epi):
    say(f"small batch tiled M={M} N={N} K={K} epi={epi}")
    a, b = _forward_pair(ql, M, N, K, epi, False, 50 + M + epi)
    assert torch.equal(_bits(a), _bits(b))


# MFMA kernel: 32-, 64- and 128-row tiles, ragged N (not a multiple of 256)
GEMM_SHAPES = [(17, 1296, 1024), (64, 528, 512), (300, 4112, 2048), (2048, 12288, 12288)]


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("epi", [0, 1, 2])
@pytest.mark.parametrize("with_ws", [False, True])
def test_mfma_tiled_equals_rows(ql, M, N, K, epi, with_ws):
    say(f"mfma tiled M={M} N={N} K={K} epi={epi} ws={with_ws}")
    a, b = _forward_pair(ql, M, N, K, epi, with_ws, 60 + M + epi)
    assert torch.equal(_bits(a), _bits(b))


# The small-batch kernel's pair loop: each wave takes every W-th pair of
# groups, runs its main loop while two pairs ahead exist and its last two or
# three pairs after it, requesting nothing past them; an odd G's last pair
# has one group.  Group counts G that give every wave 0-5 pairs, with odd and
# even counts and odd G, for the widths N selects: 6 fragments (N = 24576),
# 3 with pair tiles (36864), 3 with eight waves (12288), 4 single tiles
# (12304).  Exact arithmetic (ternary x, per-(column, group) power-of-two
# scales), so both layouts must equal the oracle bit for bit on sampled
# columns (every 5th, and the last 40).
PAIR_TAILS = [(8, 24576, 1), (8, 24576, 3), (8, 24576, 9), (16, 24576, 17), (1, 24576, 37),
              (8, 24576, 31), (8, 36864, 5), (13, 36864, 25), (8, 12288, 13), (4, 12288, 26),
              (8, 12304, 3), (16, 12304, 10)]


@pytest.mark.parametrize("M,N,G", PAIR_TAILS)
def test_small_batch_pair_tails_exact(ql, M, N, G):
    K = 128 * G
    say(f"pair tails M={M} N={N} G={G}")
    x = synth.ternary_bf16(300 + G, M, K)
    qw = synth.random_packed_bytes(301 + G, N, K)
    sc = synth.pow2_scales_f16(302 + G, N, G)
    cols = np.unique(np.concatenate([np.arange(0, N, 5), np.arange(N - 40, N)]))
    want = O.f64_to_bf16_bits(O.qlinear_ref_cols(x, qw, sc, cols))
    qd = dev(qw)
    for q, tiled in ((qd, False), (ql.tile_codes(qd), True)):
        y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
        ql.forward_ex(dev_u16(x), q, dev_u16(sc), y, ql.EPI_NONE, None, tiled=tiled)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host_u16(y)[:, cols], want, err_msg=f"tiled={tiled}")


@pytest.mark.parametrize("M,N,K,with_ws", [(8, 4096, 1024, False), (300, 1296, 2048, False),
                                           (300, 1296, 2048, True)])
def test_tiled_exact_arithmetic_against_oracle(ql, M, N, K, with_ws):
    """Ternary x, uniform codes, per-(column, group) power-of-two scales:
    every partial sum is exact, so the tiled path equals the oracle bit for bit."""
    say(f"tiled exact M={M} N={N} K={K} ws={with_ws}")
    x = synth.ternary_bf16(70, M, K)
    qw = synth.random_packed_bytes(71, N, K)
    sc = synth.pow2_scales_f16(72, N, K // 128)
    qt = ql.tile_codes(dev(qw))
    ws = None
    if with_ws:
        ws = torch.empty(ql.workspace_bytes(M, K), dtype=torch.uint8, device="cuda")
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    ql.forward_ex(dev_u16(x), qt, dev_u16(sc), y, ql.EPI_NONE, ws, tiled=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host_u16(y), O.f64_to_bf16_bits(O.qlinear_ref(x, qw, sc)))


def test_tiled_launch_split_equals_rows(ql):
    """Codes past 2^31 bytes: the column chunks of the split start on 16-column
    block boundaries, so the tiled chunk offsets match the row-major ones."""
    M, N, K = 256, 360000, 12288
    say(f"tiled split M={M} N={N} K={K}")
    x = synth.ternary_bf16_cuda(81, M, K)
    qw = synth.random_packed_bytes_cuda(82, N, K)
    sc = synth.pow2_scales_f16_cuda(83, N, K // 128)
    qt = ql.tile_codes(qw)
    ya = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    yb = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    ql.forward_ex(x, qw, sc, ya, ql.EPI_NONE, None)
    del qw
    ql.forward_ex(x, qt, sc, yb, ql.EPI_NONE, None, tiled=True)
    torch.cuda.synchronize()
    assert torch.equal(_bits(ya), _bits(yb))
    del x, qt, sc, ya, yb
    torch.cuda.empty_cache()


# ------------------------------------------------------------------ stack entry points

def _layers(ql, seed, d, dff, n):
    shapes = {"qkv": (3 * d, d), "out": (d, d), "up": (dff, d), "down": (d, dff)}
    rows, tiled = [], []
    for l in range(n):
        r, t = {}, {}
        for i, (name, (nn, k)) in enumerate(shapes.items()):
            s = synth.matrix_seed(seed, l, i)
            q = synth.random_packed_bytes_cuda(s, nn, k)
            sc = synth.random_scales_f16_cuda(s + 1, nn, k // 128)
            r[name] = (q, sc)
            t[name] = (ql.tile_codes(q), sc, ql.LAYOUT_TILED)
        rows.append(r)
        tiled.append(t)
    return rows, tiled


@pytest.mark.parametrize("M,attn", [(8, None), (64, None), (300, None), (128, (2, 64, 32))])
def test_stack_tiled_equals_rows(ql, M, attn):
    d, dff, L = 256, 1024, 3
    say(f"stack tiled M={M} attn={attn}")
    rows, tiled = _layers(ql, 90 + M, d, dff, L)
    h0 = synth.residual_f32(91 + M, M, d)
    ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
    a, b = dev(h0), dev(h0)
    ql.stack_forward(ql.make_layers(rows), a, dff, ws, attn=attn)
    ql.stack_forward(ql.make_layers(tiled), b, dff, ws, attn=attn)
    torch.cuda.synchronize()
    assert torch.equal(_bits(a), _bits(b))


@pytest.mark.parametrize("M", [8, 300])
def test_streamed_and_noalloc_tiled_equal_rows(ql, M):
    """Host-streamed blocks keep the host matrices' layouts in the device
    slots; the allocation-free entry point takes tiled layers as well."""
    d, dff, L = 256, 1024, 3
    say(f"streamed / noalloc tiled M={M}")
    rows, tiled = _layers(ql, 95 + M, d, dff, L)
    pinned = [{k: (q.cpu().pin_memory(), s.cpu().pin_memory(), lay)
               for k, (q, s, lay) in layer.items()} for layer in tiled]
    h0 = synth.residual_f32(96 + M, M, d)
    ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
    slots = torch.empty(2 * ql.stack_slot_bytes(d, dff), dtype=torch.uint8, device="cuda")
    a, b, c = dev(h0), dev(h0), dev(h0)
    ql.stack_forward(ql.make_layers(rows), a, dff, ws)
    cs = torch.cuda.Stream()
    ql.stack_forward_streamed(ql.make_layers(pinned), b, dff, ws, slots, cs)
    torch.cuda.synchronize()
    ql.stack_forward_noalloc(ql.make_layers(tiled), c, dff)
    torch.cuda.synchronize()
    assert torch.equal(_bits(a), _bits(b))
    assert torch.equal(_bits(a), _bits(c))
