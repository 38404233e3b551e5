"""GPU parity of the sliding-window attention kernel (qlinear_attention) and
of the stack with attention, against the oracle's attention_ref.

Tolerance, from the kernel's arithmetic: the scores are exact bf16 products
summed in fp32 (negligible error); the probabilities are rounded to bf16
(relative error <= 2^-9 each) and the normaliser sums the rounded values, so
every normalised weight is within a factor (1 +- 2^-9)/(1 -+ 2^-9) of the
exact one and the weighted sum moves by at most 2^-8 * max|v| (v over the
window); the bf16 store adds 2^-9 * |o|.  Each element must therefore lie
within 2^-8 * (max|V| + |o|) of the fp64 oracle -- a bound with a factor of
two of slack -- and the relative Frobenius error within 5e-3.
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from tests.gpu_util import bf16_as_f64, dev, dev_u16, host_u16, say

pytestmark = pytest.mark.gpu

TOL = 2.0 ** -8


@pytest.fixture(scope="module")
def ql():
    import paper_2608_30877_amd as ql

    return ql


def _check(got_bits, qkv_bits, d, heads, seq_len, window, ref=None):
    ref = O.attention_ref(qkv_bits, d, heads, seq_len, window) if ref is None else ref
    got = bf16_as_f64(got_bits)
    vmax = np.abs(bf16_as_f64(qkv_bits[:, 2 * d:3 * d])).max()
    bad = np.abs(got - ref) > TOL * (vmax + np.abs(ref))
    assert not bad.any(), f"{bad.sum()} elements outside the bound, first at {np.argwhere(bad)[0]}"
    err = O.rel_fro(got, ref)
    assert err <= 5e-3, err
    return err


CASES = [
    # M, heads, seq_len, window
    (64, 1, 64, 64),        # one block, plain causal
    (128, 2, 64, 1),        # window 1: O = V
    (200, 2, 100, 7),       # ragged sequences, query blocks straddle nothing
    (130, 1, 130, 64),      # window = block size, ragged tail
    (5, 2, 1, 1),           # one-token sequences
    (510, 2, 255, 3000),    # window beyond the sequence: causal
    (1024, 2, 512, 32768),  # the paper's window over 512-token pairs
    (1024, 2, 512, 100),    # window shorter than the sequence, not a block multiple
    (640, 2, 320, 65),      # window one past a block
    (63, 1, 63, 63),        # a single partial block
    (768, 3, 256, 129),
]


@pytest.mark.parametrize("M,heads,L,W", CASES)
def test_attention_parity(ql, M, heads, L, W):
    d = 128 * heads
    say(f"attention M={M} heads={heads} L={L} W={W}")
    qkv = synth.qkv_bf16(100 + M + W, M, d)
    out = ql.attention(dev_u16(qkv), heads, L, W)
    torch.cuda.synchronize()
    err = _check(host_u16(out), qkv, d, heads, L, W)
    say(f"  rel err {err:.3e}")


@pytest.mark.parametrize("std", [0.05, 6.0])
def test_attention_flat_and_peaked_scores(ql, std):
    """Nearly uniform weights (small scores) and nearly one-hot weights
    (scores of tens of units) over 512-token causal windows."""
    M, heads, L, W = 1024, 2, 512, 32768
    d = 128 * heads
    qkv = synth.qkv_bf16(7, M, d, std=std)
    out = ql.attention(dev_u16(qkv), heads, L, W)
    torch.cuda.synchronize()
    _check(host_u16(out), qkv, d, heads, L, W)


@pytest.mark.parametrize("M,heads,L,W", [(256, 2, 64, 1), (300, 1, 1, 5), (128, 3, 128, 1)])
def test_attention_single_key_is_v_bit_exact(ql, M, heads, L, W):
    """With one visible key (window 1, or one-token sequences) the weight is
    exactly 1 and the output is V, bit for bit."""
    d = 128 * heads
    qkv = synth.qkv_bf16(11, M, d)
    out = host_u16(ql.attention(dev_u16(qkv), heads, L, W))
    np.testing.assert_array_equal(out, qkv[:, 2 * d:3 * d])


def test_attention_strided_operands(ql):
    """qkv with a row stride beyond 3d and out written into a wider buffer:
    only out's first d columns change."""
    M, heads, L, W = 192, 2, 96, 40
    d = 128 * heads
    qkv = synth.qkv_bf16(12, M, d)
    wide = np.zeros((M, 3 * d + 64), dtype=np.uint16)
    wide[:, :3 * d] = qkv
    dq = dev_u16(wide)
    dout = torch.full((M, d + 128), 0x1234, dtype=torch.int16, device="cuda")
    ql.attention(dq, heads, L, W, out=dout)
    torch.cuda.synchronize()
    got = host_u16(dout)
    assert (got[:, d:] == 0x1234).all()
    _check(got[:, :d].copy(), qkv, d, heads, L, W)


def test_attention_full_size_sampled_heads(ql):
    """175B width: 8 pairs x 512 tokens, 96 heads, window 32768.  Six sampled
    (pair, head) blocks -- all 512 x 128 of their outputs -- against the
    oracle (heads and pairs are independent in its definition)."""
    M, heads, L, W = 4096, 96, 512, 32768
    d = 128 * heads
    say("attention full size")
    qkv = synth.qkv_bf16(synth.SEED_STACK, M, d)
    out = host_u16(ql.attention(dev_u16(qkv), heads, L, W))
    rng = np.random.default_rng(21)
    for _ in range(6):
        pair, hh = int(rng.integers(M // L)), int(rng.integers(heads))
        rows = slice(pair * L, pair * L + L)
        cols = np.concatenate([np.arange(hh * 128, hh * 128 + 128) + t * d for t in range(3)])
        sub = np.ascontiguousarray(qkv[rows][:, cols])
        got = out[rows, hh * 128:hh * 128 + 128].copy()
        err = _check(got, sub, 128, 1, L, W)
        say(f"  pair {pair} head {hh}: rel err {err:.3e}")


@pytest.mark.parametrize("L,W", [(32768, 32768), (16384, 5000)])
def test_attention_32k_window_sampled_rows(ql, L, W):
    """The paper's 32K window used in full: sequences of 32768 (or 16384)
    tokens, one head; 48 sampled query rows (first, last, window edges and
    random) against the oracle's row-sampled attention."""
    M, heads = 32768, 1
    d = 128 * heads
    say(f"attention long sequences L={L} W={W}")
    qkv = synth.qkv_bf16(31 + W, M, d, std=1.0)
    out = host_u16(ql.attention(dev_u16(qkv), heads, L, W))
    rng = np.random.default_rng(W)
    edges = [0, 1, W - 1, W, W + 1, L - 1, L, L + 1, L + W - 1, L + W, M - 1]
    rows = sorted(set([r for r in edges if 0 <= r < M] + [int(r) for r in rng.choice(M, 39, replace=False)]))
    ref = O.attention_rows_ref(qkv, d, heads, L, W, rows)
    got = bf16_as_f64(out[rows])
    vmax = np.abs(bf16_as_f64(qkv[:, 2 * d:])).max()
    bad = np.abs(got - ref) > TOL * (vmax + np.abs(ref))
    assert not bad.any(), f"rows {np.array(rows)[bad.any(axis=1)]}"
    assert O.rel_fro(got, ref) <= 5e-3


def test_attention_argument_errors(ql):
    qkv = torch.zeros((128, 3 * 256), dtype=torch.int16, device="cuda")
    with pytest.raises(ql.QLError) as e:
        ql.attention(qkv, 2, 100, 4)          # 128 % 100 != 0
    assert e.value.code == 1
    with pytest.raises(ql.QLError) as e:
        ql.attention(qkv, 2, 64, 0)           # window 0
    assert e.value.code == 1
    with pytest.raises(ql.QLError) as e:      # out inside qkv
        ql.attention(qkv, 2, 64, 4, out=qkv[:, :256])
    assert e.value.code == 1


# ---- ragged batches (pairs of different lengths, no padding) -----------------

def _cu(lengths):
    return torch.tensor(np.concatenate([[0], np.cumsum(lengths)]), dtype=torch.int32,
                        device="cuda")


@pytest.mark.parametrize("lengths,heads,W", [
    ([512, 300, 1, 129, 64, 450], 2, 32768),
    ([7, 130, 0, 255, 128, 3], 1, 100),       # an empty sequence, block-edge lengths
    ([1, 1, 1, 1], 3, 1),
    ([200], 2, 65),
])
def test_attention_varlen_parity(ql, lengths, heads, W):
    d = 128 * heads
    M = int(sum(lengths))
    say(f"attention varlen lengths={lengths} heads={heads} W={W}")
    qkv = synth.qkv_bf16(300 + M + W, M, d)
    out = ql.attention_varlen(dev_u16(qkv), heads, _cu(lengths), max(lengths), W)
    torch.cuda.synchronize()
    _check(host_u16(out), qkv, d, heads, [n for n in lengths if n], W)


def test_attention_varlen_uniform_matches_uniform_kernel(ql):
    """Equal lengths given as offsets run the same arithmetic: bit-equal."""
    M, heads, L, W = 1024, 2, 256, 300
    d = 128 * heads
    qkv = dev_u16(synth.qkv_bf16(13, M, d))
    a = ql.attention(qkv, heads, L, W)
    b = ql.attention_varlen(qkv, heads, _cu([L] * (M // L)), L, W)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_attention_varlen_full_width_sampled(ql):
    """175B width, 96 heads: a ragged batch of 9 pairs (380-450 residue plus
    40-62 ligand tokens each, packed without padding); five sampled (pair,
    head) blocks against the oracle."""
    heads, W = 96, 32768
    d = 128 * heads
    lengths = synth.pair_lengths(synth.SEED_STACK, 9)
    M = int(lengths.sum())
    say(f"attention varlen full width M={M}")
    qkv = synth.qkv_bf16(synth.SEED_STACK + 2, M, d)
    out = host_u16(ql.attention_varlen(dev_u16(qkv), heads, _cu(lengths), int(lengths.max()), W))
    starts = np.concatenate([[0], np.cumsum(lengths)])
    rng = np.random.default_rng(22)
    for _ in range(5):
        pr, hh = int(rng.integers(len(lengths))), int(rng.integers(heads))
        rows = slice(starts[pr], starts[pr + 1])
        cols = np.concatenate([np.arange(hh * 128, hh * 128 + 128) + t * d for t in range(3)])
        sub = np.ascontiguousarray(qkv[rows][:, cols])
        got = out[rows, hh * 128:hh * 128 + 128].copy()
        _check(got, sub, 128, 1, int(lengths[pr]), W)


# ---- the stack with attention -------------------------------------------

def _packed_layer_oracle(seed, layer, d, dff):
    mk = lambda i, n, k: O.quantize_pack(synth.weights_f32(synth.matrix_seed(seed, layer, i), n, k))
    return {"qkv": mk(0, 3 * d, d), "out": mk(1, d, d), "up": mk(2, dff, d), "down": mk(3, d, dff)}


def _to_dev(layer):
    return {k: (dev(q), dev_u16(s)) for k, (q, s) in layer.items()}


@pytest.mark.parametrize("M,L,W", [(8, 8, 3), (16, 4, 32768), (64, 64, 17), (200, 100, 32768),
                                   (256, 128, 64)])
def test_small_stack_with_attention(ql, M, L, W):
    """4 blocks at d = 256 (2 heads), d_ff = 1024, attention between the QKV
    and out projections; small-batch kernels for M <= 16, MFMA above."""
    d, dff, nl, heads = 256, 1024, 4, 2
    say(f"stack+attention M={M} L={L} W={W}")
    layers = [_packed_layer_oracle(50, l, d, dff) for l in range(nl)]
    h0 = synth.residual_f32(50 + M, M, d)
    ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
    h = dev(h0)
    ql.stack_forward(ql.make_layers([_to_dev(x) for x in layers]), h, dff, ws,
                     attn=(heads, L, W))
    torch.cuda.synchronize()
    ref = h0
    for x in layers:
        ref = O.stack_layer(ref, x, attn=(heads, L, W))
    err = O.rel_fro(h.cpu().numpy().astype(np.float64) - h0, ref.astype(np.float64) - h0)
    say(f"  end-to-end rel err of the residual update: {err:.3e}")
    assert err <= 5e-3


@pytest.mark.parametrize("M", [16, 192])
def test_stack_attention_window_one_equals_stand_in(ql, M):
    """Window 1 makes attention the identity on V, so the stack with
    attention matches the stand-in stack: bit for bit on the small-batch
    path (the out projection reads the same V values), and to fp32 rounding
    on the MFMA path (there the stand-in takes V's group sums from the QKV
    epilogue and the attention path from the operand-preparation kernel,
    which add in a different order)."""
    d, dff = 256, 1024
    layers = [_to_dev(_packed_layer_oracle(51, l, d, dff)) for l in range(2)]
    arr = ql.make_layers(layers)
    h0 = synth.residual_f32(51, M, d)
    ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
    a, b = dev(h0), dev(h0)
    ql.stack_forward(arr, a, dff, ws)
    ql.stack_forward(arr, b, dff, ws, attn=(2, 16, 1))
    torch.cuda.synchronize()
    if M <= 16:
        assert torch.equal(a, b)
    else:
        ua = a.cpu().numpy().astype(np.float64) - h0
        ub = b.cpu().numpy().astype(np.float64) - h0
        assert O.rel_fro(ub, ua) <= 1e-3


def test_full_width_block_with_attention_sampled_sequence(ql):
    """One 175B-width block (96 heads) with attention at M = 4096 tokens in
    sequences of 128: one sampled sequence -- every one of its tokens --
    against the oracle's block on that sequence alone (sequences never mix)."""
    d, dff, M, L, W = 12288, 49152, 4096, 128, 32768
    say("stack+attention full-width block")

    def mk(i, n, k):
        s = synth.matrix_seed(synth.SEED_STACK + 1, 0, i)
        return synth.random_packed_bytes(s, n, k), synth.random_scales_f16(s, n, k // 128)

    layer = {"qkv": mk(0, 3 * d, d), "out": mk(1, d, d), "up": mk(2, dff, d), "down": mk(3, d, dff)}
    h0 = synth.residual_f32(synth.SEED_STACK + 1, M, d)
    ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
    h = dev(h0)
    ql.stack_forward(ql.make_layers([_to_dev(layer)]), h, dff, ws, attn=(96, L, W))
    torch.cuda.synchronize()
    seq = 13
    rows = slice(seq * L, seq * L + L)
    got = h.cpu().numpy()[rows].astype(np.float64)
    say("  oracle on the sampled sequence")
    ref = O.stack_layer(h0[rows], layer, attn=(96, L, W)).astype(np.float64)
    err = O.rel_fro(got - h0[rows], ref - h0[rows])
    say(f"  rel err of the residual update: {err:.3e}")
    assert err <= 5e-3


@pytest.mark.parametrize("lengths", [[5, 3, 8], [40, 1, 77, 8], [130, 70, 120, 50]])
def test_small_stack_with_ragged_attention(ql, lengths):
    """4 blocks at d = 256 on a ragged batch (small-batch kernels for 16
    tokens, MFMA above): attention over each pair's own tokens only."""
    d, dff, nl, heads, W = 256, 1024, 4, 2, 32768
    M = sum(lengths)
    say(f"stack+ragged attention lengths={lengths}")
    layers = [_packed_layer_oracle(52, l, d, dff) for l in range(nl)]
    h0 = synth.residual_f32(52 + M, M, d)
    ws = torch.empty(ql.stack_workspace_bytes(M, d, dff), dtype=torch.uint8, device="cuda")
    h = dev(h0)
    ql.stack_forward(ql.make_layers([_to_dev(x) for x in layers]), h, dff, ws,
                     attn=(heads, _cu(lengths), max(lengths), W))
    torch.cuda.synchronize()
    ref = h0
    for x in layers:
        ref = O.stack_layer(ref, x, attn=(heads, lengths, W))
    err = O.rel_fro(h.cpu().numpy().astype(np.float64) - h0, ref.astype(np.float64) - h0)
    say(f"  end-to-end rel err of the residual update: {err:.3e}")
    assert err <= 5e-3
