"""CPU check of the attention kernel's LDS layouts (host logic, no GPU).

The index functions of csrc/ql_attn.hip are restated here: the K swizzle
(chunk ^ k_msk(key)), the V swizzle (chunk ^ 2 (key mod 8)), the slot each
direct-to-LDS copy fills, and the transposing LDS read (ds_read_b64_tr_b16),
whose lane mapping on gfx950 was measured on the device: within each group of
16 lanes, lane 4a + b receives element b of the 8-byte pieces addressed by
lanes a, a + 4, a + 8, a + 12.  The tests check that every lane then holds
exactly the operand elements the 16x16x32 MFMA layout needs (S^T = K Q^T with
K as the row operand; O^T += V^T P^T with key 32 t + 16 f + 4 h + j as element
4 f + j), that the copies cover the tile once, and that every access stays
inside its 16 KB stage and is free of bank conflicts per half-wave."""
import numpy as np
import pytest

WAVES = 8          # waves per workgroup
SLOTS = 64 * 16    # 16-byte slots per 64-key stage


def k_msk(r):
    r &= 15
    return r ^ ((((r >> 2) ^ (r >> 3)) & 1) << 2)


def v_swz(r):
    return (r & 7) << 1


def stage_contents(swz):
    """slot -> (key, chunk) after the copies of one stage."""
    tile = {}
    copies = SLOTS // 64 // WAVES
    for wave in range(WAVES):
        for i in range(copies):
            for lane in range(64):
                slot = (i * WAVES + wave) * 64 + lane
                key, ps = slot >> 4, slot & 15
                assert slot not in tile
                tile[slot] = (key, ps ^ swz(key))
    return tile


def test_copies_cover_each_tile_once():
    for swz in (k_msk, v_swz):
        tile = stage_contents(swz)
        assert len(tile) == SLOTS
        assert sorted(tile.values()) == [(k, c) for k in range(64) for c in range(16)]


def test_k_operand_reads():
    tile = stage_contents(k_msk)
    for lane in range(64):
        h, lr = lane >> 4, lane & 15
        for kf in range(4):
            key = kf * 16 + lr
            for s in range(4):
                assert tile[key * 16 + ((h * 4 + s) ^ k_msk(key))] == (key, h * 4 + s)


def _vt_byte(df, t2, f, h, lr):
    key = 32 * t2 + 16 * f + 4 * h + (lr >> 2)
    chunk = 2 * df + ((lr >> 1) & 1)
    return key * 256 + ((chunk ^ v_swz(key)) << 4) + ((lr & 1) << 3)


@pytest.mark.parametrize("df", range(8))
def test_v_transposed_operand(df):
    tile = stage_contents(v_swz)

    def element(byte):
        key, chunk = tile[byte // 16]
        return key, chunk * 8 + (byte % 16) // 2

    for t2 in range(2):
        for f in range(2):
            addr = [_vt_byte(df, t2, f, lane >> 4, lane & 15) for lane in range(64)]
            assert max(addr) + 8 <= SLOTS * 16
            # the constant (t2, f) part is an immediate offset of the read
            assert all(addr[l] - _vt_byte(df, 0, 0, l >> 4, l & 15) == (32 * t2 + 16 * f) * 256
                       for l in range(64))
            for half in range(2):
                pairs = [(addr[l] // 8) % 32 for l in range(half * 32, half * 32 + 32)]
                assert len(set(pairs)) == 32, "bank conflict in a transposing read"
            for lane in range(64):
                g, i = lane >> 4, lane & 15
                a, b = i >> 2, i & 3
                for j in range(4):
                    got = element(addr[g * 16 + a + 4 * j] + 2 * b)
                    h, lr = g, i
                    assert got == (32 * t2 + 16 * f + 4 * h + j, 16 * df + lr)
