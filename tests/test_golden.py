"""Hand-worked quantization groups (tests/golden/quant_hand_worked.json)
against the oracle (CPU) and the GPU packer.  The expected scales, codes
and bytes were derived by hand from the scheme's definition; the
derivation of each is stored beside it."""
import json
import os

import numpy as np
import pytest

import oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))
FIX = json.load(open(os.path.join(HERE, "golden", "quant_hand_worked.json")))


def _weights():
    g = FIX["group"]
    w = np.zeros((len(FIX["groups"]), g), dtype=np.float32)
    for i, grp in enumerate(FIX["groups"]):
        w[i, :len(grp["w_head"])] = np.array(grp["w_head"], dtype=np.float32)
    return w


def _check(qw, sc):
    for i, grp in enumerate(FIX["groups"]):
        assert int(sc[i, 0]) == grp["scale_bits"], grp["name"]
        nb = len(grp["bytes_head"])
        assert list(qw[i, :nb]) == grp["bytes_head"], grp["name"]
        assert not qw[i, nb:].any(), grp["name"]
        q = O.unpack_codes(qw[i:i + 1])[0]
        assert list(q[:len(grp["codes_head"])]) == grp["codes_head"], grp["name"]


def test_oracle_matches_hand_worked_groups():
    qw, sc = O.quantize_pack(_weights())
    _check(qw, sc)


@pytest.mark.gpu
def test_gpu_pack_matches_hand_worked_groups():
    import torch

    import paper_2608_30877_amd as ql

    qw, sc = ql.pack(torch.from_numpy(_weights()).cuda())
    torch.cuda.synchronize()
    _check(qw.cpu().numpy(), sc.cpu().numpy().view(np.uint16))
