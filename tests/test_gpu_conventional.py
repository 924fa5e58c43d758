"""The conventional PyTorch path that bench.py times beside this one
(``torch.cat`` cache growth, ``repeat_interleave`` GQA) computes the same
outputs as the oracle on the same inputs, so the comparison is like for
like."""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2607_19456_amd import workloads

pytestmark = pytest.mark.gpu

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


@pytest.mark.parametrize("G,steps", [(4, 3), (1, 2), (8, 0)])
def test_conventional_path_matches_the_oracle(cuda_device, G, steps):
    shape = workloads.custom(f"conv{G}", B=3, h_q=8, h_kv=8 // G, d_k=64, d_v=64, n_max=300,
                             len_lo=100, len_hi=250, steps=steps)
    inp = workloads.make(shape, seed=G, pad=0.0)
    outs = []
    res = bench.conventional_leg(shape, inp, cuda_device, 1.0, outputs=outs)
    hK, hV, hl = inp.K.copy(), inp.V.copy(), inp.lens.copy()
    n_out = len(outs) if steps else 1
    for t in range(n_out):
        if steps:
            oracle.append(hK, hV, inp.k_new[t], inp.v_new[t], hl)
            ref = oracle.decode(inp.q_step[t], hK, hV, hl, shape.scale32())
        else:
            ref = oracle.decode(inp.q, hK, hV, hl, shape.scale32())
        for o in (outs[t:t + 1] if steps else outs):
            assert np.max(np.abs(o - ref)) <= 1e-5, t
    assert res["final_len"] == hl.tolist()
