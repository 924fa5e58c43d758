"""The no-allocation decode (da_decode_attn_noalloc, the library's static
64 MiB workspace) against da_decode_attn with a caller workspace: two calls
in a row, the second with smaller shapes (so its counter region overlaps
what the first call left in the array), each compared with da_decode_attn's
output and with the oracle at 1e-5; then shapes too large for the array are
rejected.  Called through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_19456_amd import binding, workloads

pytestmark = pytest.mark.gpu

TOL = 1e-5


def say(msg):
    print(msg, flush=True)


def dev(a, device):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


CALLS = [
    # name, B, h_q, h_kv, d, n_max, lengths (several segments per slab: the
    # partial + merge path), then a smaller problem
    ("large", 4, 32, 8, 128, 20000, [20000, 13001, 7777, 1]),
    ("smaller", 2, 8, 2, 64, 3000, [2999, 1500]),
]


def test_noalloc_matches_decode_attn_on_consecutive_calls(cuda_device):
    for name, B, h_q, h_kv, d, n_max, lens in CALLS:
        shape = workloads.custom(name, B=B, h_q=h_q, h_kv=h_kv, d_k=d, d_v=d, n_max=n_max)
        inp = workloads.make(shape, seed=41, lens=np.array(lens, np.int32))
        dq, dK, dV, dl = (dev(a, cuda_device) for a in (inp.q, inp.K, inp.V, inp.lens))
        scale = float(shape.scale32())
        say(f"no-alloc decode, {name}: B={B} h_q={h_q} h_kv={h_kv} d={d} lens={lens}")
        assert binding.workspace_bytes(B, h_q, h_kv, n_max, d, d) <= \
            binding.NOALLOC_MAX_WORKSPACE_BYTES
        out_na = torch.full((B, h_q, d), float("nan"), device=cuda_device)
        binding.decode_attn_noalloc(dq, dK, dV, dl, scale, out_na)
        out_ws = binding.decode_attn(dq, dK, dV, dl, scale)
        torch.cuda.synchronize()
        got_na = out_na.cpu().numpy().astype(np.float64)
        got_ws = out_ws.cpu().numpy().astype(np.float64)
        ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
        for what, got in (("no-alloc", got_na), ("workspace", got_ws)):
            assert np.all(np.isfinite(got)), what
            err = float(np.max(np.abs(got - ref)))
            say(f"  {name} {what} vs oracle: max-abs-err {err:.3e}")
            assert err <= TOL
        diff = float(np.max(np.abs(got_na - got_ws)))
        say(f"  {name} no-alloc vs da_decode_attn: max-abs-diff {diff:.3e}")
        assert diff <= TOL


def test_noalloc_rejects_shapes_beyond_its_array(cuda_device):
    """B=128, 32/8 heads, n_max=32768 needs more than 64 MiB of workspace:
    rejected on the host before anything is enqueued (the pointers are
    never dereferenced)."""
    assert binding.workspace_bytes(128, 32, 8, 32768, 128, 128) > \
        binding.NOALLOC_MAX_WORKSPACE_BYTES
    p = torch.zeros(16, device=cuda_device).data_ptr()
    st = binding._lib.da_decode_attn_noalloc(p, p, p, p, 0.1, p, 128, 32, 8, 32768, 128, 128,
                                             None)
    assert st == 6
