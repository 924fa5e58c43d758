"""Seeded random shapes through the C ABI against the CPU oracle.

Every combination the planner distinguishes -- one or two MFMA column
blocks, several head groups, d_k != d_v, head sizes 64/128/256, the direct
form (single-chunk caches), the 14/16 static share with dynamic units
(forced where the planner would make a small cache wholly static: the
``schedule`` fixture runs every case both ways), whole-slab ranges (many
slabs), large batches scheduled dynamically only,
empty and full caches -- is drawn from one fixed seed, so a failure names a
reproducible case.  Decode: max-abs-err <= 1e-5 with the cache rows beyond
len[b] poisoned with NaN; the fused step (append + decode) also checks the
cache, bit for bit, and the advanced lengths.
"""
import random

import numpy as np
import pytest
import torch

import oracle
from paper_2607_19456_amd import binding, workloads

pytestmark = pytest.mark.gpu

TOL = 1e-5
GROUPS = [1, 2, 3, 4, 5, 8, 12, 16, 17, 20, 24, 32, 33, 40, 64]
HEAD_DIMS = [64, 64, 128, 128, 128, 256]


def _cases(n, seed):
    rng = random.Random(seed)
    out = []
    while len(out) < n:
        h_kv = rng.choice([1, 1, 2, 3, 4, 8])
        G = rng.choice(GROUPS)
        d_k, d_v = rng.choice(HEAD_DIMS), rng.choice(HEAD_DIMS)
        B = rng.choice([1, 2, 3, 5, 8, 16, 40, 64, 300])
        n_max = rng.choice([1, 17, 100, 500, 768, 769, 1200, 2600])
        # keep the oracle's work (B * h_q * n * (d_k + d_v) products) small
        if B * h_kv * G * n_max * (d_k + d_v) > 1.5e8:
            continue
        if B * h_kv * n_max * (d_k + d_v) * 4 > 256e6:
            continue
        lens = [rng.randint(0, n_max) for _ in range(B)]
        if B > 1:
            lens[0] = n_max
        chunk = rng.choice([0, 0, 768, 1536])
        out.append((f"r{len(out)}_B{B}_hkv{h_kv}_G{G}_dk{d_k}_dv{d_v}_n{n_max}_c{chunk}",
                    B, h_kv * G, h_kv, d_k, d_v, n_max, lens, chunk))
    return out


DECODE_CASES = _cases(36, 20261) + [
    # the two many-slab regimes, drawn rarely above: whole-slab ranges (two
    # or more slabs per workgroup) and, beyond 256 sequences, dynamic units only
    ("fixed_whole_slab_B64_hkv8_G2_n1100", 64, 16, 8, 64, 64, 1100,
     [(37 * b) % 1101 for b in range(64)], 0),
    ("fixed_dynamic_only_B300_hkv2_G1_n1600", 300, 2, 2, 64, 64, 1600,
     [(53 * b) % 1601 for b in range(300)], 0),
]
STEP_CASES = _cases(12, 771)


def _long_cases(n, seed):
    """Short batches of long slabs: the wholly static plans at one or two
    workgroups per CU, and (under the fixture's dynamic mode) dynamic units
    on slabs longer than the two-wave form's 4608 rows."""
    rng = random.Random(seed)
    out = []
    while len(out) < n:
        h_kv = rng.choice([1, 2, 4, 8])
        G = rng.choice([1, 2, 4, 8, 16, 20, 32])
        d_k, d_v = rng.choice(HEAD_DIMS), rng.choice(HEAD_DIMS)
        B = rng.choice([1, 2, 3, 4, 6])
        n_max = rng.choice([4609, 6000, 9000, 16384, 25000])
        if B * h_kv * G * n_max * (d_k + d_v) > 1.2e8:
            continue
        lens = [rng.randint(0, n_max) for _ in range(B)]
        lens[0] = n_max
        out.append((f"long{len(out)}_B{B}_hkv{h_kv}_G{G}_dk{d_k}_dv{d_v}_n{n_max}",
                    B, h_kv * G, h_kv, d_k, d_v, n_max, lens, 0))
    return out


DECODE_CASES += _long_cases(10, 4099)
STEP_CASES += _long_cases(4, 4117)


def say(msg):
    print(msg, flush=True)


def dev(a, device):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def poisoned_workspace(dq, dK, dV, chunk_rows):
    ws = binding.alloc_workspace(dq, dK, dV, chunk_rows)
    ws.fill_(0xFF)
    B, h_q, d_k = dq.shape
    _, h_kv, n_max, _ = dK.shape
    ws[:binding.workspace_counter_bytes(B, h_q, h_kv, n_max, d_k, dV.shape[3])].zero_()
    return ws


def check(got, ref, what):
    assert got.shape == ref.shape
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = float(np.max(np.abs(got - ref))) if got.size else 0.0
    say(f"  {what}: max-abs-err {err:.3e}")
    assert err <= TOL, f"{what}: max-abs-err {err:.3e} > {TOL}"


def _inputs(case, steps=0):
    name, B, h_q, h_kv, d_k, d_v, n_max, lens, chunk = case
    shape = workloads.custom(name, B=B, h_q=h_q, h_kv=h_kv, d_k=d_k, d_v=d_v,
                             n_max=n_max, steps=steps)
    seed = sum(ord(c) for c in name) % 997
    return shape, workloads.make(shape, seed=seed, lens=np.array(lens, np.int32)), chunk


@pytest.mark.parametrize("case", DECODE_CASES, ids=[c[0] for c in DECODE_CASES])
def test_random_shape_decode(cuda_device, schedule, case):
    shape, inp, chunk = _inputs(case)
    say(f"decode {case[0]} lens={inp.lens.tolist()[:8]}")
    dq, dK, dV = dev(inp.q, cuda_device), dev(inp.K, cuda_device), dev(inp.V, cuda_device)
    ws = poisoned_workspace(dq, dK, dV, chunk)
    out = binding.decode_attn(dq, dK, dV, dev(inp.lens, cuda_device), float(shape.scale32()),
                              workspace=ws, chunk_rows=chunk)
    torch.cuda.synchronize()
    nc = binding.workspace_counter_bytes(*dq.shape[:2], dK.shape[1], dK.shape[2],
                                         dq.shape[2], dV.shape[3])
    assert not ws[:nc].any(), "counters not reset by the merge"
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    check(out.cpu().numpy().astype(np.float64), ref, case[0])


@pytest.mark.parametrize("case", STEP_CASES, ids=[c[0] for c in STEP_CASES])
def test_random_shape_fused_step(cuda_device, schedule, case):
    shape, inp, chunk = _inputs(case, steps=2)
    dK, dV, dl = dev(inp.K, cuda_device), dev(inp.V, cuda_device), dev(inp.lens, cuda_device)
    hK, hV, hl = inp.K.copy(), inp.V.copy(), inp.lens.copy()
    ws = poisoned_workspace(dev(inp.q, cuda_device), dK, dV, chunk)
    for t in range(shape.steps):
        say(f"step {case[0]} t={t}")
        out = binding.decode_step(dev(inp.q_step[t], cuda_device), dK, dV,
                                  dev(inp.k_new[t], cuda_device), dev(inp.v_new[t], cuda_device),
                                  dl, float(shape.scale32()), workspace=ws, chunk_rows=chunk)
        torch.cuda.synchronize()
        oracle.append(hK, hV, inp.k_new[t], inp.v_new[t], hl)
        ref = oracle.decode(inp.q_step[t], hK, hV, hl, shape.scale32())
        assert dl.cpu().numpy().tolist() == hl.tolist()
        assert np.array_equal(dK.cpu().numpy().view(np.uint32), hK.view(np.uint32))
        assert np.array_equal(dV.cpu().numpy().view(np.uint32), hV.view(np.uint32))
        check(out.cpu().numpy().astype(np.float64), ref, f"{case[0]} t={t}")
