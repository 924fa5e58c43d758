"""Parity of the multi-row (causal) decode, the fused multi-row step and the
T-row append on the GPU (through the C ABI) with the CPU oracle.

Decode: max-abs-err <= 1e-5 against the fp64 oracle on seeded N(0,1) inputs,
cache rows at or beyond len[b] poisoned with NaN; rows with no visible key
must be exactly zero.  Appends: bit-exact.
"""
import zlib

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


def rand(seed, shape):
    from paper_2607_19456_amd.workloads import normal
    return normal(seed, 77, shape)


def poisoned_multi_workspace(dq, dK, dV, chunk_rows=0):
    ws = binding.alloc_multi_workspace(dq, dK, dV, chunk_rows)
    ws.fill_(0xFF)
    B, h_q, T, d_k = dq.shape
    _, h_kv, n_max, _ = dK.shape
    nc = binding.workspace_counter_bytes(B, h_q * T, h_kv, n_max, d_k, dV.shape[3])
    ws[:nc].zero_()
    return ws, nc


def check(got, ref, what):
    assert got.shape == ref.shape
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = float(np.max(np.abs(got - ref))) if got.size else 0.0
    say(f"  {what}: max-abs-err {err:.3e}")
    assert err <= TOL, f"{what}: max-abs-err {err:.3e} > {TOL}"


MULTI = [
    # name, B, h_q, h_kv, d_k, d_v, n_max, T, lens
    ("gqa8_T4", 2, 16, 2, 128, 128, 900, 4, [900, 37]),
    ("mha_d64_T2", 2, 4, 4, 64, 64, 300, 2, [300, 1]),
    ("mqa32_T3_headgroups", 2, 32, 1, 128, 128, 513, 3, [513, 2]),
    ("dk64_dv128_T8", 2, 8, 2, 64, 128, 400, 8, [400, 5]),
    ("T16_two_groups", 1, 4, 1, 128, 128, 1000, 16, [1000]),
    ("dk128_dv64_T5_odd", 3, 6, 3, 128, 64, 97, 5, [97, 4, 60]),
    ("empty_and_short", 2, 8, 4, 128, 128, 70, 4, [0, 3]),
    ("d256_T4", 2, 8, 2, 256, 256, 600, 4, [600, 2]),
]


@pytest.mark.parametrize("case", MULTI, ids=[c[0] for c in MULTI])
@pytest.mark.parametrize("chunk_rows", [0, 768])
def test_decode_multi(cuda_device, case, chunk_rows):
    name, B, h_q, h_kv, d_k, d_v, n_max, T, lens = case
    shape = workloads.custom(name, B=B, h_q=h_q, h_kv=h_kv, d_k=d_k, d_v=d_v, n_max=n_max)
    seed = zlib.crc32(name.encode()) % 1000
    inp = workloads.make(shape, seed=seed, lens=np.array(lens, np.int32))
    q = rand(seed, (B, h_q, T, d_k))
    say(f"decode_multi {name} T={T} chunk_rows={chunk_rows} lens={lens}")
    dq, dK, dV = dev(q, cuda_device), dev(inp.K, cuda_device), dev(inp.V, cuda_device)
    dl = dev(inp.lens, cuda_device)
    ws, nc = poisoned_multi_workspace(dq, dK, dV, chunk_rows)
    out = binding.decode_multi(dq, dK, dV, dl, float(shape.scale32()), workspace=ws,
                               chunk_rows=chunk_rows)
    torch.cuda.synchronize()
    assert not ws[:nc].any(), "counters not reset by the merge"
    got = out.cpu().numpy().astype(np.float64)
    ref = oracle.decode_multi(q, inp.K, inp.V, inp.lens, shape.scale32())
    check(got, ref, name)
    for b, n in enumerate(lens):
        for r in range(T):
            if n - T + r < 0:
                assert not got[b, :, r].any(), (b, r)


STEPS = [
    # name, B, h_q, h_kv, d_k, d_v, n_max, T, lens
    ("gqa8_T4", 3, 16, 2, 128, 128, 700, 4, [0, 333, 698]),     # empty, middle, clipped
    ("mha_d64_T2_full", 2, 4, 4, 64, 64, 300, 2, [299, 300]),   # one row fits / none
    ("mqa_T3_dkdv", 2, 32, 1, 64, 128, 200, 3, [5, 190]),
    ("neg_len_T6", 2, 8, 4, 128, 128, 100, 6, [-3, 40]),
    # one launch per step (single-segment slabs, G*T <= 16), near capacity
    ("one_launch_T3", 9, 8, 2, 128, 128, 150, 3, [0, 149, 150, -1, 75, 147, 148, 10, 3]),
    # 1024 slabs: whole-slab ranges at two workgroups per CU, causal rows
    ("two_wave_T2", 128, 8, 8, 64, 64, 900, 2, [0, 1, 898, 899, 900, 450, 3, 777] * 16),
]


@pytest.mark.parametrize("case", STEPS, ids=[c[0] for c in STEPS])
def test_decode_multi_step_equals_sequential_steps(cuda_device, case):
    name, B, h_q, h_kv, d_k, d_v, n_max, T, lens = case
    shape = workloads.custom(name, B=B, h_q=h_q, h_kv=h_kv, d_k=d_k, d_v=d_v, n_max=n_max)
    seed = zlib.crc32(name.encode()) % 1000
    inp = workloads.make(shape, seed=seed, lens=np.array(lens, np.int32))
    dK, dV, dl = dev(inp.K, cuda_device), dev(inp.V, cuda_device), dev(inp.lens, cuda_device)
    hK, hV, hl = inp.K.copy(), inp.V.copy(), inp.lens.copy()
    ws = None
    for step in range(2):
        q = rand(seed + 10 * step, (B, h_q, T, d_k))
        kn = rand(seed + 10 * step + 1, (B, h_kv, T, d_k))
        vn = rand(seed + 10 * step + 2, (B, h_kv, T, d_v))
        dq = dev(q, cuda_device)
        if ws is None:
            ws, nc = poisoned_multi_workspace(dq, dK, dV)
        say(f"multi step {name} step {step} len={hl.tolist()}")
        out = binding.decode_multi_step(dq, dK, dV, dev(kn, cuda_device), dev(vn, cuda_device),
                                        dl, float(shape.scale32()), workspace=ws)
        torch.cuda.synchronize()
        # the definition: T single steps (append one row, decode its query)
        ref = np.zeros((B, h_q, T, d_v))
        for r in range(T):
            oracle.append(hK, hV, np.ascontiguousarray(kn[:, :, r]),
                          np.ascontiguousarray(vn[:, :, r]), hl)
            ref[:, :, r] = oracle.decode(np.ascontiguousarray(q[:, :, r]), hK, hV, hl,
                                         shape.scale32())
        assert dl.cpu().numpy().tolist() == hl.tolist()
        assert np.array_equal(dK.cpu().numpy().view(np.uint32), hK.view(np.uint32))
        assert np.array_equal(dV.cpu().numpy().view(np.uint32), hV.view(np.uint32))
        assert not ws[:nc].any()
        check(out.cpu().numpy().astype(np.float64), ref, f"{name} step {step}")


@pytest.mark.parametrize("T", [1, 3, 8])
def test_append_rows_bit_exact(cuda_device, T):
    B, h_kv, n_max, d_k, d_v = 4, 3, 12, 8, 12
    rng = np.random.default_rng(T)
    K = rng.standard_normal((B, h_kv, n_max, d_k)).astype(np.float32)
    V = rng.standard_normal((B, h_kv, n_max, d_v)).astype(np.float32)
    lens = np.array([0, 5, 11, -2], np.int32)
    dK, dV, dl = dev(K, cuda_device), dev(V, cuda_device), dev(lens, cuda_device)
    for step in range(3):
        kn = rng.standard_normal((B, h_kv, T, d_k)).astype(np.float32)
        vn = rng.standard_normal((B, h_kv, T, d_v)).astype(np.float32)
        kn.view(np.uint32)[0, 0, 0, :3] = [0x7FC01234, 0x80000000, 0x00000001]
        say(f"append_rows T={T} step {step}")
        binding.kv_append_rows(dK, dV, dev(kn, cuda_device), dev(vn, cuda_device), dl)
        oracle.append_rows(K, V, kn, vn, lens)
        torch.cuda.synchronize()
        assert np.array_equal(dl.cpu().numpy(), lens)
        assert np.array_equal(dK.cpu().numpy().view(np.uint32), K.view(np.uint32))
        assert np.array_equal(dV.cpu().numpy().view(np.uint32), V.view(np.uint32))


def test_multi_row_long_context(cuda_device):
    """The 4-row speculative workload through the fused path: all 16 steps,
    every head and query row against the oracle (the host mirror replays
    the appends; row r of a step is the single step r, so it attends
    len + r + 1 rows)."""
    shape = workloads.get("spec4")
    say("multi-row long context: generating inputs")
    inp = workloads.make(shape, seed=4)
    dK, dV, dl = dev(inp.K, cuda_device), dev(inp.V, cuda_device), dev(inp.lens, cuda_device)
    hK, hV, hl = inp.K, inp.V, inp.lens.copy()
    ws = binding.alloc_multi_workspace(dev(inp.q_step[0], cuda_device), dK, dV)
    T = shape.rows
    for t in range(shape.steps):
        out = binding.decode_multi_step(dev(inp.q_step[t], cuda_device), dK, dV,
                                        dev(inp.k_new[t], cuda_device),
                                        dev(inp.v_new[t], cuda_device), dl,
                                        float(shape.scale32()), workspace=ws)
        len0 = hl.copy()
        oracle.append_rows(hK, hV, inp.k_new[t], inp.v_new[t], hl)
        torch.cuda.synchronize()
        got = out.cpu().numpy().astype(np.float64)
        for r in range(T):
            lens_r = np.minimum(len0 + r + 1, shape.n_max).astype(np.int32)
            ref = oracle.decode(np.ascontiguousarray(inp.q_step[t][:, :, r]), hK, hV, lens_r,
                                shape.scale32())
            check(got[:, :, r], ref, f"spec4 step {t} row {r}")
        assert dl.cpu().numpy().tolist() == hl.tolist()


@pytest.mark.parametrize("lens,agree", [([96, 40], True), ([98, 100], False)],
                         ids=["room_for_every_row", "near_capacity"])
def test_multi_step_and_append_then_multi_near_capacity(cuda_device, lens, agree):
    """da_decode_multi_step (T single steps) and da_kv_append_rows followed by
    da_decode_multi each match their own definition on the GPU, also when the
    cache fills up during the step; the two coincide exactly while every row
    fits (len + T <= n_max) and differ, as documented, once it does not."""
    B, h_q, h_kv, n_max, d, T = 2, 8, 2, 100, 64, 4
    shape = workloads.custom("near_cap", B=B, h_q=h_q, h_kv=h_kv, d_k=d, d_v=d, n_max=n_max)
    inp = workloads.make(shape, seed=23, lens=np.array(lens, np.int32))
    q = rand(70, (B, h_q, T, d))
    kn, vn = rand(71, (B, h_kv, T, d)), rand(72, (B, h_kv, T, d))
    scale = float(shape.scale32())
    # fused: T single steps
    dK, dV, dl = dev(inp.K, cuda_device), dev(inp.V, cuda_device), dev(inp.lens, cuda_device)
    fused = binding.decode_multi_step(dev(q, cuda_device), dK, dV, dev(kn, cuda_device),
                                      dev(vn, cuda_device), dl, scale)
    # append T rows, then the multi-row decode over the cache's last T positions
    dK2, dV2, dl2 = dev(inp.K, cuda_device), dev(inp.V, cuda_device), dev(inp.lens, cuda_device)
    binding.kv_append_rows(dK2, dV2, dev(kn, cuda_device), dev(vn, cuda_device), dl2)
    chunked = binding.decode_multi(dev(q, cuda_device), dK2, dV2, dl2, scale)
    torch.cuda.synchronize()
    hK, hV, hl = inp.K.copy(), inp.V.copy(), inp.lens.copy()
    oracle.append_rows(hK, hV, kn, vn, hl)
    ref_chunked = oracle.decode_multi(q, hK, hV, hl, scale)
    ref_fused = np.zeros_like(ref_chunked)
    for r in range(T):
        lr = np.minimum(inp.lens + r + 1, n_max).astype(np.int32)
        ref_fused[:, :, r] = oracle.decode(np.ascontiguousarray(q[:, :, r]), hK, hV, lr, scale)
    assert dl.cpu().numpy().tolist() == dl2.cpu().numpy().tolist() == hl.tolist()
    got_f = fused.cpu().numpy().astype(np.float64)
    got_c = chunked.cpu().numpy().astype(np.float64)
    check(got_f, ref_fused, "multi_step")
    check(got_c, ref_chunked, "append_rows + decode_multi")
    assert np.array_equal(ref_fused, ref_chunked) == agree
    if agree:
        assert np.max(np.abs(got_f - got_c)) <= 2 * TOL


def test_graph_replay_of_multi_row_steps(cuda_device):
    """Two multi-row steps captured in one HIP graph, replayed three times
    from the same initial cache with eager work in between."""
    B, h_q, h_kv, n_max, d, T = 2, 16, 2, 600, 128, 4
    shape = workloads.custom("graph_multi", B=B, h_q=h_q, h_kv=h_kv, d_k=d, d_v=d, n_max=n_max)
    inp = workloads.make(shape, seed=31, lens=np.array([0, 597], np.int32))
    dK0, dV0, dl0 = dev(inp.K, cuda_device), dev(inp.V, cuda_device), dev(inp.lens, cuda_device)
    dK, dV, dl = dK0.clone(), dV0.clone(), dl0.clone()
    qs = [rand(40 + t, (B, h_q, T, d)) for t in range(2)]
    kns = [rand(50 + t, (B, h_kv, T, d)) for t in range(2)]
    vns = [rand(60 + t, (B, h_kv, T, d)) for t in range(2)]
    dq = [dev(x, cuda_device) for x in qs]
    dkn = [dev(x, cuda_device) for x in kns]
    dvn = [dev(x, cuda_device) for x in vns]
    ws = binding.alloc_multi_workspace(dq[0], dK, dV)
    outs = [torch.empty((B, h_q, T, d), device=cuda_device) for _ in range(2)]
    scale = float(shape.scale32())
    # the definition: single steps on the host mirror
    hK, hV, hl = inp.K.copy(), inp.V.copy(), inp.lens.copy()
    refs = []
    for t in range(2):
        ref = np.zeros((B, h_q, T, d))
        for r in range(T):
            oracle.append(hK, hV, np.ascontiguousarray(kns[t][:, :, r]),
                          np.ascontiguousarray(vns[t][:, :, r]), hl)
            ref[:, :, r] = oracle.decode(np.ascontiguousarray(qs[t][:, :, r]), hK, hV, hl,
                                         shape.scale32())
        refs.append(ref)
    for t in range(2):   # eager pass first (loads the kernels)
        binding.decode_multi_step(dq[t], dK, dV, dkn[t], dvn[t], dl, scale, out=outs[t],
                                  workspace=ws)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for t in range(2):
            binding.decode_multi_step(dq[t], dK, dV, dkn[t], dvn[t], dl, scale, out=outs[t],
                                      workspace=ws)
    for rep in range(3):
        dK.copy_(dK0)
        dV.copy_(dV0)
        dl.copy_(dl0)
        for o in outs:
            o.fill_(float("nan"))
        torch.cuda.synchronize()
        say(f"multi-row graph replay {rep}")
        graph.replay()
        torch.cuda.synchronize()
        for t in range(2):
            check(outs[t].cpu().numpy().astype(np.float64), refs[t], f"replay {rep} step {t}")
        assert dl.cpu().numpy().tolist() == hl.tolist()
        assert np.array_equal(dK.cpu().numpy().view(np.uint32), hK.view(np.uint32))
