"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Decode: max-abs-err <= 1e-5 against the fp64 oracle on the same seeded
N(0,1) inputs, with every cache row at or beyond len[b] poisoned with NaN.
Append: bit-exact against the oracle's host mirror.
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


def poisoned_workspace(dq, dK, dV, chunk_rows=0):
    """Workspace whose partial slots hold NaN bit patterns (a decode must
    never read a slot it did not write) and whose counters are zero."""
    ws = binding.alloc_workspace(dq, dK, dV, chunk_rows)
    ws.fill_(0xFF)
    B, h_q, d_k = dq.shape
    _, h_kv, n_max, _ = dK.shape
    ws[:binding.workspace_counter_bytes(B, h_q, h_kv, n_max, d_k, dV.shape[3])].zero_()
    return ws


def run_decode(inp, device, q=None, lens=None, chunk_rows=0, K=None, V=None):
    s = inp.shape
    q = inp.q if q is None else q
    lens = inp.lens if lens is None else lens
    dK = dev(inp.K, device) if K is None else K
    dV = dev(inp.V, device) if V is None else V
    dq, dl = dev(q, device), dev(lens, device)
    ws = poisoned_workspace(dq, dK, dV, chunk_rows)
    out = binding.decode_attn(dq, dK, dV, dl, float(s.scale32()), workspace=ws,
                              chunk_rows=chunk_rows)
    torch.cuda.synchronize()
    # a completed decode leaves the counters zero for the next call
    nc = binding.workspace_counter_bytes(*dq.shape[:2], dK.shape[1], dK.shape[2],
                                         dq.shape[2], dV.shape[3])
    assert not ws[:nc].any(), "counters not reset by the merge"
    return out.cpu().numpy().astype(np.float64)


def check(got, ref, what):
    assert got.shape == ref.shape
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = float(np.max(np.abs(got - ref))) if got.size else 0.0
    say(f"  {what}: max-abs-err {err:.3e}")
    assert err <= TOL, f"{what}: max-abs-err {err:.3e} > {TOL}"


# --- decode on small shapes: several tiles, ragged tails, every group size --

SMALL = [
    # name, B, h_q, h_kv, d_k, d_v, n_max, lens
    ("mha_d64", 2, 4, 4, 64, 64, 300, [300, 1]),
    ("mha_d128_tail", 3, 2, 2, 128, 128, 1000, [17, 999, 64]),
    ("gqa4", 2, 16, 4, 128, 128, 777, [777, 130]),
    ("gqa8", 2, 16, 2, 128, 128, 2050, [2050, 1025]),
    ("gqa16", 1, 16, 1, 128, 128, 333, [333]),
    ("gqa20_twoblocks", 2, 40, 2, 128, 128, 200, [200, 63]),
    ("mqa32", 2, 32, 1, 128, 128, 513, [513, 16]),
    ("gqa64_headgroups", 1, 64, 1, 128, 128, 150, [150]),
    ("dk64_dv128", 2, 8, 2, 64, 128, 400, [400, 65]),
    ("dk128_dv64", 2, 8, 4, 128, 64, 400, [15, 400]),
    ("g3_odd", 2, 9, 3, 64, 64, 97, [97, 2]),
    ("empty_and_full", 3, 8, 8, 128, 128, 70, [0, 70, 1]),
    ("d256", 2, 8, 2, 256, 256, 900, [900, 33]),
    ("d256_mqa_twoblocks", 1, 32, 1, 256, 256, 500, [500]),
    ("dk256_dv64", 2, 4, 2, 256, 64, 300, [1, 300]),
    ("dk64_dv256_g20", 2, 40, 2, 64, 256, 200, [200, 17]),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
@pytest.mark.parametrize("chunk_rows", [0, 768, 1536])
def test_decode_small_shapes(cuda_device, case, chunk_rows):
    name, B, h_q, h_kv, d_k, d_v, n_max, lens = case
    shape = workloads.custom(name, B=B, h_q=h_q, h_kv=h_kv, d_k=d_k, d_v=d_v,
                             n_max=n_max)
    inp = workloads.make(shape, seed=zlib.crc32(name.encode()) % 1000, lens=np.array(lens, np.int32))
    say(f"decode {name} chunk_rows={chunk_rows} lens={lens}")
    got = run_decode(inp, cuda_device, chunk_rows=chunk_rows)
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    check(got, ref, name)
    for b, n in enumerate(lens):
        if n == 0:
            assert np.array_equal(got[b], np.zeros_like(got[b]))


def test_chunk_size_invariance(cuda_device):
    shape = workloads.custom("chunks", B=2, h_q=8, h_kv=2, d_k=128, d_v=128, n_max=4096)
    inp = workloads.make(shape, seed=5, lens=np.array([4096, 3000], np.int32))
    outs = [run_decode(inp, cuda_device, chunk_rows=c) for c in (768, 1536, 4608, 0)]
    for o in outs[1:]:
        assert np.max(np.abs(o - outs[0])) <= 1e-6


def test_workspace_reuse_across_calls_and_shapes(cuda_device):
    """One workspace, many decodes in a row (counters must come back to zero
    after each), including a smaller problem in the same buffer."""
    shape = workloads.custom("reuse", B=3, h_q=16, h_kv=4, d_k=128, d_v=128, n_max=3000)
    inp = workloads.make(shape, seed=11, lens=np.array([3000, 1500, 77], np.int32))
    dq, dK, dV, dl = (dev(a, cuda_device) for a in (inp.q, inp.K, inp.V, inp.lens))
    ws = binding.alloc_workspace(dq, dK, dV)
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    for rep in range(5):
        out = binding.decode_attn(dq, dK, dV, dl, float(shape.scale32()), workspace=ws)
        torch.cuda.synchronize()
        check(out.cpu().numpy().astype(np.float64), ref, f"reuse {rep}")
    small = np.array([500, 0, 9], np.int32)
    out = binding.decode_attn(dq[:, :8].contiguous(), dK[:, :2].contiguous(),
                              dV[:, :2].contiguous(), dev(small, cuda_device),
                              float(shape.scale32()), workspace=ws)
    torch.cuda.synchronize()
    ref = oracle.decode(np.ascontiguousarray(inp.q[:, :8]), np.ascontiguousarray(inp.K[:, :2]),
                        np.ascontiguousarray(inp.V[:, :2]), small, shape.scale32())
    check(out.cpu().numpy().astype(np.float64), ref, "reuse smaller")


def test_len_beyond_capacity_is_clamped(cuda_device):
    shape = workloads.custom("clamp", B=2, h_q=4, h_kv=2, d_k=64, d_v=64, n_max=100)
    inp = workloads.make(shape, seed=6, lens=np.array([100, 100], np.int32))
    got = run_decode(inp, cuda_device, lens=np.array([100000, -5], np.int32))
    ref = oracle.decode(inp.q, inp.K, inp.V, np.array([100, 0], np.int32), shape.scale32())
    check(got, ref, "clamped len")


def test_identical_keys_give_mean_of_v(cuda_device):
    shape = workloads.custom("ident", B=1, h_q=8, h_kv=1, d_k=128, d_v=128, n_max=1000)
    inp = workloads.make(shape, seed=7)
    inp.K[:] = inp.K[:, :, :1]
    got = run_decode(inp, cuda_device)
    mean = inp.V[0, 0].astype(np.float64).mean(axis=0)
    for h in range(8):
        assert np.max(np.abs(got[0, h] - mean)) <= TOL


def test_large_logits_stay_finite(cuda_device):
    shape = workloads.custom("big", B=1, h_q=4, h_kv=1, d_k=128, d_v=128, n_max=500,
                             scale=1.0)
    inp = workloads.make(shape, seed=8)
    inp.q *= 4                       # scores of several hundred
    got = run_decode(inp, cuda_device)
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    check(got, ref, "large logits")


@pytest.mark.parametrize("h_q", [8, 32], ids=["one_block", "two_blocks"])
def test_rising_and_jumping_scores(cuda_device, h_q):
    """Scores that climb steadily along the rows (about 100 base-2 units
    over the sequence, so the softmax reference of the online form moves many
    times, with weights of up to 2^8 between moves), then fall, then jump far
    above everything before (a reference move that wipes the old weights)."""
    n = 3000
    shape = workloads.custom(f"rising_{h_q}", B=1, h_q=h_q, h_kv=1, d_k=128, d_v=128,
                             n_max=n)
    inp = workloads.make(shape, seed=31)
    u = inp.q[0, 0].astype(np.float64)
    u /= np.linalg.norm(u)
    # log2-unit score of head 0 along u: log2(e) * scale * |q0| per unit of K
    per_unit = np.log2(np.e) * shape.scale32() * np.linalg.norm(inp.q[0, 0].astype(np.float64))
    ramp = np.concatenate([np.linspace(0.0, 100.0, 2000), np.linspace(100.0, 20.0, 999),
                           [130.0]]) / per_unit
    inp.K[0, 0, :n] += (ramp[:, None] * u[None, :]).astype(np.float32)
    got = run_decode(inp, cuda_device)
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    check(got, ref, f"rising scores h_q={h_q}")


def test_plain_decode_leaves_cache_and_len_alone(cuda_device):
    shape = workloads.custom("plain", B=2, h_q=16, h_kv=2, d_k=128, d_v=128, n_max=900)
    inp = workloads.make(shape, seed=9, lens=np.array([900, 450], np.int32))
    dq, dK, dV, dl = (dev(a, cuda_device) for a in (inp.q, inp.K, inp.V, inp.lens))
    ws = poisoned_workspace(dq, dK, dV)
    out = binding.decode_attn(dq, dK, dV, dl, float(shape.scale32()), workspace=ws)
    torch.cuda.synchronize()
    assert dl.cpu().numpy().tolist() == [900, 450]
    assert np.array_equal(dK.cpu().numpy().view(np.uint32), inp.K.view(np.uint32))
    assert np.array_equal(dV.cpu().numpy().view(np.uint32), inp.V.view(np.uint32))
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    check(out.cpu().numpy().astype(np.float64), ref, "plain decode")


@pytest.mark.parametrize("h_q,h_kv", [(4, 1), (1, 1), (32, 1)])
def test_one_slab_many_visits(cuda_device, schedule, h_q, h_kv):
    """A single long slab in small chunks: every resident workgroup visits it,
    so its merge combines hundreds of partials."""
    n = 150_000
    shape = workloads.custom(f"one_slab_{h_q}", B=1, h_q=h_q, h_kv=h_kv, d_k=128, d_v=128,
                             n_max=n)
    inp = workloads.make(shape, seed=12, lens=np.array([n - 5], np.int32))
    say(f"one slab h_q={h_q}: decode")
    got = run_decode(inp, cuda_device, chunk_rows=768)
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    check(got, ref, f"one slab h_q={h_q}")


def test_decode_partial_then_merge_equals_decode(cuda_device):
    shape = workloads.custom("pm", B=2, h_q=16, h_kv=2, d_k=128, d_v=128, n_max=900)
    inp = workloads.make(shape, seed=9, lens=np.array([900, 450], np.int32))
    dq, dK, dV, dl = (dev(a, cuda_device) for a in (inp.q, inp.K, inp.V, inp.lens))
    ws = poisoned_workspace(dq, dK, dV)
    out = torch.empty((2, 16, 128), device=cuda_device)
    binding.decode_partial(dq, dK, dV, dl, float(shape.scale32()), ws)
    binding.decode_merge(out, ws, 2, 16, 2, 900, 128, 128)
    torch.cuda.synchronize()
    assert dl.cpu().numpy().tolist() == [900, 450]   # a plain decode leaves len alone
    torch.cuda.synchronize()
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    check(out.cpu().numpy().astype(np.float64), ref, "partial+merge")


def test_workspace_reset_after_a_lone_partial(cuda_device):
    """A partial without its merge leaves the scheduling counters set;
    da_decode_workspace_reset clears them, after which a decode on the same
    workspace matches the oracle (and leaves the counters zero again)."""
    shape = workloads.custom("reset", B=3, h_q=16, h_kv=4, d_k=128, d_v=128, n_max=5000)
    inp = workloads.make(shape, seed=17, lens=np.array([5000, 2500, 130], np.int32))
    dq, dK, dV, dl = (dev(a, cuda_device) for a in (inp.q, inp.K, inp.V, inp.lens))
    ws = poisoned_workspace(dq, dK, dV)
    nc = binding.workspace_counter_bytes(3, 16, 4, 5000, 128, 128)
    binding.decode_partial(dq, dK, dV, dl, float(shape.scale32()), ws)
    torch.cuda.synchronize()
    assert ws[:nc].any(), "a lone partial should leave counters set"
    binding.workspace_reset(ws, 3, 16, 4, 5000, 128, 128)
    torch.cuda.synchronize()
    assert not ws[:nc].any(), "reset left counters set"
    out = binding.decode_attn(dq, dK, dV, dl, float(shape.scale32()), workspace=ws)
    torch.cuda.synchronize()
    assert not ws[:nc].any()
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    check(out.cpu().numpy().astype(np.float64), ref, "decode after reset")


def test_validation_errors_raise(cuda_device):
    shape = workloads.custom("err", B=1, h_q=2, h_kv=1, d_k=64, d_v=64, n_max=64)
    inp = workloads.make(shape, seed=1)
    dq, dK, dV, dl = (dev(a, cuda_device) for a in (inp.q, inp.K, inp.V, inp.lens))
    small = torch.empty(8, dtype=torch.uint8, device=cuda_device)
    with pytest.raises(binding.DecodeAttnError, match="WORKSPACE"):
        binding.decode_attn(dq, dK, dV, dl, 0.1, workspace=small)
    with pytest.raises(binding.DecodeAttnError, match="SCALE"):
        binding.decode_attn(dq, dK, dV, dl, float("nan"))


def test_thousands_of_slabs_ragged(cuda_device):
    """2400 slabs (many more than resident workgroups, and than the 64 slabs
    one search step looks at), ragged lengths from 0 to 300."""
    B, h_q, h_kv, n_max = 300, 16, 8, 300
    shape = workloads.custom("many_slabs", B=B, h_q=h_q, h_kv=h_kv, d_k=64, d_v=64,
                             n_max=n_max)
    lens = np.random.default_rng(3).integers(0, n_max + 1, size=B).astype(np.int32)
    lens[:3] = [0, 1, n_max]
    inp = workloads.make(shape, seed=13, lens=lens)
    say("thousands of slabs: decode")
    got = run_decode(inp, cuda_device)
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    check(got, ref, "2400 slabs")


SCHEDULE = [
    # name, B, h_q, h_kv, d_k, d_v, n_max, lens
    # fewer static units than workgroups: most ranges are empty, most rows
    # dynamic, several sequences without any static unit
    ("sparse_static", 8, 8, 1, 64, 64, 8192, [10, 20, 30, 5, 0, 1, 200, 1000]),
    # two or more slabs per workgroup (one column block): every slab wholly
    # static, no dynamic units; a range walks from slab to slab, within a
    # sequence and across sequences
    ("ranges_span_slabs", 64, 16, 8, 64, 64, 800, "ragged"),
    # the same with 128 slabs per sequence
    ("wide_sequences_all_static", 4, 128, 128, 64, 64, 1000, "ragged"),
    # more sequences than the static part handles: dynamic units of whole
    # segments only, on multi-segment slabs
    ("many_sequences_dynamic", 300, 4, 2, 64, 64, 1000, "ragged"),
    # two column blocks with many slabs per workgroup: the 14/16 static share
    # with dynamic remainders where they pay (here only under the fixture's
    # dynamic schedule: 16 units per workgroup)
    ("two_blocks_many_slabs", 128, 256, 8, 64, 64, 800, "ragged"),
    # two column blocks: the full resident grid of two workgroups per CU
    # (interleaved ranks) on a ragged batch
    ("two_blocks_ragged", 8, 64, 2, 64, 64, 16384, "ragged"),
    # 1024 slabs or more of multi-segment caches: whole-slab ranges at two
    # workgroups per CU (512 ranges), a range walking several slabs
    ("two_wave_ranges", 128, 16, 8, 64, 64, 1000, "ragged"),
    ("two_wave_wide_sequences", 8, 128, 128, 128, 128, 900, "ragged"),
]


@pytest.mark.parametrize("case", SCHEDULE, ids=[c[0] for c in SCHEDULE])
def test_schedule_edge_cases(cuda_device, schedule, case):
    """Static ranges and dynamic units cover every row exactly once however
    the lengths fall: compared with the oracle, with NaN-poisoned partial
    slots (a slot never written would show)."""
    name, B, h_q, h_kv, d_k, d_v, n_max, lens = case
    if lens == "ragged":
        lens = np.random.default_rng(zlib.crc32(name.encode())).integers(0, n_max + 1, size=B)
        lens[:2] = [0, n_max]
    lens = np.asarray(lens, dtype=np.int32)
    shape = workloads.custom(name, B=B, h_q=h_q, h_kv=h_kv, d_k=d_k, d_v=d_v, n_max=n_max)
    inp = workloads.make(shape, seed=21, lens=lens)
    say(f"schedule {name}: decode")
    got = run_decode(inp, cuda_device)
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    check(got, ref, name)


def test_two_million_rows_one_slab(cuda_device):
    """One sequence of 2^21 + 5 rows (a slab of 512 MiB per tensor at d=64):
    row offsets beyond 2^31 bytes."""
    n = (1 << 21) + 5
    shape = workloads.custom("huge", B=1, h_q=4, h_kv=1, d_k=64, d_v=64, n_max=n)
    say("two million rows: generating inputs")
    inp = workloads.make(shape, seed=14)
    say("two million rows: decode")
    got = run_decode(inp, cuda_device)
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    check(got, ref, "2^21+5 rows")


# --- fused append + decode step ------------------------------------------------

STEP_CASES = [
    # name, B, h_q, h_kv, d_k, d_v, n_max, lens (initial)
    ("gqa8", 3, 16, 2, 128, 128, 700, [0, 333, 699]),     # empty, middle, fills up
    ("mha_d64", 2, 4, 4, 64, 64, 300, [299, 300]),         # one full cache: no append
    ("mqa32_dkdv", 2, 32, 1, 64, 128, 200, [5, 190]),
    ("neg_len", 2, 8, 4, 128, 128, 100, [-3, 40]),
    ("d256", 2, 8, 2, 256, 256, 400, [0, 399]),
    # many sequences in the one-launch form (single-segment slabs, G <= 16):
    # the last workgroup of each sequence advances len
    ("many_seqs_one_launch", 40, 12, 3, 128, 128, 257,
     [0, 1, 2, 128, 255, 256, 257, -1, 7, 200] * 4),
    # 1024 slabs of multi-segment caches: whole-slab ranges at two
    # workgroups per CU, then the merge
    ("two_wave_ranges_step", 128, 8, 8, 128, 128, 1200,
     [0, 1, 799, 800, 1199, 1200, -2, 500] * 16),
]


@pytest.mark.parametrize("case", STEP_CASES, ids=[c[0] for c in STEP_CASES])
def test_fused_step_equals_append_then_decode(cuda_device, case):
    name, B, h_q, h_kv, d_k, d_v, n_max, lens = case
    shape = workloads.custom(name, B=B, h_q=h_q, h_kv=h_kv, d_k=d_k, d_v=d_v,
                             n_max=n_max, steps=3)
    inp = workloads.make(shape, seed=zlib.crc32(name.encode()) % 1000,
                         lens=np.array(lens, np.int32))
    dK, dV, dl = dev(inp.K, cuda_device), dev(inp.V, cuda_device), dev(inp.lens, cuda_device)
    hK, hV, hl = inp.K.copy(), inp.V.copy(), inp.lens.copy()
    ws = poisoned_workspace(dev(inp.q, cuda_device), dK, dV)
    for t in range(shape.steps):
        say(f"step {name} t={t} len={hl.tolist()}")
        out = binding.decode_step(dev(inp.q_step[t], cuda_device), dK, dV,
                                  dev(inp.k_new[t], cuda_device), dev(inp.v_new[t], cuda_device),
                                  dl, float(shape.scale32()), workspace=ws)
        torch.cuda.synchronize()
        oracle.append(hK, hV, inp.k_new[t], inp.v_new[t], hl)
        ref = oracle.decode(inp.q_step[t], hK, hV, hl, shape.scale32())
        assert dl.cpu().numpy().tolist() == hl.tolist()
        assert np.array_equal(dK.cpu().numpy().view(np.uint32), hK.view(np.uint32))
        assert np.array_equal(dV.cpu().numpy().view(np.uint32), hV.view(np.uint32))
        nc = binding.workspace_counter_bytes(B, h_q, h_kv, n_max, d_k, d_v)
        assert not ws[:nc].any(), "counters not back to zero after the step"
        check(out.cpu().numpy().astype(np.float64), ref, f"step {name} t={t}")


def test_fused_step_long_context(cuda_device):
    """The long-context workload's first steps through the fused step call
    (da_decode_step), every head checked (the oracle replays the appends on
    the host)."""
    shape = workloads.get("c5")
    say("fused step long-context: generating inputs")
    inp = workloads.make(shape, seed=3)
    dK, dV, dl = dev(inp.K, cuda_device), dev(inp.V, cuda_device), dev(inp.lens, cuda_device)
    hK, hV, hl = inp.K, inp.V, inp.lens.copy()
    ws = binding.alloc_workspace(dev(inp.q, cuda_device), dK, dV)
    for t in range(4):
        out = binding.decode_step(dev(inp.q_step[t], cuda_device), dK, dV,
                                  dev(inp.k_new[t], cuda_device), dev(inp.v_new[t], cuda_device),
                                  dl, float(shape.scale32()), workspace=ws)
        oracle.append(hK, hV, inp.k_new[t], inp.v_new[t], hl)
        torch.cuda.synchronize()
        ref = oracle.decode(inp.q_step[t], hK, hV, hl, shape.scale32())
        check(out.cpu().numpy().astype(np.float64), ref, f"fused step {t}")
        assert dl.cpu().numpy().tolist() == hl.tolist()


@pytest.mark.parametrize("n_max", [1200, 500, 20000],
                         ids=["two_launches", "one_launch", "long_slabs"])
def test_graph_replay_of_fused_steps(cuda_device, schedule, n_max):
    """Several fused steps captured in one HIP graph and replayed three times,
    each replay from the same initial cache with eager work in between: every
    replay matches the oracle step by step (the kernels hold no memset and
    leave the workspace counters zero, so replays are independent).  At
    n_max = 500 every slab is one segment and each step is a single launch;
    at 20000 the short batch of long slabs runs as two-wave ranges (the
    library's schedule) or with dynamic units (the fixture's other mode)."""
    T = 4
    shape = workloads.custom("graph", B=3, h_q=16, h_kv=2, d_k=128, d_v=128, n_max=n_max,
                             steps=T)
    inp = workloads.make(shape, seed=21, lens=np.array([0, n_max // 2, n_max - 2], np.int32))
    dK0, dV0, dl0 = dev(inp.K, cuda_device), dev(inp.V, cuda_device), dev(inp.lens, cuda_device)
    dK, dV, dl = dK0.clone(), dV0.clone(), dl0.clone()
    qs = [dev(inp.q_step[t], cuda_device) for t in range(T)]
    kn = [dev(inp.k_new[t], cuda_device) for t in range(T)]
    vn = [dev(inp.v_new[t], cuda_device) for t in range(T)]
    ws = binding.alloc_workspace(qs[0], dK, dV)
    outs = [torch.empty((3, 16, 128), device=cuda_device) for _ in range(T)]
    scale = float(shape.scale32())
    # host mirror and oracle outputs of the T steps
    hK, hV, hl = inp.K.copy(), inp.V.copy(), inp.lens.copy()
    refs = []
    for t in range(T):
        oracle.append(hK, hV, inp.k_new[t], inp.v_new[t], hl)
        refs.append(oracle.decode(inp.q_step[t], hK, hV, hl, shape.scale32()))
    # one eager pass first (loads the kernels before capture)
    for t in range(T):
        binding.decode_step(qs[t], dK, dV, kn[t], vn[t], dl, scale, out=outs[t], workspace=ws)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for t in range(T):
            binding.decode_step(qs[t], dK, dV, kn[t], vn[t], dl, scale, out=outs[t],
                                workspace=ws)
    for rep in range(3):
        dK.copy_(dK0)
        dV.copy_(dV0)
        dl.copy_(dl0)
        for o in outs:
            o.fill_(float("nan"))
        torch.cuda.synchronize()
        say(f"graph replay {rep}")
        graph.replay()
        torch.cuda.synchronize()
        for t in range(T):
            check(outs[t].cpu().numpy().astype(np.float64), refs[t], f"replay {rep} step {t}")
        assert dl.cpu().numpy().tolist() == hl.tolist()
        assert np.array_equal(dK.cpu().numpy().view(np.uint32), hK.view(np.uint32))
        assert np.array_equal(dV.cpu().numpy().view(np.uint32), hV.view(np.uint32))
        nc = binding.workspace_counter_bytes(3, 16, 2, n_max, 128, 128)
        assert not ws[:nc].any()


# --- append: bit-exact --------------------------------------------------------

@pytest.mark.parametrize("d_k,d_v", [(128, 128), (64, 128), (4, 12)])
def test_append_bit_exact(cuda_device, d_k, d_v):
    B, h_kv, n_max = 3, 5, 9
    rng = np.random.default_rng([d_k, d_v])
    K = rng.standard_normal((B, h_kv, n_max, d_k)).astype(np.float32)
    V = rng.standard_normal((B, h_kv, n_max, d_v)).astype(np.float32)
    lens = np.array([0, 4, 8], np.int32)
    dK, dV, dl = dev(K, cuda_device), dev(V, cuda_device), dev(lens, cuda_device)
    for step in range(3):   # the third sequence fills up after one append
        kn = rng.standard_normal((B, h_kv, d_k)).astype(np.float32)
        vn = rng.standard_normal((B, h_kv, d_v)).astype(np.float32)
        # odd bit patterns must survive: NaN payloads, -0, denormals, inf
        kn.view(np.uint32)[0, 0, :4] = [0x7FC01234, 0xFFA00001, 0x80000000, 0x00000001]
        vn.view(np.uint32)[1, 2, :2] = [0x7F800000, 0x7F812345]
        say(f"append d_k={d_k} d_v={d_v} step={step}")
        binding.kv_append(dK, dV, dev(kn, cuda_device), dev(vn, cuda_device), dl)
        oracle.append(K, V, kn, vn, lens)
        torch.cuda.synchronize()
        assert np.array_equal(dl.cpu().numpy(), lens)
        assert np.array_equal(dK.cpu().numpy().view(np.uint32), K.view(np.uint32))
        assert np.array_equal(dV.cpu().numpy().view(np.uint32), V.view(np.uint32))
    assert lens.tolist() == [3, 7, 9]


def test_append_with_negative_len_is_a_no_op(cuda_device):
    K = torch.zeros((2, 1, 4, 4), device=cuda_device)
    V = torch.zeros((2, 1, 4, 4), device=cuda_device)
    lens = torch.tensor([-1, 4], dtype=torch.int32, device=cuda_device)
    one = torch.ones((2, 1, 4), device=cuda_device)
    binding.kv_append(K, V, one, one, lens)
    torch.cuda.synchronize()
    assert lens.tolist() == [-1, 4] and not K.any() and not V.any()


# --- the five workloads, every head of every step -------------------------------

@pytest.mark.parametrize("name", ["c1", "c3", "c4"])
def test_single_step_workloads(cuda_device, name):
    shape = workloads.get(name)
    say(f"workload {shape.name}: generating inputs")
    inp = workloads.make(shape, seed=0)
    say(f"workload {shape.name}: decode")
    got = run_decode(inp, cuda_device)
    say(f"workload {shape.name}: oracle")
    ref = oracle.decode(inp.q, inp.K, inp.V, inp.lens, shape.scale32())
    check(got, ref, shape.name)


@pytest.mark.parametrize("fused", [False, True], ids=["append_then_decode", "fused_step"])
@pytest.mark.parametrize("name", ["c2", "c5"])
def test_multi_step_workloads(cuda_device, name, fused):
    """Append then decode, step after step, with len kept on the device --
    as two calls, or fused as the benchmark times it (the partial kernel with
    the append, then the merge); the host mirror replays every append and the
    oracle checks every head of every step, and the appended rows bit for
    bit."""
    shape = workloads.get(name)
    say(f"workload {shape.name}: generating inputs")
    inp = workloads.make(shape, seed=0)
    dK, dV = dev(inp.K, cuda_device), dev(inp.V, cuda_device)
    dl = dev(inp.lens, cuda_device)
    hK, hV, hl = inp.K, inp.V, inp.lens.copy()
    dq0 = dev(inp.q_step[0], cuda_device)
    ws = binding.alloc_workspace(dq0, dK, dV)
    out = torch.empty((shape.B, shape.h_q, shape.d_v), device=cuda_device)
    for t in range(shape.steps):
        dq = dev(inp.q_step[t], cuda_device)
        kn, vn = dev(inp.k_new[t], cuda_device), dev(inp.v_new[t], cuda_device)
        if fused:
            binding.decode_partial(dq, dK, dV, dl, float(shape.scale32()), ws, k_new=kn, v_new=vn)
            binding.decode_merge(out, ws, shape.B, shape.h_q, shape.h_kv, shape.n_max,
                                 shape.d_k, shape.d_v, lens=dl)
        else:
            binding.kv_append(dK, dV, kn, vn, dl)
            binding.decode_attn(dq, dK, dV, dl, float(shape.scale32()), out=out, workspace=ws)
        oracle.append(hK, hV, inp.k_new[t], inp.v_new[t], hl)
        torch.cuda.synchronize()
        assert np.array_equal(dl.cpu().numpy(), hl)
        got = out.cpu().numpy().astype(np.float64)
        ref = oracle.decode(inp.q_step[t], hK, hV, hl, shape.scale32())
        check(got, ref, f"{shape.name} step {t}")
        # the appended rows themselves, bit for bit
        rows = hl.astype(np.int64) - 1
        for b in range(shape.B):
            r = int(rows[b])
            assert np.array_equal(dK[b, :, r].cpu().numpy().view(np.uint32),
                                  hK[b, :, r].view(np.uint32))
            assert np.array_equal(dV[b, :, r].cpu().numpy().view(np.uint32),
                                  hV[b, :, r].view(np.uint32))
    torch.cuda.synchronize()
    assert np.array_equal(dl.cpu().numpy(), hl)
