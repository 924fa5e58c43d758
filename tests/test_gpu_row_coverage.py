"""Row coverage at full length: every cache row, the appended one included,
is counted exactly once (eq. (3) and Algorithm 1 sum over every l < n;
Proposition 2 adds exactly one row per step).

With N(0,1) inputs one row of a 10^5-row slab weighs about 1/(1.65 n), so a
dropped or doubled row moves the output by less than the 1e-5 tolerance for
many rows.  Here the rows where a decomposition of the slab can cut it --
the first and last row of every 64-row turn of the workgroup's waves (every
tile-ring unit, segment, static range and visit starts and ends on such a
row), row len-1 and the appended row -- are planted: each gets the key of
one query head of its group, scaled so that this head scores it 10 natural
units above the N(0,1) rows, and the G heads of a group have orthonormal
query directions, so a planted row weighs about 1/(planted rows of its head)
for its head and nothing for the others.  Dropping or doubling any planted
row then moves its head's output by more than 1e-4, which the tests assert
on the CPU from the oracle's own weights before comparing the GPU with the
oracle at 1e-5.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_19456_amd import workloads

TOL = 1e-5
GRID = 64          # rows per turn of a workgroup's four waves (4 x 16-row tiles)
SCORE = 10.0       # planted score, natural units
SENSITIVITY = 1e-4


def say(msg):
    print(msg, flush=True)


def dev(a, device):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def planted_rows(n_old, n):
    """Rows of a slab with n rows (n_old before this step's append) that lie
    on a boundary of some 64-row turn, plus rows n_old-1 .. n-1."""
    if n <= 0:
        return np.zeros(0, np.int64)
    first = np.arange(0, n, GRID)
    last = np.minimum(first + GRID - 1, n - 1)
    extra = np.arange(max(n_old - 1, 0), n)
    return np.unique(np.concatenate([first, last, extra]))


def orthonormal_queries(B, h_q, h_kv, d, seed):
    """q [B][h_q][d] fp32 whose G heads of each group are orthonormal
    directions scaled to |q| = sqrt(d) (the norm of an N(0,1) vector), and
    the unit directions u [B][h_kv][G][d] (fp64)."""
    G = h_q // h_kv
    a = workloads.normal(seed, 91, (B, h_kv, d, G)).astype(np.float64)
    u = np.empty((B, h_kv, G, d))
    for b in range(B):
        for g in range(h_kv):
            qmat, _ = np.linalg.qr(a[b, g])
            u[b, g] = qmat.T
    q = (u * np.sqrt(d)).reshape(B, h_q, d).astype(np.float32)
    return q, u


def plant(K, u, lens_old, lens_new, n_max):
    """Plant rows of every slab in place: row l (the i-th planted row of its
    slab) gets SCORE/scale along head i mod G's direction, so that head
    scores it SCORE (scale = 1/sqrt(d)).  Returns the planted rows and
    their heads per (b, g)."""
    B, h_kv, G, d = u.shape
    mag = SCORE * np.sqrt(d)
    rows = {}
    for b in range(B):
        n_old = int(min(max(lens_old[b], 0), n_max))
        n = int(min(max(lens_new[b], 0), n_max))
        r = planted_rows(n_old, n)
        r_old = r[r < n_old]
        for g in range(h_kv):
            heads = (np.arange(len(r)) + b + g) % G
            K[b, g, r_old] = (mag * u[b, g, heads[:len(r_old)]]).astype(np.float32)
            rows[(b, g)] = (r, heads)
    return rows


def plant_new_rows(k_new, u, rows, lens_old, n_max):
    """The appended row of every (b, g) (row len_old), planted like the
    cache rows (its head from the same numbering)."""
    B, h_kv, G, d = u.shape
    for b in range(B):
        if not 0 <= lens_old[b] < n_max:
            continue
        for g in range(h_kv):
            r, heads = rows[(b, g)]
            i = int(np.searchsorted(r, lens_old[b]))
            assert r[i] == lens_old[b]
            k_new[b, g] = (SCORE * np.sqrt(d) * u[b, g, heads[i]]).astype(np.float32)


def assert_sensitive(q, K, V, lens, scale, rows, G):
    """For every planted row: deleting it (or counting it twice) changes its
    head's oracle output by more than SENSITIVITY.  From the head's weights
    a: deleting row l gives (out - a_l v_l) / (1 - a_l), so the change is
    a_l (out - v_l) / (1 - a_l); doubling it a_l (v_l - out) / (1 + a_l)."""
    worst = np.inf
    for (b, g), (r, heads) in rows.items():
        for j in range(G):
            sel = r[heads == j]
            if sel.size == 0:
                continue
            w, out = oracle.decode_weights(q, K, V, lens, scale, b, g * G + j)
            a = w[sel][:, None]
            diff = np.abs(out[None, :] - V[b, g, sel].astype(np.float64)).max(axis=1)[:, None]
            change = (a / (1 + a) * diff).min()      # doubling moves it least
            worst = min(worst, float(change))
    say(f"  smallest output change from one dropped/doubled planted row: {worst:.2e}")
    assert worst > SENSITIVITY


def check(got, ref, what):
    assert got.shape == ref.shape
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = float(np.max(np.abs(got - ref)))
    say(f"  {what}: max-abs-err {err:.3e}")
    assert err <= TOL, f"{what}: max-abs-err {err:.3e} > {TOL}"


def test_the_change_formula_is_the_oracle_itself():
    """CPU pin of the algebra assert_sensitive relies on: removing a row (its
    key moved so far down that its weight underflows to zero) or adding a
    copy changes the oracle's output by exactly a_l (out - v_l) / (1 - a_l),
    resp. a_l (v_l - out) / (1 + a_l), for rows of any weight."""
    B, h_q, h_kv, d, n = 1, 4, 1, 32, 300
    shape = workloads.custom("cov_pin", B=B, h_q=h_q, h_kv=h_kv, d_k=d, d_v=d, n_max=n + 1)
    inp = workloads.make(shape, seed=5, lens=np.array([n], np.int32))
    q, u = orthonormal_queries(B, h_q, h_kv, d, seed=6)
    rows = plant(inp.K, u, inp.lens, inp.lens, n + 1)
    scale = shape.scale32()
    r, heads = rows[(0, 0)]
    for l, j in [(r[0], heads[0]), (r[5], heads[5]), (7, 2), (n - 1, heads[-1])]:
        w, out = oracle.decode_weights(q, inp.K, inp.V, inp.lens, scale, 0, int(j))
        a, v = w[l], inp.V[0, 0, l].astype(np.float64)
        K2 = inp.K.copy()
        K2[0, 0, l] = (-1e4 * u[0, 0, j]).astype(np.float32)        # weight exp(-1e4) = 0
        gone = oracle.decode(q, K2, inp.V, inp.lens, scale)[0, j]
        assert np.allclose(gone - out, a * (out - v) / (1 - a), rtol=1e-9, atol=1e-15)
        K3 = np.zeros((1, 1, n + 1, d), np.float32)
        V3 = np.zeros_like(K3)
        K3[0, 0, :n], V3[0, 0, :n] = inp.K[0, 0, :n], inp.V[0, 0, :n]
        K3[0, 0, n], V3[0, 0, n] = inp.K[0, 0, l], inp.V[0, 0, l]     # row l twice
        twice = oracle.decode(q, K3, V3, np.array([n + 1], np.int32), scale)[0, j]
        assert np.allclose(twice - out, a * (v - out) / (1 + a), rtol=1e-9, atol=1e-15)


@pytest.mark.gpu
def test_long_context_rows_each_counted_once(cuda_device):
    """The long-context workload's shapes and lengths (B=4, 64/8 heads,
    d=128, n_max=131072, len ~ U{65536..131008}): a plain decode, then two
    fused append+decode steps with planted appended rows, every head
    against the oracle."""
    from paper_2607_19456_amd import binding

    shape = workloads.get("c5")
    say("row coverage, long context: generating inputs")
    inp = workloads.make(shape, seed=7)
    B, h_q, h_kv, d = shape.B, shape.h_q, shape.h_kv, shape.d_k
    G = h_q // h_kv
    q, u = orthonormal_queries(B, h_q, h_kv, d, seed=8)
    scale = shape.scale32()
    lens = inp.lens.copy()
    rows = plant(inp.K, u, lens, lens, shape.n_max)
    assert_sensitive(q, inp.K, inp.V, lens, scale, rows, G)
    dK, dV, dl = dev(inp.K, cuda_device), dev(inp.V, cuda_device), dev(lens, cuda_device)
    dq = dev(q, cuda_device)
    ws = binding.alloc_workspace(dq, dK, dV)
    say("row coverage, long context: plain decode")
    out = binding.decode_attn(dq, dK, dV, dl, float(scale), workspace=ws)
    torch.cuda.synchronize()
    check(out.cpu().numpy().astype(np.float64),
          oracle.decode(q, inp.K, inp.V, lens, scale), "plain decode")
    hK, hV, hl = inp.K, inp.V, lens.copy()
    for t in range(2):
        kn, vn = inp.k_new[t].copy(), inp.v_new[t]
        new_lens = np.minimum(hl + 1, shape.n_max)
        rows = plant(hK, u, hl, new_lens, shape.n_max)
        plant_new_rows(kn, u, rows, hl, shape.n_max)
        dK.copy_(dev(hK, cuda_device))              # the cache rows planted for this step
        say(f"row coverage, long context: fused step {t}")
        out = binding.decode_step(dq, dK, dV, dev(kn, cuda_device), dev(vn, cuda_device), dl,
                                  float(scale), workspace=ws)
        oracle.append(hK, hV, kn, vn, hl)
        torch.cuda.synchronize()
        assert dl.cpu().numpy().tolist() == hl.tolist()
        assert_sensitive(q, hK, hV, hl, scale, rows, G)
        check(out.cpu().numpy().astype(np.float64), oracle.decode(q, hK, hV, hl, scale),
              f"fused step {t}")


@pytest.mark.gpu
def test_two_million_row_slab_rows_each_counted_once(cuda_device):
    """One sequence of 2^21 + 5 rows (16 query heads on one KV head, d=64):
    a plain decode, then a fused step that appends row 2^21 + 5."""
    from paper_2607_19456_amd import binding

    n = (1 << 21) + 5
    shape = workloads.custom("cov_huge", B=1, h_q=16, h_kv=1, d_k=64, d_v=64, n_max=n + 1,
                             steps=1)
    say("row coverage, 2^21+5 rows: generating inputs")
    inp = workloads.make(shape, seed=9, lens=np.array([n], np.int32))
    q, u = orthonormal_queries(1, 16, 1, 64, seed=10)
    scale = shape.scale32()
    lens = inp.lens.copy()
    rows = plant(inp.K, u, lens, lens, shape.n_max)
    assert_sensitive(q, inp.K, inp.V, lens, scale, rows, 16)
    dK, dV, dl = dev(inp.K, cuda_device), dev(inp.V, cuda_device), dev(lens, cuda_device)
    dq = dev(q, cuda_device)
    ws = binding.alloc_workspace(dq, dK, dV)
    say("row coverage, 2^21+5 rows: plain decode")
    out = binding.decode_attn(dq, dK, dV, dl, float(scale), workspace=ws)
    torch.cuda.synchronize()
    check(out.cpu().numpy().astype(np.float64),
          oracle.decode(q, inp.K, inp.V, lens, scale), "plain decode")
    kn = inp.k_new[0].copy()
    rows = plant(inp.K, u, lens, lens + 1, shape.n_max)
    plant_new_rows(kn, u, rows, lens, shape.n_max)
    say("row coverage, 2^21+5 rows: fused step")
    out = binding.decode_step(dq, dK, dV, dev(kn, cuda_device), dev(inp.v_new[0], cuda_device),
                              dl, float(scale), workspace=ws)
    hK, hV, hl = inp.K, inp.V, lens.copy()
    oracle.append(hK, hV, kn, inp.v_new[0], hl)
    torch.cuda.synchronize()
    assert dl.cpu().numpy().tolist() == [n + 1]
    assert_sensitive(q, hK, hV, hl, scale, rows, 16)
    check(out.cpu().numpy().astype(np.float64), oracle.decode(q, hK, hV, hl, scale),
          "fused step")
