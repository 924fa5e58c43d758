"""The C-ABI library on the CPU: it loads, exports every symbol the header
declares, and its host-side validation rejects bad arguments before anything
is enqueued (these calls never reach the GPU, so they run without one)."""
import ctypes
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "decode_attn.h")

binding = pytest.importorskip("paper_2607_19456_amd.binding",
                              reason="HIP library not built")
lib = binding._lib

FAKE = 0x10000   # a 16-byte aligned, never dereferenced address


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return set(re.findall(r"\b(da_[a-z_]+)\s*\(", text))


# The boundary's core, exactly as specified: argument types in order
# (pointers, scalars) and the result type.
CORE_PROTOTYPES = {
    "da_status_string": ("const char *", ["da_status"]),
    "da_decode_workspace_bytes": ("size_t", ["int"] * 6),
    "da_decode_attn": ("da_status", ["const float *"] * 3 + ["const int32_t *", "float",
                                                              "float *"] + ["int"] * 6
                       + ["void *", "size_t", "void *"]),
    "da_kv_append": ("da_status", ["float *", "float *", "const float *", "const float *",
                                   "int32_t *"] + ["int"] * 5 + ["void *"]),
}


def _norm(t):
    """A C type with canonical spacing: 'const float*' -> 'const float *'."""
    return " ".join(t.replace("*", " * ").split())


def _prototypes():
    """name -> (result type, [parameter types]) for every declaration in the
    header (parameter names dropped)."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    protos = {}
    for m in re.finditer(r"([A-Za-z_][\w \t\*]*?)\b(da_[a-z_]+)\s*\(([^)]*)\)\s*;", text):
        params = []
        for p in m.group(3).split(","):
            toks = _norm(p).split(" ")
            params.append(" ".join(toks[:-1]))          # drop the parameter name
        protos[m.group(2)] = (_norm(m.group(1).split("\n")[-1]), params)
    return protos


def test_core_prototypes_are_exactly_the_specified_ones():
    protos = _prototypes()
    for name, (ret, params) in CORE_PROTOTYPES.items():
        assert name in protos, name
        got_ret, got_params = protos[name]
        assert got_ret == _norm(ret), (name, got_ret)
        assert got_params == [_norm(p) for p in params], (name, got_params)
    # the tuning knob appears only in the tuning calls
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    for m in re.finditer(r"\b(da_[a-z_]+)\s*\(([^)]*)\)\s*;", text):
        if "chunk_rows" in m.group(2):
            assert m.group(1).endswith("_ex"), m.group(1)


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert names == set(binding.SIGNATURES), names ^ set(binding.SIGNATURES)
    protos = _prototypes()
    for n, (_, params) in protos.items():
        assert len(params) == len(binding.SIGNATURES[n][1]), n
    for n in names:
        assert hasattr(lib, n)
    out = subprocess.run(["nm", "-D", "--defined-only", binding.LIBRARY_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (da_[a-z_]+)\b", out))
    assert names <= exported


def test_status_strings():
    for code, name in binding.STATUS.items():
        assert lib.da_status_string(code).decode().startswith(name)
    assert b"unknown" in lib.da_status_string(99)


def _expected_workspace(B, h_q, h_kv, n_max, d_k, d_v, c):
    """The sizing rule, restated: rows are scheduled in units of one ring
    turn (64 rows per tile of the ring: 3 tiles for one column block, 4 for
    two, 2 for large heads); per (b, query head) one visit slot for each static
    visit a slab can have (at most one per unit plus one, and at most one per
    resident workgroup) and, for dynamic visits, up to 4x the even share of
    resident workgroups per slab (at most one per unit); one 128-byte
    counter line per slab and one visit count per (b, query head).
    Single-chunk caches and batches of more than 256 sequences are scheduled
    dynamically only, in whole chunks.  Caches of at most 4608 rows (one
    column block, d_k + d_v <= 256) run as whole-slab ranges at two
    workgroups per CU with a two-tile ring, and so may batches of fewer
    than 16 * 256 one-wave units (192 rows each) of any length: the
    workspace is sized for that form whenever it may be chosen."""
    pad = lambda x: -(-x // 256) * 256
    G = h_q // h_kv
    groups = -(-G // 32)
    slabs = B * h_kv * groups
    chunks = -(-n_max // c)
    resident = 256                      # one workgroup per CU
    grid = max(1, min(resident, chunks * slabs))
    static = chunks > 1 and B <= 256
    ring = 2 if d_k + d_v > 256 else (4 if G > 16 else 3)
    units = slabs * -(-n_max // (ring * 64))
    if static and G <= 16 and d_k + d_v <= 256 and (n_max <= 4608 or units < 16 * resident):
        grid = min(2 * resident, chunks * slabs)
        ring = 2
    dyn_rows = ring * 64 if static else c
    Js = min(grid, -(-n_max // dyn_rows)) + 1 if static else 0
    Jd = max(1, min(-(-n_max // dyn_rows), 4 * -(-grid // slabs)))
    J = Js + Jd
    slots = B * h_q * J
    counters = pad(slabs * 128) + pad(B * h_q * 4)
    return counters, counters + pad(slots * 8) + slots * d_v * 4


def expected_chunk_rows(B, h_q, h_kv, n_max, d_k, d_v):
    """The library's segment size: 768 rows, or the whole cache rounded up to
    768 if shorter, or if there are at least 2048 slabs of at most 4608 rows
    with one column block (G <= 16) and d_k + d_v <= 256 (the direct form)."""
    whole = -(-n_max // 768) * 768
    G = h_q // h_kv
    slabs = B * h_kv * -(-G // 32)
    c = 768
    if G <= 16 and d_k + d_v <= 256 and slabs >= 2048 and n_max <= 4608:
        c = whole
    return min(c, whole)


def test_chunk_rows_and_workspace_sizes():
    for args in [(1, 1, 1, 128, 64, 64), (8, 32, 32, 4112, 128, 128),
                 (16, 32, 8, 8192, 128, 128), (32, 32, 1, 16384, 128, 128),
                 (4, 64, 8, 131072, 128, 128), (3, 40, 5, 77, 64, 128),
                 (2, 64, 2, 5000, 256, 256), (2, 16, 2, 900, 256, 64),
                 (256, 8, 8, 1536, 128, 128), (64, 32, 32, 1040, 128, 128),
                 (2048, 8, 8, 4608, 64, 64), (2048, 8, 8, 4609, 64, 64),
                 (1024, 16, 2, 1000, 128, 128), (1024, 17, 1, 1000, 64, 64),
                 (512, 8, 4, 2000, 128, 256), (128, 32, 8, 8192, 128, 128),
                 (256, 16, 4, 2048, 64, 64), (1024, 8, 1, 5000, 128, 128),
                 (2, 32, 8, 32768, 128, 128), (1, 32, 8, 65536, 128, 128),
                 (4, 32, 8, 16384, 64, 64), (16, 16, 4, 16384, 128, 128)]:
        c = binding.chunk_rows(*args)
        assert c == expected_chunk_rows(*args), args
        counters, total = _expected_workspace(*args, c)
        assert binding.workspace_counter_bytes(*args) == counters
        assert binding.workspace_bytes(*args) == total
        assert lib.da_decode_workspace_bytes(*args) == total
        assert lib.da_decode_workspace_bytes_ex(*args, 0) == total
        assert binding.workspace_bytes(*args, 1536) == _expected_workspace(*args, 1536)[1]
    assert binding.chunk_rows(1, 3, 2, 10, 64, 64) == 0       # h_kv does not divide h_q
    assert binding.workspace_bytes(1, 1, 1, 10, 96, 64) == 0  # unsupported d_k
    assert binding.workspace_bytes(1, 1, 1, 10, 64, 64, 192) == 0  # chunk not a multiple of 768
    assert binding.workspace_bytes(1, 1, 1, 10, 64, 64, 384) == 0
    assert lib.da_decode_workspace_bytes(1, 3, 2, 10, 64, 64) == 0


@pytest.mark.parametrize("value", ["0", "32", "1000", "bad", ""])
def test_dynamic_share_override_leaves_sizes_alone(monkeypatch, value):
    """The tuning override of the dynamic share (DECODE_ATTN_DYNAMIC_MIN_UNITS,
    read at every call) changes which rows are scheduled how, never the
    workspace a caller must provide or the segment size."""
    args = [(32, 32, 1, 16384, 128, 128), (16, 32, 8, 8192, 128, 128),
            (4, 64, 8, 131072, 128, 128), (3, 40, 5, 77, 64, 128),
            (2, 32, 8, 32768, 128, 128), (1, 32, 8, 65536, 128, 128)]
    monkeypatch.delenv("DECODE_ATTN_DYNAMIC_MIN_UNITS", raising=False)
    ref = [(lib.da_decode_workspace_bytes(*a), binding.chunk_rows(*a)) for a in args]
    monkeypatch.setenv("DECODE_ATTN_DYNAMIC_MIN_UNITS", value)
    assert [(lib.da_decode_workspace_bytes(*a), binding.chunk_rows(*a)) for a in args] == ref


def _decode(**kw):
    """da_decode_attn, or with ``chunk`` its tuning form da_decode_multi_ex."""
    a = dict(q=FAKE, K=FAKE, V=FAKE, len=FAKE, scale=0.125, out=FAKE, B=1, h_q=1,
             h_kv=1, n_max=128, d_k=64, d_v=64, chunk=None, ws=FAKE, wsn=1 << 30,
             stream=None)
    a.update(kw)
    head = (a["q"], a["K"], a["V"], a["len"], a["scale"], a["out"], a["B"], a["h_q"],
            a["h_kv"], a["n_max"], a["d_k"], a["d_v"])
    if a["chunk"] is None:
        return lib.da_decode_attn(*head, a["ws"], a["wsn"], a["stream"])
    return lib.da_decode_multi_ex(*head, 1, a["chunk"], a["ws"], a["wsn"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), 1), (dict(K=None), 1), (dict(V=None), 1), (dict(len=None), 1),
    (dict(out=None), 1),
    (dict(B=0), 2), (dict(h_q=0), 2), (dict(h_kv=0), 2), (dict(n_max=0), 2),
    (dict(h_q=3, h_kv=2), 2), (dict(B=1 << 21), 2), (dict(chunk=100), 2),
    (dict(chunk=192), 2), (dict(chunk=384), 2), (dict(chunk=-768), 2),
    (dict(d_k=96), 3), (dict(d_v=32), 3), (dict(d_k=512), 3),
    (dict(q=FAKE + 4), 4), (dict(K=FAKE + 8), 4), (dict(out=FAKE + 4), 4),
    (dict(len=FAKE + 2), 4),
    (dict(scale=float("nan")), 5), (dict(scale=float("inf")), 5),
    (dict(ws=None), 6), (dict(wsn=16), 6),
    (dict(ws=FAKE + 4), 4),
])
def test_decode_validation(kw, status):
    assert _decode(**kw) == status


def test_partial_and_merge_validation():
    P = lib.da_decode_partial
    assert P(None, FAKE, FAKE, None, None, FAKE, 0.1, 1, 1, 1, 64, 64, 64,
             FAKE, 1 << 20, None) == 1
    assert P(FAKE, FAKE, FAKE, None, None, FAKE, 0.1, 1, 1, 1, 64, 64, 64,
             FAKE, 8, None) == 6
    # k_new and v_new come together or not at all
    assert P(FAKE, FAKE, FAKE, FAKE, None, FAKE, 0.1, 1, 1, 1, 64, 64, 64,
             FAKE, 1 << 20, None) == 1
    assert P(FAKE, FAKE, FAKE, FAKE, FAKE + 4, FAKE, 0.1, 1, 1, 1, 64, 64, 64,
             FAKE, 1 << 20, None) == 4
    M = lib.da_decode_merge
    assert M(None, None, 1, 1, 1, 64, 64, 64, FAKE, 1 << 20, None) == 1
    assert M(FAKE, None, 1, 2, 3, 64, 64, 64, FAKE, 1 << 20, None) == 2
    assert M(FAKE, None, 1, 1, 1, 64, 64, 64, FAKE, 4, None) == 6
    assert M(FAKE + 4, None, 1, 1, 1, 64, 64, 64, FAKE, 1 << 20, None) == 4
    assert M(FAKE, FAKE + 2, 1, 1, 1, 64, 64, 64, FAKE, 1 << 20, None) == 4
    # the tuning forms take T and chunk_rows
    PX = lib.da_decode_partial_ex
    assert PX(FAKE, FAKE, FAKE, None, None, FAKE, 0.1, 1, 1, 1, 64, 64, 64, 1, 384,
              FAKE, 1 << 20, None) == 2
    assert PX(FAKE, FAKE, FAKE, None, None, FAKE, 0.1, 1, 1, 1, 64, 64, 64, 0, 0,
              FAKE, 1 << 20, None) == 2
    MX = lib.da_decode_merge_ex
    assert MX(FAKE, None, 1, 1, 1, 64, 64, 64, 1, 100, FAKE, 1 << 20, None) == 2
    assert MX(FAKE, None, 1, 1, 1, 64, 64, 64, 4097, 0, FAKE, 1 << 20, None) == 2


def test_workspace_reset_validation():
    R = lib.da_decode_workspace_reset
    nc = binding.workspace_counter_bytes(2, 8, 2, 1000, 128, 128)
    assert R(None, 1 << 20, 2, 8, 2, 1000, 128, 128, None) == 1
    assert R(FAKE, 1 << 20, 2, 3, 2, 1000, 128, 128, None) == 2
    assert R(FAKE, 1 << 20, 2, 8, 2, 1000, 96, 128, None) == 3
    assert R(FAKE, nc - 16, 2, 8, 2, 1000, 128, 128, None) == 6
    assert R(FAKE + 4, 1 << 20, 2, 8, 2, 1000, 128, 128, None) == 4


def test_step_validation():
    S = lib.da_decode_step
    args = [FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0.1, FAKE, 1, 1, 1, 64, 64, 64,
            FAKE, 1 << 20, None]
    for pos in (0, 1, 2, 3, 4, 5, 7):
        a = list(args); a[pos] = None
        assert S(*a) == 1, pos
    for pos in (3, 4, 7):
        a = list(args); a[pos] = FAKE + 4
        assert S(*a) == 4, pos
    a = list(args); a[15] = 8
    assert S(*a) == 6
    a = list(args); a[6] = float("nan")
    assert S(*a) == 5
    a = list(args); a[9] = 3; a[10] = 2
    assert S(*a) == 2
    a = list(args); a[12] = 96
    assert S(*a) == 3


def test_multi_row_validation():
    D = lib.da_decode_multi
    base = [FAKE, FAKE, FAKE, FAKE, 0.1, FAKE, 1, 2, 1, 64, 64, 64, 4, FAKE, 1 << 20, None]
    for pos in (0, 1, 2, 3, 5):
        a = list(base); a[pos] = None
        assert D(*a) == 1, pos
    for T in (0, -1, 4097):
        a = list(base); a[12] = T
        assert D(*a) == 2, T
    a = list(base); a[14] = 16
    assert D(*a) == 6
    a = list(base); a[5] = FAKE + 4
    assert D(*a) == 4
    S = lib.da_decode_multi_step
    sb = [FAKE] * 6 + [0.1, FAKE, 1, 2, 1, 64, 64, 64, 4, FAKE, 1 << 20, None]
    for pos in (3, 4, 5, 7):
        a = list(sb); a[pos] = None
        assert S(*a) == 1, pos
    a = list(sb); a[14] = 0
    assert S(*a) == 2
    R = lib.da_kv_append_rows
    rb = [FAKE] * 5 + [1, 1, 8, 64, 64, 3, None]
    assert R(*rb[:4], None, *rb[5:]) == 1
    for T in (0, 4097):
        a = list(rb); a[10] = T
        assert R(*a) == 2, T
    a = list(rb); a[8] = 62
    assert R(*a) == 3
    a = list(rb); a[2] = FAKE + 4
    assert R(*a) == 4
    # the workspace of a T-row decode is that of h_q*T query heads
    assert binding.workspace_bytes(2, 8 * 4, 2, 1000, 128, 128) > binding.workspace_bytes(
        2, 8, 2, 1000, 128, 128)


@pytest.mark.parametrize("args,status", [
    ((None, FAKE, FAKE, FAKE, FAKE, 1, 1, 8, 64, 64), 1),
    ((FAKE, FAKE, FAKE, FAKE, None, 1, 1, 8, 64, 64), 1),
    ((FAKE, FAKE, FAKE, FAKE, FAKE, 0, 1, 8, 64, 64), 2),
    ((FAKE, FAKE, FAKE, FAKE, FAKE, 1, 1, 0, 64, 64), 2),
    ((FAKE, FAKE, FAKE, FAKE, FAKE, 1, 1, 8, 62, 64), 3),
    ((FAKE, FAKE + 4, FAKE, FAKE, FAKE, 1, 1, 8, 64, 64), 4),
    ((FAKE, FAKE, FAKE, FAKE + 8, FAKE, 1, 1, 8, 64, 64), 4),
])
def test_append_validation(args, status):
    assert lib.da_kv_append(*args, None) == status


def test_noalloc_validation():
    """The no-allocation decode validates like da_decode_attn and rejects
    shapes whose workspace exceeds its 64 MiB array, all on the host."""
    N = lib.da_decode_attn_noalloc
    args = [FAKE, FAKE, FAKE, FAKE, 0.125, FAKE, 4, 64, 8, 131072, 128, 128, None]
    for pos in (0, 1, 2, 3, 5):
        a = list(args); a[pos] = None
        assert N(*a) == 1, pos
    a = list(args); a[7] = 7
    assert N(*a) == 2
    a = list(args); a[10] = 96
    assert N(*a) == 3
    a = list(args); a[0] = FAKE + 4
    assert N(*a) == 4
    a = list(args); a[4] = float("nan")
    assert N(*a) == 5
    big = [FAKE, FAKE, FAKE, FAKE, 0.125, FAKE, 128, 32, 8, 32768, 128, 128, None]
    assert binding.workspace_bytes(*big[6:12]) > binding.NOALLOC_MAX_WORKSPACE_BYTES
    assert N(*big) == 6
    assert binding.workspace_bytes(4, 64, 8, 131072, 128, 128) <= \
        binding.NOALLOC_MAX_WORKSPACE_BYTES


def test_binding_fails_loudly_without_the_library(tmp_path):
    env = dict(os.environ, DECODE_ATTN_LIB=str(tmp_path / "missing.so"))
    code = ("import paper_2607_19456_amd as p\n"
            "try:\n    p.decode_attn\nexcept ImportError as e:\n    print('IMPORTERROR', e)\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=120)
    assert "IMPORTERROR" in r.stdout and "no CPU fallback" in r.stdout


def test_product_path_does_not_reference_the_oracle():
    pkg = os.path.join(ROOT, "paper_2607_19456_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".c", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f
                assert "liboracle" not in text, f


def test_read_probe_library_loads_and_validates():
    """The read-ceiling probe the benchmark uses: its library loads, and bad
    arguments are rejected on the host (no launch)."""
    from paper_2607_19456_amd import hbm_probe
    p = hbm_probe._lib
    assert p.hbm_probe_threads() == 256
    assert p.hbm_read_probe(FAKE, 16, FAKE, 16, None, 1, None) == 1      # no output
    assert p.hbm_read_probe(None, 16, FAKE, 16, FAKE, 1, None) == 1      # NULL input
    assert p.hbm_read_probe(FAKE + 4, 16, FAKE, 16, FAKE, 1, None) == 1  # misaligned
    assert p.hbm_read_probe(FAKE, 20, FAKE, 16, FAKE, 1, None) == 2      # size not 16k
    assert p.hbm_read_probe(FAKE, 16, FAKE, 16, FAKE, 0, None) == 2      # no workgroups
