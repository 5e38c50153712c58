"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every symbol include/kmip.h declares, sizes its workspace, and rejects bad
arguments before touching the device."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

kmip = pytest.importorskip("paper_2604_03815_amd")
from paper_2604_03815_amd import _lib  # noqa: E402


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2604_03815_amd import build
        build.build()
    return _lib.load()


def _declared_symbols():
    with open(os.path.join(ROOT, "include", "kmip.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kmip_[a-z_]+)\s*\(", text)))


def test_header_matches_binding():
    assert sorted(_lib.EXPORTS) == _declared_symbols()


def test_all_declared_symbols_exported(lib):
    for name in _declared_symbols():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for s in range(5):
        assert lib.kmip_status_string(s)
    assert lib.kmip_status_string(99) == b"unknown status"


def test_workspace_size(lib):
    # tiled copy of K, padded to whole 32-key tiles, 256-byte aligned
    n = lib.kmip_topk_workspace_size(500_000, 4, 16, 32, 1)
    packed = 4 * (15625 + 16) * 32 * 16 * 2 + 512   # tiled K, then 512 B of work counters
    # one graph of >= 8192 nodes: query grouping adds reference directions
    # [H][256][d] bf16, labels [H][N] u16, a histogram and the seed references
    # [2][H][256] i32 and the permutation [H][N] i32, each 256-byte aligned
    grouping = 4 * 256 * 16 * 2 + 4 * 500_000 * 2 + 2 * 4 * 256 * 4 + 4 * 500_000 * 4
    # ... and the stored key order: two position buffers [H][N] i32, two
    # head-major copies of the key rows in that order [H][N][d] bf16, projection
    # codes [H][N] u16, per-node data of the widest tree level (1954
    # superblocks -> 11 levels, 1024 nodes) [H][1024][2d + 2] f32 and
    # [H][1024][520] i32, votes [2H] i32 (padded to 256 B), the bound tiles:
    # 1954 superblocks of 256 keys -> 31 windows of 64 -> 62 tiles per head of
    # (d/16 + 1) chunks of 64 x 16 B, and the window tiles: 31 windows -> one
    # pair of tiles per head
    key_order = (2 * 4 * 500_000 * 4 + 2 * 4 * 500_000 * 16 * 2 + 4 * 500_000 * 2 + 4 * 1024 * 34 * 4
                 + 4 * 1024 * 520 * 4
                 + 256 + 4 * 62 * 2 * 64 * 16 + 4 * 2 * 2 * 64 * 16)
    assert n == packed + grouping + key_order
    assert lib.kmip_topk_workspace_size(8191, 1, 16, 4, 1) == (256 + 16) * 32 * 16 * 2 + 512
    assert lib.kmip_topk_workspace_size(33, 1, 16, 4, 1) == (2 + 16) * 32 * 16 * 2 + 512
    multi = lib.kmip_topk_workspace_size(1000, 2, 32, 16, 7)
    assert multi > lib.kmip_topk_workspace_size(1000, 2, 32, 16, 1)
    assert lib.kmip_topk_workspace_size(100, 1, 24, 4, 1) == 0   # unsupported d
    assert lib.kmip_topk_workspace_size(-1, 1, 16, 4, 1) == 0
    assert lib.kmip_fwd_workspace_size(1000, 2, 32, 16, 1) == lib.kmip_topk_workspace_size(1000, 2, 32, 16, 1)
    # backward: per-pair atomics need none; key aggregation groups the queries
    # (reference directions in bf16, labels, histogram + seed slots, permutation)
    assert lib.kmip_bwd_workspace_size(1000, 2, 32, 16, 1) == 0
    agg = 2 * 256 * 32 * 2 + 4096 + 2 * 2 * 256 * 4 + 8192
    assert lib.kmip_bwd_workspace_size(1000, 2, 32, 16, _lib.BWD_KEY_AGGREGATED) == agg
    # the segmented reduction: pair coefficients (2 f32), the key-sorted pair
    # records (16 B), per-key counts and the scan's block sums, each 256-byte
    # aligned
    csr = 32000 * 8 + 32000 * 16 + 8192 + 256
    assert lib.kmip_bwd_workspace_size(1000, 2, 32, 16, _lib.BWD_SEGMENTED) == csr
    # the bucketed reduction: the bucket-sorted records (12 B: packed
    # key-row offset and query row, then the coefficients),
    # three arrays over the 2000 / (4096 / 32) = 16 key-row buckets (+1:
    # counts, kept starts, pieces), the scan's block sums and the head-major
    # interleaved copy of Q and dO (bf16, 2d per query-head)
    # ... and the records in super-bucket order between the two placement
    # passes (16 B), with three arrays of 65 super-bucket entries
    # ... and the grouping of the queries by direction, the order in which the
    # coefficient pass takes them (the key-aggregated variant's workspace)
    bucket = 32000 * 12 + 3 * 256 + 256 + 2 * 2000 * 32 * 2 + 32000 * 16 + 3 * 512 + agg
    assert lib.kmip_bwd_workspace_size(1000, 2, 32, 16, _lib.BWD_BUCKETED) == bucket
    # the library picks the bucketed reduction where it fits
    assert lib.kmip_bwd_workspace_size(1000, 2, 32, 16, 0) == bucket
    # buckets widen up to 512 key rows: N*H = 4M still fits 8192 buckets;
    # beyond that the variant is unsupported (size 0) and the library picks
    # the full key sort
    assert lib.kmip_bwd_workspace_size(1_000_000, 4, 16, 16, _lib.BWD_BUCKETED) > 0
    assert lib.kmip_bwd_workspace_size(1_100_000, 4, 16, 16, _lib.BWD_BUCKETED) == 0
    assert (lib.kmip_bwd_workspace_size(1_100_000, 4, 16, 16, 0)
            == lib.kmip_bwd_workspace_size(1_100_000, 4, 16, 16, _lib.BWD_SEGMENTED) > 0)
    assert lib.kmip_bwd_workspace_size(1000, 2, 32, 16, 5) == 0
    # k > 128 and d = 128: the bucketed reduction is not built for them, the
    # library picks the key sort
    # (the key sort's arrays as above: 2000 k pairs of 8 + 16 B, each array
    # rounded up to 256 B, 8192 B of counts and 256 B of block sums)
    def al(x):
        return (x + 255) // 256 * 256

    for d, k in ((16, 129), (64, 512), (128, 16)):
        csr_k = al(2000 * k * 8) + al(2000 * k * 16) + 8192 + 256
        assert lib.kmip_bwd_workspace_size(1000, 2, d, k, _lib.BWD_BUCKETED) == 0
        assert lib.kmip_bwd_workspace_size(1000, 2, d, k, _lib.BWD_SEGMENTED) == csr_k
        assert lib.kmip_bwd_workspace_size(1000, 2, d, k, 0) == csr_k
    assert lib.kmip_bwd_ex_workspace_size(1000, 2, 128, 64, 128, _lib.BWD_SEGMENTED) > 0
    assert lib.kmip_bwd_ex_workspace_size(1000, 2, 128, 256, 16, _lib.BWD_SEGMENTED) == 0
    # one graph of d = 128 is not grouped: tiles of K and the counters only
    assert lib.kmip_topk_workspace_size(20000, 1, 128, 16, 1) == (625 + 16) * 32 * 128 * 2 + 512
    assert lib.kmip_topk_workspace_size(100, 1, 128, 129, 1) == 0
    assert lib.kmip_topk_workspace_size(100, 1, 64, 512, 1) > 0
    assert lib.kmip_topk_workspace_size(100, 1, 64, 513, 1) == 0


P = ctypes.c_void_p
FAKE = P(256)  # never dereferenced: every call below fails validation first


def _topk(lib, N=64, H=1, d=16, k=4, offsets=None, G=1, ws=FAKE, ws_bytes=1 << 20, q=FAKE):
    optr = None if offsets is None else np.ascontiguousarray(offsets, np.int32).ctypes.data_as(P)
    return lib.kmip_topk(q, FAKE, optr, G, N, H, d, k, FAKE, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(N=-1), 1), (dict(H=0), 1), (dict(k=0), 1), (dict(d=24), 2), (dict(d=256), 2), (dict(k=513), 2),
    (dict(d=128, k=129), 2),
    (dict(N=1 << 31), 1), (dict(N=1 << 28, H=8, d=16), 1),
    (dict(offsets=[1, 64], G=1), 1), (dict(offsets=[0, 40, 30, 64], G=3), 1),
    (dict(offsets=[0, 32, 63], G=2), 1), (dict(offsets=[0, 64], G=0), 1),
    (dict(ws=None), 3), (dict(ws_bytes=10), 3), (dict(ws=P(256 + 16)), 3),
    (dict(q=None), 1), (dict(q=P(258)), 1),
])
def test_topk_rejects(lib, kw, status):
    assert _topk(lib, **kw) == status
    assert lib.kmip_last_error()


def test_zero_nodes_is_a_no_op(lib):
    assert lib.kmip_topk(None, None, None, 1, 0, 1, 16, 4, None, None, 0, None) == 0
    assert lib.kmip_attend(None, None, None, 0, 1, 16, 4, ctypes.c_float(1.0), None, None, None, None) == 0


def test_attend_rejects(lib):
    f = ctypes.c_float
    assert lib.kmip_attend(FAKE, FAKE, FAKE, 64, 1, 16, 4, f(0.0), FAKE, FAKE, FAKE, None) == 1
    assert lib.kmip_attend(FAKE, FAKE, FAKE, 64, 1, 16, 4, f(float("nan")), FAKE, FAKE, FAKE, None) == 1
    assert lib.kmip_attend(FAKE, FAKE, FAKE, 64, 1, 16, 4, f(float("inf")), FAKE, FAKE, FAKE, None) == 1
    assert lib.kmip_attend(FAKE, FAKE, None, 64, 1, 16, 4, f(1.0), FAKE, FAKE, FAKE, None) == 1
    assert lib.kmip_attend(FAKE, FAKE, FAKE, 64, 1, 48, 4, f(1.0), FAKE, FAKE, FAKE, None) == 2


def test_bwd_rejects(lib):
    f = ctypes.c_float
    args = [FAKE] * 6 + [64, 1, 16, 4, f(1.0), FAKE, FAKE, FAKE]
    assert lib.kmip_bwd(*args, 7, None, 0, None) == 2            # unknown variant
    assert lib.kmip_bwd(*args, _lib.BWD_SEGMENTED, None, 0, None) == 3        # needs workspace
    assert lib.kmip_bwd(*args, _lib.BWD_KEY_AGGREGATED, None, 0, None) == 3   # needs workspace
    assert lib.kmip_bwd(*args, _lib.BWD_BUCKETED, None, 0, None) == 3         # needs workspace
    assert lib.kmip_bwd(*args, 0, FAKE, 16, None) == 3           # workspace too small
    bad = list(args)
    bad[3] = None                                                 # dOut
    assert lib.kmip_bwd(*bad, 0, None, 0, None) == 1
    bad = list(args)
    bad[10] = f(-2.0)
    assert lib.kmip_bwd(*bad, 0, None, 0, None) == 1


def test_fwd_validates_before_launch(lib):
    f = ctypes.c_float
    assert lib.kmip_fwd(FAKE, FAKE, None, None, 1, 64, 1, 16, 4, f(1.0), FAKE, FAKE, FAKE,
                        FAKE, 1 << 20, None) == 1
    assert lib.kmip_fwd(FAKE, FAKE, FAKE, None, 1, 64, 1, 16, 4, f(-1.0), FAKE, FAKE, FAKE,
                        FAKE, 1 << 20, None) == 1


def _prototypes():
    """{function name: [parameter names]} of every prototype in include/kmip.h."""
    with open(os.path.join(ROOT, "include", "kmip.h")) as f:
        text = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
    protos = {}
    for m in re.finditer(r"\b(kmip_[a-z_]+)\s*\(([^)]*)\)\s*;", text):
        params = [p.strip() for p in m.group(2).split(",") if p.strip() and p.strip() != "void"]
        protos[m.group(1)] = [re.findall(r"[A-Za-z_][A-Za-z_0-9]*", p)[-1] for p in params]
    return protos


def test_bwd_signature_as_documented():
    # kmip_bwd takes (inputs, saved tensors, sizes, scale, outputs, variant,
    # workspace, stream); the forward's graph_offsets and out are not
    # parameters (the header states why).
    assert _prototypes()["kmip_bwd"] == [
        "Q", "K", "V", "dOut", "topk_idx", "lse", "N", "H", "d", "k", "scale", "dQ", "dK", "dV",
        "variant", "workspace", "workspace_bytes", "stream"]


def test_bwd_variant_codes_as_documented():
    with open(os.path.join(ROOT, "include", "kmip.h")) as f:
        text = f.read()
    codes = dict((n, int(v)) for n, v in re.findall(r"\b(KMIP_BWD_[A-Z_]+)\s*=\s*(\d+)", text))
    assert codes == {"KMIP_BWD_AUTO": 0, "KMIP_BWD_ATOMIC": 1, "KMIP_BWD_SEGMENTED": 2,
                     "KMIP_BWD_BUCKETED": 3, "KMIP_BWD_KEY_AGGREGATED": 4}
    assert (_lib.BWD_AUTO, _lib.BWD_ATOMIC, _lib.BWD_SEGMENTED, _lib.BWD_BUCKETED,
            _lib.BWD_KEY_AGGREGATED) == (0, 1, 2, 3, 4)


def test_binding_argument_counts_match_header(lib):
    for name, params in _prototypes().items():
        argtypes = getattr(lib, name).argtypes
        assert argtypes is not None and len(argtypes) == len(params), name


def test_noalloc_scratch_size_matches_header():
    with open(os.path.join(ROOT, "include", "kmip.h")) as f:
        m = re.search(r"#define KMIP_NOALLOC_SCRATCH_BYTES \((\d+)u \* (\d+)u \* (\d+)u\)", f.read())
    assert m and int(m.group(1)) * int(m.group(2)) * int(m.group(3)) == _lib.NOALLOC_SCRATCH_BYTES


def test_noalloc_validates_before_launch(lib):
    f = ctypes.c_float
    # sizes whose working data exceed the fixed array: rejected with a clear
    # error before any HIP call (this host has no GPU)
    assert lib.kmip_fwd_noalloc(FAKE, FAKE, FAKE, 1_000_000, 4, 16, 32, f(0.25), FAKE, FAKE, FAKE, None) == 2
    assert b"scratch" in lib.kmip_last_error()
    assert lib.kmip_fwd_workspace_size(1_000_000, 4, 16, 32, 1) > _lib.NOALLOC_SCRATCH_BYTES
    # the benchmark's workload fits
    assert 0 < lib.kmip_fwd_workspace_size(500_000, 4, 16, 32, 1) <= _lib.NOALLOC_SCRATCH_BYTES
    # argument errors come first
    assert lib.kmip_fwd_noalloc(FAKE, FAKE, None, 64, 1, 16, 4, f(1.0), FAKE, FAKE, FAKE, None) == 1
    assert lib.kmip_fwd_noalloc(FAKE, FAKE, FAKE, 64, 1, 16, 4, f(-1.0), FAKE, FAKE, FAKE, None) == 1
    assert lib.kmip_fwd_noalloc(FAKE, FAKE, FAKE, 64, 1, 24, 4, f(1.0), FAKE, FAKE, FAKE, None) == 2
    assert lib.kmip_fwd_noalloc(P(258), FAKE, FAKE, 64, 1, 16, 4, f(1.0), FAKE, FAKE, FAKE, None) == 1
    # nothing to do
    assert lib.kmip_fwd_noalloc(None, None, None, 0, 1, 16, 4, f(1.0), None, None, None, None) == 0


def test_extended_entry_points_validate(lib):
    f = ctypes.c_float
    # value widths outside {16, 32, 64}
    assert lib.kmip_attend_ex(FAKE, FAKE, FAKE, 64, 1, 16, 48, 4, f(1.0), FAKE, None, f(0.0), FAKE, FAKE,
                              None) == 2
    assert lib.kmip_fwd_ex(FAKE, FAKE, FAKE, None, 1, 64, 1, 16, 8, 4, f(1.0), None, f(0.0), FAKE, FAKE, FAKE,
                           FAKE, 1 << 20, None) == 2
    args = [FAKE] * 6
    sizes = [64, 1, 32, 16, 4, f(1.0), FAKE, FAKE, FAKE]
    # the bucketed variant needs d_V == d_K; the others take any pair
    assert lib.kmip_bwd_ex(*args, None, f(0.0), *sizes, _lib.BWD_BUCKETED, FAKE, 1 << 30, None) == 2
    assert lib.kmip_bwd_ex_workspace_size(64, 1, 32, 16, 4, _lib.BWD_BUCKETED) == 0
    assert lib.kmip_bwd_ex_workspace_size(64, 1, 32, 16, 4, _lib.BWD_AUTO) == \
        lib.kmip_bwd_ex_workspace_size(64, 1, 32, 16, 4, _lib.BWD_SEGMENTED) > 0
    assert lib.kmip_bwd_ex(*args, None, f(0.0), *sizes, _lib.BWD_SEGMENTED, None, 0, None) == 3
    # d_V = d_K: the plain entry points are this case
    for v in (0, 1, 2, 3, 4):
        assert lib.kmip_bwd_ex_workspace_size(5000, 2, 32, 32, 16, v) == lib.kmip_bwd_workspace_size(5000, 2, 32, 16, v)
    assert lib.kmip_attend_ex(FAKE, FAKE, FAKE, 64, 1, 16, 32, 4, f(-1.0), FAKE, None, f(0.0), FAKE, FAKE,
                              None) == 1
    # dropout: a rate in [0, 1), and keep draws for a rate above 0
    for rate, keep in ((1.0, FAKE), (-0.1, FAKE), (float("nan"), FAKE), (0.5, None)):
        assert lib.kmip_attend_ex(FAKE, FAKE, FAKE, 64, 1, 16, 16, 4, f(1.0), FAKE, keep, f(rate), FAKE, FAKE,
                                  None) == 1
        assert lib.kmip_bwd_ex(*args, keep, f(rate), 64, 1, 16, 16, 4, f(1.0), FAKE, FAKE, FAKE, 0, None, 0,
                               None) == 1


def test_prefilter_sizes_and_rejects(lib):
    # the select's tiles and counters, then the int8 tiles (H x (ceil(N/32)
    # + 16) tiles of ceil(d/32) 1 KB chunks), 4 words a head, 1024 candidates
    # and 2 lengths per query-head, a flag per (head, block), the redo count
    # and one task per block, each rounded up to 256 bytes
    def al(x):
        return (x + 255) // 256 * 256

    N, H, d, k = 1000, 2, 32, 16
    nb = 32
    want = (al(H * (nb + 16) * 32 * d * 2) + 512 + al(H * (nb + 16) * 1024) + 256 + al(N * H * 1024 * 4)
            + al(N * H * 2 * 4) + al(H * nb * 4) + 256 + al(nb * 16))
    assert lib.kmip_topk_prefilter_workspace_size(N, H, d, k) == want
    assert lib.kmip_topk_prefilter_workspace_size(N, H, d, 33) == 0      # k <= 32 only
    assert lib.kmip_topk_prefilter_workspace_size(N, H, 24, 16) == 0     # unsupported d
    assert lib.kmip_topk_prefilter(FAKE, FAKE, 64, 1, 16, 33, FAKE, None, FAKE, 1 << 30, None) == 2
    assert lib.kmip_topk_prefilter(FAKE, FAKE, 64, 1, 16, 8, FAKE, None, FAKE, 10, None) == 3
    assert lib.kmip_topk_prefilter(FAKE, FAKE, 64, 1, 16, 8, FAKE, None, P(256 + 16), 1 << 30, None) == 3
    assert lib.kmip_topk_prefilter(None, FAKE, 64, 1, 16, 8, FAKE, None, FAKE, 1 << 30, None) == 1
    assert lib.kmip_topk_prefilter(None, None, 0, 1, 16, 8, None, None, None, 0, None) == 0
