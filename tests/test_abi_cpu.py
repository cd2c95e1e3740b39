"""Host-side checks of the C ABI (no GPU needed, nothing is launched).

* libfva.so loads and exports every function include/fva.h declares;
* the host-only queries (block count, workspace sizes, trace size, status
  strings) return the documented values;
* every argument error is reported before any launch, with the documented
  status: the calls below never reach a kernel, so fake device addresses
  are safe.
"""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2607_16190_amd as fva

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "fva.h")
FAKE = ctypes.c_void_p(0x7F0000001000)  # 4 KiB aligned, never dereferenced


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fva_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert "fva_route" in names and "fva_attn" in names
    lib = ctypes.CDLL(fva.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(fva.EXPORTED)


def test_num_blocks():
    assert fva.fva_num_blocks(fva.Tiling(3, 16, 16, 1, 8, 8)) == 12
    assert fva.fva_num_blocks(fva.Tiling(21, 30, 52, 2, 8, 8)) == 308
    assert fva.fva_num_blocks(fva.Tiling(21, 45, 80, 2, 8, 8)) == 660
    assert fva.fva_num_blocks(fva.Tiling(31, 45, 80, 2, 8, 8)) == 960
    assert fva.fva_num_blocks(fva.Tiling(0, 45, 80, 2, 8, 8)) == -1


def desc(B=1, H=40, N=75600, D=128):
    return fva._Desc(B, H, N, D, H * N * D, N * D, D)


T720 = fva.Tiling(21, 45, 80, 2, 8, 8)


def test_workspace_sizes():
    nb = 660
    rows = 40 * nb
    # fp64 means of Q and K, blocks padded to a multiple of 16 (660 -> 672),
    # then the fp64 score rows
    assert fva.fva_route_workspace_size(desc(), T720) == 2 * 40 * 672 * 128 * 8 + 40 * nb * nb * 8
    al = lambda x: (x + 255) // 256 * 256
    heads = 40
    part = 66560  # one chunk's partial result: 128 x 128 fp32 O, 128 references, 128 sums

    def attn_ws(cap, pairs=0):
        # counts, kept lists, queue items (rows + chunks), 9 queue bases, 8 queue
        # counters, per-head plan scratch, per-row prefixes, split count, chunk and
        # split records, partial results, one 32-byte record per block, then the
        # query-block pairs' union lists, their lengths, the first block of each
        # pair of a head and the plan's chunk size
        ws = (al(rows * 4) + al(rows * nb * 4) + al((rows + cap) * 4) + al(9 * 4) + al(8 * 4)
              + al(heads * 19 * 4) + al(2 * (rows + 1) * 4) + al(4) + 2 * al(cap * 16) + al(cap * part)
              + al(nb * 32))
        if pairs:
            ws += al(pairs * nb * 4) + al(pairs * 4) + al(pairs // heads * 4) + al(4)
        return ws

    # 720p: the 60 blocks of the last (one-frame) t-row hold 64 or 40 tokens,
    # 6 lines of 10 blocks, so 5 x-pairs per line and 30 per head
    pairs = heads * 30
    assert fva.fva_attn_workspace_size(desc(), T720) == attn_ws(2048, pairs)
    assert fva.fva_attn_workspace_size(desc(), T720, fva.FVA_SCHED_UNPAIRED) == attn_ws(2048)
    assert fva.fva_attn_workspace_size(desc(), T720, fva.FVA_SCHED_NAIVE) == attn_ws(0)
    assert fva.fva_attn_workspace_size(desc(), T720, fva.FVA_SPLIT_BLOCKS(200)) == attn_ws(rows * 4, pairs)
    assert fva.fva_trace_words(desc(), T720) == (rows + 2048) * 4


def _pairs_by_definition(T, H, W, bt, bh, bw):
    """Query-block pairs of one head, counted block by block: x-neighbours
    (ix even, ix + 1) of one (t, y) line, both holding <= 64 tokens; then,
    among the blocks no x-pair holds, y-neighbours (iy even, iy + 1) of one
    (t, x) column, both holding <= 64 tokens."""
    from oracle import tile_geometry

    geo = tile_geometry(T, H, W, bt, bh, bw)
    n = geo.block_sizes.reshape(geo.nbt, geo.nby, geo.nbx)
    taken = np.zeros(n.shape, bool)
    count = 0
    for t in range(geo.nbt):
        for y in range(geo.nby):
            for x in range(0, geo.nbx - 1, 2):
                if n[t, y, x] <= 64 and n[t, y, x + 1] <= 64:
                    taken[t, y, x] = taken[t, y, x + 1] = True
                    count += 1
    for t in range(geo.nbt):
        for x in range(geo.nbx):
            for y in range(0, geo.nby - 1, 2):
                if not taken[t, y, x] and not taken[t, y + 1, x] and n[t, y, x] <= 64 and n[t, y + 1, x] <= 64:
                    count += 1
    return count


@pytest.mark.parametrize(
    "grid,tile,expect",
    [
        ((21, 45, 80), (2, 8, 8), 30),      # 720p: the one-frame last t-row
        ((31, 45, 80), (2, 8, 8), 30),      # long clip
        ((21, 30, 52), (2, 8, 8), 34),      # 480p: 12 x-pairs, 22 y-pairs of the 4-token-wide column
        ((3, 16, 16), (1, 8, 8), 6),        # 64-token boxes: every line pairs
        ((5, 17, 23), (1, 8, 8), None),     # odd block counts per line
        ((9, 20, 40), (2, 4, 8), None),     # 64-token boxes of another shape
        ((1, 1, 60000), (1, 1, 64), 469),   # curve blocks of 64 tokens (the last holds 32)
        ((1, 1, 75600), (1, 1, 128), 0),    # curve blocks of 128: none
    ],
)
def test_pair_count_matches_definition(grid, tile, expect):
    T, H, W = grid
    want = _pairs_by_definition(T, H, W, *tile)
    if expect is not None:
        assert want == expect
    heads = 3
    d = fva._Desc(1, heads, T * H * W, 128, heads * T * H * W * 128, T * H * W * 128, 128)
    t = fva.Tiling(T, H, W, *tile)
    nb = fva.fva_num_blocks(t)
    al = lambda x: (x + 255) // 256 * 256
    extra = fva.fva_attn_workspace_size(d, t) - fva.fva_attn_workspace_size(d, t, fva.FVA_SCHED_UNPAIRED)
    P = heads * want
    assert extra == ((al(P * nb * 4) + al(P * 4) + al(want * 4) + al(4)) if P else 0)


@pytest.mark.parametrize(
    "d,t,status",
    [
        (desc(N=75601), T720, fva.FVA_ERR_SHAPE),
        (desc(D=64), T720, fva.FVA_ERR_UNSUPPORTED),
        (desc(N=21 * 45 * 80), fva.Tiling(21, 45, 80, 1, 4, 4), fva.FVA_ERR_UNSUPPORTED),  # tile volume 16
        (desc(N=64 * 64 * 64), fva.Tiling(64, 64, 64, 2, 8, 8), fva.FVA_ERR_UNSUPPORTED),  # nb > 1024
        (desc(), fva.Tiling(21, 45, 80, 0, 8, 8), fva.FVA_ERR_SHAPE),
    ],
)
def test_shape_errors(d, t, status):
    with pytest.raises(fva.FvaError) as e:
        fva.fva_route_workspace_size(d, t)
    assert e.value.status == status


def _route(p=0.9, k_min=4, d=None, t=T720, q=FAKE, ws=FAKE, wsb=1 << 40, mask=FAKE, counts=FAKE):
    d = d or desc()
    return fva.lib.fva_route(q, FAKE, ctypes.byref(d), p, k_min, ctypes.byref(t.c()), mask, counts, None, ws,
                             ctypes.c_size_t(wsb), None)


def test_route_argument_errors():
    assert _route(p=float("nan")) == fva.FVA_ERR_INVALID_ARG
    assert _route(p=-0.01) == fva.FVA_ERR_INVALID_ARG
    assert _route(p=1.5) == fva.FVA_ERR_INVALID_ARG
    assert _route(k_min=-1) == fva.FVA_ERR_INVALID_ARG
    assert _route(q=None) == fva.FVA_ERR_INVALID_ARG
    assert _route(mask=None) == fva.FVA_ERR_INVALID_ARG
    assert _route(counts=None) == fva.FVA_ERR_INVALID_ARG
    assert _route(q=ctypes.c_void_p(0x7F0000001002)) == fva.FVA_ERR_INVALID_ARG  # misaligned rows
    assert _route(ws=None) == fva.FVA_ERR_WORKSPACE
    assert _route(wsb=100) == fva.FVA_ERR_WORKSPACE
    assert _route(ws=ctypes.c_void_p(0x7F0000001080)) == fva.FVA_ERR_WORKSPACE  # not 256-aligned
    assert _route(d=desc(N=10)) == fva.FVA_ERR_SHAPE
    bad = desc()
    bad.stride_n = 100  # rows overlap and are not 16-byte aligned
    assert _route(d=bad) == fva.FVA_ERR_SHAPE
    assert _route(d=desc(B=2, H=40000)) == fva.FVA_ERR_UNSUPPORTED  # more than 65535 heads in all


def _attn(flags=0, counts=None, kv=None, mask=FAKE, trace=None, scale=0.0, ws=FAKE, wsb=1 << 40, o=FAKE):
    d = desc()
    return fva.lib.fva_attn(FAKE, FAKE, FAKE, ctypes.byref(d), ctypes.byref(T720.c()), mask, counts, kv,
                            ctypes.c_float(scale), flags, o, ws, ctypes.c_size_t(wsb), trace, None)


def test_attn_argument_errors():
    assert _attn(flags=8) == fva.FVA_ERR_INVALID_ARG
    assert _attn(flags=1 << 24) == fva.FVA_ERR_INVALID_ARG  # beyond the chunk-size field
    assert _attn(counts=FAKE, kv=None) == fva.FVA_ERR_INVALID_ARG
    assert _attn(counts=None, kv=FAKE) == fva.FVA_ERR_INVALID_ARG
    assert _attn(mask=None) == fva.FVA_ERR_INVALID_ARG
    assert _attn(flags=fva.FVA_TRACE, trace=None) == fva.FVA_ERR_INVALID_ARG
    assert _attn(scale=float("nan")) == fva.FVA_ERR_INVALID_ARG
    assert _attn(o=None) == fva.FVA_ERR_INVALID_ARG
    assert _attn(wsb=10) == fva.FVA_ERR_WORKSPACE


def test_attn_rejects_work_item_overflow():
    # batch * heads * nb must leave room for the chunk items below 2^31
    # (32-bit work-item indices): rejected on the host, before any launch.
    big = desc(B=1024, H=3200)  # 3,276,800 heads x 660 blocks = 2.16e9 rows
    for flags in (0, fva.FVA_SCHED_NAIVE, fva.FVA_SPLIT_BLOCKS(4)):
        st = fva.lib.fva_attn(FAKE, FAKE, FAKE, ctypes.byref(big), ctypes.byref(T720.c()), FAKE, None, None,
                              ctypes.c_float(0.0), flags, FAKE, FAKE, ctypes.c_size_t(1 << 62), None, None)
        assert st == fva.FVA_ERR_UNSUPPORTED, flags
        with pytest.raises(fva.FvaError) as e:
            fva.fva_attn_workspace_size(big, T720, flags)
        assert e.value.status == fva.FVA_ERR_UNSUPPORTED
    assert fva.lib.fva_trace_words(ctypes.byref(big), ctypes.byref(T720.c())) == -1
    # just inside the limit with the automatic chunk size, outside with forced splits
    n_ok = (2**31 - 1 - 2048) // 660
    ok = desc(B=1, H=n_ok)
    assert fva.fva_attn_workspace_size(ok, T720) > 0
    with pytest.raises(fva.FvaError):
        fva.fva_attn_workspace_size(ok, T720, fva.FVA_SPLIT_BLOCKS(4))
    assert fva.fva_attn_workspace_size(desc(B=1, H=n_ok + 4), T720, fva.FVA_SCHED_NAIVE) > 0


def test_curve_workspace_sizes():
    al = lambda x: (x + 255) // 256 * 256
    # 8^k-bit bitmap and its word prefixes (max(1, 8^k / 32) words each), one index per token
    for (T, H, W), k in (((21, 45, 80), 7), ((3, 16, 16), 4), ((1, 1, 1), 0), ((2, 2, 1), 1), ((1, 256, 3), 8)):
        words = max(1, 8**k // 32)
        assert fva.fva_curve_workspace_size(T, H, W) == 2 * al(words * 4) + al(T * H * W * 4)
    for grid, status in (((0, 4, 4), fva.FVA_ERR_SHAPE), ((4, -1, 4), fva.FVA_ERR_SHAPE),
                         ((257, 4, 4), fva.FVA_ERR_UNSUPPORTED), ((4, 4, 300), fva.FVA_ERR_UNSUPPORTED)):
        with pytest.raises(fva.FvaError) as e:
            fva.fva_curve_workspace_size(*grid)
        assert e.value.status == status


def test_curve_argument_errors():
    L = fva.lib
    assert L.fva_curve_order(21, 45, 80, None, FAKE, ctypes.c_size_t(1 << 30), None) == fva.FVA_ERR_INVALID_ARG
    assert L.fva_curve_order(21, 45, 80, FAKE, None, ctypes.c_size_t(1 << 30), None) == fva.FVA_ERR_WORKSPACE
    assert L.fva_curve_order(21, 45, 80, FAKE, FAKE, ctypes.c_size_t(1000), None) == fva.FVA_ERR_WORKSPACE
    assert L.fva_curve_order(21, 45, 0, FAKE, FAKE, ctypes.c_size_t(1 << 30), None) == fva.FVA_ERR_SHAPE
    assert L.fva_curve_order(300, 45, 8, FAKE, FAKE, ctypes.c_size_t(1 << 30), None) == fva.FVA_ERR_UNSUPPORTED
    other = ctypes.c_void_p(0x7F0000100000)
    d = desc()
    P = lambda src=FAKE, dst=other, dd=d, perm=FAKE, direction=fva.FVA_TO_CURVE: L.fva_permute_tokens(
        src, dst, ctypes.byref(dd) if dd is not None else None, perm, direction, None)
    assert P(src=None) == fva.FVA_ERR_INVALID_ARG
    assert P(perm=None) == fva.FVA_ERR_INVALID_ARG
    assert P(dd=None) == fva.FVA_ERR_INVALID_ARG
    assert P(dst=FAKE) == fva.FVA_ERR_INVALID_ARG  # in place
    assert P(direction=2) == fva.FVA_ERR_INVALID_ARG
    assert P(dst=ctypes.c_void_p(0x7F0000100008)) == fva.FVA_ERR_INVALID_ARG  # not 16-byte aligned
    assert P(dd=desc(D=64)) == fva.FVA_ERR_UNSUPPORTED
    assert P(dd=desc(N=0)) == fva.FVA_ERR_SHAPE
    bad = desc()
    bad.stride_n = 100
    assert P(dd=bad) == fva.FVA_ERR_SHAPE
    assert P(dd=desc(B=2, H=40000)) == fva.FVA_ERR_UNSUPPORTED  # more than 65535 heads in all


def test_curve_tiling_block_counts():
    assert fva.fva_num_blocks(fva.Tiling.curve(75600, 128)) == 591
    assert fva.fva_num_blocks(fva.Tiling.curve(32760, 128)) == 256
    assert fva.fva_num_blocks(fva.Tiling.curve(768, 64)) == 12
    assert fva.fva_attn_workspace_size(desc(), fva.Tiling.curve(75600, 128)) > 0


def test_fp8_sizes_and_argument_errors():
    d = desc()
    assert fva.fva_v8_size(d, T720) == 40 * 660 * 16384
    assert fva.fva_quantize_v_workspace_size(d, T720) == 40 * 128 * 4
    assert fva.fva_quantize_v_workspace_size(desc(H=3), T720) == 1536  # 3 * 128 * 4 rounded up to 256
    L = fva.lib
    Q = lambda v=FAKE, v8=FAKE, e=FAKE, ws=FAKE, wsb=1 << 30, dd=None: L.fva_quantize_v(
        v, ctypes.byref(dd or d), ctypes.byref(T720.c()), v8, e, ws, ctypes.c_size_t(wsb), None)
    assert Q(v=None) == fva.FVA_ERR_INVALID_ARG
    assert Q(v8=None) == fva.FVA_ERR_INVALID_ARG
    assert Q(e=None) == fva.FVA_ERR_INVALID_ARG
    assert Q(e=ctypes.c_void_p(0x7F0000001002)) == fva.FVA_ERR_INVALID_ARG  # v_exp not 4-byte aligned
    assert Q(v8=ctypes.c_void_p(0x7F0000001008)) == fva.FVA_ERR_INVALID_ARG  # V8 not 16-byte aligned
    assert Q(ws=None) == fva.FVA_ERR_WORKSPACE
    assert Q(wsb=100) == fva.FVA_ERR_WORKSPACE
    assert Q(dd=desc(N=10)) == fva.FVA_ERR_SHAPE
    assert Q(dd=desc(D=64)) == fva.FVA_ERR_UNSUPPORTED
    A = lambda v8=FAKE, e=FAKE, flags=0, wsb=1 << 40: L.fva_attn_fp8v(
        FAKE, FAKE, v8, e, ctypes.byref(d), ctypes.byref(T720.c()), FAKE, None, None, ctypes.c_float(0.0), flags,
        FAKE, FAKE, ctypes.c_size_t(wsb), None, None)
    assert A(v8=None) == fva.FVA_ERR_INVALID_ARG
    assert A(e=None) == fva.FVA_ERR_INVALID_ARG
    assert A(flags=8) == fva.FVA_ERR_INVALID_ARG
    assert A(wsb=10) == fva.FVA_ERR_WORKSPACE
    assert L.fva_attn(FAKE, FAKE, None, ctypes.byref(d), ctypes.byref(T720.c()), FAKE, None, None,
                      ctypes.c_float(0.0), 0, FAKE, FAKE, ctypes.c_size_t(1 << 40), None, None) == fva.FVA_ERR_INVALID_ARG


def test_route_sasa_sizes_and_argument_errors():
    d = desc()
    # 40 int32 extra-block counts, then one 16-byte cut record per routed row (40 x 660)
    assert fva.fva_route_sasa_workspace_size(d, T720) == fva.fva_route_workspace_size(d, T720) + 256 + 40 * 660 * 16
    L = fva.lib
    R = lambda rank_of=FAKE, n=8, n1=0.8, n2=0.07, ws=FAKE, wsb=1 << 40, extra=None: L.fva_route_sasa(
        FAKE, FAKE, ctypes.byref(d), 0.9, 4, ctypes.byref(T720.c()), rank_of, n, n1, n2, FAKE, FAKE, None, extra,
        ws, ctypes.c_size_t(wsb), None)
    assert R(rank_of=None) == fva.FVA_ERR_INVALID_ARG
    assert R(rank_of=ctypes.c_void_p(0x7F0000001002)) == fva.FVA_ERR_INVALID_ARG
    assert R(extra=ctypes.c_void_p(0x7F0000001001)) == fva.FVA_ERR_INVALID_ARG
    assert R(n=0) == fva.FVA_ERR_INVALID_ARG
    assert R(n=1025) == fva.FVA_ERR_INVALID_ARG
    assert R(n1=-0.1) == fva.FVA_ERR_INVALID_ARG
    assert R(n1=1.5) == fva.FVA_ERR_INVALID_ARG
    assert R(n1=float("nan")) == fva.FVA_ERR_INVALID_ARG
    assert R(n2=2.0) == fva.FVA_ERR_INVALID_ARG
    plain = fva.fva_route_workspace_size(d, T720)
    assert R(wsb=plain) == fva.FVA_ERR_WORKSPACE  # the augmentation needs the tail


def test_status_strings():
    assert fva.fva_status_string(0) == "ok"
    for s in (-1, -2, -3, -4, -5):
        assert fva.fva_status_string(s) != "unknown status"
    assert fva.fva_status_string(7) == "unknown status"


def test_host_tensors_are_refused_no_cpu_fallback():
    # Every compute entry point takes device tensors only: host tensors are an
    # error, never a slower path.
    import torch

    t = fva.Tiling(3, 16, 16, 1, 8, 8)
    q = torch.zeros(1, 2, 3 * 16 * 16, 128, dtype=torch.bfloat16)
    mask = torch.ones(1, 2, 12, 12, dtype=torch.uint8)
    with pytest.raises(ValueError):
        fva.fva_route(q, q, 0.9, 2, t)
    with pytest.raises(ValueError):
        fva.fva_attn(q, q, q, t, mask)
    with pytest.raises(ValueError):
        fva.fva_quantize_v(q, t)
    with pytest.raises(ValueError):
        fva.fva_route_sasa(q, q, 0.9, 2, t, torch.zeros(2, dtype=torch.int32), 2, 0.8, 0.07)


def _noalloc(d=None, flags=0, counts=FAKE, kv=FAKE, trace=None, scale=0.0, o=FAKE, v=FAKE):
    d = d or desc()
    return fva.lib.fva_attn_noalloc(FAKE, FAKE, v, ctypes.byref(d), ctypes.byref(T720.c()), counts, kv,
                                    ctypes.c_float(scale), flags, o, trace, None)


def noalloc_scratch_bytes(heads, nb, batch=1):
    """The layout include/fva.h documents for fva_attn_noalloc's scratch."""
    al = lambda x: (x + 255) // 256 * 256
    rows = batch * heads * nb
    # queue items, 9 queue bases, 8 counters, per-head plan scratch, per-row
    # prefixes, split count, one 32-byte record per block
    return (al(rows * 4) + al(36) + al(32) + al(batch * heads * 19 * 4) + al(2 * (rows + 1) * 4) + al(4)
            + al(nb * 32))


def test_noalloc_scratch_limit_and_argument_errors():
    cap = 16 << 20
    nb = 660
    h_ok = max(h for h in range(1, 4000) if noalloc_scratch_bytes(h, nb) <= cap)
    assert 2000 < h_ok < 2200  # "about 2,000 heads fit" at nb = 660
    # one head past the limit: rejected before any launch (the fake pointers
    # are never touched); shapes inside it would launch, so none is called here
    assert _noalloc(d=desc(H=h_ok + 1)) == fva.FVA_ERR_SCRATCH
    assert _noalloc(d=desc(B=2, H=h_ok)) == fva.FVA_ERR_SCRATCH
    assert "static" in fva.fva_status_string(fva.FVA_ERR_SCRATCH)
    assert _noalloc(flags=fva.FVA_SCHED_NAIVE) == fva.FVA_ERR_INVALID_ARG
    assert _noalloc(flags=fva.FVA_SPLIT_BLOCKS(4)) == fva.FVA_ERR_INVALID_ARG
    assert _noalloc(flags=fva.FVA_SCHED_UNPAIRED) == fva.FVA_ERR_INVALID_ARG
    assert _noalloc(flags=fva.FVA_TRACE, trace=None) == fva.FVA_ERR_INVALID_ARG
    assert _noalloc(counts=None) == fva.FVA_ERR_INVALID_ARG
    assert _noalloc(kv=None) == fva.FVA_ERR_INVALID_ARG
    assert _noalloc(v=None) == fva.FVA_ERR_INVALID_ARG
    assert _noalloc(o=None) == fva.FVA_ERR_INVALID_ARG
    assert _noalloc(scale=float("inf")) == fva.FVA_ERR_INVALID_ARG
    assert _noalloc(d=desc(N=10)) == fva.FVA_ERR_SHAPE
    assert _noalloc(d=desc(B=1024, H=3200)) == fva.FVA_ERR_UNSUPPORTED
