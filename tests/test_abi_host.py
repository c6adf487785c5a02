"""The C-ABI library loads, exports every call the header declares, and its
host-side logic (coverage check, argument and consistency checks that run
before anything is enqueued) agrees with the oracle.  No GPU needed: every
call here is rejected before it touches device memory."""
import ctypes as C
import os
import re

import pytest

from helpers import ensure_lib
from oracle import paged
import test_oracle_paged as top

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000  # a non-null, aligned address that no call here dereferences


@pytest.fixture(scope="module")
def P():
    return ensure_lib()


def header_functions():
    src = open(os.path.join(ROOT, "include", "pallas.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(pallas_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_call(P):
    names = header_functions()
    assert "pallas_prefill_prefix" in names and "pallas_assemble_kv" in names
    h = P.lib()
    for n in names:
        assert hasattr(h, n), n
    assert set(names) == set(P.EXPORTS), "binding and header disagree"
    assert P.pallas_abi_version() == 3


@pytest.mark.parametrize("prefix,ranges,n,ok", top.test_check_coverage.pytestmark[0].args[1])
def test_coverage_matches_oracle(P, prefix, ranges, n, ok):
    st = P.pallas_check_coverage(prefix, [r[0] for r in ranges], [r[1] for r in ranges], n)
    want = paged.check_coverage(prefix, [r[0] for r in ranges], [r[1] for r in ranges], n)
    assert want is ok
    assert (st == P.Status.OK) is ok
    if not ok:
        assert st == P.Status.COVERAGE
        assert "coverage" in P.pallas_last_error()


def fake_pool(P, L=2, pages=8, page=16, hkv=2, d=64):
    from paper_2608_16477_amd.binding import KVPoolC
    return KVPoolC(FAKE, pages, page, L, hkv, d)


def assemble_rc(P, hdrs, req=7, epoch=3, max_pages=4, arena_bytes=1 << 30):
    h = P.lib()
    arr = (P.ChunkHeader * len(hdrs))(*hdrs)
    pool = fake_pool(P)
    return h.pallas_assemble_kv(C.byref(pool), FAKE, max_pages, arr, FAKE, arena_bytes,
                                len(hdrs), req, epoch, None, None)


def hdr(P, start, cnt, req=7, epoch=3, off=0, shape=(2, 2, 64)):
    return P.ChunkHeader(req, epoch, start, cnt, off, *shape, 2)


@pytest.mark.parametrize("case,code", [
    ("request", "WRONG_REQUEST"), ("epoch", "STALE_EPOCH"), ("shape", "INVALID_ARG"),
    ("range", "OUT_OF_RANGE"), ("overlap", "COVERAGE"), ("arena", "OUT_OF_RANGE"),
])
def test_assemble_host_rejections_match_oracle(P, case, code):
    row = 2 * 2 * 64 * 2   # bytes per position over 2 layers x K|V
    good = hdr(P, 0, 16)
    bad = {
        "request": hdr(P, 16, 8, req=8, off=16 * row),
        "epoch": hdr(P, 16, 8, epoch=2, off=16 * row),
        "shape": hdr(P, 16, 8, off=16 * row, shape=(2, 2, 128)),
        "range": hdr(P, 60, 8, off=16 * row),
        "overlap": hdr(P, 15, 8, off=16 * row),
        "arena": hdr(P, 16, 8, off=(1 << 30) - row),
    }[case]
    rc = assemble_rc(P, [good, bad])
    assert P.Status(rc).name == code, P.pallas_last_error()
    if case != "arena":   # the oracle has no arena; the other rules are shared
        oh = [paged.ChunkHeader(x.request_id, x.epoch, x.start_pos, x.num_tokens, x.n_layers,
                                x.n_kv_heads, x.head_dim, x.elem_bytes) for x in (good, bad)]
        import numpy as np
        pool = np.zeros((2, 2, 8, 16, 2, 64), np.uint16)
        with pytest.raises(paged.Rejected) as e:
            paged.check_chunks(pool, 4 * 16, oh, 7, 3)
        assert e.value.code == code


def test_empty_copy_calls_enqueue_nothing(P):
    """Pack and assemble with no chunks, or only zero-token ones, pass their
    checks and enqueue nothing: here, with no GPU, they still return OK.
    An empty header is still checked (a stale epoch rejects the call), as
    the oracle's assembly checks every header."""
    h = P.lib()
    pool = fake_pool(P)

    def pack(descs):
        arr = (P.ChunkDesc * max(1, len(descs)))(*descs)
        return P.Status(h.pallas_pack_suffix_blocks(C.byref(pool), FAKE, 4, arr, len(descs), FAKE, 1 << 20,
                                                    None, None))
    assert pack([]) == P.Status.OK
    assert pack([P.ChunkDesc(3, 0, 0), P.ChunkDesc(9, 0, 16)]) == P.Status.OK
    assert P.Status(assemble_rc(P, [])) == P.Status.OK
    assert P.Status(assemble_rc(P, [hdr(P, 5, 0), hdr(P, 20, 0, off=64)])) == P.Status.OK
    assert P.Status(assemble_rc(P, [hdr(P, 5, 0, epoch=2)])) == P.Status.STALE_EPOCH
    import numpy as np
    onp = np.zeros((2, 2, 8, 16, 2, 64), np.uint16)
    with pytest.raises(paged.Rejected) as e:
        paged.check_chunks(onp, 4 * 16, [paged.ChunkHeader(7, 2, 5, 0, 2, 2, 64, 2)], 7, 3)
    assert e.value.code == "STALE_EPOCH"


def test_pack_host_rejections(P):
    h = P.lib()
    pool = fake_pool(P)
    def rc(descs, arena_bytes=1 << 20, max_pages=4):
        arr = (P.ChunkDesc * max(1, len(descs)))(*descs)
        return P.Status(h.pallas_pack_suffix_blocks(C.byref(pool), FAKE, max_pages, arr, len(descs),
                                                    FAKE, arena_bytes, None, None))
    row = 2 * 2 * 64 * 2
    assert rc([P.ChunkDesc(60, 8, 0)]) == P.Status.OUT_OF_RANGE
    assert rc([P.ChunkDesc(0, 8, 8)]) == P.Status.INVALID_ARG             # unaligned offset
    assert rc([P.ChunkDesc(0, 8, 0)], arena_bytes=8 * row - 16) == P.Status.OUT_OF_RANGE
    assert rc([P.ChunkDesc(0, 8, 0), P.ChunkDesc(8, 8, 4 * row)]) == P.Status.INVALID_ARG  # arena overlap
    assert rc([P.ChunkDesc(-1, 8, 0)]) == P.Status.OUT_OF_RANGE


def test_model_create_rejects_bad_shapes(P):
    from workloads import configs
    from paper_2608_16477_amd.binding import ModelConfigC, WeightsC, LayerWeightsC
    h = P.lib()
    def rc(**kw):
        c = configs.TINY.replace(**kw)
        cc = ModelConfigC(c.n_layers, c.hidden, c.n_q_heads, c.n_kv_heads, c.head_dim, c.ffn,
                          c.vocab, c.rms_eps, c.rope_theta, int(c.qk_norm), c.page_size)
        la = (LayerWeightsC * c.n_layers)()
        for l in range(c.n_layers):
            for name, _ in LayerWeightsC._fields_:
                setattr(la[l], name, FAKE)
        w = WeightsC(FAKE, FAKE, FAKE, la)
        out = C.c_void_p()
        r = h.pallas_model_create(C.byref(cc), C.byref(w), C.byref(out))
        if r == 0:
            h.pallas_model_destroy(out)
        return P.Status(r)
    assert rc() == P.Status.OK
    assert rc(n_q_heads=3) == P.Status.INVALID_ARG
    assert rc(head_dim=96) == P.Status.UNSUPPORTED
    assert rc(page_size=32) == P.Status.UNSUPPORTED
    assert rc(hidden=200) == P.Status.UNSUPPORTED


def test_prefill_rejects_sequences_beyond_the_length_limit(P):
    """A sequence longer than PALLAS_MAX_PREFILL_LEN tokens is refused on the
    host (UNSUPPORTED) before anything touches the device; one at the limit
    passes that check and stops at the (undersized) workspace instead."""
    from workloads import configs
    from paper_2608_16477_amd.binding import ModelConfigC, WeightsC, LayerWeightsC, KVPoolC
    h = P.lib()
    c = configs.TINY
    cc = ModelConfigC(c.n_layers, c.hidden, c.n_q_heads, c.n_kv_heads, c.head_dim, c.ffn,
                      c.vocab, c.rms_eps, c.rope_theta, int(c.qk_norm), c.page_size)
    la = (LayerWeightsC * c.n_layers)()
    for l in range(c.n_layers):
        for name, _ in LayerWeightsC._fields_:
            setattr(la[l], name, FAKE)
    w = WeightsC(FAKE, FAKE, FAKE, la)
    model = C.c_void_p()
    assert h.pallas_model_create(C.byref(cc), C.byref(w), C.byref(model)) == 0
    limit = 32768
    pool = KVPoolC(FAKE, 4096, c.page_size, c.n_layers, c.n_kv_heads, c.head_dim)
    try:
        def rc(n):
            cu = (C.c_int32 * 2)(0, n)
            return P.Status(h.pallas_prefill_prefix(model, 1, FAKE, cu, FAKE, 4096, C.byref(pool),
                                                    FAKE, 256, None, None))
        assert rc(limit + 1) == P.Status.UNSUPPORTED
        assert rc(limit) == P.Status.WORKSPACE
    finally:
        h.pallas_model_destroy(model)


def test_prefill_rejects_k_planes_beyond_4_gib(P):
    """Prefill attention addresses one layer's K plane with 32-bit offsets:
    a pool whose plane (num_pages * page * n_kv_heads * head_dim * 2 bytes)
    exceeds 4 GiB - 1 is refused on the host (UNSUPPORTED) before anything
    touches the device; one page fewer passes that check and stops at the
    (undersized) workspace instead.  Both prefill calls apply it."""
    from workloads import configs
    from paper_2608_16477_amd.binding import ModelConfigC, WeightsC, LayerWeightsC, KVPoolC
    h = P.lib()
    c = configs.TINY
    cc = ModelConfigC(c.n_layers, c.hidden, c.n_q_heads, c.n_kv_heads, c.head_dim, c.ffn,
                      c.vocab, c.rms_eps, c.rope_theta, int(c.qk_norm), c.page_size)
    la = (LayerWeightsC * c.n_layers)()
    for l in range(c.n_layers):
        for name, _ in LayerWeightsC._fields_:
            setattr(la[l], name, FAKE)
    w = WeightsC(FAKE, FAKE, FAKE, la)
    model = C.c_void_p()
    assert h.pallas_model_create(C.byref(cc), C.byref(w), C.byref(model)) == 0
    page_bytes = c.page_size * c.n_kv_heads * c.head_dim * 2
    first_refused = (1 << 32) // page_bytes          # plane of exactly 4 GiB
    assert (first_refused * page_bytes) == 1 << 32
    try:
        def rc(pages, chunk):
            pool = KVPoolC(FAKE, pages, c.page_size, c.n_layers, c.n_kv_heads, c.head_dim)
            cu = (C.c_int32 * 2)(0, 16)
            if chunk:
                start = (C.c_int32 * 1)(16)
                return P.Status(h.pallas_prefill_chunk(model, 1, FAKE, cu, start, FAKE, 4, C.byref(pool),
                                                       FAKE, 256, None, None))
            return P.Status(h.pallas_prefill_prefix(model, 1, FAKE, cu, FAKE, 4, C.byref(pool),
                                                    FAKE, 256, None, None))
        for chunk in (False, True):
            assert rc(first_refused, chunk) == P.Status.UNSUPPORTED
            assert "4 GiB" in P.pallas_last_error()
            assert rc(first_refused - 1, chunk) == P.Status.WORKSPACE
    finally:
        h.pallas_model_destroy(model)


def test_profile_clock_arguments(P):
    """The clock query rejects a class outside the enumeration; with nothing
    sampled it reports 0 GHz and 0 workgroups."""
    h = P.lib()
    ghz, wgs = C.c_double(7.0), C.c_int64(7)
    assert h.pallas_profile_clock(13, C.byref(ghz), C.byref(wgs)) == P.Status.INVALID_ARG
    assert h.pallas_profile_clock(-1, C.byref(ghz), C.byref(wgs)) == P.Status.INVALID_ARG
    assert h.pallas_profile_clock(7, None, C.byref(wgs)) == P.Status.INVALID_ARG
    assert h.pallas_profile_clock(7, C.byref(ghz), C.byref(wgs)) == P.Status.OK
    assert ghz.value == 0.0 and wgs.value == 0


def fake_model(P, c):
    """A model handle over fake (never dereferenced) weight pointers."""
    from paper_2608_16477_amd.binding import ModelConfigC, WeightsC, LayerWeightsC
    h = P.lib()
    cc = ModelConfigC(c.n_layers, c.hidden, c.n_q_heads, c.n_kv_heads, c.head_dim, c.ffn,
                      c.vocab, c.rms_eps, c.rope_theta, int(c.qk_norm), c.page_size)
    la = (LayerWeightsC * c.n_layers)()
    for l in range(c.n_layers):
        for name, _ in LayerWeightsC._fields_:
            setattr(la[l], name, FAKE)
    w = WeightsC(FAKE, FAKE, FAKE, la)
    model = C.c_void_p()
    assert h.pallas_model_create(C.byref(cc), C.byref(w), C.byref(model)) == 0
    return model


def test_prefill_rejects_operands_beyond_2_gib(P):
    """The projections address their bf16 operands with 32-bit offsets, so
    the [M][ffn] SwiGLU product must stay below 2 GiB: at the 64-layer shape
    (ffn 25600) a prefill of 41,944 rows (two sequences of 20,972 tokens,
    within the per-sequence and table limits) is refused on the host with
    UNSUPPORTED, before anything is enqueued (no device exists here, so any
    launch would have failed with HIP instead).  41,943 rows pass that check
    and stop at the undersized workspace.  Both prefill calls apply it."""
    from workloads import configs
    from paper_2608_16477_amd.binding import KVPoolC
    h = P.lib()
    c = configs.LARGE
    assert 41943 * c.ffn * 2 < (1 << 31) <= 41944 * c.ffn * 2
    model = fake_model(P, c)
    pool = KVPoolC(FAKE, 8192, c.page_size, c.n_layers, c.n_kv_heads, c.head_dim)
    try:
        def rc(total, chunk):
            a = total // 2
            cu = (C.c_int32 * 3)(0, a, total)
            if chunk:
                start = (C.c_int32 * 2)(0, 0)
                return P.Status(h.pallas_prefill_chunk(model, 2, FAKE, cu, start, FAKE, 2048, C.byref(pool),
                                                       FAKE, 1 << 40, None, None))
            return P.Status(h.pallas_prefill_prefix(model, 2, FAKE, cu, FAKE, 2048, C.byref(pool),
                                                    FAKE, 256, None, None))
        for chunk in (False, True):
            assert rc(41944, chunk) == P.Status.UNSUPPORTED
            assert "SwiGLU product" in P.pallas_last_error()
        assert rc(41943, False) == P.Status.WORKSPACE
    finally:
        h.pallas_model_destroy(model)


def test_decode_rejects_positions_and_operands_beyond_limits(P):
    """Decode positions above PALLAS_MAX_DECODE_POS (16383) are refused with
    UNSUPPORTED.  More than 8 sequences run the MFMA GEMM, whose operands
    must stay below 2 GiB: an lm_head of 262144 x 5120 bf16 (2.5 GiB) is
    refused for 9 sequences and accepted for 8 (the skinny kernel); those
    calls then stop at the undersized workspace."""
    from workloads import configs
    from paper_2608_16477_amd.binding import KVPoolC
    h = P.lib()
    c = configs.LARGE.replace(n_layers=2, vocab=262144)
    model = fake_model(P, c)
    pool = KVPoolC(FAKE, 8192, c.page_size, c.n_layers, c.n_kv_heads, c.head_dim)
    try:
        def rc(positions):
            pos = (C.c_int32 * len(positions))(*positions)
            return P.Status(h.pallas_decode_step(model, len(positions), FAKE, pos, FAKE, 2048, C.byref(pool),
                                                 FAKE, FAKE, 256, None, None))
        assert rc([16384]) == P.Status.UNSUPPORTED
        assert "16383" in P.pallas_last_error()
        assert rc([16383]) == P.Status.WORKSPACE
        assert rc([10] * 9) == P.Status.UNSUPPORTED
        assert "lm_head" in P.pallas_last_error()
        assert rc([10] * 8) == P.Status.WORKSPACE
    finally:
        h.pallas_model_destroy(model)


def test_static_decode_host_rejections(P):
    """pallas_decode_step_static applies pallas_decode_step's checks, then
    its own limits, all before it touches the device: more than
    PALLAS_STATIC_DECODE_MAX_SEQS (8) sequences, or a step whose scratch
    need exceeds PALLAS_STATIC_SCRATCH_BYTES (64 MiB): 8 sequences at
    position 15,744 of the large shape need 64.22 MiB (at 15,743, 63.97
    MiB: the decode-attention records grow by one 64-key split there).
    (A call that
    passes every check is not made here: with a device present it would
    launch kernels on the fake pointers.)"""
    from workloads import configs
    from paper_2608_16477_amd.binding import KVPoolC
    h = P.lib()
    c = configs.LARGE.replace(n_layers=2)
    model = fake_model(P, c)
    pool = KVPoolC(FAKE, 8192, c.page_size, c.n_layers, c.n_kv_heads, c.head_dim)
    try:
        def rc(positions):
            pos = (C.c_int32 * len(positions))(*positions)
            return P.Status(h.pallas_decode_step_static(model, len(positions), FAKE, pos, FAKE, 2048,
                                                        C.byref(pool), FAKE, None, None))
        assert rc([16384]) == P.Status.UNSUPPORTED
        assert rc([5] * 9) == P.Status.UNSUPPORTED
        assert "at most 8" in P.pallas_last_error()
        assert rc([15744] * 8) == P.Status.UNSUPPORTED
        assert "scratch" in P.pallas_last_error()
        assert rc([-1]) == P.Status.OUT_OF_RANGE
    finally:
        h.pallas_model_destroy(model)
