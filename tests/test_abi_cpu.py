"""Host-side checks of the C ABI: symbols, arena sizing and argument validation.

None of these calls reaches the GPU: validation precedes all device work.
"""
import ctypes as C
import os
import re

import pytest

import pard_inputs as pi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pard.h")
LIB = os.path.join(ROOT, "paper_2504_18583_amd", "libpard.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libpard.so not built")


@pytest.fixture(scope="module")
def b():
    from paper_2504_18583_amd import binding
    return binding


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pard_[a-z_]+)\s*\(", text)))


def test_every_declared_function_is_exported(b):
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(b.lib, n), n
    assert set(names) == set(b.EXPORTED)


def _pair(name="llama8b_1b"):
    wl = pi.WORKLOADS[name]
    return wl, pi.with_dtype(wl.target, "bf16"), pi.with_dtype(wl.draft, "bf16")


def test_arena_bytes_covers_weights_and_cache(b):
    wl, t, d = _pair()
    n = b.pard_arena_bytes(b.spec_from(t), b.spec_from(d), 1, 1100, 8)
    weights = 2 * (t.n_params() + d.n_params())
    kv = 1100 * (131072 + 32768)
    assert weights + kv < n < weights + kv + 2.0e9
    n2 = b.pard_arena_bytes(b.spec_from(t), b.spec_from(d), 2, 1100, 8)
    assert n2 - n >= kv


@pytest.mark.parametrize("field,value", [("head_dim", 96), ("dtype", 0), ("vocab", 1000),
                                         ("d_model", 100), ("n_kv_heads", 3), ("n_layers", 0),
                                         ("rms_eps", 0.0), ("rope_factor", 0.5)])
def test_arena_bytes_rejects_bad_spec(b, field, value):
    _, t, d = _pair("tiny")
    ts = b.spec_from(t)
    setattr(ts, field, value)
    assert b.pard_arena_bytes(ts, b.spec_from(d), 1, 256, 4) == 0


def test_rope_scaling_fields_cross_the_abi(b):
    """The scaling fields sit after the seed in the C struct: a valid set is
    accepted, each inconsistent one rejected."""
    from dataclasses import replace
    _, t, d = _pair("tiny")
    good = b.spec_from(replace(t, rope_scaling=(8.0, 1.0, 4.0, 8192)))
    assert (good.rope_factor, good.rope_original_max_pos) == (8.0, 8192)
    assert b.pard_arena_bytes(good, b.spec_from(d), 1, 256, 4) > 0
    for field, value in (("rope_low_freq_factor", 0.0), ("rope_high_freq_factor", 1.0),
                         ("rope_original_max_pos", 0), ("rope_factor", float("inf"))):
        bad = b.spec_from(replace(t, rope_scaling=(8.0, 1.0, 4.0, 8192)))
        setattr(bad, field, value)
        assert b.pard_arena_bytes(bad, b.spec_from(d), 1, 256, 4) == 0, field


def test_arena_bytes_rejects_bad_capacity(b):
    _, t, d = _pair("tiny")
    ts, ds = b.spec_from(t), b.spec_from(d)
    assert b.pard_arena_bytes(ts, ds, 1, 256, 0) == 0
    assert b.pard_arena_bytes(ts, ds, 1, 256, 33) == 0
    assert b.pard_arena_bytes(ts, ds, 0, 256, 4) == 0
    assert b.pard_arena_bytes(ts, ds, 1, 9, 4) == 0
    ds.vocab = 2048
    assert b.pard_arena_bytes(ts, ds, 1, 256, 4) == 0


def _load(b, t, d, mask, arena, nbytes, max_k=4):
    ctx = b._CTX()
    st = b.lib.pard_model_load(C.byref(t), C.byref(d), mask, 1, 256, max_k, C.c_void_p(arena),
                               nbytes, None, C.byref(ctx))
    return st, ctx.value


def test_model_load_validates_before_device_work(b):
    _, t, d = _pair("tiny")
    ts, ds = b.spec_from(t), b.spec_from(d)
    need = b.pard_arena_bytes(ts, ds, 1, 256, 4)
    assert _load(b, ts, ds, 1023, 0, need)[0] == b.PARD_ERR_ARG            # null arena
    assert _load(b, ts, ds, 1023, 0x1000 + 8, need)[0] == b.PARD_ERR_ARG   # misaligned
    assert _load(b, ts, ds, 1023, 0x1000, need - 1)[0] == b.PARD_ERR_NOMEM
    assert _load(b, ts, ds, 1024, 0x1000, need)[0] == b.PARD_ERR_ARG       # mask id
    assert _load(b, ts, ds, 1023, 0x1000, need, max_k=0)[0] == b.PARD_ERR_ARG
    bad = b.spec_from(t)
    bad.head_dim = 96
    assert _load(b, bad, ds, 1023, 0x1000, need)[0] == b.PARD_ERR_UNSUPPORTED
    bad = b.spec_from(t)
    bad.dtype = b.PARD_F32
    assert _load(b, bad, ds, 1023, 0x1000, need)[0] == b.PARD_ERR_UNSUPPORTED


def test_null_context_calls_return_arg(b):
    one = (C.c_int32 * 4)(1, 2, 3, 4)
    out = C.c_int32()
    assert b.lib.pard_prefill(None, 0, one, 4, C.byref(out)) == b.PARD_ERR_ARG
    assert b.lib.pard_draft(None, 0, one, 4, 2, one) == b.PARD_ERR_ARG
    assert b.lib.pard_verify(None, 0, one, 2, C.byref(out), C.byref(out)) == b.PARD_ERR_ARG
    assert b.lib.pard_kv_truncate(None, 0, 0, 0) == b.PARD_ERR_ARG
    assert b.lib.pard_kv_len(None, 0, 0, C.byref(out)) == b.PARD_ERR_ARG
    assert b.lib.pard_generate(None, 1, one, 2, 4, 0, one, None) == b.PARD_ERR_ARG
    assert b.lib.pard_generate_ex(None, 1, one, 2, b.PARD_MODE_VANILLA, 4, 0, one, None) == b.PARD_ERR_ARG
    assert b.lib.pard_last_error(None) == b"null context"
    b.lib.pard_free(None)
    assert b.lib.pard_status_string(b.PARD_ERR_CAPACITY) == b"PARD_ERR_CAPACITY"
    assert b.lib.pard_status_string(b.PARD_ERR_RANGE) == b"PARD_ERR_RANGE"


def test_cod_capacity_and_argument_checks(b):
    """Host-side COD checks (no device work): the capacity equals subtask 1's
    columns plus each later subtask's keep target; bad parameters, lengths and
    undersized output regions are refused before any device call."""
    import ctypes as C
    from oracle import cod
    for n_tok, k, r, r_min in ((5, 3, 0.5, 0.0), (1001, 8, 0.7, 0.2), (2, 8, 0.7, 0.2), (8193, 4, 0.9, 0.0)):
        n = n_tok - 1
        want = n + sum(cod.keep_target(n, kk, r, r_min) for kk in range(2, k + 1))
        assert b.cod_capacity(n_tok, k, r, r_min) == want
    assert b.cod_capacity(1, 4, 0.5, 0.0) == -1 and b.cod_capacity(8194, 4, 0.5, 0.0) == -1
    assert b.cod_capacity(10, 0, 0.5, 0.0) == -1 and b.cod_capacity(10, 4, 0.0, 0.0) == -1
    assert b.cod_capacity(10, 4, 1.5, 0.0) == -1 and b.cod_capacity(10, 4, 0.5, -0.1) == -1
    dummy = C.c_void_p(16)                       # never dereferenced: the checks fail first
    P64 = C.POINTER(C.c_int64)

    def build(tok_offs, out_offs, k=4, r=0.5, ws=256, ws_bytes=None):
        t = (C.c_int64 * len(tok_offs))(*tok_offs)
        o = (C.c_int64 * len(out_offs))(*out_offs)
        n = len(tok_offs) - 1
        if ws_bytes is None:
            ws_bytes = b.lib.pard_cod_workspace_bytes(n)
        return b.lib.pard_cod_build(dummy, C.cast(t, P64), n, k, r, 0.0, 0, 0, C.cast(o, P64),
                                    dummy, dummy, dummy, dummy, dummy, dummy, C.c_void_p(ws), ws_bytes, None, None)
    cap = b.cod_capacity(10, 4, 0.5, 0.0)
    # the device workspace holds both offset arrays (int64, n_samples + 1 each)
    assert b.lib.pard_cod_workspace_bytes(1) >= 32 and b.lib.pard_cod_workspace_bytes(1000) >= 16 * 1001
    assert b.lib.pard_cod_workspace_bytes(0) == 0
    assert build([0, 10], [0, cap], ws=0) == b.PARD_ERR_ARG                 # no workspace
    assert build([0, 10], [0, cap], ws=256 + 8) == b.PARD_ERR_ARG           # misaligned
    assert build([0, 10], [0, cap], ws_bytes=31) == b.PARD_ERR_NOMEM        # too small
    assert build([0, 10], [0, cap - 1]) == b.PARD_ERR_CAPACITY
    assert build([0, 1], [0, 100]) == b.PARD_ERR_ARG          # a one-token sample
    assert build([0, 10], [0, cap], k=0) == b.PARD_ERR_ARG
    assert build([0, 10], [0, cap], r=2.0) == b.PARD_ERR_ARG
    # the layout is the capacities' prefix sum
    offs = (C.c_int64 * 4)(0, 10, 12, 500)
    lay = (C.c_int64 * 4)()
    total = b.lib.pard_cod_layout(C.cast(offs, P64), 3, 4, 0.5, 0.0, C.cast(lay, P64))
    caps = [b.cod_capacity(n, 4, 0.5, 0.0) for n in (10, 2, 488)]
    assert list(lay) == [0, caps[0], caps[0] + caps[1], sum(caps)] and total == sum(caps)


def test_matrices_of_2gib_or_more_are_refused(b):
    """The kernels address a strip-packed weight with 32-bit byte offsets: a
    spec whose largest matrix (here a 152 064 x 8192 lm_head, 2.49 GB in two
    bytes per weight) reaches 2 GiB is refused, one just below is accepted."""
    from dataclasses import replace
    _, t, d = _pair("tiny")
    big = replace(t, n_layers=1, d_model=8192, n_heads=64, n_kv_heads=8, head_dim=128, ffn_dim=1024,
                  vocab=152064)
    drf = replace(d, vocab=152064)
    ts, ds = b.spec_from(big), b.spec_from(drf)
    assert b.pard_arena_bytes(ts, ds, 1, 256, 4) == 0
    assert _load(b, ts, ds, 152063, 0x1000, 1 << 40)[0] == b.PARD_ERR_UNSUPPORTED
    # 131 056 x 8192 x 2 = 2 147 221 504 bytes < 2^31: accepted
    ok = replace(big, vocab=131056)
    assert b.pard_arena_bytes(b.spec_from(ok), b.spec_from(replace(d, vocab=131056)), 1, 256, 4) > 0
    # gate/up: 2 x 65 536 x 8192 x 2 bytes = 2 GiB exactly
    ffn = replace(t, n_layers=1, d_model=8192, n_heads=64, n_kv_heads=8, head_dim=128, ffn_dim=65536)
    assert b.pard_arena_bytes(b.spec_from(ffn), b.spec_from(d), 1, 256, 4) == 0


def test_cod_noalloc_refuses_batches_above_its_scratch(b):
    """The allocation-free COD call stages its offsets in a fixed device
    scratch of PARD_COD_NOALLOC_MAX_SAMPLES samples: a larger batch is refused
    with CAPACITY before any device work (nothing is dereferenced)."""
    import numpy as np
    P64 = C.POINTER(C.c_int64)
    dummy = C.c_void_p(16)
    n = b.PARD_COD_NOALLOC_MAX_SAMPLES + 1
    offs = np.arange(0, 3 * (n + 1), 3, dtype=np.int64)
    out = np.zeros(n + 1, np.int64)
    rc = b.lib.pard_cod_build_noalloc(dummy, offs.ctypes.data_as(P64), n, 4, 0.5, 0.0, 0, 0, out.ctypes.data_as(P64),
                                      dummy, dummy, dummy, dummy, dummy, dummy, None)
    assert rc == b.PARD_ERR_CAPACITY
    # bad parameters are refused the same way as by pard_cod_build
    rc = b.lib.pard_cod_build_noalloc(dummy, offs.ctypes.data_as(P64), 3, 0, 0.5, 0.0, 0, 0, out.ctypes.data_as(P64),
                                      dummy, dummy, dummy, dummy, dummy, dummy, None)
    assert rc == b.PARD_ERR_ARG
