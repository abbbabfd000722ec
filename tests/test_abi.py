"""The C-ABI library loads, exports every symbol its header declares, and
rejects bad arguments before launching anything (no GPU needed: every call
here fails validation)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2605_22850_amd as oc
from paper_2605_22850_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "objectcache.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(oc_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = oc.lib()
    names = declared_functions()
    assert len(names) >= 10
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, f"not exported: {missing}"
    assert set(names) == set(L.EXPORTS)


def test_abi_version():
    assert oc.oc_abi_version() == 6


def _layout(**kw):
    base = dict(num_layers=2, num_q_heads=4, num_kv_heads=2, head_dim=64, page_size=16, chunk_tokens=16, num_pages=64)
    base.update(kw)
    return L.c_layout(*base.values())


FAKE = 1 << 20            # aligned non-null "device" address; never dereferenced


def _ingest(layout, num_chunks=16, slice_bytes=None, table_entries=16, num_tokens=256, layer=0, data=FAKE,
            base=FAKE):
    if slice_bytes is None:
        slice_bytes = 2 * layout.chunk_tokens * layout.num_kv_heads * layout.head_dim * 2
    st = L.c_staging(data, num_chunks, slice_bytes)
    bt = L.c_block_table(FAKE, table_entries, num_tokens)
    kp = L.c_kv_pool(base, layout)
    return oc.lib().oc_kv_layer_ingest(ctypes.byref(st), ctypes.byref(bt), ctypes.byref(kp), layer, None)


def test_ingest_validation():
    lay = _layout()
    assert _ingest(lay, slice_bytes=1000) == L.OC_ESHAPE
    assert b"2*G*n_kv*d*2" in oc.lib().oc_last_error()
    assert _ingest(lay, layer=2) == L.OC_ERANGE
    assert _ingest(lay, layer=-1) == L.OC_ERANGE
    assert _ingest(lay, table_entries=15) == L.OC_ERANGE
    assert _ingest(lay, num_chunks=15) == L.OC_ESHAPE
    assert _ingest(lay, data=FAKE + 8) == L.OC_EALIGN
    assert _ingest(lay, base=FAKE + 2) == L.OC_EALIGN
    assert _ingest(_layout(num_q_heads=3)) == L.OC_ESHAPE
    assert _ingest(_layout(page_size=12)) == L.OC_ESHAPE
    assert _ingest(_layout(head_dim=60)) == L.OC_ESHAPE
    assert _ingest(_layout(chunk_tokens=0)) == L.OC_EINVAL
    assert _ingest(_layout(num_pages=8)) == L.OC_ERANGE
    # nothing to do is not an error
    assert _ingest(lay, num_chunks=0, table_entries=0, num_tokens=0) == L.OC_OK
    assert oc.lib().oc_kv_layer_ingest(None, None, None, 0, None) == L.OC_EINVAL


def _chunks(layout, num_chunks=4, first_chunk=0, slice_bytes=None, table_entries=16, num_tokens=256, data=FAKE,
            base=FAKE):
    if slice_bytes is None:
        slice_bytes = 2 * layout.chunk_tokens * layout.num_kv_heads * layout.head_dim * 2
    st = L.c_staging(data, num_chunks, slice_bytes)
    bt = L.c_block_table(FAKE, table_entries, num_tokens)
    kp = L.c_kv_pool(base, layout)
    return oc.lib().oc_kv_chunks_ingest(ctypes.byref(st), first_chunk, ctypes.byref(bt), ctypes.byref(kp), None)


def test_chunks_ingest_validation():
    lay = _layout()
    assert _chunks(lay, slice_bytes=1000) == L.OC_ESHAPE
    assert _chunks(lay, first_chunk=-1) == L.OC_EINVAL
    assert _chunks(lay, num_chunks=-1) == L.OC_EINVAL
    # chunks 13..16 of a 16-chunk (256-token) prefix run past its end
    assert _chunks(lay, first_chunk=13) == L.OC_ERANGE
    assert b"past the end" in oc.lib().oc_last_error()
    assert _chunks(lay, table_entries=15) == L.OC_ERANGE
    assert _chunks(lay, data=FAKE + 8) == L.OC_EALIGN
    assert _chunks(lay, base=FAKE + 2) == L.OC_EALIGN
    assert _chunks(_layout(num_q_heads=3)) == L.OC_ESHAPE
    # no objects is not an error, wherever they would start
    assert _chunks(lay, num_chunks=0, first_chunk=16) == L.OC_OK
    assert oc.lib().oc_kv_chunks_ingest(None, 0, None, None, None) == L.OC_EINVAL


def _gather_chunks(layout, first_chunk=0, num_chunks=4, table_entries=16, num_tokens=256, out=FAKE, base=FAKE):
    bt = L.c_block_table(FAKE, table_entries, num_tokens)
    kp = L.c_kv_pool(base, layout)
    return oc.lib().oc_kv_chunks_gather(ctypes.byref(bt), ctypes.byref(kp), first_chunk, num_chunks, out, None)


def test_chunks_gather_validation():
    lay = _layout()
    assert _gather_chunks(lay, first_chunk=-1) == L.OC_EINVAL
    assert _gather_chunks(lay, num_chunks=-1) == L.OC_EINVAL
    assert _gather_chunks(lay, first_chunk=13) == L.OC_ERANGE
    assert b"past the end" in oc.lib().oc_last_error()
    assert _gather_chunks(lay, table_entries=15) == L.OC_ERANGE
    assert _gather_chunks(lay, out=FAKE + 8) == L.OC_EALIGN
    assert _gather_chunks(lay, base=FAKE + 2) == L.OC_EALIGN
    assert _gather_chunks(lay, out=None) == L.OC_EINVAL
    assert _gather_chunks(_layout(head_dim=60)) == L.OC_ESHAPE
    assert _gather_chunks(lay, num_chunks=0, first_chunk=16) == L.OC_OK
    assert oc.lib().oc_kv_chunks_gather(None, None, 0, 0, None, None) == L.OC_EINVAL


def _append(layout, suffix_tokens=32, table_entries=18, num_tokens=256, layer=0, k=FAKE, v=FAKE, base=FAKE):
    bt = L.c_block_table(FAKE, table_entries, num_tokens)
    kp = L.c_kv_pool(base, layout)
    return oc.lib().oc_kv_suffix_append(k, v, suffix_tokens, ctypes.byref(bt), ctypes.byref(kp), layer, None)


def test_suffix_append_validation():
    lay = _layout()
    # 256 prefix + 32 suffix tokens need 18 pages of 16
    assert _append(lay, table_entries=17) == L.OC_ERANGE
    assert b"18 entries" in oc.lib().oc_last_error()
    assert _append(lay, suffix_tokens=-1) == L.OC_EINVAL
    assert _append(lay, layer=2) == L.OC_ERANGE
    assert _append(lay, k=FAKE + 4) == L.OC_EALIGN
    assert _append(lay, v=FAKE + 8) == L.OC_EALIGN
    assert _append(lay, k=None) == L.OC_EINVAL
    assert _append(_layout(num_pages=17)) == L.OC_ERANGE
    assert _append(_layout(page_size=12)) == L.OC_ESHAPE
    # nothing to append is not an error, even with a table that has no room
    assert _append(lay, suffix_tokens=0, table_entries=16) == L.OC_OK
    assert oc.lib().oc_kv_suffix_append(None, None, 1, None, None, 0, None) == L.OC_EINVAL


def _rest(layout, ffn=64, tokens=8, layer=0, weights=(FAKE, FAKE, FAKE, FAKE), attn=FAKE,
          bufs=(FAKE, FAKE, FAKE, FAKE, FAKE)):
    w = L.c_layer_weights(ffn, *weights)
    b = L.c_layer_buffers(*bufs)
    return oc.lib().oc_rest_of_layer(attn, tokens, ctypes.byref(layout), ctypes.byref(w), layer, ctypes.byref(b),
                                     None)


def test_rest_of_layer_validation():
    lay = _layout()
    assert _rest(lay, ffn=60) == L.OC_ESHAPE
    assert _rest(lay, ffn=0) == L.OC_ESHAPE
    assert _rest(lay, weights=(FAKE, None, FAKE, FAKE)) == L.OC_EINVAL
    assert _rest(lay, weights=(FAKE, FAKE, FAKE + 8, FAKE)) == L.OC_EALIGN
    assert _rest(lay, layer=2) == L.OC_ERANGE
    assert _rest(lay, tokens=-1) == L.OC_EINVAL
    assert _rest(lay, attn=None) == L.OC_EINVAL
    assert _rest(lay, attn=FAKE + 2) == L.OC_EALIGN
    assert _rest(lay, bufs=(FAKE, FAKE, None, FAKE, FAKE)) == L.OC_EINVAL
    assert _rest(lay, bufs=(FAKE, FAKE, FAKE, FAKE, FAKE + 4)) == L.OC_EALIGN
    assert _rest(_layout(num_q_heads=3)) == L.OC_ESHAPE
    # no tokens is not an error (nothing is launched)
    assert _rest(lay, tokens=0, attn=None, bufs=(None,) * 5) == L.OC_OK
    assert oc.lib().oc_rest_of_layer(FAKE, 8, None, None, 0, None, None) == L.OC_EINVAL


def test_attention_validation():
    lay = _layout()
    bt = L.c_block_table(FAKE, 16, 256)
    kp = L.c_kv_pool(FAKE, lay)
    f = oc.lib().oc_suffix_prefill_layer
    need = oc.lib().oc_attention_workspace_bytes(ctypes.byref(lay), 256, 32)
    assert need > 0
    args = [FAKE, FAKE, FAKE, 32, ctypes.byref(kp), ctypes.byref(bt), 0, FAKE, FAKE, need, None]
    bad = list(args); bad[9] = need - 1
    assert f(*bad) == L.OC_EINVAL and b"workspace too small" in oc.lib().oc_last_error()
    bad = list(args); bad[3] = 0
    assert f(*bad) == L.OC_EINVAL
    bad = list(args); bad[0] = FAKE + 4
    assert f(*bad) == L.OC_EALIGN
    bad = list(args); bad[8] = FAKE + 16
    assert f(*bad) == L.OC_EALIGN
    bad = list(args); bad[6] = 5
    assert f(*bad) == L.OC_ERANGE
    lay96 = _layout(head_dim=96)
    assert oc.lib().oc_attention_workspace_bytes(ctypes.byref(lay96), 256, 32) == 0
    lay_p32 = _layout(page_size=32)
    assert oc.lib().oc_attention_workspace_bytes(ctypes.byref(lay_p32), 256, 32) == 0


def test_workspace_grows_with_lengths():
    lay = _layout(num_layers=32, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=16384)
    f = oc.lib().oc_attention_workspace_bytes
    small = f(ctypes.byref(lay), 4096, 128)
    big = f(ctypes.byref(lay), 65536, 512)
    assert 0 < small < big < (1 << 30)


def test_block_table_check():
    oc.oc_block_table_check([3, 1, 2], 40, 4, 16)
    with pytest.raises(oc.OcError) as e:
        oc.oc_block_table_check([3, 1, 3], 40, 4, 16)
    assert e.value.status == L.OC_ERANGE
    with pytest.raises(oc.OcError):
        oc.oc_block_table_check([3, 1, 4], 40, 4, 16)
    with pytest.raises(oc.OcError):
        oc.oc_block_table_check([3, 1], 40, 4, 16)
    oc.oc_block_table_check(np.zeros(0, np.int32), 0, 4, 16)
    # the check's memory follows the table, not the pool: a pool of 2^62
    # pages is no reason to fail
    oc.oc_block_table_check([5, 1 << 30, 7], 40, 1 << 62, 16)
    with pytest.raises(oc.OcError) as e:
        oc.oc_block_table_check([5, 1 << 30, 5], 40, 1 << 62, 16)
    assert e.value.status == L.OC_ERANGE and "repeats" in str(e.value)


def test_context_rejects_an_absent_device():
    lay = _layout()
    kp = L.c_kv_pool(FAKE, lay)
    opts = L.c_pipeline_opts()
    ctx = ctypes.c_void_p()
    rc = oc.lib().oc_context_create(4096, ctypes.byref(kp), ctypes.byref(opts), 256, 32, ctypes.byref(ctx))
    assert rc == L.OC_EINVAL and not ctx.value
    assert b"no such device" in oc.lib().oc_last_error()


def test_lengths_past_the_kernels_32bit_arithmetic_are_rejected():
    big = _layout(num_layers=2, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=1 << 26)
    ws = oc.lib().oc_attention_workspace_bytes
    # suffix K/V byte offsets: T_s * n_kv * d * 2 must stay below 2^31
    assert ws(ctypes.byref(big), 4096, (1 << 20) - 1) > 0
    assert ws(ctypes.byref(big), 4096, 1 << 20) == 0
    assert b"2^31" in oc.lib().oc_last_error()
    # key positions: prefix + suffix tokens up to 2^30
    assert ws(ctypes.byref(big), (1 << 30) - 512, 512) > 0
    assert ws(ctypes.byref(big), (1 << 30) - 511, 512) == 0
    assert b"2^30" in oc.lib().oc_last_error()
    # the single-layer call rejects the same lengths before launching anything
    bt = L.c_block_table(FAKE, 1 << 26, 4096)
    kp = L.c_kv_pool(FAKE, big)
    f = oc.lib().oc_suffix_prefill_layer
    assert f(FAKE, FAKE, FAKE, 1 << 20, ctypes.byref(kp), ctypes.byref(bt), 0, FAKE, FAKE, 1 << 40, None) == \
        L.OC_ERANGE
    g = oc.lib().oc_suffix_prefill_layer_noalloc
    assert g(FAKE, FAKE, FAKE, 1 << 20, ctypes.byref(kp), ctypes.byref(bt), 0, FAKE, None) == L.OC_ERANGE
    bt_long = L.c_block_table(FAKE, 1 << 26, (1 << 30) - 16)
    assert f(FAKE, FAKE, FAKE, 512, ctypes.byref(kp), ctypes.byref(bt_long), 0, FAKE, FAKE, 1 << 40, None) == \
        L.OC_ERANGE
    # a context for such lengths is refused before any device is touched
    opts = L.c_pipeline_opts()
    ctx = ctypes.c_void_p()
    rc = oc.lib().oc_context_create(0, ctypes.byref(kp), ctypes.byref(opts), 4096, 1 << 20, ctypes.byref(ctx))
    assert rc == L.OC_ERANGE and not ctx.value


def test_copies_past_a_32bit_grid_are_rejected():
    # 2^24 prefix tokens of 8 heads x 128 dims are 2^32 16-byte pieces per layer
    lay = _layout(num_layers=2, num_q_heads=32, num_kv_heads=8, head_dim=128, num_pages=1 << 21)
    n = 1 << 24
    ok = n - 16
    assert _ingest(lay, num_chunks=n // 16, table_entries=1 << 20, num_tokens=n) == L.OC_ERANGE
    assert b"2^32" in oc.lib().oc_last_error()
    st = L.c_staging(FAKE, n // 16, 2 * 16 * 8 * 128 * 2)
    bt = L.c_block_table(FAKE, 1 << 20, n)
    kp = L.c_kv_pool(FAKE, lay)
    assert oc.lib().oc_kv_chunks_ingest(ctypes.byref(st), 0, ctypes.byref(bt), ctypes.byref(kp), None) == \
        L.OC_ERANGE
    assert oc.lib().oc_kv_layer_gather(ctypes.byref(bt), ctypes.byref(kp), 0, FAKE, n // 16, 2 * 16 * 8 * 128 * 2,
                                       None) == L.OC_ERANGE
    assert oc.lib().oc_kv_chunks_gather(ctypes.byref(bt), ctypes.byref(kp), 0, n // 16, FAKE, None) == L.OC_ERANGE
    # the append moves K and V in two grid rows: 2^25 tokens are 2^32 pieces of each
    bt0 = L.c_block_table(FAKE, 1 << 21, 0)
    assert oc.lib().oc_kv_suffix_append(FAKE, FAKE, 1 << 25, ctypes.byref(bt0), ctypes.byref(kp), 0, None) == \
        L.OC_ERANGE
    # one chunk fewer is accepted by validation (it is not launched here: the
    # NULL data pointer stops it)
    assert _ingest(lay, num_chunks=ok // 16, table_entries=1 << 20, num_tokens=ok, data=None) == L.OC_EINVAL


def test_noalloc_attention_validation_and_workspace_bound():
    lay = _layout()
    bt = L.c_block_table(FAKE, 16, 256)
    kp = L.c_kv_pool(FAKE, lay)
    g = oc.lib().oc_suffix_prefill_layer_noalloc
    args = [FAKE, FAKE, FAKE, 32, ctypes.byref(kp), ctypes.byref(bt), 0, FAKE, None]
    for i, v, want in ((3, 0, L.OC_EINVAL), (0, FAKE + 4, L.OC_EALIGN), (7, None, L.OC_EINVAL), (6, 2, L.OC_ERANGE)):
        bad = list(args)
        bad[i] = v
        assert g(*bad) == want, (i, v)
    lay96 = _layout(head_dim=96)
    assert g(FAKE, FAKE, FAKE, 32, ctypes.byref(L.c_kv_pool(FAKE, lay96)), ctypes.byref(bt), 0, FAKE, None) == \
        L.OC_ESHAPE
    # every accepted shape's workspace fits the static array: fewer than 512
    # (row tile, key split) pairs; the largest comes from 255 row tiles split in two
    ws = oc.lib().oc_attention_workspace_bytes
    worst = _layout(num_q_heads=1, num_kv_heads=1, head_dim=128, num_pages=1 << 16)
    w = ws(ctypes.byref(worst), 65536, 255 * 256)
    assert 64 << 20 < w <= L.OC_NOALLOC_WORKSPACE_BYTES
    rng = np.random.default_rng(0)
    for _ in range(3000):
        nkv = int(rng.choice([1, 2, 4, 8, 16]))
        grp = int(rng.choice([1, 2, 4, 8]))
        d = int(rng.choice([64, 128]))
        lay_r = _layout(num_q_heads=nkv * grp, num_kv_heads=nkv, head_dim=d, num_pages=1 << 20)
        ts = int(rng.integers(1, 1 << int(rng.integers(1, 18))))
        tp = int(rng.integers(0, 1 << int(rng.integers(1, 22))))
        n = ws(ctypes.byref(lay_r), tp, ts)
        assert 0 < n <= L.OC_NOALLOC_WORKSPACE_BYTES, (nkv, grp, d, tp, ts, n)
