"""Host-side checks of the C ABI: the library loads, exports every declared
symbol, and rejects bad arguments before touching the GPU.  No kernel is
launched here, so these run without a GPU."""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2602_07721_amd as pk
import workloads
from oracle import quantizer

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pariskv.h")

pytestmark = pytest.mark.skipif(not os.path.exists(pk.LIB_PATH), reason="library not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pariskv_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 12
    L = pk.lib()
    for n in names:
        assert hasattr(L, n), n
    assert L.pariskv_abi_version() == pk.ABI_VERSION == 4


def test_error_strings():
    L = pk.lib()
    for code in (0, -1, -2, -3, -4, -5):
        assert L.pariskv_strerror(code)


def test_quantizer_table_is_bit_identical_to_the_oracle():
    # The library derives the table in closed form with binary128 arithmetic,
    # the oracle through Beta incomplete integrals in mpmath; both round the
    # same fixed point to double.
    tau_l, a_l = pk.quantizer_table(8)
    tau_o, a_o, _ = quantizer.lloyd_max(8)
    assert [x.hex() for x in tau_l] == [float(x).hex() for x in tau_o]
    assert [x.hex() for x in a_l] == [float(x).hex() for x in a_o]
    with pytest.raises(pk.PariskvError) as e:
        pk.quantizer_table(4)
    assert e.value.code == pk.ERR_UNSUPPORTED


def _cfg(**kw):
    base = dict(n_kv_heads=8, q_per_kv=4, capacity=4096, rot_signs=workloads.rotation_signs(0))
    base.update(kw)
    return pk.Config(**base)


FAKE = 1 << 20  # an aligned address that is never dereferenced: validation fails first


def _index(ids=FAKE, rec=FAKE, counts=FAKE):
    return pk._Index(ids, rec, counts)


def _encode(cfg, idx, keys=FAKE, n=16, batch=1):
    L = pk.lib()
    return L.pariskv_encode(cfg.c(), ctypes.byref(idx), ctypes.c_void_p(keys), n, batch, None)


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=100), pk.ERR_INVALID),
    (dict(head_dim=64, n_subspaces=8), pk.ERR_UNSUPPORTED),
    (dict(n_subspaces=32), pk.ERR_UNSUPPORTED),
    (dict(n_kv_heads=0), pk.ERR_INVALID),
    (dict(q_per_kv=0), pk.ERR_INVALID),
    (dict(q_per_kv=17), pk.ERR_INVALID),
    (dict(capacity=0), pk.ERR_INVALID),
    (dict(capacity=1 << 31), pk.ERR_INVALID),
])
def test_config_validation(kw, code):
    assert _encode(_cfg(**kw), _index()) == code


def test_sign_validation():
    s = workloads.rotation_signs(0).copy()
    s[5] = 0
    assert _encode(_cfg(rot_signs=s), _index()) == pk.ERR_INVALID
    assert b"rot_signs[5]" in pk.lib().pariskv_last_error()


def test_encode_pointer_and_capacity_validation():
    cfg = _cfg()
    assert _encode(cfg, _index(ids=0)) == pk.ERR_INVALID
    assert _encode(cfg, _index(rec=FAKE + 8)) == pk.ERR_INVALID
    assert _encode(cfg, _index(), keys=0) == pk.ERR_INVALID
    assert _encode(cfg, _index(), keys=FAKE + 2) == pk.ERR_INVALID
    assert _encode(cfg, _index(), n=-1) == pk.ERR_INVALID
    assert _encode(cfg, _index(), n=4097) == pk.ERR_CAPACITY
    assert _encode(cfg, _index(), batch=0) == pk.ERR_INVALID
    L = pk.lib()
    rc = L.pariskv_append(cfg.c(), ctypes.byref(_index()), ctypes.c_void_p(FAKE), 4000, 97, 1, None)
    assert rc == pk.ERR_CAPACITY


def test_workspace_layout_is_consistent():
    cfg = _cfg()
    b = pk.Budget(512, 1024, 64)
    lay = pk.workspace_layout(cfg, 2, 4000, b)
    assert lay["total"] == pk.retrieve_workspace_size(cfg, 2, 4000, b)
    assert lay["n_pad"] == 4032 and lay["n_chunks"] == 1 and lay["c_eff"] == 512 and lay["quads"] == 1
    offs = [lay[k] for k in ("zq", "lut", "score8", "chunk_sfx", "chunk_base", "thresh", "cand",
                             "cand_score", "stats", "surv", "group_rows", "group_part")]
    assert offs == sorted(offs) and all(o % 256 == 0 for o in offs) and lay["total"] >= offs[-1]
    # the regions a plain call does not use are empty
    assert lay["surv"] == lay["group_rows"] == lay["group_part"] == lay["total"]
    assert lay["topk_parts"] == 1 and lay["group_splits"] == 0
    assert lay["score8"] - lay["lut"] >= 2 * 8 * 1 * 16 * 256 * 4
    lay2 = pk.workspace_layout(_cfg(q_per_kv=6), 1, 100, pk.Budget(512, 1024, 64))
    assert lay2["quads"] == 2 and lay2["c_eff"] == 100
    assert pk.workspace_layout(cfg, 1, 0, b)["n_chunks"] == 0


@pytest.mark.parametrize("budget,n,code", [
    ((0, 10, 1), 100, pk.ERR_INVALID),
    ((10, 0, 1), 100, pk.ERR_INVALID),
    ((10, 10, 11), 100, pk.ERR_INVALID),
    ((10, 10, 0), 100, pk.ERR_INVALID),
    ((70000, 10, 5), 100, pk.ERR_UNSUPPORTED),
    ((4000, 4000, 3000), 100, pk.ERR_UNSUPPORTED),
    ((10, 10, 5), 5000, pk.ERR_INVALID),     # n > capacity
    ((10, 10, 5), -1, pk.ERR_INVALID),
])
def test_retrieve_budget_validation(budget, n, code):
    cfg = _cfg()
    b = pk.Budget(*budget)
    L = pk.lib()
    rc = L.pariskv_retrieve(cfg.c(), ctypes.byref(_index()), ctypes.c_void_p(FAKE), n, 1, b.c(),
                            ctypes.c_void_p(FAKE), None, ctypes.c_void_p(FAKE), 1 << 40, None)
    assert rc == code
    assert L.pariskv_retrieve_workspace(cfg.c(), 1, n, b.c()) == 0


def test_retrieve_workspace_validation():
    cfg = _cfg()
    b = pk.Budget(512, 1024, 64)
    need = pk.retrieve_workspace_size(cfg, 1, 4000, b)
    L = pk.lib()
    args = lambda ws, size: (cfg.c(), ctypes.byref(_index()), ctypes.c_void_p(FAKE), 4000, 1, b.c(),
                             ctypes.c_void_p(FAKE), None, ctypes.c_void_p(ws), size, None)
    assert L.pariskv_retrieve(*args(FAKE, need - 1)) == pk.ERR_WORKSPACE
    assert L.pariskv_retrieve(*args(FAKE + 128, need)) == pk.ERR_WORKSPACE
    assert L.pariskv_retrieve(*args(0, need)) == pk.ERR_WORKSPACE


def test_sparse_attend_validation():
    cfg = _cfg()
    L = pk.lib()

    def call(k=8, host=0, cap=4096, scale=0.1, idx=FAKE, out=FAKE):
        return L.pariskv_sparse_attend(cfg.c(), ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE),
                                       ctypes.c_void_p(FAKE), host, cap, ctypes.c_void_p(idx), k, 1,
                                       ctypes.c_float(scale), ctypes.c_void_p(out), None)
    assert call(k=0) == pk.ERR_INVALID
    assert call(host=2) == pk.ERR_INVALID
    assert call(cap=0) == pk.ERR_INVALID
    assert call(scale=float("nan")) == pk.ERR_INVALID
    assert call(idx=FAKE + 2) == pk.ERR_INVALID
    assert call(out=0) == pk.ERR_INVALID


def test_id_slot_encoding_spreads_near_ids_over_banks():
    # The documented stored form of a centroid id: a bijection, its own inverse,
    # and ids within Hamming distance 3 never share a value mod 32.
    from parity import SLOT
    s = SLOT.astype(np.int64)
    assert sorted(s.tolist()) == list(range(256))
    assert np.all(s[s] == np.arange(256))
    assert np.all((s >> 5) == (np.arange(256) >> 5))
    for c in range(256):
        for d in range(1, 256):
            if bin(d).count("1") <= 3:
                assert s[c] % 32 != s[c ^ d] % 32, (c, d)


def test_rotation_signs_match_the_oracle():
    from oracle import rotation
    for seed in (0, 1, 977, 2**63 + 11):
        for D in (1, 7, 128, 256):
            np.testing.assert_array_equal(pk.rotation_signs(seed, D), rotation.seeded_signs(seed, D))
    L = pk.lib()
    out = (ctypes.c_int8 * 4)()
    assert L.pariskv_rotation_signs(ctypes.c_uint64(1), 0, out) == pk.ERR_INVALID
    assert L.pariskv_rotation_signs(ctypes.c_uint64(1), 4, None) == pk.ERR_INVALID


def test_retrieve_attend_validation():
    cfg = _cfg()
    b = pk.Budget(512, 1024, 64)
    need = pk.retrieve_workspace_size(cfg, 1, 4000, b)
    L = pk.lib()

    def call(K=FAKE, V=FAKE, host=0, cap=4096, scale=0.1, out=FAKE, ws=FAKE, size=None):
        return L.pariskv_retrieve_attend(cfg.c(), ctypes.byref(_index()), ctypes.c_void_p(FAKE), 4000, 1,
                                         b.c(), ctypes.c_void_p(FAKE), None, ctypes.c_void_p(K),
                                         ctypes.c_void_p(V), host, cap, ctypes.c_float(scale),
                                         ctypes.c_void_p(out), ctypes.c_void_p(ws),
                                         need if size is None else size, None)
    assert call(K=0) == pk.ERR_INVALID
    assert call(V=FAKE + 4) == pk.ERR_INVALID
    assert call(out=0) == pk.ERR_INVALID
    assert call(host=3) == pk.ERR_INVALID
    assert call(cap=0) == pk.ERR_INVALID
    assert call(scale=float("inf")) == pk.ERR_INVALID
    assert call(size=need - 1) == pk.ERR_WORKSPACE


def test_noalloc_validation_before_any_hip_call():
    # The shapes are checked against the 64 MiB static scratch before the library
    # touches HIP (no device here): 8 x 32 query heads over 300000 keys need more.
    L = pk.lib()
    b = pk.Budget(8192, 16384, 512)

    def call(cfg, n, batch, K=FAKE, out=FAKE, bud=b):
        return L.pariskv_retrieve_attend_noalloc(cfg.c(), ctypes.byref(_index()), ctypes.c_void_p(FAKE), n,
                                                 batch, bud.c(), ctypes.c_void_p(FAKE), None,
                                                 ctypes.c_void_p(K), ctypes.c_void_p(FAKE), 0, 4096,
                                                 ctypes.c_float(0.1), ctypes.c_void_p(out), None)
    big = _cfg(capacity=300000)
    assert pk.retrieve_workspace_size(big, 8, 300000, b) > pk.NOALLOC_SCRATCH_BYTES
    assert call(big, 300000, 8) == pk.ERR_WORKSPACE
    assert b"static scratch" in L.pariskv_last_error()
    # the bench workload's intermediates fit
    assert pk.retrieve_workspace_size(_cfg(capacity=131072), 8, 131072, b) <= pk.NOALLOC_SCRATCH_BYTES
    small = _cfg()
    assert call(small, 5000, 1) == pk.ERR_INVALID                       # n above capacity
    assert call(small, 4000, 1, bud=pk.Budget(512, 1024, 600)) == pk.ERR_INVALID  # k > C
    assert pk.NOALLOC_SCRATCH_BYTES == 64 << 20


@pytest.mark.parametrize("P,sink,local,m", [(10, 2, 4, 3), (5, 4, 4, 2), (2000, 128, 512, 256), (2000, 128, 512, 512),
                                            (700, 128, 512, 256), (100, 128, 512, 64), (3000, 0, 512, 1),
                                            (1000, 16, 8, 32), (0, 128, 512, 256), (130, 128, 512, 7)])
def test_window_regions_match_the_oracle_replay(P, sink, local, m):
    # The library's closed form against the oracle's token-by-token replay of Sec. "Buffer Update".
    from oracle import window
    R = window.after_prefill(P, sink, local, m)
    for t in range(0, 1200):
        if t > 0:
            window.decode_step(R)
        w, n = pk.window_regions(P, t, sink, local, m)
        assert (w.sink_len, w.retr_begin) == (len(R.sink), len(R.sink)), t
        assert n == len(R.retrieval), t
        assert list(range(w.retr_begin, w.retr_begin + n)) == R.retrieval, t
        assert list(range(w.dense_begin, w.dense_end)) == R.local + R.buffer, t


def test_window_regions_validation():
    L = pk.lib()
    w, n = pk._Window(), ctypes.c_int64()
    for args in ((-1, 0, 1, 1, 1), (1, -1, 1, 1, 1), (1, 0, -1, 1, 1), (1, 0, 1, -1, 1), (1, 0, 1, 1, 0),
                 (2**41, 0, 1, 1, 1)):
        assert L.pariskv_window_regions(*args, ctypes.byref(w), ctypes.byref(n)) == pk.ERR_INVALID
    assert L.pariskv_window_regions(1, 0, 1, 1, 1, None, ctypes.byref(n)) == pk.ERR_INVALID


def test_window_attend_validation():
    cfg = _cfg()
    L = pk.lib()

    def call(win, k=8, cap=4096):
        return L.pariskv_window_attend(cfg.c(), ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE),
                                       ctypes.c_void_p(FAKE), 0, cap, ctypes.c_void_p(FAKE), k,
                                       None if win is None else win.c(), 1, ctypes.c_float(0.1),
                                       ctypes.c_void_p(FAKE), None)
    W = pk.Window
    assert call(None) == pk.ERR_INVALID
    assert call(W(-1, 0, 0, 0)) == pk.ERR_INVALID                 # negative sink
    assert call(W(8, 4, 10, 12)) == pk.ERR_INVALID                # retrieval before the sink ends
    assert call(W(4, 4, 3, 12)) == pk.ERR_INVALID                 # dense before retrieval
    assert call(W(4, 4, 10, 9)) == pk.ERR_INVALID                 # empty range reversed
    assert call(W(4, 4, 10, 5000)) == pk.ERR_INVALID              # past the cache
    assert call(W(128, 128, 3000, 4000), k=2969) == pk.ERR_UNSUPPORTED  # 128 + 1000 + 2969 = 4097 rows
    # (every case here fails validation: a valid window would launch a kernel on fake pointers)


def test_retrieve_window_attend_validation():
    cfg = _cfg()
    b = pk.Budget(512, 1024, 64)
    need = pk.retrieve_workspace_size(cfg, 1, 4000, b)
    L = pk.lib()

    def call(win, n=4000, cap=8192):
        return L.pariskv_retrieve_window_attend(cfg.c(), ctypes.byref(_index()), ctypes.c_void_p(FAKE), n, 1,
                                                b.c(), ctypes.c_void_p(FAKE), None, ctypes.c_void_p(FAKE),
                                                ctypes.c_void_p(FAKE), 0, cap,
                                                None if win is None else win.c(), ctypes.c_float(0.1),
                                                ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), need, None)
    W = pk.Window
    assert call(None) == pk.ERR_INVALID
    assert call(W(128, 128, 4000, 4600)) == pk.ERR_INVALID        # retrieval rows run into the dense rows
    assert call(W(128, 128, 4128, 9000)) == pk.ERR_INVALID        # past the cache
    assert call(W(2048, 2048, 6048, 8192)) == pk.ERR_UNSUPPORTED  # 2048 + 2144 + 64 rows > 4096


def test_append_rows_validation():
    cfg = _cfg()
    L = pk.lib()

    def call(cap=4096, row_begin=0, n_cur=0, t=16, K=FAKE):
        return L.pariskv_append_rows(cfg.c(), ctypes.byref(_index()), ctypes.c_void_p(K), cap, row_begin,
                                     n_cur, t, 1, None)
    assert call(cap=0) == pk.ERR_INVALID
    assert call(row_begin=-1) == pk.ERR_INVALID
    assert call(row_begin=4090, t=7) == pk.ERR_INVALID            # rows past the cache
    assert call(t=-1) == pk.ERR_INVALID
    assert call(K=0) == pk.ERR_INVALID
    assert call(n_cur=4090, t=16) == pk.ERR_CAPACITY              # index rows past its capacity


def test_variant_flag_validation():
    L = pk.lib()
    bad = _cfg(flags=4)
    b = pk.Budget(512, 1024, 64)
    assert L.pariskv_retrieve_workspace(bad.c(), 1, 4000, b.c()) == 0
    assert _encode(bad, _index()) == pk.ERR_INVALID
    assert pk.retrieve_workspace_size(_cfg(flags=pk.NO_ROTATION | pk.NO_ALPHA_CORRECTION), 1, 4000, b) > 0
    assert L.pariskv_retrieve_workspace(_cfg().c(), 1, 4000, pk.Budget(512, 1024, 64, flags=8).c()) == 0
    every = pk.BINARY_COLLISIONS | pk.EXACT_RECOUNT | pk.GROUP_FETCH
    assert every == 7 and pk.retrieve_workspace_size(_cfg(), 1, 4000, pk.Budget(512, 1024, 64, flags=every)) > 0
    assert pk.retrieve_workspace_size(_cfg(), 1, 4000, pk.Budget(512, 1024, 64, flags=pk.EXACT_RECOUNT)) > 0
    assert pk.retrieve_workspace_size(_cfg(), 1, 4000, pk.Budget(512, 1024, 64, flags=pk.BINARY_COLLISIONS)) > 0


def test_tiered_attend_and_offload_validation():
    cfg = _cfg()
    L = pk.lib()
    W = pk.Window

    def call(win, wcap=1000, kw=FAKE, k=8, cap=4096):
        return L.pariskv_tiered_attend(cfg.c(), ctypes.c_void_p(FAKE), ctypes.c_void_p(kw), ctypes.c_void_p(FAKE),
                                       wcap, ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), 0, cap,
                                       ctypes.c_void_p(FAKE), k, None if win is None else win.c(), 1,
                                       ctypes.c_float(0.1), ctypes.c_void_p(FAKE), None)
    assert call(None) == pk.ERR_INVALID
    assert call(W(128, 128, 3000, 3600), kw=0) == pk.ERR_INVALID           # no window cache
    assert call(W(128, 128, 3000, 3600), wcap=0) == pk.ERR_INVALID
    assert call(W(128, 128, 3000, 3600), wcap=700) == pk.ERR_INVALID       # 128 + ring 572 < 600 rows
    assert call(W(128, 128, 3000, 3600), wcap=2 ** 30) == pk.ERR_INVALID  # past the row limit
    assert call(W(128, 128, 3000, 3600), cap=2 ** 30) == pk.ERR_INVALID    # main cache past the limit
    assert call(W(128, 128, 3000, 3600), k=3400) == pk.ERR_UNSUPPORTED     # 128 + 600 + 3400 rows
    # dense rows may lie past the main cache: they live in the window cache (would launch: not run here)

    def off(src_row=0, dst_row=0, t=16, scap=100, dcap=100, kd=FAKE):
        return L.pariskv_offload_rows(ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), scap, src_row,
                                      ctypes.c_void_p(kd), ctypes.c_void_p(FAKE), dcap, dst_row, t, 1, 8, None)
    assert off(kd=0) == pk.ERR_INVALID
    assert off(src_row=90) == pk.ERR_INVALID
    assert off(dst_row=-1) == pk.ERR_INVALID
    assert off(t=-1) == pk.ERR_INVALID
    assert off(dcap=0) == pk.ERR_INVALID
    assert off(t=0) == pk.OK                                               # nothing to copy


def test_group_attend_validation():
    L = pk.lib()

    def call(cfg, k=256, union=FAKE, cap=4096):
        return L.pariskv_group_attend(cfg.c(), ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), 0,
                                      cap, ctypes.c_void_p(FAKE), k, 1, ctypes.c_float(0.1), ctypes.c_void_p(FAKE),
                                      ctypes.c_void_p(union), None)
    assert call(_cfg(), k=1025) == pk.ERR_UNSUPPORTED        # 4 heads x 1025 entries per quad
    assert call(_cfg(q_per_kv=2), k=2049) == pk.ERR_UNSUPPORTED
    assert call(_cfg(), k=0) == pk.ERR_INVALID
    assert call(_cfg(), union=FAKE + 2) == pk.ERR_INVALID
    assert call(_cfg(), cap=2 ** 30) == pk.ERR_INVALID


def test_binding_refuses_mismatched_tensors_before_any_launch():
    # The Python binding derives sizes from tensor shapes; a wrong dtype or shape is refused
    # on the host (CPU tensors here: the checks run before the device check and the call).
    import torch
    signs = workloads.rotation_signs(3)
    cfg = pk.Config(2, 4, 64, signs)
    f16 = torch.float16
    keys = torch.zeros((1, 2, 64, 128), dtype=f16)
    index = pk.Index(torch.zeros((1, 2, 64, 16), dtype=torch.uint8), torch.zeros((1, 2, 64, 128), dtype=torch.uint8),
                     torch.zeros((1, 2, 16, 256), dtype=torch.int32))
    with pytest.raises(TypeError, match="keys must be torch.float16"):
        pk.encode(cfg, index, keys.to(torch.int8))
    with pytest.raises(ValueError, match="keys must have shape"):
        pk.encode(cfg, index, torch.zeros((1, 3, 64, 128), dtype=f16))     # 3 KV heads, config has 2
    with pytest.raises(ValueError, match="keys must have shape"):
        pk.encode(cfg, index, torch.zeros((1, 2, 64, 64), dtype=f16))      # D = 64
    with pytest.raises(ValueError, match="must be a GPU tensor"):
        pk.encode(cfg, index, keys)                                        # right shapes, host memory
    short = pk.Index(index.ids[:, :, :32].contiguous(), index.rec, index.counts)
    with pytest.raises(ValueError, match="index.ids must have shape"):
        short.c(cfg, 1)                                                    # rows below the capacity
    with pytest.raises(TypeError, match="index.counts must be torch.int32"):
        pk.Index(index.ids, index.rec, index.counts.long()).c(cfg, 1)

    bud = pk.Budget(16, 32, 8)
    q = torch.zeros((1, 8, 128), dtype=f16)
    ws = torch.zeros(1024, dtype=torch.uint8)
    with pytest.raises(TypeError, match="q must be torch.float16"):
        pk.retrieve(cfg, index, q.float(), 64, bud, workspace=ws)
    with pytest.raises(ValueError, match="q must have shape"):
        pk.retrieve(cfg, index, torch.zeros((1, 4, 128), dtype=f16), 64, bud, workspace=ws)
    with pytest.raises(ValueError, match="out_idx must have shape"):
        pk.retrieve(cfg, index, q, 64, bud, out_idx=torch.zeros((1, 8, 4), dtype=torch.int32), workspace=ws)
    with pytest.raises(TypeError, match="out_score must be torch.float32"):
        pk.retrieve(cfg, index, q, 64, bud, out_idx=torch.zeros((1, 8, 8), dtype=torch.int32),
                    out_score=torch.zeros((1, 8, 8), dtype=torch.float64), workspace=ws)

    K = torch.zeros((1, 2, 64, 128), dtype=f16)
    idx = torch.zeros((1, 8, 8), dtype=torch.int32)
    with pytest.raises(TypeError, match="idx must be torch.int32"):
        pk.sparse_attend(cfg, q, K, K, idx.long(), 0.1)
    with pytest.raises(ValueError, match="V must have shape"):
        pk.sparse_attend(cfg, q, K, K[:, :, :32].contiguous(), idx, 0.1)  # V rows != K rows
    with pytest.raises(ValueError, match="must be pinned host memory"):
        pk.sparse_attend(cfg, q, K, K, idx, 0.1, kv_host_mapped=True)      # pageable host memory
    with pytest.raises(ValueError, match="out must have shape"):
        pk.sparse_attend(cfg, q, K, K, idx, 0.1, out=torch.zeros((1, 8, 64), dtype=torch.float32))
    with pytest.raises(ValueError, match="union_rows must have shape"):
        pk.group_attend(cfg, q, K, K, idx, 0.1, union_rows=torch.zeros((1, 2, 2), dtype=torch.int32))
    with pytest.raises(ValueError, match="K_win must have shape"):
        pk.tiered_attend(cfg, q, torch.zeros((1, 1, 16, 128), dtype=f16), K, K, K, idx, pk.Window(), 0.1)
    with pytest.raises(ValueError, match="V_dst must have shape"):
        pk.offload_rows(K, K, 0, K, K[:1, :1].contiguous(), 0, 4)


def test_stream_kernels_validation():
    L = pk.lib()
    assert L.pariskv_stream_copy(ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), 100, None) == pk.ERR_INVALID
    assert L.pariskv_stream_copy(ctypes.c_void_p(FAKE + 4), ctypes.c_void_p(FAKE), 256, None) == pk.ERR_INVALID
    assert L.pariskv_stream_copy(None, ctypes.c_void_p(FAKE), 256, None) == pk.ERR_INVALID
    assert L.pariskv_stream_read(ctypes.c_void_p(FAKE), 100, 0, ctypes.c_void_p(FAKE), None) == pk.ERR_INVALID
    assert L.pariskv_stream_read(ctypes.c_void_p(FAKE), 256, 0, None, None) == pk.ERR_INVALID


def test_group_fetch_validation():
    # PARISKV_GROUP_FETCH: min(G, 4) * k within one block's list, n within 64 key ranges
    L = pk.lib()
    cfg = _cfg()
    ok = pk.Budget(512, 1024, 64, flags=pk.GROUP_FETCH)
    lay = pk.workspace_layout(cfg, 1, 4000, ok)
    assert lay["group_rows"] > 0 and lay["total"] >= lay["group_rows"] + 8 * 4
    # 8 quads with 4 x 64 entries each: one block per quad (a share needs >= 256 rows)
    assert lay["group_splits"] == 1 and lay["group_part"] == lay["total"]
    assert pk.workspace_layout(cfg, 1, 4000, pk.Budget(512, 1024, 64))["group_splits"] == 0
    # the host1m shape: 8 quads of 4 x 1024 entries -> 16 shares each, states of 4 x 132 floats
    h1m = pk.workspace_layout(pk.Config(8, 4, 1 << 20, workloads.rotation_signs(0)), 1, 1 << 20,
                              pk.Budget(32768, 65536, 1024, flags=pk.GROUP_FETCH))
    assert h1m["group_splits"] == 16 and h1m["group_part"] > h1m["group_rows"]
    assert h1m["total"] - h1m["group_part"] == 8 * 16 * 4 * 132 * 4
    # batch 8 of the same: 64 quads -> 4 shares each
    b8 = pk.workspace_layout(pk.Config(8, 4, 1 << 17, workloads.rotation_signs(0)), 8, 1 << 17,
                             pk.Budget(8192, 16384, 512, flags=pk.GROUP_FETCH))
    assert b8["group_splits"] == 4
    # G = 2: 2 x 64 entries per quad, too few to share
    g2 = pk.workspace_layout(_cfg(q_per_kv=2), 1, 4000, ok)
    assert g2["group_splits"] == 1
    # key ranges of at most 65536: 1.1M keys need 17 shares even where 16 would do
    big = pk.Config(8, 4, 1100000, workloads.rotation_signs(0))
    assert pk.workspace_layout(big, 1, 1100000, pk.Budget(8192, 16384, 1024, flags=pk.GROUP_FETCH))[
        "group_splits"] == 17
    assert pk.workspace_layout(big, 1, 1100000, pk.Budget(8192, 16384, 16, flags=pk.GROUP_FETCH))[
        "group_splits"] == 17
    # beyond 64 ranges of 65536 keys the flag is refused
    huge = pk.Config(1, 4, 5000000, workloads.rotation_signs(0))
    hb = pk.Budget(8192, 16384, 64, flags=pk.GROUP_FETCH)
    need = pk.retrieve_workspace_size(huge, 1, 4200000, hb)
    rc = L.pariskv_retrieve_attend(huge.c(), ctypes.byref(_index()), ctypes.c_void_p(FAKE), 4200000, 1, hb.c(),
                                   ctypes.c_void_p(FAKE), None, ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), 0,
                                   4200000, ctypes.c_float(0.1), ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), need,
                                   None)
    assert rc == pk.ERR_UNSUPPORTED and "4194304" in L.pariskv_last_error().decode()
    big = pk.Budget(8192, 16384, 2048, flags=pk.GROUP_FETCH)   # 4 x 2048 > 4096
    need = pk.retrieve_workspace_size(cfg, 1, 4000, big)
    rc = L.pariskv_retrieve_attend(cfg.c(), ctypes.byref(_index()), ctypes.c_void_p(FAKE), 4000, 1, big.c(),
                                   ctypes.c_void_p(FAKE), None, ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), 0,
                                   4096, ctypes.c_float(0.1), ctypes.c_void_p(FAKE), ctypes.c_void_p(FAKE), need,
                                   None)
    assert rc == pk.ERR_UNSUPPORTED
