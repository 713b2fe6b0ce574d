"""ParisKV decode-step KV retrieval for AMD MI355X (gfx950).

Python binding of ``libpariskv.so`` (declared in ``include/pariskv.h``).  It
only marshals arguments: torch tensors provide device memory and streams,
every step of the path runs in the library's HIP kernels, and a missing
library raises instead of falling back to anything.

Method: ParisKV (arXiv 2602.07721), Alg. 1 -- encode keys into centroid ids,
4-bit codes and weights; per decode step rank clusters, score collisions,
select top-beta candidates, rerank them with the RSQ-IP estimator, keep the
top-k; then attend over the fetched K/V rows only.
"""

import ctypes
import os
from dataclasses import dataclass

import numpy as np

__all__ = [
    "PariskvError", "Config", "Budget", "Index", "Window", "lib", "encode", "append", "append_rows",
    "retrieve", "retrieve_workspace_size", "workspace_layout", "sparse_attend", "retrieve_attend",
    "retrieve_attend_noalloc", "NOALLOC_SCRATCH_BYTES",
    "window_regions", "window_attend", "retrieve_window_attend", "tiered_attend", "retrieve_tiered_attend",
    "offload_rows", "window_slot", "group_attend", "quantizer_table", "rotation_signs",
    "profile_enable", "profile_reset", "profile_read", "stream_copy", "stream_read",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpariskv.so")
# pariskv_abi_version() of the library this binding marshals for (struct layouts, entry points)
ABI_VERSION = 4

OK, ERR_INVALID, ERR_CAPACITY, ERR_WORKSPACE, ERR_HIP, ERR_UNSUPPORTED = 0, -1, -2, -3, -4, -5
HEAD_DIM, SUBSPACES, CENTROIDS, REC_BYTES = 128, 16, 256, 128
MAX_ATTEND_ROWS = 4096
# Ablation variants (Sec. "Ablation Studies"): Config.flags, Budget.flags.
NO_ROTATION, NO_ALPHA_CORRECTION = 1, 2
BINARY_COLLISIONS = 1
# Diagnostic Budget.flags bit: every selection threshold from the exact recount.
EXACT_RECOUNT = 2
# Budget.flags bit for retrieve_attend: GQA-group de-duplication of the K/V fetch.
GROUP_FETCH = 4


class PariskvError(RuntimeError):
    def __init__(self, code, message):
        super().__init__(f"pariskv error {code}: {message}")
        self.code = code


class _Config(ctypes.Structure):
    _fields_ = [("head_dim", ctypes.c_int32), ("n_subspaces", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("q_per_kv", ctypes.c_int32),
                ("capacity", ctypes.c_int64), ("rot_signs", ctypes.POINTER(ctypes.c_int8)),
                ("flags", ctypes.c_uint32)]


class _Index(ctypes.Structure):
    _fields_ = [("ids", ctypes.c_void_p), ("rec", ctypes.c_void_p), ("counts", ctypes.c_void_p)]


class _Budget(ctypes.Structure):
    _fields_ = [("n_cand", ctypes.c_int64), ("n_collide", ctypes.c_int64), ("top_k", ctypes.c_int32),
                ("flags", ctypes.c_int32)]


class _Window(ctypes.Structure):
    _fields_ = [("sink_len", ctypes.c_int64), ("retr_begin", ctypes.c_int64),
                ("dense_begin", ctypes.c_int64), ("dense_end", ctypes.c_int64)]


class _Layout(ctypes.Structure):
    _fields_ = [(name, ctypes.c_size_t) for name in
                ("total", "zq", "lut", "score8", "chunk_sfx", "chunk_base", "thresh", "cand",
                 "cand_score", "stats", "surv", "group_rows", "group_part")] + \
               [(name, ctypes.c_int64) for name in ("n_pad", "n_chunks", "chunk_keys", "c_eff")] + \
               [(name, ctypes.c_int32) for name in ("quads", "topk_parts", "group_splits")]


_lib = None


def lib():
    """The loaded library; raises ImportError when it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2602_07721_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, VP, I32, I64, SZ = ctypes.POINTER, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        L.pariskv_encode.argtypes = [P(_Config), P(_Index), VP, I64, I32, VP]
        L.pariskv_append.argtypes = [P(_Config), P(_Index), VP, I64, I64, I32, VP]
        L.pariskv_append_rows.argtypes = [P(_Config), P(_Index), VP, I64, I64, I64, I64, I32, VP]
        L.pariskv_window_regions.argtypes = [I64, I64, I64, I64, I64, P(_Window), P(I64)]
        L.pariskv_window_attend.argtypes = [P(_Config), VP, VP, VP, I32, I64, VP, I32, P(_Window), I32,
                                            ctypes.c_float, VP, VP]
        L.pariskv_retrieve_window_attend.argtypes = [P(_Config), P(_Index), VP, I64, I32, P(_Budget), VP,
                                                     VP, VP, VP, I32, I64, P(_Window), ctypes.c_float, VP,
                                                     VP, SZ, VP]
        L.pariskv_retrieve_workspace.argtypes = [P(_Config), I32, I64, P(_Budget)]
        L.pariskv_retrieve_workspace.restype = SZ
        L.pariskv_workspace_layout.argtypes = [P(_Config), I32, I64, P(_Budget), P(_Layout)]
        L.pariskv_retrieve.argtypes = [P(_Config), P(_Index), VP, I64, I32, P(_Budget), VP, VP, VP,
                                       SZ, VP]
        L.pariskv_retrieve_attend_noalloc.argtypes = [P(_Config), P(_Index), VP, I64, I32, P(_Budget), VP, VP,
                                                      VP, VP, I32, I64, ctypes.c_float, VP, VP]
        L.pariskv_sparse_attend.argtypes = [P(_Config), VP, VP, VP, I32, I64, VP, I32, I32,
                                            ctypes.c_float, VP, VP]
        L.pariskv_retrieve_attend.argtypes = [P(_Config), P(_Index), VP, I64, I32, P(_Budget), VP, VP,
                                              VP, VP, I32, I64, ctypes.c_float, VP, VP, SZ, VP]
        L.pariskv_tiered_attend.argtypes = [P(_Config), VP, VP, VP, I64, VP, VP, I32, I64, VP, I32, P(_Window),
                                            I32, ctypes.c_float, VP, VP]
        L.pariskv_retrieve_tiered_attend.argtypes = [P(_Config), P(_Index), VP, I64, I32, P(_Budget), VP, VP,
                                                     VP, VP, I64, VP, VP, I32, I64, P(_Window),
                                                     ctypes.c_float, VP, VP, SZ, VP]
        L.pariskv_group_attend.argtypes = [P(_Config), VP, VP, VP, I32, I64, VP, I32, I32, ctypes.c_float, VP,
                                           VP, VP]
        L.pariskv_offload_rows.argtypes = [VP, VP, I64, I64, VP, VP, I64, I64, I64, I32, I32, VP]
        L.pariskv_stream_copy.argtypes = [VP, VP, SZ, VP]
        L.pariskv_stream_read.argtypes = [VP, SZ, ctypes.c_uint32, VP, VP]
        L.pariskv_quantizer_table.argtypes = [I32, P(ctypes.c_double), P(ctypes.c_double)]
        L.pariskv_rotation_signs.argtypes = [ctypes.c_uint64, I32, P(ctypes.c_int8)]
        L.pariskv_profile_enable.argtypes = [I32]
        L.pariskv_profile_read.argtypes = [I32, P(ctypes.c_char_p), P(I64), P(ctypes.c_double)]
        L.pariskv_strerror.restype = ctypes.c_char_p
        L.pariskv_strerror.argtypes = [ctypes.c_int]
        L.pariskv_last_error.restype = ctypes.c_char_p
        L.pariskv_abi_version.restype = I32
        if L.pariskv_abi_version() != ABI_VERSION:
            raise ImportError(f"{LIB_PATH} has ABI version {L.pariskv_abi_version()}, this binding expects "
                              f"{ABI_VERSION}: rebuild the library")
        _lib = L
    return _lib


def _check(rc):
    if rc != OK:
        msg = lib().pariskv_last_error().decode()
        raise PariskvError(rc, msg or lib().pariskv_strerror(rc).decode())
    return rc


@dataclass
class Config:
    """Layer shape, rotation signs and index variant flags (see ``pariskv_config``)."""
    n_kv_heads: int
    q_per_kv: int
    capacity: int
    rot_signs: np.ndarray
    head_dim: int = HEAD_DIM
    n_subspaces: int = SUBSPACES
    flags: int = 0

    def __post_init__(self):
        self._signs = np.ascontiguousarray(np.asarray(self.rot_signs, dtype=np.int8))
        self._c = _Config(self.head_dim, self.n_subspaces, self.n_kv_heads, self.q_per_kv,
                          self.capacity, self._signs.ctypes.data_as(ctypes.POINTER(ctypes.c_int8)),
                          self.flags)

    @property
    def n_q_heads(self):
        return self.n_kv_heads * self.q_per_kv

    def c(self):
        return ctypes.byref(self._c)


@dataclass
class Budget:
    """C = n_cand, C_rho = n_collide, k = top_k, flags (see ``pariskv_budget``)."""
    n_cand: int
    n_collide: int
    top_k: int
    flags: int = 0

    def c(self):
        self._c = _Budget(self.n_cand, self.n_collide, self.top_k, self.flags)
        return ctypes.byref(self._c)


def _ptr(t, name, device=True):
    if t is None:
        return None
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if device and not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _arg(t, name, dtype, shape, dev=None, optional=False):
    """Pointer of a tensor argument after checking its dtype and its shape (None entries are
    free; the sizes the library derives from shapes must be consistent).  The kernels trust
    these, so a mismatch is refused here rather than read past the end of an allocation.
    A tensor that must live on the GPU is appended to the list `dev`, checked by
    _require_device once every argument of the call has passed these checks."""
    import torch
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != len(shape) or any(w is not None and int(d) != int(w) for d, w in zip(t.shape, shape)):
        want = "[" + ", ".join("*" if w is None else str(w) for w in shape) + "]"
        raise ValueError(f"{name} must have shape {want}, got {list(t.shape)}")
    if dev is not None:
        dev.append((t, name))
    return _ptr(t, name, False)


def _require_device(dev):
    for t, name in dev:
        if not t.is_cuda:
            raise ValueError(f"{name} must be a GPU tensor")


def _kv_args(cfg, batch, K, V, kv_host_mapped, dev, names=("K", "V")):
    """Pointers of a K/V cache pair [batch][Hkv][capacity][D] float16 (pinned host memory when
    kv_host_mapped) and its capacity."""
    import torch
    shape = (batch, cfg.n_kv_heads, None, HEAD_DIM)
    kp = _arg(K, names[0], torch.float16, shape, None if kv_host_mapped else dev)
    cap = int(K.shape[2])
    vp = _arg(V, names[1], torch.float16, (batch, cfg.n_kv_heads, cap, HEAD_DIM), None if kv_host_mapped else dev)
    if kv_host_mapped:
        for t, nm in ((K, names[0]), (V, names[1])):
            if t.is_cuda or not t.is_pinned():
                raise ValueError(f"{nm} must be pinned host memory when kv_host_mapped")
    return kp, vp, cap


def _q_arg(cfg, q, dev):
    import torch
    if not isinstance(q, torch.Tensor) or q.dim() != 3:
        raise ValueError("q must be a [batch][Hq][D] tensor")
    batch = int(q.shape[0])
    return _arg(q, "q", torch.float16, (batch, cfg.n_q_heads, HEAD_DIM), dev), batch


def _out_arg(cfg, out, batch, device, dev):
    import torch
    if out is None:
        out = torch.empty((batch, cfg.n_q_heads, HEAD_DIM), dtype=torch.float32, device=device)
    return out, _arg(out, "out", torch.float32, (batch, cfg.n_q_heads, HEAD_DIM), dev)


def _idx_arg(cfg, idx, batch, dev, name="idx"):
    import torch
    if not isinstance(idx, torch.Tensor) or idx.dim() != 3:
        raise ValueError(f"{name} must be a [batch][Hq][k] int32 tensor")
    k = int(idx.shape[-1])
    return _arg(idx, name, torch.int32, (batch, cfg.n_q_heads, k), dev), k


def _retrieve_outs(cfg, budget, batch, out_idx, out_score, workspace, n, device, dev):
    """Allocate what the caller left out and check the rest: (out_idx, out_score, workspace, ptrs)."""
    import torch
    if out_idx is None:
        out_idx = torch.empty((batch, cfg.n_q_heads, budget.top_k), dtype=torch.int32, device=device)
    if workspace is None:
        workspace = torch.empty(max(256, retrieve_workspace_size(cfg, batch, n, budget)),
                                dtype=torch.uint8, device=device)
    rows = (batch, cfg.n_q_heads, budget.top_k)
    ptrs = (_arg(out_idx, "out_idx", torch.int32, rows, dev),
            _arg(out_score, "out_score", torch.float32, rows, dev, optional=True),
            _arg(workspace, "workspace", torch.uint8, (None,), dev))
    return out_idx, out_score, workspace, ptrs


class Index:
    """Device arrays of the per-key metadata (see ``pariskv_index``)."""

    def __init__(self, ids, rec, counts):
        self.ids, self.rec, self.counts = ids, rec, counts

    @classmethod
    def empty(cls, cfg, batch, device="cuda"):
        import torch
        ids = torch.empty((batch, cfg.n_kv_heads, cfg.capacity, SUBSPACES), dtype=torch.uint8, device=device)
        rec = torch.empty((batch, cfg.n_kv_heads, cfg.capacity, REC_BYTES), dtype=torch.uint8, device=device)
        counts = torch.zeros((batch, cfg.n_kv_heads, SUBSPACES, CENTROIDS), dtype=torch.int32, device=device)
        return cls(ids, rec, counts)

    @property
    def batch(self):
        return int(self.ids.shape[0])

    def c(self, cfg=None, batch=None, dev=None):
        if cfg is not None:
            import torch
            b = self.batch if batch is None else batch
            cap = cfg.capacity
            own = dev is None
            dev = [] if own else dev
            ptrs = (_arg(self.ids, "index.ids", torch.uint8, (b, cfg.n_kv_heads, cap, SUBSPACES), dev),
                    _arg(self.rec, "index.rec", torch.uint8, (b, cfg.n_kv_heads, cap, REC_BYTES), dev),
                    _arg(self.counts, "index.counts", torch.int32, (b, cfg.n_kv_heads, SUBSPACES, CENTROIDS), dev))
            if own:
                _require_device(dev)
        else:
            ptrs = (_ptr(self.ids, "ids"), _ptr(self.rec, "rec"), _ptr(self.counts, "counts"))
        self._c = _Index(*ptrs)
        return ctypes.byref(self._c)


def _keys_arg(cfg, keys, dev, name="keys"):
    import torch
    if not isinstance(keys, torch.Tensor) or keys.dim() != 4:
        raise ValueError(f"{name} must be a [batch][Hkv][n][D] float16 tensor")
    b = int(keys.shape[0])
    return _arg(keys, name, torch.float16, (b, cfg.n_kv_heads, None, HEAD_DIM), dev), b


def encode(cfg, index, keys, stream=None):
    """Prefill: encode keys [batch][Hkv][n][D] float16 into rows [0, n); resets counts."""
    dev = []
    kp, b = _keys_arg(cfg, keys, dev)
    ic = index.c(cfg, b, dev)
    _require_device(dev)
    _check(lib().pariskv_encode(cfg.c(), ic, kp, int(keys.shape[2]), b, _stream(stream)))


def append(cfg, index, keys, n_cur, stream=None):
    """Streaming update: encode keys [batch][Hkv][t][D] into rows [n_cur, n_cur + t)."""
    dev = []
    kp, b = _keys_arg(cfg, keys, dev)
    ic = index.c(cfg, b, dev)
    _require_device(dev)
    _check(lib().pariskv_append(cfg.c(), ic, kp, int(n_cur), int(keys.shape[2]), b, _stream(stream)))


def append_rows(cfg, index, K, row_begin, t, n_cur, stream=None):
    """Streaming update from the key cache K [batch][Hkv][kv_capacity][D]: encode cache rows
    [row_begin, row_begin + t) into index rows [n_cur, n_cur + t)."""
    dev = []
    kp, b = _keys_arg(cfg, K, dev, "K")
    ic = index.c(cfg, b, dev)
    _require_device(dev)
    _check(lib().pariskv_append_rows(cfg.c(), ic, kp, int(K.shape[2]), int(row_begin), int(n_cur), int(t), b,
                                     _stream(stream)))


@dataclass
class Window:
    """Rows attended besides the retrieved keys (see ``pariskv_window``): Sink rows
    [0, sink_len), retrieved index row i at cache row retr_begin + i, Local + Update Buffer
    rows [dense_begin, dense_end)."""
    sink_len: int = 0
    retr_begin: int = 0
    dense_begin: int = 0
    dense_end: int = 0

    @property
    def dense_rows(self):
        return self.sink_len + self.dense_end - self.dense_begin

    def c(self):
        self._c = _Window(self.sink_len, self.retr_begin, self.dense_begin, self.dense_end)
        return ctypes.byref(self._c)


def window_regions(P, t, sink=128, local=512, m=256):
    """(Window, n_retrieval) after a prompt of P tokens and t decode steps, buffer updates
    every m steps (Sec. "Buffer Update"); see ``pariskv_window_regions``."""
    w = _Window()
    n = ctypes.c_int64()
    _check(lib().pariskv_window_regions(int(P), int(t), int(sink), int(local), int(m), ctypes.byref(w),
                                        ctypes.byref(n)))
    return Window(w.sink_len, w.retr_begin, w.dense_begin, w.dense_end), int(n.value)


def retrieve_workspace_size(cfg, batch, n, budget):
    return int(lib().pariskv_retrieve_workspace(cfg.c(), batch, n, budget.c()))


def workspace_layout(cfg, batch, n, budget):
    L = _Layout()
    _check(lib().pariskv_workspace_layout(cfg.c(), batch, n, budget.c(), ctypes.byref(L)))
    return {name: getattr(L, name) for name, _ in _Layout._fields_}


def retrieve(cfg, index, q, n, budget, out_idx=None, out_score=None, workspace=None, stream=None):
    """Alg. 1 decode for all query heads; returns (idx, score, workspace) tensors."""
    dev = []
    qp, batch = _q_arg(cfg, q, dev)
    out_idx, out_score, workspace, (ip, sp, wp) = _retrieve_outs(cfg, budget, batch, out_idx, out_score,
                                                                 workspace, n, q.device, dev)
    ic = index.c(cfg, batch, dev)
    _require_device(dev)
    _check(lib().pariskv_retrieve(cfg.c(), ic, qp, int(n), batch, budget.c(), ip, sp, wp,
                                  workspace.numel(), _stream(stream)))
    return out_idx, out_score, workspace


def retrieve_attend(cfg, index, q, n, budget, K, V, scale, out_idx=None, out_score=None, out=None,
                    workspace=None, kv_host_mapped=False, stream=None):
    """retrieve + sparse_attend in one call (the attention runs inside the final top-k kernel);
    returns (idx, score, out, workspace)."""
    dev = []
    qp, batch = _q_arg(cfg, q, dev)
    kp, vp, cap = _kv_args(cfg, batch, K, V, kv_host_mapped, dev)
    out, op = _out_arg(cfg, out, batch, q.device, dev)
    out_idx, out_score, workspace, (ip, sp, wp) = _retrieve_outs(cfg, budget, batch, out_idx, out_score,
                                                                 workspace, n, q.device, dev)
    ic = index.c(cfg, batch, dev)
    _require_device(dev)
    _check(lib().pariskv_retrieve_attend(cfg.c(), ic, qp, int(n), batch, budget.c(), ip, sp,
                                         kp, vp, int(bool(kv_host_mapped)), cap, float(scale), op, wp,
                                         workspace.numel(), _stream(stream)))
    return out_idx, out_score, out, workspace


NOALLOC_SCRATCH_BYTES = 64 << 20


def retrieve_attend_noalloc(cfg, index, q, n, budget, K, V, scale, out_idx, out, out_score=None,
                            kv_host_mapped=False, stream=None):
    """pariskv_retrieve_attend_noalloc: retrieve_attend with the intermediates in the library's
    static per-device scratch array (NOALLOC_SCRATCH_BYTES), for callers that cannot allocate.
    Allocates nothing, so out_idx [batch][Hq][k] int32 and out [batch][Hq][D] float32 must be
    given.  Calls that overlap on one device race on the shared array."""
    import torch
    dev = []
    qp, batch = _q_arg(cfg, q, dev)
    kp, vp, cap = _kv_args(cfg, batch, K, V, kv_host_mapped, dev)
    rows = (batch, cfg.n_q_heads, budget.top_k)
    ip = _arg(out_idx, "out_idx", torch.int32, rows, dev)
    sp = _arg(out_score, "out_score", torch.float32, rows, dev, optional=True)
    op = _arg(out, "out", torch.float32, (batch, cfg.n_q_heads, HEAD_DIM), dev)
    ic = index.c(cfg, batch, dev)
    _require_device(dev)
    _check(lib().pariskv_retrieve_attend_noalloc(cfg.c(), ic, qp, int(n), batch, budget.c(), ip, sp,
                                                 kp, vp, int(bool(kv_host_mapped)), cap, float(scale), op,
                                                 _stream(stream)))
    return out_idx, out_score, out


def sparse_attend(cfg, q, K, V, idx, scale, out=None, kv_host_mapped=False, stream=None):
    """Attention over idx only; K, V [batch][Hkv][kv_capacity][D] float16 (device or pinned host)."""
    dev = []
    qp, batch = _q_arg(cfg, q, dev)
    kp, vp, cap = _kv_args(cfg, batch, K, V, kv_host_mapped, dev)
    xp, k = _idx_arg(cfg, idx, batch, dev)
    out, op = _out_arg(cfg, out, batch, q.device, dev)
    _require_device(dev)
    _check(lib().pariskv_sparse_attend(cfg.c(), qp, kp, vp, int(bool(kv_host_mapped)), cap, xp, k, batch,
                                       float(scale), op, _stream(stream)))
    return out


def window_attend(cfg, q, K, V, idx, win, scale, out=None, kv_host_mapped=False, stream=None):
    """Attention over Sink + retrieved (retr_begin + idx) + Local/Buffer rows of ``win``."""
    dev = []
    qp, batch = _q_arg(cfg, q, dev)
    kp, vp, cap = _kv_args(cfg, batch, K, V, kv_host_mapped, dev)
    xp, k = _idx_arg(cfg, idx, batch, dev)
    out, op = _out_arg(cfg, out, batch, q.device, dev)
    _require_device(dev)
    _check(lib().pariskv_window_attend(cfg.c(), qp, kp, vp, int(bool(kv_host_mapped)), cap, xp, k, win.c(),
                                       batch, float(scale), op, _stream(stream)))
    return out


def retrieve_window_attend(cfg, index, q, n, budget, K, V, win, scale, out_idx=None, out_score=None,
                           out=None, workspace=None, kv_host_mapped=False, stream=None):
    """retrieve over the Retrieval region + window_attend in one call; returns
    (idx, score, out, workspace)."""
    dev = []
    qp, batch = _q_arg(cfg, q, dev)
    kp, vp, cap = _kv_args(cfg, batch, K, V, kv_host_mapped, dev)
    out, op = _out_arg(cfg, out, batch, q.device, dev)
    out_idx, out_score, workspace, (ip, sp, wp) = _retrieve_outs(cfg, budget, batch, out_idx, out_score,
                                                                 workspace, n, q.device, dev)
    ic = index.c(cfg, batch, dev)
    _require_device(dev)
    _check(lib().pariskv_retrieve_window_attend(
        cfg.c(), ic, qp, int(n), batch, budget.c(), ip, sp, kp, vp, int(bool(kv_host_mapped)),
        cap, win.c(), float(scale), op, wp, workspace.numel(), _stream(stream)))
    return out_idx, out_score, out, workspace


def group_attend(cfg, q, K, V, idx, scale, out=None, union_rows=None, kv_host_mapped=False, stream=None):
    """sparse_attend with each distinct K/V row fetched once per KV head (quads of query heads
    attend over the union of their ascending lists); union_rows: optional int32 tensor
    [batch][Hkv][ceil(G/4)] that receives the number of rows fetched."""
    import torch
    dev = []
    qp, batch = _q_arg(cfg, q, dev)
    kp, vp, cap = _kv_args(cfg, batch, K, V, kv_host_mapped, dev)
    xp, k = _idx_arg(cfg, idx, batch, dev)
    out, op = _out_arg(cfg, out, batch, q.device, dev)
    up = _arg(union_rows, "union_rows", torch.int32, (batch, cfg.n_kv_heads, (cfg.q_per_kv + 3) // 4), dev,
              optional=True)
    _require_device(dev)
    _check(lib().pariskv_group_attend(cfg.c(), qp, kp, vp, int(bool(kv_host_mapped)), cap, xp, k, batch,
                                      float(scale), op, up, _stream(stream)))
    return out


def window_slot(r, sink_len, win_capacity):
    """Slot of cache row r in a window cache (see ``pariskv_tiered_attend``)."""
    return r if r < sink_len else sink_len + (r - sink_len) % (win_capacity - sink_len)


def tiered_attend(cfg, q, K_win, V_win, K, V, idx, win, scale, out=None, kv_host_mapped=False, stream=None):
    """window_attend with Sink + Local/Buffer rows read from the GPU window cache K_win/V_win
    [batch][Hkv][win_capacity][D] and the retrieved rows from K/V (pinned host memory when
    kv_host_mapped)."""
    dev = []
    qp, batch = _q_arg(cfg, q, dev)
    kwp, vwp, wcap = _kv_args(cfg, batch, K_win, V_win, False, dev, ("K_win", "V_win"))
    kp, vp, cap = _kv_args(cfg, batch, K, V, kv_host_mapped, dev)
    xp, k = _idx_arg(cfg, idx, batch, dev)
    out, op = _out_arg(cfg, out, batch, q.device, dev)
    _require_device(dev)
    _check(lib().pariskv_tiered_attend(cfg.c(), qp, kwp, vwp, wcap, kp, vp, int(bool(kv_host_mapped)), cap,
                                       xp, k, win.c(), batch, float(scale), op, _stream(stream)))
    return out


def retrieve_tiered_attend(cfg, index, q, n, budget, K_win, V_win, K, V, win, scale, out_idx=None,
                           out_score=None, out=None, workspace=None, kv_host_mapped=False, stream=None):
    """retrieve over the Retrieval region + tiered_attend in one call; returns (idx, score, out, ws)."""
    dev = []
    qp, batch = _q_arg(cfg, q, dev)
    kwp, vwp, wcap = _kv_args(cfg, batch, K_win, V_win, False, dev, ("K_win", "V_win"))
    kp, vp, cap = _kv_args(cfg, batch, K, V, kv_host_mapped, dev)
    out, op = _out_arg(cfg, out, batch, q.device, dev)
    out_idx, out_score, workspace, (ip, sp, wp) = _retrieve_outs(cfg, budget, batch, out_idx, out_score,
                                                                 workspace, n, q.device, dev)
    ic = index.c(cfg, batch, dev)
    _require_device(dev)
    _check(lib().pariskv_retrieve_tiered_attend(
        cfg.c(), ic, qp, int(n), batch, budget.c(), ip, sp, kwp, vwp, wcap, kp, vp,
        int(bool(kv_host_mapped)), cap, win.c(), float(scale), op, wp, workspace.numel(), _stream(stream)))
    return out_idx, out_score, out, workspace


def offload_rows(K_src, V_src, src_row, K_dst, V_dst, dst_row, t, stream=None):
    """Copy rows [src_row, src_row + t) of every (sequence, KV head) of K_src/V_src to rows
    [dst_row, dst_row + t) of K_dst/V_dst (device or pinned host tensors [b][Hkv][cap][D])."""
    import torch
    named = ((K_src, "K_src"), (V_src, "V_src"), (K_dst, "K_dst"), (V_dst, "V_dst"))
    for x, nm in named:
        if not isinstance(x, torch.Tensor) or x.dim() != 4:
            raise ValueError(f"{nm} must be a [batch][Hkv][capacity][D] float16 tensor")
    b, hkv = int(K_src.shape[0]), int(K_src.shape[1])
    src_cap, dst_cap = int(K_src.shape[2]), int(K_dst.shape[2])
    ps = [_arg(x, nm, torch.float16, (b, hkv, c, HEAD_DIM))
          for x, nm, c in ((K_src, "K_src", src_cap), (V_src, "V_src", src_cap),
                           (K_dst, "K_dst", dst_cap), (V_dst, "V_dst", dst_cap))]
    for x, nm in named:
        if not x.is_cuda and not x.is_pinned():
            raise ValueError(f"{nm} must be device or pinned host memory")
    _check(lib().pariskv_offload_rows(ps[0], ps[1], src_cap, int(src_row), ps[2], ps[3], dst_cap, int(dst_row),
                                      int(t), b, hkv, _stream(stream)))


def stream_copy(dst, src, stream=None):
    """Reference streaming copy of src into dst (device tensors of equal byte size, a
    multiple of 16): measurement only."""
    nb = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nb:
        raise ValueError("dst and src must hold the same number of bytes")
    _check(lib().pariskv_stream_copy(_ptr(dst, "dst"), _ptr(src, "src"), nb, _stream(stream)))


def stream_read(src, sink, key=0xFFFFFFFF, stream=None):
    """Reference streaming read of src (a device tensor, multiple of 16 bytes); writes sink
    (a 4-byte device tensor) only if the folded data equals key: measurement only."""
    if sink.numel() * sink.element_size() < 4:
        raise ValueError("sink needs 4 bytes")
    _check(lib().pariskv_stream_read(_ptr(src, "src"), src.numel() * src.element_size(), key,
                                     _ptr(sink, "sink"), _stream(stream)))


def quantizer_table(m=8):
    """(tau[7], a[8]) float64 of the library's offline Lloyd-Max quantizer."""
    tau = (ctypes.c_double * 7)()
    a = (ctypes.c_double * 8)()
    _check(lib().pariskv_quantizer_table(m, tau, a))
    return np.array(tau[:]), np.array(a[:])


def rotation_signs(seed, D=HEAD_DIM):
    """The library's seeded rotation signs s in {+1, -1}^D (int8), see pariskv_rotation_signs."""
    out = (ctypes.c_int8 * D)()
    _check(lib().pariskv_rotation_signs(ctypes.c_uint64(seed & (2**64 - 1)), D, out))
    return np.array(out[:], dtype=np.int8)


def profile_enable(on=True):
    _check(lib().pariskv_profile_enable(1 if on else 0))


def profile_reset():
    _check(lib().pariskv_profile_reset())


def profile_read(max_entries=64):
    """{kernel name: (launches, total ms)} from events recorded since the last reset."""
    names = (ctypes.c_char_p * max_entries)()
    launches = (ctypes.c_int64 * max_entries)()
    ms = (ctypes.c_double * max_entries)()
    n = lib().pariskv_profile_read(max_entries, names, launches, ms)
    if n < 0:
        _check(n)
    return {names[i].decode(): (launches[i], ms[i]) for i in range(min(n, max_entries))}
