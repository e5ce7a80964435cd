"""ctypes binding of libspanq.so.  Argument marshalling only."""
from __future__ import annotations

import ctypes
import os
import struct
import weakref
from typing import Iterable, List, Optional, Sequence

import numpy as np

try:  # bind to torch's HIP runtime when torch is present (one runtime per process)
    import torch  # noqa: F401
except ImportError:  # pragma: no cover
    torch = None

HERE = os.path.dirname(os.path.abspath(__file__))

SPAN_OK, SPAN_EINVAL, SPAN_ENOMEM, SPAN_EHIP, SPAN_ESTATE = 0, -1, -2, -3, -4
SPAN_F32, SPAN_BF16 = 0, 1
SPAN_HASH_SPAN, SPAN_HASH_STOCK = 0, 1
SPAN_KERNEL = {"auto": 0, "generic": 1, "mfma": 2}
SPAN_HASH_ROOT = 0x243F6A8885A308D3
SPAN_HASH_FRAG_TAG = 0x13198A2E03707344

EXPORTS = [
    "span_last_error", "span_hash_mix", "span_pool_bytes", "span_pool_create", "span_pool_destroy",
    "span_pool_reset", "span_pool_get_info", "span_pool_page_address", "span_pool_read_page",
    "span_hash_pages", "kv_lookup", "span_plan", "span_plan_stats", "span_plan_block_table",
    "span_plan_evicted", "span_plan_rows", "span_prefill_fragments", "span_cross_attend",
    "span_plan_commit", "span_plan_destroy", "span_plan_kernel_times", "span_probe_mfma_peak",
    "span_probe_read_peak", "span_plan_static", "span_model_create", "span_model_destroy", "span_model_forward",
    "span_parse_serialized", "span_bulk_order", "span_plan_moves", "span_plan_decode", "span_decode_attend",
    "span_model_decode", "span_probe_gemm",
]
SPAN_STATIC_SCRATCH_BYTES = 64 << 20
SPAN_FLAG_TIMING = 1
SPAN_FLAG_MATERIALIZE = 2


class SpanError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"[{code}] {msg}")
        self.code = code


class PoolConfig(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("hash_mode", ctypes.c_int32), ("kernel", ctypes.c_int32), ("device", ctypes.c_int32),
                ("flags", ctypes.c_int32), ("rope_theta", ctypes.c_float), ("num_pages", ctypes.c_int64),
                ("device_buf", ctypes.c_void_p), ("device_bytes", ctypes.c_size_t)]


class PoolInfo(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in
                ("num_pages", "free_pages", "cached_pages", "pinned_pages", "tick", "total_evictions")]


class SpanTokens(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_void_p), ("n", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("row", ctypes.c_int64)]


class SpanQuery(ctypes.Structure):
    _fields_ = [("prefix", SpanTokens), ("frags", ctypes.POINTER(SpanTokens)), ("n_frags", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("cross", SpanTokens)]


STAT_FIELDS = ("pages_hit", "pages_new", "pages_cross", "pages_evicted", "tokens_hit", "tokens_new", "tokens_cross",
               "prefill_pairs", "cross_pairs", "prefill_tiles", "cross_tiles", "kv_splits", "cross_kv_pages")


class SpanStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in STAT_FIELDS] + [("host_plan_us", ctypes.c_double),
                                                            ("host_upload_us", ctypes.c_double),
                                                            ("pages_moved", ctypes.c_int64),
                                                            ("tokens_moved", ctypes.c_int64),
                                                            ("prefill_queues", ctypes.c_int64),
                                                            ("decode_steps", ctypes.c_int64),
                                                            ("decode_tokens", ctypes.c_int64),
                                                            ("decode_pages", ctypes.c_int64),
                                                            ("decode_pairs", ctypes.c_int64)]


TIME_FIELDS = ("page_write_prefill_ms", "prefill_attention_ms", "page_write_cross_ms", "cross_attention_ms",
               "combine_ms", "page_move_ms", "decode_ms")


class KernelTimes(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in TIME_FIELDS] + [("prefill_calls", ctypes.c_int32),
                                                            ("cross_calls", ctypes.c_int32),
                                                            ("decode_calls", ctypes.c_int32)]


class SpanRange(ctypes.Structure):
    _fields_ = [("begin", ctypes.c_int64), ("n", ctypes.c_int64)]


class ModelConfig(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("hidden", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("reserved", ctypes.c_int32),
                ("embed", ctypes.c_void_p),
                ("attn_norm", ctypes.POINTER(ctypes.c_void_p)), ("w_qkv", ctypes.POINTER(ctypes.c_void_p)),
                ("w_o", ctypes.POINTER(ctypes.c_void_p)), ("ffn_norm", ctypes.POINTER(ctypes.c_void_p)),
                ("w_gate_up", ctypes.POINTER(ctypes.c_void_p)), ("w_down", ctypes.POINTER(ctypes.c_void_p)),
                ("final_norm", ctypes.c_void_p), ("lm_head", ctypes.c_void_p)]


_LIB = None


def library_path() -> str:
    return os.environ.get("SPANQ_LIB", os.path.join(HERE, "libspanq.so"))


def load():
    """Load libspanq.so (built by ``paper_2511_02749_amd/build.py``); raise if missing."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = library_path()
    if not os.path.exists(path):
        raise FileNotFoundError(f"{path} not built: run python -m paper_2511_02749_amd.build")
    lib = ctypes.CDLL(path)
    P, I32, I64, U64, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p
    sig = {
        "span_last_error": (ctypes.c_char_p, []),
        "span_hash_mix": (U64, [U64]),
        "span_pool_bytes": (I32, [P(PoolConfig), P(ctypes.c_size_t)]),
        "span_pool_create": (I32, [P(PoolConfig), P(VP)]),
        "span_pool_destroy": (I32, [VP]),
        "span_pool_reset": (I32, [VP]),
        "span_pool_get_info": (I32, [VP, P(PoolInfo)]),
        "span_pool_page_address": (I32, [VP, I32, I32, P(VP), P(I64)]),
        "span_pool_read_page": (I32, [VP, I32, I32, VP, ctypes.c_size_t]),
        "span_hash_pages": (I32, [U64, P(I32), I32, I32, I32, P(U64), P(I32)]),
        "kv_lookup": (I32, [VP, P(U64), I32, P(I32), P(I32)]),
        "span_plan": (I32, [VP, P(SpanQuery), I32, VP, P(VP)]),
        "span_plan_static": (I32, [VP, P(SpanQuery), I32, VP, P(VP)]),
        "span_model_create": (I32, [VP, P(ModelConfig), P(VP)]),
        "span_model_destroy": (I32, [VP]),
        "span_model_forward": (I32, [VP, VP, P(I32), I64, I32, VP, VP, P(I32), VP]),
        "span_model_decode": (I32, [VP, VP, P(I32), VP, P(I32), VP]),
        "span_bulk_order": (I32, [VP, P(SpanQuery), I32, P(I32)]),
        "span_parse_serialized": (I32, [P(I32), I64, I32, P(I32), P(SpanRange), I32, P(I32), P(SpanRange),
                                        P(SpanRange)]),
        "span_plan_stats": (I32, [VP, P(SpanStats)]),
        "span_plan_block_table": (I32, [VP, I32, I32, P(I32), I32, P(I32), P(I32)]),
        "span_plan_evicted": (I32, [VP, P(I32), I32, P(I32)]),
        "span_plan_moves": (I32, [VP, P(I32), I32, P(I32)]),
        "span_plan_decode": (I32, [VP, P(I32), P(I64), VP]),
        "span_decode_attend": (I32, [VP, I32, VP, VP, VP, VP, VP]),
        "span_plan_rows": (I32, [VP, P(I64), I64, P(I64), P(I64)]),
        "span_prefill_fragments": (I32, [VP, I32, VP, VP, VP, VP, VP]),
        "span_cross_attend": (I32, [VP, I32, VP, VP, VP, VP, VP]),
        "span_plan_commit": (I32, [VP]),
        "span_plan_destroy": (I32, [VP]),
        "span_plan_kernel_times": (I32, [VP, P(KernelTimes)]),
        "span_probe_mfma_peak": (I32, [I32, I32, VP, P(ctypes.c_double)]),
        "span_probe_read_peak": (I32, [VP, ctypes.c_size_t, I32, VP, P(ctypes.c_double)]),
        "span_probe_gemm": (I32, [VP, VP, VP, I64, I64, I64, I32, I32, VP, P(I32), P(ctypes.c_double)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    _LIB = lib
    return lib


def _check(rc: int):
    if rc != SPAN_OK:
        raise SpanError(rc, load().span_last_error().decode())


def _i32p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _ptr(x) -> Optional[int]:
    """Device pointer of a torch tensor (or an int address); None stays None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s) -> Optional[int]:
    if s is None:
        if torch is not None and torch.cuda.is_available():
            return torch.cuda.current_stream().cuda_stream
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def probe_mfma_peak(iters: int = 20000, reps: int = 5, stream=None) -> float:
    """bf16 MFMA TFLOP/s this GPU attains with an MFMA-only loop (span_probe_mfma_peak)."""
    out = ctypes.c_double()
    _check(load().span_probe_mfma_peak(iters, reps, _stream(stream), ctypes.byref(out)))
    return float(out.value)


def probe_read_peak(buf, reps: int = 5, stream=None) -> float:
    """HBM read GB/s this GPU attains streaming a device tensor (span_probe_read_peak)."""
    out = ctypes.c_double()
    nbytes = buf.numel() * buf.element_size()
    _check(load().span_probe_read_peak(_ptr(buf), nbytes - nbytes % 16, reps, _stream(stream), ctypes.byref(out)))
    return float(out.value)


def probe_gemm(x, w, y, residual: bool = False, reps: int = 0, stream=None):
    """The model stack's GEMM y = x @ w (+ y) on bf16 device tensors (span_probe_gemm).
    Returns (kernel, seconds per call): kernel 1 GEMV, 2 skinny MFMA, 0 hipBLASLt."""
    M, K = x.shape
    K2, N = w.shape
    assert K2 == K and tuple(y.shape) == (M, N)
    kern, sec = ctypes.c_int32(), ctypes.c_double()
    _check(load().span_probe_gemm(_ptr(x), _ptr(w), _ptr(y), M, N, K, 1 if residual else 0, reps, _stream(stream),
                                  ctypes.byref(kern), ctypes.byref(sec)))
    return int(kern.value), float(sec.value)


def hash_mix(x: int) -> int:
    return int(load().span_hash_mix(x))


def hash_pages(seed: int, tokens: Sequence[int], page_size: int = 16, include_partial: bool = True) -> List[int]:
    lib = load()
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    out = np.zeros(max(1, (t.size + page_size - 1) // page_size), np.uint64)
    n = ctypes.c_int32()
    _check(lib.span_hash_pages(seed, _i32p(t), t.size, page_size, int(include_partial),
                               out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)), ctypes.byref(n)))
    return [int(x) for x in out[: n.value]]


class Pool:
    """A paged KV pool and its cache index.  device=-1 gives a host-only pool."""

    def __init__(self, *, num_q_heads: int, num_kv_heads: int, head_dim: int, num_pages: int, dtype: str = "bf16",
                 num_layers: int = 1, rope_theta: float = 1e4, page_size: int = 16, device: int = 0,
                 hash_mode: str = "span", kernel: str = "auto", timing: bool = False, materialize: bool = False,
                 device_buf=None):
        """device_buf: optional caller-owned device memory for the pages (a torch tensor of
        at least span_pool_bytes bytes, kept referenced by the pool)."""
        lib = load()
        self.cfg = PoolConfig(num_layers=num_layers, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                              head_dim=head_dim, page_size=page_size,
                              dtype=SPAN_BF16 if dtype == "bf16" else SPAN_F32,
                              hash_mode=SPAN_HASH_STOCK if hash_mode == "stock" else SPAN_HASH_SPAN,
                              kernel=SPAN_KERNEL[kernel], device=device,
                              flags=(SPAN_FLAG_TIMING if timing else 0) | (SPAN_FLAG_MATERIALIZE if materialize else 0),
                              rope_theta=rope_theta,
                              num_pages=num_pages, device_buf=_ptr(device_buf),
                              device_bytes=0 if device_buf is None else device_buf.numel() * device_buf.element_size())
        self._buf = device_buf
        self.dtype = dtype
        self._plans = weakref.WeakSet()
        self._h = ctypes.c_void_p()
        _check(lib.span_pool_create(ctypes.byref(self.cfg), ctypes.byref(self._h)))

    @property
    def handle(self):
        return self._h

    def page_bytes(self) -> int:
        es = 2 if self.dtype == "bf16" else 4
        return 2 * self.cfg.num_kv_heads * self.cfg.page_size * self.cfg.head_dim * es

    def close(self):
        if self._h:
            for p in list(self._plans):
                p.destroy()
            _check(load().span_pool_destroy(self._h))
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def reset(self):
        _check(load().span_pool_reset(self._h))

    def info(self) -> dict:
        i = PoolInfo()
        _check(load().span_pool_get_info(self._h, ctypes.byref(i)))
        return {n: int(getattr(i, n)) for n, _ in PoolInfo._fields_}

    def lookup(self, hashes: Sequence[int]):
        h = np.ascontiguousarray(hashes, dtype=np.uint64)
        ids = np.zeros(max(1, h.size), np.int32)
        lead = ctypes.c_int32()
        _check(load().kv_lookup(self._h, h.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)), h.size, _i32p(ids),
                                ctypes.byref(lead)))
        return [int(x) for x in ids[: h.size]], lead.value

    def read_page(self, layer: int, page_id: int) -> np.ndarray:
        """Raw page (K then V) as uint16 (bf16 bits) or float32 values."""
        buf = np.zeros(self.page_bytes() // (2 if self.dtype == "bf16" else 4),
                       np.uint16 if self.dtype == "bf16" else np.float32)
        _check(load().span_pool_read_page(self._h, layer, page_id, buf.ctypes.data, buf.nbytes))
        return buf

    def bulk_order(self, queries: Iterable) -> List[int]:
        """Execution order clustering fragment reuse (span_bulk_order)."""
        qs = list(queries)
        keep: list = []
        arr = _query_array(qs, keep)
        order = np.zeros(max(1, len(qs)), np.int32)
        _check(load().span_bulk_order(self._h, arr, len(qs), _i32p(order)))
        return [int(x) for x in order[: len(qs)]]

    def plan(self, queries: Iterable, stream=None, static: bool = False) -> "Plan":
        """queries: objects with .prefix, .frags, .cross; each span has .tokens (int32) and .row.
        static=True plans through span_plan_static (no device allocation)."""
        return Plan(self, list(queries), stream, static)


# Data addresses of int32 token arrays already marshalled, by id: the entry holds the
# array itself, so its id cannot be reused while the entry lives, and an array whose
# buffer this cache references cannot be resized in place.  Bounded; cleared when full.
_ADDR: dict = {}
_ADDR_CAP = 1 << 14

# span_tokens and span_query (include/spanq.h) as packed little-endian records
_SPAN_REC = struct.Struct("<QiiQ")
_QUERY_REC = struct.Struct("<QiiQ" "Qii" "QiiQ")
assert _SPAN_REC.size == ctypes.sizeof(SpanTokens) and _QUERY_REC.size == ctypes.sizeof(SpanQuery)


def _tokens(t, keep: list):
    """(array, data address or 0, length) of a span's int32 tokens."""
    hit = _ADDR.get(id(t))
    if hit is not None and hit[0] is t:
        return hit
    if not (isinstance(t, np.ndarray) and t.dtype == np.int32 and t.flags.c_contiguous):
        t = np.ascontiguousarray(t, dtype=np.int32)
        keep.append(t)
        return t, (t.ctypes.data if t.size else 0), t.size
    if len(_ADDR) >= _ADDR_CAP:
        _ADDR.clear()
    hit = _ADDR[id(t)] = (t, t.ctypes.data if t.size else 0, t.size)
    return hit


def _query_array(queries: list, keep: list):
    """A span_query array over the queries (the buffers it points into go to keep)."""
    n = max(1, len(queries))
    qb = bytearray(_QUERY_REC.size * n)
    pack_span, pack_query, get = _SPAN_REC.pack_into, _QUERY_REC.pack_into, _ADDR.get
    for i, q in enumerate(queries):
        frags = q.frags
        fb = bytearray(_SPAN_REC.size * max(1, len(frags)))
        o = 0
        for f in frags:
            t = f.tokens
            hit = get(id(t))  # the cached entry inline: this loop runs once per fragment
            if hit is None or hit[0] is not t:
                hit = _tokens(t, keep)
            pack_span(fb, o, hit[1], hit[2], 0, int(f.row))
            o += _SPAN_REC.size
        keep.append(fb)
        p, c = q.prefix, q.cross
        _, pa, pm = _tokens(p.tokens, keep)
        _, ca, cm = _tokens(c.tokens, keep)
        pack_query(qb, _QUERY_REC.size * i, pa, pm, 0, int(p.row), ctypes.addressof(ctypes.c_char.from_buffer(fb)),
                   len(frags), 0, ca, cm, 0, int(c.row))
    keep.append(qb)
    return (SpanQuery * n).from_buffer(qb)


class Plan:
    def __init__(self, pool: Pool, queries: list, stream=None, static: bool = False):
        lib = load()
        self.pool = pool
        keep: list = []
        arr = _query_array(queries, keep)
        self.n_queries = len(queries)
        self.n_frags = [len(q.frags) for q in queries]
        self._h = ctypes.c_void_p()
        self._stream = _stream(stream)
        entry = lib.span_plan_static if static else lib.span_plan
        _check(entry(pool.handle, arr, len(queries), self._stream, ctypes.byref(self._h)))
        pool._plans.add(self)

    def stats(self) -> dict:
        s = SpanStats()
        _check(load().span_plan_stats(self._h, ctypes.byref(s)))
        d = {n: int(getattr(s, n)) for n in STAT_FIELDS}
        d["host_plan_us"], d["host_upload_us"] = float(s.host_plan_us), float(s.host_upload_us)
        d["pages_moved"], d["tokens_moved"] = int(s.pages_moved), int(s.tokens_moved)
        for n in ("prefill_queues", "decode_steps", "decode_tokens", "decode_pages", "decode_pairs"):
            d[n] = int(getattr(s, n))
        return d

    def block_table(self, query: int, span: int):
        """span: -1 prefix, 0..n-1 fragment children, n cross.  Returns (page ids, n_hit)."""
        n, nh = ctypes.c_int32(), ctypes.c_int32()
        _check(load().span_plan_block_table(self._h, query, span, None, 0, ctypes.byref(n), ctypes.byref(nh)))
        ids = np.zeros(max(1, n.value), np.int32)
        _check(load().span_plan_block_table(self._h, query, span, _i32p(ids), n.value, ctypes.byref(n),
                                            ctypes.byref(nh)))
        return [int(x) for x in ids[: n.value]], nh.value

    def moves(self) -> List[tuple]:
        """Repositioned copies (materialize pools): (source page, copy page, shift, filled slots)."""
        n = ctypes.c_int32()
        _check(load().span_plan_moves(self._h, None, 0, ctypes.byref(n)))
        rec = np.zeros(max(4, 4 * n.value), np.int32)
        _check(load().span_plan_moves(self._h, _i32p(rec), n.value, ctypes.byref(n)))
        return [tuple(int(x) for x in rec[4 * i: 4 * i + 4]) for i in range(n.value)]

    def evicted(self) -> List[int]:
        n = ctypes.c_int32()
        _check(load().span_plan_evicted(self._h, None, 0, ctypes.byref(n)))
        ids = np.zeros(max(1, n.value), np.int32)
        _check(load().span_plan_evicted(self._h, _i32p(ids), n.value, ctypes.byref(n)))
        return [int(x) for x in ids[: n.value]]

    def rows(self):
        """(prefill rows, cross rows) the plan computes."""
        npf, ncr = ctypes.c_int64(), ctypes.c_int64()
        _check(load().span_plan_rows(self._h, None, 0, ctypes.byref(npf), ctypes.byref(ncr)))
        buf = np.zeros(max(1, npf.value + ncr.value), np.int64)
        _check(load().span_plan_rows(self._h, buf.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), buf.size,
                                     ctypes.byref(npf), ctypes.byref(ncr)))
        return buf[: npf.value].copy(), buf[npf.value: npf.value + ncr.value].copy()

    def prefill(self, layer: int, q, k, v, out, stream=None):
        _check(load().span_prefill_fragments(self._h, layer, _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                             _stream(stream) if stream is not None else self._stream))

    def cross(self, layer: int, q, k, v, out, stream=None):
        _check(load().span_cross_attend(self._h, layer, _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                        _stream(stream) if stream is not None else self._stream))

    def decode(self, n_new, rows, stream=None):
        """Plan a decode step: n_new[q] tokens appended to query q's cross segment, taken
        from caller rows rows[q] .. (span_plan_decode)."""
        n = np.ascontiguousarray(n_new, np.int32)
        r = np.ascontiguousarray(rows, np.int64)
        _check(load().span_plan_decode(self._h, _i32p(n), r.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                       _stream(stream) if stream is not None else self._stream))

    def decode_attend(self, layer: int, q, k, v, out, stream=None):
        _check(load().span_decode_attend(self._h, layer, _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                         _stream(stream) if stream is not None else self._stream))

    def kernel_times(self) -> dict:
        t = KernelTimes()
        _check(load().span_plan_kernel_times(self._h, ctypes.byref(t)))
        d = {n: float(getattr(t, n)) for n in TIME_FIELDS}
        d["prefill_calls"], d["cross_calls"] = int(t.prefill_calls), int(t.cross_calls)
        d["decode_calls"] = int(t.decode_calls)
        return d

    def commit(self):
        _check(load().span_plan_commit(self._h))

    def destroy(self):
        if self._h:
            _check(load().span_plan_destroy(self._h))
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


class Model:
    """A decoder stack bound to a pool (span_model_*).  Weights are device tensors or
    device addresses (bf16, x @ W layout); per-layer weights are sequences."""

    def __init__(self, pool: Pool, *, hidden: int, ffn: int, vocab: int, rms_eps: float, embed, attn_norm, w_qkv,
                 w_o, ffn_norm, w_gate_up, w_down, final_norm, lm_head):
        lib = load()
        L = pool.cfg.num_layers
        self._keep = [embed, attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down, final_norm, lm_head]
        tables = []
        for seq in (attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down):
            assert len(seq) == L
            tables.append((ctypes.c_void_p * L)(*[_ptr(x) for x in seq]))
        self._tables = tables
        self.cfg = ModelConfig(num_layers=L, hidden=hidden, num_q_heads=pool.cfg.num_q_heads,
                               num_kv_heads=pool.cfg.num_kv_heads, head_dim=pool.cfg.head_dim, ffn=ffn, vocab=vocab,
                               rms_eps=rms_eps, reserved=0, embed=_ptr(embed),
                               attn_norm=ctypes.cast(tables[0], ctypes.POINTER(ctypes.c_void_p)),
                               w_qkv=ctypes.cast(tables[1], ctypes.POINTER(ctypes.c_void_p)),
                               w_o=ctypes.cast(tables[2], ctypes.POINTER(ctypes.c_void_p)),
                               ffn_norm=ctypes.cast(tables[3], ctypes.POINTER(ctypes.c_void_p)),
                               w_gate_up=ctypes.cast(tables[4], ctypes.POINTER(ctypes.c_void_p)),
                               w_down=ctypes.cast(tables[5], ctypes.POINTER(ctypes.c_void_p)),
                               final_norm=_ptr(final_norm), lm_head=_ptr(lm_head))
        self.pool = pool
        self._h = ctypes.c_void_p()
        _check(lib.span_model_create(pool.handle, ctypes.byref(self.cfg), ctypes.byref(self._h)))

    def forward(self, plan: "Plan", row_tokens, n_layers: Optional[int] = None, hidden_out=None, logits_out=None,
                first_tokens: bool = True, stream=None):
        """Run the plan's computed rows through the stack; returns the first token of
        each query (or None with first_tokens=False)."""
        rt = np.ascontiguousarray(row_tokens, dtype=np.int32)
        L = self.cfg.num_layers if n_layers is None else n_layers
        toks = np.zeros(max(1, plan.n_queries), np.int32) if first_tokens else None
        _check(load().span_model_forward(self._h, plan._h, _i32p(rt), rt.size, L, _ptr(hidden_out), _ptr(logits_out),
                                         _i32p(toks) if toks is not None else None,
                                         _stream(stream) if stream is not None else plan._stream))
        return [int(t) for t in toks[: plan.n_queries]] if toks is not None else None

    def decode(self, plan: "Plan", tokens, logits_out=None, stream=None):
        """One greedy decode step (span_model_decode): tokens[q] >= 0 is fed to query q;
        returns the next token of each query (-1 where tokens[q] < 0)."""
        t = np.ascontiguousarray(tokens, dtype=np.int32)
        nxt = np.zeros(max(1, plan.n_queries), np.int32)
        _check(load().span_model_decode(self._h, plan._h, _i32p(t), _ptr(logits_out), _i32p(nxt),
                                        _stream(stream) if stream is not None else plan._stream))
        return [int(x) for x in nxt[: plan.n_queries]]

    def close(self):
        if self._h:
            _check(load().span_model_destroy(self._h))
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
