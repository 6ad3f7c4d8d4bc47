"""ctypes binding of libsparse_engine.so (argument marshalling only).

The functions carry the C names of include/sparse_engine.h.  They take torch
tensors (device memory owned by the caller) or None, check dtype, device and
contiguity, and pass raw pointers plus the current HIP stream to the library.
Every step of the computation runs in the library's HIP kernels; there is no
fallback of any kind, and importing this module fails if the library has not
been built.
"""

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsparse_engine.so")

SE_OK = 0
SE_ERR_INVALID_ARGUMENT = 1
SE_ERR_UNSUPPORTED = 2
SE_ERR_WORKSPACE = 3
SE_ERR_HIP = 4

SE_DEVERR_BAD_PAGE = 1
SE_DEVERR_CAPACITY = 2
SE_DEVERR_BAD_LENGTH = 4
SE_DEVERR_BAD_SELECTION = 8
SE_DEVERR_BAD_POSITIONS = 16
SE_DEVERR_BAD_INTERVAL = 32

SE_ATTEND_ACCUMULATE = 1
SE_QUEST_SCORES_GIVEN = 1
SE_OP_DECODE_ATTEND = 1
SE_OP_QUEST_SELECT = 2
SE_OP_QUEST_STEP = 3
SE_OP_SNAPKV = 4
SE_OP_OMNIKV_SELECT = 5
SE_OP_H2O_PREFILL = 6
SE_SNAPKV_SCORE_ONLY = 1

EXPORTED = (
    "se_decode_attend", "se_decode_step_h2o", "se_decode_step_quest", "se_accumulate_scores", "se_evict_compact", "se_quest_summarize",
    "se_quest_select", "se_workspace_bytes", "se_read_device_errors", "se_status_string",
    "se_version", "se_snapkv_compact", "se_omnikv_select", "se_attend_slots", "se_h2o_prefill_chunk",
    "se_prune_interval", "se_decode_step_h2o_noalloc", "se_static_scratch_bytes", "se_probe_read_pages",
)


class SparseEngineError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} returned {status_string(status)} ({status})")
        self.status = status


class se_kv_view(ctypes.Structure):
    _fields_ = [
        ("kv_pool", ctypes.c_void_p),
        ("pos_pool", ctypes.c_void_p),
        ("score_pool", ctypes.c_void_p),
        ("meta_pool", ctypes.c_void_p),
        ("block_table", ctypes.c_void_p),
        ("lengths", ctypes.c_void_p),
        ("num_pages", ctypes.c_int64),
        ("num_units", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("max_pages", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
    ]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python paper_2609_39068_amd/build.py` "
            "(hipcc, gfx950); there is no fallback path")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, U32, F32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_float, ctypes.c_size_t
    V = ctypes.POINTER(se_kv_view)
    sig = {
        "se_decode_attend": (I32, [V, I32, P, P, P, P, P, I32, F32, I32, U32, P, P, P, I32, P, SZ, P, P]),
        "se_decode_step_h2o": (I32, [V, I32, P, P, P, P, F32, I32, I32, I32, P, P, P, I32, P, P, SZ, P, P]),
        "se_decode_step_h2o_noalloc": (I32, [V, I32, P, P, P, P, F32, I32, I32, I32, P, P, P, I32, P, P, P]),
        "se_static_scratch_bytes": (SZ, []),
        "se_accumulate_scores": (I32, [V, I32, P, I32, P, I32, P, P]),
        "se_evict_compact": (I32, [V, I32, I32, I32, P, I32, P, P, P]),
        "se_quest_summarize": (I32, [V, I32, P, P]),
        "se_quest_select": (I32, [V, I32, P, F32, I32, I32, U32, P, P, I32, P, SZ, P, P]),
        "se_decode_step_quest": (I32, [V, I32, P, P, P, P, F32, I32, I32, P, P, P, P, SZ, P, P]),
        "se_snapkv_compact": (I32, [V, I32, P, I32, I32, F32, I32, I32, U32, P, I32, P, P, SZ, P, P]),
        "se_omnikv_select": (I32, [V, I32, P, I32, I32, I32, P, P, SZ, P, P]),
        "se_h2o_prefill_chunk": (I32, [V, I32, P, I32, I32, F32, I32, I32, I32, P, I32, P, P, SZ, P, P]),
        "se_attend_slots": (I32, [V, I32, P, P, P, P, P, I32, F32, I32, P, P, P, P]),
        "se_prune_interval": (I32, [V, P, P, I32, P, I32, P, I32, P, P, P]),
        "se_workspace_bytes": (SZ, [I32, I32, I32, I32, I32, I32, I32]),
        "se_read_device_errors": (I32, [P, P, P]),
        "se_status_string": (ctypes.c_char_p, [I32]),
        "se_version": (I32, []),
        "se_probe_read_pages": (I32, [P, ctypes.c_int64, P, ctypes.c_int64, I32, I32, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def status_string(status: int) -> str:
    return _lib.se_status_string(int(status)).decode()


def _ptr(t, dtype=None, name="tensor"):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor or None")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must live in device memory")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _check(fn, status):
    if status != SE_OK:
        raise SparseEngineError(fn, status)


class KVView:
    """Owns the se_kv_view struct of a set of pool tensors (and keeps them alive)."""

    def __init__(self, kv_pool, pos_pool, score_pool, meta_pool, block_table, lengths,
                 num_kv_heads: int, page_size: int = 16):
        self.tensors = (kv_pool, pos_pool, score_pool, meta_pool, block_table, lengths)
        num_pages, two, ps, d = kv_pool.shape
        if two != 2 or ps != page_size:
            raise ValueError("kv_pool must be [num_pages][2][page_size][head_dim]")
        for t, per_page, name in ((pos_pool, page_size, "pos_pool"), (score_pool, page_size, "score_pool"),
                                  (meta_pool, 2 * d, "meta_pool")):
            _need(t, num_pages * per_page, name)
        if lengths.numel() < block_table.shape[0]:
            raise ValueError("lengths needs one entry per block-table row")
        self.struct = se_kv_view(
            kv_pool=_ptr(kv_pool, torch.bfloat16, "kv_pool"),
            pos_pool=_ptr(pos_pool, torch.int32, "pos_pool"),
            score_pool=_ptr(score_pool, torch.float32, "score_pool"),
            meta_pool=_ptr(meta_pool, torch.bfloat16, "meta_pool"),
            block_table=_ptr(block_table, torch.int32, "block_table"),
            lengths=_ptr(lengths, torch.int32, "lengths"),
            num_pages=num_pages, num_units=block_table.shape[0], num_kv_heads=num_kv_heads,
            max_pages=block_table.shape[1], page_size=page_size, head_dim=d)

    @property
    def num_units(self) -> int:
        return self.struct.num_units

    def ref(self):
        return ctypes.byref(self.struct)


def se_workspace_bytes(op, num_units, max_len, max_pages, q_per_kv, head_dim, top_k=0) -> int:
    return int(_lib.se_workspace_bytes(op, num_units, max_len, max_pages, q_per_kv, head_dim, top_k))


def _need(t, n, name):
    if t is not None and t.numel() < n:
        raise ValueError(f"{name} holds {t.numel()} elements, the call needs {n}")


def se_decode_attend(view: KVView, q_per_kv, q, k_new, v_new, new_pos, sel_pages, top_k, scale,
                     max_len, flags, out, lse, logits, logits_stride, ws, dev_err, stream=None):
    s = view.struct
    nreq = s.num_units // s.num_kv_heads
    hq = s.num_kv_heads * q_per_kv
    _need(q, nreq * hq * s.head_dim, "q")
    _need(out, nreq * hq * s.head_dim, "out")
    _need(lse, nreq * hq, "lse")
    _need(k_new, s.num_units * s.head_dim, "k_new")
    _need(v_new, s.num_units * s.head_dim, "v_new")
    _need(new_pos, nreq, "new_pos")
    if sel_pages is not None:
        _need(sel_pages, s.num_units * int(top_k), "sel_pages")
    if logits is not None:
        _need(logits, s.num_units * q_per_kv * int(logits_stride), "logits")
    st = _lib.se_decode_attend(
        view.ref(), q_per_kv, _ptr(q, torch.bfloat16, "q"), _ptr(k_new, torch.bfloat16, "k_new"),
        _ptr(v_new, torch.bfloat16, "v_new"), _ptr(new_pos, torch.int32, "new_pos"),
        _ptr(sel_pages, torch.int32, "sel_pages"), int(top_k), float(scale), int(max_len),
        int(flags), _ptr(out, torch.float32, "out"), _ptr(lse, torch.float32, "lse"),
        _ptr(logits, torch.float32, "logits"), int(logits_stride), _ptr(ws, None, "ws"),
        0 if ws is None else ws.numel() * ws.element_size(), _ptr(dev_err, torch.int32, "dev_err"),
        _stream(stream))
    _check("se_decode_attend", st)


def se_decode_step_h2o(view: KVView, q_per_kv, q, k_new, v_new, new_pos, scale, budget, recent,
                       max_len, out, lse, freed_pages, freed_stride, freed_count, ws, dev_err,
                       stream=None):
    s = view.struct
    nreq = s.num_units // s.num_kv_heads
    hq = s.num_kv_heads * q_per_kv
    _need(q, nreq * hq * s.head_dim, "q")
    _need(out, nreq * hq * s.head_dim, "out")
    _need(lse, nreq * hq, "lse")
    _need(k_new, s.num_units * s.head_dim, "k_new")
    _need(v_new, s.num_units * s.head_dim, "v_new")
    _need(new_pos, nreq, "new_pos")
    if freed_pages is not None:
        _need(freed_pages, s.num_units * int(freed_stride), "freed_pages")
    _need(freed_count, s.num_units, "freed_count")
    st = _lib.se_decode_step_h2o(
        view.ref(), q_per_kv, _ptr(q, torch.bfloat16, "q"), _ptr(k_new, torch.bfloat16, "k_new"),
        _ptr(v_new, torch.bfloat16, "v_new"), _ptr(new_pos, torch.int32, "new_pos"), float(scale),
        int(budget), int(recent), int(max_len), _ptr(out, torch.float32, "out"),
        _ptr(lse, torch.float32, "lse"), _ptr(freed_pages, torch.int32, "freed_pages"),
        int(freed_stride), _ptr(freed_count, torch.int32, "freed_count"), _ptr(ws, None, "ws"),
        0 if ws is None else ws.numel() * ws.element_size(), _ptr(dev_err, torch.int32, "dev_err"),
        _stream(stream))
    _check("se_decode_step_h2o", st)


def se_decode_step_h2o_noalloc(view: KVView, q_per_kv, q, k_new, v_new, new_pos, scale, budget, recent,
                               max_len, out, lse, freed_pages, freed_stride, freed_count, dev_err, stream=None):
    s = view.struct
    nreq = s.num_units // s.num_kv_heads
    hq = s.num_kv_heads * q_per_kv
    _need(q, nreq * hq * s.head_dim, "q")
    _need(out, nreq * hq * s.head_dim, "out")
    _need(lse, nreq * hq, "lse")
    _need(k_new, s.num_units * s.head_dim, "k_new")
    _need(v_new, s.num_units * s.head_dim, "v_new")
    _need(new_pos, nreq, "new_pos")
    if freed_pages is not None:
        _need(freed_pages, s.num_units * int(freed_stride), "freed_pages")
    _need(freed_count, s.num_units, "freed_count")
    st = _lib.se_decode_step_h2o_noalloc(
        view.ref(), q_per_kv, _ptr(q, torch.bfloat16, "q"), _ptr(k_new, torch.bfloat16, "k_new"),
        _ptr(v_new, torch.bfloat16, "v_new"), _ptr(new_pos, torch.int32, "new_pos"), float(scale),
        int(budget), int(recent), int(max_len), _ptr(out, torch.float32, "out"),
        _ptr(lse, torch.float32, "lse"), _ptr(freed_pages, torch.int32, "freed_pages"),
        int(freed_stride), _ptr(freed_count, torch.int32, "freed_count"), _ptr(dev_err, torch.int32, "dev_err"),
        _stream(stream))
    _check("se_decode_step_h2o_noalloc", st)


def se_static_scratch_bytes() -> int:
    return int(_lib.se_static_scratch_bytes())


def se_accumulate_scores(view: KVView, q_per_kv, logits, logits_stride, lse, max_len, dev_err,
                         stream=None):
    s = view.struct
    _need(logits, s.num_units * q_per_kv * int(logits_stride), "logits")
    _need(lse, s.num_units * q_per_kv, "lse")
    st = _lib.se_accumulate_scores(view.ref(), q_per_kv, _ptr(logits, torch.float32, "logits"),
                                   int(logits_stride), _ptr(lse, torch.float32, "lse"),
                                   int(max_len), _ptr(dev_err, torch.int32, "dev_err"),
                                   _stream(stream))
    _check("se_accumulate_scores", st)


def se_evict_compact(view: KVView, budget, recent, max_len, freed_pages, freed_stride,
                     freed_count, dev_err, stream=None):
    s = view.struct
    if freed_pages is not None:
        _need(freed_pages, s.num_units * int(freed_stride), "freed_pages")
    _need(freed_count, s.num_units, "freed_count")
    st = _lib.se_evict_compact(view.ref(), int(budget), int(recent), int(max_len),
                               _ptr(freed_pages, torch.int32, "freed_pages"), int(freed_stride),
                               _ptr(freed_count, torch.int32, "freed_count"),
                               _ptr(dev_err, torch.int32, "dev_err"), _stream(stream))
    _check("se_evict_compact", st)


def se_quest_summarize(view: KVView, max_len, dev_err, stream=None):
    st = _lib.se_quest_summarize(view.ref(), int(max_len), _ptr(dev_err, torch.int32, "dev_err"),
                                 _stream(stream))
    _check("se_quest_summarize", st)


def se_quest_select(view: KVView, q_per_kv, q, scale, top_k, max_len, flags, sel_pages,
                    page_scores, scores_stride, ws, dev_err, stream=None):
    s = view.struct
    _need(sel_pages, s.num_units * int(top_k), "sel_pages")
    if q is not None:
        _need(q, (s.num_units // s.num_kv_heads) * s.num_kv_heads * q_per_kv * s.head_dim, "q")
    if page_scores is not None:
        _need(page_scores, s.num_units * int(scores_stride), "page_scores")
    st = _lib.se_quest_select(
        view.ref(), int(q_per_kv), _ptr(q, torch.bfloat16, "q"), float(scale), int(top_k),
        int(max_len), int(flags), _ptr(sel_pages, torch.int32, "sel_pages"),
        _ptr(page_scores, torch.float32, "page_scores"), int(scores_stride),
        _ptr(ws, None, "ws"), 0 if ws is None else ws.numel() * ws.element_size(),
        _ptr(dev_err, torch.int32, "dev_err"), _stream(stream))
    _check("se_quest_select", st)


def se_read_device_errors(dev_err, stream=None) -> int:
    out = ctypes.c_int32(0)
    st = _lib.se_read_device_errors(_ptr(dev_err, torch.int32, "dev_err"), ctypes.byref(out),
                                    _stream(stream))
    _check("se_read_device_errors", st)
    return int(out.value)


def se_version() -> int:
    return int(_lib.se_version())


def se_probe_read_pages(pool, pool_pages, pages, n_pages, page_bytes, grid, sink, stream=None):
    """Measurement aid: reads the listed pages of `pool` (the read-rate ceiling of a page gather)."""
    _need(pool, int(pool_pages) * int(page_bytes) // pool.element_size(), "pool")
    _need(pages, int(n_pages), "pages")
    _need(sink, int(grid) * 512, "sink")
    st = _lib.se_probe_read_pages(_ptr(pool, None, "pool"), int(pool_pages), _ptr(pages, torch.int32, "pages"),
                                  int(n_pages), int(page_bytes), int(grid), _ptr(sink, torch.int32, "sink"),
                                  _stream(stream))
    _check("se_probe_read_pages", st)


def raw_library():
    """The loaded ctypes library (for symbol checks)."""
    return _lib


def se_decode_step_quest(view: KVView, q_per_kv, q, k_new, v_new, new_pos, scale, top_k, max_len, sel_pages,
                         out, lse, ws, dev_err, stream=None):
    s = view.struct
    nreq = s.num_units // s.num_kv_heads
    hq = s.num_kv_heads * q_per_kv
    _need(q, nreq * hq * s.head_dim, "q")
    _need(out, nreq * hq * s.head_dim, "out")
    _need(lse, nreq * hq, "lse")
    _need(k_new, s.num_units * s.head_dim, "k_new")
    _need(v_new, s.num_units * s.head_dim, "v_new")
    _need(new_pos, nreq, "new_pos")
    _need(sel_pages, s.num_units * int(top_k), "sel_pages")
    st = _lib.se_decode_step_quest(
        view.ref(), int(q_per_kv), _ptr(q, torch.bfloat16, "q"), _ptr(k_new, torch.bfloat16, "k_new"),
        _ptr(v_new, torch.bfloat16, "v_new"), _ptr(new_pos, torch.int32, "new_pos"), float(scale),
        int(top_k), int(max_len), _ptr(sel_pages, torch.int32, "sel_pages"), _ptr(out, torch.float32, "out"),
        _ptr(lse, torch.float32, "lse"), _ptr(ws, None, "ws"),
        0 if ws is None else ws.numel() * ws.element_size(), _ptr(dev_err, torch.int32, "dev_err"),
        _stream(stream))
    _check("se_decode_step_quest", st)


def se_snapkv_compact(view: KVView, q_per_kv, q_obs, window, kernel, scale, budget, max_len, flags,
                      freed_pages, freed_stride, freed_count, ws, dev_err, stream=None):
    s = view.struct
    nreq = s.num_units // s.num_kv_heads
    _need(q_obs, nreq * int(window) * s.num_kv_heads * q_per_kv * s.head_dim, "q_obs")
    if freed_pages is not None:
        _need(freed_pages, s.num_units * int(freed_stride), "freed_pages")
    _need(freed_count, s.num_units, "freed_count")
    st = _lib.se_snapkv_compact(
        view.ref(), int(q_per_kv), _ptr(q_obs, torch.bfloat16, "q_obs"), int(window), int(kernel),
        float(scale), int(budget), int(max_len), int(flags), _ptr(freed_pages, torch.int32, "freed_pages"),
        int(freed_stride), _ptr(freed_count, torch.int32, "freed_count"), _ptr(ws, None, "ws"),
        0 if ws is None else ws.numel() * ws.element_size(), _ptr(dev_err, torch.int32, "dev_err"),
        _stream(stream))
    _check("se_snapkv_compact", st)


def se_omnikv_select(view: KVView, q_per_kv, logits, logits_stride, budget, max_len, sel_slots, ws, dev_err,
                     stream=None):
    s = view.struct
    nreq = s.num_units // s.num_kv_heads
    _need(logits, s.num_units * q_per_kv * int(logits_stride), "logits")
    _need(sel_slots, nreq * int(budget), "sel_slots")
    st = _lib.se_omnikv_select(
        view.ref(), int(q_per_kv), _ptr(logits, torch.float32, "logits"), int(logits_stride), int(budget),
        int(max_len), _ptr(sel_slots, torch.int32, "sel_slots"), _ptr(ws, None, "ws"),
        0 if ws is None else ws.numel() * ws.element_size(), _ptr(dev_err, torch.int32, "dev_err"),
        _stream(stream))
    _check("se_omnikv_select", st)


def se_attend_slots(view: KVView, q_per_kv, q, k_new, v_new, new_pos, sel_slots, sel_count, scale, max_len,
                    out, lse, dev_err, stream=None):
    s = view.struct
    nreq = s.num_units // s.num_kv_heads
    hq = s.num_kv_heads * q_per_kv
    _need(q, nreq * hq * s.head_dim, "q")
    _need(out, nreq * hq * s.head_dim, "out")
    _need(lse, nreq * hq, "lse")
    _need(k_new, s.num_units * s.head_dim, "k_new")
    _need(v_new, s.num_units * s.head_dim, "v_new")
    _need(new_pos, nreq, "new_pos")
    _need(sel_slots, nreq * int(sel_count), "sel_slots")
    st = _lib.se_attend_slots(
        view.ref(), int(q_per_kv), _ptr(q, torch.bfloat16, "q"), _ptr(k_new, torch.bfloat16, "k_new"),
        _ptr(v_new, torch.bfloat16, "v_new"), _ptr(new_pos, torch.int32, "new_pos"),
        _ptr(sel_slots, torch.int32, "sel_slots"), int(sel_count), float(scale), int(max_len),
        _ptr(out, torch.float32, "out"), _ptr(lse, torch.float32, "lse"), _ptr(dev_err, torch.int32, "dev_err"),
        _stream(stream))
    _check("se_attend_slots", st)


def se_h2o_prefill_chunk(view: KVView, q_per_kv, q_score, score_window, chunk_len, scale, budget, recent, max_len,
                         freed_pages, freed_stride, freed_count, ws, dev_err, stream=None):
    s = view.struct
    nreq = s.num_units // s.num_kv_heads
    _need(q_score, nreq * int(score_window) * s.num_kv_heads * q_per_kv * s.head_dim, "q_score")
    if freed_pages is not None:
        _need(freed_pages, s.num_units * int(freed_stride), "freed_pages")
    _need(freed_count, s.num_units, "freed_count")
    st = _lib.se_h2o_prefill_chunk(
        view.ref(), int(q_per_kv), _ptr(q_score, torch.bfloat16, "q_score"), int(score_window), int(chunk_len),
        float(scale), int(budget), int(recent), int(max_len), _ptr(freed_pages, torch.int32, "freed_pages"),
        int(freed_stride), _ptr(freed_count, torch.int32, "freed_count"), _ptr(ws, None, "ws"),
        0 if ws is None else ws.numel() * ws.element_size(), _ptr(dev_err, torch.int32, "dev_err"),
        _stream(stream))
    _check("se_h2o_prefill_chunk", st)


def se_prune_interval(view: KVView, interval, keep_mask, mask_stride, keep_budget, max_len, freed_pages,
                      freed_stride, freed_count, dev_err, stream=None):
    """interval int32 [num_units][2]; exactly one of keep_mask (uint8 [num_units][mask_stride])
    and keep_budget (int32 [num_units])."""
    s = view.struct
    _need(interval, 2 * s.num_units, "interval")
    if keep_mask is not None:
        _need(keep_mask, s.num_units * int(mask_stride), "keep_mask")
    if keep_budget is not None:
        _need(keep_budget, s.num_units, "keep_budget")
    if freed_pages is not None:
        _need(freed_pages, s.num_units * int(freed_stride), "freed_pages")
    if freed_count is not None:
        _need(freed_count, s.num_units, "freed_count")
    st = _lib.se_prune_interval(
        view.ref(), _ptr(interval, torch.int32, "interval"), _ptr(keep_mask, torch.uint8, "keep_mask"),
        int(mask_stride), _ptr(keep_budget, torch.int32, "keep_budget"), int(max_len),
        _ptr(freed_pages, torch.int32, "freed_pages"), int(freed_stride),
        _ptr(freed_count, torch.int32, "freed_count"), _ptr(dev_err, torch.int32, "dev_err"), _stream(stream))
    _check("se_prune_interval", st)
