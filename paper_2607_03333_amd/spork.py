"""Thin ctypes binding of ``libspork.so`` (C ABI in ``include/spork.h``).

Argument marshalling only: every function has the name of the C entry point
it calls, turns torch tensors into device pointers and numpy arrays into host
pointers, and raises :class:`SporkError` on a non-zero status. Kernels run on
the given stream, or torch's current stream. Nothing here computes any part
of the method, and nothing falls back to the CPU: without the built library
every call raises.
"""

import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspork.so")
# The sanitizer test of the host code loads an AddressSanitizer/UBSan build of
# the host sources instead (its kernel launches all fail); unset otherwise.
_HOST_SANITIZER_LIB = os.environ.get("SPORK_HOST_SANITIZER_LIB")

SPORK_OK = 0
SPORK_E_INVAL = -1
SPORK_E_NOBLOCKS = -2
SPORK_E_UNSUPPORTED = -3
SPORK_E_CAPACITY = -4
SPORK_E_HIP = -5
SPORK_DTYPE_F32 = 0
SPORK_DTYPE_BF16 = 1
SPORK_KERNEL_ATTN = 0
SPORK_KERNEL_MERGE = 1
SPORK_KERNEL_ARGMAX = 2
SPORK_KERNEL_ACCEPT = 3
SPORK_KERNEL_CONF_CHUNKS = 4
SPORK_KERNEL_CONF_FINAL = 5
SPORK_KERNEL_NGRAM_SCAN = 6
SPORK_KERNEL_NGRAM_DRAFTS = 7
SPORK_KERNEL_READ_CEILING = 8
SPORK_KERNEL_KINDS = 9
KERNEL_NAMES = ("attn_partial", "merge", "argmax", "accept", "conf_chunks", "conf_final", "ngram_scan",
                "ngram_drafts", "read_ceiling")

_c_i32 = ctypes.c_int32
_c_i64 = ctypes.c_int64
_p = ctypes.c_void_p
_pi32 = ctypes.POINTER(ctypes.c_int32)
_pi64 = ctypes.POINTER(ctypes.c_int64)


class SporkError(RuntimeError):
    def __init__(self, code, message):
        super().__init__(f"spork status {code}: {message}")
        self.code = code


class spork_shape(ctypes.Structure):
    _fields_ = [("hq", _c_i32), ("hkv", _c_i32), ("head_dim", _c_i32),
                ("block_size", _c_i32), ("dtype", _c_i32), ("sm_scale", ctypes.c_float)]


class spork_plan_info(ctypes.Structure):
    _fields_ = [("n_threads", _c_i32), ("n_rows", _c_i32), ("n_groups", _c_i32),
                ("n_items", _c_i32), ("n_units", _c_i32), ("n_partials", _c_i32),
                ("max_row_tiles", _c_i32), ("attn_grid", _c_i32),
                ("image_bytes", ctypes.c_size_t), ("workspace_bytes", ctypes.c_size_t),
                ("shared_tokens", _c_i64), ("private_tokens", _c_i64),
                ("unique_kv_bytes", _c_i64), ("flat_kv_bytes", _c_i64), ("attn_waves", _c_i32),
                ("control_bytes", ctypes.c_size_t)]


# name -> (restype, argtypes); every name is declared in include/spork.h
_SIGNATURES = {
    "spork_last_error": (ctypes.c_char_p, []),
    "spork_version": (ctypes.c_int, []),
    "spork_cache_create": (ctypes.c_int, [_c_i32, _c_i32, _p, ctypes.POINTER(_p)]),
    "spork_cache_destroy": (ctypes.c_int, [_p]),
    "spork_seq_new": (ctypes.c_int, [_p, _pi32]),
    "spork_seq_append": (ctypes.c_int, [_p, _c_i32, _c_i32, _p, _p, _pi32]),
    "spork_seq_append_batch": (ctypes.c_int, [_p, _p, _p, _c_i32, _p, _p, _pi32]),
    "spork_fork": (ctypes.c_int, [_p, _c_i32, _pi32]),
    "spork_seq_free": (ctypes.c_int, [_p, _c_i32]),
    "spork_seq_len": (ctypes.c_int, [_p, _c_i32, _pi32]),
    "spork_block_table": (ctypes.c_int, [_p, _c_i32, _p, _c_i32, _pi32]),
    "spork_refcount": (ctypes.c_int, [_p, _c_i32, _pi32]),
    "spork_free_blocks": (ctypes.c_int, [_p, _p, _c_i32, _pi32]),
    "spork_kv_write": (ctypes.c_int, [ctypes.POINTER(spork_shape), _p, _p, _c_i32, _p, _p, _p,
                                      _c_i32, _p, _p]),
    "spork_kv_copy": (ctypes.c_int, [ctypes.POINTER(spork_shape), _p, _p, _c_i32, _c_i32, _c_i32,
                                     _c_i32, _p]),
    "spork_plan_create": (ctypes.c_int, [_p, ctypes.POINTER(spork_shape), _p, _p, _p, _c_i32,
                                         _c_i32, ctypes.POINTER(_p)]),
    "spork_plan_destroy": (ctypes.c_int, [_p]),
    "spork_plan_get_info": (ctypes.c_int, [_p, ctypes.POINTER(spork_plan_info)]),
    "spork_plan_image": (ctypes.c_int, [_p, _p, ctypes.c_size_t]),
    "spork_plan_advance": (ctypes.c_int, [_p, _p, _p, _p]),
    "spork_workspace_clear": (ctypes.c_int, [_p, _p, ctypes.c_size_t, _p]),
    "spork_attn_decode": (ctypes.c_int, [_p, _p, _p, _p, _p, _p, _p, _p, ctypes.c_size_t, _p]),
    "spork_verify_workspace_bytes": (ctypes.c_int, [_c_i32, _c_i32, _c_i32,
                                                    ctypes.POINTER(ctypes.c_size_t)]),
    "spork_verify_accept": (ctypes.c_int, [_p, _p, _p, _p, _p, _p, _p, _p, _c_i32, _c_i32, _p,
                                           _c_i32, _c_i32, _p, _p, _p, _p, ctypes.c_size_t, _p]),
    "spork_verify_accept_noalloc": (ctypes.c_int, [_p, _p, _p, _p, _p, _p, _p, _p, _c_i32, _c_i32, _p,
                                                   _c_i32, _c_i32, _p, _p, _p, _p]),
    "spork_confidence_workspace_bytes": (ctypes.c_int, [_c_i32, _c_i32,
                                                        ctypes.POINTER(ctypes.c_size_t)]),
    "spork_probe_confidence": (ctypes.c_int, [_p, _c_i32, _c_i32, _c_i32, _p, _c_i32, ctypes.c_float,
                                              _p, _p, _p, _p, _p, ctypes.c_size_t, _p]),
    "spork_ngram_workspace_bytes": (ctypes.c_int, [_c_i32, _c_i64, ctypes.POINTER(ctypes.c_size_t)]),
    "spork_ngram_propose": (ctypes.c_int, [_p, _p, _c_i32, _c_i64, _c_i32, _c_i32, _c_i32, _p, _p, _p,
                                           ctypes.c_size_t, _p]),
    "spork_read_ceiling": (ctypes.c_int, [_p, _c_i64, _c_i32, _c_i32, _p, _p]),
    "spork_timing_enable": (ctypes.c_int, [_c_i32]),
    "spork_timing_read": (ctypes.c_int, [_p, _p]),
}

_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        path = _HOST_SANITIZER_LIB or LIB_PATH
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with "
                               "`python -m paper_2607_03333_amd.build` (there is no fallback)")
        handle = ctypes.CDLL(path)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def _check(rc):
    if rc != SPORK_OK:
        raise SporkError(rc, lib().spork_last_error().decode())


def _ptr(x):
    """Device pointer of a torch tensor, host pointer of a numpy array, or NULL."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        if not x.flags["C_CONTIGUOUS"]:
            raise ValueError("numpy arguments must be C-contiguous")
        return x.ctypes.data
    if not x.is_contiguous():
        raise ValueError("tensor arguments must be contiguous")
    return x.data_ptr()


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _i32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def make_shape(hq, hkv, head_dim, block_size, dtype, sm_scale):
    return spork_shape(hq, hkv, head_dim, block_size, dtype, sm_scale)


# ---- block manager ------------------------------------------------------------
def spork_version():
    return lib().spork_version()


def spork_cache_create(num_blocks, block_size, free_order=None):
    out = _p()
    order = None if free_order is None else _i32(free_order)
    _check(lib().spork_cache_create(num_blocks, block_size, _ptr(order), ctypes.byref(out)))
    return out


def spork_cache_destroy(cache):
    _check(lib().spork_cache_destroy(cache))


def spork_seq_new(cache):
    s = _c_i32()
    _check(lib().spork_seq_new(cache, ctypes.byref(s)))
    return s.value


def spork_seq_append(cache, seq, n_tokens):
    """Returns (slots int64 array, list of (src, dst, n_valid) copies)."""
    slots = np.zeros(max(n_tokens, 1), dtype=np.int64)
    cow = np.zeros(3, dtype=np.int32)
    n_cow = _c_i32()
    _check(lib().spork_seq_append(cache, seq, n_tokens, _ptr(slots), _ptr(cow), ctypes.byref(n_cow)))
    return slots[:n_tokens], ([tuple(int(x) for x in cow)] if n_cow.value else [])


def spork_seq_append_batch(cache, seqs, n_tokens):
    """Returns (slots int64 array in batch order, list of (src, dst, n_valid) copies)."""
    seqs, n_tokens = _i32(seqs), _i32(n_tokens)
    slots = np.zeros(max(int(np.maximum(n_tokens, 0).sum()), 1), dtype=np.int64)
    cow = np.zeros(max(3 * len(seqs), 3), dtype=np.int32)
    n_cow = _c_i32()
    _check(lib().spork_seq_append_batch(cache, _ptr(seqs), _ptr(n_tokens), len(seqs), _ptr(slots), _ptr(cow),
                                        ctypes.byref(n_cow)))
    return slots[:int(np.maximum(n_tokens, 0).sum())], [tuple(int(x) for x in cow[3 * i:3 * i + 3])
                                                        for i in range(n_cow.value)]


def spork_fork(cache, parent_seq):
    c = _c_i32()
    _check(lib().spork_fork(cache, parent_seq, ctypes.byref(c)))
    return c.value


def spork_seq_free(cache, seq):
    _check(lib().spork_seq_free(cache, seq))


def spork_seq_len(cache, seq):
    n = _c_i32()
    _check(lib().spork_seq_len(cache, seq, ctypes.byref(n)))
    return n.value


def spork_block_table(cache, seq):
    n = _c_i32()
    rc = lib().spork_block_table(cache, seq, None, 0, ctypes.byref(n))
    if rc not in (SPORK_OK, SPORK_E_CAPACITY):
        _check(rc)
    out = np.zeros(max(n.value, 1), dtype=np.int32)
    _check(lib().spork_block_table(cache, seq, _ptr(out), n.value, ctypes.byref(n)))
    return out[: n.value]


def spork_refcount(cache, block):
    r = _c_i32()
    _check(lib().spork_refcount(cache, block, ctypes.byref(r)))
    return r.value


def spork_free_blocks(cache):
    n = _c_i32()
    rc = lib().spork_free_blocks(cache, None, 0, ctypes.byref(n))
    if rc not in (SPORK_OK, SPORK_E_CAPACITY):
        _check(rc)
    out = np.zeros(max(n.value, 1), dtype=np.int32)
    _check(lib().spork_free_blocks(cache, _ptr(out), n.value, ctypes.byref(n)))
    return out[: n.value]


# ---- KV writes --------------------------------------------------------------
def spork_kv_write(shape, k_cache, v_cache, num_blocks, slots, k_new, v_new, bad_slots=None,
                   stream=None):
    _check(lib().spork_kv_write(ctypes.byref(shape), _ptr(k_cache), _ptr(v_cache), num_blocks,
                                _ptr(slots), _ptr(k_new), _ptr(v_new), int(slots.numel()),
                                _ptr(bad_slots), _stream(stream)))


def spork_kv_copy(shape, k_cache, v_cache, num_blocks, src_block, dst_block, n_valid, stream=None):
    _check(lib().spork_kv_copy(ctypes.byref(shape), _ptr(k_cache), _ptr(v_cache), num_blocks,
                               src_block, dst_block, n_valid, _stream(stream)))


# ---- plan -------------------------------------------------------------------
def spork_plan_create(cache, shape, seqs, n_rows, groups, n_cu=0):
    seqs, n_rows, groups = _i32(seqs), _i32(n_rows), _i32(groups)
    if not (len(seqs) == len(n_rows) == len(groups)):
        raise ValueError("seqs, n_rows and groups must have one entry per thread")
    out = _p()
    _check(lib().spork_plan_create(cache, ctypes.byref(shape), _ptr(seqs), _ptr(n_rows), _ptr(groups),
                                   len(seqs), n_cu, ctypes.byref(out)))
    return out


def spork_plan_destroy(plan):
    _check(lib().spork_plan_destroy(plan))


def spork_plan_get_info(plan):
    info = spork_plan_info()
    _check(lib().spork_plan_get_info(plan, ctypes.byref(info)))
    return {name: getattr(info, name) for name, _ in spork_plan_info._fields_}


def spork_plan_advance(plan, cache, dev_image, stream=None):
    _check(lib().spork_plan_advance(plan, cache, _ptr(dev_image), _stream(stream)))


def spork_plan_image(plan):
    n = spork_plan_get_info(plan)["image_bytes"]
    img = np.zeros(max(n, 1), dtype=np.uint8)
    _check(lib().spork_plan_image(plan, _ptr(img), img.nbytes))
    return img[:n]


# ---- hot path ---------------------------------------------------------------
def spork_workspace_clear(plan, workspace, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().spork_workspace_clear(plan, _ptr(workspace), ws_bytes, _stream(stream)))


def spork_attn_decode(plan, dev_image, q, k_cache, v_cache, out, lse, workspace, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().spork_attn_decode(plan, _ptr(dev_image), _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                   _ptr(out), _ptr(lse), _ptr(workspace), ws_bytes, _stream(stream)))


def spork_verify_workspace_bytes(n_verify, k_drafts, vocab):
    b = ctypes.c_size_t()
    _check(lib().spork_verify_workspace_bytes(n_verify, k_drafts, vocab, ctypes.byref(b)))
    return b.value


def spork_verify_accept(plan, dev_image, q, k_cache, v_cache, out, lse, logits, logits_dtype, vocab,
                        drafts, n_verify, k_drafts, accept_len, next_token, argmax_out, workspace,
                        stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().spork_verify_accept(plan, _ptr(dev_image), _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                     _ptr(out), _ptr(lse), _ptr(logits), logits_dtype, vocab,
                                     _ptr(drafts), n_verify, k_drafts, _ptr(accept_len),
                                     _ptr(next_token), _ptr(argmax_out), _ptr(workspace), ws_bytes,
                                     _stream(stream)))


def spork_verify_accept_noalloc(plan, dev_image, q, k_cache, v_cache, out, lse, logits, logits_dtype, vocab,
                                drafts, n_verify, k_drafts, accept_len, next_token, argmax_out, stream=None):
    _check(lib().spork_verify_accept_noalloc(plan, _ptr(dev_image), _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                             _ptr(out), _ptr(lse), _ptr(logits), logits_dtype, vocab,
                                             _ptr(drafts), n_verify, k_drafts, _ptr(accept_len),
                                             _ptr(next_token), _ptr(argmax_out), _stream(stream)))


def spork_confidence_workspace_bytes(n_rows, vocab):
    b = ctypes.c_size_t()
    _check(lib().spork_confidence_workspace_bytes(n_rows, vocab, ctypes.byref(b)))
    return b.value


def spork_probe_confidence(logits, logits_dtype, vocab, n_rows, span_off, n_probes, theta,
                           argmax_out, logprob_out, confidence_out, commit_out, workspace, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().spork_probe_confidence(_ptr(logits), logits_dtype, vocab, n_rows, _ptr(span_off),
                                        n_probes, float(theta), _ptr(argmax_out), _ptr(logprob_out),
                                        _ptr(confidence_out), _ptr(commit_out), _ptr(workspace),
                                        ws_bytes, _stream(stream)))


def spork_ngram_workspace_bytes(n_seqs, max_len):
    b = ctypes.c_size_t()
    _check(lib().spork_ngram_workspace_bytes(n_seqs, max_len, ctypes.byref(b)))
    return b.value


def spork_ngram_propose(tokens, seq_off, n_seqs, max_len, n_min, n_max, k, drafts, n_drafts, workspace,
                        stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib().spork_ngram_propose(_ptr(tokens), _ptr(seq_off), n_seqs, max_len, n_min, n_max, k,
                                     _ptr(drafts), _ptr(n_drafts), _ptr(workspace), ws_bytes,
                                     _stream(stream)))


# ---- measurement aid --------------------------------------------------------
def spork_read_ceiling(src, nbytes, grid, mode, sink, stream=None):
    _check(lib().spork_read_ceiling(_ptr(src), nbytes, grid, mode, _ptr(sink), _stream(stream)))


# ---- kernel timing ------------------------------------------------------------
def spork_timing_enable(on):
    _check(lib().spork_timing_enable(1 if on else 0))


def spork_timing_read():
    """{kernel name: (total ms, launches)} since the last read."""
    ms = np.zeros(SPORK_KERNEL_KINDS, dtype=np.float32)
    n = np.zeros(SPORK_KERNEL_KINDS, dtype=np.int32)
    _check(lib().spork_timing_read(_ptr(ms), _ptr(n)))
    return {KERNEL_NAMES[k]: (float(ms[k]), int(n[k])) for k in range(SPORK_KERNEL_KINDS)}
