"""ctypes binding of libchimera.so (include/chimera.h).  Argument marshalling
only: every function keeps the C name and raises ChimeraError on a
non-zero status.  Loading fails loudly when the library is not built."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libchimera.so")

CHIMERA_F32, CHIMERA_BF16 = 0, 1
CHIMERA_DECODE_GREEDY, CHIMERA_DECODE_TYPICAL = 0, 1
CHIMERA_DRAFT_CHAIN, CHIMERA_DRAFT_BRANCH = 0, 1
DBG_VERIFY_LOGITS, DBG_DRAFT_LOGITS, DBG_TREE_TOKENS, DBG_DRAFT_LISTS, DBG_SEQ_LEN, DBG_TOKENS = range(6)
CHIMERA_MAX_PIPELINED_STEPS = 64
CHIMERA_OK, CHIMERA_EINVAL, CHIMERA_ENOMEM, CHIMERA_ECAPACITY, CHIMERA_EHIP, CHIMERA_ESTATE = 0, -1, -2, -3, -4, -5
STATUS = {0: "OK", -1: "EINVAL", -2: "ENOMEM", -3: "ECAPACITY", -4: "EHIP", -5: "ESTATE"}


class ChimeraError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class chimera_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("n_draft_heads", ctypes.c_int32), ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("dtype", ctypes.c_int32), ("max_positions", ctypes.c_int32)]


class chimera_tensor(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("data", ctypes.c_void_p), ("numel", ctypes.c_int64),
                ("dtype", ctypes.c_int32), ("on_device", ctypes.c_int32)]


class chimera_profile(ctypes.Structure):
    _fields_ = [("steps", ctypes.c_int64), ("ms_draft", ctypes.c_double), ("ms_verify", ctypes.c_double),
                ("ms_tail", ctypes.c_double), ("ms_gemm_verify", ctypes.c_double),
                ("gemm_verify_launches", ctypes.c_int64), ("gemm_verify_bytes", ctypes.c_double),
                ("verify_bytes", ctypes.c_double), ("ms_draft_median", ctypes.c_double),
                ("ms_verify_median", ctypes.c_double), ("ms_step_median", ctypes.c_double)]


_lib = None
P = ctypes.c_void_p
I32, I64 = ctypes.c_int32, ctypes.c_int64
PI32 = ctypes.POINTER(ctypes.c_int32)
PI64 = ctypes.POINTER(ctypes.c_int64)

_PROTOS = {
    "chimera_weight_bytes": [ctypes.POINTER(chimera_config), PI64],
    "chimera_load": [ctypes.POINTER(chimera_config), ctypes.POINTER(chimera_tensor), I32, P, I64, P,
                     ctypes.POINTER(P)],
    "chimera_kv_bytes": [P, I32, I32, I32, I32, PI64],
    "chimera_kv_create": [P, I32, I32, I32, I32, PI32, P, I64, ctypes.POINTER(P)],
    "chimera_ctx_bytes": [P, P, I32, PI64],
    "chimera_ctx_create": [P, P, PI32, PI32, I32, P, I64, ctypes.POINTER(P)],
    "chimera_prefill": [P, P, P, PI32, PI32, I32, PI32, P],
    "chimera_step": [P, P, P, PI32, PI32, PI32, P],
    "chimera_steps": [P, P, P, I32, PI32, PI32, PI32, P],
    "chimera_set_forcing": [P, P, P, I32],
    "chimera_set_tree_tokens": [P, PI32, I32],
    "chimera_debug_copy": [P, I32, P, I64],
    "chimera_kv_read": [P, I32, I32, I32, I32, P, P],
    "chimera_profile_enable": [P, I32],
    "chimera_set_graph": [P, I32],
    "chimera_profile_read": [P, ctypes.POINTER(chimera_profile)],
    "chimera_debug_gemm": [I32, P, P, I32, I32, I32, ctypes.POINTER(ctypes.c_float)],
    "chimera_gemm_static": [I32, P, P, I32, I32, I32, P, P],
    "chimera_trigram_cache_bytes": [P, I32, PI64],
    "chimera_set_decoding": [P, I32, ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_uint64],
    "chimera_set_drafting": [P, I32],
    "chimera_set_trigram_cache": [P, P, I64, I32],
    "chimera_trigram_cache_stats": [P, PI64, PI64],
    "chimera_compaction_check_bytes": [P, PI64],
    "chimera_set_compaction_check": [P, P, I64],
    "chimera_compaction_check_read": [P, PI64, PI64],
}


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2402_15758_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, args in _PROTOS.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = ctypes.c_int
        L.chimera_last_error.restype = ctypes.c_char_p
        L.chimera_last_error.argtypes = []
        for name in ("chimera_ctx_free", "chimera_kv_free", "chimera_free"):
            getattr(L, name).argtypes = [P]
            getattr(L, name).restype = None
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        raise ChimeraError(status, lib().chimera_last_error().decode(errors="replace"))


def _i32p(arr):
    """A ctypes int32 pointer to a contiguous numpy int32 array (or None)."""
    if arr is None:
        return None
    return arr.ctypes.data_as(PI32)


def chimera_last_error() -> str:
    return lib().chimera_last_error().decode(errors="replace")


def chimera_weight_bytes(cfg: chimera_config) -> int:
    out = I64()
    _check(lib().chimera_weight_bytes(ctypes.byref(cfg), ctypes.byref(out)))
    return out.value


def chimera_load(cfg: chimera_config, tensors, arena_ptr: int, arena_bytes: int, stream: int) -> int:
    arr = (chimera_tensor * len(tensors))(*tensors)
    out = P()
    _check(lib().chimera_load(ctypes.byref(cfg), arr, len(tensors), arena_ptr, arena_bytes, stream, ctypes.byref(out)))
    return out.value


def chimera_kv_bytes(model: int, max_batch: int, max_len: int, n_pages: int, page_size: int) -> int:
    out = I64()
    _check(lib().chimera_kv_bytes(model, max_batch, max_len, n_pages, page_size, ctypes.byref(out)))
    return out.value


def chimera_kv_create(model: int, max_batch: int, max_len: int, n_pages: int, page_size: int, page_order,
                      arena_ptr: int, arena_bytes: int) -> int:
    out = P()
    _check(lib().chimera_kv_create(model, max_batch, max_len, n_pages, page_size, _i32p(page_order), arena_ptr,
                                   arena_bytes, ctypes.byref(out)))
    return out.value


def chimera_ctx_bytes(model: int, kv: int, n_nodes: int) -> int:
    out = I64()
    _check(lib().chimera_ctx_bytes(model, kv, n_nodes, ctypes.byref(out)))
    return out.value


def chimera_ctx_create(model: int, kv: int, parent, rank, arena_ptr: int, arena_bytes: int) -> int:
    out = P()
    _check(lib().chimera_ctx_create(model, kv, _i32p(parent), _i32p(rank), len(parent), arena_ptr, arena_bytes,
                                    ctypes.byref(out)))
    return out.value


def chimera_prefill(model: int, kv: int, ctx: int, tokens, lens, first_tokens, stream: int):
    _check(lib().chimera_prefill(model, kv, ctx, _i32p(tokens), _i32p(lens), len(lens), _i32p(first_tokens), stream))


def chimera_step(model: int, kv: int, ctx: int, new_tokens, n_new, path_nodes, stream: int):
    _check(lib().chimera_step(model, kv, ctx, _i32p(new_tokens), _i32p(n_new), _i32p(path_nodes), stream))


def chimera_steps(model: int, kv: int, ctx: int, n_steps: int, new_tokens, n_new, path_nodes, stream: int):
    _check(lib().chimera_steps(model, kv, ctx, n_steps, _i32p(new_tokens), _i32p(n_new), _i32p(path_nodes),
                               stream))


def chimera_set_forcing(ctx: int, ref_ptr, ok_ptr, stride: int):
    _check(lib().chimera_set_forcing(ctx, ref_ptr, ok_ptr, stride))


def chimera_set_tree_tokens(ctx: int, tokens, batch: int):
    _check(lib().chimera_set_tree_tokens(ctx, _i32p(tokens), batch))


def chimera_debug_copy(ctx: int, what: int, dst_ptr: int, nbytes: int):
    _check(lib().chimera_debug_copy(ctx, what, dst_ptr, nbytes))


def chimera_kv_read(kv: int, layer: int, b: int, pos0: int, count: int, k_ptr: int, v_ptr: int):
    _check(lib().chimera_kv_read(kv, layer, b, pos0, count, k_ptr, v_ptr))


def chimera_profile_enable(ctx: int, enable: bool):
    _check(lib().chimera_profile_enable(ctx, 1 if enable else 0))


def chimera_set_graph(ctx: int, enable: bool):
    _check(lib().chimera_set_graph(ctx, 1 if enable else 0))


def chimera_profile_read(ctx: int) -> chimera_profile:
    out = chimera_profile()
    _check(lib().chimera_profile_read(ctx, ctypes.byref(out)))
    return out


def chimera_debug_gemm(dtype: int, x_ptr: int, w_ptr: int, M: int, N: int, K: int, y_ptr: int):
    _check(lib().chimera_debug_gemm(dtype, x_ptr, w_ptr, M, N, K, ctypes.cast(y_ptr, ctypes.POINTER(ctypes.c_float))))


def chimera_gemm_static(dtype: int, x_ptr: int, w_ptr: int, M: int, N: int, K: int, y_ptr: int, stream: int):
    _check(lib().chimera_gemm_static(dtype, x_ptr, w_ptr, M, N, K, y_ptr, stream))


def chimera_set_drafting(ctx: int, mode: int):
    _check(lib().chimera_set_drafting(ctx, mode))


def chimera_set_decoding(ctx: int, mode: int, temperature: float = 1.0, eps: float = 0.09, delta: float = 0.3,
                         seed: int = 0):
    _check(lib().chimera_set_decoding(ctx, mode, temperature, eps, delta, seed))


def chimera_trigram_cache_bytes(model: int, n_entries: int) -> int:
    out = I64()
    _check(lib().chimera_trigram_cache_bytes(model, n_entries, ctypes.byref(out)))
    return out.value


def chimera_set_trigram_cache(ctx: int, arena_ptr, arena_bytes: int, n_entries: int):
    _check(lib().chimera_set_trigram_cache(ctx, arena_ptr, arena_bytes, n_entries))


def chimera_trigram_cache_stats(ctx: int):
    lookups, hits = I64(), I64()
    _check(lib().chimera_trigram_cache_stats(ctx, ctypes.byref(lookups), ctypes.byref(hits)))
    return lookups.value, hits.value


def chimera_compaction_check_bytes(ctx: int) -> int:
    out = I64()
    _check(lib().chimera_compaction_check_bytes(ctx, ctypes.byref(out)))
    return out.value


def chimera_set_compaction_check(ctx: int, arena_ptr, arena_bytes: int):
    _check(lib().chimera_set_compaction_check(ctx, arena_ptr, arena_bytes))


def chimera_compaction_check_read(ctx: int):
    rows, bad = I64(), I64()
    _check(lib().chimera_compaction_check_read(ctx, ctypes.byref(rows), ctypes.byref(bad)))
    return rows.value, bad.value


def chimera_ctx_free(ctx: int):
    lib().chimera_ctx_free(ctx)


def chimera_kv_free(kv: int):
    lib().chimera_kv_free(kv)


def chimera_free(model: int):
    lib().chimera_free(model)
