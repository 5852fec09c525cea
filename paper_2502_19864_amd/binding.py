"""ctypes binding of libringada.so (include/ringada.h): same names, argument
marshalling only.  Every function raises RingadaError on a non-OK status,
with the library's message."""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, byref, c_char, c_char_p, c_double, c_float, c_int32, c_int64, c_size_t, c_void_p

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libringada.so")

RINGADA_OK, RINGADA_E_INVALID, RINGADA_E_STATE, RINGADA_E_WORKSPACE, RINGADA_E_UNSUPPORTED, RINGADA_E_HIP = range(6)
ARCH_POSTLN_GELU, ARCH_PRERMS_SWIGLU = 0, 1
F32, BF16 = 0, 1
PLACEMENT_HOULSBY, PLACEMENT_FFN = 0, 1
STATUS_NAMES = {0: "OK", 1: "E_INVALID", 2: "E_STATE", 3: "E_WORKSPACE", 4: "E_UNSUPPORTED", 5: "E_HIP"}


class RingadaError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), msg))
        self.status = status


class StageDesc(ctypes.Structure):
    _fields_ = [("arch", c_int32), ("dtype", c_int32), ("n_blocks", c_int32), ("d_model", c_int32),
                ("n_heads", c_int32), ("d_ffn", c_int32), ("d_adapter", c_int32),
                ("max_batch", c_int32), ("max_seq", c_int32), ("norm_eps", c_float),
                ("rope_theta", c_float), ("placement", c_int32)]


class BlockWeights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("w_qkv", "b_qkv", "w_o", "b_o", "norm1_g", "norm1_b", "w_in",
                                        "b_in", "w_out", "b_out", "norm2_g", "norm2_b")]


class Adapter(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("w_down", "w_up", "g_down", "g_up")]


class Optim(ctypes.Structure):
    _fields_ = [("kind", c_int32), ("lr", c_float)]


class ProfEntry(ctypes.Structure):
    _fields_ = [("name", c_char * 64), ("launches", c_int32), ("total_ms", c_double),
                ("flops", c_double), ("bytes", c_double)]


# (name, restype, argtypes): every symbol declared in include/ringada.h
SIGNATURES = [
    ("ringada_stage_plan", c_int32, [POINTER(StageDesc), c_int32, c_int32, c_int32,
                                     POINTER(c_size_t), POINTER(c_size_t)]),
    ("ringada_local_cutoff", c_int32, [c_int32, c_int32, c_int32, c_int32]),
    ("ringada_stage_plan_weights", c_int32, [POINTER(StageDesc), POINTER(c_size_t), POINTER(c_size_t)]),
    ("ringada_stage_create", c_int32, [POINTER(StageDesc), c_void_p, c_size_t, POINTER(c_void_p)]),
    ("ringada_stage_bind_block", c_int32, [c_void_p, c_int32, POINTER(BlockWeights), POINTER(Adapter),
                                           POINTER(Adapter), c_void_p, c_size_t, c_void_p]),
    ("ringada_stage_sync_adapters", c_int32, [c_void_p, c_void_p]),
    ("ringada_stage_destroy", None, [c_void_p]),
    ("ringada_stage_forward", c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_int32, c_int32, c_int32,
                                        c_void_p, c_size_t, c_void_p, c_size_t]),
    ("ringada_stage_backward", c_int32, [c_void_p, c_void_p, c_void_p, c_int32, c_void_p]),
    ("ringada_adapter_step", c_int32, [c_void_p, c_void_p, c_int32, POINTER(Optim)]),
    ("ringada_loss_mse", c_int32, [c_void_p, c_int32, c_void_p, c_void_p, c_int64, c_void_p, c_void_p]),
    ("ringada_head_ce", c_int32, [c_void_p, c_int32, c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                  c_int32, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]),
    ("ringada_sgd_f32", c_int32, [c_void_p, c_void_p, c_void_p, c_int64, c_float]),
    ("ringada_last_error", c_char_p, []),
    ("ringada_prof_begin", c_int32, [c_void_p]),
    ("ringada_prof_end", c_int32, [c_void_p, POINTER(ProfEntry), c_int32, POINTER(c_int32)]),
]

_lib = None


def lib():
    """Loads libringada.so (built in-tree); raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libringada.so is not built (run `python -m paper_2502_19864_amd.build`); "
                               "there is no fallback implementation")
        L = ctypes.CDLL(LIB_PATH)
        for name, res, args in SIGNATURES:
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(status):
    if status != RINGADA_OK:
        msg = lib().ringada_last_error()
        raise RingadaError(status, msg.decode() if msg else "")


def _p(x):
    """Device pointer of a torch tensor, an int address or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def ringada_stage_plan(desc, batch, seq, lowest_unfrozen):
    st, sc = c_size_t(0), c_size_t(0)
    _check(lib().ringada_stage_plan(byref(desc), batch, seq, lowest_unfrozen, byref(st), byref(sc)))
    return st.value, sc.value


def ringada_local_cutoff(n_tm, depth, first_block, n_local):
    return lib().ringada_local_cutoff(n_tm, depth, first_block, n_local)


def ringada_stage_plan_weights(desc):
    blk, stg = c_size_t(0), c_size_t(0)
    _check(lib().ringada_stage_plan_weights(byref(desc), byref(blk), byref(stg)))
    return blk.value, stg.value


def ringada_stage_create(desc, stage_mem, stage_mem_bytes):
    h = c_void_p()
    _check(lib().ringada_stage_create(byref(desc), _p(stage_mem), stage_mem_bytes, byref(h)))
    return h


def ringada_stage_bind_block(stage, block, frozen, attn_adapter, ffn_adapter, block_mem, block_mem_bytes, stream):
    """attn_adapter is None for a stage with the single (FFN) placement."""
    _check(lib().ringada_stage_bind_block(stage, block, byref(frozen),
                                          None if attn_adapter is None else byref(attn_adapter),
                                          byref(ffn_adapter), _p(block_mem), block_mem_bytes, stream))


def ringada_stage_sync_adapters(stage, stream):
    _check(lib().ringada_stage_sync_adapters(stage, stream))


def ringada_stage_destroy(stage):
    lib().ringada_stage_destroy(stage)


def ringada_stage_forward(stage, stream, x, y, batch, seq, lowest_unfrozen, stash, stash_bytes, scratch,
                          scratch_bytes):
    _check(lib().ringada_stage_forward(stage, stream, _p(x), _p(y), batch, seq, lowest_unfrozen, _p(stash),
                                       stash_bytes, _p(scratch), scratch_bytes))


def ringada_stage_backward(stage, stream, dy, lowest_unfrozen, dx_in):
    _check(lib().ringada_stage_backward(stage, stream, _p(dy), lowest_unfrozen, _p(dx_in)))


def ringada_adapter_step(stage, stream, lowest_unfrozen, lr, kind=0):
    opt = Optim(kind, lr)
    _check(lib().ringada_adapter_step(stage, stream, lowest_unfrozen, byref(opt)))


def ringada_loss_mse(stream, dtype, y, target, n, dy, loss):
    _check(lib().ringada_loss_mse(stream, dtype, _p(y), _p(target), n, _p(dy), _p(loss)))


def ringada_head_ce(stream, dtype, y, batch, seq, d, w_h, b_h, n_classes, labels, dy, g_wh, g_bh, loss):
    _check(lib().ringada_head_ce(stream, dtype, _p(y), batch, seq, d, _p(w_h), _p(b_h), n_classes, _p(labels),
                                 _p(dy), _p(g_wh), _p(g_bh), _p(loss)))


def ringada_sgd_f32(stream, w, g, n, lr):
    _check(lib().ringada_sgd_f32(stream, _p(w), _p(g), n, lr))


def ringada_last_error():
    m = lib().ringada_last_error()
    return m.decode() if m else ""


def ringada_prof_begin(stage):
    _check(lib().ringada_prof_begin(stage))


def ringada_prof_end(stage, max_entries=64):
    arr = (ProfEntry * max_entries)()
    n = c_int32(0)
    _check(lib().ringada_prof_end(stage, arr, max_entries, byref(n)))
    return [dict(name=arr[i].name.decode(), launches=arr[i].launches, total_ms=arr[i].total_ms,
                 flops=arr[i].flops, bytes=arr[i].bytes) for i in range(min(n.value, max_entries))]
