"""Thin Python binding of libams (C ABI in include/ams.h).

Each ``ams_*`` function here marshals torch tensors (device memory) and the
current HIP stream into the C call of the same name and raises AmsError on a
non-OK status.  No step of the method runs in Python: there is no fallback,
and loading fails loudly when libams.so has not been built.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libams.so")

AMS_F32, AMS_BF16, AMS_F32_X3 = 0, 1, 2
AMS_POOL_SUM, AMS_POOL_MAX, AMS_POOL_ATT = 0, 1, 2
POOL = {"sum": AMS_POOL_SUM, "max": AMS_POOL_MAX, "att": AMS_POOL_ATT}
STATUS = {0: "AMS_OK", 1: "AMS_ERR_NULL", 2: "AMS_ERR_SIZE", 3: "AMS_ERR_DTYPE", 4: "AMS_ERR_DIMS",
          5: "AMS_ERR_WORKSPACE", 6: "AMS_ERR_HIP", 7: "AMS_ERR_ID_RANGE", 8: "AMS_ERR_MODE",
          9: "AMS_ERR_CAPACITY"}
DEDUP_NOALLOC_MAX_OCC = 1 << 20     # AMS_DEDUP_NOALLOC_MAX_OCC
EXPORTS = ["ams_status_str", "ams_build_info", "ams_dedup_workspace", "ams_dedup", "ams_dedup_noalloc",
           "ams_embed_workspace", "ams_embed_fwd", "ams_embed_bwd", "ams_pool_fwd",
           "ams_pool_workspace", "ams_pool_bwd", "ams_timing_enable", "ams_timing_read",
           "ams_bag_fwd", "ams_bag_workspace", "ams_bag_bwd", "ams_ctr_workspace", "ams_ctr_fwd_bwd",
           "ams_adagrad_rows", "ams_pool_query_fwd", "ams_pool_query_bwd",
           "ams_adam_update", "ams_pool_concat_fwd", "ams_pool_concat_bwd", "ams_dssm_workspace",
           "ams_dssm_fwd_bwd", "ams_peak_copy", "ams_peak_read", "ams_peak_gather", "ams_peak_mfma"]


class AmsError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)} ({_text(status)})")


class ams_kernel_time(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int64), ("total_ms", ctypes.c_double)]


class ams_mlp(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("dims", ctypes.c_int32 * 4),
                ("dtype", ctypes.c_int32), ("final_relu", ctypes.c_int32)]


class ams_ctr(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("dims", ctypes.c_int32 * 4)]


_lib = None


def load() -> ctypes.CDLL:
    """Load libams.so (raises if it has not been built: there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing; build it with `python -m paper_1711_06505_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    M = ctypes.POINTER(ams_mlp)
    PP = ctypes.POINTER(ctypes.c_void_p)
    lib.ams_status_str.restype = ctypes.c_char_p
    lib.ams_status_str.argtypes = [ctypes.c_int]
    lib.ams_build_info.restype = ctypes.c_char_p
    lib.ams_dedup_workspace.restype = sz
    lib.ams_dedup_workspace.argtypes = [i64, i32]
    lib.ams_dedup.restype = ctypes.c_int
    lib.ams_dedup.argtypes = [P, i64, i32, P, P, P, P, P, P, P, sz, P]
    lib.ams_dedup_noalloc.restype = ctypes.c_int
    lib.ams_dedup_noalloc.argtypes = [P, i64, i32, P, P, P, P, P, P, P]
    lib.ams_embed_workspace.restype = sz
    lib.ams_embed_workspace.argtypes = [M, i32]
    lib.ams_embed_fwd.restype = ctypes.c_int
    lib.ams_embed_fwd.argtypes = [M, P, i64, P, P, i32, P, P, P, P, P, P, PP, P, P, P, P, sz, P]
    lib.ams_embed_bwd.restype = ctypes.c_int
    lib.ams_embed_bwd.argtypes = [M, P, i64, P, P, i32, P, P, P, PP, P, P, P, P, P, P, P, P, P, P, PP, P, sz,
                                  P]
    lib.ams_pool_fwd.restype = ctypes.c_int
    lib.ams_pool_fwd.argtypes = [i32, i32, i32, P, i64, P, i32, P, P, P, P, P]
    lib.ams_pool_workspace.restype = sz
    lib.ams_pool_workspace.argtypes = [i32, i32, i64, i32, i32]
    lib.ams_pool_bwd.restype = ctypes.c_int
    lib.ams_pool_bwd.argtypes = [i32, i32, i32, P, i64, P, P, P, P, i32, P, P, P, P, P, P, P, P, sz, P]
    C = ctypes.POINTER(ams_ctr)
    lib.ams_bag_fwd.restype = ctypes.c_int
    lib.ams_bag_fwd.argtypes = [i32, i32, P, i64, P, P, i64, P, P]
    lib.ams_bag_workspace.restype = sz
    lib.ams_bag_workspace.argtypes = [i32, i64, i32, i32]
    lib.ams_bag_bwd.restype = ctypes.c_int
    lib.ams_bag_bwd.argtypes = [i32, i32, P, i64, P, P, P, P, i32, P, P, P, P, sz, P]
    lib.ams_ctr_workspace.restype = sz
    lib.ams_ctr_workspace.argtypes = [C, i32]
    lib.ams_ctr_fwd_bwd.restype = ctypes.c_int
    lib.ams_ctr_fwd_bwd.argtypes = [C, i32, i32, PP, ctypes.POINTER(i32), P, PP, PP, PP, P, P, PP, PP, PP, PP,
                                    P, sz, P]
    lib.ams_dssm_workspace.restype = sz
    lib.ams_dssm_workspace.argtypes = [C, C, i32]
    lib.ams_dssm_fwd_bwd.restype = ctypes.c_int
    lib.ams_dssm_fwd_bwd.argtypes = [C, C, i32, i32, PP, ctypes.POINTER(i32), i32, PP, ctypes.POINTER(i32), P,
                                     PP, PP, PP, PP, PP, PP, P, P, PP, PP, PP, PP, PP, PP, PP, PP, P, sz, P]
    lib.ams_adagrad_rows.restype = ctypes.c_int
    lib.ams_adagrad_rows.argtypes = [i32, P, P, i32, P, P, i64, P, ctypes.c_float, ctypes.c_float, P]
    lib.ams_pool_query_fwd.restype = ctypes.c_int
    lib.ams_pool_query_fwd.argtypes = [i32, i32, P, i64, P, i32, P, P, P, P, P]
    lib.ams_pool_query_bwd.restype = ctypes.c_int
    lib.ams_pool_query_bwd.argtypes = [i32, i32, P, i64, P, P, P, P, i32, P, P, P, P, P, P, P, i32, P, sz, P]
    lib.ams_pool_concat_fwd.restype = ctypes.c_int
    lib.ams_pool_concat_fwd.argtypes = [i32, i32, i32, P, i64, P, i32, P, P, P, P]
    lib.ams_pool_concat_bwd.restype = ctypes.c_int
    lib.ams_pool_concat_bwd.argtypes = [i32, i32, i32, P, i64, P, P, P, P, i32, P, P, P, P, sz, P]
    f = ctypes.c_float
    lib.ams_adam_update.restype = ctypes.c_int
    lib.ams_adam_update.argtypes = [i64, P, P, P, P, f, f, f, f, i64, P, P]
    for name, args in (("ams_peak_copy", [P, P, i64, i32, P]), ("ams_peak_read", [P, i64, i32, P, P]),
                       ("ams_peak_gather", [P, i64, i32, P, i32, i32, P, i32, P, P]),
                       ("ams_peak_mfma", [i32, P, i32, i32, P, P])):
        getattr(lib, name).restype = ctypes.c_int
        getattr(lib, name).argtypes = args
    lib.ams_timing_enable.restype = ctypes.c_int
    lib.ams_timing_enable.argtypes = [ctypes.c_int]
    lib.ams_timing_read.restype = ctypes.c_int
    lib.ams_timing_read.argtypes = [ctypes.POINTER(ams_kernel_time), ctypes.c_int, ctypes.POINTER(ctypes.c_int)]
    _lib = lib
    return lib


def _text(status: int) -> str:
    try:
        return load().ams_status_str(status).decode()
    except Exception:  # pragma: no cover
        return "?"


def _check(rc: int, where: str):
    if rc != 0:
        raise AmsError(rc, where)


def _p(t):
    """Raw pointer of a tensor (None -> NULL)."""
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _rows_at_least(n: int, **tensors):
    """Every named tensor must hold at least n rows (the capacity the call is told)."""
    for name, t in tensors.items():
        if t is not None and t.shape[0] < int(n):
            raise ValueError(f"{name} has {t.shape[0]} rows, fewer than the capacity {int(n)}")


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def make_mlp(dims, dtype: str = "f32", final_relu: bool = False) -> ams_mlp:
    """ams_mlp for layer widths `dims`; dtype "f32", "bf16" or "f32x3" (float32
    storage, the first layer's forward product on bf16 MFMA with an exact
    three-part split of each operand)."""
    m = ams_mlp()
    m.n_layers = len(dims) - 1
    for i, d in enumerate(dims):
        m.dims[i] = int(d)
    m.dtype = {"f32": AMS_F32, "bf16": AMS_BF16, "f32x3": AMS_F32_X3}[dtype]
    m.final_relu = int(final_relu)
    return m


# ------------------------------------------------------------- C calls

def ams_dedup_workspace(n_occ: int, n_ids: int) -> int:
    return load().ams_dedup_workspace(int(n_occ), int(n_ids))


def ams_dedup(ids, n_ids, uniq, inv, occ_perm, uniq_off, n_uniq, dev_status, ws, stream=None):
    _check(load().ams_dedup(_p(ids), ids.numel(), int(n_ids), _p(uniq), _p(inv), _p(occ_perm),
                            _p(uniq_off), _p(n_uniq), _p(dev_status), _p(ws),
                            ws.numel() * ws.element_size() if ws is not None else 0,
                            _stream(stream)), "ams_dedup")


def ams_dedup_noalloc(ids, n_ids, uniq, inv, occ_perm, uniq_off, n_uniq, dev_status, stream=None):
    """ams_dedup on the library's fixed per-device scratch (no workspace, no
    allocation); at most DEDUP_NOALLOC_MAX_OCC occurrences."""
    _check(load().ams_dedup_noalloc(_p(ids), ids.numel(), int(n_ids), _p(uniq), _p(inv), _p(occ_perm),
                                    _p(uniq_off), _p(n_uniq), _p(dev_status), _stream(stream)), "ams_dedup_noalloc")


def ams_embed_workspace(mlp: ams_mlp, n_uniq_cap: int) -> int:
    return load().ams_embed_workspace(ctypes.byref(mlp), int(n_uniq_cap))


def ams_embed_fwd(mlp, T, uniq, n_uniq, n_uniq_cap, W, b, H1_save, H2_save, E, ws, stream=None, slopes=None):
    """slopes: None (ReLU) or the PReLU slopes of every hidden layer."""
    W3 = W[2] if len(W) > 2 else None
    b3 = b[2] if len(b) > 2 else None
    _check(load().ams_embed_fwd(ctypes.byref(mlp), _p(T), T.shape[0], _p(uniq), _p(n_uniq),
                                int(n_uniq_cap), _p(W[0]), _p(b[0]), _p(W[1]), _p(b[1]), _p(W3), _p(b3),
                                _opt_parray(slopes), _p(H1_save), _p(H2_save), _p(E), _p(ws),
                                ws.numel() * ws.element_size() if ws is not None else 0,
                                _stream(stream)), "ams_embed_fwd")


def ams_embed_bwd(mlp, T, uniq, n_uniq, n_uniq_cap, W, H1_save, H2_save, E_fwd, dE, dW, db, ws,
                  stream=None, slopes=None, dslopes=None):
    """slopes as in ams_embed_fwd; dslopes: where the slope gradients go (None: not stored)."""
    W3 = W[2] if len(W) > 2 else None
    dW3 = dW[2] if len(dW) > 2 else None
    db3 = db[2] if len(db) > 2 else None
    _check(load().ams_embed_bwd(ctypes.byref(mlp), _p(T), T.shape[0], _p(uniq), _p(n_uniq),
                                int(n_uniq_cap), _p(W[0]), _p(W[1]), _p(W3), _opt_parray(slopes), _p(H1_save),
                                _p(H2_save), _p(E_fwd), _p(dE), _p(dW[0]), _p(db[0]), _p(dW[1]), _p(db[1]),
                                _p(dW3), _p(db3), _opt_parray(dslopes), _p(ws), ws.numel() * ws.element_size(),
                                _stream(stream)), "ams_embed_bwd")


def ams_pool_fwd(mode, seg_off, n_beh, inv, E, U, A, saved, stream=None):
    m = POOL[mode] if isinstance(mode, str) else int(mode)
    B = seg_off.numel() - 1
    _check(load().ams_pool_fwd(m, B, U.shape[1], _p(seg_off), int(n_beh), _p(inv), E.shape[0], _p(E), _p(U),
                               _p(A), _p(saved), _stream(stream)), "ams_pool_fwd")


def ams_pool_workspace(mode, B: int, n_beh: int, D: int, n_uniq_cap: int) -> int:
    m = POOL[mode] if isinstance(mode, str) else int(mode)
    return load().ams_pool_workspace(m, int(B), int(n_beh), int(D), int(n_uniq_cap))


def ams_pool_bwd(mode, seg_off, n_beh, inv, occ_perm, uniq_off, n_uniq, n_uniq_cap, E, U, A, saved,
                 dU, dA, dE, ws, stream=None):
    m = POOL[mode] if isinstance(mode, str) else int(mode)
    B = seg_off.numel() - 1
    _rows_at_least(n_uniq_cap, E=E, dE=dE)
    _check(load().ams_pool_bwd(m, B, U.shape[1], _p(seg_off), int(n_beh), _p(inv), _p(occ_perm),
                               _p(uniq_off), _p(n_uniq), int(n_uniq_cap), _p(E), _p(U), _p(A), _p(saved),
                               _p(dU), _p(dA), _p(dE), _p(ws),
                               ws.numel() * ws.element_size() if ws is not None else 0,
                               _stream(stream)), "ams_pool_bwd")


# ------------------------------------------------------- one whole step

def ams_timing_enable(on: bool):
    _check(load().ams_timing_enable(1 if on else 0), "ams_timing_enable")


def ams_timing_read(cap: int = 64) -> dict:
    """{kernel name: (launches, total ms)} recorded since the last read
    (waits for the recorded events; clears the record)."""
    buf = (ams_kernel_time * cap)()
    n = ctypes.c_int(0)
    _check(load().ams_timing_read(buf, cap, ctypes.byref(n)), "ams_timing_read")
    if n.value > cap:
        raise RuntimeError(f"ams_timing_read: {n.value} kernels recorded, buffer holds {cap}")
    return {buf[k].name.decode(): (int(buf[k].launches), float(buf[k].total_ms)) for k in range(n.value)}


def ams_pool_query_fwd(seg_off, n_beh: int, inv, E, Q, U, w, stream=None):
    B, D = Q.shape
    _check(load().ams_pool_query_fwd(B, D, _p(seg_off), int(n_beh), _p(inv), E.shape[0], _p(E), _p(Q), _p(U),
                                     _p(w), _stream(stream)), "ams_pool_query_fwd")


def ams_pool_query_bwd(seg_off, n_beh: int, inv, occ_perm, uniq_off, n_uniq, n_uniq_cap: int, E, Q, U, w, dU, dQ,
                       dE, accumulate: bool, ws, stream=None):
    B, D = Q.shape
    _rows_at_least(n_uniq_cap, E=E, dE=dE)
    _check(load().ams_pool_query_bwd(B, D, _p(seg_off), int(n_beh), _p(inv), _p(occ_perm), _p(uniq_off),
                                     _p(n_uniq), int(n_uniq_cap), _p(E), _p(Q), _p(U), _p(w), _p(dU), _p(dQ),
                                     _p(dE), int(bool(accumulate)), _p(ws), ws.numel() * ws.element_size(),
                                     _stream(stream)), "ams_pool_query_bwd")


def ams_adam_update(param, grad, m, v, lr: float, t: int, b1: float = 0.9, b2: float = 0.999, eps: float = 1e-8,
                    param_bf16=None, stream=None):
    _check(load().ams_adam_update(param.numel(), _p(param), _p(grad), _p(m), _p(v), float(lr), float(b1), float(b2),
                                  float(eps), int(t), _p(param_bf16), _stream(stream)), "ams_adam_update")


def ams_pool_concat_fwd(Lc: int, seg_off, n_beh: int, inv, E, U, A, stream=None):
    B, D = seg_off.numel() - 1, E.shape[1]
    _check(load().ams_pool_concat_fwd(B, D, int(Lc), _p(seg_off), int(n_beh), _p(inv), E.shape[0], _p(E), _p(U),
                                      _p(A), _stream(stream)), "ams_pool_concat_fwd")


def ams_pool_concat_bwd(Lc: int, seg_off, n_beh: int, inv, occ_perm, uniq_off, n_uniq, n_uniq_cap: int, dU, dA,
                        dE, ws, stream=None):
    B, D = seg_off.numel() - 1, dE.shape[1]
    _rows_at_least(n_uniq_cap, dE=dE)
    _check(load().ams_pool_concat_bwd(B, D, int(Lc), _p(seg_off), int(n_beh), _p(inv), _p(occ_perm), _p(uniq_off),
                                      _p(n_uniq), int(n_uniq_cap), _p(dU), _p(dA), _p(dE), _p(ws),
                                      ws.numel() * ws.element_size(), _stream(stream)), "ams_pool_concat_bwd")


def make_ctr(dims) -> ams_ctr:
    c = ams_ctr()
    c.n_layers = len(dims) - 1
    for i, d in enumerate(dims):
        c.dims[i] = int(d)
    return c


def _parray(ts):
    """Host array of device pointers (None -> NULL)."""
    return (ctypes.c_void_p * len(ts))(*[t.data_ptr() if t is not None else None for t in ts])


def ams_bag_fwd(seg_off, n_beh: int, ids, table, bag, stream=None):
    B, D = bag.shape
    _check(load().ams_bag_fwd(B, D, _p(seg_off), int(n_beh), _p(ids), _p(table), table.shape[0], _p(bag),
                              _stream(stream)), "ams_bag_fwd")


def ams_bag_workspace(B: int, n_beh: int, D: int, n_uniq_cap: int) -> int:
    return load().ams_bag_workspace(int(B), int(n_beh), int(D), int(n_uniq_cap))


def ams_bag_bwd(seg_off, n_beh: int, inv, occ_perm, uniq_off, n_uniq, n_uniq_cap: int, dbag, grad, ws,
                stream=None, dad=None):
    """dad: None, or a second gradient [B x D] of each sample's ad row."""
    B, D = dbag.shape
    _rows_at_least(n_uniq_cap, grad=grad)
    if dad is not None and tuple(dad.shape) != (B, D):
        raise ValueError("dad must be [B x D] like dbag")
    _check(load().ams_bag_bwd(B, D, _p(seg_off), int(n_beh), _p(inv), _p(occ_perm), _p(uniq_off), _p(n_uniq),
                              int(n_uniq_cap), _p(dbag), _p(dad), _p(grad), _p(ws),
                              ws.numel() * ws.element_size(), _stream(stream)), "ams_bag_bwd")


def ams_ctr_workspace(net: ams_ctr, B: int) -> int:
    return load().ams_ctr_workspace(ctypes.byref(net), int(B))


def _opt_parray(ts):
    return _parray(ts) if ts is not None else None


def _widths(fields):
    return (ctypes.c_int32 * len(fields))(*[int(f.shape[1]) for f in fields])


def ams_ctr_fwd_bwd(net: ams_ctr, fields, labels, W, b, loss, prob, dW, db, dfields, ws, stream=None, slopes=None,
                    dslopes=None):
    """slopes: PReLU slopes of the hidden layers (None, or None entries: ReLU);
    dslopes: where their gradients go (None: not stored)."""
    B = fields[0].shape[0]
    _check(load().ams_ctr_fwd_bwd(ctypes.byref(net), B, len(fields), _parray(fields), _widths(fields), _p(labels),
                                  _parray(W), _parray(b), _opt_parray(slopes), _p(loss), _p(prob), _parray(dW),
                                  _parray(db), _opt_parray(dslopes), _opt_parray(dfields), _p(ws),
                                  ws.numel() * ws.element_size(), _stream(stream)), "ams_ctr_fwd_bwd")


def ams_dssm_workspace(user_net: ams_ctr, ad_net: ams_ctr, B: int) -> int:
    return load().ams_dssm_workspace(ctypes.byref(user_net), ctypes.byref(ad_net), int(B))


def ams_dssm_fwd_bwd(user_net: ams_ctr, ad_net: ams_ctr, user_fields, ad_fields, labels, user, ad, loss, prob,
                     duser, dad, duser_fields, dad_fields, ws, stream=None):
    """user / ad: (W, b, slopes) of each tower; duser / dad: (dW, db, dslopes)."""
    B = user_fields[0].shape[0]
    _check(load().ams_dssm_fwd_bwd(ctypes.byref(user_net), ctypes.byref(ad_net), B, len(user_fields),
                                   _parray(user_fields), _widths(user_fields), len(ad_fields), _parray(ad_fields),
                                   _widths(ad_fields), _p(labels), _parray(user[0]), _parray(user[1]),
                                   _opt_parray(user[2]), _parray(ad[0]), _parray(ad[1]), _opt_parray(ad[2]),
                                   _p(loss), _p(prob), _parray(duser[0]), _parray(duser[1]), _opt_parray(duser[2]),
                                   _parray(dad[0]), _parray(dad[1]), _opt_parray(dad[2]),
                                   _opt_parray(duser_fields), _opt_parray(dad_fields), _p(ws),
                                   ws.numel() * ws.element_size(), _stream(stream)), "ams_dssm_fwd_bwd")


def ams_adagrad_rows(uniq, n_uniq, n_uniq_cap: int, grad, table, accum, lr: float, eps: float, stream=None):
    _check(load().ams_adagrad_rows(table.shape[1], _p(uniq), _p(n_uniq), int(n_uniq_cap), _p(grad), _p(table),
                                   table.shape[0], _p(accum), float(lr), float(eps), _stream(stream)),
           "ams_adagrad_rows")


# ---------------------------------------------------------------- probes

def ams_peak_copy(src, dst, blocks: int, stream=None):
    _check(load().ams_peak_copy(_p(src), _p(dst), src.numel() * src.element_size(), int(blocks), _stream(stream)),
           "ams_peak_copy")


def ams_peak_read(src, blocks: int, out, stream=None):
    _check(load().ams_peak_read(_p(src), src.numel() * src.element_size(), int(blocks), _p(out), _stream(stream)),
           "ams_peak_read")


def ams_peak_gather(T, rows, pattern: int, blocks: int, out, W=None, stream=None):
    """Gather probe over T's rows (8192 bytes each); pattern 0-4 as in ams.h
    (4 also streams slices of W, 2 MB)."""
    _check(load().ams_peak_gather(_p(T), T.shape[0], T.shape[1] * T.element_size(), _p(rows), rows.numel(),
                                  int(pattern), _p(W) if W is not None else None, int(blocks), _p(out),
                                  _stream(stream)), "ams_peak_gather")


def ams_peak_mfma(dtype: str, ops, iters: int, blocks: int, out, stream=None):
    if ops.numel() * ops.element_size() < 524288:
        raise ValueError("ams_peak_mfma reads 524288 bytes of operands")
    _check(load().ams_peak_mfma({"f32": AMS_F32, "bf16": AMS_BF16}[dtype], _p(ops), int(iters), int(blocks), _p(out),
                                _stream(stream)), "ams_peak_mfma")


class Step:
    """Buffers for one training step of the embedding hot path, and the five
    calls in order on one stream: dedup -> embed fwd -> pool fwd -> pool bwd
    -> embed bwd.  Inputs (table, weights, batch) stay caller-owned tensors.

    Buffers are sized for up to B samples and n_beh_max behaviors; `cap`
    (default B + n_beh_max) bounds the unique count used for grids, since n_u
    is only known on the device.  A cap below B + n_beh_max saves memory but
    can be exceeded by a batch with more distinct images: the kernels then
    stay inside the buffers and the results are unspecified, so such a Step
    is only built with ``cap_checked=True``, by a caller that checks
    `capacity_ok()` after its steps.  With `prelu` the hidden layers use
    PReLU (float32 models, and bf16 ones whose first hidden layer is 256
    wide): the slopes are passed to run / embed_fwd / embed_bwd and their
    gradients land in `dslope`.
    """

    def __init__(self, dims, dtype: str, mode: str, B: int, n_beh_max: int, final_relu: bool = False,
                 device="cuda", cap: int | None = None, prelu: bool = False, cap_checked: bool = False):
        self.mlp = make_mlp(dims, dtype, final_relu)
        self.dims = tuple(dims)
        self.dtype = dtype
        self.mode = mode
        self.B, self.n_beh = int(B), int(n_beh_max)
        self.n_occ = self.n_beh + self.B
        self.cap = self.n_occ if cap is None else int(cap)
        if self.cap < 0 or (self.cap < self.n_occ and not cap_checked):
            raise ValueError(f"cap {self.cap} is below the {self.n_occ} occurrences a batch may hold: "
                             "pass cap_checked=True and check capacity_ok() after the step")
        D, H = dims[-1], dims[1]
        dev = torch.device(device)
        i32, f32 = torch.int32, torch.float32
        n = max(self.n_occ, 1)
        self.uniq = torch.empty(n, dtype=i32, device=dev)
        self.inv = torch.empty(n, dtype=i32, device=dev)
        self.occ_perm = torch.empty(n, dtype=i32, device=dev)
        self.uniq_off = torch.empty(n + 1, dtype=i32, device=dev)
        self.n_uniq = torch.zeros(1, dtype=i32, device=dev)
        self.dev_status = torch.zeros(1, dtype=i32, device=dev)
        cap1 = max(self.cap, 1)
        h1_dtype = torch.bfloat16 if dtype == "bf16" else f32
        self.H1 = torch.empty((cap1, H), dtype=h1_dtype, device=dev)
        self.H2 = torch.empty((cap1, dims[2]), dtype=f32, device=dev) if len(dims) == 4 else None
        self.E = torch.empty((cap1, D), dtype=f32, device=dev)
        self.U = torch.empty((max(self.B, 1), D), dtype=f32, device=dev)
        self.A = torch.empty((max(self.B, 1), D), dtype=f32, device=dev)
        if mode == "max":
            self.saved = torch.empty((max(self.B, 1), D), dtype=i32, device=dev)
        elif mode == "att":
            self.saved = torch.empty(max(self.n_beh, 1), dtype=f32, device=dev)
        else:
            self.saved = None
        self.dE = torch.empty((cap1, D), dtype=f32, device=dev)
        self.dW = [torch.empty((o, i), dtype=f32, device=dev) for i, o in zip(dims[:-1], dims[1:])]
        self.db = [torch.empty((o,), dtype=f32, device=dev) for o in dims[1:]]
        self.dslope = [torch.empty((o,), dtype=f32, device=dev) for o in dims[1:-1]] if prelu else None
        self.ws = None
        self.n_ids = None

    def capacity_ok(self) -> bool:
        """True when the last dedup's unique count fits the cap (synchronises)."""
        return int(self.n_uniq.item()) <= self.cap

    def alloc_workspace(self, n_ids: int):
        """One workspace shared by the five calls (they run in order on one stream)."""
        need = max(ams_dedup_workspace(self.n_occ, n_ids),
                   ams_embed_workspace(self.mlp, self.cap),
                   ams_pool_workspace(self.mode, self.B, self.n_beh, self.dims[-1], self.cap), 256)
        if self.ws is None or self.ws.numel() < need:
            self.ws = torch.empty(need, dtype=torch.uint8, device=self.uniq.device)
        self.n_ids = int(n_ids)

    def dedup(self, ids, n_ids, stream=None):
        if self.ws is None or self.n_ids != int(n_ids):
            self.alloc_workspace(n_ids)
        ams_dedup(ids, n_ids, self.uniq, self.inv, self.occ_perm, self.uniq_off, self.n_uniq,
                  self.dev_status, self.ws, stream)

    def embed_fwd(self, T, W, b, stream=None, slopes=None):
        ams_embed_fwd(self.mlp, T, self.uniq, self.n_uniq, self.cap, W, b, self.H1, self.H2, self.E,
                      self.ws, stream, slopes=slopes)

    def pool_fwd(self, seg_off, n_beh, stream=None):
        ams_pool_fwd(self.mode, seg_off, n_beh, self.inv, self.E, self.U, self.A, self.saved, stream)

    def pool_bwd(self, seg_off, n_beh, dU, dA, stream=None):
        ams_pool_bwd(self.mode, seg_off, n_beh, self.inv, self.occ_perm, self.uniq_off, self.n_uniq,
                     self.cap, self.E, self.U, self.A, self.saved, dU, dA, self.dE, self.ws, stream)

    def embed_bwd(self, T, W, stream=None, slopes=None):
        ams_embed_bwd(self.mlp, T, self.uniq, self.n_uniq, self.cap, W, self.H1, self.H2, self.E,
                      self.dE, self.dW, self.db, self.ws, stream, slopes=slopes,
                      dslopes=self.dslope if slopes is not None else None)

    def run(self, ids, n_ids, T, W, b, seg_off, dU, dA, stream=None, slopes=None):
        """The whole step, enqueued on one stream with no host synchronisation."""
        n_beh = ids.numel() - (seg_off.numel() - 1)
        if n_beh > self.n_beh or seg_off.numel() - 1 > self.B:
            raise ValueError("batch larger than the buffers of this Step")
        if slopes is not None and self.dslope is None:
            raise ValueError("this Step was built without prelu=True")
        self.dedup(ids, n_ids, stream)
        self.embed_fwd(T, W, b, stream, slopes=slopes)
        self.pool_fwd(seg_off, n_beh, stream)
        self.pool_bwd(seg_off, n_beh, dU, dA, stream)
        self.embed_bwd(T, W, stream, slopes=slopes)


class StepPipeline:
    """Steps of a Step over a sequence of batches, with the dedup of batch
    k + 1 on a second stream (default priority) beside batch k's pooling and
    backward.  Two sets of dedup outputs are used alternately, each with its
    own dedup workspace; events order every use: dedup k + 1 starts after
    batch k's forward has been enqueued and after batch k - 1 (the last user
    of its set) has finished, and batch k + 1 waits for it.  Each batch still
    runs the whole path; only the dedup leaves the critical path.
    """

    _SET = ("uniq", "inv", "occ_perm", "uniq_off", "n_uniq", "dev_status")

    def __init__(self, step: Step, n_ids: int):
        self.st = step
        self.n_ids = int(n_ids)
        step.alloc_workspace(n_ids)
        dev = step.uniq.device
        self.side = torch.cuda.Stream(device=dev)
        other = {k: torch.empty_like(getattr(step, k)) for k in self._SET}
        self.sets = [{k: getattr(step, k) for k in self._SET}, other]
        need = max(ams_dedup_workspace(step.n_occ, self.n_ids), 256)
        self.dd_ws = [torch.empty(need, dtype=torch.uint8, device=dev) for _ in range(2)]
        self.ev_dd = [torch.cuda.Event() for _ in range(2)]
        self.ev_done = [torch.cuda.Event() for _ in range(2)]
        self.ev_fwd = torch.cuda.Event()

    def _dedup(self, b, s, stream):
        b["ids"].record_stream(stream)
        d = self.sets[s]
        ams_dedup(b["ids"], self.n_ids, d["uniq"], d["inv"], d["occ_perm"], d["uniq_off"], d["n_uniq"],
                  d["dev_status"], self.dd_ws[s], stream)

    def run(self, batches, T, W, b, slopes=None):
        """batches: dicts with ids, seg_off, dU, dA, n_beh (device tensors and
        an int).  Enqueues everything; returns the dedup set index of the last
        batch (whose outputs the Step's attributes then point at)."""
        st, main = self.st, torch.cuda.current_stream()
        n = len(batches)
        if n == 0:
            return None
        self.side.wait_stream(main)               # inputs and earlier users of both sets
        self._dedup(batches[0], 0, self.side)
        self.ev_dd[0].record(self.side)
        for k, bt in enumerate(batches):
            s = k % 2
            for key in self._SET:
                setattr(st, key, self.sets[s][key])
            main.wait_event(self.ev_dd[s])
            st.embed_fwd(T, W, b, main, slopes=slopes)
            if k + 1 < n:
                self.ev_fwd.record(main)
                self.side.wait_event(self.ev_fwd)
                if k >= 1:
                    self.side.wait_event(self.ev_done[(k + 1) % 2])   # batch k - 1 is done with that set
                self._dedup(batches[k + 1], (k + 1) % 2, self.side)
                self.ev_dd[(k + 1) % 2].record(self.side)
            st.pool_fwd(bt["seg_off"], bt["n_beh"], main)
            st.pool_bwd(bt["seg_off"], bt["n_beh"], bt["dU"], bt["dA"], main)
            st.embed_bwd(T, W, main, slopes=slopes)
            self.ev_done[s].record(main)
        main.wait_stream(self.side)
        return (n - 1) % 2


class JointStep:
    """Buffers and calls of one joint training step (Algorithm 1: worker
    iteration with the server's embed and update):

      image dedup                     ams_dedup
      image embed + pool forward      ams_embed_fwd, ams_pool_fwd
      ID dedups, ID bags              ams_dedup, ams_bag_fwd x tables       (side stream)
      CTR forward + backward          ams_ctr_fwd_bwd (fields: U, A, bags)
      image pool + embed backward     ams_pool_bwd(dU, dA), ams_embed_bwd
      ID rows: merged grad, Adagrad   ams_bag_bwd, ams_adagrad_rows x tables (side stream)

    With ``query_table`` t_q (MultiQueryAttentivePooling, section 5.2) the
    image embeddings are pooled by a second attentive channel whose query is
    each sample's ad row of ID table t_q (gathered by ams_bag_fwd over the ad
    IDs alone): ams_pool_query_fwd gives U2, the CTR fields are
    [U, U2, A, bags...], ams_pool_query_bwd adds that channel's dE to the image
    channel's and yields dQ, which table t_q's ams_bag_bwd adds to the ad
    occurrences' row gradients before its Adagrad step.

    With ``overlap`` (the default) each ID table's work runs on a stream of
    its own (default priority), forked from the caller's stream at the start
    and joined before the CTR call and at the end, so the tables' dedups, bags
    and row updates (latency-bound kernels) overlap one another and the image
    path's own small kernels; each stream has its own workspace.  Without it,
    every call is on the caller's stream in the order above.  The ID tables and their Adagrad
    accumulators are caller tensors updated in place; everything else is held
    here.
    """

    def __init__(self, dims, dtype: str, mode: str, B: int, n_beh_max: int, id_rows, id_dim: int, ctr_dims,
                 device="cuda", overlap: bool = True, query_table: int | None = None):
        if query_table is not None:
            if mode != "att":
                raise ValueError("the query channel pairs with attentive pooling of the image channel")
            if not 0 <= int(query_table) < len(id_rows) or int(id_dim) != dims[-1]:
                raise ValueError("query_table must name an ID table whose rows are as wide as the embeddings")
        self.query_table = None if query_table is None else int(query_table)
        self.img = Step(dims, dtype, mode, B, n_beh_max, device=device)
        self.B, self.n_beh = int(B), int(n_beh_max)
        self.n_occ = self.B + self.n_beh
        self.id_rows = [int(x) for x in id_rows]
        self.id_dim = int(id_dim)
        self.ctr = make_ctr(ctr_dims)
        self.ctr_dims = tuple(ctr_dims)
        dev = torch.device(device)
        i32, f32 = torch.int32, torch.float32
        n = max(self.n_occ, 1)
        T = len(self.id_rows)
        self.t_uniq = [torch.empty(n, dtype=i32, device=dev) for _ in range(T)]
        self.t_inv = [torch.empty(n, dtype=i32, device=dev) for _ in range(T)]
        self.t_perm = [torch.empty(n, dtype=i32, device=dev) for _ in range(T)]
        self.t_off = [torch.empty(n + 1, dtype=i32, device=dev) for _ in range(T)]
        self.t_nu = [torch.zeros(1, dtype=i32, device=dev) for _ in range(T)]
        self.t_status = [torch.zeros(1, dtype=i32, device=dev) for _ in range(T)]
        Bm = max(self.B, 1)
        self.bags = [torch.empty((Bm, self.id_dim), dtype=f32, device=dev) for _ in range(T)]
        self.dbags = [torch.empty((Bm, self.id_dim), dtype=f32, device=dev) for _ in range(T)]
        self.row_grad = [torch.empty((n, self.id_dim), dtype=f32, device=dev) for _ in range(T)]
        D = dims[-1]
        self.dU = torch.empty((Bm, D), dtype=f32, device=dev)
        self.dA = torch.empty((Bm, D), dtype=f32, device=dev)
        self.loss = torch.zeros(1, dtype=f32, device=dev)
        self.prob = torch.empty((Bm, self.ctr_dims[-1]), dtype=f32, device=dev)
        self.ctr_dW = [torch.empty((o, i), dtype=f32, device=dev) for i, o in zip(ctr_dims[:-1], ctr_dims[1:])]
        self.ctr_db = [torch.empty((o,), dtype=f32, device=dev) for o in ctr_dims[1:]]
        if self.query_table is not None:
            self.Q = torch.empty((Bm, D), dtype=f32, device=dev)
            self.U2 = torch.empty((Bm, D), dtype=f32, device=dev)
            self.w2 = torch.empty((max(self.n_beh, 1),), dtype=f32, device=dev)
            self.dU2 = torch.empty((Bm, D), dtype=f32, device=dev)
            self.dQ = torch.empty((Bm, D), dtype=f32, device=dev)
            self.no_beh = torch.zeros(Bm + 1, dtype=i32, device=dev)      # offsets of bags holding the ad alone
        self.ws = None
        self.ws_id = None
        self.sides = [torch.cuda.Stream(device=dev) for _ in range(T)] if overlap else None

    def alloc_workspace(self, n_ids: int):
        id_need = max(ams_dedup_workspace(self.n_occ, max(self.id_rows)),
                      ams_bag_workspace(self.B, self.n_beh, self.id_dim, self.n_occ), 256)
        img_need = max(ams_dedup_workspace(self.n_occ, n_ids), ams_embed_workspace(self.img.mlp, self.img.cap),
                       ams_pool_workspace(self.img.mode, self.B, self.n_beh, self.img.dims[-1], self.img.cap),
                       ams_ctr_workspace(self.ctr, max(self.B, 1)), 256)
        if self.sides is None:
            img_need = max(img_need, id_need)
        self.img.ws = torch.empty(img_need, dtype=torch.uint8, device=self.loss.device)
        self.img.n_ids = int(n_ids)
        self.ws = self.img.ws
        self.ws_id = ([torch.empty(id_need, dtype=torch.uint8, device=self.loss.device) for _ in self.sides]
                      if self.sides is not None else [self.ws] * len(self.id_rows))

    def run(self, ids, n_ids, T, W, b, seg_off, id_ids, id_tables, accum, labels, ctr_W, ctr_b, lr: float,
            eps: float, stream=None):
        """The whole joint step, enqueued with no host synchronisation.
        id_ids[t]: behavior then ad IDs of table t; id_tables[t] and accum[t]
        are updated in place on the touched rows."""
        n_beh = ids.numel() - (seg_off.numel() - 1)
        if n_beh > self.n_beh or seg_off.numel() - 1 > self.B:
            raise ValueError("batch larger than the buffers of this JointStep")
        if self.ws is None or self.img.n_ids != int(n_ids):
            self.alloc_workspace(n_ids)
        st = self.img
        main = stream if stream is not None else torch.cuda.current_stream()
        nt = len(self.id_rows)
        sides = self.sides if self.sides is not None else [main] * nt
        forked = self.sides is not None
        B = seg_off.numel() - 1
        if forked:
            for t, sd in enumerate(sides):
                sd.wait_stream(main)                # the caller's inputs are ready
                for x in (seg_off, labels, id_ids[t], id_tables[t], accum[t]):
                    x.record_stream(sd)
        tq = self.query_table
        # ID tables, beside the image forward: dedup (needed from bag_bwd on) and
        # bags; with a query table also each sample's ad row of it (a bag of the
        # ad alone).  (Issuing the bags first and letting the CTR call wait for
        # them alone moves the dedups into the image backward, where they meet
        # the dW1 product that fills every CU: slower.)
        for t in range(nt):
            ams_dedup(id_ids[t], self.id_rows[t], self.t_uniq[t], self.t_inv[t], self.t_perm[t], self.t_off[t],
                      self.t_nu[t], self.t_status[t], self.ws_id[t], sides[t])
            ams_bag_fwd(seg_off, n_beh, id_ids[t], id_tables[t], self.bags[t], sides[t])
            if t == tq:
                ams_bag_fwd(self.no_beh[:B + 1], 0, id_ids[t][n_beh:], id_tables[t], self.Q[:B], sides[t])
        st.dedup(ids, n_ids, main)
        st.embed_fwd(T, W, b, main)
        st.pool_fwd(seg_off, n_beh, main)
        if forked:
            for sd in sides:
                main.wait_stream(sd)                # bags (and the queries) ready
        users, dusers = [st.U[:B]], [self.dU[:B]]
        if tq is not None:
            ams_pool_query_fwd(seg_off, n_beh, st.inv, st.E, self.Q[:B], self.U2[:B], self.w2, main)
            users.append(self.U2[:B])
            dusers.append(self.dU2[:B])
        fields = users + [st.A[:B]] + [x[:B] for x in self.bags]
        dfields = dusers + [self.dA[:B]] + [x[:B] for x in self.dbags]
        ams_ctr_fwd_bwd(self.ctr, fields, labels, ctr_W, ctr_b, self.loss, self.prob, self.ctr_dW, self.ctr_db,
                        dfields, self.ws, main)
        if forked:
            for sd in sides:
                sd.wait_stream(main)                # bag gradients ready
        # ID rows: merged gradients and Adagrad, beside the image backward (the
        # query table after the query channel's backward has produced dQ)
        def id_update(t, dad=None):
            ams_bag_bwd(seg_off, n_beh, self.t_inv[t], self.t_perm[t], self.t_off[t], self.t_nu[t], self.n_occ,
                        self.dbags[t][:B], self.row_grad[t], self.ws_id[t], sides[t], dad=dad)
            ams_adagrad_rows(self.t_uniq[t], self.t_nu[t], self.n_occ, self.row_grad[t], id_tables[t], accum[t],
                             lr, eps, sides[t])
        for t in range(nt):
            if t != tq:
                id_update(t)
        st.pool_bwd(seg_off, n_beh, self.dU, self.dA, main)
        if tq is not None:
            ams_pool_query_bwd(seg_off, n_beh, st.inv, st.occ_perm, st.uniq_off, st.n_uniq, st.cap, st.E,
                               self.Q[:B], self.U2[:B], self.w2, self.dU2[:B], self.dQ[:B], st.dE, True, st.ws, main)
            if forked:
                sides[tq].wait_stream(main)         # dQ ready
            id_update(tq, self.dQ[:B])
        st.embed_bwd(T, W, main)
        if forked:
            for sd in sides:
                main.wait_stream(sd)                # the whole step is ordered before later work on main
