"""Thin ctypes binding of libflashloop.so (argument marshalling only).

Every function takes torch tensors that live on the ROCm device, checks dtype/shape/contiguity,
allocates outputs with torch, and passes raw device pointers plus the current HIP stream to the C ABI
declared in include/flashloop.h.  All arithmetic happens in the library's HIP kernels; if the library
is missing this module raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libflashloop.so")

AXIS_TOKEN = 0
AXIS_CHANNEL = 1
DQ_COMPACT = 0
DQ_COMMIT = 1
ATTN_DENSE = 1
PASS_ADD, PASS_SUBTRACT, PASS_BOTH = 0, 1, 2

_c_p = ctypes.c_void_p
_c_i = ctypes.c_int
_c_d = ctypes.c_double
_c_f = ctypes.c_float
_c_sz = ctypes.c_size_t

_SIGNATURES = {
    "fl_status_str": (ctypes.c_char_p, [_c_i]),
    "fl_last_error": (ctypes.c_char_p, []),
    "fl_abi_version": (_c_i, []),
    "fl_set_index_checks": (None, [_c_i]),
    "fl_select_tokens": (_c_i, [_c_p, _c_p, _c_p, _c_p, _c_i, _c_i, _c_i, _c_p, _c_i, _c_i, _c_i, _c_d,
                                _c_p, _c_p, _c_p, _c_p]),
    "fl_kv_residual_quant": (_c_i, [_c_p, _c_p, _c_p, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i,
                                    _c_p, _c_p, _c_p, _c_p, _c_p]),
    "fl_kv_residual_quant_commit": (_c_i, [_c_p, _c_p, _c_p, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i,
                                           _c_p, _c_p, _c_p, _c_p]),
    "fl_kv_residual_dequant": (_c_i, [_c_p, _c_p, _c_p, _c_p, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i,
                                      _c_i, _c_i, _c_p, _c_p, _c_p]),
    "fl_kv_residual_dequant_kv": (_c_i, [_c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i, _c_i, _c_i, _c_i, _c_i,
                                         _c_i, _c_i, _c_i, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "fl_kv_residual_quant_kv": (_c_i, [_c_p, _c_p, _c_p, _c_p, _c_p, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i,
                                       _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i, _c_p]),
    "fl_kv_residual_quant_kv_v16": (_c_i, [_c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i,
                                           _c_i, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p]),
    "fl_kv_f16_rows": (_c_i, [_c_p, _c_p, _c_i, _c_i, _c_i, _c_i, _c_i, _c_p, _c_p]),
    "fl_loop_sparse_attn_ws": (_c_sz, [_c_i, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i]),
    "fl_loop_sparse_attn": (_c_i, [_c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i, _c_p, _c_i, _c_i,
                                   _c_i, _c_i, _c_i, _c_i, _c_f, _c_i, _c_p, _c_p, _c_p, _c_sz, _c_p]),
    "fl_loop_sparse_attn_terms": (_c_i, [_c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i, _c_p, _c_i, _c_i,
                                         _c_i, _c_i, _c_i, _c_i, _c_f, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i, _c_p,
                                         _c_p, _c_p, _c_sz, _c_p]),
    "fl_loop_subtract_terms_supported": (_c_i, [_c_i, _c_i, _c_i, _c_i, _c_i]),
    "fl_attn_kernel_name": (ctypes.c_char_p, [_c_i, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i]),
    "fl_loop_subtract_terms": (_c_i, [_c_p, _c_p, _c_p, _c_p, _c_i, _c_p, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i, _c_f,
                                      _c_p, _c_p, _c_p, _c_p]),
    "fl_loop_sparse_attn_terms_v16": (_c_i, [_c_p, _c_p, _c_p, _c_p, _c_p, _c_i, _c_p, _c_i, _c_i, _c_i, _c_i,
                                             _c_i, _c_i, _c_f, _c_p, _c_p, _c_p, _c_p, _c_p, _c_i, _c_p, _c_p,
                                             _c_p]),
    "fl_loop_subtract_terms_v16": (_c_i, [_c_p, _c_p, _c_p, _c_p, _c_p, _c_i, _c_p, _c_i, _c_i, _c_i, _c_i, _c_i,
                                          _c_i, _c_f, _c_p, _c_p, _c_p, _c_p]),
    "fl_column_scores_ws": (_c_sz, [_c_i, _c_i, _c_i]),
    "fl_column_scores": (_c_i, [_c_p, _c_p, _c_i, _c_i, _c_i, _c_i, _c_p, _c_p, _c_sz, _c_p]),
    "fl_select_columns": (_c_i, [_c_p, _c_i, _c_i, _c_i, _c_i, _c_i, _c_p, _c_p]),
    "fl_decode_step_ws": (_c_sz, [_c_i, _c_i, _c_i, _c_i, _c_i, _c_i]),
    "fl_decode_step": (_c_i, [_c_p, _c_p, _c_p, _c_p, _c_i, _c_p, _c_p, _c_i, _c_i, _c_i, _c_i, _c_f, _c_p, _c_p,
                              _c_i, _c_i, _c_i, _c_p, _c_p, _c_p, _c_p, _c_sz, _c_p]),
    "fl_decode_step_noalloc": (_c_i, [_c_p, _c_p, _c_p, _c_p, _c_i, _c_p, _c_p, _c_i, _c_i, _c_i, _c_i, _c_f, _c_p,
                                      _c_p, _c_i, _c_i, _c_i, _c_p, _c_p, _c_p, _c_p]),
    "fl_prune_columns_ws": (_c_sz, [_c_i, _c_i, _c_i, _c_i, _c_i]),
    "fl_kv_keep_recent": (_c_i, [_c_p, _c_p, _c_i, _c_i, _c_i, _c_i, _c_i, _c_i, _c_p, _c_p, _c_p]),
    "fl_prune_columns": (_c_i, [_c_p, _c_p, _c_p, _c_i, _c_p, _c_i, _c_p, _c_i, _c_i, _c_i, _c_i, _c_d, _c_i, _c_i,
                                _c_p, _c_p, _c_p, _c_sz, _c_p]),
}

EXPORTS = tuple(_SIGNATURES)

_lib = None


class FlashLoopError(RuntimeError):
    pass


def load(path: str = LIB_PATH):
    """Load the HIP library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FlashLoopError(f"{path} is missing: build it with `python -m paper_2609_29812_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def set_index_checks(on: bool):
    """Turn the library's index-list checks on or off (every call then validates its lists on the host)."""
    load().fl_set_index_checks(1 if on else 0)


def _check(rc: int, fn: str):
    if rc != 0:
        lib = load()
        raise FlashLoopError(f"{fn}: {lib.fl_status_str(rc).decode()}: {lib.fl_last_error().decode()}")


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev(t, dtype, name, shape=None):
    if t is None:
        return
    if not t.is_cuda:
        raise FlashLoopError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise FlashLoopError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise FlashLoopError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise FlashLoopError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


# ---- (1) token selection ----------------------------------------------------------------------------
def select_tokens(k_cur, k_prev, v_cur, v_prev, k, cand=None, normalize=True, eps=1e-6, slot=True,
                  out_key=None, out_idx=None, out_slot=None):
    """Active rows of the loop: returns (idx int32 [B, k], slot int32 [B, N] or None, key fp32 [B, n])."""
    B, N = k_cur.shape[:2]
    D = k_cur.numel() // (B * N)
    for name, t in (("k_cur", k_cur), ("k_prev", k_prev), ("v_cur", v_cur), ("v_prev", v_prev)):
        _dev(t, torch.bfloat16, name, None if t is None else k_cur.shape)
    n_cand = N if cand is None else cand.shape[1]
    _dev(cand, torch.int32, "cand", None if cand is None else (B, n_cand))
    dev = k_cur.device
    out_key = torch.empty(B, n_cand, dtype=torch.float32, device=dev) if out_key is None else out_key
    out_idx = torch.empty(B, k, dtype=torch.int32, device=dev) if out_idx is None else out_idx
    if slot and out_slot is None:
        out_slot = torch.empty(B, N, dtype=torch.int32, device=dev)
    rc = load().fl_select_tokens(_p(k_cur), _p(k_prev), _p(v_cur), _p(v_prev), B, N, D, _p(cand), n_cand,
                                 k, 1 if normalize else 0, eps, _p(out_key), _p(out_idx),
                                 _p(out_slot) if slot else None, _stream())
    _check(rc, "fl_select_tokens")
    return out_idx, (out_slot if slot else None), out_key


# ---- (2) residual codec -----------------------------------------------------------------------------
def meta_shape(B, k, H, d, group, axis):
    return (B, -(-k // group), H, d) if axis == AXIS_TOKEN else (B, k, H, d // group)


def kv_residual_quant(x_cur, x_ref, idx, bits, group, axis, rows=True, out=None):
    """Quantize the residual of rows idx (None = all rows).  Returns (codes, scale, zero, rows)."""
    B, N, H, d = x_cur.shape
    _dev(x_cur, torch.bfloat16, "x_cur")
    _dev(x_ref, torch.bfloat16, "x_ref", x_cur.shape)
    k = N if idx is None else idx.shape[1]
    _dev(idx, torch.int32, "idx", None if idx is None else (B, k))
    dev = x_cur.device
    o = out or {}
    codes = o.get("codes")
    if codes is None:
        codes = torch.empty(B, k, H, d * bits // 8, dtype=torch.uint8, device=dev)
    scale = zero = None
    if bits != 16:
        shp = meta_shape(B, k, H, d, group, axis)
        scale = o.get("scale") if o.get("scale") is not None else torch.empty(shp, dtype=torch.float16, device=dev)
        zero = o.get("zero") if o.get("zero") is not None else torch.empty(shp, dtype=torch.float16, device=dev)
    out_rows = None
    if rows is True:
        out_rows = torch.empty(B, k, H, d, dtype=torch.bfloat16, device=dev)
    elif rows is not None and rows is not False:
        out_rows = rows
    rc = load().fl_kv_residual_quant(_p(x_cur), _p(x_ref), _p(idx), k, B, N, H, d, bits, group, axis,
                                     _p(codes), _p(scale), _p(zero), _p(out_rows), _stream())
    _check(rc, "fl_kv_residual_quant")
    return codes, scale, zero, out_rows


def kv_residual_quant_commit(x_cur, x_hat, idx, bits, group, axis, out=None):
    """Quantize the residual of rows idx against x_hat and commit the reconstruction into x_hat in place.
    Returns (codes, scale, zero)."""
    B, N, H, d = x_cur.shape
    _dev(x_cur, torch.bfloat16, "x_cur")
    _dev(x_hat, torch.bfloat16, "x_hat", x_cur.shape)
    k = N if idx is None else idx.shape[1]
    _dev(idx, torch.int32, "idx", None if idx is None else (B, k))
    dev = x_cur.device
    o = out or {}
    codes = o.get("codes")
    if codes is None:
        codes = torch.empty(B, k, H, d * bits // 8, dtype=torch.uint8, device=dev)
    scale = zero = None
    if bits != 16:
        shp = meta_shape(B, k, H, d, group, axis)
        scale = o.get("scale") if o.get("scale") is not None else torch.empty(shp, dtype=torch.float16, device=dev)
        zero = o.get("zero") if o.get("zero") is not None else torch.empty(shp, dtype=torch.float16, device=dev)
    rc = load().fl_kv_residual_quant_commit(_p(x_cur), _p(x_hat), _p(idx), k, B, N, H, d, bits, group, axis,
                                            _p(codes), _p(scale), _p(zero), _stream())
    _check(rc, "fl_kv_residual_quant_commit")
    return codes, scale, zero


def kv_residual_quant_kv(k_cur, k_ref, v_cur, v_ref, idx, bits, group, mode=DQ_COMPACT, rows=True, v_f16=None):
    """Keys (token axis) and values (channel axis) in one call.  COMPACT: returns
    ((codes, scale, zero, rows) for keys, the same for values), rows None unless rows=True;
    COMMIT: rows idx of k_ref / v_ref are updated in place and the rows entries are None; with v_f16 (fp16
    [B, N, H, d], COMMIT only) its rows idx receive the fp16 copy of the updated values
    (fl_kv_residual_quant_kv_v16)."""
    B, N, H, d = k_cur.shape
    _dev(k_cur, torch.bfloat16, "k_cur")
    _dev(v_cur, torch.bfloat16, "v_cur", k_cur.shape)
    _dev(k_ref, torch.bfloat16, "k_ref", k_cur.shape)
    _dev(v_ref, torch.bfloat16, "v_ref", k_cur.shape)
    k = N if idx is None else idx.shape[1]
    _dev(idx, torch.int32, "idx", None if idx is None else (B, k))
    dev = k_cur.device

    def outputs(axis):
        codes = torch.empty(B, k, H, d * bits // 8, dtype=torch.uint8, device=dev)
        scale = zero = None
        if bits != 16:
            shp = meta_shape(B, k, H, d, group, axis)
            scale = torch.empty(shp, dtype=torch.float16, device=dev)
            zero = torch.empty(shp, dtype=torch.float16, device=dev)
        out_rows = None
        if mode == DQ_COMPACT and rows:
            out_rows = torch.empty(B, k, H, d, dtype=torch.bfloat16, device=dev)
        return codes, scale, zero, out_rows

    ko, vo = outputs(AXIS_TOKEN), outputs(AXIS_CHANNEL)
    if v_f16 is not None:
        if mode != DQ_COMMIT:
            raise FlashLoopError("kv_residual_quant_kv: v_f16 needs mode=DQ_COMMIT")
        _dev(v_f16, torch.float16, "v_f16", k_cur.shape)
        rc = load().fl_kv_residual_quant_kv_v16(_p(k_cur), _p(k_ref), _p(v_cur), _p(v_ref), _p(v_f16), _p(idx), k,
                                                B, N, H, d, bits, group, _p(ko[0]), _p(ko[1]), _p(ko[2]),
                                                _p(vo[0]), _p(vo[1]), _p(vo[2]), _stream())
        _check(rc, "fl_kv_residual_quant_kv_v16")
        return ko, vo
    rc = load().fl_kv_residual_quant_kv(_p(k_cur), _p(k_ref), _p(v_cur), _p(v_ref), _p(idx), k, B, N, H, d, bits,
                                        group, _p(ko[0]), _p(ko[1]), _p(ko[2]), _p(vo[0]), _p(vo[1]), _p(vo[2]),
                                        _p(ko[3]), _p(vo[3]), mode, _stream())
    _check(rc, "fl_kv_residual_quant_kv")
    return ko, vo


def kv_f16_rows(x, idx=None, out=None):
    """fp16 copy of rows of a bf16 [B, N, H, d] tensor (fl_kv_f16_rows): every row when idx is None, else
    rows idx of `out` (fp16 [B, N, H, d], allocated when None); returns out."""
    B, N, H, d = x.shape
    _dev(x, torch.bfloat16, "x")
    k = N if idx is None else idx.shape[1]
    _dev(idx, torch.int32, "idx", None if idx is None else (B, k))
    out = torch.empty(B, N, H, d, dtype=torch.float16, device=x.device) if out is None else out
    _dev(out, torch.float16, "out", x.shape)
    rc = load().fl_kv_f16_rows(_p(x), _p(idx), k, B, N, H, d, _p(out), _stream())
    _check(rc, "fl_kv_f16_rows")
    return out


def kv_residual_dequant_kv(k_enc, v_enc, idx, bits, group, k_hat, v_hat, mode=DQ_COMPACT):
    """Keys (token axis) and values (channel axis) in one call; k_enc / v_enc = (codes, scale, zero).
    COMPACT: returns (key rows, value rows) [B, k, H, d]; COMMIT: updates k_hat and v_hat in place."""
    B, N, H, d = k_hat.shape
    _dev(k_hat, torch.bfloat16, "k_hat")
    _dev(v_hat, torch.bfloat16, "v_hat", k_hat.shape)
    k = N if idx is None else idx.shape[1]
    _dev(idx, torch.int32, "idx", None if idx is None else (B, k))
    for name, enc, axis in (("k", k_enc, AXIS_TOKEN), ("v", v_enc, AXIS_CHANNEL)):
        _dev(enc[0], torch.uint8, f"{name} codes", (B, k, H, d * bits // 8))
        if bits != 16:
            shp = meta_shape(B, k, H, d, group, axis)
            _dev(enc[1], torch.float16, f"{name} scale", shp)
            _dev(enc[2], torch.float16, f"{name} zero", shp)
    k_rows = v_rows = None
    if mode == DQ_COMPACT:
        k_rows = torch.empty(B, k, H, d, dtype=torch.bfloat16, device=k_hat.device)
        v_rows = torch.empty(B, k, H, d, dtype=torch.bfloat16, device=k_hat.device)
    rc = load().fl_kv_residual_dequant_kv(_p(k_enc[0]), _p(k_enc[1]), _p(k_enc[2]), _p(v_enc[0]), _p(v_enc[1]),
                                          _p(v_enc[2]), _p(idx), k, B, N, H, d, bits, group, mode, _p(k_hat),
                                          _p(v_hat), _p(k_rows), _p(v_rows), _stream())
    _check(rc, "fl_kv_residual_dequant_kv")
    return k_rows, v_rows


def kv_residual_dequant(codes, scale, zero, idx, bits, group, axis, x_hat, mode=DQ_COMPACT):
    """COMPACT: returns the reconstructed rows [B, k, H, d]; COMMIT: updates x_hat in place."""
    B, N, H, d = x_hat.shape
    _dev(x_hat, torch.bfloat16, "x_hat")
    k = N if idx is None else idx.shape[1]
    _dev(idx, torch.int32, "idx", None if idx is None else (B, k))
    _dev(codes, torch.uint8, "codes", (B, k, H, d * bits // 8))
    if bits != 16:
        shp = meta_shape(B, k, H, d, group, axis)
        _dev(scale, torch.float16, "scale", shp)
        _dev(zero, torch.float16, "zero", shp)
    out_rows = None
    if mode == DQ_COMPACT:
        out_rows = torch.empty(B, k, H, d, dtype=torch.bfloat16, device=x_hat.device)
    rc = load().fl_kv_residual_dequant(_p(codes), _p(scale), _p(zero), _p(idx), k, B, N, H, d, bits, group,
                                       axis, mode, _p(x_hat), _p(out_rows), _stream())
    _check(rc, "fl_kv_residual_dequant")
    return out_rows if mode == DQ_COMPACT else x_hat


# ---- (3) attention ----------------------------------------------------------------------------------
def loop_sparse_attn(q_cur, q_prev, k_cache, v_cache, k_new, v_new, slot, rows, cols, window, lse_ref, o,
                     sm_scale=None, ws=None, term_prev=None, mass_prev=None, slot_prev=None, term_out=None,
                     mass_out=None, v16=None):
    """Mass-corrected update of rows `rows` (in place on lse_ref and o).

    term_out/mass_out (fp32 [B, k, H, d] / [B, k, H]) also keep this loop's add terms; term_prev/mass_prev with
    slot_prev (the previous loop's slot map) reuse the previous loop's add terms as the subtract terms, in
    which case q_prev may be None, and k_new/v_new may be None when the caches already hold this loop's rows.
    v16: the fp16 copy of v_cache (given terms over current caches only; fl_loop_sparse_attn_terms_v16)."""
    B, N, H, d = q_cur.shape
    k = rows.shape[1]
    reuse = term_prev is not None
    for name, t in (("q_cur", q_cur), ("q_prev", q_prev), ("k_cache", k_cache), ("v_cache", v_cache)):
        _dev(t, torch.bfloat16, name, q_cur.shape)
    _dev(k_new, torch.bfloat16, "k_new", (B, k, H, d))
    _dev(v_new, torch.bfloat16, "v_new", (B, k, H, d))
    _dev(slot, torch.int32, "slot", (B, N))
    _dev(rows, torch.int32, "rows", (B, k))
    c_list = 0 if cols is None else cols.shape[2]
    _dev(cols, torch.int32, "cols", None if cols is None else (B, H, c_list))
    _dev(lse_ref, torch.float32, "lse_ref", (B, N, H))
    _dev(o, torch.float32, "o", (B, N, H, d))
    k_prev = 0
    if reuse:
        k_prev = term_prev.shape[1]
        _dev(term_prev, torch.float32, "term_prev", (B, k_prev, H, d))
        _dev(mass_prev, torch.float32, "mass_prev", (B, k_prev, H))
        _dev(slot_prev, torch.int32, "slot_prev", (B, N))
    _dev(term_out, torch.float32, "term_out", (B, k, H, d))
    _dev(mass_out, torch.float32, "mass_out", (B, k, H))
    sm_scale = 1.0 / math.sqrt(d) if sm_scale is None else sm_scale
    lib = load()
    if v16 is not None:
        if not reuse or k_new is not None or v_new is not None:
            raise FlashLoopError("loop_sparse_attn: v16 needs term_prev and current caches (k_new = v_new = None)")
        _dev(v16, torch.float16, "v16", q_cur.shape)
        rc = lib.fl_loop_sparse_attn_terms_v16(_p(q_cur), _p(k_cache), _p(v_cache), _p(v16), _p(rows), k, _p(cols),
                                               c_list, window, B, N, H, d, sm_scale, _p(lse_ref), _p(o),
                                               _p(term_prev), _p(mass_prev), _p(slot_prev), k_prev, _p(term_out),
                                               _p(mass_out), _stream())
        _check(rc, "fl_loop_sparse_attn_terms_v16")
        return o, lse_ref
    need = lib.fl_loop_sparse_attn_ws(B, N, H, d, k, c_list, window, 0)
    if need and (ws is None or ws.numel() < need):
        ws = torch.empty(need, dtype=torch.uint8, device=q_cur.device)
    if reuse or term_out is not None:
        rc = lib.fl_loop_sparse_attn_terms(_p(q_cur), _p(q_prev), _p(k_cache), _p(v_cache), _p(k_new), _p(v_new),
                                           _p(slot), _p(rows), k, _p(cols), c_list, window, B, N, H, d, sm_scale,
                                           _p(lse_ref), _p(o), _p(term_prev), _p(mass_prev), _p(slot_prev), k_prev,
                                           _p(term_out), _p(mass_out), _p(ws) if need else None, need, _stream())
        _check(rc, "fl_loop_sparse_attn_terms")
    else:
        rc = lib.fl_loop_sparse_attn(_p(q_cur), _p(q_prev), _p(k_cache), _p(v_cache), _p(k_new), _p(v_new),
                                     _p(slot), _p(rows), k, _p(cols), c_list, window, B, N, H, d, sm_scale, 0,
                                     _p(lse_ref), _p(o), _p(ws) if need else None, need, _stream())
        _check(rc, "fl_loop_sparse_attn")
    return o, lse_ref


def attn_kernel_name(pass_, k, c_list, window, B, N, H, d):
    """Name of the kernel an attention pass launches for the shape, or None (fl_attn_kernel_name; host only).
    pass_: PASS_ADD (add pass over current caches), PASS_SUBTRACT or PASS_BOTH."""
    name = load().fl_attn_kernel_name(pass_, k, c_list, window, B, N, H, d)
    return None if name is None else name.decode()


def subtract_terms_supported(k, c_list, window, N, d):
    """Whether fl_loop_subtract_terms covers the shape (a column list of at most 3072 entries)."""
    return bool(load().fl_loop_subtract_terms_supported(k, c_list, window, N, d))


def subtract_terms(q_prev, k_cache, v_cache, rows, cols, window, lse_ref, term_out=None, mass_out=None,
                   sm_scale=None, v16=None):
    """Subtract term and mass of Eq. 7 over the previous loop's state: (term fp32 [B, k, H, d], m fp32 [B, k, H])
    in the row order of `rows` (fl_loop_subtract_terms; with v16, the fp16 copy of v_cache,
    fl_loop_subtract_terms_v16)."""
    B, N, H, d = q_prev.shape
    k = rows.shape[1]
    for name, t in (("q_prev", q_prev), ("k_cache", k_cache), ("v_cache", v_cache)):
        _dev(t, torch.bfloat16, name, q_prev.shape)
    _dev(rows, torch.int32, "rows", (B, k))
    c_list = 0 if cols is None else cols.shape[2]
    _dev(cols, torch.int32, "cols", None if cols is None else (B, H, c_list))
    _dev(lse_ref, torch.float32, "lse_ref", (B, N, H))
    term_out = torch.empty(B, k, H, d, dtype=torch.float32, device=q_prev.device) if term_out is None else term_out
    mass_out = torch.empty(B, k, H, dtype=torch.float32, device=q_prev.device) if mass_out is None else mass_out
    _dev(term_out, torch.float32, "term_out", (B, k, H, d))
    _dev(mass_out, torch.float32, "mass_out", (B, k, H))
    sm_scale = 1.0 / math.sqrt(d) if sm_scale is None else sm_scale
    if v16 is not None:
        _dev(v16, torch.float16, "v16", q_prev.shape)
        rc = load().fl_loop_subtract_terms_v16(_p(q_prev), _p(k_cache), _p(v_cache), _p(v16), _p(rows), k, _p(cols),
                                               c_list, window, B, N, H, d, sm_scale, _p(lse_ref), _p(term_out),
                                               _p(mass_out), _stream())
        _check(rc, "fl_loop_subtract_terms_v16")
        return term_out, mass_out
    rc = load().fl_loop_subtract_terms(_p(q_prev), _p(k_cache), _p(v_cache), _p(rows), k, _p(cols), c_list, window,
                                       B, N, H, d, sm_scale, _p(lse_ref), _p(term_out), _p(mass_out), _stream())
    _check(rc, "fl_loop_subtract_terms")
    return term_out, mass_out


def dense_attn(q, k_cache, v_cache, o=None, lse=None, sm_scale=None):
    """Dense causal loop: returns (o fp32 [B, N, H, d], lse fp32 [B, N, H])."""
    B, N, H, d = q.shape
    for name, t in (("q", q), ("k_cache", k_cache), ("v_cache", v_cache)):
        _dev(t, torch.bfloat16, name, q.shape)
    o = torch.empty(B, N, H, d, dtype=torch.float32, device=q.device) if o is None else o
    lse = torch.empty(B, N, H, dtype=torch.float32, device=q.device) if lse is None else lse
    sm_scale = 1.0 / math.sqrt(d) if sm_scale is None else sm_scale
    lib = load()
    need = lib.fl_loop_sparse_attn_ws(B, N, H, d, N, 0, 0, ATTN_DENSE)
    ws = torch.empty(need, dtype=torch.uint8, device=q.device) if need else None
    rc = lib.fl_loop_sparse_attn(_p(q), None, _p(k_cache), _p(v_cache), None, None, None, None, N, None, 0, 0,
                                 B, N, H, d, sm_scale, ATTN_DENSE, _p(lse), _p(o), _p(ws), need, _stream())
    _check(rc, "fl_loop_sparse_attn(dense)")
    return o, lse


def column_scores(q, k_cache):
    """fp32 column keys [B, H, N] of a dense source loop (fp64 inside)."""
    B, N, H, d = q.shape
    _dev(q, torch.bfloat16, "q")
    _dev(k_cache, torch.bfloat16, "k_cache", q.shape)
    lib = load()
    need = lib.fl_column_scores_ws(B, N, H)
    ws = torch.empty(need, dtype=torch.uint8, device=q.device)
    col_key = torch.empty(B, H, N, dtype=torch.float32, device=q.device)
    rc = lib.fl_column_scores(_p(q), _p(k_cache), B, N, H, d, _p(col_key), _p(ws), need, _stream())
    _check(rc, "fl_column_scores")
    return col_key


def select_columns(col_key, n_sink, t):
    """Column list [B, H, min(n_sink, N) + t], ascending."""
    B, H, N = col_key.shape
    _dev(col_key, torch.float32, "col_key")
    ns = min(n_sink, N)
    cols = torch.empty(B, H, ns + t, dtype=torch.int32, device=col_key.device)
    rc = load().fl_select_columns(_p(col_key), B, H, N, n_sink, t, _p(cols), _stream())
    _check(rc, "fl_select_columns")
    return cols


# ---- (6) decode ---------------------------------------------------------------------------------------
def decode_ws(k_cache, cols, c_next):
    """A workspace for decode_step over these shapes (reusable across calls of the same or smaller size)."""
    B, T, H, d = k_cache.shape
    c = 0 if cols is None else cols.shape[2]
    need = load().fl_decode_step_ws(B, T, H, d, c, c_next)
    return torch.empty(max(need, 1), dtype=torch.uint8, device=k_cache.device)


def _decode_args(q, k_cache, v_cache, cols, mass, sub, o, c_next, lse, out):
    B, T, H, d = k_cache.shape
    _dev(q, torch.bfloat16, "q", (B, H, d))
    _dev(k_cache, torch.bfloat16, "k_cache")
    _dev(v_cache, torch.bfloat16, "v_cache", k_cache.shape)
    _dev(o, torch.float32, "o", (B, H, d))
    c = 0 if cols is None else cols.shape[2]
    if cols is not None:
        _dev(cols, torch.int32, "cols", (B, H, c))
        _dev(mass, torch.float32, "mass", (B, H))
        _dev(sub, torch.float32, "sub", (B, H, d))
    _dev(lse, torch.float32, "lse", (B, H))
    cols_next = mass_next = sub_next = None
    if c_next > 0:
        if out is None:
            dev = q.device
            out = (torch.empty(B, H, c_next, dtype=torch.int32, device=dev),
                   torch.empty(B, H, dtype=torch.float32, device=dev),
                   torch.empty(B, H, d, dtype=torch.float32, device=dev))
        cols_next, mass_next, sub_next = out
        _dev(cols_next, torch.int32, "cols_next", (B, H, c_next))
        _dev(mass_next, torch.float32, "mass_next", (B, H))
        _dev(sub_next, torch.float32, "sub_next", (B, H, d))
    return B, T, H, d, c, cols_next, mass_next, sub_next


def decode_step(q, k_cache, v_cache, cols, mass, sub, o, c_next, n_sink=0, window=0, sm_scale=None, lse=None,
                out=None, ws=None):
    """One loop of the decode position T-1.  q bf16 [B, H, d]; caches bf16 [B, T, H, d]; cols int32 [B, H, c]
    (or None for a dense source loop, then mass and sub are unused); o fp32 [B, H, d] updated in place.
    out: optional (cols_next, mass_next, sub_next) to write into; ws: optional workspace (decode_ws).  With
    both given nothing is allocated.  Returns (cols_next [B, H, c_next], mass_next [B, H], sub_next
    [B, H, d]) or Nones when c_next == 0."""
    B, T, H, d, c, cols_next, mass_next, sub_next = _decode_args(q, k_cache, v_cache, cols, mass, sub, o, c_next,
                                                                 lse, out)
    sm_scale = 1.0 / math.sqrt(d) if sm_scale is None else sm_scale
    lib = load()
    need = lib.fl_decode_step_ws(B, T, H, d, c, c_next)
    if ws is None:
        ws = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    _dev(ws, torch.uint8, "ws")
    rc = lib.fl_decode_step(_p(q), _p(k_cache), _p(v_cache), _p(cols), c, _p(mass), _p(sub), B, T, H, d, sm_scale,
                            _p(o), _p(lse), n_sink, window, c_next, _p(cols_next), _p(mass_next), _p(sub_next),
                            _p(ws), ws.numel(), _stream())
    _check(rc, "fl_decode_step")
    return cols_next, mass_next, sub_next


def decode_step_noalloc(q, k_cache, v_cache, cols, mass, sub, o, c_next, out=None, n_sink=0, window=0,
                        sm_scale=None, lse=None):
    """decode_step without a caller workspace: the library's own device scratch serves as the workspace
    (calls overlapping on one GPU race on it).  Nothing is allocated when `out` is given (or c_next == 0)."""
    B, T, H, d, c, cols_next, mass_next, sub_next = _decode_args(q, k_cache, v_cache, cols, mass, sub, o, c_next,
                                                                 lse, out)
    sm_scale = 1.0 / math.sqrt(d) if sm_scale is None else sm_scale
    rc = load().fl_decode_step_noalloc(_p(q), _p(k_cache), _p(v_cache), _p(cols), c, _p(mass), _p(sub), B, T, H, d,
                                       sm_scale, _p(o), _p(lse), n_sink, window, c_next, _p(cols_next),
                                       _p(mass_next), _p(sub_next), _stream())
    _check(rc, "fl_decode_step_noalloc")
    return cols_next, mass_next, sub_next


# ---- (7) list pruning for a smaller budget --------------------------------------------------------------
def prune_columns(q, k_cache, rows, cols, lse_ref, n_sink, t_next, sm_scale=None):
    """Keep the sinks and the t_next list entries that loop r's updated rows gave the most probability mass.
    q, k_cache bf16 [B, N, H, d] (loop r); rows int32 [B, k] (or None when k = 0); cols int32 [B, H, c_list];
    lse_ref fp32 [B, N, H].  Returns (cols_next int32 [B, H, ns + t_next], col_key fp32 [B, H, c_list - ns])."""
    B, N, H, d = k_cache.shape
    _dev(q, torch.bfloat16, "q", k_cache.shape)
    _dev(k_cache, torch.bfloat16, "k_cache")
    c_list = cols.shape[2]
    _dev(cols, torch.int32, "cols", (B, H, c_list))
    _dev(lse_ref, torch.float32, "lse_ref", (B, N, H))
    k = 0 if rows is None else rows.shape[1]
    if rows is not None:
        _dev(rows, torch.int32, "rows", (B, k))
    ns = min(n_sink, c_list)
    dev = q.device
    col_key = torch.empty(B, H, c_list - ns, dtype=torch.float32, device=dev)
    cols_next = torch.empty(B, H, ns + t_next, dtype=torch.int32, device=dev)
    sm_scale = 1.0 / math.sqrt(d) if sm_scale is None else sm_scale
    lib = load()
    need = lib.fl_prune_columns_ws(B, H, k, c_list, n_sink)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    rc = lib.fl_prune_columns(_p(q), _p(k_cache), _p(rows), k, _p(cols), c_list, _p(lse_ref), B, N, H, d,
                              sm_scale, n_sink, t_next, _p(col_key) if c_list > ns else None, _p(cols_next),
                              _p(ws), need, _stream())
    _check(rc, "fl_prune_columns")
    return cols_next, col_key


# ---- (8) recent tokens kept in bf16 --------------------------------------------------------------------
def kv_keep_recent(x_cur, idx, tail, cache=None, rows=None):
    """Store the active rows i >= N - tail exactly: cache [B, N, H, d] at i and/or the compact rows
    [B, k, H, d] at their position (x_cur bf16 [B, N, H, d]; idx int32 [B, k] or None for every row)."""
    B, N, H, d = x_cur.shape
    _dev(x_cur, torch.bfloat16, "x_cur")
    k = N if idx is None else idx.shape[1]
    _dev(idx, torch.int32, "idx", None if idx is None else (B, k))
    _dev(cache, torch.bfloat16, "cache", None if cache is None else x_cur.shape)
    _dev(rows, torch.bfloat16, "rows", None if rows is None else (B, k, H, d))
    rc = load().fl_kv_keep_recent(_p(x_cur), _p(idx), k, B, N, H, d, tail, _p(cache), _p(rows), _stream())
    _check(rc, "fl_kv_keep_recent")
