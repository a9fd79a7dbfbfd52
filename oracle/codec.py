"""Cross-loop K/V residual codec (test infrastructure only).

Follows Section 4.3, Eq. (4) and Appendix D.3, Eq. (8): loop 1 stores a quantized base
X^(1)_hat = D(Q(X^(1))); every later loop quantizes only the active rows' residual against the previous
reconstruction, Delta_i = X^(r)_i - X^(r-1)_hat_i, and reconstructs X^(r)_hat_i = X^(r-1)_hat_i +
D(Q(Delta))_i for active rows while inactive rows keep X^(r-1)_hat.  The quantizer is the one fixed in
Appendix E ("Quantization Setting"): asymmetric, group-wise, scale and offset from the group's min and
max, the same scheme for base and residuals; keys grouped per channel, values per token.

Readings (where the paper is silent):
* K (axis TOKEN): a group is G consecutive packed active rows x one (head, channel); the last group is
  partial.  V (axis CHANNEL): a group is one (row, head) x G consecutive channels (G divides d).
* zero z = largest fp16 <= min; scale s = smallest fp16 >= (max - z) / (2^b - 1), computed in fp64,
  so the grid covers [min, max]; s == 0 gives all-zero codes.
* code q = clamp(rint(fp32(fp32(Delta - z) / s)), 0, 2^b - 1): IEEE fp32 division, ties to even.
* dequantized residual dq = fp32(z + q * s) (q * s is exact in fp32); the reconstruction is a bf16
  state: X_hat = bf16(fp32(X_prev_hat) + dq).
* codes are packed LSB-first along channels: channel e of a (row, head) goes to byte e*b//8 at bit
  (e mod 8/b)*b; b = 8 is one byte per code; b = 16 means "no quantization" and the payload is the
  raw bf16 state (X_hat = X).
"""
from __future__ import annotations

import numpy as np

from .numerics import bf16_to_f32, f16_down, f16_up, f32_to_bf16

AXIS_TOKEN = 0
AXIS_CHANNEL = 1


def _rows(x, idx):
    """Gather the packed rows [B, k, H, d] of a [B, N, H, d] array."""
    B = x.shape[0]
    if idx is None:
        return x
    return np.stack([x[b, np.asarray(idx[b], dtype=np.int64)] for b in range(B)])


def group_minmax(delta, group, axis):
    """Per-group min and max of fp32 residuals delta [B, k, H, d].

    TOKEN: returns [B, ceil(k/G), H, d];  CHANNEL: returns [B, k, H, d/G].
    """
    B, k, H, d = delta.shape
    if axis == AXIS_TOKEN:
        ng = -(-k // group)
        mn = np.empty((B, ng, H, d), np.float32)
        mx = np.empty((B, ng, H, d), np.float32)
        for g in range(ng):
            blk = delta[:, g * group:min(g * group + group, k)]
            mn[:, g] = blk.min(axis=1)
            mx[:, g] = blk.max(axis=1)
        return mn, mx
    if d % group:
        raise ValueError("CHANNEL axis needs G | d")
    blk = delta.reshape(B, k, H, d // group, group)
    return blk.min(axis=4), blk.max(axis=4)


def _expand(meta, group, axis, k):
    """Broadcast per-group metadata back to element shape [B, k, H, d]."""
    if axis == AXIS_TOKEN:
        return np.repeat(meta, group, axis=1)[:, :k]
    return np.repeat(meta, group, axis=3)


def quantize(x_cur, x_ref, idx, bits, group, axis):
    """Q(Delta) for the packed rows idx, Delta = fp32(X^(r)) - fp32(X^(r-1)_hat) (Eq. (8)).

    x_cur, x_ref : uint16 bf16 [B, N, H, d] (x_ref None = zeros, the base loop)
    idx          : None (all rows) or int [B, k] ascending
    Returns the dict of `encode`, plus the raw bf16 payload when bits == 16.
    """
    cur = bf16_to_f32(_rows(x_cur, idx))
    ref = np.zeros_like(cur) if x_ref is None else bf16_to_f32(_rows(x_ref, idx))
    delta = cur - ref                                          # fp32, round to nearest even
    if bits == 16:
        B, k, H, d = delta.shape
        raw = _rows(x_cur, idx).astype(np.uint16)
        return dict(codes=raw.view(np.uint8).reshape(B, k, H, 2 * d), scale=None, zero=None,
                    q=raw, delta=delta)
    return encode(delta, bits, group, axis)


def encode(delta, bits, group, axis):
    """Group-wise asymmetric quantization of fp32 residuals delta [B, k, H, d].

    Returns dict(codes uint8 [B, k, H, d*bits/8], scale/zero float16 (TOKEN: [B, ceil(k/G), H, d],
    CHANNEL: [B, k, H, d/G]), q uint8 [B, k, H, d], delta).
    """
    if bits not in (2, 4, 8):
        raise ValueError("bits must be 2, 4, 8 or 16")
    delta = np.asarray(delta, dtype=np.float32)
    k = delta.shape[1]
    qmax = (1 << bits) - 1
    mn, mx = group_minmax(delta, group, axis)
    z = f16_down(mn.astype(np.float64))
    s = f16_up((mx.astype(np.float64) - z.astype(np.float64)) / qmax)
    z32 = _expand(z, group, axis, k).astype(np.float32)
    s32 = _expand(s, group, axis, k).astype(np.float32)
    with np.errstate(divide="ignore", invalid="ignore"):
        t = (delta - z32) / s32                                # two fp32 roundings, IEEE division
        q = np.where(s32 == 0, 0, np.clip(np.rint(t), 0, qmax))
    q = q.astype(np.uint8)
    return dict(codes=pack(q, bits), scale=s, zero=z, q=q, delta=delta)


def pack(q, bits):
    """Pack codes [..., d] LSB-first along the last axis into bytes [..., d*bits/8]."""
    if bits == 8:
        return q.astype(np.uint8)
    per = 8 // bits
    d = q.shape[-1]
    q = q.astype(np.uint8).reshape(*q.shape[:-1], d // per, per)
    out = np.zeros(q.shape[:-1], dtype=np.uint8)
    for t in range(per):
        out |= (q[..., t] << np.uint8(t * bits)).astype(np.uint8)
    return out


def unpack(codes, bits, d):
    """Inverse of pack: bytes [..., d*bits/8] -> codes [..., d] (uint8)."""
    if bits == 8:
        return codes.astype(np.uint8)
    per = 8 // bits
    mask = np.uint8((1 << bits) - 1)
    parts = [(codes >> np.uint8(t * bits)) & mask for t in range(per)]
    return np.stack(parts, axis=-1).reshape(*codes.shape[:-1], d)


def dequantize(codes, scale, zero, bits, group, axis, d):
    """D(Q(Delta)) as fp32 [B, k, H, d] (bits 2/4/8)."""
    q = unpack(codes, bits, d).astype(np.float32)
    k = q.shape[1]
    z32 = _expand(zero, group, axis, k).astype(np.float32)
    s32 = _expand(scale, group, axis, k).astype(np.float32)
    return z32 + q * s32                                       # q * s exact; one rounding


def reconstruct(x_hat_prev, x_cur, idx, enc, bits, group, axis):
    """Eq. (8): X^(r)_hat = X^(r-1)_hat with active rows replaced by bf16(X^(r-1)_hat + dq).

    x_hat_prev : uint16 bf16 [B, N, H, d] or None (base loop: zeros)
    Returns (x_hat uint16 [B, N, H, d], new_rows uint16 [B, k, H, d]).
    """
    B, N, H, d = x_cur.shape
    if bits == 16:
        new_rows = _rows(x_cur, idx).astype(np.uint16)
    else:
        dq = dequantize(enc["codes"], enc["scale"], enc["zero"], bits, group, axis, d)
        base = (np.zeros(dq.shape, np.float32) if x_hat_prev is None
                else bf16_to_f32(_rows(x_hat_prev, idx)))
        new_rows = f32_to_bf16(base + dq)
    x_hat = (np.zeros((B, N, H, d), np.uint16) if x_hat_prev is None else x_hat_prev.copy())
    for b in range(B):
        rows = np.arange(N) if idx is None else np.asarray(idx[b], dtype=np.int64)
        x_hat[b, rows] = new_rows[b]
    return x_hat, new_rows


def keep_recent(x_hat, new_rows, x_cur, idx, tail):
    """Appendix E keeps the most recent `tail` tokens in bf16: every stored row i >= N - tail is the exact
    X^(r) row instead of its reconstruction.  Reading: the rows are still encoded with the others (the groups
    and codes are unchanged); only what the state stores for them is exact.  x_hat [B, N, H, d] and the
    compact new_rows [B, k, H, d] (either may be None) are returned as updated copies."""
    if tail <= 0:
        return x_hat, new_rows
    B, N = x_cur.shape[:2]
    lo = max(0, N - tail)
    if x_hat is not None:
        x_hat = x_hat.copy()
        for b in range(B):
            rows = np.arange(N) if idx is None else np.asarray(idx[b], dtype=np.int64)
            rows = rows[rows >= lo]
            x_hat[b, rows] = x_cur[b, rows]
    if new_rows is not None:
        new_rows = new_rows.copy()
        for b in range(B):
            rows = np.arange(N) if idx is None else np.asarray(idx[b], dtype=np.int64)
            sel = np.nonzero(rows >= lo)[0]
            new_rows[b, sel] = x_cur[b, rows[sel]]
    return x_hat, new_rows
