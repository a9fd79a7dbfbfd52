"""Per-layer sequencing of the FlashLoop step on one GPU (device tensors only; all math is in the library).

setup()       dense source loop 1: base codec of K (per-channel groups) and V (per-token groups) with the
              reconstruction written straight into the caches (the most recent `tail` rows stored exactly,
              Appendix E), dense causal attention over the
              reconstructed base, fp64 column statistic and the column list (Appendix D.2, Eq. 6).
sparse_step() one sparse loop r >= 2: select the active rows among the previous loop's (Eq. 5), quantize
              their K/V residuals against the caches and reconstruct the new rows (Eq. 8), apply the
              mass-corrected update to their outputs (Eq. 7), then commit the new rows into the caches.
              Each loop keeps its add terms; from the second sparse loop on they serve as the subtract
              terms (equal in exact arithmetic: the column sets are fixed and the active rows nested).
              Such a loop needs only the new state, so the quantizers commit the new rows straight into
              the caches and the attention reads every column from them.  A loop without stored terms
              computes its subtract terms first, over the loop r-1 state, where the segment kernel covers
              the shape, and then runs as such a loop; otherwise it runs both passes in one kernel and
              commits after it.
The layer also keeps an fp16 copy of the value cache (v16): the quantizers write it with the committed rows,
and the attention's segment kernels load value tiles from it instead of converting bf16 tiles in LDS
(bitwise the same results).
prune_list()  a smaller column budget for the next loop (Section 4.2): keep the sinks and the entries the
              last loop's updated rows gave the most probability mass.  The next loop then runs both passes
              (its subtract pass recomputes the kept columns' share with the same lse_ref).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

from . import flashloop as fl


@dataclass
class LayerState:
    k_hat: torch.Tensor            # bf16 [B, N, H, d]  X_hat of the last finished loop
    v_hat: torch.Tensor
    o: torch.Tensor                # fp32 [B, N, H, d]
    lse: torch.Tensor              # fp32 [B, N, H]
    cols: torch.Tensor             # int32 [B, H, c_list]
    cand: torch.Tensor | None = None   # int32 [B, k] active rows of the last loop (None after loop 1)
    window: int = 0
    group: int = 64
    base: dict = field(default_factory=dict)
    reuse: bool = True                  # keep add terms and reuse them as the next loop's subtract terms
    term: torch.Tensor | None = None    # fp32 [B, k, H, d] add terms of the last loop (row order of cand)
    mass: torch.Tensor | None = None    # fp32 [B, k, H]
    slot_prev: torch.Tensor | None = None   # int32 [B, N] slot map of the last loop
    tail: int = 0                       # the most recent positions stored exactly in bf16 (Appendix E)
    v16: torch.Tensor | None = None     # fp16 [B, N, H, d] copy of v_hat (kept current with it), or None


def setup(q1, k1, v1, base_bits, group, n_sink, t, window, tail=0, v16=True):
    B, N, H, d = k1.shape
    k_hat = torch.empty_like(k1)
    v_hat = torch.empty_like(v1)
    ck, sk, zk, _ = fl.kv_residual_quant(k1, None, None, base_bits, group, fl.AXIS_TOKEN, rows=k_hat)
    cv, sv, zv, _ = fl.kv_residual_quant(v1, None, None, base_bits, group, fl.AXIS_CHANNEL, rows=v_hat)
    if tail:
        fl.kv_keep_recent(k1, None, tail, cache=k_hat)
        fl.kv_keep_recent(v1, None, tail, cache=v_hat)
    o, lse = fl.dense_attn(q1, k_hat, v_hat)
    col_key = fl.column_scores(q1, k_hat)
    cols = fl.select_columns(col_key, n_sink, t)
    st = LayerState(k_hat, v_hat, o, lse, cols, None, window, group)
    st.tail = tail
    st.v16 = fl.kv_f16_rows(v_hat) if v16 else None
    st.base = dict(codes_k=ck, scale_k=sk, zero_k=zk, codes_v=cv, scale_v=sv, zero_v=zv, col_key=col_key)
    return st


def subtract_pass_first(k, c_list, window, B, N, H, d):
    """Whether a loop without stored terms runs as the subtract pass, the commit and the add pass (rather
    than the two-pass kernel): where a segment kernel (one team or two) takes the subtract pass.  Each
    segment pass streams the list tiles once more than the two-pass kernel does, but loads the value tiles
    from the fp16 copy and keeps its rows on the chip; with the copy the three calls measured 15-25% faster
    than quantize, two-pass kernel, commit and copy refresh, with a band and without one.  Shapes that only
    the 64-row kernels cover keep the two-pass kernel."""
    return fl.attn_kernel_name(fl.PASS_SUBTRACT, k, c_list, window, B, N, H, d) in ("seg_sub_kernel",
                                                                                    "seg1_sub_kernel")


def sparse_step(st: LayerState, qr, qp, kr, kp, vr, vp, k_r, bits, keep=False):
    """Advance the layer by one sparse loop.  Returns the loop's outputs when keep=True."""
    idx, slot, key = fl.select_tokens(kr, kp, vr, vp, k_r, cand=st.cand)
    B, N, H, d = kr.shape
    k = idx.shape[1]
    term = mass = None
    if st.reuse:
        term = torch.empty(B, k, H, d, dtype=torch.float32, device=kr.device)
        mass = torch.empty(B, k, H, dtype=torch.float32, device=kr.device)
    k_new = v_new = None
    reuse = st.reuse and st.term is not None
    split = not reuse and subtract_pass_first(k, st.cols.shape[2], st.window, B, N, H, d)
    if reuse or split:
        term_prev, mass_prev, slot_prev = st.term, st.mass, st.slot_prev
        if split:
            # no stored terms: the subtract pass over the loop r-1 state first (its terms index this loop's
            # rows), so that the new rows can be committed before the add pass
            term_prev, mass_prev = fl.subtract_terms(qp, st.k_hat, st.v_hat, idx, st.cols, st.window, st.lse,
                                                     v16=st.v16)
            slot_prev = slot
        # the add pass alone: commit the new rows first (and their fp16 values), then attend over the caches
        (ck, sk, zk, _), (cv, sv, zv, _) = fl.kv_residual_quant_kv(kr, st.k_hat, vr, st.v_hat, idx, bits,
                                                                   st.group, mode=fl.DQ_COMMIT, v_f16=st.v16)
        if st.tail:
            fl.kv_keep_recent(kr, idx, st.tail, cache=st.k_hat)
            fl.kv_keep_recent(vr, idx, st.tail, cache=st.v_hat)
            if st.v16 is not None:
                fl.kv_f16_rows(st.v_hat, idx, out=st.v16)
        fl.loop_sparse_attn(qr, None, st.k_hat, st.v_hat, None, None, slot, idx, st.cols, st.window, st.lse,
                            st.o, term_prev=term_prev, mass_prev=mass_prev, slot_prev=slot_prev, term_out=term,
                            mass_out=mass, v16=st.v16)
    else:
        # both passes: the subtract pass needs the loop r-1 caches, so commit after the attention
        (ck, sk, zk, k_new), (cv, sv, zv, v_new) = fl.kv_residual_quant_kv(kr, st.k_hat, vr, st.v_hat, idx, bits,
                                                                           st.group)
        if st.tail:
            fl.kv_keep_recent(kr, idx, st.tail, rows=k_new)
            fl.kv_keep_recent(vr, idx, st.tail, rows=v_new)
        fl.loop_sparse_attn(qr, qp, st.k_hat, st.v_hat, k_new, v_new, slot, idx, st.cols, st.window, st.lse,
                            st.o, term_out=term, mass_out=mass)
        fl.kv_residual_dequant_kv((ck, sk, zk), (cv, sv, zv), idx, bits, st.group, st.k_hat, st.v_hat,
                                  mode=fl.DQ_COMMIT)
        if st.tail:
            fl.kv_keep_recent(kr, idx, st.tail, cache=st.k_hat)
            fl.kv_keep_recent(vr, idx, st.tail, cache=st.v_hat)
        if st.v16 is not None:
            fl.kv_f16_rows(st.v_hat, idx, out=st.v16)
    st.term, st.mass, st.slot_prev = term, mass, slot
    st.cand = idx
    if keep:   # (k_new / v_new are None when the loop committed straight into the caches)
        return dict(idx=idx, slot=slot, key=key, codes_k=ck, scale_k=sk, zero_k=zk, codes_v=cv,
                    scale_v=sv, zero_v=zv, k_new=k_new, v_new=v_new)
    return None


def prune_list(st: LayerState, qr, t_next, n_sink):
    """Shrink the column lists to the sinks plus t_next entries after the loop whose queries are qr."""
    st.cols, _ = fl.prune_columns(qr, st.k_hat, st.cand, st.cols, st.lse, n_sink, t_next)
    st.term = st.mass = None   # the stored add terms cover the old lists: the next loop recomputes
