"""Helpers for the GPU tests: upload seeded inputs, run one verify step through
the C ABI, and compare with the CPU reference at the parity tolerances."""

from __future__ import annotations

import numpy as np
import torch

import paper_2505_07680_amd as sr

# Parity tolerances.
ATT_ATOL, ATT_RTOL = 2e-2, 1e-2      # bf16 in, fp32 accumulate
# Relative L2 error of every (sequence, row, head) output vector. With
# Q, K, V ~ N(0, 1) the outputs are small (RMS ~0.04 at 2K keys, ~0.01 at 32K),
# so the elementwise bound above is loose there; this one is not (bf16
# probabilities in the PV products give ~1e-3).
ATT_REL_L2 = 1e-2
PROB_RTOL = 1e-5                     # accept_prob, p_tok, q_tok
DIV_RTOL, DIV_ATOL = 1e-4, 1e-7      # KL and TV (absolute floor for near-zero values)


def dev(x, device="cuda"):
    x = np.ascontiguousarray(x)
    if x.dtype == np.uint16:
        x = x.view(np.int16)
    return torch.from_numpy(x).to(device)


def host(t):
    return t.detach().cpu().numpy()


def run_attention(inp, mask=None, q=None):
    B, G1, Hq, D = inp.q.shape
    Hkv, cap = inp.k.shape[1], inp.k.shape[2]
    qd = dev(inp.q if q is None else q)
    kd, vd = dev(inp.k), dev(inp.v)
    kv = dev(inp.kv_len.astype(np.int32))
    gm = dev(inp.gamma.astype(np.int32))
    md = None if mask is None else dev(mask.astype(np.uint8))
    out = torch.full((B, G1, Hq, D), float("nan"), dtype=torch.float32, device="cuda")
    ws = sr.attention_workspace(B, G1 - 1, Hq, Hkv, D, cap)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    sr.specrouter_verify_attention(qd, kd, vd, md, kv, gm, out, inp.scale, ws, st)
    torch.cuda.synchronize()
    return host(out), int(host(st)[0])


def run_accept(p_logits, q_logits, drafts, gamma, u_acc, u_res, kv_len=None, bufs=None,
               p_dev=None, q_dev=None, temperature=None, top_k=0, top_p=1.0):
    B, G1, V = p_logits.shape if p_dev is None else p_dev.shape
    code = sr.SR_BF16 if (p_dev is None and p_logits.dtype == np.uint16) or (
        p_dev is not None and p_dev.element_size() == 2) else sr.SR_F32
    pd = dev(p_logits) if p_dev is None else p_dev
    qd = dev(q_logits) if q_dev is None else q_dev
    if bufs is None:
        bufs = sr.AcceptBuffers(B, G1 - 1, V, code)
    bufs.status.zero_()
    kvd = None if kv_len is None else dev(np.asarray(kv_len, np.int32))
    args = (pd, qd, dev(np.asarray(drafts, np.int32)), dev(np.asarray(gamma, np.int32)),
            None if u_acc is None else dev(np.asarray(u_acc, np.float32)),
            None if u_res is None else dev(np.asarray(u_res, np.float32)), kvd,
            bufs.accept_len, bufs.out_tokens, bufs.new_len if kvd is not None else None,
            bufs.accept_prob, bufs.p_tok, bufs.q_tok, bufs.kl, bufs.tv, bufs.workspace, bufs.status)
    if temperature is None and top_k == 0 and top_p == 1.0:
        sr.specrouter_accept_and_diverge(*args)
    else:
        sr.specrouter_accept_and_diverge_sampled(*args, temperature=1.0 if temperature is None else temperature,
                                                 top_k=top_k, top_p=top_p)
    torch.cuda.synchronize()
    res = dict(
        accept_len=host(bufs.accept_len), out_tokens=host(bufs.out_tokens),
        accept_prob=host(bufs.accept_prob), p_tok=host(bufs.p_tok), q_tok=host(bufs.q_tok),
        kl=host(bufs.kl), tv=host(bufs.tv), status=int(host(bufs.status)[0]),
    )
    if kvd is not None:
        res["new_len"] = host(bufs.new_len)
    return res


def run_rollback(kv_len, mask, new_len, cap):
    kv = dev(np.asarray(kv_len, np.int32))
    md = None if mask is None else dev(np.asarray(mask, np.uint8))
    phys = torch.zeros(1, dtype=torch.int32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    sr.specrouter_rollback(kv, md, dev(np.asarray(new_len, np.int32)), phys, st, L_cap=cap)
    torch.cuda.synchronize()
    return host(kv), (None if md is None else host(md)), int(host(phys)[0]), int(host(st)[0])


def check_attention(got, want, seqs=None, atol=ATT_ATOL, rtol=ATT_RTOL, rel_l2=ATT_REL_L2):
    """Elementwise |got - want| <= atol + rtol |want|, and the relative L2 error
    ||got - want|| / ||want|| of every (sequence, row, head) vector with a
    non-zero reference at most rel_l2 (a vector whose reference is zero must
    be zero). Returns the worst relative L2 error."""
    if seqs is not None:
        got, want = got[list(seqs)], want[list(seqs)]
    assert np.isfinite(got).all(), "non-finite attention output"
    err = np.abs(got - want)
    bad = err > atol + rtol * np.abs(want)
    assert not bad.any(), f"{bad.sum()} attention elements outside tolerance; max err {err.max():.3e}"
    num = np.linalg.norm(got - want, axis=-1)
    den = np.linalg.norm(want, axis=-1)
    live = den > 0
    assert (num[~live] == 0).all(), "output rows whose reference is zero are not zero"
    worst = float((num[live] / den[live]).max()) if live.any() else 0.0
    assert worst <= rel_l2, f"attention relative L2 error {worst:.3e} > {rel_l2:.0e}"
    return worst


def _close(got, want, rtol, atol=0.0):
    nan_g, nan_w = np.isnan(got), np.isnan(want)
    assert (nan_g == nan_w).all(), "NaN padding differs"
    g, w = got[~nan_w], want[~nan_w]
    with np.errstate(invalid="ignore"):
        same = g == w  # equal infinities (a KL with q = 0 where p > 0) included
        ok = same | (np.abs(g - w) <= rtol * np.abs(w) + atol)
        rel = np.where(same, 0.0, np.abs(g - w) / np.maximum(np.abs(w), 1e-30))
    return ok.all(), float(np.nanmax(rel)) if g.size else 0.0


def check_accept(got, ref, seqs=None, check_new_len=True):
    """Bit-exact lengths/tokens except reference boundary cases; float outputs
    at their tolerances. Returns (n_boundary, n_boundary_mismatches)."""
    B = ref["accept_len"].shape[0]
    seqs = list(range(B)) if seqs is None else list(seqs)
    n_bd = n_bd_mis = 0
    for b in seqs:
        same = (got["accept_len"][b] == ref["accept_len"][b]) and (
            got["out_tokens"][b] == ref["out_tokens"][b]).all()
        if check_new_len and ref.get("new_len") is not None and "new_len" in got:
            same = same and got["new_len"][b] == ref["new_len"][b]
        if ref["boundary"][b]:
            n_bd += 1
            n_bd_mis += int(not same)
        else:
            assert same, (f"sequence {b}: accept_len {got['accept_len'][b]} vs {ref['accept_len'][b]}, "
                          f"tokens {got['out_tokens'][b]} vs {ref['out_tokens'][b]}, margin {ref['margin'][b]:.3e}")
        # per-position probabilities and divergences do not depend on the decisions
        for key in ("accept_prob", "p_tok", "q_tok"):
            ok, worst = _close(got[key][b], ref[key][b], PROB_RTOL)
            assert ok, f"sequence {b}: {key} rel err {worst:.3e}"
        for key in ("kl", "tv"):
            ok, worst = _close(got[key][b], ref[key][b], DIV_RTOL, DIV_ATOL)
            assert ok, f"sequence {b}: {key} rel err {worst:.3e}"
    return n_bd, n_bd_mis
