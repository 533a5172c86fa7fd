"""Seeded input generation for verify-step workloads.

Every random array comes from numpy's Philox counter-based generator keyed by
(seed, stream, index), so any slab (one sequence's Q block, one (sequence,
kv-head) K or V slab, one logits row) can be regenerated on its own without
materialising the rest. Streams:

    0 Q   1 K   2 V   3 verifier logits   4 draft noise   5 draft sampling
    6 accept uniforms   7 resample uniforms   8 ragged parameters
    10 second noise level (chain)

A chain level adds a per-level offset (32 target level, 64 draft level).

Layouts (all C-contiguous, what the verify step consumes):
    q        bf16 bits  [B, gmax+1, Hq, D]       rows i > gamma_b are NaN
    k, v     bf16 bits  [B, Hkv, cap, D]         rows >= kv_len_b are +-1e4
    kv_len   int32      [B]                      ctx_b + gamma_b + 1
    gamma    int32      [B]
    p_logits f32 or bf16 bits [B, gmax+1, V]     rows j > gamma_b are NaN
    q_logits f32 or bf16 bits [B, gmax,   V]     rows j >= gamma_b are NaN
    drafts   int32      [B, gmax]                exact samples of softmax(q row)
    u_acc    fp32       [B, gmax]
    u_res    fp32       [B, gmax+1]
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

from .configs import ChainShape, VerifyShape

S_Q, S_K, S_V, S_P, S_NOISE, S_DRAFT, S_UACC, S_URES, S_RAGGED = range(9)
S_NOISE2 = 10
LEVEL_TARGET = 32
LEVEL_DRAFT = 64

BF16_NAN = np.uint16(0x7FC0)
BF16_POS_1E4 = np.uint16(0x461C)
BF16_NEG_1E4 = np.uint16(0xC61C)


def _gen(seed: int, stream: int, index: int = 0) -> np.random.Generator:
    key = (int(seed) << 64) | (int(stream) << 40) | int(index)
    return np.random.Generator(np.random.Philox(key=key))


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def bf16_bits_from_f32(x) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even); return the bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def f32_from_bf16_bits(bits) -> np.ndarray:
    """Widen bf16 bit patterns to the fp32 values they encode (exact)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def ragged_params(shape: VerifyShape):
    """Per-sequence (ctx_b, gamma_b, sigma_b) for a shape."""
    B = shape.B
    rng = _gen(shape.seed, S_RAGGED)
    lo, hi = shape.ctx
    ctx = rng.integers(lo, hi + 1, size=B) if lo < hi else np.full(B, lo)
    lo, hi = shape.gamma
    gam = rng.integers(lo, hi + 1, size=B) if lo < hi else np.full(B, lo)
    lo, hi = shape.noise
    sig = rng.uniform(lo, hi, size=B) if lo < hi else np.full(B, float(lo))
    return ctx.astype(np.int32), gam.astype(np.int32), sig.astype(np.float64)


def _garbage(rows: int, D: int) -> np.ndarray:
    """Finite filler (+-1e4 in bf16) for cache rows that hold no valid entry."""
    out = np.empty((rows, D), dtype=np.uint16)
    idx = np.add.outer(np.arange(rows), np.arange(D)) & 1
    out[...] = np.where(idx == 0, BF16_POS_1E4, BF16_NEG_1E4)
    return out


def kv_slab(seed: int, b: int, g: int, which: str, kv_len_b: int, cap: int, D: int,
            level: int = 0) -> np.ndarray:
    """K ('k') or V ('v') slab of sequence b, kv-head g: bf16 bits [cap, D]."""
    stream = (S_K if which == "k" else S_V) + level
    out = np.empty((cap, D), dtype=np.uint16)
    n = int(kv_len_b)
    vals = _gen(seed, stream, (b << 8) | g).standard_normal(n * D, dtype=np.float32)
    out[:n] = bf16_bits_from_f32(vals).reshape(n, D)
    if n < cap:
        out[n:] = _garbage(cap - n, D)
    return out


def q_block(seed: int, b: int, gamma_b: int, gmax: int, Hq: int, D: int, level: int = 0) -> np.ndarray:
    """Query rows of sequence b: bf16 bits [gmax+1, Hq, D]; padding rows NaN."""
    out = np.full((gmax + 1, Hq, D), BF16_NAN, dtype=np.uint16)
    n = int(gamma_b) + 1
    vals = _gen(seed, S_Q + level, b).standard_normal(n * Hq * D, dtype=np.float32)
    out[:n] = bf16_bits_from_f32(vals).reshape(n, Hq, D)
    return out


def _normal_row(seed, stream, b, j, V, sigma) -> np.ndarray:
    x = _gen(seed, stream, (b << 8) | j).standard_normal(V, dtype=np.float32)
    return (x * np.float32(sigma)).astype(np.float32)


def _gumbel_argmax(seed, stream, b, j, logits_seen: np.ndarray) -> int:
    """Exact sample of softmax(logits_seen) by the Gumbel-max construction."""
    e = _gen(seed, stream, (b << 8) | j).standard_exponential(logits_seen.shape[0])
    e = np.maximum(e, np.finfo(np.float64).tiny)
    return int(np.argmax(logits_seen.astype(np.float64) - np.log(e)))


def _store(vals_f32: np.ndarray, dtype: str):
    """Return (stored array in the logits dtype, fp32 values as stored)."""
    if dtype == "bf16":
        bits = bf16_bits_from_f32(vals_f32)
        return bits, f32_from_bf16_bits(bits)
    v = np.ascontiguousarray(vals_f32, dtype=np.float32)
    return v, v


def logits_rows(shape: VerifyShape, b: int, gamma_b: int, sigma_b: float, level: int = 0):
    """Verifier/draft logits rows and drafts of sequence b.

    Returns (p_store [gmax+1, V], q_store [gmax, V], drafts [gmax] int32).
    """
    V, gmax = shape.V, shape.gmax
    if shape.logits == "bf16":
        p_store = np.full((gmax + 1, V), BF16_NAN, dtype=np.uint16)
        q_store = np.full((gmax, V), BF16_NAN, dtype=np.uint16)
    else:
        p_store = np.full((gmax + 1, V), np.nan, dtype=np.float32)
        q_store = np.full((gmax, V), np.nan, dtype=np.float32)
    drafts = np.zeros(gmax, dtype=np.int32)
    for j in range(int(gamma_b) + 1):
        zp = _normal_row(shape.seed, S_P + level, b, j, V, shape.p_sigma)
        p_store[j], _ = _store(zp, shape.logits)
        if j < gamma_b:
            zq = (zp + _normal_row(shape.seed, S_NOISE + level, b, j, V, sigma_b)).astype(np.float32)
            q_store[j], seen = _store(zq, shape.logits)
            drafts[j] = _gumbel_argmax(shape.seed, S_DRAFT + level, b, j, seen)
    return p_store, q_store, drafts


def uniforms(seed: int, b: int, gmax: int, level: int = 0):
    u_acc = _gen(seed, S_UACC + level, b).random(gmax, dtype=np.float32)
    u_res = _gen(seed, S_URES + level, b).random(gmax + 1, dtype=np.float32)
    return u_acc, u_res


@dataclass
class LevelInputs:
    """Host arrays for one verify step at one level."""

    shape: object
    q: np.ndarray
    k: np.ndarray | None
    v: np.ndarray | None
    kv_len: np.ndarray
    gamma: np.ndarray
    mask: np.ndarray | None
    p_logits: np.ndarray
    q_logits: np.ndarray
    drafts: np.ndarray
    u_acc: np.ndarray
    u_res: np.ndarray
    scale: float
    sigma: np.ndarray = field(default=None)
    ctx: np.ndarray = field(default=None)

    @property
    def B(self):
        return self.kv_len.shape[0]


def _materialise_kv(seed, kv_len, Hkv, cap, D, level, threads):
    B = kv_len.shape[0]
    k = np.empty((B, Hkv, cap, D), dtype=np.uint16)
    v = np.empty((B, Hkv, cap, D), dtype=np.uint16)

    def job(bg):
        b, g = divmod(bg, Hkv)
        k[b, g] = kv_slab(seed, b, g, "k", int(kv_len[b]), cap, D, level)
        v[b, g] = kv_slab(seed, b, g, "v", int(kv_len[b]), cap, D, level)

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(job, range(B * Hkv)))
    return k, v


def level_inputs(shape: VerifyShape, kv: bool = True, logits: bool = True,
                 threads: int | None = None) -> LevelInputs:
    """All inputs of one verify step for `shape` (seeded by shape.seed)."""
    threads = threads or _threads()
    B, gmax = shape.B, shape.gmax
    ctx, gam, sig = ragged_params(shape)
    kv_len = (ctx + gam + 1).astype(np.int32)
    cap = shape.cap
    if int(kv_len.max()) > cap:
        raise ValueError("capacity too small for the drawn lengths")
    q = np.empty((B, gmax + 1, shape.Hq, shape.D), dtype=np.uint16)
    for b in range(B):
        q[b] = q_block(shape.seed, b, int(gam[b]), gmax, shape.Hq, shape.D)
    k = v = None
    if kv:
        k, v = _materialise_kv(shape.seed, kv_len, shape.Hkv, cap, shape.D, 0, threads)
    ldt = np.uint16 if shape.logits == "bf16" else np.float32
    p_l = np.empty((B, gmax + 1, shape.V), dtype=ldt)
    q_l = np.empty((B, gmax, shape.V), dtype=ldt)
    drafts = np.zeros((B, gmax), dtype=np.int32)
    if logits:
        def job(b):
            p_l[b], q_l[b], drafts[b] = logits_rows(shape, b, int(gam[b]), float(sig[b]))

        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(job, range(B)))
    u_acc = np.empty((B, gmax), dtype=np.float32)
    u_res = np.empty((B, gmax + 1), dtype=np.float32)
    for b in range(B):
        u_acc[b], u_res[b] = uniforms(shape.seed, b, gmax)
    return LevelInputs(
        shape=shape, q=q, k=k, v=v, kv_len=kv_len, gamma=gam.astype(np.int32), mask=None,
        p_logits=p_l, q_logits=q_l, drafts=drafts, u_acc=u_acc, u_res=u_res,
        scale=float(1.0 / np.sqrt(shape.D)), sigma=sig, ctx=ctx,
    )


def chain_inputs(shape: ChainShape, threads: int | None = None, kv: bool = True):
    """Inputs of the three-level chain.

    Target logits z3 ~ N(0, p_sigma^2); intermediate z2 = z3 + N(0, s23^2);
    draft z1 = z2 + N(0, s12^2). The intermediate level verifies gamma_int
    drafts sampled from softmax(z1) with (p, q) = (z2, z1). The target level's
    drafts and lengths depend on the intermediate level's outcome and are
    assembled by the caller; this returns every array that does not.
    """
    threads = threads or _threads()
    B, V, cap, seed = shape.B, shape.V, shape.cap, shape.seed
    gi, gt = shape.gamma_int, shape.gamma_tgt
    z3 = np.empty((B, gi + 1, V), dtype=np.float32)
    z2 = np.empty((B, gi + 1, V), dtype=np.float32)
    z1 = np.full((B, gi, V), np.nan, dtype=np.float32)
    drafts = np.zeros((B, gi), dtype=np.int32)

    def job(b):
        for j in range(gi + 1):
            z3[b, j] = _normal_row(seed, S_P, b, j, V, shape.p_sigma)
            z2[b, j] = (z3[b, j] + _normal_row(seed, S_NOISE, b, j, V, shape.sigma_int_tgt)).astype(np.float32)
            if j < gi:
                z1[b, j] = (z2[b, j] + _normal_row(seed, S_NOISE2, b, j, V, shape.sigma_draft_int)).astype(np.float32)
                drafts[b, j] = _gumbel_argmax(seed, S_DRAFT, b, j, z1[b, j])

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(job, range(B)))

    def level(hq, hkv, d, gamma, lvl):
        kvl = np.full(B, shape.ctx + gamma + 1, dtype=np.int32)
        q = np.stack([q_block(seed, b, gamma, gamma, hq, d, lvl) for b in range(B)])
        k = v = None
        if kv:
            k, v = _materialise_kv(seed, kvl, hkv, cap, d, lvl, threads)
        return q, k, v, kvl

    out = {}
    qi, ki, vi, kvl_i = level(*shape.inter, gi, 0)
    ua_i = np.empty((B, gi), dtype=np.float32)
    ur_i = np.empty((B, gi + 1), dtype=np.float32)
    ua_t = np.empty((B, gt), dtype=np.float32)
    ur_t = np.empty((B, gt + 1), dtype=np.float32)
    for b in range(B):
        ua_i[b], ur_i[b] = uniforms(seed, b, gi, 0)
        ua_t[b], ur_t[b] = uniforms(seed, b, gt, LEVEL_TARGET)
    out["inter"] = LevelInputs(
        shape=shape, q=qi, k=ki, v=vi, kv_len=kvl_i, gamma=np.full(B, gi, dtype=np.int32), mask=None,
        p_logits=z2, q_logits=z1, drafts=drafts, u_acc=ua_i, u_res=ur_i,
        scale=float(1.0 / np.sqrt(shape.inter[2])),
    )
    # Target level: Q/K/V for the widest draft window (gamma_tgt); the real
    # per-sequence window gamma3_b <= gamma_tgt shortens kv_len at run time.
    hq, hkv, d = shape.target
    qt = np.stack([q_block(seed, b, gt, gt, hq, d, LEVEL_TARGET) for b in range(B)])
    kt = vt = None
    if kv:
        base_len = np.full(B, shape.ctx + gt + 1, dtype=np.int32)
        kt, vt = _materialise_kv(seed, base_len, hkv, cap, d, LEVEL_TARGET, threads)
    out["target"] = dict(q=qt, k=kt, v=vt, p_logits=np.ascontiguousarray(z3[:, : gt + 1]),
                         u_acc=ua_t, u_res=ur_t, scale=float(1.0 / np.sqrt(d)))
    # Draft level: one decode-attention call (gamma = 0) per drafted token.
    hq, hkv, d = shape.draft
    qd, kd, vd, kvl_d = level(hq, hkv, d, 0, LEVEL_DRAFT)
    out["draft"] = dict(q=qd, k=kd, v=vd, kv_len=kvl_d, scale=float(1.0 / np.sqrt(d)))
    out["z"] = (z1, z2, z3)
    return out
