"""ctypes binding of libspecrouter.so (the verify-step C ABI).

Argument marshalling only: every function takes torch tensors that already
live on the HIP device, checks their shapes against each other, and passes
raw pointers, sizes and the current stream to the C entry point of the same
name. All arithmetic happens in the library's kernels. A missing library or
a non-zero return code raises.
"""

from __future__ import annotations

import ctypes
import os
import re

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libspecrouter.so")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
HEADERS = [os.path.join(INCLUDE, h) for h in ("specrouter.h", "specrouter_sched.h", "specrouter_probe.h")]

SR_OK, SR_EINVAL, SR_EUNSUPPORTED, SR_EWORKSPACE, SR_ELAUNCH, SR_ESCRATCH = 0, -1, -2, -3, -4, -5
SR_F32, SR_BF16 = 0, 1
SR_ST_GAMMA, SR_ST_KVLEN, SR_ST_TOKEN, SR_ST_UNIFORM, SR_ST_ROLLBACK_GROW, SR_ST_TIMEOUT, SR_ST_CHAIN = 1, 2, 4, 8, 16, 32, 64

_c_p = ctypes.c_void_p
_c_i = ctypes.c_int
_c_i64 = ctypes.c_int64
_c_sz = ctypes.c_size_t
_c_f = ctypes.c_float
_c_d = ctypes.c_double
_c_dp = ctypes.POINTER(ctypes.c_double)
_c_ip = ctypes.POINTER(ctypes.c_int32)

class SamplingParams(ctypes.Structure):
    """specrouter_sampling: temperature (0 = greedy), top_k (0), top_p (1)."""

    _fields_ = [("temperature", ctypes.c_float), ("top_k", ctypes.c_int), ("top_p", ctypes.c_float)]


_SIGNATURES = {
    "specrouter_abi_version": (_c_i, []),
    "specrouter_status_string": (ctypes.c_char_p, [_c_i]),
    "specrouter_verify_attention_workspace_size": (_c_sz, [_c_i] * 6),
    "specrouter_verify_attention": (
        _c_i,
        [_c_p] * 7 + [_c_i] * 6 + [_c_f, _c_p, _c_sz, _c_p, _c_p],
    ),
    "specrouter_accept_workspace_size": (_c_sz, [_c_i] * 4),
    "specrouter_accept_and_diverge": (
        _c_i,
        [_c_p, _c_i64, _c_p, _c_i64, _c_i] + [_c_p] * 13 + [_c_i] * 3 + [_c_p, _c_sz, _c_p, _c_p],
    ),
    "specrouter_accept_and_diverge_sampled": (
        _c_i,
        [_c_p, _c_i64, _c_p, _c_i64, _c_i] + [_c_p] * 13 + [_c_i] * 3
        + [ctypes.POINTER(SamplingParams), _c_p, _c_sz, _c_p, _c_p],
    ),
    "specrouter_accept_and_rollback": (
        _c_i,
        [_c_p, _c_i64, _c_p, _c_i64, _c_i] + [_c_p] * 13 + [_c_i] * 3
        + [ctypes.POINTER(SamplingParams), _c_p, _c_p, _c_p, _c_i, _c_p, _c_sz, _c_p, _c_p],
    ),
    "specrouter_accept_and_rollback_noalloc": (
        _c_i,
        [_c_p, _c_i64, _c_p, _c_i64, _c_i] + [_c_p] * 13 + [_c_i] * 3
        + [ctypes.POINTER(SamplingParams), _c_p, _c_p, _c_p, _c_i, _c_p, _c_p],
    ),
    "specrouter_rollback": (_c_i, [_c_p] * 4 + [_c_i, _c_i, _c_p, _c_p]),
    "specrouter_chain_window": (_c_i, [_c_p, _c_p, _c_i, _c_i, _c_i] + [_c_p] * 5),
    "specrouter_kv_append": (_c_i, [_c_p] * 8 + [_c_i] * 5 + [_c_p, _c_p]),
    "specrouter_kv_compact": (_c_i, [_c_p] * 4 + [_c_i] * 4 + [_c_p, _c_p]),
    "specrouter_chain_consensus": (_c_i, [_c_p, _c_p, _c_p, _c_i, _c_p, _c_p, _c_i, _c_i] + [_c_p] * 6),
    "specrouter_hbm_read_probe": (_c_i, [_c_p, _c_sz, _c_p, _c_p]),
    # chain scheduler (host code; host pointers)
    "specrouter_sched_create": (_c_i, [_c_i, _c_dp, _c_i, _c_i, _c_i, _c_d, _c_d, _c_d, ctypes.POINTER(_c_p)]),
    "specrouter_sched_destroy": (None, [_c_p]),
    "specrouter_sched_observe_time": (_c_i, [_c_p, _c_i, _c_d]),
    "specrouter_sched_set_similarity": (_c_i, [_c_p, _c_i, _c_i, _c_d]),
    "specrouter_sched_observe_step": (_c_i, [_c_p, _c_i, _c_i, _c_i, _c_i, _c_ip, _c_ip,
                                             ctypes.POINTER(ctypes.c_float)]),
    "specrouter_sched_calibrate": (_c_i, [_c_p, _c_dp, _c_dp]),
    "specrouter_sched_metrics": (_c_i, [_c_p, _c_dp, _c_dp, _c_dp, ctypes.POINTER(_c_i)]),
    "specrouter_sched_effective_time": (_c_i, [_c_p, _c_ip, _c_i, _c_dp]),
    "specrouter_sched_optimal_chain": (_c_i, [_c_p, _c_ip, ctypes.POINTER(_c_i), _c_dp, ctypes.POINTER(_c_i)]),
}

_lib = None


def load() -> ctypes.CDLL:
    """Load the library (once). Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2505_07680_amd.build`"
            )
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def header_functions() -> list[str]:
    """Names of the functions declared in include/*.h."""
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names.update(re.findall(r"\b(specrouter_\w+)\s*\(", text))
    return sorted(names)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(rc: int, what: str) -> None:
    if rc != SR_OK:
        msg = load().specrouter_status_string(rc).decode()
        raise RuntimeError(f"{what} failed: {rc} ({msg})")


def _dev(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("all tensors must be on the HIP device")


def _i32(t, name):
    if t is not None and t.dtype != torch.int32:
        raise TypeError(f"{name} must be int32")


def logits_dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return SR_F32
    if t.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        return SR_BF16
    raise TypeError("logits must be float32 or bf16 (bfloat16 or 16-bit bit patterns)")


def specrouter_abi_version() -> int:
    return load().specrouter_abi_version()


def specrouter_status_string(code: int) -> str:
    return load().specrouter_status_string(code).decode()


def specrouter_verify_attention_workspace_size(B, gamma_max, Hq, Hkv, D, L_cap) -> int:
    return load().specrouter_verify_attention_workspace_size(B, gamma_max, Hq, Hkv, D, L_cap)


def specrouter_verify_attention(q, k_cache, v_cache, cache_mask, kv_len, gamma, out, scale,
                                workspace=None, status=None):
    """q [B, gmax+1, Hq, D] bf16; k/v [B, Hkv, L_cap, D] bf16; out [B, gmax+1, Hq, D] fp32."""
    _dev(q, k_cache, v_cache, cache_mask, kv_len, gamma, out, workspace, status)
    _i32(kv_len, "kv_len")
    _i32(gamma, "gamma")
    B, G1, Hq, D = q.shape
    Hkv, L_cap = k_cache.shape[1], k_cache.shape[2]
    if k_cache.shape != (B, Hkv, L_cap, D) or v_cache.shape != k_cache.shape:
        raise ValueError("k_cache/v_cache must be [B, Hkv, L_cap, D]")
    if out.shape != (B, G1, Hq, D) or out.dtype != torch.float32:
        raise ValueError("out must be fp32 [B, gamma_max+1, Hq, D]")
    if q.element_size() != 2 or k_cache.element_size() != 2 or v_cache.element_size() != 2:
        raise TypeError("q, k_cache, v_cache must hold bf16")
    for t in (q, k_cache, v_cache, out):
        if not t.is_contiguous():
            raise ValueError("q, k_cache, v_cache and out must be contiguous")
    if cache_mask is not None and (cache_mask.shape != (B, L_cap) or cache_mask.element_size() != 1
                                   or not cache_mask.is_contiguous()):
        raise ValueError("cache_mask must be u8 [B, L_cap]")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    rc = load().specrouter_verify_attention(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(cache_mask), _ptr(kv_len), _ptr(gamma), _ptr(out),
        B, G1 - 1, Hq, Hkv, D, L_cap, float(scale), _ptr(workspace), ws_bytes, _ptr(status), _stream(),
    )
    _check(rc, "specrouter_verify_attention")
    return out


def specrouter_accept_workspace_size(B, gamma_max, V, logits_dtype) -> int:
    return load().specrouter_accept_workspace_size(B, gamma_max, V, logits_dtype)


def _row_view(t, rows, V, name):
    if t.dim() != 3 or t.shape[1] < rows or t.shape[2] != V or t.stride(2) != 1 or t.stride(1) != V:
        raise ValueError(f"{name} must be [B, >= {rows}, V] with contiguous rows")
    return t.stride(0)


def specrouter_accept_and_diverge(p_logits, q_logits, draft_tokens, gamma, u_accept, u_resample,
                                  kv_len, accept_len, out_tokens, new_len, accept_prob, p_tok,
                                  q_tok, kl, tv, workspace, status=None):
    """p_logits [B, gmax+1, V]; q_logits [B, gmax, V] (rows contiguous, batch stride free)."""
    _accept(p_logits, q_logits, draft_tokens, gamma, u_accept, u_resample, kv_len, accept_len, out_tokens,
            new_len, accept_prob, p_tok, q_tok, kl, tv, workspace, status, None)


def specrouter_accept_and_diverge_sampled(p_logits, q_logits, draft_tokens, gamma, u_accept, u_resample,
                                          kv_len, accept_len, out_tokens, new_len, accept_prob, p_tok,
                                          q_tok, kl, tv, workspace, status=None, temperature=1.0, top_k=0,
                                          top_p=1.0):
    """As specrouter_accept_and_diverge under softmax(logits / temperature);
    temperature 0 is greedy decoding (u_accept and u_resample may be None)."""
    _accept(p_logits, q_logits, draft_tokens, gamma, u_accept, u_resample, kv_len, accept_len, out_tokens,
            new_len, accept_prob, p_tok, q_tok, kl, tv, workspace, status,
            SamplingParams(float(temperature), int(top_k), float(top_p)))


def specrouter_accept_and_rollback(p_logits, q_logits, draft_tokens, gamma, u_accept, u_resample, kv_len,
                                   accept_len, out_tokens, new_len, accept_prob, p_tok, q_tok, kl, tv,
                                   cache_kv_len, cache_mask, phys_len, workspace, status=None, temperature=1.0,
                                   L_cap=None, top_k=0, top_p=1.0):
    """specrouter_accept_and_diverge_sampled, then specrouter_rollback of
    cache_kv_len / cache_mask to the accepted lengths, in one call."""
    _dev(cache_kv_len, cache_mask, phys_len)
    _i32(cache_kv_len, "cache_kv_len")
    B = out_tokens.shape[0]
    if cache_kv_len.shape != (B,):
        raise ValueError("cache_kv_len must be [B]")
    if cache_mask is not None:
        if cache_mask.shape[0] != B or not cache_mask.is_contiguous():
            raise ValueError("cache_mask must be contiguous [B, L_cap]")
        L_cap = cache_mask.shape[1]
    if L_cap is None:
        raise ValueError("L_cap is required when cache_mask is None")
    _accept(p_logits, q_logits, draft_tokens, gamma, u_accept, u_resample, kv_len, accept_len, out_tokens,
            new_len, accept_prob, p_tok, q_tok, kl, tv, workspace, status,
            SamplingParams(float(temperature), int(top_k), float(top_p)),
            rollback=(cache_kv_len, cache_mask, phys_len, int(L_cap)))


def specrouter_accept_and_rollback_noalloc(p_logits, q_logits, draft_tokens, gamma, u_accept, u_resample, kv_len,
                                           accept_len, out_tokens, new_len, accept_prob, p_tok, q_tok, kl, tv,
                                           cache_kv_len, cache_mask, phys_len, status=None, temperature=1.0,
                                           L_cap=None, top_k=0, top_p=1.0):
    """specrouter_accept_and_rollback with the library's own fixed device
    array as the workspace (no workspace argument, nothing allocated)."""
    _dev(cache_kv_len, cache_mask, phys_len)
    _i32(cache_kv_len, "cache_kv_len")
    B = out_tokens.shape[0]
    if cache_kv_len.shape != (B,):
        raise ValueError("cache_kv_len must be [B]")
    if cache_mask is not None:
        if cache_mask.shape[0] != B or not cache_mask.is_contiguous():
            raise ValueError("cache_mask must be contiguous [B, L_cap]")
        L_cap = cache_mask.shape[1]
    if L_cap is None:
        raise ValueError("L_cap is required when cache_mask is None")
    _accept(p_logits, q_logits, draft_tokens, gamma, u_accept, u_resample, kv_len, accept_len, out_tokens,
            new_len, accept_prob, p_tok, q_tok, kl, tv, None, status,
            SamplingParams(float(temperature), int(top_k), float(top_p)),
            rollback=(cache_kv_len, cache_mask, phys_len, int(L_cap)), noalloc=True)


def _accept(p_logits, q_logits, draft_tokens, gamma, u_accept, u_resample, kv_len, accept_len, out_tokens,
            new_len, accept_prob, p_tok, q_tok, kl, tv, workspace, status, sampling, rollback=None, noalloc=False):
    tensors = (p_logits, q_logits, draft_tokens, gamma, u_accept, u_resample, kv_len, accept_len,
               out_tokens, new_len, accept_prob, p_tok, q_tok, kl, tv, workspace, status)
    _dev(*tensors)
    for t, n in ((draft_tokens, "draft_tokens"), (gamma, "gamma"), (kv_len, "kv_len"),
                 (accept_len, "accept_len"), (out_tokens, "out_tokens"), (new_len, "new_len")):
        _i32(t, n)
    B, G1 = out_tokens.shape
    gmax = G1 - 1
    V = p_logits.shape[2]
    code = logits_dtype_code(p_logits)
    ps = _row_view(p_logits, G1, V, "p_logits")
    qs = 0
    if gmax > 0:
        if logits_dtype_code(q_logits) != code:
            raise TypeError("p_logits and q_logits must share a dtype")
        qs = _row_view(q_logits, gmax, V, "q_logits")
    if (u_resample is not None and u_resample.shape != (B, G1)) or (
            gmax > 0 and u_accept is not None and u_accept.shape != (B, gmax)):
        raise ValueError("u_accept [B, gmax] and u_resample [B, gmax+1] expected")
    for t in (accept_prob, p_tok, q_tok, kl, tv):
        if t is not None and (t.shape != (B, gmax) or t.dtype != torch.float32):
            raise ValueError("float outputs must be fp32 [B, gamma_max]")
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    common = (_ptr(p_logits), ps, _ptr(q_logits), qs, code, _ptr(draft_tokens), _ptr(gamma),
              _ptr(u_accept), _ptr(u_resample), _ptr(kv_len), _ptr(accept_len), _ptr(out_tokens),
              _ptr(new_len), _ptr(accept_prob), _ptr(p_tok), _ptr(q_tok), _ptr(kl), _ptr(tv),
              B, gmax, V, None if sampling is None else ctypes.byref(sampling))
    if noalloc:
        rkv, rmask, rphys, L_cap = rollback
        rc = load().specrouter_accept_and_rollback_noalloc(*common, _ptr(rkv), _ptr(rmask), _ptr(rphys), L_cap,
                                                           _ptr(status), _stream())
        _check(rc, "specrouter_accept_and_rollback_noalloc")
        return
    if rollback is not None:
        rkv, rmask, rphys, L_cap = rollback
        rc = load().specrouter_accept_and_rollback(*common, _ptr(rkv), _ptr(rmask), _ptr(rphys), L_cap,
                                                   _ptr(workspace), ws_bytes, _ptr(status), _stream())
        _check(rc, "specrouter_accept_and_rollback")
        return
    rc = load().specrouter_accept_and_diverge_sampled(*common, _ptr(workspace), ws_bytes, _ptr(status), _stream())
    _check(rc, "specrouter_accept_and_diverge" + ("" if sampling is None else "_sampled"))


def specrouter_hbm_read_probe(buf, sink=None):
    """Stream the bytes of the contiguous device tensor `buf` once (the read
    bandwidth probe); `sink` is an optional one-element int32 device tensor."""
    _dev(buf, sink)
    if not buf.is_contiguous():
        raise ValueError("buf must be contiguous")
    rc = load().specrouter_hbm_read_probe(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink), _stream())
    _check(rc, "specrouter_hbm_read_probe")


def specrouter_rollback(kv_len, cache_mask, new_len, phys_len=None, status=None, L_cap=None):
    _dev(kv_len, cache_mask, new_len, phys_len, status)
    _i32(kv_len, "kv_len")
    _i32(new_len, "new_len")
    B = kv_len.shape[0]
    if cache_mask is not None:
        if cache_mask.shape[0] != B or not cache_mask.is_contiguous():
            raise ValueError("cache_mask must be contiguous [B, L_cap]")
        L_cap = cache_mask.shape[1]
    if L_cap is None:
        raise ValueError("L_cap is required when cache_mask is None")
    rc = load().specrouter_rollback(_ptr(kv_len), _ptr(cache_mask), _ptr(new_len), _ptr(phys_len),
                                    B, int(L_cap), _ptr(status), _stream())
    _check(rc, "specrouter_rollback")


def specrouter_chain_window(accept_len, out_tokens, gamma_cap, gamma_next, drafts_next, ctx_len=None,
                            kv_len_next=None):
    """accept_len [B], out_tokens [B, gmax+1] of the level below -> gamma_next [B],
    drafts_next [B, gamma_cap] (and kv_len_next [B] from ctx_len [B])."""
    _dev(accept_len, out_tokens, gamma_next, drafts_next, ctx_len, kv_len_next)
    for t, n in ((accept_len, "accept_len"), (out_tokens, "out_tokens"), (gamma_next, "gamma_next"),
                 (drafts_next, "drafts_next"), (ctx_len, "ctx_len"), (kv_len_next, "kv_len_next")):
        _i32(t, n)
    B, G1 = out_tokens.shape
    if drafts_next.shape != (B, gamma_cap) or gamma_next.shape != (B,) or accept_len.shape != (B,):
        raise ValueError("accept_len [B], gamma_next [B] and drafts_next [B, gamma_cap] expected")
    rc = load().specrouter_chain_window(_ptr(accept_len), _ptr(out_tokens), B, G1 - 1, int(gamma_cap),
                                        _ptr(ctx_len), _ptr(gamma_next), _ptr(drafts_next), _ptr(kv_len_next),
                                        _stream())
    _check(rc, "specrouter_chain_window")


def specrouter_chain_consensus(ctx_len, k_lower, out_lower, k_upper, out_upper, len_upper, len_lower, pending,
                               n_pending, status=None):
    """Rows each level keeps after a two-level verify and the pending tokens."""
    _dev(ctx_len, k_lower, out_lower, k_upper, out_upper, len_upper, len_lower, pending, n_pending, status)
    for t in (ctx_len, k_lower, out_lower, k_upper, out_upper, len_upper, len_lower, pending, n_pending):
        _i32(t, "chain tensor")
    B = ctx_len.shape[0]
    if pending.shape != (B, 2) or out_lower.shape[0] != B or out_upper.shape[0] != B:
        raise ValueError("pending [B, 2], out_lower [B, gl+1], out_upper [B, gu+1] expected")
    rc = load().specrouter_chain_consensus(_ptr(ctx_len), _ptr(k_lower), _ptr(out_lower), out_lower.shape[1] - 1,
                                           _ptr(k_upper), _ptr(out_upper), out_upper.shape[1] - 1, B,
                                           _ptr(len_upper), _ptr(len_lower), _ptr(pending), _ptr(n_pending),
                                           _ptr(status), _stream())
    _check(rc, "specrouter_chain_consensus")


def specrouter_kv_append(k_new, v_new, gamma, k_cache, v_cache, cache_mask, kv_len, shared_len=None, status=None):
    """k_new/v_new [B, gmax+1, Hkv, D] bf16 -> k_cache/v_cache [B, Hkv, L_cap, D] at each cursor."""
    _dev(k_new, v_new, gamma, k_cache, v_cache, cache_mask, kv_len, shared_len, status)
    _i32(gamma, "gamma")
    _i32(kv_len, "kv_len")
    B, G1, Hkv, D = k_new.shape
    L_cap = k_cache.shape[2]
    if v_new.shape != k_new.shape or k_cache.shape != (B, Hkv, L_cap, D) or v_cache.shape != k_cache.shape:
        raise ValueError("k_new/v_new [B, gmax+1, Hkv, D] and k_cache/v_cache [B, Hkv, L_cap, D] expected")
    for t in (k_new, v_new, k_cache, v_cache):
        if not t.is_contiguous() or t.element_size() != 2:
            raise ValueError("K/V tensors must be contiguous bf16")
    if cache_mask is not None and (cache_mask.shape != (B, L_cap) or not cache_mask.is_contiguous()):
        raise ValueError("cache_mask must be u8 [B, L_cap]")
    rc = load().specrouter_kv_append(_ptr(k_new), _ptr(v_new), _ptr(gamma), _ptr(k_cache), _ptr(v_cache),
                                     _ptr(cache_mask), _ptr(kv_len), _ptr(shared_len), B, G1 - 1, Hkv, D, L_cap,
                                     _ptr(status), _stream())
    _check(rc, "specrouter_kv_append")


def specrouter_kv_compact(k_cache, v_cache, cache_mask, kv_len, status=None):
    _dev(k_cache, v_cache, cache_mask, kv_len, status)
    _i32(kv_len, "kv_len")
    B, Hkv, L_cap, D = k_cache.shape
    if v_cache.shape != k_cache.shape or cache_mask.shape != (B, L_cap):
        raise ValueError("k_cache/v_cache [B, Hkv, L_cap, D] and cache_mask [B, L_cap] expected")
    for t in (k_cache, v_cache, cache_mask):
        if not t.is_contiguous():
            raise ValueError("cache tensors must be contiguous")
    rc = load().specrouter_kv_compact(_ptr(k_cache), _ptr(v_cache), _ptr(cache_mask), _ptr(kv_len), B, Hkv, D, L_cap,
                                      _ptr(status), _stream())
    _check(rc, "specrouter_kv_compact")


# ----------------------------------------------------------------------------
# Buffer helpers (allocation only).

class AcceptBuffers:
    """Outputs and the self-resetting workspace of one accept-and-diverge call shape."""

    def __init__(self, B: int, gamma_max: int, V: int, logits_dtype: int, device="cuda"):
        i32 = dict(dtype=torch.int32, device=device)
        f32 = dict(dtype=torch.float32, device=device)
        self.accept_len = torch.empty(B, **i32)
        self.out_tokens = torch.empty(B, gamma_max + 1, **i32)
        self.new_len = torch.empty(B, **i32)
        self.accept_prob = torch.empty(B, gamma_max, **f32)
        self.p_tok = torch.empty(B, gamma_max, **f32)
        self.q_tok = torch.empty(B, gamma_max, **f32)
        self.kl = torch.empty(B, gamma_max, **f32)
        self.tv = torch.empty(B, gamma_max, **f32)
        n = specrouter_accept_workspace_size(B, gamma_max, V, logits_dtype)
        if n == 0:
            raise RuntimeError("accept workspace query failed")
        self.workspace = torch.zeros(n, dtype=torch.uint8, device=device)  # zero before first use
        self.status = torch.zeros(1, **i32)


def attention_workspace(B, gamma_max, Hq, Hkv, D, L_cap, device="cuda"):
    n = specrouter_verify_attention_workspace_size(B, gamma_max, Hq, Hkv, D, L_cap)
    return None if n == 0 else torch.zeros(n, dtype=torch.uint8, device=device)


# ----------------------------------------------------------------------------
# Chain scheduler (host code). Inputs are copied into host arrays; the
# arithmetic is the library's.

def _host(t, dtype):
    """A contiguous host numpy array of `t` (a torch tensor on any device, or
    array-like) with the given numpy dtype."""
    import numpy as np

    if isinstance(t, torch.Tensor):
        t = t.detach().cpu().numpy()
    return np.ascontiguousarray(np.asarray(t), dtype=dtype)


def _as_ptr(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def specrouter_sched_create(capability, target, window, max_levels=None, ema_time=0.2, ema_sim=0.1,
                            prior_weight=1.0):
    import numpy as np

    cap = _host(capability, np.float64)
    n = int(cap.shape[0])
    h = ctypes.c_void_p()
    rc = load().specrouter_sched_create(n, _as_ptr(cap, ctypes.c_double), int(target), int(window),
                                        n if max_levels is None else int(max_levels), float(ema_time),
                                        float(ema_sim), float(prior_weight), ctypes.byref(h))
    _check(rc, "specrouter_sched_create")
    return h


def specrouter_sched_destroy(handle) -> None:
    load().specrouter_sched_destroy(handle)


def specrouter_sched_observe_time(handle, model, seconds_per_token) -> None:
    _check(load().specrouter_sched_observe_time(handle, int(model), float(seconds_per_token)),
           "specrouter_sched_observe_time")


def specrouter_sched_set_similarity(handle, draft, verifier, simscore) -> None:
    _check(load().specrouter_sched_set_similarity(handle, int(draft), int(verifier), float(simscore)),
           "specrouter_sched_set_similarity")


def specrouter_sched_observe_step(handle, draft, verifier, gamma, accept_len, tv) -> None:
    """gamma [B], accept_len [B], tv [B, gamma_max]: the accept call's outputs
    (device tensors are copied to the host)."""
    import numpy as np

    g = _host(gamma, np.int32)
    k = _host(accept_len, np.int32)
    t = _host(tv, np.float32)
    if t.ndim != 2 or g.shape != (t.shape[0],) or k.shape != g.shape:
        raise ValueError("gamma [B], accept_len [B] and tv [B, gamma_max] expected")
    rc = load().specrouter_sched_observe_step(handle, int(draft), int(verifier), int(t.shape[0]), int(t.shape[1]),
                                              _as_ptr(g, ctypes.c_int32), _as_ptr(k, ctypes.c_int32),
                                              _as_ptr(t, ctypes.c_float))
    _check(rc, "specrouter_sched_observe_step")


def specrouter_sched_calibrate(handle):
    A, B = ctypes.c_double(), ctypes.c_double()
    _check(load().specrouter_sched_calibrate(handle, ctypes.byref(A), ctypes.byref(B)), "specrouter_sched_calibrate")
    return A.value, B.value


def specrouter_sched_metrics(handle, n_models):
    """(T [n], SimScore [n, n], (A, B), number of kept observations)."""
    import numpy as np

    T = np.empty(n_models, np.float64)
    S = np.empty((n_models, n_models), np.float64)
    c = np.empty(2, np.float64)
    n_obs = ctypes.c_int()
    _check(load().specrouter_sched_metrics(handle, _as_ptr(T, ctypes.c_double), _as_ptr(S, ctypes.c_double),
                                           _as_ptr(c, ctypes.c_double), ctypes.byref(n_obs)),
           "specrouter_sched_metrics")
    return T, S, (float(c[0]), float(c[1])), n_obs.value


def specrouter_sched_effective_time(handle, chain) -> float:
    import numpy as np

    c = _host(chain, np.int32)
    t = ctypes.c_double()
    _check(load().specrouter_sched_effective_time(handle, _as_ptr(c, ctypes.c_int32), int(c.shape[0]),
                                                  ctypes.byref(t)), "specrouter_sched_effective_time")
    return t.value


def specrouter_sched_optimal_chain(handle, n_models):
    """(chain as a list of model indices, predicted T_eff, number of candidates)."""
    import numpy as np

    out = np.empty(n_models, np.int32)
    n, cnt = ctypes.c_int(), ctypes.c_int()
    t = ctypes.c_double()
    _check(load().specrouter_sched_optimal_chain(handle, _as_ptr(out, ctypes.c_int32), ctypes.byref(n),
                                                 ctypes.byref(t), ctypes.byref(cnt)),
           "specrouter_sched_optimal_chain")
    return out[:n.value].tolist(), t.value, cnt.value


class ChainScheduler:
    """Owning wrapper of a scheduler handle (Section 4.2, Algorithm 1)."""

    def __init__(self, capability, target, window, max_levels=None, ema_time=0.2, ema_sim=0.1,
                 prior_weight=1.0):
        self.n = len(capability)
        self.handle = specrouter_sched_create(capability, target, window, max_levels, ema_time, ema_sim,
                                              prior_weight)

    def close(self):
        if self.handle is not None:
            specrouter_sched_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def observe_time(self, model, seconds_per_token):
        specrouter_sched_observe_time(self.handle, model, seconds_per_token)

    def set_similarity(self, draft, verifier, simscore):
        specrouter_sched_set_similarity(self.handle, draft, verifier, simscore)

    def observe_step(self, draft, verifier, gamma, accept_len, tv):
        specrouter_sched_observe_step(self.handle, draft, verifier, gamma, accept_len, tv)

    def calibrate(self):
        return specrouter_sched_calibrate(self.handle)

    def metrics(self):
        return specrouter_sched_metrics(self.handle, self.n)

    def effective_time(self, chain):
        return specrouter_sched_effective_time(self.handle, chain)

    def optimal_chain(self):
        return specrouter_sched_optimal_chain(self.handle, self.n)
