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
HEADER = os.path.join(os.path.dirname(HERE), "include", "specrouter.h")

SR_OK, SR_EINVAL, SR_EUNSUPPORTED, SR_EWORKSPACE, SR_ELAUNCH = 0, -1, -2, -3, -4
SR_F32, SR_BF16 = 0, 1
SR_ST_GAMMA, SR_ST_KVLEN, SR_ST_TOKEN, SR_ST_UNIFORM, SR_ST_ROLLBACK_GROW, SR_ST_TIMEOUT = 1, 2, 4, 8, 16, 32

_c_p = ctypes.c_void_p
_c_i = ctypes.c_int
_c_i64 = ctypes.c_int64
_c_sz = ctypes.c_size_t
_c_f = ctypes.c_float

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
    "specrouter_rollback": (_c_i, [_c_p] * 4 + [_c_i, _c_i, _c_p, _c_p]),
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
    """Names of the functions declared in include/specrouter.h."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(specrouter_\w+)\s*\(", text)))


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
    if u_resample.shape != (B, G1) or (gmax > 0 and u_accept.shape != (B, gmax)):
        raise ValueError("u_accept [B, gmax] and u_resample [B, gmax+1] expected")
    for t in (accept_prob, p_tok, q_tok, kl, tv):
        if t is not None and (t.shape != (B, gmax) or t.dtype != torch.float32):
            raise ValueError("float outputs must be fp32 [B, gamma_max]")
    ws_bytes = workspace.numel() * workspace.element_size()
    rc = load().specrouter_accept_and_diverge(
        _ptr(p_logits), ps, _ptr(q_logits), qs, code, _ptr(draft_tokens), _ptr(gamma),
        _ptr(u_accept), _ptr(u_resample), _ptr(kv_len), _ptr(accept_len), _ptr(out_tokens),
        _ptr(new_len), _ptr(accept_prob), _ptr(p_tok), _ptr(q_tok), _ptr(kl), _ptr(tv),
        B, gmax, V, _ptr(workspace), ws_bytes, _ptr(status), _stream(),
    )
    _check(rc, "specrouter_accept_and_diverge")


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
