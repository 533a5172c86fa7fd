"""MI355X (gfx950) verify step of multi-level speculative decoding.

The compute lives in libspecrouter.so (hand-written HIP kernels behind a C
ABI, declared in include/specrouter.h) together with the host-side chain
scheduler (include/specrouter_sched.h) and an HBM read-bandwidth probe
(include/specrouter_probe.h); this package holds their sources, the
build script and a thin ctypes binding with the same function names as the C
entry points.
"""

from . import _lib
from ._lib import (
    SR_BF16,
    SR_ESCRATCH,
    SR_F32,
    AcceptBuffers,
    ChainScheduler,
    attention_workspace,
    load,
    specrouter_abi_version,
    specrouter_accept_and_diverge,
    specrouter_accept_and_diverge_sampled,
    specrouter_accept_and_rollback,
    specrouter_accept_and_rollback_noalloc,
    specrouter_accept_workspace_size,
    specrouter_chain_consensus,
    specrouter_chain_window,
    specrouter_hbm_read_probe,
    specrouter_kv_append,
    specrouter_kv_compact,
    specrouter_rollback,
    specrouter_status_string,
    specrouter_verify_attention,
    specrouter_verify_attention_workspace_size,
)

__all__ = [
    "SR_BF16",
    "SR_ESCRATCH",
    "SR_F32",
    "AcceptBuffers",
    "ChainScheduler",
    "attention_workspace",
    "load",
    "specrouter_abi_version",
    "specrouter_accept_and_diverge",
    "specrouter_accept_and_diverge_sampled",
    "specrouter_accept_and_rollback",
    "specrouter_accept_and_rollback_noalloc",
    "specrouter_accept_workspace_size",
    "specrouter_chain_consensus",
    "specrouter_chain_window",
    "specrouter_hbm_read_probe",
    "specrouter_kv_append",
    "specrouter_kv_compact",
    "specrouter_rollback",
    "specrouter_status_string",
    "specrouter_verify_attention",
    "specrouter_verify_attention_workspace_size",
]
