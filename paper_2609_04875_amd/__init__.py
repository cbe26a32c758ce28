"""MI355X-native hot path of Provenance-Guided Selective Replay.

Restore a checkpoint by cropping a paged KV cache to the injection boundary
tau - 1 (Algorithm 1, restore step; Lemma 1), then replay the T - tau + 1
sanitized transitions as a prefix + causal prefill against the kept prefix
(Algorithm 1, replay loop; Theorem 1; Corollary 1).  The work runs in the HIP
kernels of ``lib/libpgsr.so`` behind the C ABI of ``include/pgsr.h``; this
package only allocates device memory with torch and marshals arguments.  The
forget front-end (provenance queries and checkpoint choice that yield the crop
length) is host code in the same library.
"""
from ._native import (BF16, COMMIT, EHIP, EINVAL, ENOENT, ENOMEM, EUNSUPPORTED, ERANGE, F32, FP8_E4M3,
                      OK, POISON, PgsrError)
from .frontend import CheckpointStore, ForgetPlan, ProvenanceGraph, forget_plan
from .sampling import sample_tokens, sample_workspace_bytes
from .decoder import DecoderReplay, rmsnorm, rope_, silu_mul
from .pool import KVPool, gemm_bf16, workspace_bytes
from .stack import StackedReplay

__all__ = ["KVPool", "StackedReplay", "DecoderReplay", "rmsnorm", "rope_", "silu_mul", "gemm_bf16", "workspace_bytes", "ProvenanceGraph", "CheckpointStore",
           "ForgetPlan", "forget_plan", "sample_tokens", "sample_workspace_bytes", "PgsrError", "OK", "EINVAL", "ERANGE", "ENOMEM", "EUNSUPPORTED",
           "EHIP", "ENOENT", "F32", "BF16", "FP8_E4M3", "COMMIT", "POISON"]
