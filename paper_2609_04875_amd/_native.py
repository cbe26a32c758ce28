"""ctypes binding of libpgsr.so (the C ABI in include/pgsr.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  Importing this module fails loudly when the library is not built;
there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
# PGSR_LIB may name another build of the same library (e.g. a variant built
# with different compile-time options); the default is the in-tree build.
LIB_PATH = os.environ.get("PGSR_LIB") or os.path.join(_PKG, "lib", "libpgsr.so")

OK, EINVAL, ERANGE, ENOMEM, EUNSUPPORTED, EHIP, ENOENT = range(7)
STATIC_SCRATCH_BYTES = 64 << 20      # PGSR_STATIC_SCRATCH_BYTES
F32, BF16, FP8_E4M3 = 0, 1, 2
COMMIT, POISON = 1, 2

EXPORTS = (
    "pgsr_last_error", "pgsr_abi_version", "pgsr_pool_create", "pgsr_pool_destroy",
    "pgsr_pool_refresh", "pgsr_seq_len", "pgsr_free_blocks", "pgsr_workspace_bytes",
    "pgsr_kv_crop", "pgsr_kv_fork", "pgsr_replay_prefill", "pgsr_replay_prefill_static",
    "pgsr_restore_replay_prefill",
    "pgsr_full_reset_prefill", "pgsr_gemm_bf16",
    "pgsr_pool_enable_timing", "pgsr_pool_last_times", "pgsr_pool_set_kv_scales",
    "pgsr_pool_set_prefill_kernel", "pgsr_pool_set_clock_buffer", "pgsr_pool_last_clock",
    "pgsr_graph_create", "pgsr_graph_destroy", "pgsr_graph_append", "pgsr_graph_size",
    "pgsr_graph_session_length", "pgsr_graph_kv_length_after", "pgsr_graph_locate_source",
    "pgsr_graph_taint_closure", "pgsr_graph_policy_boundaries", "pgsr_ckpt_create",
    "pgsr_ckpt_destroy", "pgsr_ckpt_register", "pgsr_ckpt_count", "pgsr_forget_plan_query",
    "pgsr_sample_workspace_bytes", "pgsr_sample_tokens", "pgsr_rmsnorm_bf16", "pgsr_rope_bf16",
    "pgsr_silu_mul_bf16",
)


class ForgetPlanC(ctypes.Structure):
    """struct pgsr_forget_plan."""
    _fields_ = [(name, ctypes.c_int64) for name in (
        "tau", "checkpoint", "boundary", "crop_len", "seq", "env_snapshot", "manifest",
        "replay_transitions", "minimal_transitions", "n_sources", "closure_size",
        "clean_artifacts", "committed_after_tau")]


class PgsrError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"pgsr status {code}: {msg}")
        self.code = code


def _load() -> ctypes.CDLL:
    # torch ships its own HIP runtime; it must be the one in the process before
    # the library is opened, so that both share one runtime (and device memory,
    # streams and events pass between them).  Opening the library first would
    # bring in the system runtime alongside torch's.
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python paper_2609_04875_amd/build.py` "
            "(or __graft_entry__.build()); there is no fallback path")
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, u32, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_float
    i32p = ctypes.POINTER(ctypes.c_int32)
    lib.pgsr_last_error.restype = ctypes.c_char_p
    lib.pgsr_last_error.argtypes = []
    lib.pgsr_abi_version.restype = ctypes.c_int
    lib.pgsr_pool_create.restype = ctypes.c_int
    lib.pgsr_pool_create.argtypes = [i32, i32, i32, i32, i32, i32, i32, i32, i32, P, P, P, P, P, P, P, P,
                                     ctypes.c_size_t, i32p, P, ctypes.POINTER(P)]
    lib.pgsr_kv_fork.restype = ctypes.c_int
    lib.pgsr_kv_fork.argtypes = [P, i32, i32p, i32p, P]
    lib.pgsr_pool_destroy.restype = ctypes.c_int
    lib.pgsr_pool_destroy.argtypes = [P]
    lib.pgsr_pool_refresh.restype = ctypes.c_int
    lib.pgsr_pool_refresh.argtypes = [P, P]
    lib.pgsr_seq_len.restype = ctypes.c_int
    lib.pgsr_seq_len.argtypes = [P, i32, i32p]
    lib.pgsr_free_blocks.restype = ctypes.c_int
    lib.pgsr_free_blocks.argtypes = [P, i32p]
    lib.pgsr_workspace_bytes.restype = ctypes.c_size_t
    lib.pgsr_workspace_bytes.argtypes = [i32, i32, i64, i32]
    lib.pgsr_kv_crop.restype = ctypes.c_int
    lib.pgsr_kv_crop.argtypes = [P, i32, i32p, i32p, u32, P]
    for name in ("pgsr_replay_prefill", "pgsr_full_reset_prefill"):
        f = getattr(lib, name)
        f.restype = ctypes.c_int
        f.argtypes = [P, i32, i32, i32p, i32p, P, P, P, P, f32, u32, ctypes.POINTER(i64), P]
    lib.pgsr_restore_replay_prefill.restype = ctypes.c_int
    lib.pgsr_restore_replay_prefill.argtypes = [P, i32, i32, i32p, i32p, i32p, P, P, P, P, f32, u32,
                                                ctypes.POINTER(i64), P]
    lib.pgsr_replay_prefill_static.restype = ctypes.c_int
    lib.pgsr_replay_prefill_static.argtypes = [P, i32, i32, i32p, i32p, P, P, P, P, f32, u32, ctypes.c_size_t,
                                               ctypes.POINTER(i64), P]
    lib.pgsr_pool_set_kv_scales.restype = ctypes.c_int
    lib.pgsr_pool_set_kv_scales.argtypes = [P, P, P]
    lib.pgsr_pool_enable_timing.restype = ctypes.c_int
    lib.pgsr_pool_enable_timing.argtypes = [P, ctypes.c_int]
    lib.pgsr_pool_last_times.restype = ctypes.c_int
    lib.pgsr_pool_last_times.argtypes = [P, ctypes.POINTER(f32), ctypes.POINTER(f32)]
    lib.pgsr_pool_set_clock_buffer.restype = ctypes.c_int
    lib.pgsr_pool_set_clock_buffer.argtypes = [P, P, ctypes.c_size_t]
    lib.pgsr_pool_last_clock.restype = ctypes.c_int
    lib.pgsr_pool_last_clock.argtypes = [P, P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64),
                                         ctypes.POINTER(i64)]
    lib.pgsr_pool_set_prefill_kernel.restype = ctypes.c_int
    lib.pgsr_pool_set_prefill_kernel.argtypes = [P, ctypes.c_int]
    lib.pgsr_gemm_bf16.restype = ctypes.c_int
    lib.pgsr_gemm_bf16.argtypes = [i32, i32, i32, P, P, P, P, P]
    lib.pgsr_sample_workspace_bytes.restype = ctypes.c_size_t
    lib.pgsr_sample_workspace_bytes.argtypes = [i32, i32]
    lib.pgsr_sample_tokens.restype = ctypes.c_int
    lib.pgsr_sample_tokens.argtypes = [i32, i32, i32, P, f32, ctypes.c_uint64, P, P, P, ctypes.c_size_t,
                                       P, P]
    lib.pgsr_rmsnorm_bf16.restype = ctypes.c_int
    lib.pgsr_rmsnorm_bf16.argtypes = [i32, i32, P, P, f32, P, P]
    lib.pgsr_rope_bf16.restype = ctypes.c_int
    lib.pgsr_rope_bf16.argtypes = [i32, i32, i32, P, P, ctypes.c_double, P]
    lib.pgsr_silu_mul_bf16.restype = ctypes.c_int
    lib.pgsr_silu_mul_bf16.argtypes = [i32, i32, P, P, P]
    # forget front-end (host only)
    i64p = ctypes.POINTER(i64)
    for name, args in (
            ("pgsr_graph_create", [i64, i64, i64, ctypes.POINTER(P)]),
            ("pgsr_graph_destroy", [P]),
            ("pgsr_graph_append", [P, i64, P, P, P, P, P, P, P, P, P, i64p]),
            ("pgsr_graph_size", [P, i64p]),
            ("pgsr_graph_session_length", [P, i64p]),
            ("pgsr_graph_kv_length_after", [P, i64, i64p]),
            ("pgsr_graph_locate_source", [P, i64, P, i64, i64p]),
            ("pgsr_graph_taint_closure", [P, P, i64, P, i64, i64p]),
            ("pgsr_graph_policy_boundaries", [P, i32, i64, P, i64, i64p]),
            ("pgsr_ckpt_create", [i64, ctypes.POINTER(P)]),
            ("pgsr_ckpt_destroy", [P]),
            ("pgsr_ckpt_register", [P, i64, i64, i64, i64, i64]),
            ("pgsr_ckpt_count", [P, i64p]),
            ("pgsr_forget_plan_query", [P, P, i64, P, i64, ctypes.POINTER(ForgetPlanC)])):
        f = getattr(lib, name)
        f.restype = ctypes.c_int
        f.argtypes = args
    return lib


lib = _load()


def check(code: int) -> None:
    if code != OK:
        raise PgsrError(code, lib.pgsr_last_error().decode())


def int32_array(values):
    values = [int(v) for v in values]
    return (ctypes.c_int32 * max(1, len(values)))(*values)
