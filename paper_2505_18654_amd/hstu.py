"""ctypes binding of libmtgr_hstu.so: the C entry points under the same names.

Argument marshalling only.  Every computation runs in the HIP kernels of the
library; torch is used for device buffers and the current stream.  Importing
this module does not need a GPU, but loading fails loudly (MtgrLibraryMissing)
when the library has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmtgr_hstu.so")

MTGR_SUCCESS = 0
MTGR_ERROR_NULL_POINTER = 1
MTGR_ERROR_INVALID_ARGUMENT = 2
MTGR_ERROR_UNSUPPORTED = 3
MTGR_ERROR_WORKSPACE_TOO_SMALL = 4
MTGR_ERROR_DEVICE = 5
MTGR_DTYPE_BF16 = 0
MTGR_DTYPE_FP32 = 1
MTGR_SEG_USER, MTGR_SEG_HIST, MTGR_SEG_RT, MTGR_SEG_CAND = 0, 1, 2, 3
MTGR_MAX_RAB_BUCKETS = 64
MTGR_MAX_HEADS = 255
MTGR_MAX_GROUPS = 127
MTGR_MAX_LD = 1 << 24
MTGR_ATTN_PLANNED = 1
MTGR_BWD_SKIP_DQ = 2
MTGR_BWD_SKIP_DKDV = 4
MTGR_BWD_KEEP_DS = 8
MTGR_BWD_DS_READY = 16
MTGR_FWD_CAND_ROWS = 32
MTGR_VALIDATE_SCRATCH_BYTES = 64
MTGR_NOALLOC_SCRATCH_BYTES = 16 * 1024 * 1024
MTGR_GEMM_NN, MTGR_GEMM_NT, MTGR_GEMM_TN = 0, 1, 2
MTGR_GEMM_EPI_NONE, MTGR_GEMM_EPI_BIAS_SILU, MTGR_GEMM_EPI_BIAS_RESIDUAL = 0, 1, 2
MTGR_EMB_KEY_EMPTY = 0xFFFFFFFFFFFFFFFF
MTGR_EMB_KEY_DELETED = 0xFFFFFFFFFFFFFFFE
MTGR_EMB_STATE_WORDS = 8
MTGR_EMB_STATE_NEXT_ROW, MTGR_EMB_STATE_FREE_TOP, MTGR_EMB_STATE_NUM_KEYS, MTGR_EMB_STATE_OVERFLOW = 0, 1, 2, 3

EXPORTED = (
    "mtgr_hstu_attn_workspace_size", "mtgr_hstu_attn_plan", "mtgr_hstu_attn_fwd", "mtgr_hstu_attn_bwd",
    "mtgr_hstu_attn_fwd_noalloc", "mtgr_hstu_attn_fwd_cached",
    "mtgr_group_layernorm_workspace_size", "mtgr_group_layernorm_fwd", "mtgr_group_layernorm_bwd",
    "mtgr_bias_silu_fwd", "mtgr_bias_silu_bwd", "mtgr_add", "mtgr_gemm_workspace_size", "mtgr_gemm_bf16",
    "mtgr_debug_validate_inputs", "mtgr_debug_clock_probe", "mtgr_status_string", "mtgr_last_error_message", "mtgr_version",
    "mtgr_embedding_init", "mtgr_embedding_dedup_workspace_size", "mtgr_embedding_dedup",
    "mtgr_embedding_lookup_workspace_size", "mtgr_embedding_lookup", "mtgr_embedding_gather",
    "mtgr_embedding_sgd_workspace_size", "mtgr_embedding_sgd", "mtgr_embedding_evict",
    "mtgr_embedding_rehash",
)


class MtgrLibraryMissing(RuntimeError):
    pass


class MtgrError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


class HstuProblem(ctypes.Structure):
    _fields_ = [
        ("num_users", ctypes.c_int32), ("max_seqlen", ctypes.c_int32),
        ("total_tokens", ctypes.c_int64), ("num_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32), ("alpha", ctypes.c_float),
        ("num_rab_buckets", ctypes.c_int32), ("flags", ctypes.c_uint32),
        ("ld_q", ctypes.c_int64), ("ld_k", ctypes.c_int64), ("ld_v", ctypes.c_int64),
        ("ld_o", ctypes.c_int64),
    ]


class GlnProblem(ctypes.Structure):
    _fields_ = [
        ("num_tokens", ctypes.c_int64), ("dim", ctypes.c_int32), ("num_groups", ctypes.c_int32),
        ("dtype", ctypes.c_int32), ("eps", ctypes.c_float),
        ("ld_x", ctypes.c_int64), ("ld_u", ctypes.c_int64), ("ld_y", ctypes.c_int64),
    ]


class EmbeddingTable(ctypes.Structure):
    _fields_ = [
        ("key_capacity", ctypes.c_int64), ("row_capacity", ctypes.c_int64), ("dim", ctypes.c_int32),
        ("dtype", ctypes.c_int32), ("keys", ctypes.c_void_p), ("key_rows", ctypes.c_void_p),
        ("values", ctypes.c_void_p), ("counts", ctypes.c_void_p), ("last_ts", ctypes.c_void_p),
        ("free_rows", ctypes.c_void_p), ("state", ctypes.c_void_p),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise MtgrLibraryMissing(
                f"{LIB_PATH} is not built; run `python -m paper_2505_18654_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32
        P = ctypes.POINTER(HstuProblem)
        G = ctypes.POINTER(GlnProblem)
        L.mtgr_hstu_attn_workspace_size.argtypes = [P, ctypes.c_int, ctypes.POINTER(sz)]
        L.mtgr_hstu_attn_plan.argtypes = [P, vp, vp, vp, vp, sz, vp]
        L.mtgr_hstu_attn_fwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.mtgr_hstu_attn_fwd_noalloc.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.mtgr_hstu_attn_fwd_cached.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, P, vp, vp, vp, vp, vp, sz,
                                                vp, sz, vp]
        L.mtgr_hstu_attn_bwd.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.mtgr_group_layernorm_workspace_size.argtypes = [G, ctypes.c_int, ctypes.POINTER(sz)]
        L.mtgr_group_layernorm_fwd.argtypes = [G, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.mtgr_group_layernorm_bwd.argtypes = [G, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.mtgr_debug_validate_inputs.argtypes = [P, vp, vp, vp, i32, vp, sz, vp]
        i64 = ctypes.c_int64
        L.mtgr_bias_silu_fwd.argtypes = [i64, i32, ctypes.c_int, vp, i64, vp, vp, i64, vp]
        L.mtgr_bias_silu_bwd.argtypes = [i64, i32, ctypes.c_int, vp, i64, vp, vp, i64, vp, i64, vp]
        L.mtgr_add.argtypes = [i64, i32, ctypes.c_int, vp, i64, vp, i64, vp, i64, vp]
        L.mtgr_debug_clock_probe.argtypes = [i32, i32, vp, ctypes.POINTER(i32), vp]
        L.mtgr_gemm_workspace_size.argtypes = [i32, i64, i64, i64, ctypes.POINTER(sz)]
        L.mtgr_gemm_bf16.argtypes = [i32, i64, i64, i64, vp, i64, vp, i64, vp, i64, i32, vp, vp, i64, vp, i64, vp,
                                     vp, sz, vp]
        E = ctypes.POINTER(EmbeddingTable)
        L.mtgr_embedding_init.argtypes = [E, vp]
        L.mtgr_embedding_dedup_workspace_size.argtypes = [i64, ctypes.POINTER(sz)]
        L.mtgr_embedding_dedup.argtypes = [i64, vp, vp, vp, vp, vp, vp, sz, vp]
        L.mtgr_embedding_lookup_workspace_size.argtypes = [i64, ctypes.POINTER(sz)]
        L.mtgr_embedding_lookup.argtypes = [E, i64, vp, vp, vp, i32, i32, vp, vp, sz, vp]
        L.mtgr_embedding_gather.argtypes = [E, i64, vp, vp, vp, i64, vp]
        L.mtgr_embedding_sgd_workspace_size.argtypes = [i64, i64, i32, ctypes.POINTER(sz)]
        L.mtgr_embedding_sgd.argtypes = [E, i64, vp, vp, vp, i64, i64, vp, vp, ctypes.c_float, vp, sz, vp]
        L.mtgr_embedding_evict.argtypes = [E, i32, ctypes.c_uint32, vp, vp]
        L.mtgr_embedding_rehash.argtypes = [E, E, vp]
        for name in EXPORTED:
            if name not in ("mtgr_status_string", "mtgr_last_error_message", "mtgr_version"):
                getattr(L, name).restype = ctypes.c_int
        L.mtgr_status_string.argtypes = [ctypes.c_int]
        L.mtgr_status_string.restype = ctypes.c_char_p
        L.mtgr_last_error_message.argtypes = []
        L.mtgr_last_error_message.restype = ctypes.c_char_p
        L.mtgr_version.argtypes = []
        L.mtgr_version.restype = i32
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != MTGR_SUCCESS:
        msg = lib().mtgr_last_error_message().decode()
        kind = lib().mtgr_status_string(status).decode()
        raise MtgrError(status, f"{kind}: {msg}")


def _ptr(x) -> Optional[int]:
    """Device (or host) address of a tensor, an int address, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ------------------------------------------------------------------ raw entry points

def mtgr_version() -> int:
    return int(lib().mtgr_version())


def mtgr_status_string(status: int) -> str:
    return lib().mtgr_status_string(status).decode()


def mtgr_last_error_message() -> str:
    return lib().mtgr_last_error_message().decode()


def mtgr_hstu_attn_workspace_size(problem: HstuProblem, backward: bool = False) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().mtgr_hstu_attn_workspace_size(ctypes.byref(problem), int(backward), ctypes.byref(out)))
    return int(out.value)


def mtgr_hstu_attn_plan(problem, offsets, seg, ts, workspace, workspace_bytes, stream=None) -> None:
    _check(lib().mtgr_hstu_attn_plan(ctypes.byref(problem), _ptr(offsets), _ptr(seg), _ptr(ts),
                                     _ptr(workspace), int(workspace_bytes), _stream(stream)))


def mtgr_hstu_attn_fwd(problem, offsets, seg, ts, q, k, v, rab, out, workspace, workspace_bytes,
                       stream=None) -> None:
    _check(lib().mtgr_hstu_attn_fwd(ctypes.byref(problem), _ptr(offsets), _ptr(seg), _ptr(ts),
                                    _ptr(q), _ptr(k), _ptr(v), _ptr(rab), _ptr(out), _ptr(workspace),
                                    int(workspace_bytes), _stream(stream)))


def mtgr_hstu_attn_fwd_cached(problem, offsets, seg, ts, q, k, v, rab, out, cache_problem, offsets_c, ts_c,
                              kc, vc, cache_plan, cache_plan_bytes, workspace, workspace_bytes,
                              stream=None) -> None:
    _check(lib().mtgr_hstu_attn_fwd_cached(
        ctypes.byref(problem), _ptr(offsets), _ptr(seg), _ptr(ts), _ptr(q), _ptr(k), _ptr(v), _ptr(rab),
        _ptr(out), None if cache_problem is None else ctypes.byref(cache_problem), _ptr(offsets_c), _ptr(ts_c), _ptr(kc), _ptr(vc),
        _ptr(cache_plan), int(cache_plan_bytes), _ptr(workspace), int(workspace_bytes), _stream(stream)))


def mtgr_hstu_attn_fwd_noalloc(problem, offsets, seg, ts, q, k, v, rab, out, stream=None) -> None:
    _check(lib().mtgr_hstu_attn_fwd_noalloc(ctypes.byref(problem), _ptr(offsets), _ptr(seg), _ptr(ts),
                                            _ptr(q), _ptr(k), _ptr(v), _ptr(rab), _ptr(out), _stream(stream)))


def mtgr_hstu_attn_bwd(problem, offsets, seg, ts, q, k, v, rab, dout, dq, dk, dv, drab, workspace,
                       workspace_bytes, stream=None) -> None:
    _check(lib().mtgr_hstu_attn_bwd(ctypes.byref(problem), _ptr(offsets), _ptr(seg), _ptr(ts),
                                    _ptr(q), _ptr(k), _ptr(v), _ptr(rab), _ptr(dout), _ptr(dq),
                                    _ptr(dk), _ptr(dv), _ptr(drab), _ptr(workspace),
                                    int(workspace_bytes), _stream(stream)))


def mtgr_group_layernorm_workspace_size(problem: GlnProblem, backward: bool = False) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().mtgr_group_layernorm_workspace_size(ctypes.byref(problem), int(backward),
                                                     ctypes.byref(out)))
    return int(out.value)


def mtgr_group_layernorm_fwd(problem, x, u, group_ids, gamma, beta, y, mean, rstd, stream=None) -> None:
    _check(lib().mtgr_group_layernorm_fwd(ctypes.byref(problem), _ptr(x), _ptr(u), _ptr(group_ids),
                                          _ptr(gamma), _ptr(beta), _ptr(y), _ptr(mean), _ptr(rstd),
                                          _stream(stream)))


def mtgr_group_layernorm_bwd(problem, dy, x, u, group_ids, gamma, mean, rstd, dx, du, dgamma, dbeta,
                             workspace=None, workspace_bytes=0, stream=None) -> None:
    _check(lib().mtgr_group_layernorm_bwd(ctypes.byref(problem), _ptr(dy), _ptr(x), _ptr(u),
                                          _ptr(group_ids), _ptr(gamma), _ptr(mean), _ptr(rstd),
                                          _ptr(dx), _ptr(du), _ptr(dgamma), _ptr(dbeta),
                                          _ptr(workspace), int(workspace_bytes), _stream(stream)))


def mtgr_bias_silu_fwd(rows, cols, dtype, h, ld_h, bias, out, ld_out, stream=None) -> None:
    _check(lib().mtgr_bias_silu_fwd(int(rows), int(cols), int(dtype), _ptr(h), int(ld_h), _ptr(bias), _ptr(out),
                                    int(ld_out), _stream(stream)))


def mtgr_bias_silu_bwd(rows, cols, dtype, h, ld_h, bias, dout, ld_dout, dh, ld_dh, stream=None) -> None:
    _check(lib().mtgr_bias_silu_bwd(int(rows), int(cols), int(dtype), _ptr(h), int(ld_h), _ptr(bias), _ptr(dout),
                                    int(ld_dout), _ptr(dh), int(ld_dh), _stream(stream)))


def mtgr_add(rows, cols, dtype, a, ld_a, b, ld_b, out, ld_out, stream=None) -> None:
    _check(lib().mtgr_add(int(rows), int(cols), int(dtype), _ptr(a), int(ld_a), _ptr(b), int(ld_b), _ptr(out),
                          int(ld_out), _stream(stream)))


def mtgr_gemm_workspace_size(layout, M, N, K) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().mtgr_gemm_workspace_size(int(layout), int(M), int(N), int(K), ctypes.byref(out)))
    return out.value


def mtgr_gemm_bf16(layout, M, N, K, A, lda, B, ldb, C, ldc, epilogue=MTGR_GEMM_EPI_NONE, bias=None, R=None,
                   ldr=0, C2=None, ldc2=0, colsum=None, workspace=None, workspace_bytes=0, stream=None) -> None:
    _check(lib().mtgr_gemm_bf16(int(layout), int(M), int(N), int(K), _ptr(A), int(lda), _ptr(B), int(ldb),
                                _ptr(C), int(ldc), int(epilogue), _ptr(bias), _ptr(R), int(ldr), _ptr(C2),
                                int(ldc2), _ptr(colsum), _ptr(workspace), int(workspace_bytes),
                                _stream(stream)))


def mtgr_debug_clock_probe(mfma_iterations, blocks, out, stream=None) -> int:
    """Launches the clock probe into `out` (device int64 [3 * blocks]); returns the constant
    counter's rate in kHz."""
    khz = ctypes.c_int32(0)
    _check(lib().mtgr_debug_clock_probe(int(mfma_iterations), int(blocks), _ptr(out), ctypes.byref(khz),
                                        _stream(stream)))
    return khz.value


def mtgr_debug_validate_inputs(problem, offsets, seg, group_ids, num_groups, scratch, scratch_bytes,
                               stream=None) -> None:
    _check(lib().mtgr_debug_validate_inputs(ctypes.byref(problem), _ptr(offsets), _ptr(seg),
                                            _ptr(group_ids), int(num_groups), _ptr(scratch),
                                            int(scratch_bytes), _stream(stream)))


# ------------------------------------------------------------------ problem builders

def attn_problem(num_users: int, total_tokens: int, max_seqlen: int, heads: int, head_dim: int,
                 dtype: int = MTGR_DTYPE_BF16, alpha: float = 1.0, rab_buckets: int = 0,
                 ld_q: Optional[int] = None, ld_k: Optional[int] = None, ld_v: Optional[int] = None,
                 ld_o: Optional[int] = None, flags: int = 0) -> HstuProblem:
    row = heads * head_dim
    return HstuProblem(num_users, max_seqlen, total_tokens, heads, head_dim, dtype, alpha, rab_buckets,
                       flags, ld_q or row, ld_k or row, ld_v or row, ld_o or row)


def gln_problem(num_tokens: int, dim: int, groups: int, dtype: int = MTGR_DTYPE_BF16,
                eps: float = 1e-5, ld_x: Optional[int] = None, ld_u: Optional[int] = None,
                ld_y: Optional[int] = None) -> GlnProblem:
    return GlnProblem(num_tokens, dim, groups, dtype, eps, ld_x or dim, ld_u or dim, ld_y or dim)


# ------------------------------------------------------------------ embedding table

def mtgr_embedding_init(table: EmbeddingTable, stream=None) -> None:
    _check(lib().mtgr_embedding_init(ctypes.byref(table), _stream(stream)))


def mtgr_embedding_dedup_workspace_size(n: int) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().mtgr_embedding_dedup_workspace_size(n, ctypes.byref(out)))
    return out.value


def mtgr_embedding_dedup(n, ids, unique, occurrences, inverse, num_unique, workspace, workspace_bytes,
                         stream=None) -> None:
    _check(lib().mtgr_embedding_dedup(n, _ptr(ids), _ptr(unique), _ptr(occurrences), _ptr(inverse),
                                      _ptr(num_unique), _ptr(workspace), workspace_bytes, _stream(stream)))


def mtgr_embedding_lookup_workspace_size(n_max: int) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().mtgr_embedding_lookup_workspace_size(n_max, ctypes.byref(out)))
    return out.value


def mtgr_embedding_lookup(table, n_max, unique, occurrences, num_unique, now, insert, rows, workspace,
                          workspace_bytes, stream=None) -> None:
    _check(lib().mtgr_embedding_lookup(ctypes.byref(table), n_max, _ptr(unique), _ptr(occurrences),
                                       _ptr(num_unique), now, int(bool(insert)), _ptr(rows), _ptr(workspace),
                                       workspace_bytes, _stream(stream)))


def mtgr_embedding_gather(table, n, inverse, rows, out, ld_out, stream=None) -> None:
    _check(lib().mtgr_embedding_gather(ctypes.byref(table), n, _ptr(inverse), _ptr(rows), _ptr(out), ld_out,
                                       _stream(stream)))


def mtgr_embedding_sgd_workspace_size(n: int, n_max: int, dim: int) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().mtgr_embedding_sgd_workspace_size(n, n_max, dim, ctypes.byref(out)))
    return out.value


def mtgr_embedding_sgd(table, n, inverse, occurrences, grad_out, ld_grad, n_max, rows, num_unique, lr,
                       workspace, workspace_bytes, stream=None) -> None:
    _check(lib().mtgr_embedding_sgd(ctypes.byref(table), n, _ptr(inverse), _ptr(occurrences), _ptr(grad_out),
                                    ld_grad, n_max, _ptr(rows), _ptr(num_unique), lr, _ptr(workspace),
                                    workspace_bytes, _stream(stream)))


def mtgr_embedding_evict(table, threshold, min_count, num_evicted, stream=None) -> None:
    _check(lib().mtgr_embedding_evict(ctypes.byref(table), threshold, min_count, _ptr(num_evicted),
                                      _stream(stream)))


def mtgr_embedding_rehash(src, dst, stream=None) -> None:
    _check(lib().mtgr_embedding_rehash(ctypes.byref(src), ctypes.byref(dst), _stream(stream)))
