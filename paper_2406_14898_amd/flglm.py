"""ctypes binding of libflglm.so (include/flglm.h, include/flglm_testing.h).

Argument marshalling only: every step of the server stack runs in the HIP
library.  Functions keep the C names; device buffers may be passed as torch
tensors (their data_ptr() is used) or as integer addresses, streams as
torch.cuda.Stream, an integer hipStream_t, or None (the current torch
stream when torch has a GPU, else the default stream).
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libflglm.so")

FL_OK = 0
FL_ERR_NULL, FL_ERR_SHAPE, FL_ERR_SEQLENS, FL_ERR_CLIENTS, FL_ERR_PREFIX = -1, -2, -3, -4, -5
FL_ERR_WORKSPACE, FL_ERR_ALIAS, FL_ERR_ALIGN, FL_ERR_HIP, FL_ERR_ARG = -6, -7, -8, -9, -10
FL_ERR_NOMEM = -11
FL_BF16, FL_F32 = 0, 1
FL_MASK_CAUSAL, FL_MASK_PREFIX = 0, 1
FL_GEMM_NT, FL_GEMM_NN, FL_GEMM_TN = 0, 1, 2
FL_EPI_STORE, FL_EPI_BIAS, FL_EPI_BIAS_RES, FL_EPI_BIAS_GELU, FL_EPI_GELU_BWD, FL_EPI_ACC_F32, FL_EPI_RES = range(7)
FL_PROF_NUM_CLASSES = 14
FL_NOALLOC_SCRATCH_BYTES = 256 << 20
FL_NOALLOC_MAX_SEQS = 256

PARAM_FIELDS = ("w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2",
                "ln1_g", "ln1_b", "ln2_g", "ln2_b")
PREFIX_FIELDS = ("prefix_k", "prefix_v")  # P-tuning v2 prefix keys / values

#: every extern "C" symbol the headers declare
EXPORTS = (
    "fl_stack_create", "fl_stack_destroy", "fl_stack_saved_bytes", "fl_stack_workspace_bytes",
    "fl_server_stack_forward", "fl_server_stack_forward_noalloc", "fl_server_stack_backward",
    "fl_client_token_range",
    "fl_pack_clients", "fl_unpack_clients", "fl_last_error",
    "fl_adam_step", "fl_average_replicas",
    "fl_client_create", "fl_client_destroy", "fl_client_workspace_bytes", "fl_embedding_forward",
    "fl_embedding_backward", "fl_lm_head_forward", "fl_lm_head_backward",
    "fl_stack_profile", "fl_stack_profile_classes", "fl_stack_profile_read", "fl_profile_class_name",
    "fl_test_gemm", "fl_test_layernorm_fwd", "fl_test_layernorm_bwd", "fl_test_layernorm_bwd_fused",
    "fl_test_colsum",
    "fl_test_rope", "fl_test_attention_fwd", "fl_test_attention_bwd", "fl_test_attention_ds_bytes",
)


class FlglmError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"flglm error {code}: {msg}")
        self.code = code


class fl_stack_desc(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("hidden", ctypes.c_int32), ("num_heads", ctypes.c_int32),
                ("ffn_hidden", ctypes.c_int32), ("rotary_dim", ctypes.c_int32), ("rope_base", ctypes.c_float),
                ("ln_eps", ctypes.c_float), ("dtype", ctypes.c_int32), ("num_prefix", ctypes.c_int32),
                ("residual_alpha", ctypes.c_float), ("rotary_2d", ctypes.c_int32)]


class fl_batch_desc(ctypes.Structure):
    _fields_ = [("num_clients", ctypes.c_int32), ("num_seqs", ctypes.c_int32), ("total_tokens", ctypes.c_int64),
                ("max_seqlen", ctypes.c_int32), ("cu_seqlens", ctypes.POINTER(ctypes.c_int32)),
                ("client_seq_ptr", ctypes.POINTER(ctypes.c_int32)), ("mask_kind", ctypes.c_int32),
                ("prefix_len", ctypes.POINTER(ctypes.c_int32))]


class fl_client_desc(ctypes.Structure):
    _fields_ = [("vocab", ctypes.c_int64), ("hidden", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("ln_eps", ctypes.c_float)]


class fl_layer_params(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PARAM_FIELDS + PREFIX_FIELDS]


class fl_layer_grads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PARAM_FIELDS + PREFIX_FIELDS]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads the HIP library; raises if it has not been built (there is no
    fallback implementation)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise FlglmError(FL_ERR_ARG, f"HIP library not built: {path} is missing "
                                     f"(run paper_2406_14898_amd/build.py)")
    lib = ctypes.CDLL(path)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    P = ctypes.POINTER
    sig = {
        "fl_stack_create": [P(fl_stack_desc), P(vp)],
        "fl_stack_destroy": [vp],
        "fl_stack_saved_bytes": [vp, P(fl_batch_desc), ctypes.c_int, P(sz)],
        "fl_stack_workspace_bytes": [vp, P(fl_batch_desc), ctypes.c_int, P(sz)],
        "fl_server_stack_forward": [vp, P(fl_batch_desc), P(fl_layer_params), vp, vp, vp, ctypes.c_int, vp, sz, vp],
        "fl_server_stack_forward_noalloc": [vp, P(fl_batch_desc), P(fl_layer_params), vp, vp, vp],
        "fl_server_stack_backward": [vp, P(fl_batch_desc), P(fl_layer_params), P(fl_layer_grads), vp, vp, vp, vp,
                                     ctypes.c_int, vp, sz, vp],
        "fl_client_token_range": [P(fl_batch_desc), i32, P(i64), P(i64)],
        "fl_pack_clients": [vp, P(fl_batch_desc), P(vp), vp, vp, sz, vp],
        "fl_unpack_clients": [vp, P(fl_batch_desc), vp, P(vp), vp, sz, vp],
        "fl_adam_step": [vp, vp, vp, vp, vp, i64, i64, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                         ctypes.c_double, ctypes.c_int, vp],
        "fl_average_replicas": [i32, P(vp), P(vp), i64, vp],
        "fl_client_create": [P(fl_client_desc), P(vp)],
        "fl_client_destroy": [vp],
        "fl_client_workspace_bytes": [vp, i64, P(sz)],
        "fl_embedding_forward": [vp, vp, P(i32), i64, vp, vp, sz, vp],
        "fl_embedding_backward": [vp, P(i32), i64, vp, vp, vp, sz, vp],
        "fl_lm_head_forward": [vp, vp, vp, vp, vp, P(i32), i64, vp, vp, vp, sz, vp],
        "fl_lm_head_backward": [vp, vp, vp, vp, i64, ctypes.c_float, vp, vp, vp, vp, vp, sz, vp],
        "fl_stack_profile": [vp, ctypes.c_int],
        "fl_stack_profile_classes": [vp, ctypes.c_uint32],
        "fl_stack_profile_read": [vp, ctypes.c_int, P(i64), P(ctypes.c_double), P(ctypes.c_double),
                                  P(ctypes.c_double)],
        "fl_test_gemm": [ctypes.c_int] * 3 + [vp] * 3 + [ctypes.c_int] * 3 + [i64] * 3 + [vp, vp, i64, vp, i64, vp,
                                                                                          i64, vp, i64, ctypes.c_int,
                                                                                          ctypes.c_float, vp, vp],
        "fl_test_layernorm_fwd": [ctypes.c_int, vp, vp, vp, vp, vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_float,
                                  vp],
        "fl_test_layernorm_bwd": [ctypes.c_int] + [vp] * 7 + [ctypes.c_int, ctypes.c_int, vp],
        "fl_test_layernorm_bwd_fused": [ctypes.c_int] + [vp] * 7 + [ctypes.c_int, ctypes.c_int] + [vp] * 5,
        "fl_test_colsum": [ctypes.c_int, ctypes.c_int, vp, vp, vp, vp, ctypes.c_int, ctypes.c_int, vp, vp, vp, vp],
        "fl_test_rope": [ctypes.c_int, vp, vp] + [ctypes.c_int] * 6 + [ctypes.c_float, vp, vp, vp, vp],
        "fl_test_attention_fwd": [ctypes.c_int, vp, vp, vp, vp, vp] + [ctypes.c_int] * 5 + [vp, vp, ctypes.c_int, vp],
        "fl_test_attention_bwd": [ctypes.c_int] + [vp] * 11 + [ctypes.c_int] * 6 + [vp, vp, ctypes.c_int, vp, vp,
                                                                                    ctypes.c_size_t, vp],
        "fl_test_attention_ds_bytes": [vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                       ctypes.POINTER(ctypes.c_size_t)],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.fl_last_error.argtypes = []
    lib.fl_last_error.restype = ctypes.c_char_p
    lib.fl_profile_class_name.argtypes = [ctypes.c_int]
    lib.fl_profile_class_name.restype = ctypes.c_char_p
    _lib = lib
    return lib


def fl_last_error() -> str:
    return load().fl_last_error().decode()


def _check(rc: int) -> None:
    if rc != FL_OK:
        raise FlglmError(rc, fl_last_error())


def _ptr(t) -> Optional[int]:
    """Device address of a tensor (None and integer addresses pass through).
    Every tensor argument of the library is device memory: a host tensor is
    refused here instead of handing its address to a kernel."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if getattr(t, "is_cuda", True) is False:
        raise FlglmError(FL_ERR_ARG, f"tensor on {t.device}: the library takes device memory")
    return t.data_ptr()


def _stream(s) -> Optional[int]:
    if s is None:
        try:
            import torch
            if torch.cuda.is_available():
                return torch.cuda.current_stream().cuda_stream
        except Exception:  # pragma: no cover
            pass
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


# ---------------------------------------------------------------------------
# Descriptors
# ---------------------------------------------------------------------------

def stack_desc(num_layers: int, hidden: int, num_heads: int, ffn_hidden: int, rotary_dim: int,
               dtype: int = FL_BF16, rope_base: float = 10000.0, ln_eps: float = 1e-5,
               num_prefix: int = 0, residual_alpha: float = 0.0, rotary_2d: bool = False) -> fl_stack_desc:
    return fl_stack_desc(num_layers, hidden, num_heads, ffn_hidden, rotary_dim, rope_base, ln_eps, dtype, num_prefix,
                         residual_alpha, int(rotary_2d))


class BatchDesc:
    """Owns the host arrays an fl_batch_desc points at."""

    def __init__(self, cu_seqlens, client_seq_ptr, prefix_len=None, max_seqlen: Optional[int] = None):
        self.cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
        self.csp = np.ascontiguousarray(client_seq_ptr, dtype=np.int32)
        self.prefix = None if prefix_len is None else np.ascontiguousarray(prefix_len, dtype=np.int32)
        P = ctypes.POINTER(ctypes.c_int32)
        lens = np.diff(self.cu)
        self.desc = fl_batch_desc(
            len(self.csp) - 1, len(self.cu) - 1, int(self.cu[-1]) if len(self.cu) else 0,
            int(lens.max()) if max_seqlen is None and len(lens) else int(max_seqlen or 0),
            self.cu.ctypes.data_as(P), self.csp.ctypes.data_as(P),
            FL_MASK_PREFIX if self.prefix is not None else FL_MASK_CAUSAL,
            self.prefix.ctypes.data_as(P) if self.prefix is not None else None)

    @property
    def total_tokens(self) -> int:
        return int(self.desc.total_tokens)

    @classmethod
    def from_batch(cls, b) -> "BatchDesc":
        """From any record with cu_seqlens, client_seq_ptr, mask, prefix_len."""
        pre = b.prefix_len if getattr(b, "mask", "causal") == "prefix" else None
        return cls(b.cu_seqlens, b.client_seq_ptr, pre)


def layer_params(tensors: dict) -> fl_layer_params:
    """Device tensors by name; the prefix entries are optional."""
    return fl_layer_params(*[_ptr(tensors.get(n)) for n in PARAM_FIELDS + PREFIX_FIELDS])


def layer_grads(tensors: dict) -> fl_layer_grads:
    """Device fp32 accumulators by name; a dict without the weight names
    means frozen weights (P-tuning v2), the prefix entries are optional."""
    return fl_layer_grads(*[_ptr(tensors.get(n)) for n in PARAM_FIELDS + PREFIX_FIELDS])


# ---------------------------------------------------------------------------
# C entry points
# ---------------------------------------------------------------------------

def fl_stack_create(desc: fl_stack_desc) -> int:
    h = ctypes.c_void_p()
    _check(load().fl_stack_create(ctypes.byref(desc), ctypes.byref(h)))
    return h.value


def fl_stack_destroy(handle: int) -> None:
    _check(load().fl_stack_destroy(handle))


def fl_stack_saved_bytes(handle: int, batch: BatchDesc, recompute: bool) -> int:
    n = ctypes.c_size_t()
    _check(load().fl_stack_saved_bytes(handle, ctypes.byref(batch.desc), int(recompute), ctypes.byref(n)))
    return n.value


def fl_stack_workspace_bytes(handle: int, batch: BatchDesc, recompute: bool) -> int:
    n = ctypes.c_size_t()
    _check(load().fl_stack_workspace_bytes(handle, ctypes.byref(batch.desc), int(recompute), ctypes.byref(n)))
    return n.value


def fl_server_stack_forward(handle: int, batch: BatchDesc, layers: Sequence[fl_layer_params], x, y, saved,
                            recompute: bool, workspace, workspace_bytes: int, stream=None) -> None:
    arr = (fl_layer_params * len(layers))(*layers)
    _check(load().fl_server_stack_forward(handle, ctypes.byref(batch.desc), arr, _ptr(x), _ptr(y), _ptr(saved),
                                          int(recompute), _ptr(workspace), workspace_bytes, _stream(stream)))


def fl_server_stack_forward_noalloc(handle: int, batch: BatchDesc, layers: Sequence[fl_layer_params], x, y,
                                    stream=None) -> None:
    arr = (fl_layer_params * len(layers))(*layers)
    _check(load().fl_server_stack_forward_noalloc(handle, ctypes.byref(batch.desc), arr, _ptr(x), _ptr(y),
                                                  _stream(stream)))


def fl_server_stack_backward(handle: int, batch: BatchDesc, layers: Sequence[fl_layer_params],
                             grads: Sequence[fl_layer_grads], x, saved, dy, dx, recompute: bool, workspace,
                             workspace_bytes: int, stream=None) -> None:
    pa = (fl_layer_params * len(layers))(*layers)
    ga = (fl_layer_grads * len(grads))(*grads)
    _check(load().fl_server_stack_backward(handle, ctypes.byref(batch.desc), pa, ga, _ptr(x), _ptr(saved), _ptr(dy),
                                           _ptr(dx), int(recompute), _ptr(workspace), workspace_bytes,
                                           _stream(stream)))


def fl_client_token_range(batch: BatchDesc, client: int):
    b, e = ctypes.c_int64(), ctypes.c_int64()
    _check(load().fl_client_token_range(ctypes.byref(batch.desc), client, ctypes.byref(b), ctypes.byref(e)))
    return b.value, e.value


def fl_pack_clients(handle: int, batch: BatchDesc, client_bufs, packed, workspace, workspace_bytes: int,
                    stream=None) -> None:
    arr = (ctypes.c_void_p * len(client_bufs))(*[_ptr(c) for c in client_bufs])
    _check(load().fl_pack_clients(handle, ctypes.byref(batch.desc), arr, _ptr(packed), _ptr(workspace),
                                  workspace_bytes, _stream(stream)))


def fl_unpack_clients(handle: int, batch: BatchDesc, packed, client_bufs, workspace, workspace_bytes: int,
                      stream=None) -> None:
    arr = (ctypes.c_void_p * len(client_bufs))(*[_ptr(c) for c in client_bufs])
    _check(load().fl_unpack_clients(handle, ctypes.byref(batch.desc), _ptr(packed), arr, _ptr(workspace),
                                    workspace_bytes, _stream(stream)))


def fl_adam_step(param, grad, exp_avg, exp_avg_sq, param_bf16, n: int, step: int, lr: float = 2e-2,
                 beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8, zero_grad: bool = False,
                 stream=None) -> None:
    _check(load().fl_adam_step(_ptr(param), _ptr(grad), _ptr(exp_avg), _ptr(exp_avg_sq), _ptr(param_bf16), n, step,
                               lr, beta1, beta2, eps, int(zero_grad), _stream(stream)))


def fl_average_replicas(params, params_bf16, n: int, stream=None) -> None:
    arr = (ctypes.c_void_p * len(params))(*[_ptr(p) for p in params])
    arr16 = None if params_bf16 is None else (ctypes.c_void_p * len(params_bf16))(*[_ptr(p) for p in params_bf16])
    _check(load().fl_average_replicas(len(params), arr, arr16, n, _stream(stream)))


def _host_i32(a):
    import numpy as np
    arr = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return arr, arr.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def fl_client_create(vocab: int, hidden: int, dtype: int = FL_BF16, ln_eps: float = 1e-5) -> int:
    h = ctypes.c_void_p()
    _check(load().fl_client_create(ctypes.byref(fl_client_desc(vocab, hidden, dtype, ln_eps)), ctypes.byref(h)))
    return h.value


def fl_client_destroy(handle: int) -> None:
    _check(load().fl_client_destroy(handle))


def fl_client_workspace_bytes(handle: int, T: int) -> int:
    n = ctypes.c_size_t()
    _check(load().fl_client_workspace_bytes(handle, T, ctypes.byref(n)))
    return n.value


def fl_embedding_forward(handle: int, table, ids, out, workspace, stream=None) -> None:
    arr, p = _host_i32(ids)
    _check(load().fl_embedding_forward(handle, _ptr(table), p, len(arr), _ptr(out), _ptr(workspace),
                                       workspace.numel() * workspace.element_size(), _stream(stream)))


def fl_embedding_backward(handle: int, ids, dout, dtable, workspace, stream=None) -> None:
    arr, p = _host_i32(ids)
    _check(load().fl_embedding_backward(handle, p, len(arr), _ptr(dout), _ptr(dtable), _ptr(workspace),
                                        workspace.numel() * workspace.element_size(), _stream(stream)))


def fl_lm_head_forward(handle: int, h, w, labels, loss_tok, loss_sum, workspace, stream=None, ln_g=None,
                       ln_b=None) -> None:
    arr, p = _host_i32(labels)
    _check(load().fl_lm_head_forward(handle, _ptr(h), _ptr(ln_g), _ptr(ln_b), _ptr(w), p, len(arr), _ptr(loss_tok),
                                     _ptr(loss_sum), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                     _stream(stream)))


def fl_lm_head_backward(handle: int, h, w, T: int, grad_scale: float, dh, dw, workspace, stream=None, ln_g=None,
                        dln_g=None, dln_b=None) -> None:
    _check(load().fl_lm_head_backward(handle, _ptr(h), _ptr(ln_g), _ptr(w), T, grad_scale, _ptr(dh), _ptr(dln_g),
                                      _ptr(dln_b), _ptr(dw), _ptr(workspace),
                                      workspace.numel() * workspace.element_size(), _stream(stream)))


def fl_stack_profile(handle: int, enable: bool) -> None:
    _check(load().fl_stack_profile(handle, int(enable)))


def fl_stack_profile_classes(handle: int, class_mask: int) -> None:
    """Time only the launches of the classes whose bits are set (0: off)."""
    _check(load().fl_stack_profile_classes(handle, int(class_mask) & 0xffffffff))


def fl_profile_class_name(cls: int) -> str:
    return load().fl_profile_class_name(cls).decode()


def fl_stack_profile_read(handle: int, cls: int):
    """(launches, milliseconds, flops, bytes) for one class; waits for the events."""
    n, ms, fl, by = ctypes.c_int64(), ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(load().fl_stack_profile_read(handle, cls, ctypes.byref(n), ctypes.byref(ms), ctypes.byref(fl),
                                        ctypes.byref(by)))
    return n.value, ms.value, fl.value, by.value


def profile_table(handle: int):
    """{class name: dict(launches, ms, flops, bytes)} for every class with launches."""
    out = {}
    for c in range(FL_PROF_NUM_CLASSES):
        n, ms, fl, by = fl_stack_profile_read(handle, c)
        if n:
            out[fl_profile_class_name(c)] = dict(launches=n, ms=ms, flops=fl, bytes=by)
    return out


# ---------------------------------------------------------------------------
# Test-only single-kernel entry points
# ---------------------------------------------------------------------------

def fl_test_gemm(dtype, layout, epi, A, B, C, M, N, K, lda, ldb, ldc, bias=None, R=None, ldr=0, C2=None, ldc2=0,
                 Z=None, ldz=0, part=None, b_rows=0, res_scale=1.0, colsum=None, stream=None) -> None:
    """part: optional fp32 device tensor, split-reduction scratch; b_rows:
    rows B really has (0 = all); colsum: fp32 [ceil(M/256), N] per-block
    column sums of C (bf16 NN GELU_BWD only)."""
    nbytes = part.numel() * part.element_size() if part is not None else 0
    _check(load().fl_test_gemm(dtype, layout, epi, _ptr(A), _ptr(B), _ptr(C), M, N, K, lda, ldb, ldc, _ptr(bias),
                               _ptr(R), ldr, _ptr(C2), ldc2, _ptr(Z), ldz, _ptr(part), nbytes, b_rows,
                               res_scale, _ptr(colsum), _stream(stream)))


def fl_test_layernorm_fwd(dtype, x, g, b, y, mean, rstd, T, H, eps, stream=None) -> None:
    _check(load().fl_test_layernorm_fwd(dtype, _ptr(x), _ptr(g), _ptr(b), _ptr(y), _ptr(mean), _ptr(rstd), T, H,
                                        eps, _stream(stream)))


def fl_test_layernorm_bwd(dtype, dy, x, mean, rstd, g, dres, dx, T, H, stream=None) -> None:
    _check(load().fl_test_layernorm_bwd(dtype, _ptr(dy), _ptr(x), _ptr(mean), _ptr(rstd), _ptr(g), _ptr(dres),
                                        _ptr(dx), T, H, _stream(stream)))


def fl_test_layernorm_bwd_fused(dtype, dy, x, mean, rstd, g, dres, dx, T, H, dgamma=None, dbeta=None, dsum=None,
                                partial=None, stream=None) -> None:
    _check(load().fl_test_layernorm_bwd_fused(dtype, _ptr(dy), _ptr(x), _ptr(mean), _ptr(rstd), _ptr(g), _ptr(dres),
                                              _ptr(dx), T, H, _ptr(dgamma), _ptr(dbeta), _ptr(dsum), _ptr(partial),
                                              _stream(stream)))


def fl_test_colsum(dtype, mode, X, Y, mean, rstd, T, N, out, out2, partial, stream=None) -> None:
    _check(load().fl_test_colsum(dtype, mode, _ptr(X), _ptr(Y), _ptr(mean), _ptr(rstd), T, N, _ptr(out), _ptr(out2),
                                 _ptr(partial), _stream(stream)))


def fl_test_rope(dtype, qkv, cu_dev, S, T, max_seqlen, H, num_heads, rotary_dim, base, pos, cos_t, sin_t,
                 stream=None) -> None:
    _check(load().fl_test_rope(dtype, _ptr(qkv), _ptr(cu_dev), S, T, max_seqlen, H, num_heads, rotary_dim, base,
                               _ptr(pos), _ptr(cos_t), _ptr(sin_t), _stream(stream)))


def fl_test_attention_fwd(dtype, qkv, o, lse, cu_dev, prefix_dev, T, S, max_seqlen, H, num_heads,
                          pk=None, pv=None, num_prefix=0, stream=None) -> None:
    _check(load().fl_test_attention_fwd(dtype, _ptr(qkv), _ptr(o), _ptr(lse), _ptr(cu_dev), _ptr(prefix_dev), T, S,
                                        max_seqlen, H, num_heads, _ptr(pk), _ptr(pv), num_prefix, _stream(stream)))


def fl_test_attention_bwd(dtype, qkv, o, lse, dout, dqkv, delta, cu_dev, prefix_dev, pos, cos_t, sin_t, rotary_dim,
                          T, S, max_seqlen, H, num_heads, pk=None, pv=None, num_prefix=0, dprefix_part=None,
                          ds_work=None, stream=None) -> None:
    """ds_work: device byte tensor of fl_test_attention_ds_bytes bytes (dq
    reads the stored softmax gradient), or None (dq recomputes it)."""
    nbytes = ds_work.numel() * ds_work.element_size() if ds_work is not None else 0
    _check(load().fl_test_attention_bwd(dtype, _ptr(qkv), _ptr(o), _ptr(lse), _ptr(dout), _ptr(dqkv), _ptr(delta),
                                        _ptr(cu_dev), _ptr(prefix_dev), _ptr(pos), _ptr(cos_t), _ptr(sin_t),
                                        rotary_dim, T, S, max_seqlen, H, num_heads, _ptr(pk), _ptr(pv), num_prefix,
                                        _ptr(dprefix_part), _ptr(ds_work), nbytes, _stream(stream)))


def fl_test_attention_ds_bytes(cu_host, prefix_host, num_heads, num_prefix=0) -> int:
    """Bytes of ds_work for these host sequence bounds (numpy int32 cu_host
    [S+1], prefix_host [S] or None)."""
    cu = np.ascontiguousarray(cu_host, dtype=np.int32)
    pre = None if prefix_host is None else np.ascontiguousarray(prefix_host, dtype=np.int32)
    out = ctypes.c_size_t(0)
    _check(load().fl_test_attention_ds_bytes(cu.ctypes.data, None if pre is None else pre.ctypes.data,
                                             len(cu) - 1, num_heads, num_prefix, ctypes.byref(out)))
    return int(out.value)
