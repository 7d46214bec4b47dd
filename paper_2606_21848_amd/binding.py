"""Thin ctypes binding of libkeyless.so (the C ABI in include/keyless.h).

Argument marshalling only: torch supplies device memory and the current HIP
stream; every step of the computation runs in the library's HIP kernels.
There is no fallback: if the library is not built, every call raises.
"""

from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkeyless.so")

KL_OK, KL_ERR_INVALID_ARG, KL_ERR_UNSUPPORTED, KL_ERR_WORKSPACE, KL_ERR_HIP = 0, -1, -2, -3, -4
KL_F32, KL_BF16 = 0, 1
KL_CONTIGUOUS, KL_PAGED = 0, 1

# Every symbol include/keyless.h declares.
EXPORTS = (
    "keyless_fold_routing", "keyless_prefill", "keyless_prefill_workspace_size",
    "keyless_packed_weights_size", "keyless_pack_weights", "keyless_prefill_packed",
    "keyless_cross_attention", "keyless_cross_attention_workspace_size",
    "keyless_cross_attention_packed",
    "keyless_latent_decode", "keyless_latent_decode_workspace_size",
    "keyless_attention_forward", "keyless_attention_backward",
    "keyless_attention_backward_workspace_size", "keyless_weight_gradients",
    "keyless_weight_gradients_workspace_size",
    "keyless_decode_project", "keyless_decode", "keyless_decode_chunked", "keyless_decode_workspace_size",
    "keyless_decode_append", "keyless_decode_noalloc",
    "value_cache_append", "standard_decode", "standard_decode_chunked",
    "keyless_set_kernel_timer", "keyless_probe_read", "keyless_probe_mfma",
    "keyless_last_error", "keyless_version",
)


class KeylessError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"status {status}: {message}")
        self.status = status


class KLValueCache(ctypes.Structure):
    _fields_ = [
        ("data", ctypes.c_void_p), ("dtype", ctypes.c_int), ("layout", ctypes.c_int),
        ("G", ctypes.c_int), ("d_head", ctypes.c_int), ("L_max", ctypes.c_int),
        ("block_size", ctypes.c_int), ("num_blocks", ctypes.c_int),
        ("max_blocks_per_seq", ctypes.c_int), ("block_table", ctypes.c_void_p),
    ]


_lib = None


def load(path: str = LIB_PATH):
    """Load the shared library (once). Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2606_21848_amd.build`")
    # torch's HIP runtime must be loaded first so the library binds to it.
    import torch.cuda  # noqa: F401
    lib = ctypes.CDLL(path)
    vp, i, f, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    cp = ctypes.POINTER(KLValueCache)
    sig = {
        "keyless_fold_routing": (i, [vp, vp, i, i, i, i, vp, vp]),
        "keyless_prefill": (i, [vp, vp, vp, vp, i, i, i, i, i, i, i, f, i, vp, vp, vp, vp, sz, vp]),
        "keyless_prefill_workspace_size": (sz, [i, i, i, i, i, i, i, i, i, i]),
        "keyless_packed_weights_size": (sz, [i, i, i, i, i]),
        "keyless_pack_weights": (i, [vp, vp, vp, i, i, i, i, i, vp, vp]),
        "keyless_prefill_packed": (i, [vp, vp, i, i, i, i, i, i, i, f, i, vp, vp, vp, vp, sz, vp]),
        "keyless_cross_attention": (i, [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, f, i, vp, vp, vp,
                                        vp, sz, vp]),
        "keyless_cross_attention_workspace_size": (sz, [i, i, i, i, i, i, i, i, i, i, i]),
        "keyless_cross_attention_packed": (i, [vp, vp, vp, i, i, i, i, i, i, i, f, i, vp, vp, vp,
                                               vp, sz, vp]),
        "keyless_decode_project": (i, [vp, vp, i, i, i, i, i, i, vp, vp, cp, vp, vp]),
        "keyless_decode": (i, [vp, cp, vp, i, i, f, vp, vp, sz, vp]),
        "keyless_decode_chunked": (i, [vp, cp, vp, i, i, f, vp, vp, sz, i, vp]),
        "keyless_decode_append": (i, [vp, vp, cp, vp, i, i, f, vp, vp, sz, vp]),
        "keyless_decode_noalloc": (i, [vp, cp, vp, i, i, f, vp, vp]),
        "keyless_decode_workspace_size": (sz, [cp, i, i, i]),
        "keyless_latent_decode": (i, [vp, vp, cp, vp, i, i, i, f, vp, vp, sz, vp]),
        "keyless_latent_decode_workspace_size": (sz, [cp, i, i, i]),
        "keyless_attention_forward": (i, [vp, vp, i, i, i, i, i, i, f, i, vp, vp, vp, vp]),
        "keyless_attention_backward": (i, [vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, f, i, vp,
                                           vp, vp, sz, vp]),
        "keyless_attention_backward_workspace_size": (sz, [i, i, i]),
        "keyless_weight_gradients": (i, [vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, vp, vp, vp,
                                         vp, vp, sz, vp]),
        "keyless_weight_gradients_workspace_size": (sz, [i, i, i, i, i, i, i]),
        "value_cache_append": (i, [cp, vp, vp, i, i, vp]),
        "standard_decode": (i, [vp, cp, cp, vp, i, i, f, vp, vp, sz, vp]),
        "standard_decode_chunked": (i, [vp, cp, cp, vp, i, i, f, vp, vp, sz, i, vp]),
        "keyless_set_kernel_timer": (None, [vp, vp]),
        "keyless_probe_read": (i, [vp, sz, vp, i, vp]),
        "keyless_probe_mfma": (i, [vp, i, i, vp]),
        "keyless_last_error": (ctypes.c_char_p, []),
        "keyless_version": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int):
    if status != KL_OK:
        raise KeylessError(status, _lib.keyless_last_error().decode())


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return KL_BF16
    if t.dtype == torch.float32:
        return KL_F32
    raise TypeError(f"unsupported dtype {t.dtype} (bf16 or fp32)")


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensors must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


class ValueCache:
    """A value-only cache: contiguous [B, G, L_max, d] or paged [num_blocks, G, bs, d]."""

    def __init__(self, data: torch.Tensor, block_table: torch.Tensor | None = None):
        self.data = data
        self.block_table = block_table
        d = KLValueCache()
        d.data = data.data_ptr()
        d.dtype = _dt(data)
        d.G = data.shape[1]
        d.d_head = data.shape[3]
        if block_table is None:
            d.layout = KL_CONTIGUOUS
            d.L_max = data.shape[2]
        else:
            if block_table.dtype != torch.int32:
                raise TypeError("block_table must be int32")
            _ptr(block_table)
            d.layout = KL_PAGED
            d.block_size = data.shape[2]
            d.num_blocks = data.shape[0]
            d.max_blocks_per_seq = block_table.shape[1]
            d.block_table = block_table.data_ptr()
        _ptr(data)
        self.desc = d

    @property
    def ref(self):
        return ctypes.byref(self.desc)


def decode_workspace_bytes(cache: ValueCache, B: int, H: int, chunk_rows: int = 0) -> int:
    load()
    return int(_lib.keyless_decode_workspace_size(cache.ref, B, H, chunk_rows))


def keyless_decode(q_routed: torch.Tensor, cache: ValueCache, lengths: torch.Tensor,
                   scale: float = 0.0, out: torch.Tensor | None = None,
                   workspace: torch.Tensor | None = None, chunk_rows: int = 0) -> torch.Tensor:
    """out[b, h] = softmax over the cached values of <q~, v> * scale, applied to the values."""
    load()
    B, H, _ = q_routed.shape
    if lengths.dtype != torch.int32:
        raise TypeError("lengths must be int32")
    if out is None:
        out = torch.empty_like(q_routed)
    if workspace is None:
        workspace = torch.zeros(max(decode_workspace_bytes(cache, B, H, chunk_rows), 256),
                                dtype=torch.uint8, device=q_routed.device)
    _check(_lib.keyless_decode_chunked(_ptr(q_routed), cache.ref, _ptr(lengths), B, H, scale,
                                       _ptr(out), _ptr(workspace), workspace.numel(), chunk_rows,
                                       _stream(q_routed)))
    return out


def standard_decode(q: torch.Tensor, k_cache: ValueCache, v_cache: ValueCache,
                    lengths: torch.Tensor, scale: float = 0.0, out: torch.Tensor | None = None,
                    workspace: torch.Tensor | None = None, chunk_rows: int = 0) -> torch.Tensor:
    load()
    B, H, _ = q.shape
    if out is None:
        out = torch.empty_like(q)
    if workspace is None:
        workspace = torch.zeros(max(decode_workspace_bytes(v_cache, B, H, chunk_rows), 256),
                                dtype=torch.uint8, device=q.device)
    _check(_lib.standard_decode_chunked(_ptr(q), k_cache.ref, v_cache.ref, _ptr(lengths), B, H,
                                        scale, _ptr(out), _ptr(workspace), workspace.numel(),
                                        chunk_rows, _stream(q)))
    return out


def value_cache_append(cache: ValueCache, values: torch.Tensor, lengths_before: torch.Tensor):
    """Write values[b, t, g, :] at position lengths_before[b] + t of sequence b."""
    load()
    B, T = values.shape[0], values.shape[1]
    _check(_lib.value_cache_append(cache.ref, _ptr(values), _ptr(lengths_before), B, T,
                                   _stream(values)))


def keyless_fold_routing(W_Q: torch.Tensor, W_R: torch.Tensor) -> torch.Tensor:
    """W~^Q_h = W^Q_h W^R_h for every head; W_Q [d, H*d_k], W_R [H, d_k, d_k]."""
    load()
    H, dk, _ = W_R.shape
    out = torch.empty_like(W_Q)
    _check(_lib.keyless_fold_routing(_ptr(W_Q), _ptr(W_R), W_Q.shape[0], H, dk, _dt(W_Q),
                                     _ptr(out), _stream(W_Q)))
    return out


def keyless_prefill(x: torch.Tensor, W_Q: torch.Tensor, W_R: torch.Tensor | None,
                    W_V: torch.Tensor, H: int, G: int, causal: bool = True, scale: float = 0.0,
                    return_qv: bool = False, out=None, q_routed_out=None, v_out=None,
                    workspace=None):
    """Keyless self-attention; returns out [B, N, H, d] (and Q~, V if return_qv)."""
    load()
    B, N, d_model = x.shape
    dk = W_Q.shape[1] // H
    if out is None:
        out = torch.empty((B, N, H, dk), dtype=x.dtype, device=x.device)
    if return_qv:
        if q_routed_out is None:
            q_routed_out = torch.empty((B, N, H, dk), dtype=x.dtype, device=x.device)
        if v_out is None:
            v_out = torch.empty((B, N, G, dk), dtype=x.dtype, device=x.device)
    need = int(_lib.keyless_prefill_workspace_size(B, N, d_model, H, G, dk, _dt(x),
                                                   int(W_R is not None), int(q_routed_out is not None),
                                                   int(v_out is not None)))
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=x.device)
    _check(_lib.keyless_prefill(_ptr(x), _ptr(W_Q), _ptr(W_R), _ptr(W_V), B, N, d_model, H, G, dk,
                                int(causal), scale, _dt(x), _ptr(out), _ptr(q_routed_out),
                                _ptr(v_out), _ptr(workspace), workspace.numel(), _stream(x)))
    if return_qv:
        return out, q_routed_out, v_out
    return out


def set_kernel_timer(start: "torch.cuda.Event | None", stop: "torch.cuda.Event | None"):
    """Record ``start``/``stop`` around the split kernel of later decode calls on
    this thread (both events must already have been recorded once, so that
    torch has created them); ``None, None`` turns it off."""
    load()
    if start is None or stop is None:
        _lib.keyless_set_kernel_timer(None, None)
    else:
        _lib.keyless_set_kernel_timer(ctypes.c_void_p(start.cuda_event),
                                      ctypes.c_void_p(stop.cuda_event))


def probe_read(buf: torch.Tensor, sink: torch.Tensor, workgroups: int) -> None:
    """Stream-read every byte of ``buf`` once (the practical read ceiling)."""
    load()
    _check(_lib.keyless_probe_read(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink),
                                   workgroups, _stream(buf)))


def probe_mfma(sink: torch.Tensor, iters: int, workgroups: int) -> int:
    """Run the matrix-core loop; returns its FLOP count."""
    load()
    _check(_lib.keyless_probe_mfma(_ptr(sink), iters, workgroups, _stream(sink)))
    return workgroups * 4 * iters * 16 * 16 * 16 * 32 * 2


def keyless_pack_weights(W_Q: torch.Tensor, W_R: torch.Tensor | None, W_V: torch.Tensor, H: int,
                         G: int, out: torch.Tensor | None = None) -> torch.Tensor:
    """Packed [(H+G)*d, d_model] bf16 weights: (W^Q W^R)^T over W^V^T, d_model contiguous."""
    load()
    d_model = W_Q.shape[0]
    dk = W_Q.shape[1] // H
    n = int(_lib.keyless_packed_weights_size(d_model, H, G, dk, _dt(W_Q)))
    if n == 0:
        raise KeylessError(KL_ERR_UNSUPPORTED, "packed weights are bf16 only")
    packed = out if out is not None else torch.empty(((H + G) * dk, d_model), dtype=W_Q.dtype,
                                                     device=W_Q.device)
    if packed.shape != ((H + G) * dk, d_model) or packed.dtype != W_Q.dtype:
        raise ValueError("out must be [(H + G) * d_head, d_model] in the weights' dtype")
    _check(_lib.keyless_pack_weights(_ptr(W_Q), _ptr(W_R), _ptr(W_V), d_model, H, G, dk, _dt(W_Q),
                                     _ptr(packed), _stream(W_Q)))
    return packed


def keyless_decode_project(x: torch.Tensor, packed: torch.Tensor, H: int, G: int,
                           cache: "ValueCache | None" = None, lengths_before=None,
                           q_routed_out=None, v_out=None, return_v: bool = False):
    """Decode-step projections q~ = x W~^Q [B, H, d], v = x W^V [B, G, d] from
    packed weights; with ``cache`` the values are also appended at lengths_before."""
    load()
    B, d_model = x.shape
    dk = packed.shape[0] // (H + G)
    if q_routed_out is None:
        q_routed_out = torch.empty((B, H, dk), dtype=x.dtype, device=x.device)
    if return_v and v_out is None:
        v_out = torch.empty((B, G, dk), dtype=x.dtype, device=x.device)
    _check(_lib.keyless_decode_project(_ptr(x), _ptr(packed), B, d_model, H, G, dk, _dt(x),
                                       _ptr(q_routed_out), _ptr(v_out),
                                       None if cache is None else cache.ref, _ptr(lengths_before),
                                       _stream(x)))
    if return_v:
        return q_routed_out, v_out
    return q_routed_out


def keyless_prefill_packed(x: torch.Tensor, packed: torch.Tensor, H: int, G: int,
                           causal: bool = True, scale: float = 0.0, return_qv: bool = False,
                           out=None, q_routed_out=None, v_out=None, workspace=None):
    """keyless_prefill with weights from keyless_pack_weights."""
    load()
    B, N, d_model = x.shape
    dk = packed.shape[0] // (H + G)
    if out is None:
        out = torch.empty((B, N, H, dk), dtype=x.dtype, device=x.device)
    if return_qv:
        if q_routed_out is None:
            q_routed_out = torch.empty((B, N, H, dk), dtype=x.dtype, device=x.device)
        if v_out is None:
            v_out = torch.empty((B, N, G, dk), dtype=x.dtype, device=x.device)
    need = 0
    if q_routed_out is None:
        need += -(-B * N * H * dk * 2 // 256) * 256
    if v_out is None:
        need += -(-B * N * G * dk * 2 // 256) * 256
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    _check(_lib.keyless_prefill_packed(_ptr(x), _ptr(packed), B, N, d_model, H, G, dk, int(causal),
                                       scale, _dt(x), _ptr(out), _ptr(q_routed_out), _ptr(v_out),
                                       _ptr(workspace), 0 if workspace is None else workspace.numel(),
                                       _stream(x)))
    if return_qv:
        return out, q_routed_out, v_out
    return out


def _cross_outputs(xa, xb, H, G, dk, return_qv, out, q_routed_out, v_out):
    B, Na, Nb = xa.shape[0], xa.shape[1], xb.shape[1]
    if out is None:
        out = torch.empty((B, Na, H, dk), dtype=xa.dtype, device=xa.device)
    if return_qv:
        if q_routed_out is None:
            q_routed_out = torch.empty((B, Na, H, dk), dtype=xa.dtype, device=xa.device)
        if v_out is None:
            v_out = torch.empty((B, Nb, G, dk), dtype=xa.dtype, device=xa.device)
    return out, q_routed_out, v_out


def keyless_cross_attention(xa: torch.Tensor, xb: torch.Tensor, W_Q: torch.Tensor,
                            W_R: torch.Tensor | None, W_V: torch.Tensor, H: int, G: int,
                            scale: float = 0.0, return_qv: bool = False, out=None,
                            q_routed_out=None, v_out=None, workspace=None):
    """Keyless cross-attention (queries from xa [B, N_a, d], values from xb
    [B, N_b, d]); returns out [B, N_a, H, d_k] (and Q~, V if return_qv)."""
    load()
    B, Na, d_model = xa.shape
    Nb = xb.shape[1]
    dk = W_Q.shape[1] // H
    out, q_routed_out, v_out = _cross_outputs(xa, xb, H, G, dk, return_qv, out, q_routed_out, v_out)
    need = int(_lib.keyless_cross_attention_workspace_size(
        B, Na, Nb, d_model, H, G, dk, _dt(xa), int(W_R is not None), int(q_routed_out is not None),
        int(v_out is not None)))
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=xa.device)
    _check(_lib.keyless_cross_attention(_ptr(xa), _ptr(xb), _ptr(W_Q), _ptr(W_R), _ptr(W_V), B, Na,
                                        Nb, d_model, H, G, dk, scale, _dt(xa), _ptr(out),
                                        _ptr(q_routed_out), _ptr(v_out), _ptr(workspace),
                                        workspace.numel(), _stream(xa)))
    if return_qv:
        return out, q_routed_out, v_out
    return out


def keyless_cross_attention_packed(xa: torch.Tensor, xb: torch.Tensor, packed: torch.Tensor,
                                   H: int, G: int, scale: float = 0.0, return_qv: bool = False,
                                   out=None, q_routed_out=None, v_out=None, workspace=None):
    """keyless_cross_attention with weights from keyless_pack_weights."""
    load()
    B, Na, d_model = xa.shape
    Nb = xb.shape[1]
    dk = packed.shape[0] // (H + G)
    out, q_routed_out, v_out = _cross_outputs(xa, xb, H, G, dk, return_qv, out, q_routed_out, v_out)
    need = 0
    if q_routed_out is None:
        need += -(-B * Na * H * dk * 2 // 256) * 256
    if v_out is None:
        need += -(-B * Nb * G * dk * 2 // 256) * 256
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=xa.device)
    _check(_lib.keyless_cross_attention_packed(_ptr(xa), _ptr(xb), _ptr(packed), B, Na, Nb, d_model,
                                               H, G, dk, scale, _dt(xa), _ptr(out),
                                               _ptr(q_routed_out), _ptr(v_out), _ptr(workspace),
                                               0 if workspace is None else workspace.numel(),
                                               _stream(xa)))
    if return_qv:
        return out, q_routed_out, v_out
    return out


def latent_decode_workspace_bytes(cache: "ValueCache", B: int, H: int, d_head: int) -> int:
    load()
    return int(_lib.keyless_latent_decode_workspace_size(cache.ref, B, H, d_head))


def keyless_latent_decode(q_routed: torch.Tensor, W_post: torch.Tensor, cache: "ValueCache",
                          lengths: torch.Tensor, scale: float = 0.0, out=None, workspace=None):
    """Decode over a latent value-only cache (r-wide rows): q* = q~ W_post^T,
    decode of q* at scale 1/sqrt(r), out = o* W_post. q_routed [B, H, d_k],
    W_post [H, r, d_k]; returns [B, H, d_k]."""
    load()
    B, H, dk = q_routed.shape
    if out is None:
        out = torch.empty_like(q_routed)
    if workspace is None:
        n = latent_decode_workspace_bytes(cache, B, H, dk)
        workspace = torch.empty(max(n, 256), dtype=torch.uint8, device=q_routed.device)
    _check(_lib.keyless_latent_decode(_ptr(q_routed), _ptr(W_post), cache.ref, _ptr(lengths), B, H,
                                      dk, scale, _ptr(out), _ptr(workspace), workspace.numel(),
                                      _stream(q_routed)))
    return out


def keyless_attention_forward(q_routed: torch.Tensor, v: torch.Tensor, causal: bool = True,
                              scale: float = 0.0, out=None, lse=None, out_f32=None):
    """Attention over projected routed queries [B, N, H, d] and values [B, N, G, d];
    returns (out, lse [B, H, N] fp32, the natural-log log-sum-exp per row). With
    out_f32 (a [B, N, H, d] fp32 tensor) the unrounded output is written too."""
    load()
    B, N, H, dk = q_routed.shape
    G = v.shape[2]
    if out is None:
        out = torch.empty_like(q_routed)
    if lse is None:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=q_routed.device)
    _check(_lib.keyless_attention_forward(_ptr(q_routed), _ptr(v), B, N, H, G, dk, int(causal),
                                          scale, _dt(q_routed), _ptr(out), _ptr(lse), _ptr(out_f32),
                                          _stream(q_routed)))
    return out, lse


def attention_backward_workspace_bytes(B: int, N: int, H: int) -> int:
    load()
    return int(_lib.keyless_attention_backward_workspace_size(B, N, H))


def keyless_attention_backward(q_routed: torch.Tensor, v: torch.Tensor, out: torch.Tensor,
                               dout: torch.Tensor, lse: torch.Tensor, causal: bool = True,
                               scale: float = 0.0, dq=None, dv=None, workspace=None, out_f32=None):
    """(dq_routed, dv) of the keyless attention from dout and the forward's out, lse
    (and its fp32 output, when kept)."""
    load()
    B, N, H, dk = q_routed.shape
    G = v.shape[2]
    if dq is None:
        dq = torch.empty_like(q_routed)
    if dv is None:
        dv = torch.empty_like(v)
    if workspace is None:
        n = int(_lib.keyless_attention_backward_workspace_size(B, N, H))
        workspace = torch.empty(max(n, 256), dtype=torch.uint8, device=q_routed.device)
    _check(_lib.keyless_attention_backward(_ptr(q_routed), _ptr(v), _ptr(out), _ptr(out_f32),
                                           _ptr(dout), _ptr(lse),
                                           B, N, H, G, dk, int(causal), scale, _dt(q_routed),
                                           _ptr(dq), _ptr(dv), _ptr(workspace), workspace.numel(),
                                           _stream(q_routed)))
    return dq, dv


def keyless_weight_gradients(x: torch.Tensor, W_Q: torch.Tensor, W_R: torch.Tensor,
                             W_V: torch.Tensor, dq_routed: torch.Tensor, dv: torch.Tensor,
                             H: int, G: int, workspace=None):
    """dict(dW_Q, dW_R, dW_V, dX) from the attention gradients (Eqs. 5 and 6)."""
    load()
    B, N, d_model = x.shape
    dk = W_Q.shape[1] // H
    res = dict(dW_Q=torch.empty_like(W_Q), dW_R=torch.empty_like(W_R), dW_V=torch.empty_like(W_V),
               dX=torch.empty_like(x))
    if workspace is None:
        n = int(_lib.keyless_weight_gradients_workspace_size(B, N, d_model, H, G, dk, _dt(x)))
        workspace = torch.empty(max(n, 256), dtype=torch.uint8, device=x.device)
    _check(_lib.keyless_weight_gradients(_ptr(x), _ptr(W_Q), _ptr(W_R), _ptr(W_V), _ptr(dq_routed),
                                         _ptr(dv), B, N, d_model, H, G, dk, _dt(x), _ptr(res["dW_Q"]),
                                         _ptr(res["dW_R"]), _ptr(res["dW_V"]), _ptr(res["dX"]),
                                         _ptr(workspace), workspace.numel(), _stream(x)))
    return res


def keyless_decode_append(q_routed: torch.Tensor, v_new: torch.Tensor, cache: ValueCache,
                          lengths_before: torch.Tensor, scale: float = 0.0, out=None,
                          workspace=None) -> torch.Tensor:
    """One decode step in one launch: v_new [B, G, d] joins the cache at
    lengths_before[b], and q~ [B, H, d] attends over lengths_before[b] + 1 rows."""
    load()
    B, H, _ = q_routed.shape
    if out is None:
        out = torch.empty_like(q_routed)
    if workspace is None:
        n = decode_workspace_bytes(cache, B, H)
        workspace = torch.empty(max(n, 256), dtype=torch.uint8, device=q_routed.device)
    _check(_lib.keyless_decode_append(_ptr(q_routed), _ptr(v_new), cache.ref, _ptr(lengths_before), B,
                                      H, scale, _ptr(out), _ptr(workspace), workspace.numel(),
                                      _stream(q_routed)))
    return out


def keyless_decode_noalloc(q_routed: torch.Tensor, cache: ValueCache, lengths: torch.Tensor,
                           scale: float = 0.0, out: torch.Tensor | None = None) -> torch.Tensor:
    """keyless_decode with the library's fixed scratch as its workspace (the
    call allocates no device memory; ``out`` may be passed in too)."""
    load()
    B, H, _ = q_routed.shape
    if lengths.dtype != torch.int32:
        raise TypeError("lengths must be int32")
    if out is None:
        out = torch.empty_like(q_routed)
    _check(_lib.keyless_decode_noalloc(_ptr(q_routed), cache.ref, _ptr(lengths), B, H, scale,
                                       _ptr(out), _stream(q_routed)))
    return out
