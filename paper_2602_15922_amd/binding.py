"""ctypes binding of libwamdit: argument marshalling only.

Every function here has the name of the C entry point it wraps, takes torch tensors
(device memory) and plain Python values, checks nothing the library does not check
itself, and raises ``WamError`` on a non-OK status.  Kernels are launched on torch's
current stream unless a stream is given.  There is no fallback: if the shared library
is missing, loading raises.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwamdit.so")

WAM_MAX_CHUNKS = 16
WAM_OK, WAM_EINVAL, WAM_EUNSUPPORTED, WAM_EWORKSPACE, WAM_EHIP = range(5)
WAM_EPI_BF16, WAM_EPI_GELU_BF16, WAM_EPI_RESID_F32, WAM_EPI_F32 = range(4)
WAM_SOLVER_EULER, WAM_SOLVER_UNIPC = range(2)
# the launches of a block that wam_step_io.block_events brackets (wam_block_event)
BLOCK_EVENT_NAMES = ("ln1", "qkv", "rope", "self_attn", "o", "lnc", "cq", "cross_attn", "co", "ln2", "ffn1", "ffn2")
WAM_BLOCK_EVENTS = len(BLOCK_EVENT_NAMES)

EXPORTED = (
    "wam_last_error", "wam_abi_version", "wam_attn_blockcausal", "wam_block_workspace_bytes",
    "wam_dit_block_fwd", "wam_step_workspace_bytes", "wam_dit_step_fwd",
    "wam_update_workspace_bytes", "wam_dit_update_fwd", "wam_flow_step", "wam_cosine_workspace_bytes",
    "wam_cosine_similarity", "wam_denoise_workspace_bytes", "wam_denoise_chunk", "wam_quantize_rows_fp8",
    "wam_gemm_fp8",
    "wam_time_embed_workspace_bytes", "wam_time_embed_fwd", "wam_text_proj_workspace_bytes",
    "wam_text_proj_fwd", "wam_adaln_ln_mod", "wam_rope_qkv", "wam_gemm_bf16",
    "wam_embed_workspace_bytes", "wam_embed_fwd", "wam_head_workspace_bytes", "wam_head_fwd",
    "wam_chunk_positions", "wam_rope_tables", "wam_attn_blockcausal_fp8", "wam_quantize_mx_fp8",
    "wam_quantize_scaled_fp8", "wam_rope_qkv_fp8", "wam_unipc_plan", "wam_unipc_step",
    "wam_cosine_similarity_noalloc", "wam_adaln_ln_mod_fp8", "wam_gemm_fp8_mx",
    "wam_attn_blockcausal_mx", "wam_attn_blockcausal_fp8_mx",
)

_vp, _fp, _i32, _i64, _sz = C.c_void_p, C.POINTER(C.c_float), C.c_int32, C.c_int64, C.c_size_t


class WamError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"libwamdit status {status}: {msg}")
        self.status = status


class wam_chunks(C.Structure):
    _fields_ = [("n_k_chunks", _i32), ("k_off", _i32 * (WAM_MAX_CHUNKS + 1)),
                ("n_q_chunks", _i32), ("q_off", _i32 * (WAM_MAX_CHUNKS + 1)),
                ("q_chunk_id", _i32 * WAM_MAX_CHUNKS)]


class wam_attn_desc(C.Structure):
    _fields_ = [("B", _i32), ("H", _i32), ("Dh", _i32), ("Lq", _i32), ("Lk", _i32),
                ("q_tok_stride", _i64), ("q_batch_stride", _i64),
                ("kv_tok_stride", _i64), ("kv_batch_stride", _i64),
                ("o_tok_stride", _i64), ("o_batch_stride", _i64),
                ("scale", C.c_float), ("ch", wam_chunks)]


class wam_dims(C.Structure):
    _fields_ = [(n, _i32) for n in ("d", "H", "Dh", "ffn", "n_layers", "latent_ch", "act_dim",
                                    "text_dim", "freq_dim")] + [("eps", C.c_float)]


BLOCK_MATS = ("w_qkv", "w_o", "w_cq", "w_ckv", "w_co", "w_f1", "w_f2")
BLOCK_VECS = ("b_qkv", "b_o", "b_cq", "b_ckv", "b_co", "b_f1", "b_f2", "mod6", "lnc_gamma", "lnc_beta")


class wam_block_fp8(C.Structure):
    _fields_ = [(n, _vp) for n in BLOCK_MATS] + [("s" + n[1:], _vp) for n in BLOCK_MATS]


class wam_block_weights(C.Structure):
    _fields_ = [(n, _vp) for n in BLOCK_MATS] + [(n, _vp) for n in BLOCK_VECS] + \
               [("fp8", C.POINTER(wam_block_fp8))]


class wam_block_io(C.Structure):
    _fields_ = [("x", _vp), ("e0", _vp), ("rope_cos", _vp), ("rope_sin", _vp),
                ("k_cache", _vp), ("v_cache", _vp), ("Lcap", _i32), ("cache_len", _i32),
                ("ch", wam_chunks), ("ctx", _vp), ("ctx_kv", _vp),
                ("B", _i32), ("L", _i32), ("Lc", _i32), ("k_exp", _vp), ("v_scale", C.c_float)]


MODEL_MATS = ("w_t1", "w_t2", "w_t6", "w_x1", "w_x2", "w_patch", "w_ain", "w_hv", "w_ha")
MODEL_VECS = ("b_t1", "b_t2", "b_t6", "b_x1", "b_x2", "b_patch", "b_ain", "b_hv", "b_ha")


class wam_model(C.Structure):
    _fields_ = ([("dims", wam_dims), ("blocks", C.POINTER(wam_block_weights))]
                + [(n, _vp) for n in MODEL_MATS] + [(n, _vp) for n in MODEL_VECS]
                + [("head_mod2", _vp)])


class wam_step_io(C.Structure):
    _fields_ = [("z_t", _vp), ("a_t", _vp), ("t", _vp), ("text", _vp),
                ("k_cache", C.POINTER(_vp)), ("v_cache", C.POINTER(_vp)), ("ctx_kv", C.POINTER(_vp)),
                ("rope_cos", _vp), ("rope_sin", _vp),
                ("B", _i32), ("F", _i32), ("Hl", _i32), ("Wl", _i32), ("A", _i32), ("Lc", _i32),
                ("Lcap", _i32), ("cache_len", _i32), ("ch", wam_chunks),
                ("v_video", _vp), ("v_action", _vp), ("attn_events", C.POINTER(_vp)), ("t_action", _vp),
                ("k_exp", C.POINTER(_vp)), ("v_scale", _fp), ("block_events", C.POINTER(_vp))]


class wam_flow_dims(C.Structure):
    _fields_ = [("B", _i32), ("cfg", _i32), ("cfg_scale", C.c_float), ("n_video", _i64), ("n_action", _i64)]


class wam_denoise_params(C.Structure):
    _fields_ = [("n_steps", _i32), ("t_sched", _fp), ("cfg", _i32), ("cfg_scale", C.c_float),
                ("cache_tau", C.c_float), ("cache_window", _i32), ("x", _vp), ("computed", C.POINTER(_i32)),
                ("solver", _i32), ("solver_order", _i32)]


class wam_unipc_coef(C.Structure):
    _fields_ = [("s_v", C.c_float), ("correct", _i32), ("c_x", C.c_float), ("c_new", C.c_float),
                ("c_m", C.c_float * 3), ("p_x", C.c_float), ("p_new", C.c_float), ("p_m", C.c_float * 2)]


class wam_gemm_desc(C.Structure):
    _fields_ = [("M", _i32), ("N", _i32), ("K", _i32), ("epilogue", _i32),
                ("A", _vp), ("lda", _i64), ("a_batch_stride", _i64), ("a_rows", _i32),
                ("W", _vp), ("ldw", _i64), ("bias", _vp),
                ("out", _vp), ("ldo", _i64), ("out_batch_stride", _i64), ("out_rows", _i32),
                ("gate_a", _vp), ("gate_v", _vp), ("gate_stride", _i64), ("gate_rows", _i32)]


_lib = None


def lib():
    """Load libwamdit.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        L.wam_last_error.restype = C.c_char_p
        L.wam_abi_version.restype = _i32
        for name in ("wam_block_workspace_bytes", "wam_step_workspace_bytes", "wam_update_workspace_bytes",
                     "wam_cosine_workspace_bytes", "wam_denoise_workspace_bytes",
                     "wam_time_embed_workspace_bytes", "wam_text_proj_workspace_bytes",
                     "wam_embed_workspace_bytes", "wam_head_workspace_bytes"):
            getattr(L, name).restype = _sz
        L.wam_block_workspace_bytes.argtypes = [C.POINTER(wam_dims), _i32, _i32, _i32]
        L.wam_step_workspace_bytes.argtypes = [C.POINTER(wam_model), C.POINTER(wam_step_io)]
        L.wam_update_workspace_bytes.argtypes = [C.POINTER(wam_model), C.POINTER(wam_step_io)]
        L.wam_time_embed_workspace_bytes.argtypes = [C.POINTER(wam_dims), _i32]
        L.wam_text_proj_workspace_bytes.argtypes = [C.POINTER(wam_dims), _i32, _i32]
        L.wam_embed_workspace_bytes.argtypes = [C.POINTER(wam_dims), _i32, _i32, _i32, _i32]
        L.wam_head_workspace_bytes.argtypes = [C.POINTER(wam_dims), _i32, _i32, _i32, _i32, _i32]
        L.wam_attn_blockcausal.argtypes = [C.POINTER(wam_attn_desc), _vp, _vp, _vp, _vp, _vp]
        L.wam_dit_block_fwd.argtypes = [C.POINTER(wam_dims), C.POINTER(wam_block_weights),
                                        C.POINTER(wam_block_io), _vp, _sz, _vp]
        L.wam_dit_step_fwd.argtypes = [C.POINTER(wam_model), C.POINTER(wam_step_io), _vp, _sz, _vp]
        L.wam_dit_update_fwd.argtypes = [C.POINTER(wam_model), C.POINTER(wam_step_io), _vp, _sz, _vp]
        L.wam_flow_step.argtypes = [C.POINTER(wam_flow_dims), _vp, _vp, _vp, _vp, _vp, C.c_float, C.c_float, _vp,
                                    _vp, _vp]
        L.wam_cosine_workspace_bytes.argtypes = []
        L.wam_cosine_similarity.argtypes = [_vp, _vp, _i64, _vp, _sz, _vp, _vp]
        L.wam_cosine_similarity_noalloc.argtypes = [_vp, _vp, _i64, _vp, _vp]
        L.wam_denoise_workspace_bytes.argtypes = [C.POINTER(wam_model), C.POINTER(wam_step_io),
                                                  C.POINTER(wam_denoise_params)]
        L.wam_denoise_chunk.argtypes = [C.POINTER(wam_model), C.POINTER(wam_step_io), C.POINTER(wam_denoise_params),
                                        _vp, _sz, _vp]
        L.wam_time_embed_fwd.argtypes = [C.POINTER(wam_model), _i32, _vp, _vp, _vp, _vp, _sz, _vp]
        L.wam_text_proj_fwd.argtypes = [C.POINTER(wam_model), _i32, _i32, _vp, _vp, _vp, _sz, _vp]
        L.wam_adaln_ln_mod.argtypes = [_i32, _i32, _i32, C.c_float, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                       _i64, _vp, _vp]
        L.wam_rope_qkv.argtypes = [_i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _i32, _i32, _vp]
        L.wam_gemm_bf16.argtypes = [C.POINTER(wam_gemm_desc), _vp]
        L.wam_gemm_fp8.argtypes = [C.POINTER(wam_gemm_desc), _vp, _vp, _vp]
        L.wam_gemm_fp8_mx.argtypes = [C.POINTER(wam_gemm_desc), _vp, _vp, _i64, _vp, _vp, _i64, _vp]
        L.wam_attn_blockcausal_mx.argtypes = [C.POINTER(wam_attn_desc), _vp, _vp, _vp, _vp, _vp, _i64, _vp]
        L.wam_attn_blockcausal_fp8_mx.argtypes = [C.POINTER(wam_attn_desc), _vp, _vp, _vp, _vp, _vp, C.c_float,
                                                  _vp, _vp, _i64, _vp]
        L.wam_quantize_rows_fp8.argtypes = [_i32, _i32, _vp, _i64, _vp, _i64, _vp, _vp]
        L.wam_adaln_ln_mod_fp8.argtypes = [_i32, _i32, _i32, C.c_float, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i64,
                                           _vp, _i64, _vp, _vp]
        L.wam_embed_fwd.argtypes = [C.POINTER(wam_model), _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp,
                                    _vp, _sz, _vp]
        L.wam_head_fwd.argtypes = [C.POINTER(wam_model), _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp,
                                   _vp, _vp, _sz, _vp]
        L.wam_chunk_positions.argtypes = [_i32, _i32, _i32, _i32, _i32, C.POINTER(_i32)]
        L.wam_rope_tables.argtypes = [C.POINTER(_i32), _i32, _i32, C.c_double, _fp, _fp]
        L.wam_attn_blockcausal_fp8.argtypes = [C.POINTER(wam_attn_desc), _vp, _vp, _vp, _vp, _vp, C.c_float, _vp,
                                               _vp]
        L.wam_quantize_mx_fp8.argtypes = [_i32, _i32, _vp, _i64, _vp, _i64, _vp, _vp]
        L.wam_quantize_scaled_fp8.argtypes = [_i64, _vp, C.c_float, _vp, _vp]
        L.wam_rope_qkv_fp8.argtypes = [_i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, C.c_float,
                                       _i32, _i32, _vp]
        L.wam_unipc_plan.argtypes = [_fp, _i32, _i32, C.POINTER(wam_unipc_coef)]
        L.wam_unipc_step.argtypes = [C.POINTER(wam_flow_dims), _vp, _vp, _vp, _vp, _vp, C.POINTER(_vp), _i32,
                                     C.POINTER(wam_unipc_coef), _vp, _vp, _vp, _vp]
        for name in EXPORTED[2:]:
            if not name.endswith("_bytes"):
                getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


def _check(status: int):
    if status != WAM_OK:
        raise WamError(status, lib().wam_last_error().decode())


def _p(t):
    """Device pointer of a tensor (None passes NULL)."""
    return None if t is None else t.data_ptr()


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


# ------------------------------------------------------------------------------------------
# chunk layouts
# ------------------------------------------------------------------------------------------
def make_chunks(k_sizes, q_sizes, q_ids) -> wam_chunks:
    """Key chunks of the given sizes (in key-row order); query chunks of the given sizes,
    query chunk i carrying global chunk id q_ids[i]."""
    c = wam_chunks()
    c.n_k_chunks = len(k_sizes)
    off = 0
    c.k_off[0] = 0
    for j, s in enumerate(k_sizes):
        off += int(s)
        c.k_off[j + 1] = off
    c.n_q_chunks = len(q_sizes)
    off = 0
    c.q_off[0] = 0
    for i, s in enumerate(q_sizes):
        off += int(s)
        c.q_off[i + 1] = off
        c.q_chunk_id[i] = int(q_ids[i])
    return c


def cached_chunks(cache_len: int, L: int) -> wam_chunks:
    """One query chunk of L rows after cache_len cached rows: everything visible."""
    if cache_len:
        return make_chunks([cache_len, L], [L], [1])
    return make_chunks([L], [L], [0])


def append_chunks(cached_sizes, new_sizes) -> wam_chunks:
    """Query chunks of the given sizes appended after cached chunks of the given sizes
    (global ids follow key-row order): the layout of a multi-chunk update pass."""
    n = len(cached_sizes)
    return make_chunks(list(cached_sizes) + list(new_sizes), list(new_sizes),
                       list(range(n, n + len(new_sizes))))


# ------------------------------------------------------------------------------------------
# entry points
# ------------------------------------------------------------------------------------------
def wam_abi_version() -> int:
    return lib().wam_abi_version()


def wam_attn_blockcausal(q, k, v, o, chunks: wam_chunks, scale: float = 0.0, stream=None):
    """q, o: [B, Lq, H, Dh] bf16 views; k, v: [B, Lk, H, Dh] bf16 views (token strides taken
    from the tensors; heads contiguous)."""
    B, Lq, H, Dh = q.shape
    d = wam_attn_desc(B=B, H=H, Dh=Dh, Lq=Lq, Lk=k.shape[1],
                      q_tok_stride=q.stride(1), q_batch_stride=q.stride(0),
                      kv_tok_stride=k.stride(1), kv_batch_stride=k.stride(0),
                      o_tok_stride=o.stride(1), o_batch_stride=o.stride(0), scale=scale, ch=chunks)
    if v.stride(1) != k.stride(1) or v.stride(0) != k.stride(0):
        raise ValueError("k and v must share token and batch strides")
    _check(lib().wam_attn_blockcausal(C.byref(d), _p(q), _p(k), _p(v), _p(o), _stream(stream)))


def wam_attn_blockcausal_fp8(q8, q_exp, k8, k_exp, v8, v_scale, o, chunks: wam_chunks, scale: float = 0.0,
                             stream=None):
    """FP8 attention (Dh = 128): q8 [B, Lq, H, 128] and k8, v8 [B, Lk, H, 128] uint8 E4M3 code
    views, q_exp [B, Lq, H] and k_exp [B, Lk, H] int32 block exponents (one byte per 32
    dims), o [B, Lq, H, 128] bf16; strides taken from the tensors."""
    B, Lq, H, Dh = q8.shape
    d = wam_attn_desc(B=B, H=H, Dh=Dh, Lq=Lq, Lk=k8.shape[1],
                      q_tok_stride=q8.stride(1), q_batch_stride=q8.stride(0),
                      kv_tok_stride=k8.stride(1), kv_batch_stride=k8.stride(0),
                      o_tok_stride=o.stride(1), o_batch_stride=o.stride(0), scale=scale, ch=chunks)
    if v8.stride(1) != k8.stride(1) or v8.stride(0) != k8.stride(0):
        raise ValueError("k8 and v8 must share token and batch strides")
    for e, c in ((q_exp, q8), (k_exp, k8)):
        if e.stride(1) * Dh != c.stride(1) or e.stride(0) * Dh != c.stride(0):
            raise ValueError("exponent strides must be the code strides / Dh")
    _check(lib().wam_attn_blockcausal_fp8(C.byref(d), _p(q8), _p(q_exp), _p(k8), _p(k_exp), _p(v8), v_scale,
                                          _p(o), _stream(stream)))


def wam_attn_blockcausal_mx(q, k, v, o8, o_exp, o_lde: int, chunks: wam_chunks, scale: float = 0.0, stream=None):
    """wam_attn_blockcausal with the output block-scaled: o8 [B, Lq, H, 128] uint8 E4M3 codes,
    o_exp uint8 (4 bytes per output row per head, stride o_lde between heads)."""
    B, Lq, H, Dh = q.shape
    d = wam_attn_desc(B=B, H=H, Dh=Dh, Lq=Lq, Lk=k.shape[1],
                      q_tok_stride=q.stride(1), q_batch_stride=q.stride(0),
                      kv_tok_stride=k.stride(1), kv_batch_stride=k.stride(0),
                      o_tok_stride=o8.stride(1), o_batch_stride=o8.stride(0), scale=scale, ch=chunks)
    if v.stride(1) != k.stride(1) or v.stride(0) != k.stride(0):
        raise ValueError("k and v must share token and batch strides")
    _check(lib().wam_attn_blockcausal_mx(C.byref(d), _p(q), _p(k), _p(v), _p(o8), _p(o_exp), o_lde,
                                         _stream(stream)))


def wam_attn_blockcausal_fp8_mx(q8, q_exp, k8, k_exp, v8, v_scale, o8, o_exp, o_lde: int, chunks: wam_chunks,
                                scale: float = 0.0, stream=None):
    """wam_attn_blockcausal_fp8 with the output block-scaled (o8 and o_exp as for
    wam_attn_blockcausal_mx)."""
    B, Lq, H, Dh = q8.shape
    d = wam_attn_desc(B=B, H=H, Dh=Dh, Lq=Lq, Lk=k8.shape[1],
                      q_tok_stride=q8.stride(1), q_batch_stride=q8.stride(0),
                      kv_tok_stride=k8.stride(1), kv_batch_stride=k8.stride(0),
                      o_tok_stride=o8.stride(1), o_batch_stride=o8.stride(0), scale=scale, ch=chunks)
    if v8.stride(1) != k8.stride(1) or v8.stride(0) != k8.stride(0):
        raise ValueError("k8 and v8 must share token and batch strides")
    _check(lib().wam_attn_blockcausal_fp8_mx(C.byref(d), _p(q8), _p(q_exp), _p(k8), _p(k_exp), _p(v8), v_scale,
                                             _p(o8), _p(o_exp), o_lde, _stream(stream)))


def wam_quantize_mx_fp8(x, q8, exps, stream=None):
    """MX-style E4M3 codes of bf16 rows x [M, K] (K % 32 == 0) into uint8 q8 [M, >=K] and
    uint8 exps [M, K/32] (biased block exponents)."""
    M, K = x.shape
    _check(lib().wam_quantize_mx_fp8(M, K, _p(x), x.stride(0), _p(q8), q8.stride(0), _p(exps), _stream(stream)))


def wam_quantize_scaled_fp8(x, scale, q8, stream=None):
    """One-scale E4M3 codes of a contiguous bf16 tensor into a uint8 tensor of the same size."""
    _check(lib().wam_quantize_scaled_fp8(x.numel(), _p(x), scale, _p(q8), _stream(stream)))


def wam_rope_qkv_fp8(qkv, cos_t, sin_t, q8, q_exp, k8_cache, k_exp, v8_cache, v_scale, row0, H, Dh, stream=None):
    """qkv [B, L, 3*H*Dh] bf16; code caches [B, Lcap, H, Dh] uint8, k_exp [B, Lcap, H] int32;
    q8 [B, L, H, Dh] uint8 and q_exp [B, L, H] int32 (or both None)."""
    B, L = qkv.shape[0], qkv.shape[1]
    _check(lib().wam_rope_qkv_fp8(B, L, H, Dh, _p(qkv), _p(cos_t), _p(sin_t), _p(q8), _p(q_exp), _p(k8_cache),
                                  _p(k_exp), _p(v8_cache), v_scale, k8_cache.shape[1], row0, _stream(stream)))


def wam_gemm_bf16(A, W, out, epilogue: int, bias=None, gate_a=None, gate_v=None, gate_stride=0,
                  gate_rows=0, M=None, lda=None, a_rows=0, a_batch_stride=0, ldo=None, out_rows=0,
                  out_batch_stride=0, stream=None):
    """out = epilogue(A W^T + bias); A [M, K] bf16, W [N, K] bf16 (row strides from the tensors
    unless given)."""
    N, K = W.shape
    g = wam_gemm_desc(M=A.shape[0] if M is None else M, N=N, K=K, epilogue=epilogue,
                      A=_p(A), lda=A.stride(0) if lda is None else lda, a_batch_stride=a_batch_stride,
                      a_rows=a_rows, W=_p(W), ldw=W.stride(0), bias=_p(bias), out=_p(out),
                      ldo=out.stride(0) if ldo is None else ldo, out_batch_stride=out_batch_stride,
                      out_rows=out_rows, gate_a=_p(gate_a), gate_v=_p(gate_v), gate_stride=gate_stride,
                      gate_rows=gate_rows)
    _check(lib().wam_gemm_bf16(C.byref(g), _stream(stream)))


def wam_quantize_rows_fp8(x, q, scale, stream=None):
    """Per-row E4M3 quantization of bf16 x [M, K] into uint8 q [M, >=K] and fp32 scale [M]."""
    M, K = x.shape
    _check(lib().wam_quantize_rows_fp8(M, K, _p(x), x.stride(0), _p(q), q.stride(0), _p(scale), _stream(stream)))


def wam_gemm_fp8(A, W, out, epilogue: int, a_scale, w_scale, bias=None, gate_a=None, gate_v=None, gate_stride=0,
                 gate_rows=0, M=None, lda=None, a_rows=0, a_batch_stride=0, ldo=None, out_rows=0,
                 out_batch_stride=0, stream=None):
    """out = epilogue((A8 W8^T) * a_scale[m] * w_scale[n] + bias); A [M, K] and W [N, K] uint8 E4M3 codes."""
    N, K = W.shape
    g = wam_gemm_desc(M=A.shape[0] if M is None else M, N=N, K=K, epilogue=epilogue,
                      A=_p(A), lda=A.stride(0) if lda is None else lda, a_batch_stride=a_batch_stride,
                      a_rows=a_rows, W=_p(W), ldw=W.stride(0), bias=_p(bias), out=_p(out),
                      ldo=out.stride(0) if ldo is None else ldo, out_batch_stride=out_batch_stride,
                      out_rows=out_rows, gate_a=_p(gate_a), gate_v=_p(gate_v), gate_stride=gate_stride,
                      gate_rows=gate_rows)
    _check(lib().wam_gemm_fp8(C.byref(g), _p(a_scale), _p(w_scale), _stream(stream)))


def wam_gemm_fp8_mx(A, W, out, epilogue: int, w_scale, a_scale=None, a_exp=None, a_lde=0, out_exp=None, o_lde=0,
                    bias=None, gate_a=None, gate_v=None, gate_stride=0, gate_rows=0, M=None, lda=None, ldo=None,
                    stream=None):
    """wam_gemm_fp8 with block-scaled activations: a_exp (uint8, 4 bytes per row per pair of
    64-column blocks, stride a_lde) instead of a_scale, or, with the GELU epilogue, the
    output as E4M3 codes in out (uint8) with its block exponents in out_exp (stride o_lde)."""
    N, K = W.shape
    g = wam_gemm_desc(M=A.shape[0] if M is None else M, N=N, K=K, epilogue=epilogue,
                      A=_p(A), lda=A.stride(0) if lda is None else lda, a_batch_stride=0, a_rows=0,
                      W=_p(W), ldw=W.stride(0), bias=_p(bias), out=_p(out),
                      ldo=out.stride(0) if ldo is None else ldo, out_batch_stride=0, out_rows=0,
                      gate_a=_p(gate_a), gate_v=_p(gate_v), gate_stride=gate_stride, gate_rows=gate_rows)
    _check(lib().wam_gemm_fp8_mx(C.byref(g), _p(a_scale), _p(a_exp), a_lde, _p(w_scale), _p(out_exp), o_lde,
                                 _stream(stream)))


def wam_adaln_ln_mod(x, h, eps, rows_per_batch, gamma=None, beta=None, shift_a=None, shift_v=None,
                     scale_a=None, scale_v=None, mod_stride=0, stream=None):
    d = x.shape[-1]
    rows = x.numel() // d
    B = rows // rows_per_batch if rows_per_batch else 0
    _check(lib().wam_adaln_ln_mod(B, rows_per_batch, d, eps, _p(x), _p(gamma), _p(beta), _p(shift_a),
                                  _p(shift_v), _p(scale_a), _p(scale_v), mod_stride, _p(h), _stream(stream)))


def wam_adaln_ln_mod_fp8(x, q, scale, eps, rows_per_batch, gamma=None, beta=None, shift_a=None, shift_v=None,
                         scale_a=None, scale_v=None, mod_stride=0, stream=None):
    """The LayerNorm of wam_adaln_ln_mod written as E4M3 codes q [rows, >=d] uint8 (row stride
    from the tensor) and row scales scale [rows] fp32."""
    d = x.shape[-1]
    rows = x.numel() // d
    B = rows // rows_per_batch if rows_per_batch else 0
    _check(lib().wam_adaln_ln_mod_fp8(B, rows_per_batch, d, eps, _p(x), _p(gamma), _p(beta), _p(shift_a),
                                      _p(shift_v), _p(scale_a), _p(scale_v), mod_stride, _p(q), q.stride(0),
                                      _p(scale), _stream(stream)))


def wam_rope_qkv(qkv, cos_t, sin_t, q_out, k_cache, v_cache, row0, H, Dh, stream=None):
    """qkv [B, L, 3*H*Dh] bf16; caches [B, Lcap, H, Dh] bf16."""
    B, L = qkv.shape[0], qkv.shape[1]
    _check(lib().wam_rope_qkv(B, L, H, Dh, _p(qkv), _p(cos_t), _p(sin_t), _p(q_out), _p(k_cache),
                              _p(v_cache), k_cache.shape[1], row0, _stream(stream)))


def make_dims(d, H, Dh, ffn, n_layers, latent_ch=16, act_dim=16, text_dim=4096, freq_dim=256, eps=1e-6):
    return wam_dims(d=d, H=H, Dh=Dh, ffn=ffn, n_layers=n_layers, latent_ch=latent_ch, act_dim=act_dim,
                    text_dim=text_dim, freq_dim=freq_dim, eps=eps)


def make_block_weights(t: dict) -> wam_block_weights:
    """t: name -> device tensor (missing vectors = NULL); t["fp8"], when present, the dict
    make_block_fp8 returns (the block's projections then run as FP8 GEMMs)."""
    w = wam_block_weights()
    for n in BLOCK_MATS + BLOCK_VECS:
        setattr(w, n, _p(t.get(n)))
    f8 = t.get("fp8")
    if f8 is not None:
        f = wam_block_fp8()
        for n in BLOCK_MATS:
            setattr(f, n, _p(f8.get(n)))
            setattr(f, "s" + n[1:], _p(f8.get("s" + n[1:])))
        w.fp8 = C.pointer(f)
        w._fp8 = f
    return w


def make_block_fp8(t: dict, stream=None) -> dict:
    """E4M3 copies of a block's bf16 projection matrices (device tensors in t), one scale per
    output channel, made on the device with wam_quantize_rows_fp8."""
    import torch
    out = {}
    for n in BLOCK_MATS:
        if t.get(n) is None:
            continue
        W = t[n]
        N, K = W.shape
        q = torch.empty((N, K), dtype=torch.uint8, device=W.device)
        s = torch.empty(N, dtype=torch.float32, device=W.device)
        wam_quantize_rows_fp8(W, q, s, stream=stream)
        out[n], out["s" + n[1:]] = q, s
    return out


def make_model(dims: wam_dims, top: dict, blocks: list) -> wam_model:
    m = wam_model()
    m.dims = dims
    ws = [make_block_weights(b) for b in blocks]
    arr = (wam_block_weights * max(1, len(blocks)))(*ws)
    m.blocks = C.cast(arr, C.POINTER(wam_block_weights))
    m._keep = (arr, ws)  # keep the host arrays (and any FP8 structs) alive with the model
    for n in MODEL_MATS + MODEL_VECS + ("head_mod2",):
        setattr(m, n, _p(top.get(n)))
    return m


def wam_block_workspace_bytes(dims: wam_dims, B: int, L: int, Lc: int) -> int:
    return lib().wam_block_workspace_bytes(C.byref(dims), B, L, Lc)


def wam_dit_block_fwd(dims: wam_dims, weights: wam_block_weights, x, e0, rope_cos, rope_sin, k_cache,
                      v_cache, cache_len, chunks: wam_chunks, ctx=None, ctx_kv=None, ws=None, stream=None):
    """x [B, L, d] fp32 (in place); caches [B, Lcap, H, Dh] bf16; ctx [B, Lc, d] bf16 or ctx_kv
    [B, Lc, 2d]; ws a uint8 device tensor of at least wam_block_workspace_bytes."""
    B, L = x.shape[0], x.shape[1]
    Lc = (ctx if ctx is not None else ctx_kv).shape[1]
    io = wam_block_io(x=_p(x), e0=_p(e0), rope_cos=_p(rope_cos), rope_sin=_p(rope_sin),
                      k_cache=_p(k_cache), v_cache=_p(v_cache), Lcap=k_cache.shape[1], cache_len=cache_len,
                      ch=chunks, ctx=_p(ctx), ctx_kv=_p(ctx_kv), B=B, L=L, Lc=Lc)
    _check(lib().wam_dit_block_fwd(C.byref(dims), C.byref(weights), C.byref(io), _p(ws),
                                   0 if ws is None else ws.numel(), _stream(stream)))


def wam_time_embed_workspace_bytes(dims: wam_dims, B: int) -> int:
    return lib().wam_time_embed_workspace_bytes(C.byref(dims), B)


def wam_time_embed_fwd(model: wam_model, t, e, e0, ws, stream=None):
    _check(lib().wam_time_embed_fwd(C.byref(model), t.shape[0], _p(t), _p(e), _p(e0), _p(ws), ws.numel(),
                                    _stream(stream)))


def wam_text_proj_workspace_bytes(dims: wam_dims, B: int, Lc: int) -> int:
    return lib().wam_text_proj_workspace_bytes(C.byref(dims), B, Lc)


def wam_text_proj_fwd(model: wam_model, text, ctx, ws, stream=None):
    B, Lc = text.shape[0], text.shape[1]
    _check(lib().wam_text_proj_fwd(C.byref(model), B, Lc, _p(text), _p(ctx), _p(ws), ws.numel(),
                                   _stream(stream)))


def wam_embed_workspace_bytes(dims: wam_dims, B, F, Hl, Wl) -> int:
    return lib().wam_embed_workspace_bytes(C.byref(dims), B, F, Hl, Wl)


def wam_embed_fwd(model: wam_model, z_t, a_t, x, ws, stream=None):
    B, _, F, Hl, Wl = z_t.shape
    A = a_t.shape[1] if a_t is not None else 0
    _check(lib().wam_embed_fwd(C.byref(model), B, F, Hl, Wl, A, _p(z_t), _p(a_t), _p(x), _p(ws), ws.numel(),
                               _stream(stream)))


def wam_head_workspace_bytes(dims: wam_dims, B, F, Hl, Wl, A) -> int:
    return lib().wam_head_workspace_bytes(C.byref(dims), B, F, Hl, Wl, A)


def wam_head_fwd(model: wam_model, x, e, v_video, v_action, ws, stream=None):
    B, _, F, Hl, Wl = v_video.shape
    A = v_action.shape[1] if v_action is not None else 0
    _check(lib().wam_head_fwd(C.byref(model), B, F, Hl, Wl, A, _p(x), _p(e), _p(v_video), _p(v_action),
                              _p(ws), ws.numel(), _stream(stream)))


def _ptr_array(ts):
    return (_vp * len(ts))(*[_p(t) for t in ts])


def make_step_io(z_t, a_t, t, text, k_caches, v_caches, rope_cos, rope_sin, cache_len, chunks, v_video,
                 v_action, ctx_kv=None, events=None, t_action=None, k_exps=None, v_scales=None,
                 block_events=None) -> wam_step_io:
    """Step inputs/outputs; with k_exps (per-layer [B, Lcap, H] int32) and v_scales (per-layer
    floats) the caches are FP8 code caches and the self-attention runs in FP8.  events: the
    2*n_layers self-attention events; block_events: 2*WAM_BLOCK_EVENTS*n_layers torch events
    around every launch of every block."""
    B, _, F, Hl, Wl = z_t.shape
    io = wam_step_io(z_t=_p(z_t), a_t=_p(a_t), t=_p(t), text=_p(text), rope_cos=_p(rope_cos),
                     rope_sin=_p(rope_sin), B=B, F=F, Hl=Hl, Wl=Wl, A=a_t.shape[1], Lc=text.shape[1],
                     Lcap=k_caches[0].shape[1] if k_caches else 0, cache_len=cache_len, ch=chunks,
                     v_video=_p(v_video), v_action=_p(v_action), t_action=_p(t_action))
    kc, vc = _ptr_array(k_caches), _ptr_array(v_caches)
    io.k_cache = C.cast(kc, C.POINTER(_vp))
    io.v_cache = C.cast(vc, C.POINTER(_vp))
    keep = [kc, vc]
    if ctx_kv is not None:
        ck = _ptr_array(ctx_kv)
        io.ctx_kv = C.cast(ck, C.POINTER(_vp))
        keep.append(ck)
    if k_exps is not None:
        ke = _ptr_array(k_exps)
        vs = (C.c_float * len(v_scales))(*[float(v) for v in v_scales])
        io.k_exp = C.cast(ke, C.POINTER(_vp))
        io.v_scale = C.cast(vs, _fp)
        keep += [ke, vs]
    if events is not None:
        # torch's Event.elapsed_time() only reads events torch has seen recorded; record
        # each once here so the library's later hipEventRecord on them can be read back.
        for e in events:
            e.record()
        ev = (_vp * len(events))(*[e.cuda_event for e in events])
        io.attn_events = C.cast(ev, C.POINTER(_vp))
        keep.append(ev)
    if block_events is not None:
        for e in block_events:
            e.record()
        bev = (_vp * len(block_events))(*[e.cuda_event for e in block_events])
        io.block_events = C.cast(bev, C.POINTER(_vp))
        keep.append(bev)
    io._keep = keep
    return io


def wam_step_workspace_bytes(model: wam_model, io: wam_step_io) -> int:
    return lib().wam_step_workspace_bytes(C.byref(model), C.byref(io))


def wam_dit_step_fwd(model: wam_model, io: wam_step_io, ws, stream=None):
    _check(lib().wam_dit_step_fwd(C.byref(model), C.byref(io), _p(ws), ws.numel(), _stream(stream)))


def wam_update_workspace_bytes(model: wam_model, io: wam_step_io) -> int:
    return lib().wam_update_workspace_bytes(C.byref(model), C.byref(io))


def wam_dit_update_fwd(model: wam_model, io: wam_step_io, ws, stream=None):
    """Cache-update pass: appends every layer's K/V of the io's clean rows at
    [cache_len, cache_len + L); v_video / v_action of io are not written."""
    _check(lib().wam_dit_update_fwd(C.byref(model), C.byref(io), _p(ws), ws.numel(), _stream(stream)))


def wam_flow_step(dims: wam_flow_dims, x, z_next, a_next, t, t_next, v_video=None, v_action=None, v_in=None,
                  v_out=None, stream=None):
    _check(lib().wam_flow_step(C.byref(dims), _p(v_video), _p(v_action), _p(v_in), _p(x), _p(v_out), t, t_next,
                               _p(z_next), _p(a_next), _stream(stream)))


def wam_cosine_workspace_bytes() -> int:
    return lib().wam_cosine_workspace_bytes()


def wam_cosine_similarity(a, b, out, ws, stream=None):
    """out[0] = cos(a, b) over all elements (device fp32 tensors)."""
    _check(lib().wam_cosine_similarity(_p(a), _p(b), a.numel(), _p(ws), ws.numel(), _p(out), _stream(stream)))


def wam_cosine_similarity_noalloc(a, b, out, stream=None):
    """out[0] = cos(a, b), partial sums in the library's static scratch (no workspace)."""
    _check(lib().wam_cosine_similarity_noalloc(_p(a), _p(b), a.numel(), _p(out), _stream(stream)))


def wam_unipc_plan(t_sched, order=2):
    """Host: the UniPC weights of every step of the schedule (N+1 times), a ctypes array."""
    import numpy as np
    t = np.ascontiguousarray(np.asarray(t_sched, dtype=np.float32))
    n = len(t) - 1
    out = (wam_unipc_coef * max(n, 1))()
    _check(lib().wam_unipc_plan(t.ctypes.data_as(_fp), n, order, out))
    return out


def wam_unipc_step(dims: wam_flow_dims, v_video, v_action, v_in, x, x_last, m_ring, step, coef, v_out,
                   z_next, a_next, stream=None):
    """One UniPC step (device tensors; m_ring a list of 4 state-sized fp32 tensors, coef one
    wam_unipc_coef of wam_unipc_plan's output)."""
    ring = (_vp * 4)(*[_p(t) for t in m_ring])
    _check(lib().wam_unipc_step(C.byref(dims), _p(v_video), _p(v_action), _p(v_in), _p(x), _p(x_last), ring,
                                step, C.byref(coef), _p(v_out), _p(z_next), _p(a_next), _stream(stream)))


def make_denoise_params(t_sched, x, cfg=False, cfg_scale=1.0, cache_tau=0.0, cache_window=0,
                        solver=WAM_SOLVER_EULER, order=2):
    """Loop parameters; t_sched a float sequence of N+1 times (kept on the host), x the
    device state, solver WAM_SOLVER_EULER or WAM_SOLVER_UNIPC (of the given order).
    `p.computed` is a device int32 [N] tensor the loop fills with 1 where a step called
    the network (read it after the stream has finished)."""
    import numpy as np
    import torch
    t = np.ascontiguousarray(np.asarray(t_sched, dtype=np.float32))
    n = len(t) - 1
    computed = torch.zeros(n, dtype=torch.int32, device=x.device)
    p = wam_denoise_params(n_steps=n, t_sched=t.ctypes.data_as(_fp), cfg=int(cfg), cfg_scale=cfg_scale,
                           cache_tau=cache_tau, cache_window=cache_window, x=_p(x),
                           computed=C.cast(C.c_void_p(computed.data_ptr()), C.POINTER(_i32)),
                           solver=solver, solver_order=order)
    p._keep = (t, computed)
    p.computed_steps = computed
    return p


def wam_denoise_workspace_bytes(model: wam_model, io: wam_step_io, params: wam_denoise_params) -> int:
    return lib().wam_denoise_workspace_bytes(C.byref(model), C.byref(io), C.byref(params))


def wam_denoise_chunk(model: wam_model, io: wam_step_io, params: wam_denoise_params, ws, stream=None):
    _check(lib().wam_denoise_chunk(C.byref(model), C.byref(io), C.byref(params), _p(ws), ws.numel(),
                                   _stream(stream)))


def wam_chunk_positions(c, F, Hg, Wg, A):
    """Host: (L, 3) int32 positions of chunk c (a numpy array)."""
    import numpy as np
    L = F * Hg * Wg + A
    pos = np.zeros((L, 3), np.int32)
    _check(lib().wam_chunk_positions(c, F, Hg, Wg, A, pos.ctypes.data_as(C.POINTER(_i32))))
    return pos


def wam_rope_tables(pos, Dh, theta=10000.0):
    """Host: cos, sin float32 arrays (L, Dh/2) for int positions (L, 3)."""
    import numpy as np
    pos = np.ascontiguousarray(pos, dtype=np.int32)
    L = pos.shape[0]
    cos = np.zeros((L, Dh // 2), np.float32)
    sin = np.zeros((L, Dh // 2), np.float32)
    _check(lib().wam_rope_tables(pos.ctypes.data_as(C.POINTER(_i32)), L, Dh, theta,
                                 cos.ctypes.data_as(_fp), sin.ctypes.data_as(_fp)))
    return cos, sin
