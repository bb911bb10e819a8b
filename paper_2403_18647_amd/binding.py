"""ctypes binding of ``libsdsat.so`` (C-ABI in include/sdsat.h).

Argument marshalling only: every step of the decode path runs in the HIP
library.  PyTorch provides device memory (tensors) and the HIP stream.  The
functions carry the C names; ``Context`` bundles a context with the
workspace and weight tensors it must keep alive.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsdsat.so")

SDSAT_OK = 0
ERRORS = {-1: "EINVAL", -2: "ENOMEM", -3: "EDEVICE", -4: "ECAPACITY", -5: "EUNSUPPORTED", -6: "EDATA"}
DTYPE_FP32, DTYPE_BF16 = 0, 1
MODE_GREEDY, MODE_NUCLEUS = 0, 1
PROFILE_KINDS = {"off": 0, "gateup": 1, "qkv": 2, "attention": 3, "down": 4, "o": 5, "lm_head": 6, "block": 7,
                 "prefill": 8}


class sdsat_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ffn", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("n_adaptive", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float),
                ("dtype", ctypes.c_int32), ("max_batch", ctypes.c_int32), ("max_ctx", ctypes.c_int32),
                ("max_block", ctypes.c_int32)]


class sdsat_stats(ctypes.Structure):
    _fields_ = [("loops", ctypes.c_int64), ("blocks", ctypes.c_int64), ("prefill_blocks", ctypes.c_int64),
                ("tokens", ctypes.c_int64), ("accepted", ctypes.c_int64),
                ("accept_hist", ctypes.c_int64 * 65), ("prefill_ms", ctypes.c_double),
                ("decode_ms", ctypes.c_double)]


_VP, _I32, _I64, _F32, _U64, _SZ = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                   ctypes.c_uint64, ctypes.c_size_t)
_SIGNATURES = {
    "sdsat_query_sizes": ([ctypes.POINTER(sdsat_config), ctypes.POINTER(_SZ)], _I32),
    "sdsat_init": ([ctypes.POINTER(sdsat_config), ctypes.POINTER(_VP), _I32, _VP, _SZ, _VP, ctypes.POINTER(_VP)], _I32),
    "sdsat_reset": ([_VP, _I32], _I32),
    "sdsat_set_cache_len": ([_VP, _I32, ctypes.POINTER(_I32)], _I32),
    "sdsat_cache_len_ptr": ([_VP], _VP),
    "sdsat_forward_block": ([_VP, _I32, _I32, _VP, _VP, _VP], _I32),
    "sdsat_verify_greedy": ([_VP, _I32, _I32, _VP, _VP, _VP, _VP], _I32),
    "sdsat_verify_nucleus": ([_VP, _I32, _I32, _VP, _VP, _F32, _F32, _I32, _U64, _VP, _VP, _VP], _I32),
    "sdsat_commit_kv": ([_VP, _I32, _I32, _VP, _VP], _I32),
    "sdsat_generate": ([_VP, _I32, ctypes.POINTER(_I32), _I32, _I32, _I32, ctypes.POINTER(_I32), _I32, _F32, _F32,
                        _I32, _U64, ctypes.POINTER(_I32), ctypes.POINTER(sdsat_stats)], _I32),
    "sdsat_generate_tree": ([_VP, _I32, ctypes.POINTER(_I32), _I32, _I32, _I32, _I32, ctypes.POINTER(_I32), _I32,
                             _F32, _F32, _I32, _U64, ctypes.POINTER(_I32), ctypes.POINTER(sdsat_stats)], _I32),
    "sdsat_generate_forced": ([_VP, _I32, ctypes.POINTER(_I32), _I32, _I32, _I32, ctypes.POINTER(_I32), _I32, _F32,
                               _F32, _I32, _U64, ctypes.POINTER(_I32), _I32, ctypes.POINTER(_I32),
                               ctypes.POINTER(sdsat_stats)], _I32),
    "sdsat_kv_write": ([_VP, _I32, _I32, _I32, _VP, _VP, _VP], _I32),
    "sdsat_attention": ([_VP, _I32, _I32, _I32, _VP, _VP, _VP], _I32),
    "sdsat_linear_packed_bytes": ([_I32, _I32, _I32], _SZ),
    "sdsat_linear_pack": ([_I32, _I32, _I32, _VP, _VP, _VP], _I32),
    "sdsat_linear_scratch_bytes": ([_I32, _I32, _I32], _SZ),
    "sdsat_linear": ([_I32, _I32, _I32, _I32, _VP, _VP, _VP, _VP, _VP], _I32),
    "sdsat_linear_noalloc": ([_I32, _I32, _I32, _I32, _VP, _VP, _VP, _VP], _I32),
    "sdsat_profile_kernel": ([_VP, _I32, _I32], _I32),
    "sdsat_kernel_time": ([_VP, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_I64)], _I32),
    "sdsat_kernel_samples": ([_VP, ctypes.POINTER(ctypes.c_float), _I64, ctypes.POINTER(_I64)], _I32),
    "sdsat_stream_read": ([_VP, _SZ, _VP], _I32),
    "sdsat_destroy": ([_VP], _I32),
    "sdsat_last_error": ([_VP], ctypes.c_char_p),
}
EXPORTS = tuple(_SIGNATURES)

_lib = None


def lib():
    """Load libsdsat.so (raises if it has not been built: there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGNATURES.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


class SdsatError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"sdsat error {ERRORS.get(code, code)}: {msg}")
        self.code = code


def _check(rc: int, ctx=None) -> None:
    if rc != SDSAT_OK:
        msg = lib().sdsat_last_error(ctx)
        raise SdsatError(rc, msg.decode() if msg else "")


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def make_config(shape, max_batch: int, max_ctx: int, max_block: int) -> sdsat_config:
    """Config from any object with the shape fields of ``synth.ModelShape``."""
    return sdsat_config(shape.n_layers, shape.d_model, shape.n_heads, shape.head_dim, shape.d_ffn, shape.vocab,
                        shape.n_adaptive, shape.rms_eps, shape.rope_base,
                        DTYPE_BF16 if shape.dtype == "bf16" else DTYPE_FP32, max_batch, max_ctx, max_block)


# ------------------------------------------------------------------ C names
def sdsat_query_sizes(cfg: sdsat_config) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().sdsat_query_sizes(ctypes.byref(cfg), ctypes.byref(n)))
    return n.value


def sdsat_init(cfg, weights, workspace, stream=None):
    arr = (ctypes.c_void_p * len(weights))(*[_ptr(w) for w in weights])
    out = ctypes.c_void_p()
    _check(lib().sdsat_init(ctypes.byref(cfg), arr, len(weights), _ptr(workspace), workspace.numel(),
                            _stream(stream), ctypes.byref(out)))
    return out


def sdsat_reset(ctx, batch):
    _check(lib().sdsat_reset(ctx, batch), ctx)


def sdsat_set_cache_len(ctx, lengths):
    a = np.ascontiguousarray(lengths, np.int32)
    _check(lib().sdsat_set_cache_len(ctx, a.size, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))), ctx)


def sdsat_cache_len_ptr(ctx) -> int:
    return lib().sdsat_cache_len_ptr(ctx)


def sdsat_forward_block(ctx, batch, q, tokens, mask=None, logits=None):
    _check(lib().sdsat_forward_block(ctx, batch, q, _ptr(tokens), _ptr(mask), _ptr(logits)), ctx)


def sdsat_verify_greedy(ctx, batch, q, logits, drafts, tokens_out, n_accept):
    _check(lib().sdsat_verify_greedy(ctx, batch, q, _ptr(logits), _ptr(drafts), _ptr(tokens_out),
                                     _ptr(n_accept)), ctx)


def sdsat_verify_nucleus(ctx, batch, q, logits, drafts, temperature, top_p, top_k, seed, pos0, tokens_out,
                         n_accept):
    _check(lib().sdsat_verify_nucleus(ctx, batch, q, _ptr(logits), _ptr(drafts), temperature, top_p, top_k,
                                      seed, _ptr(pos0), _ptr(tokens_out), _ptr(n_accept)), ctx)


def sdsat_commit_kv(ctx, batch, q, n_commit, rows=None):
    _check(lib().sdsat_commit_kv(ctx, batch, q, _ptr(n_commit), _ptr(rows)), ctx)


def sdsat_generate(ctx, prompts, max_new, k, adaptive_ids, mode=MODE_GREEDY, temperature=0.0, top_p=1.0,
                   top_k=0, seed=0, ref=None, width=1):
    """prompts: host int32 [batch, P].  Returns (tokens int32 [batch, max_new], stats dict).  With ref
    (host int32 [batch, ref_len]) calls sdsat_generate_forced: draft step 2 takes its drafts from ref.
    With width > 1 calls sdsat_generate_tree (draft tree of that width)."""
    p = np.ascontiguousarray(prompts, np.int32)
    batch, P = p.shape
    ad = np.ascontiguousarray(adaptive_ids if k else np.zeros(1), np.int32)
    out = np.zeros((batch, max_new), np.int32)
    st = sdsat_stats()
    ip = ctypes.POINTER(ctypes.c_int32)
    if width > 1:
        if ref is not None:
            raise ValueError("ref and width > 1 cannot be combined")
        _check(lib().sdsat_generate_tree(ctx, batch, p.ctypes.data_as(ip), P, max_new, k, width,
                                         ad.ctypes.data_as(ip), mode, temperature, top_p, top_k, seed,
                                         out.ctypes.data_as(ip), ctypes.byref(st)), ctx)
    elif ref is None:
        _check(lib().sdsat_generate(ctx, batch, p.ctypes.data_as(ip), P, max_new, k, ad.ctypes.data_as(ip), mode,
                                    temperature, top_p, top_k, seed, out.ctypes.data_as(ip), ctypes.byref(st)), ctx)
    else:
        r = np.ascontiguousarray(ref, np.int32)
        if r.ndim != 2 or r.shape[0] != batch:
            raise ValueError("ref must be [batch, ref_len]")
        _check(lib().sdsat_generate_forced(ctx, batch, p.ctypes.data_as(ip), P, max_new, k, ad.ctypes.data_as(ip),
                                           mode, temperature, top_p, top_k, seed, r.ctypes.data_as(ip), r.shape[1],
                                           out.ctypes.data_as(ip), ctypes.byref(st)), ctx)
    stats = {"loops": st.loops, "blocks": st.blocks, "prefill_blocks": st.prefill_blocks, "tokens": st.tokens,
             "accepted": st.accepted, "accept_hist": list(st.accept_hist)[: k + 1],
             "prefill_ms": st.prefill_ms, "decode_ms": st.decode_ms}
    return out, stats


def sdsat_kv_write(ctx, layer, batch, n, k, v, pos):
    _check(lib().sdsat_kv_write(ctx, layer, batch, n, _ptr(k), _ptr(v), _ptr(pos)), ctx)


def sdsat_attention(ctx, layer, batch, q, qin, mask, out):
    _check(lib().sdsat_attention(ctx, layer, batch, q, _ptr(qin), _ptr(mask), _ptr(out)), ctx)


def sdsat_linear_packed_bytes(dtype, N, K) -> int:
    return lib().sdsat_linear_packed_bytes(dtype, N, K)


def sdsat_linear_pack(dtype, N, K, w, packed, stream=None):
    _check(lib().sdsat_linear_pack(dtype, N, K, _ptr(w), _ptr(packed), _stream(stream)))


def sdsat_linear_scratch_bytes(M, N, K) -> int:
    return lib().sdsat_linear_scratch_bytes(M, N, K)


def sdsat_linear(dtype, M, N, K, x, packed, y, scratch, stream=None):
    _check(lib().sdsat_linear(dtype, M, N, K, _ptr(x), _ptr(packed), _ptr(y), _ptr(scratch), _stream(stream)))


def sdsat_linear_noalloc(dtype, M, N, K, x, packed, y, stream=None):
    _check(lib().sdsat_linear_noalloc(dtype, M, N, K, _ptr(x), _ptr(packed), _ptr(y), _stream(stream)))


def sdsat_profile_kernel(ctx, kind, period=1):
    _check(lib().sdsat_profile_kernel(ctx, PROFILE_KINDS.get(kind, kind), period), ctx)


def sdsat_kernel_time(ctx):
    ms = ctypes.c_double(0)
    n = ctypes.c_int64(0)
    _check(lib().sdsat_kernel_time(ctx, ctypes.byref(ms), ctypes.byref(n)), ctx)
    return ms.value, n.value


def sdsat_kernel_samples(ctx, cap=1 << 16):
    """Milliseconds of each timed launch since the last call (a list, launch order)."""
    buf = (ctypes.c_float * cap)()
    n = ctypes.c_int64(0)
    _check(lib().sdsat_kernel_samples(ctx, buf, cap, ctypes.byref(n)), ctx)
    return [buf[i] for i in range(min(cap, n.value))]


def sdsat_stream_read(src, nbytes=None, stream=None):
    """Stream nbytes (default: all) of the device tensor src with the library's read-only kernel."""
    nbytes = src.numel() * src.element_size() if nbytes is None else nbytes
    _check(lib().sdsat_stream_read(_ptr(src), nbytes, _stream(stream)))


def sdsat_destroy(ctx):
    _check(lib().sdsat_destroy(ctx))


# ------------------------------------------------------------------ convenience
class Context:
    """A library context plus the device tensors it needs kept alive."""

    def __init__(self, cfg: sdsat_config, weights, device="cuda"):
        import torch
        self.cfg = cfg
        self.weights = list(weights)
        self.workspace = torch.empty(sdsat_query_sizes(cfg), dtype=torch.uint8, device=device)
        self.stream = torch.cuda.current_stream(device)
        self.handle = sdsat_init(cfg, self.weights, self.workspace, self.stream)

    def close(self):
        if getattr(self, "handle", None):
            sdsat_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def cache_len(self) -> np.ndarray:
        """Current cache_len[max_batch] (synchronises the stream)."""
        self.stream.synchronize()
        out = np.zeros(self.cfg.max_batch, np.int32)
        _hip_memcpy_d2h(out, sdsat_cache_len_ptr(self.handle))
        return out


_hip = None


def _hip_memcpy_d2h(dst: np.ndarray, src_ptr: int) -> None:
    """Blocking device-to-host copy through the HIP runtime that torch already loaded."""
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        _hip.hipMemcpy.restype = ctypes.c_int
    rc = _hip.hipMemcpy(dst.ctypes.data, src_ptr, dst.nbytes, 2)   # hipMemcpyDeviceToHost
    if rc != 0:
        raise RuntimeError(f"hipMemcpy failed ({rc})")
