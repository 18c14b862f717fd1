"""ctypes binding of libdard.so (include/dard.h).

Every function here only marshals arguments: torch tensors become device
pointers, shapes become sizes, the current torch stream becomes the HIP
stream.  All computation happens in the HIP kernels of libdard.so; if the
library is missing, loading fails loudly -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdard.so")

DARD_OK = 0
STATE_M, STATE_C, STATE_U = 0, 1, 2
DTYPE_F32, DTYPE_BF16, DTYPE_BF16_KV_FP8 = 0, 1, 2
KV_DTYPE, KV_FP8 = 0, 1
F_XSELF_SHADOW, F_MKEYS_SHADOW, F_VERIFY_PCUR, F_PROGRESS = 1, 2, 4, 8
F_C_BIDIR, F_ORDER_L2R, F_ORDER_ENTROPY, F_ORDER_MARGIN, F_FIXED_W = 16, 32, 64, 128, 256
F_CHECK_STATES = 512
F_HIDDEN_MIX = 1024
BAD_STATE = -1
GEMM_STREAM, GEMM_PIPE, GEMM_BIG, GEMM_TILED, GEMM_F32 = range(5)
PHASE_VERIFY, PHASE_FINAL = 0, 1
(K_GEMM_QKV, K_GEMM_O, K_GEMM_GU, K_GEMM_DOWN, K_GEMM_HEAD, K_ATTENTION, K_CONFIDENCE,
 K_DECIDE, K_NORM, K_MASK, K_COUNT) = range(11)

EXPORTS = [
    "dard_last_error", "dard_version", "dard_check_states", "dard_build_state_mask", "dard_attention_workspace_bytes",
    "dard_masked_attention", "dard_confidence_workspace_bytes", "dard_confidence", "dard_confidence_noalloc",
    "dard_commit_remask", "dard_packed_weight_bytes", "dard_pack_weights", "dard_kv_bytes",
    "dard_workspace_bytes", "dard_prefill", "dard_prefill_extend", "dard_step", "dard_step_full", "dard_prefill_suffix",
    "dard_step_shared", "dard_pack_matrix", "dard_linear", "dard_gemm_plan",
    "dard_trace_enable",
    "dard_trace_read", "dard_trace_reset", "dard_trace_sample",
]


class DardError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"libdard status {status}: {msg}")
        self.status = status


class dard_params(ctypes.Structure):
    _fields_ = [("tau_c", ctypes.c_float), ("tau_u", ctypes.c_float), ("lambda_", ctypes.c_double),
                ("p0", ctypes.c_double), ("mask_id", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("w_fixed", ctypes.c_float)]


class dard_dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_layers", "d_model", "n_heads", "n_kv_heads", "head_dim",
                                              "ffn_dim", "vocab", "max_pos", "dtype")] + \
               [("norm_eps", ctypes.c_float), ("rope_theta", ctypes.c_float), ("kv_format", ctypes.c_int32)]


class dard_step_debug(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("logits", "w", "maxprob_s", "argmax_s", "pcur_s",
                                               "maxprob_mix", "argmax_mix", "entropy", "margin")]


_lib = None


def lib():
    """Load libdard.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, u32, sz, f32, i64 = (ctypes.c_void_p, ctypes.c_int, ctypes.c_uint32, ctypes.c_size_t,
                                      ctypes.c_float, ctypes.c_int64)
        sig = {
            "dard_last_error": (ctypes.c_char_p, []),
            "dard_version": (i32, []),
            "dard_check_states": (i32, [vp, i32, vp, vp]),
            "dard_build_state_mask": (i32, [vp, vp, i32, i32, u32, vp, vp]),
            "dard_attention_workspace_bytes": (sz, [i32, i32, i32, i32, i32, i32]),
            "dard_masked_attention": (i32, [i32, vp, vp, vp, i32, i32, vp, vp, i32, i32, i32, i32, i32, f32,
                                            u32, vp, vp, sz, vp]),
            "dard_confidence_workspace_bytes": (sz, [i32, i32]),
            "dard_confidence": (i32, [vp, vp, vp, vp, i32, i32, i64, vp, vp, vp, vp, vp, vp, sz, vp]),
            "dard_confidence_noalloc": (i32, [vp, vp, vp, vp, i32, i32, i64, vp, vp, vp, vp, vp, vp]),
            "dard_commit_remask": (i32, [i32, vp, i32, i32] + [vp] * 14),
            "dard_packed_weight_bytes": (sz, [vp]),
            "dard_pack_weights": (i32, [vp, vp, i32, vp, sz, vp]),
            "dard_kv_bytes": (sz, [vp, i32, i32]),
            "dard_workspace_bytes": (sz, [vp, i32, i32, i32]),
            "dard_prefill": (i32, [vp, vp, vp, i32, i32, i32, vp, vp, vp, sz, vp]),
            "dard_step": (i32, [vp, vp, vp, i32, i32, vp, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
            "dard_step_full": (i32, [vp, vp, vp, i32, i32, i32, vp, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                     vp]),
            "dard_prefill_suffix": (i32, [vp, vp, vp, i32, vp, i32, i32, i32, i32, vp, vp, sz, vp]),
            "dard_prefill_extend": (i32, [vp, vp, vp, i32, i32, i32, i32, vp, vp, sz, vp]),
            "dard_step_shared": (i32, [vp, vp, vp, i32, vp, i32, i32, i32, vp, i32, i32, vp, vp, vp, vp, vp, vp, vp,
                                       vp, vp, sz, vp]),
            "dard_pack_matrix": (i32, [i32, vp, i32, i32, vp, vp]),
            "dard_linear": (i32, [i32, vp, i32, i32, vp, i32, vp, vp]),
            "dard_gemm_plan": (i32, [i32, i32, i32, i32, i32, i32, ctypes.POINTER(ctypes.c_int32)]),
            "dard_trace_enable": (i32, [u32]),
            "dard_trace_read": (i32, [i32, ctypes.POINTER(i64), ctypes.POINTER(ctypes.c_double)]),
            "dard_trace_reset": (i32, []),
            "dard_trace_sample": (i32, [i32]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(status):
    if status != DARD_OK:
        raise DardError(status, lib().dard_last_error().decode())
    return status


def _p(t):
    """Device pointer of a tensor (None -> NULL)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        return t
    if not t.is_cuda:
        raise ValueError("libdard takes device tensors")
    if not t.is_contiguous():
        raise ValueError("libdard takes contiguous tensors")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def _dt(t):
    return DTYPE_BF16 if t.dtype == torch.bfloat16 else DTYPE_F32


def _ref(x):
    return ctypes.byref(x) if x is not None else None


def make_params(tau_c=0.4, tau_u=0.9, lam=0.5 ** (1 / 8), p0=0.1, mask_id=0, flags=0, w_fixed=0.0):
    return dard_params(tau_c, tau_u, lam, p0, mask_id, flags, w_fixed)


def make_dims(d):
    """From a synth.Dims (or anything with the same attributes)."""
    kv = getattr(d, "kv_dtype", "")
    if kv not in ("", "fp8", d.dtype):
        raise ValueError(f"unknown kv_dtype {kv!r}")
    return dard_dims(d.n_layers, d.d_model, d.n_heads, d.n_kv_heads, d.head_dim, d.ffn_dim, d.vocab, d.max_pos,
                     DTYPE_BF16 if d.dtype == "bf16" else DTYPE_F32, d.norm_eps, d.rope_theta,
                     KV_FP8 if kv == "fp8" else KV_DTYPE)


# ------------------------------------------------------------------ entry points
def dard_version():
    return lib().dard_version()


def dard_check_states(state, status, stream=None):
    """status (int32 [2] on the device) = (codes outside {0,1,2}, first index or -1)."""
    _check(lib().dard_check_states(_p(state), state.numel(), _p(status), _stream(stream)))


def dard_gemm_plan(M, N, K, partial=False, frag_x=True, dtype=DTYPE_BF16):
    """(kernel, tile rows / 32, tile columns / 32, K split) the library runs for
    a projection of these sizes."""
    plan = (ctypes.c_int32 * 4)()
    _check(lib().dard_gemm_plan(dtype, M, N, K, int(partial), int(frag_x), plan))
    return tuple(plan)


def dard_build_state_mask(state, conf, flags, sel, stream=None):
    b, B = state.shape
    _check(lib().dard_build_state_mask(_p(state), _p(conf), b, B, flags, _p(sel), _stream(stream)))


def dard_attention_workspace_bytes(dtype, b, B, Hq, dh, P):
    return lib().dard_attention_workspace_bytes(dtype, b, B, Hq, dh, P)


def dard_masked_attention(q, k, v, P, state, conf, scale, flags, out, ws=None, stream=None):
    """q [b][2B][Hq][dh], k [b][Hkv][cap][dh], v [b][Hkv][dh][cap] (dims-major);
    uint8 k / v hold OCP FP8 E4M3 codes (bf16 q / out)."""
    b, R, Hq, dh = q.shape
    _, Hkv, cap, _ = k.shape
    if tuple(v.shape) != (b, Hkv, dh, cap):
        raise ValueError(f"v must be [b][Hkv][dh][cap] = {(b, Hkv, dh, cap)}, got {tuple(v.shape)}")
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    dt = DTYPE_BF16_KV_FP8 if k.dtype == torch.uint8 else _dt(q)
    _check(lib().dard_masked_attention(dt, _p(q), _p(k), _p(v), P, cap, _p(state), _p(conf), b, R // 2, Hq,
                                       Hkv, dh, scale, flags, _p(out), _p(ws), nbytes, _stream(stream)))


def dard_confidence_workspace_bytes(rows, V):
    return lib().dard_confidence_workspace_bytes(rows, V)


def dard_confidence(logits_s, argmax, maxprob, logits_x=None, w=None, cur_tok=None, pcur=None, ws=None,
                    stream=None, entropy=None, margin=None):
    rows, V = logits_s.shape
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check(lib().dard_confidence(_p(logits_s), _p(logits_x), _p(w), _p(cur_tok), rows, V, logits_s.stride(0),
                                 _p(argmax), _p(maxprob), _p(pcur), _p(entropy), _p(margin), _p(ws), nbytes,
                                 _stream(stream)))


def dard_confidence_noalloc(logits_s, argmax, maxprob, logits_x=None, w=None, cur_tok=None, pcur=None,
                            stream=None, entropy=None, margin=None):
    """dard_confidence with the library's preallocated scratch (no workspace)."""
    rows, V = logits_s.shape
    _check(lib().dard_confidence_noalloc(_p(logits_s), _p(logits_x), _p(w), _p(cur_tok), rows, V,
                                         logits_s.stride(0), _p(argmax), _p(maxprob), _p(pcur), _p(entropy),
                                         _p(margin), _stream(stream)))


def dard_commit_remask(phase, params, state_in, maxprob_s=None, pcur_s=None, argmax_s=None, maxprob_mix=None,
                       argmax_mix=None, w_out=None, state_out=None, tok_out=None, conf_out=None,
                       block_done=None, stream=None, key_s=None, key_mix=None):
    b, B = state_in.shape
    _check(lib().dard_commit_remask(phase, ctypes.byref(params), b, B, _p(state_in), _p(maxprob_s), _p(pcur_s),
                                    _p(argmax_s), _p(maxprob_mix), _p(argmax_mix), _p(key_s), _p(key_mix),
                                    _p(w_out), _p(state_out), _p(tok_out), _p(conf_out), _p(block_done),
                                    _stream(stream)))


def dard_pack_matrix(W, Wp, stream=None):
    N, K = W.shape
    _check(lib().dard_pack_matrix(_dt(W), _p(W), N, K, _p(Wp), _stream(stream)))


def dard_linear(X, Wp, N, Y, stream=None):
    """Y = X W^T with W packed by dard_pack_matrix (Wp has N*K elements)."""
    M, K = X.shape
    _check(lib().dard_linear(_dt(X), _p(X), M, K, _p(Wp), N, _p(Y), _stream(stream)))


def dard_trace_enable(mask):
    _check(lib().dard_trace_enable(mask))


def dard_trace_read(cls):
    n = ctypes.c_int64(0)
    ms = ctypes.c_double(0.0)
    _check(lib().dard_trace_read(cls, ctypes.byref(n), ctypes.byref(ms)))
    return n.value, ms.value


def dard_trace_reset():
    _check(lib().dard_trace_reset())


def dard_trace_sample(period):
    _check(lib().dard_trace_sample(period))


def _debug(debug):
    if debug is None:
        return None
    return dard_step_debug(*[_p(debug.get(k)) for k in ("logits", "w", "maxprob_s", "argmax_s", "pcur_s",
                                                        "maxprob_mix", "argmax_mix", "entropy", "margin")])


class Engine:
    """Device state of one decoding job: packed weights, KV cache and
    workspace (torch allocations), plus calls of dard_prefill / dard_step."""

    def __init__(self, dims, weights, b, B, cap, stream=None, device="cuda", packed=None):
        """weights: name -> tensor (packed here), or None with `packed` = the
        packed image of another Engine of the same dims (shared, not copied)."""
        self.dims = dims
        self.cdims = make_dims(dims)
        self.b, self.B, self.cap = b, B, cap
        L = lib()
        nbytes = L.dard_packed_weight_bytes(ctypes.byref(self.cdims))
        if nbytes == 0:
            raise DardError(-2, L.dard_last_error().decode())
        if packed is not None:
            if packed.numel() < nbytes:
                raise ValueError("packed image too small for these dims")
            self.packed = packed
        else:
            self.packed = torch.empty(nbytes, dtype=torch.uint8, device=device)
            names = [n for n in weights]
            srcs = (ctypes.c_void_p * len(names))(*[_p(weights[n].contiguous()) for n in names])
            _check(L.dard_pack_weights(ctypes.byref(self.cdims), srcs, len(names), _p(self.packed), nbytes,
                                       _stream(stream)))
        kvb = L.dard_kv_bytes(ctypes.byref(self.cdims), b, cap)
        self.kv = torch.zeros(max(kvb, 16), dtype=torch.uint8, device=device)
        wsb = L.dard_workspace_bytes(ctypes.byref(self.cdims), b, B, cap)
        if wsb == 0:
            raise DardError(-2, L.dard_last_error().decode())
        self.ws = torch.zeros(wsb, dtype=torch.uint8, device=device)

    def kv_view(self, dtype):
        """KV cache as (K, V) tensors [layers][b][Hkv][cap][dh] (V read out of
        its dims-major storage [layers][b][Hkv][dh][cap] as a transposed view);
        dtype torch.uint8 for an FP8 cache (E4M3 codes)."""
        d = self.dims
        n = d.n_layers * 2 * self.b * d.n_kv_heads * self.cap * d.head_dim
        kv = self.kv.view(dtype)[:n].view(d.n_layers, 2, self.b, d.n_kv_heads, self.cap * d.head_dim)
        k = kv[:, 0].view(d.n_layers, self.b, d.n_kv_heads, self.cap, d.head_dim)
        v = kv[:, 1].view(d.n_layers, self.b, d.n_kv_heads, d.head_dim, self.cap).transpose(-1, -2)
        return k, v

    def dard_prefill(self, ids, embeds=None, stream=None):
        b, P = ids.shape
        _check(lib().dard_prefill(ctypes.byref(self.cdims), _p(self.packed), _p(self.kv), self.cap, b, P, _p(ids),
                                  _p(embeds), _p(self.ws), self.ws.numel(), _stream(stream)))

    def dard_step(self, P, params, tok_in, state_in, conf_in, tok_out, state_out, conf_out, block_done=None,
                  debug=None, stream=None):
        b, B = tok_in.shape
        dbg = None
        dbg = _debug(debug)
        _check(lib().dard_step(ctypes.byref(self.cdims), _p(self.packed), _p(self.kv), self.cap, P,
                               ctypes.byref(params), b, B, _p(tok_in), _p(state_in), _p(conf_in), _p(tok_out),
                               _p(state_out), _p(conf_out), _p(block_done), _ref(dbg), _p(self.ws),
                               self.ws.numel(), _stream(stream)))

    def dard_prefill_extend(self, P, ids, stream=None):
        """Extend-only refresh: positions P..P+Pn-1 of each sequence (ids
        [b][Pn]) see the cached keys 0..P-1 and each other."""
        b, Pn = ids.shape
        _check(lib().dard_prefill_extend(ctypes.byref(self.cdims), _p(self.packed), _p(self.kv), self.cap, P, b, Pn,
                                         _p(ids), _p(self.ws), self.ws.numel(), _stream(stream)))

    def dard_prefill_suffix(self, shared, Ps, ids, stream=None):
        """Positions Ps.. of each sequence after the prompt cached in `shared`
        (an Engine of the same dims with b = 1 whose dard_prefill ran over Ps
        prompt positions); ids [b][Pc]."""
        b, Pc = ids.shape
        _check(lib().dard_prefill_suffix(ctypes.byref(self.cdims), _p(self.packed), _p(self.kv), self.cap,
                                         _p(shared.kv), shared.cap, Ps, b, Pc, _p(ids), _p(self.ws), self.ws.numel(),
                                         _stream(stream)))

    def dard_step_shared(self, shared, Ps, P, params, tok_in, state_in, conf_in, tok_out, state_out, conf_out,
                         block_done=None, debug=None, stream=None):
        b, B = tok_in.shape
        dbg = _debug(debug)
        _check(lib().dard_step_shared(ctypes.byref(self.cdims), _p(self.packed), _p(self.kv), self.cap,
                                      _p(shared.kv), shared.cap, Ps, P, ctypes.byref(params), b, B, _p(tok_in),
                                      _p(state_in), _p(conf_in), _p(tok_out), _p(state_out), _p(conf_out),
                                      _p(block_done), _ref(dbg), _p(self.ws), self.ws.numel(), _stream(stream)))

    def dard_step_full(self, blk, params, seq, state_in, conf_in, tok_out, state_out, conf_out, block_done=None,
                       debug=None, stream=None):
        """Full-sequence step: seq [b][N] (current block at blk..blk+B-1)."""
        b, N = seq.shape
        B = state_in.shape[1]
        dbg = _debug(debug)
        _check(lib().dard_step_full(ctypes.byref(self.cdims), _p(self.packed), _p(self.kv), self.cap, N, blk,
                                    ctypes.byref(params), b, B, _p(seq), _p(state_in), _p(conf_in), _p(tok_out),
                                    _p(state_out), _p(conf_out), _p(block_done), _ref(dbg), _p(self.ws),
                                    self.ws.numel(), _stream(stream)))
