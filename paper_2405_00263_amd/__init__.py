"""Python binding of libclover.so (MI355X / gfx950 Clover speculate-and-verify step).

Argument marshalling only: every step of the decoding path runs in the HIP
library.  PyTorch provides device memory and the stream.  Importing this module
loads the in-tree ``libclover.so``; it raises if the library has not been built.
"""
import ctypes
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libclover.so")

MAX_HEADS = 8
STATUS = {0: "OK", 1: "INVALID_ARG", 2: "CAPACITY", 3: "STATE", 4: "BAD_TREE", 5: "DEVICE"}
FLAG_KEEP_LOGITS = 1
FLAG_PROFILE = 2
FLAG_EAGER = 4
FLAG_AB_COMMIT = 8
KSTAT = {"gemm_verify": 0, "gemm_draft": 1, "attention": 2, "other": 3}
DRAFT_MODES = {"clover": 0, "medusa": 1}
AB_MODES = {"default": 0, "full": 1, "attn": 2, "mlp": 3, "none": 4}
AD_KEYS = {"single": 0, "two": 1, "path": 2}
REGRESSIVE = {"attention": 0, "mlp": 1}
MEDUSA_LM = {"shared": 0, "per_head": 1}


class CloverError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"clover {STATUS.get(status, status)}: {msg}")
        self.status = status


class ConfigC(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_theta", ctypes.c_float), ("dtype", ctypes.c_int32),
                ("n_spec_heads", ctypes.c_int32), ("topk", ctypes.c_int32 * MAX_HEADS),
                ("tree_tokens", ctypes.c_int32), ("max_batch", ctypes.c_int32),
                ("max_context", ctypes.c_int32), ("kv_block", ctypes.c_int32),
                ("prefill_chunk", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("draft_mode", ctypes.c_int32), ("ab_mode", ctypes.c_int32),
                ("ad_keys", ctypes.c_int32), ("ad_per_head", ctypes.c_int32),
                ("temperature", ctypes.c_float), ("sample_seed", ctypes.c_uint32),
                ("regressive", ctypes.c_int32), ("medusa_lm_heads", ctypes.c_int32)]


class TimingsC(ctypes.Structure):
    _fields_ = [("draft_ms", ctypes.c_float), ("verify_ms", ctypes.c_float),
                ("accept_ms", ctypes.c_float), ("total_ms", ctypes.c_float),
                ("steps", ctypes.c_int32)]


class KernelStatsC(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int64), ("total_ms", ctypes.c_double),
                ("bytes", ctypes.c_double), ("flops", ctypes.c_double)]


_lib = None

EXPORTS = {
    # name: (restype, argtypes)
    "clover_check_config": (ctypes.c_int, [ctypes.c_void_p]),
    "clover_weight_count": (ctypes.c_size_t, [ctypes.c_void_p]),
    "clover_weight_name": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_char_p, ctypes.c_size_t]),
    "clover_weight_shape": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "clover_packed_bytes": (ctypes.c_size_t, [ctypes.c_void_p, ctypes.c_size_t]),
    "clover_workspace_bytes": (ctypes.c_size_t, [ctypes.c_void_p]),
    "clover_pack_weight": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "clover_init": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p]),
    "clover_destroy": (None, [ctypes.c_void_p]),
    "clover_last_error": (ctypes.c_char_p, [ctypes.c_void_p]),
    "clover_prefill": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]),
    "clover_step": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]),
    "clover_verify_tree": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]),
    "clover_release": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32]),
    "clover_seq_len": (ctypes.c_int32, [ctypes.c_void_p, ctypes.c_int32]),
    "clover_debug_read": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_char_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "clover_debug_kv": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p]),
    "clover_get_timings": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p]),
    "clover_debug_trace": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t]),
    "clover_kernel_stats_get": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p]),
    "clover_kernel_stats_reset": (ctypes.c_int, [ctypes.c_void_p]),
    "clover_set_flags": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32]),
    "clover_op_scratch_bytes": (ctypes.c_size_t, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]),
    "clover_op_linear": (ctypes.c_int, [ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "clover_packed_matrix_bytes": (ctypes.c_size_t, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]),
    "clover_pack_matrix": (ctypes.c_int, [ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]),
    "clover_op_swiglu": (ctypes.c_int, [ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]),
    "clover_op_attention_scratch_bytes": (ctypes.c_size_t, [ctypes.c_int32] * 6),
    "clover_op_attention": (ctypes.c_int, [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "clover_op_argmax": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "clover_op_topk_scratch_bytes": (ctypes.c_size_t, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]),
    "clover_op_topk": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "clover_op_tree_build": (ctypes.c_int, [ctypes.c_void_p] * 4 + [ctypes.c_int32] * 3 + [ctypes.c_void_p] * 6),
    "clover_op_accept": (ctypes.c_int, [ctypes.c_void_p] * 3 + [ctypes.c_int32] * 2 + [ctypes.c_void_p] * 4),
    "clover_op_linear_noalloc_max_bytes": (ctypes.c_size_t, []),
    "clover_op_linear_noalloc": (ctypes.c_int, [ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                                ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]),
    "clover_op_compact": (ctypes.c_int, [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p] + [ctypes.c_int32] * 4
                          + [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32,
                             ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
}


def lib() -> ctypes.CDLL:
    """Load libclover.so once; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2405_00263_amd.build.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in EXPORTS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(status: int, ctx=None):
    if status != 0:
        msg = lib().clover_last_error(ctx)
        raise CloverError(status, msg.decode() if msg else "")


def make_config(cfg, max_batch: Optional[int] = None, max_context: Optional[int] = None,
                prefill_chunk: int = 0, flags: int = 0) -> ConfigC:
    """Build the C config from any object with the model/decoding attributes."""
    c = ConfigC()
    for f in ("n_layers", "d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim", "vocab"):
        setattr(c, f, int(getattr(cfg, f)))
    c.rms_eps = float(getattr(cfg, "rms_eps", 1e-6))
    c.rope_theta = float(getattr(cfg, "rope_theta", 10000.0))
    dt = getattr(cfg, "dtype")
    c.dtype = 1 if dt in ("bf16", 1) else 0
    topk = tuple(getattr(cfg, "topk"))
    c.n_spec_heads = len(topk)
    for i, k in enumerate(topk):
        c.topk[i] = int(k)
    c.tree_tokens = int(cfg.tree_tokens)
    c.max_batch = int(max_batch if max_batch is not None else getattr(cfg, "batch", 1))
    c.max_context = int(max_context if max_context is not None else cfg.max_context)
    c.kv_block = 16
    c.prefill_chunk = int(prefill_chunk)
    c.flags = int(flags)
    c.draft_mode = DRAFT_MODES[getattr(cfg, "draft", "clover")]
    c.ab_mode = AB_MODES[getattr(cfg, "ab", "default")]
    c.ad_keys = AD_KEYS[getattr(cfg, "ad_keys", "single")]
    c.ad_per_head = int(bool(getattr(cfg, "ad_per_head", False)))
    c.temperature = float(getattr(cfg, "temperature", 0.0))
    c.sample_seed = int(getattr(cfg, "sample_seed", 0)) & 0xFFFFFFFF
    c.regressive = REGRESSIVE[getattr(cfg, "regressive", "attention")]
    c.medusa_lm_heads = MEDUSA_LM[getattr(cfg, "medusa_lm", "shared")]
    return c


def weight_names(c: ConfigC) -> List[str]:
    L = lib()
    n = L.clover_weight_count(ctypes.byref(c))
    if n == 0:
        _check(1)
    out = []
    buf = ctypes.create_string_buffer(128)
    for i in range(n):
        L.clover_weight_name(ctypes.byref(c), i, buf, 128)
        out.append(buf.value.decode())
    return out


def weight_shapes(c: ConfigC) -> List[tuple]:
    L = lib()
    out = []
    arr = (ctypes.c_int64 * 2)()
    for i in range(L.clover_weight_count(ctypes.byref(c))):
        nd = L.clover_weight_shape(ctypes.byref(c), i, arr)
        out.append(tuple(arr[:nd]))
    return out


def workspace_bytes(c: ConfigC) -> int:
    n = lib().clover_workspace_bytes(ctypes.byref(c))
    if n == 0:
        _check(1)
    return n


def _stream_handle(stream=None) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


class CloverEngine:
    """One library context: packed weights, workspace, sequences."""

    def __init__(self, cfg, weights: Dict[str, "object"], max_batch: Optional[int] = None,
                 max_context: Optional[int] = None, prefill_chunk: int = 0, flags: int = 0,
                 stream=None, free_source: bool = False):
        import torch
        self.c = make_config(cfg, max_batch, max_context, prefill_chunk, flags)
        self.H = self.c.n_spec_heads
        self.T = self.c.tree_tokens
        L = lib()
        _check(L.clover_check_config(ctypes.byref(self.c)))
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        sh = self.stream.cuda_stream
        names = weight_names(self.c)
        shapes = weight_shapes(self.c)
        tdt = torch.bfloat16 if self.c.dtype == 1 else torch.float32
        self.packed = []
        for i, (n, shp) in enumerate(zip(names, shapes)):
            src = weights[n]
            if tuple(src.shape) != tuple(shp) or src.dtype != tdt or not src.is_cuda:
                raise ValueError(f"weight {n}: expected {shp} {tdt} on cuda, got "
                                 f"{tuple(src.shape)} {src.dtype} {src.device}")
            src = src.contiguous()
            dst = torch.empty(L.clover_packed_bytes(ctypes.byref(self.c), i), dtype=torch.uint8,
                              device=src.device)
            _check(L.clover_pack_weight(ctypes.byref(self.c), i, ctypes.c_void_p(src.data_ptr()),
                                        ctypes.c_void_p(dst.data_ptr()), ctypes.c_void_p(sh)))
            self.packed.append(dst)
            if free_source:
                self.stream.synchronize()
                weights[n] = None
                del src
        self.ws_bytes = workspace_bytes(self.c)
        self.ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device="cuda")
        ptrs = (ctypes.c_void_p * len(self.packed))(*[t.data_ptr() for t in self.packed])
        self.ctx = ctypes.c_void_p()
        _check(L.clover_init(ctypes.byref(self.c), ptrs, ctypes.c_void_p(self.ws.data_ptr()),
                             self.ws_bytes, ctypes.c_void_p(sh), ctypes.byref(self.ctx)))

    # -- decoding --------------------------------------------------------------------------
    def prefill(self, seq: int, tokens: Sequence[int]) -> int:
        arr = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))
        out = ctypes.c_int32()
        _check(lib().clover_prefill(self.ctx, seq, arr.ctypes.data_as(ctypes.c_void_p), len(arr),
                                    ctypes.byref(out)), self.ctx)
        return int(out.value)

    def step(self, seqs: Sequence[int]) -> List[List[int]]:
        ids = np.ascontiguousarray(np.asarray(seqs, dtype=np.int32))
        out = np.zeros((len(ids), self.H + 1), dtype=np.int32)
        cnt = np.zeros(len(ids), dtype=np.int32)
        _check(lib().clover_step(self.ctx, ids.ctypes.data_as(ctypes.c_void_p), len(ids),
                                 out.ctypes.data_as(ctypes.c_void_p),
                                 cnt.ctypes.data_as(ctypes.c_void_p)), self.ctx)
        return [list(map(int, out[i, :cnt[i]])) for i in range(len(ids))]

    def verify_tree(self, seq: int, tokens: Sequence[int], parents: Sequence[int]) -> List[int]:
        t = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))
        p = np.ascontiguousarray(np.asarray(parents, dtype=np.int32))
        out = np.zeros(self.H + 1, dtype=np.int32)
        cnt = np.zeros(1, dtype=np.int32)
        _check(lib().clover_verify_tree(self.ctx, seq, t.ctypes.data_as(ctypes.c_void_p),
                                        p.ctypes.data_as(ctypes.c_void_p), len(t),
                                        out.ctypes.data_as(ctypes.c_void_p),
                                        cnt.ctypes.data_as(ctypes.c_void_p)), self.ctx)
        return list(map(int, out[:cnt[0]]))

    def release(self, seq: int):
        _check(lib().clover_release(self.ctx, seq), self.ctx)

    def seq_len(self, seq: int) -> int:
        return int(lib().clover_seq_len(self.ctx, seq))

    # -- inspection ------------------------------------------------------------------------
    def debug(self, name: str, dtype, shape) -> np.ndarray:
        out = np.zeros(shape, dtype=dtype)
        written = ctypes.c_size_t()
        _check(lib().clover_debug_read(self.ctx, name.encode(), out.ctypes.data_as(ctypes.c_void_p),
                                       out.nbytes, ctypes.byref(written)), self.ctx)
        return out

    def debug_kv(self, seq: int, layer: int, pos: int, which_v: bool) -> np.ndarray:
        out = np.zeros(self.c.n_kv_heads * self.c.head_dim, dtype=np.float32)
        _check(lib().clover_debug_kv(self.ctx, seq, layer, pos, int(which_v),
                                     out.ctypes.data_as(ctypes.c_void_p)), self.ctx)
        return out

    def set_trace(self, buf):
        """Residual-stream trace into a cuda float32 tensor [n_layers + 2][rows][d_model]
        (None switches it off)."""
        if buf is None:
            _check(lib().clover_debug_trace(self.ctx, None, 0), self.ctx)
        else:
            _check(lib().clover_debug_trace(self.ctx, ctypes.c_void_p(buf.data_ptr()), buf.numel() * 4), self.ctx)
        self._trace = buf

    def timings(self) -> dict:
        t = TimingsC()
        _check(lib().clover_get_timings(self.ctx, ctypes.byref(t)), self.ctx)
        return dict(draft_ms=t.draft_ms, verify_ms=t.verify_ms, accept_ms=t.accept_ms,
                    total_ms=t.total_ms, steps=t.steps)

    def kernel_stats(self) -> dict:
        out = {}
        for name, k in KSTAT.items():
            st = KernelStatsC()
            _check(lib().clover_kernel_stats_get(self.ctx, k, ctypes.byref(st)), self.ctx)
            out[name] = dict(launches=st.launches, total_ms=st.total_ms, bytes=st.bytes, flops=st.flops)
        return out

    def set_flags(self, flags: int):
        _check(lib().clover_set_flags(self.ctx, int(flags)), self.ctx)

    def reset_kernel_stats(self):
        _check(lib().clover_kernel_stats_reset(self.ctx), self.ctx)

    def close(self):
        if getattr(self, "ctx", None) and self.ctx.value:
            lib().clover_destroy(self.ctx)
            self.ctx = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---- single-kernel entry points (tests at full size) ----------------------------------------

def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def pack_matrix(W):
    """Pack a row-major [N][K] cuda matrix (fp32 or bf16) into the tiled layout."""
    import torch
    dt = 1 if W.dtype == torch.bfloat16 else 0
    n = lib().clover_packed_matrix_bytes(dt, W.shape[0], W.shape[1])
    if n == 0:
        _check(1)
    out = torch.empty(n, dtype=torch.uint8, device=W.device)
    _check(lib().clover_pack_matrix(dt, _ptr(W.contiguous()), W.shape[0], W.shape[1], _ptr(out),
                                    ctypes.c_void_p(_stream_handle())))
    return out


def op_linear(X, Wp, N: int):
    import torch
    dt = 1 if X.dtype == torch.bfloat16 else 0
    M, K = X.shape
    Y = torch.empty(M, N, dtype=torch.float32, device=X.device)
    need = lib().clover_op_scratch_bytes(dt, M, N, K)
    if need == 0:
        _check(1)
    scratch = torch.empty(need, dtype=torch.uint8, device=X.device)
    _check(lib().clover_op_linear(dt, _ptr(X.contiguous()), M, K, _ptr(Wp), N, _ptr(Y), _ptr(scratch),
                                  need, ctypes.c_void_p(_stream_handle())))
    return Y


def op_linear_noalloc(X, Wp, N: int):
    """op_linear through the allocation-free entry point (split-K partials in the library's
    own device array); the output tensor is the caller's."""
    import torch
    dt = 1 if X.dtype == torch.bfloat16 else 0
    M, K = X.shape
    Y = torch.empty(M, N, dtype=torch.float32, device=X.device)
    _check(lib().clover_op_linear_noalloc(dt, _ptr(X.contiguous()), M, K, _ptr(Wp), N, _ptr(Y),
                                          ctypes.c_void_p(_stream_handle())))
    return Y


def op_swiglu(X, Wg_p, Wu_p, F: int):
    """silu(X W_gate^T) * (X W_up^T) in the storage type of X, from packed gate and up matrices."""
    import torch
    dt = 1 if X.dtype == torch.bfloat16 else 0
    M, K = X.shape
    act = torch.empty(M, F, dtype=X.dtype, device=X.device)
    _check(lib().clover_op_swiglu(dt, _ptr(X.contiguous()), M, K, _ptr(Wg_p), _ptr(Wu_p), F, _ptr(act),
                                  ctypes.c_void_p(_stream_handle())))
    return act


def op_attention(Q, Kpre, Vpre, Ktree, Vtree, parents=None, causal=False):
    """Q [T][Hq][hd]; Kpre/Vpre [L][Hkv][hd]; Ktree/Vtree [T][Hkv][hd] (cuda, storage dtype)."""
    import torch
    dt = 1 if Q.dtype == torch.bfloat16 else 0
    T, Hq, hd = Q.shape
    L, Hkv = Kpre.shape[0], Ktree.shape[1]
    O = torch.empty_like(Q)
    need = lib().clover_op_attention_scratch_bytes(dt, L, T, Hq, Hkv, hd)
    if need == 0:
        _check(1)
    scratch = torch.empty(need, dtype=torch.uint8, device=Q.device)
    par = np.ascontiguousarray(np.asarray(parents if parents is not None else [-1] * T, dtype=np.int32))
    kp = _ptr(Kpre.contiguous()) if L > 0 else ctypes.c_void_p(0)
    vp = _ptr(Vpre.contiguous()) if L > 0 else ctypes.c_void_p(0)
    _check(lib().clover_op_attention(dt, _ptr(Q.contiguous()), kp, vp, _ptr(Ktree.contiguous()),
                                     _ptr(Vtree.contiguous()), L, T, par.ctypes.data_as(ctypes.c_void_p),
                                     int(causal), Hq, Hkv, hd, _ptr(O), _ptr(scratch), need,
                                     ctypes.c_void_p(_stream_handle())))
    return O


def op_argmax(logits):
    import torch
    M, V = logits.shape
    out = torch.empty(M, dtype=torch.int32, device=logits.device)
    keys = torch.empty(M, dtype=torch.int64, device=logits.device)
    _check(lib().clover_op_argmax(_ptr(logits.contiguous()), M, V, _ptr(out), _ptr(keys),
                                  ctypes.c_void_p(_stream_handle())))
    return out


def op_topk(logits, k: int):
    import torch
    M, V = logits.shape
    tok = torch.empty(M, k, dtype=torch.int32, device=logits.device)
    logp = torch.empty(M, k, dtype=torch.float32, device=logits.device)
    need = lib().clover_op_topk_scratch_bytes(M, V, k)
    if need == 0:
        _check(1)
    scratch = torch.empty(need, dtype=torch.uint8, device=logits.device)
    _check(lib().clover_op_topk(_ptr(logits.contiguous()), M, V, k, _ptr(tok), _ptr(logp), _ptr(scratch),
                                ctypes.c_void_p(_stream_handle())))
    return tok, logp


def op_tree_build(token, parent, depth, lp, T: int, L: int):
    """Candidate arrays (cuda int32/float32, root first) -> tree arrays and mask."""
    import torch
    n = token.shape[0]
    dev = token.device
    out = {k: torch.empty(T, dtype=torch.int32, device=dev) for k in ("tokens", "parent", "depth", "pos")}
    mask = torch.empty(T * ((T + 63) // 64), dtype=torch.int64, device=dev)
    _check(lib().clover_op_tree_build(_ptr(token), _ptr(parent), _ptr(depth), _ptr(lp), n, T, L,
                                      _ptr(out["tokens"]), _ptr(out["parent"]), _ptr(out["depth"]),
                                      _ptr(out["pos"]), _ptr(mask), ctypes.c_void_p(_stream_handle())))
    out["mask"] = mask
    return out


def op_accept(tokens, parent, target, max_depth: int):
    import torch
    dev = tokens.device
    acc = torch.empty(max_depth + 1, dtype=torch.int32, device=dev)
    acc_len = torch.empty(1, dtype=torch.int32, device=dev)
    bonus = torch.empty(1, dtype=torch.int32, device=dev)
    _check(lib().clover_op_accept(_ptr(tokens), _ptr(parent), _ptr(target), tokens.shape[0], max_depth,
                                  _ptr(acc), _ptr(acc_len), _ptr(bonus), ctypes.c_void_p(_stream_handle())))
    return acc, acc_len, bonus


def op_compact(kcache, vcache, block_table, L: int, acc):
    """In-place KV compaction of one sequence: kcache/vcache cuda [layers][blocks][n_kv][16*hd]
    (storage dtype, the library's paged layout); block_table and acc host int sequences."""
    import torch
    dt = 1 if kcache.dtype == torch.bfloat16 else 0
    nl, nb, nkv, per = kcache.shape
    bt = np.ascontiguousarray(np.asarray(block_table, dtype=np.int32))
    ac = np.ascontiguousarray(np.asarray(acc, dtype=np.int32))
    scratch = torch.empty(4 * (len(bt) + len(ac)), dtype=torch.uint8, device=kcache.device)
    _check(lib().clover_op_compact(dt, _ptr(kcache), _ptr(vcache), nl, nb, nkv, per // 16,
                                   bt.ctypes.data_as(ctypes.c_void_p), len(bt), L,
                                   ac.ctypes.data_as(ctypes.c_void_p), len(ac), _ptr(scratch),
                                   scratch.numel(), ctypes.c_void_p(_stream_handle())))
