"""Thin Python binding of libbacon.so (include/bacon.h).

Argument marshalling only: every step of the pass runs in the HIP kernels of
the library.  torch tensors provide device memory and the current HIP stream.
Loading fails loudly when the library is missing; there is no other path.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbacon.so")

OK, ERR_INVALID, ERR_UNSUPPORTED, ERR_ORDER, ERR_WORKSPACE, ERR_HIP = range(6)
FP32, BF16 = 0, 1
TERM_E, TERM_L, TERM_T = 1, 2, 4

ENTRY_POINTS = [
    "bacon_default_params", "bacon_workspace_bytes", "bacon_init", "bacon_free",
    "bacon_begin_prompt", "bacon_score", "bacon_calibrate", "bacon_select_topk",
    "bacon_compact", "bacon_compress_layer", "bacon_compress_layer_lse", "bacon_compress_prompt",
    "bacon_window_lse", "bacon_window_lse_static", "bacon_debug_capture", "bacon_debug_device_errors",
    "bacon_allocate_heads", "bacon_alloc_output",
    "bacon_idx_count",
    "bacon_kept_rows",
    "bacon_profile_enable", "bacon_profile_read", "bacon_status_string", "bacon_last_error",
]


class Params(C.Structure):
    _fields_ = [("radius", C.c_int32), ("persist_m", C.c_int32), ("rho", C.c_double),
                ("gamma", C.c_float), ("eps", C.c_float), ("pool_kernel", C.c_int32),
                ("use_last_query", C.c_int32), ("terms", C.c_uint32), ("pool_mode", C.c_int32),
                ("head_alloc", C.c_int32), ("alloc_floor", C.c_float)]


# pooling of the score before the top-K (bacon_pool_mode)
POOL_MEAN_S, POOL_MAX_S, POOL_MEAN_B = 0, 1, 2
# head-wise budgets of the fused calls (bacon_head_alloc)
ALLOC_GIVEN, ALLOC_ADAPTIVE = 0, 1


class Shape(C.Structure):
    _fields_ = [("num_layers", C.c_int32), ("num_q_heads", C.c_int32),
                ("num_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("window", C.c_int32),
                ("max_batch", C.c_int32), ("max_total_tokens", C.c_int64), ("dtype", C.c_int)]


class Batch(C.Structure):
    _fields_ = [("batch", C.c_int32), ("cu_seqlens", C.POINTER(C.c_int32)),
                ("budgets", C.POINTER(C.c_int32)), ("head_budgets", C.POINTER(C.c_int32))]


class KernelTime(C.Structure):
    _fields_ = [("name", C.c_char * 32), ("launches", C.c_int64), ("total_ms", C.c_double)]


class BaconError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"status {status}: {msg}")
        self.status = status


_lib = None


def lib() -> C.CDLL:
    """Load libbacon.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2606_14782_amd.build")
        L = C.CDLL(LIB_PATH)
        vp, sz = C.c_void_p, C.c_size_t
        ctxp = C.POINTER(C.c_void_p)
        L.bacon_default_params.argtypes = [C.POINTER(Params)]
        L.bacon_workspace_bytes.argtypes = [C.POINTER(Shape), C.POINTER(Params)]
        L.bacon_workspace_bytes.restype = sz
        L.bacon_init.argtypes = [ctxp, C.POINTER(Shape), C.POINTER(Params), vp, sz]
        L.bacon_free.argtypes = [vp]
        L.bacon_begin_prompt.argtypes = [vp, C.POINTER(Batch), vp]
        L.bacon_score.argtypes = [vp, C.c_int32, C.POINTER(Batch), vp, vp, vp, vp, vp, vp]
        L.bacon_calibrate.argtypes = [vp, C.c_int32, C.POINTER(Batch), vp, vp, vp, vp, vp, vp, vp]
        L.bacon_select_topk.argtypes = [vp, C.POINTER(Batch), vp, vp, vp]
        L.bacon_compact.argtypes = [vp, C.POINTER(Batch), vp, vp, vp, vp, vp, vp]
        L.bacon_compress_layer.argtypes = [vp, C.c_int32, C.POINTER(Batch), vp, vp, vp, vp, vp,
                                           vp, vp]
        L.bacon_compress_layer_lse.argtypes = [vp, C.c_int32, C.POINTER(Batch), vp, vp, vp, vp,
                                               vp, vp, vp, vp]
        L.bacon_window_lse.argtypes = [vp, C.POINTER(Batch), vp, vp, vp, vp]
        L.bacon_compress_prompt.argtypes = [vp, C.POINTER(Batch), C.c_int32, C.c_int32, vp, vp, vp,
                                            vp, vp, vp, vp, vp, vp]
        L.bacon_debug_capture.argtypes = [vp, vp, vp, vp]
        L.bacon_allocate_heads.argtypes = [vp, C.POINTER(Batch), vp, vp, vp]
        L.bacon_alloc_output.argtypes = [vp, vp]
        L.bacon_debug_device_errors.argtypes = [vp]
        L.bacon_debug_device_errors.restype = C.c_int32
        L.bacon_window_lse_static.argtypes = [C.POINTER(Shape), C.POINTER(Batch), vp, vp, vp, vp]
        L.bacon_idx_count.argtypes = [C.POINTER(Batch), C.c_int32]
        L.bacon_idx_count.restype = C.c_int64
        L.bacon_kept_rows.argtypes = [C.POINTER(Batch), C.c_int32, C.c_int32]
        L.bacon_kept_rows.restype = C.c_int64
        L.bacon_profile_enable.argtypes = [vp, C.c_int32]
        L.bacon_profile_read.argtypes = [vp, C.POINTER(KernelTime), C.c_int32]
        L.bacon_profile_read.restype = C.c_int32
        L.bacon_status_string.argtypes = [C.c_int]
        L.bacon_status_string.restype = C.c_char_p
        L.bacon_last_error.restype = C.c_char_p
        for name in ("bacon_init", "bacon_free", "bacon_begin_prompt", "bacon_score",
                     "bacon_calibrate", "bacon_select_topk", "bacon_compact",
                     "bacon_compress_layer", "bacon_compress_layer_lse", "bacon_window_lse",
                     "bacon_compress_prompt", "bacon_debug_capture", "bacon_window_lse_static",
                     "bacon_allocate_heads", "bacon_alloc_output", "bacon_profile_enable"):
            getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != OK:
        raise BaconError(status, lib().bacon_last_error().decode())


def default_params(**overrides) -> Params:
    p = Params()
    lib().bacon_default_params(C.byref(p))
    for k, v in overrides.items():
        setattr(p, k, v)
    return p


class BatchLayout:
    """Host copy of a packed batch: cu_seqlens, per-sequence budgets, and
    optionally a budget per (sequence, KV head) [batch, Hkv]."""

    def __init__(self, cu_seqlens, budgets, head_budgets=None):
        self.cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
        self.budgets = np.ascontiguousarray(budgets, dtype=np.int32)
        self.head_budgets = (None if head_budgets is None else
                             np.ascontiguousarray(head_budgets, dtype=np.int32).reshape(len(self.budgets), -1))
        hb = (None if self.head_budgets is None else
              self.head_budgets.ctypes.data_as(C.POINTER(C.c_int32)))
        self.c = Batch(len(self.budgets), self.cu.ctypes.data_as(C.POINTER(C.c_int32)),
                       self.budgets.ctypes.data_as(C.POINTER(C.c_int32)), hb)

    @property
    def total(self) -> int:
        return int(self.cu[-1])

    def idx_count(self, num_kv_heads: int) -> int:
        return int(lib().bacon_idx_count(C.byref(self.c), num_kv_heads))

    def kept_rows(self, window: int, num_kv_heads: int = 1) -> int:
        return int(lib().bacon_kept_rows(C.byref(self.c), num_kv_heads, window))


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream():
    import torch
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


class Context:
    """A bacon_ctx with its workspace tensor on the current device."""

    def __init__(self, num_layers, num_q_heads, num_kv_heads, head_dim, window, max_batch,
                 max_total_tokens, dtype, params: Params | None = None, device="cuda"):
        import torch
        self.shape = Shape(num_layers, num_q_heads, num_kv_heads, head_dim, window, max_batch,
                           max_total_tokens, BF16 if dtype in ("bf16", BF16) else FP32)
        self.params = params or default_params()
        nbytes = lib().bacon_workspace_bytes(C.byref(self.shape), C.byref(self.params))
        if nbytes == 0:
            raise BaconError(ERR_INVALID, lib().bacon_last_error().decode())
        self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        base = self.workspace.data_ptr()
        aligned = (base + 255) & ~255
        self._h = C.c_void_p()
        _check(lib().bacon_init(C.byref(self._h), C.byref(self.shape), C.byref(self.params),
                                C.c_void_p(aligned), nbytes))
        self.device = device
        self.torch_dtype = torch.bfloat16 if self.shape.dtype == BF16 else torch.float32

    def __del__(self):
        h = getattr(self, "_h", None)
        if h and h.value and _lib is not None:
            _lib.bacon_free(h)
            self._h = C.c_void_p()

    # ---- entry points (same names as the C ABI)
    def bacon_begin_prompt(self, batch: BatchLayout):
        _check(lib().bacon_begin_prompt(self._h, C.byref(batch.c), _stream()))

    def bacon_score(self, layer, batch: BatchLayout, q_win, k, want_lse=False):
        import torch
        Hkv, T = self.shape.num_kv_heads, batch.total
        B = torch.empty((Hkv, T), dtype=torch.float32, device=k.device)
        Q = torch.empty((Hkv, T), dtype=torch.float32, device=k.device)
        lse = (torch.empty((len(batch.budgets), self.shape.num_q_heads, self.shape.window),
                           dtype=torch.float32, device=k.device) if want_lse else None)
        _check(lib().bacon_score(self._h, layer, C.byref(batch.c), _ptr(q_win), _ptr(k),
                                 _ptr(lse), _ptr(B), _ptr(Q), _stream()))
        return B, Q, lse

    def bacon_calibrate(self, layer, batch: BatchLayout, B, Q, want_E=False, want_V=False):
        import torch
        Hkv, T = self.shape.num_kv_heads, batch.total
        S = torch.empty((Hkv, T), dtype=torch.float32, device=B.device)
        lam = torch.empty((len(batch.budgets), Hkv), dtype=torch.float32, device=B.device)
        E = torch.empty_like(S) if want_E else None
        V = torch.empty_like(S) if want_V else None
        _check(lib().bacon_calibrate(self._h, layer, C.byref(batch.c), _ptr(B), _ptr(Q), _ptr(S),
                                     _ptr(lam), _ptr(E), _ptr(V), _stream()))
        return {"S": S, "lambda": lam, "E": E, "V": V}

    def bacon_select_topk(self, batch: BatchLayout, S):
        import torch
        idx = torch.empty(batch.idx_count(self.shape.num_kv_heads), dtype=torch.int32,
                          device=S.device)
        _check(lib().bacon_select_topk(self._h, C.byref(batch.c), _ptr(S), _ptr(idx), _stream()))
        return idx

    def _kv_out(self, batch: BatchLayout, like):
        import torch
        rows = batch.kept_rows(self.shape.window, self.shape.num_kv_heads)
        shp = (rows, self.shape.num_kv_heads, self.shape.head_dim)
        return (torch.empty(shp, dtype=like.dtype, device=like.device),
                torch.empty(shp, dtype=like.dtype, device=like.device))

    def bacon_compact(self, batch: BatchLayout, k, v, idx):
        k_out, v_out = self._kv_out(batch, k)
        _check(lib().bacon_compact(self._h, C.byref(batch.c), _ptr(k), _ptr(v), _ptr(idx),
                                   _ptr(k_out), _ptr(v_out), _stream()))
        return k_out, v_out

    def bacon_compress_layer(self, layer, batch: BatchLayout, q_win, k, v, out=None):
        import torch
        if out is None:
            idx = torch.empty(batch.idx_count(self.shape.num_kv_heads), dtype=torch.int32,
                              device=k.device)
            k_out, v_out = self._kv_out(batch, k)
        else:
            idx, k_out, v_out = out
        _check(lib().bacon_compress_layer(self._h, layer, C.byref(batch.c), _ptr(q_win), _ptr(k),
                                          _ptr(v), _ptr(idx), _ptr(k_out), _ptr(v_out),
                                          _stream()))
        return idx, k_out, v_out

    def bacon_compress_layer_lse(self, layer, batch: BatchLayout, q_win, k, v, lse, out=None):
        """The fused pass with the window-row normalisers lse [B, Hq, W] (natural
        log) given, e.g. by the prefill attention."""
        import torch
        if out is None:
            idx = torch.empty(batch.idx_count(self.shape.num_kv_heads), dtype=torch.int32,
                              device=k.device)
            k_out, v_out = self._kv_out(batch, k)
        else:
            idx, k_out, v_out = out
        _check(lib().bacon_compress_layer_lse(self._h, layer, C.byref(batch.c), _ptr(q_win),
                                              _ptr(k), _ptr(v), _ptr(lse), _ptr(idx),
                                              _ptr(k_out), _ptr(v_out), _stream()))
        return idx, k_out, v_out

    def bacon_compress_prompt(self, first_layer, batch: BatchLayout, q_wins, ks, vs, lses=None,
                              outs=None, layer_batches=None):
        """The pass over layers first_layer .. first_layer + len(ks) - 1 in one
        call; returns [(idx, k_out, v_out)] per layer.  layer_batches: None, or
        one BatchLayout per layer (same sequences, the layer's own budgets)."""
        import torch
        n = len(ks)
        lb = layer_batches if layer_batches is not None else [batch] * n
        if outs is None:
            outs = []
            for k, b in zip(ks, lb):
                idx = torch.empty(b.idx_count(self.shape.num_kv_heads), dtype=torch.int32,
                                  device=k.device)
                outs.append((idx, *self._kv_out(b, k)))
        arr = lambda xs: (C.c_void_p * n)(*[x.data_ptr() for x in xs])
        lse_arr = arr(lses) if lses is not None else None
        lb_arr = None
        if layer_batches is not None:
            lb_arr = (C.c_void_p * n)(*[C.cast(C.byref(b.c), C.c_void_p).value for b in layer_batches])
        _check(lib().bacon_compress_prompt(
            self._h, C.byref(batch.c), first_layer, n, arr(q_wins), arr(ks), arr(vs), lse_arr,
            arr([o[0] for o in outs]), arr([o[1] for o in outs]), arr([o[2] for o in outs]),
            lb_arr, _stream()))
        return outs

    def bacon_debug_device_errors(self) -> int:
        """Test instrumentation: the device error word (synchronises)."""
        return int(lib().bacon_debug_device_errors(self._h))

    def bacon_allocate_heads(self, batch: BatchLayout, B, out=None):
        """AdaKV's head-wise budgets K_{b,h} [batch, Hkv] (int32 device tensor)
        from a window score B [Hkv, T]."""
        import torch
        bud = out if out is not None else torch.empty(
            (batch.c.batch, self.shape.num_kv_heads), dtype=torch.int32, device=B.device)
        _check(lib().bacon_allocate_heads(self._h, C.byref(batch.c), _ptr(B), _ptr(bud), _stream()))
        return bud

    def bacon_alloc_output(self, budgets=None):
        """Where the fused calls under the adaptive allocation write each
        layer's budgets: an int32 device tensor [num_layers, max_batch, Hkv],
        or None to stop."""
        _check(lib().bacon_alloc_output(self._h, _ptr(budgets)))

    def bacon_debug_capture(self, B=None, V=None, lam=None):
        """Test instrumentation: per-layer copies of B, V [L, Hkv, T] and lambda
        [L, B, Hkv] (float32 device tensors) from the fused calls; None turns it off."""
        _check(lib().bacon_debug_capture(self._h, _ptr(B), _ptr(V), _ptr(lam)))

    def bacon_window_lse(self, batch: BatchLayout, q_win, k, out=None):
        """The window-row normalisers lse [B, Hq, W] (natural log) alone, as
        bacon_compress_layer_lse takes them."""
        import torch
        s = self.shape
        lse = out if out is not None else torch.empty(
            (batch.c.batch, s.num_q_heads, s.window), dtype=torch.float32, device=k.device)
        _check(lib().bacon_window_lse(self._h, C.byref(batch.c), _ptr(q_win), _ptr(k), _ptr(lse),
                                      _stream()))
        return lse

    def bacon_profile_enable(self, enable=True):
        _check(lib().bacon_profile_enable(self._h, 1 if enable else 0))

    def bacon_profile_read(self) -> dict:
        arr = (KernelTime * 32)()
        n = lib().bacon_profile_read(self._h, arr, 32)
        return {arr[i].name.decode(): (int(arr[i].launches), float(arr[i].total_ms))
                for i in range(max(0, n))}


# Module-level functions with the C names, for callers that prefer them.
def bacon_begin_prompt(ctx: Context, batch):
    return ctx.bacon_begin_prompt(batch)


def bacon_score(ctx: Context, layer, batch, q_win, k, want_lse=False):
    return ctx.bacon_score(layer, batch, q_win, k, want_lse)


def bacon_calibrate(ctx: Context, layer, batch, B, Q, want_E=False, want_V=False):
    return ctx.bacon_calibrate(layer, batch, B, Q, want_E, want_V)


def bacon_select_topk(ctx: Context, batch, S):
    return ctx.bacon_select_topk(batch, S)


def bacon_compact(ctx: Context, batch, k, v, idx):
    return ctx.bacon_compact(batch, k, v, idx)


def bacon_compress_layer(ctx: Context, layer, batch, q_win, k, v, out=None):
    return ctx.bacon_compress_layer(layer, batch, q_win, k, v, out)


def bacon_compress_layer_lse(ctx: Context, layer, batch, q_win, k, v, lse, out=None):
    return ctx.bacon_compress_layer_lse(layer, batch, q_win, k, v, lse, out)


def bacon_compress_prompt(ctx: Context, first_layer, batch, q_wins, ks, vs, lses=None, outs=None,
                          layer_batches=None):
    return ctx.bacon_compress_prompt(first_layer, batch, q_wins, ks, vs, lses, outs, layer_batches)


def bacon_window_lse_static(shape: Shape, batch: BatchLayout, q_win, k, out=None):
    """bacon_window_lse without a context or workspace (static device scratch);
    returns lse [B, Hq, W] (out if given)."""
    import torch
    lse = out if out is not None else torch.empty(
        (batch.c.batch, shape.num_q_heads, shape.window), dtype=torch.float32, device=k.device)
    _check(lib().bacon_window_lse_static(C.byref(shape), C.byref(batch.c), _ptr(q_win), _ptr(k),
                                         _ptr(lse), _stream()))
    return lse


def bacon_debug_capture(ctx: Context, B=None, V=None, lam=None):
    return ctx.bacon_debug_capture(B, V, lam)


def bacon_window_lse(ctx: Context, batch, q_win, k, out=None):
    return ctx.bacon_window_lse(batch, q_win, k, out)
