"""ctypes wrapper of the fp64 CPU oracle (``oracle/bacon_ref.c``).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg.  It never touches the GPU library.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libbacon_ref.so")
_SRC = os.path.join(_HERE, "bacon_ref.c")

_dp = C.POINTER(C.c_double)
_ip = C.POINTER(C.c_int32)
_fp = C.POINTER(C.c_float)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, strict IEEE doubles)."""
    if force or not os.path.exists(_LIB_PATH):
        cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
               "-ffp-contract=off", "-Wall", "-Wextra", "-o", _LIB_PATH + ".tmp", _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


class _Cfg(C.Structure):
    _fields_ = [("num_q_heads", C.c_int), ("num_kv_heads", C.c_int), ("head_dim", C.c_int),
                ("window", C.c_int), ("radius", C.c_int), ("persist_m", C.c_int),
                ("rho", C.c_double), ("gamma", C.c_double), ("eps", C.c_double),
                ("pool_kernel", C.c_int), ("use_last_query", C.c_int), ("terms", C.c_int),
                ("pool_mode", C.c_int)]


class _Out(C.Structure):
    _fields_ = [("lse", _dp), ("B", _dp), ("Q", _dp), ("E", _dp), ("L", _dp), ("T", _dp),
                ("V", _dp), ("S", _dp), ("S_pool", _dp), ("lam", _dp), ("sigma_B", _dp),
                ("sigma_V", _dp), ("m_count", _ip), ("idx", _ip), ("n_kept", _ip)]


_lib = None


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = C.CDLL(_LIB_PATH)
        L.bacon_ref_scores.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, _fp, C.c_long, C.c_long,
                                       _fp, C.c_long, _dp, _dp, _dp, _dp]
        L.bacon_ref_residual.argtypes = [C.c_int, _dp, _dp, _dp]
        L.bacon_ref_coherence.argtypes = [C.c_int, C.c_int, _dp, _dp]
        L.bacon_ref_persistence.argtypes = [C.c_int, C.c_int, C.POINTER(_dp), _dp]
        L.bacon_ref_topk.argtypes = [C.c_int, _dp, C.c_int, _ip]
        L.bacon_ref_topk.restype = C.c_int
        L.bacon_ref_lambda.argtypes = [C.c_int, _dp, _dp, C.c_int, C.c_double, C.c_double,
                                       C.c_double, _dp, _dp, _ip]
        L.bacon_ref_lambda.restype = C.c_double
        L.bacon_ref_pool.argtypes = [C.c_int, C.c_int, _dp, _dp]
        L.bacon_ref_pool_max.argtypes = [C.c_int, C.c_int, _dp, _dp]
        L.bacon_ref_adaptive_budgets.argtypes = [C.c_int, C.c_int, _dp, C.c_long, C.c_int,
                                                 C.c_double, _ip]
        L.bacon_ref_layer.argtypes = [C.POINTER(_Cfg), C.c_int, C.c_int, _ip, _ip, _fp, _fp,
                                      _dp, C.POINTER(_Out)]
        L.bacon_ref_layer.restype = C.c_int
        L.bacon_ref_compact.argtypes = [C.c_int, _ip, _ip, C.c_int, C.c_int, C.c_int, C.c_size_t,
                                        _ip, _ip, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.bacon_ref_set_threads.argtypes = [C.c_int]
        L.bacon_ref_get_threads.restype = C.c_int
        _lib = L
    return _lib


def _d(a):
    return None if a is None else a.ctypes.data_as(_dp)


def _i(a):
    return None if a is None else a.ctypes.data_as(_ip)


def _f(a):
    return a.ctypes.data_as(_fp)


def set_threads(n: int) -> None:
    lib().bacon_ref_set_threads(int(n))


def get_threads() -> int:
    return int(lib().bacon_ref_get_threads())


# ---------------------------------------------------------------- step functions

def scores(q: np.ndarray, k: np.ndarray, want_attn: bool = False) -> dict:
    """q ``[G, W, d]`` and k ``[n, d]`` float32 -> B, Q (and lse, attention rows)."""
    q = np.ascontiguousarray(q, dtype=np.float32)
    k = np.ascontiguousarray(k, dtype=np.float32)
    G, W, d = q.shape
    n = k.shape[0]
    B = np.zeros(n)
    Q = np.zeros(n)
    lse = np.zeros(G * W)
    attn = np.zeros(G * W * n) if want_attn else None
    lib().bacon_ref_scores(n, W, G, d, _f(q), d, W * d, _f(k), d, _d(lse), _d(attn), _d(B), _d(Q))
    out = {"B": B, "Q": Q, "lse": lse.reshape(G, W)}
    if want_attn:
        out["attn"] = attn.reshape(G, W, n)
    return out


def residual(B: np.ndarray, Q: np.ndarray) -> np.ndarray:
    B = np.ascontiguousarray(B, dtype=np.float64)
    Q = np.ascontiguousarray(Q, dtype=np.float64)
    E = np.zeros_like(B)
    lib().bacon_ref_residual(len(B), _d(B), _d(Q), _d(E))
    return E


def coherence(E: np.ndarray, radius: int) -> np.ndarray:
    E = np.ascontiguousarray(E, dtype=np.float64)
    L = np.zeros_like(E)
    lib().bacon_ref_coherence(len(E), radius, _d(E), _d(L))
    return L


def persistence(prev: list, n: int) -> np.ndarray:
    arrs = [np.ascontiguousarray(p, dtype=np.float64) for p in prev]
    ptrs = (_dp * max(1, len(arrs)))(*[_d(a) for a in arrs])
    T = np.zeros(n)
    lib().bacon_ref_persistence(n, len(arrs), ptrs, _d(T))
    return T


def topk(x: np.ndarray, k: int) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.zeros(max(1, k), dtype=np.int32)
    cnt = lib().bacon_ref_topk(len(x), _d(x), k, _i(out))
    return out[:cnt].copy()


def lambda_(B, V, n_cand: int, budget: int, rho=2.0, gamma=1.0, eps=1e-12) -> dict:
    B = np.ascontiguousarray(B, dtype=np.float64)
    V = np.ascontiguousarray(V, dtype=np.float64)
    sb, sv = C.c_double(), C.c_double()
    mc = C.c_int32()
    lam = lib().bacon_ref_lambda(n_cand, _d(B), _d(V), budget, rho, gamma, eps,
                                 C.byref(sb), C.byref(sv), C.byref(mc))
    return {"lambda": lam, "sigma_B": sb.value, "sigma_V": sv.value, "m_count": mc.value}


def pool(x: np.ndarray, kernel: int) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.zeros_like(x)
    lib().bacon_ref_pool(len(x), kernel, _d(x), _d(out))
    return out


def pool_max(x: np.ndarray, kernel: int) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.zeros_like(x)
    lib().bacon_ref_pool_max(len(x), kernel, _d(x), _d(out))
    return out


def adaptive_budgets(A: np.ndarray, budget: int, floor_alpha: float) -> np.ndarray:
    """AdaKV's head-wise allocation of one (layer, sequence): K_h from the
    backbone scores A [H, n_cand] (App. B; see bacon_ref_adaptive_budgets)."""
    A = np.ascontiguousarray(A, dtype=np.float64)
    H, n = A.shape
    out = np.zeros(H, np.int32)
    lib().bacon_ref_adaptive_budgets(H, n, _d(A), n, int(budget), float(floor_alpha), _i(out))
    return out


# ---------------------------------------------------------------- whole layers

@dataclass
class Params:
    radius: int = 5
    persist_m: int = 4
    rho: float = 2.0
    gamma: float = 1.0
    eps: float = 1e-12
    use_last_query: int = 1
    terms: int = 7
    pool_mode: int = 0          # 0 mean of S, 1 max of S, 2 mean of B before calibration


class Prompt:
    """Runs the oracle layer by layer over one packed batch, keeping E history."""

    def __init__(self, num_layers, num_q_heads, num_kv_heads, head_dim, window, pool_kernel,
                 cu_seqlens, budgets, params: Params | None = None):
        p = params or Params()
        self.cfg = _Cfg(num_q_heads, num_kv_heads, head_dim, window, p.radius, p.persist_m,
                        p.rho, p.gamma, p.eps, pool_kernel, p.use_last_query, p.terms,
                        p.pool_mode)
        self.cu = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
        self.budgets = np.ascontiguousarray(budgets, dtype=np.int32)
        self.batch = len(self.budgets)
        self.T = int(self.cu[-1])
        self.Hq, self.Hkv, self.d, self.W = num_q_heads, num_kv_heads, head_dim, window
        self.e_hist = np.zeros((num_layers, num_kv_heads, self.T))
        self.num_layers = num_layers

    @classmethod
    def for_workload(cls, wl, params: Params | None = None):
        return cls(wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window,
                   wl.pool_kernel, wl.cu_seqlens, wl.budgets_arr, params)

    def layer(self, layer: int, q_win: np.ndarray, k: np.ndarray, budgets=None,
              head_budgets=None) -> dict:
        """One layer.  ``budgets`` overrides the prompt's per-sequence budgets
        for this layer only (a per-layer budget schedule); ``head_budgets``
        [batch, Hkv] gives every (sequence, KV head) its own budget."""
        B_, Hq, Hkv, W, T = self.batch, self.Hq, self.Hkv, self.W, self.T
        bud = self.budgets if budgets is None else np.ascontiguousarray(budgets, dtype=np.int32)
        assert bud.shape == self.budgets.shape
        if head_budgets is None:
            bh = np.ascontiguousarray(np.repeat(bud[:, None], Hkv, axis=1), dtype=np.int32)
        else:
            bh = np.ascontiguousarray(head_budgets, dtype=np.int32).reshape(B_, Hkv)
        q_win = np.ascontiguousarray(q_win, dtype=np.float32)
        k = np.ascontiguousarray(k, dtype=np.float32)
        assert q_win.shape == (B_ * W, Hq, self.d) and k.shape == (T, Hkv, self.d)
        vec = lambda: np.zeros((Hkv, T))
        sc = lambda: np.zeros((B_, Hkv))
        r = {"lse": np.zeros((B_, Hq, W)), "B": vec(), "Q": vec(), "E": vec(), "L": vec(),
             "T": vec(), "V": vec(), "S": vec(), "S_pool": vec(), "lambda": sc(),
             "sigma_B": sc(), "sigma_V": sc(), "m_count": np.zeros((B_, Hkv), np.int32),
             "idx": np.zeros(int(bh.sum()), np.int32),
             "n_kept": np.zeros((B_, Hkv), np.int32), "budgets": bh}
        out = _Out(_d(r["lse"]), _d(r["B"]), _d(r["Q"]), _d(r["E"]), _d(r["L"]), _d(r["T"]),
                   _d(r["V"]), _d(r["S"]), _d(r["S_pool"]), _d(r["lambda"]), _d(r["sigma_B"]),
                   _d(r["sigma_V"]), _i(r["m_count"]), _i(r["idx"]), _i(r["n_kept"]))
        rc = lib().bacon_ref_layer(C.byref(self.cfg), layer, B_, _i(self.cu), _i(bh),
                                   _f(q_win), _f(k), _d(self.e_hist), C.byref(out))
        if rc != 0:
            raise ValueError("oracle rejected the layer arguments")
        return r

    def layer_adaptive(self, layer: int, q_win: np.ndarray, k: np.ndarray, floor_alpha: float,
                       budgets=None) -> dict:
        """One layer on the AdaKV backbone (App. B): the head-wise budgets
        K_{b,h} are AdaKV's allocation of each sequence's H_kv K_b slots by
        the backbone score, the mean pool of B over the candidates (the
        SnapKV-style window score, with this prompt's pool width); BACON then
        keeps the top K_{b,h} of its own score in each head.  Runs the layer
        once for B (E and the history are the same under any budgets) and
        again with the allocation."""
        bud = self.budgets if budgets is None else np.ascontiguousarray(budgets, dtype=np.int32)
        r0 = self.layer(layer, q_win, k, budgets=bud)
        bh = np.zeros((self.batch, self.Hkv), np.int32)
        for b in range(self.batch):
            s0, s1 = int(self.cu[b]), int(self.cu[b + 1])
            nc = (s1 - s0) - self.W
            if nc <= 0:
                bh[b] = bud[b]
                continue
            A = np.stack([pool(r0["B"][h, s0:s0 + nc], self.cfg.pool_kernel)
                          for h in range(self.Hkv)])
            bh[b] = adaptive_budgets(A, int(bud[b]), floor_alpha)
        r = self.layer(layer, q_win, k, budgets=bud, head_budgets=bh)
        r["alloc_budgets"] = bh
        return r

    def _bh(self, r: dict) -> np.ndarray:
        return r.get("budgets", np.repeat(self.budgets[:, None], self.Hkv, axis=1))

    def idx_of(self, r: dict, b: int, h: int) -> np.ndarray:
        """Kept positions of (sequence b, KV head h), without -1 padding."""
        bh = self._bh(r)
        off = int(bh.reshape(-1)[:b * self.Hkv + h].sum())
        ids = r["idx"][off:off + int(bh[b, h])]
        return ids[ids >= 0]

    def compact(self, r: dict, k_bytes: np.ndarray, v_bytes: np.ndarray, elem_size: int):
        bh = np.ascontiguousarray(self._bh(r), dtype=np.int32)
        rows = int((bh.max(axis=1) + self.W).sum())
        shape = (rows, self.Hkv, self.d * elem_size)
        k_out = np.zeros(shape, np.uint8)
        v_out = np.zeros(shape, np.uint8)
        kb = np.ascontiguousarray(k_bytes).view(np.uint8)
        vb = np.ascontiguousarray(v_bytes).view(np.uint8)
        lib().bacon_ref_compact(self.batch, _i(self.cu), _i(bh), self.Hkv, self.d,
                                self.W, elem_size, _i(r["idx"]), _i(r["n_kept"]),
                                kb.ctypes.data, vb.ctypes.data, k_out.ctypes.data,
                                v_out.ctypes.data)
        return k_out, v_out
