"""Helpers shared by the GPU parity tests: run the oracle and the HIP path on
the same seeded inputs and compare them with the tolerances of the contract."""
from __future__ import annotations

import sys

import numpy as np

from oracle import ref
from paper_2606_14782_amd import inputs

# Score tolerance: |x - x_ref| <= RTOL * (|x_ref| + mean |x_ref|) element by
# element; near the selection boundaries the scores are also held to the
# plain relative bound |x - x_ref| <= RTOL * |x_ref| (check_near_boundary).
RTOL = {"fp32": 1e-5, "bf16": 1e-2}

# A (sequence, KV head) whose oracle gaps at the M-th (scale-matching set)
# and K-th (kept set) boundaries both exceed GAP_TOL relative must have
# exactly the oracle's kept set.  The GPU's scores come from the same exact
# inputs in fp32 with hardware exp2; the single-read pass keeps the window-row
# probabilities between its two halves in fp16 (relative rounding at most
# 2^-11 per element), which leaves B within about 2e-4 of the oracle near the
# selection boundaries.  GAP_TOL leaves a fivefold margin.  Closer boundaries
# may swap positions whose pooled scores agree within RTOL of the K-th score.
GAP_TOL = 1e-3


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def params_for(wl, **kw):
    from paper_2606_14782_amd import bacon
    d = dict(pool_kernel=wl.pool_kernel)
    d.update(kw)
    return bacon.default_params(**d)


def oracle_params(**kw):
    return ref.Params(**kw)


def make_ctx(wl, params=None, max_total=None):
    from paper_2606_14782_amd import bacon
    return bacon.Context(wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.window,
                         wl.batch, max_total or wl.total_tokens, wl.dtype,
                         params or params_for(wl))


def to_dev(x, wl):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    return t.to(torch.bfloat16) if wl.dtype == "bf16" else t


def close(name, got, want, rtol):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, f"{name}: shape {got.shape} vs {want.shape}"
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    scale = np.abs(want) + np.mean(np.abs(want))
    err = np.abs(got - want)
    worst = float(np.max(err / np.maximum(scale, 1e-300))) if err.size else 0.0
    bad = err > rtol * scale
    assert not bad.any(), (f"{name}: {int(bad.sum())}/{bad.size} beyond rtol {rtol}; worst "
                           f"{worst:.3g}; first at {np.argwhere(bad)[0].tolist()}")
    return worst


def candidate_mask(wl):
    """[Hkv, T] mask of the candidate positions (all but each sequence's window)."""
    m = np.zeros((wl.num_kv_heads, wl.total_tokens), bool)
    for b in range(wl.batch):
        c0, c1 = int(wl.cu_seqlens[b]), int(wl.cu_seqlens[b + 1])
        m[:, c0:c1 - wl.window] = True
    return m


def seq_slices(wl):
    cu = wl.cu_seqlens
    return [(int(cu[b]), int(cu[b + 1])) for b in range(wl.batch)]


def _head_budgets(wl, hb):
    """[batch, Hkv] budgets: hb, or every head at its sequence's budget."""
    if hb is not None:
        return np.asarray(hb, np.int64).reshape(wl.batch, wl.num_kv_heads)
    return np.repeat(np.asarray(wl.budgets, np.int64)[:, None], wl.num_kv_heads, axis=1)


def rel_gap(vals, k):
    """Relative gap between the k-th and (k+1)-th largest of vals; inf when
    either does not exist (nothing to swap across)."""
    n = len(vals)
    if k <= 0 or k >= n:
        return np.inf
    part = np.partition(np.asarray(vals, np.float64), [n - k - 1, n - k])
    a, c = part[n - k], part[n - k - 1]
    return float((a - c) / max(abs(a), 1e-300))


def check_idx(name, got, r, wl, rtol, hb=None, strict=False, stats=None):
    """Kept sets against the oracle's.  With strict, or where the oracle's
    relative gaps at the M-th boundary of B and at the K-th boundary of the
    pooled score both exceed GAP_TOL, the set must be the oracle's exactly
    (ties then follow score descending, position ascending); elsewhere it may
    differ only in positions whose pooled oracle score is within rtol of the
    K-th kept score.  hb: optional per-(sequence, KV head) budgets [batch,
    Hkv].  Returns (and accumulates into stats) counts of pairs, exact sets,
    pairs held to exactness, and swaps."""
    W, Hkv = wl.window, wl.num_kv_heads
    bh = _head_budgets(wl, hb)
    if stats is None:
        stats = {}
    for key in ("pairs", "strict", "gated", "swaps"):
        stats.setdefault(key, 0)
    off = 0
    for b, (s0, s1) in enumerate(seq_slices(wl)):
        nc = (s1 - s0) - W
        for h in range(Hkv):
            K = int(bh[b, h])
            g = np.asarray(got[off:off + K])
            o = np.asarray(r["idx"][off:off + K])
            off += K
            kept = min(K, max(nc, 0))
            assert np.all(g[kept:] == -1), f"{name} b{b} h{h}: padding"
            gk = g[:kept]
            assert np.all(np.diff(gk) > 0), f"{name} b{b} h{h}: not ascending/unique"
            assert kept == 0 or (gk.min() >= 0 and gk.max() < nc), f"{name} b{b} h{h}: range"
            gs, os_ = set(gk.tolist()), set(o[:kept].tolist())
            stats["pairs"] += 1
            P = r["S_pool"][h, s0:s0 + nc]
            M = int(r["m_count"][b, h])
            exact = strict or (rel_gap(P, K) > GAP_TOL and
                               (M == 0 or rel_gap(r["B"][h, s0:s0 + nc], M) > GAP_TOL))
            stats["gated"] += int(exact)
            if gs == os_:
                stats["strict"] += 1
                continue
            assert not exact, (
                f"{name} b{b} h{h}: kept set differs from the oracle's where it must be exact "
                f"(strict={strict}, K-gap {rel_gap(P, K):.3g}, M-gap "
                f"{rel_gap(r['B'][h, s0:s0 + nc], M):.3g}); GPU-only {sorted(gs - os_)[:8]}, "
                f"oracle-only {sorted(os_ - gs)[:8]}")
            pK = float(P[list(os_)].min())
            for i in gs ^ os_:
                assert abs(P[i] - pK) <= rtol * abs(pK), (
                    f"{name} b{b} h{h}: position {i} differs, oracle score {P[i]:.9g} vs "
                    f"K-th {pK:.9g}")
            stats["swaps"] += len(gs - os_)
    return stats


def _lambda_of(B, V, sel, gamma, eps):
    """lambda = gamma Std(B) / (Std(V) + eps) over the set sel (population
    Std, in fp64; Eq. lambda_solution)."""
    return gamma * float(np.std(B[sel])) / (float(np.std(V[sel])) + eps)


def lambda_choices(r, b, h, s0, nc, gamma=1.0, eps=1e-12, max_band=10):
    """The lambdas of every scale-matching set that resolves a tie at the
    oracle's M-th boundary within GAP_TOL: the positions whose B is within
    GAP_TOL relative of the M-th largest form a band, the set takes every
    position above the band and any subset of the band of the remaining size.
    One value (the oracle's) when the boundary is not tied."""
    from itertools import combinations
    M = int(r["m_count"][b, h])
    lam = float(r["lambda"][b, h])
    if M == 0 or M >= nc or lam == 0.0:
        return [lam]
    B = np.asarray(r["B"][h, s0:s0 + nc], np.float64)
    V = np.asarray(r["V"][h, s0:s0 + nc], np.float64)
    bM = float(np.sort(B)[nc - M])
    tol = GAP_TOL * abs(bM)
    above = np.nonzero(B > bM + tol)[0]
    band = np.nonzero(np.abs(B - bM) <= tol)[0]
    need = M - len(above)
    if len(band) <= need or len(band) > max_band:
        return [lam]
    return [lam] + [_lambda_of(B, V, np.concatenate([above, list(c)]).astype(np.int64), gamma, eps)
                    for c in combinations(band.tolist(), need)]


def check_lambda(name, got, r, wl, rtol, gamma=1.0, eps=1e-12, B_gpu=None, V_gpu=None,
                 stats=None):
    """lambda of every (sequence, KV head) within rtol of the oracle's, or,
    given the GPU's own window score B_gpu [Hkv, T] (and evidence V_gpu), of
    what the GPU's B and V allow: the set the GPU's B selects may differ from
    the oracle's only in positions tied within GAP_TOL at the M-th boundary,
    and on that set, with dB and dV the largest deviations of the GPU's B and
    V from the oracle's there (each checked against the oracle on its own),
    Std(B) and Std(V) can move by at most dB and dV (Std is 1-Lipschitz in
    the max norm), which bounds gamma Std(B) / (Std(V) + eps) to an interval
    that lambda must meet within rtol.  The interval is wide only where the
    set's B or V are nearly constant (identical keys, constant evidence),
    where lambda is ill-conditioned.  Without B_gpu, lambda must be within
    rtol of the fp64 lambda of some set resolving a tie of at most a few
    positions."""
    got = np.asarray(got, np.float64)
    worst = 0.0
    for b, (s0, s1) in enumerate(seq_slices(wl)):
        nc = (s1 - s0) - wl.window
        for h in range(wl.num_kv_heads):
            g = float(got[b, h])
            want = float(r["lambda"][b, h])
            err = abs(g - want) / max(abs(want), 1e-300)
            if abs(g - want) <= rtol * abs(want):
                worst = max(worst, err)
                continue
            M = int(r["m_count"][b, h])
            if B_gpu is not None and 0 < M < nc:
                Bref = np.asarray(r["B"][h, s0:s0 + nc], np.float64)
                Vref = np.asarray(r["V"][h, s0:s0 + nc], np.float64)
                Bg = np.asarray(B_gpu[h, s0:s0 + nc], np.float64)
                sel_g = np.lexsort((np.arange(nc), -Bg))[:M]
                sel_o = np.lexsort((np.arange(nc), -Bref))[:M]
                bM = float(Bref[sel_o[-1]])
                diff = np.setxor1d(sel_g, sel_o)
                assert np.all(np.abs(Bref[diff] - bM) <= GAP_TOL * abs(bM)), (
                    f"{name} b{b} h{h}: the GPU's scale-matching set differs from the oracle's "
                    f"outside the tie at its M-th boundary")
                sb, sv = float(np.std(Bref[sel_g])), float(np.std(Vref[sel_g]))
                dB = float(np.max(np.abs(Bg[sel_g] - Bref[sel_g])))
                dV = 0.0
                if V_gpu is not None:
                    Vg = np.asarray(V_gpu[h, s0:s0 + nc], np.float64)
                    dV = float(np.max(np.abs(Vg[sel_g] - Vref[sel_g])))
                lo = gamma * max(sb - dB, 0.0) / (sv + dV + eps)
                hi = gamma * (sb + dB) / (max(sv - dV, 0.0) + eps)
                assert lo * (1 - rtol) <= g <= hi * (1 + rtol), (
                    f"{name} b{b} h{h}: lambda {g:.9g} vs oracle {want:.9g}, outside "
                    f"[{lo:.9g}, {hi:.9g}] that the GPU's B and V allow on the set its B selects "
                    f"({len(diff) // 2} swaps in the tie)")
                if stats is not None:
                    stats["lambda_by_interval"] = stats.get("lambda_by_interval", 0) + 1
                continue
            alts = lambda_choices(r, b, h, s0, nc, gamma, eps)
            assert any(abs(g - x) <= rtol * abs(x) for x in alts), (
                f"{name} b{b} h{h}: lambda {g:.9g} vs oracle {want:.9g} (rel {err:.3g}); the "
                f"{len(alts) - 1} sets resolving a tie at the M-th boundary give {alts[1:6]}")
    return worst


def box_pool(x, k):
    """Centred average of odd width k over x, truncated at the ends, in fp64
    (the pooling convention; used on the GPU's unpooled scores)."""
    x = np.asarray(x, np.float64)
    n, half = len(x), k // 2
    c = np.concatenate([[0.0], np.cumsum(x)])
    i = np.arange(n)
    lo, hi = np.maximum(i - half, 0), np.minimum(i + half, n - 1)
    return (c[hi + 1] - c[lo]) / (hi - lo + 1)


def check_near_boundary(name, got, want, order_by, k, rtol, width=32):
    """The plain relative bound |x - x_ref| <= rtol |x_ref| on the positions the
    oracle ranks k - width .. k + width by order_by (score descending, position
    ascending): the scores the selection turns on."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    n = len(want)
    if n == 0 or k <= 0:
        return 0.0
    k = min(k, n)
    rank = np.lexsort((np.arange(n), -np.asarray(order_by, np.float64)))
    sel = rank[max(0, k - width):min(n, k + width)]
    err = np.abs(got[sel] - want[sel])
    bad = err > rtol * np.abs(want[sel])
    assert not bad.any(), (f"{name}: {int(bad.sum())} of {len(sel)} near-boundary values beyond "
                           f"rtol {rtol}: first at position {int(sel[np.argmax(bad)])}, "
                           f"{got[sel][bad][0]:.9g} vs {want[sel][bad][0]:.9g}")
    return float(np.max(err / np.maximum(np.abs(want[sel]), 1e-300)))


def gather_rows(x_bytes, idx, wl, hb=None):
    """Expected compacted rows for GPU indices (bit copy of the input rows);
    each sequence has max_h K + W rows per head, zero-padded."""
    W, Hkv = wl.window, wl.num_kv_heads
    bh = _head_budgets(wl, hb)
    C = bh.max(axis=1)
    rows = int(np.sum(C + W))
    row_b = x_bytes.shape[-1]
    out = np.zeros((rows, Hkv, row_b), np.uint8)
    off, r0 = 0, 0
    for b, (s0, s1) in enumerate(seq_slices(wl)):
        n = s1 - s0
        for h in range(Hkv):
            K = int(bh[b, h])
            g = idx[off:off + K]
            off += K
            kept = g[g >= 0]
            src = np.concatenate([kept, np.arange(n - W, n)]).astype(np.int64)
            out[r0:r0 + len(src), h] = x_bytes[s0 + src, h]
        r0 += int(C[b]) + W
    return out


def as_bytes(x_f32, wl):
    """Raw bytes of an input tensor in its storage type, [T, Hkv, d*es]."""
    if wl.dtype == "bf16":
        u = inputs.bf16_bits(x_f32)
    else:
        u = np.ascontiguousarray(x_f32, np.float32)
    return u.view(np.uint8).reshape(x_f32.shape[0], x_f32.shape[1], -1)


def tensor_bytes(t):
    import torch
    a = t.detach().cpu()
    if a.dtype == torch.bfloat16:
        a = a.view(torch.int16)
    return a.numpy().view(np.uint8).reshape(a.shape[0], a.shape[1], -1)
