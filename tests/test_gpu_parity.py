"""GPU parity of the HIP path against the fp64 oracle (needs an MI355X).

Every case draws seeded inputs, runs the oracle layer by layer, and runs the
HIP path through the C ABI both as split calls (score, calibrate, select,
compact) and as the fused per-layer call.  Scores are compared element by
element with |x - x_ref| <= rtol (|x_ref| + mean|x_ref|) (rtol 1e-5 for fp32
inputs, 1e-2 for bf16), and near the M-th and K-th selection boundaries with
the plain relative bound |x - x_ref| <= rtol |x_ref|.  Kept sets must be the
oracle's exactly where its gaps at both boundaries exceed GAP_TOL (and in the
exact-tie cases), and elsewhere may swap only positions whose pooled oracle
score is within rtol of the K-th; the compacted cache must be a bit copy of
the input rows named by the GPU's indices.  The fused calls' own B, V and
lambda are read back through bacon_debug_capture and compared too.
"""
import numpy as np
import pytest

import parity as P
from oracle import ref
from paper_2606_14782_amd import inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_14782_amd import bacon
    bacon.lib()
    ref.set_threads(16)


def _small(idx, **kw):
    return inputs.shrink(inputs.workload(idx), **kw)


CASES = {
    # model-shaped workloads at full sequence length and head count, fewer layers
    "tiny-fp32": lambda: inputs.workload(0),
    "llava-n2048": lambda: inputs.workload(1).with_(num_layers=6),
    "qwen2vl-n8192": lambda: inputs.workload(2).with_(num_layers=6),
    # seven layers: the E history (m + 1 = 5 slots) wraps around
    "video-n32768": lambda: inputs.workload(3).with_(num_layers=7),
    "ragged-b8": lambda: inputs.workload(4).with_(num_layers=7),
    # reduced shapes with ragged tails (lengths not multiples of the tile sizes)
    "llava-small": lambda: _small(1, num_layers=5, max_len=1500, num_kv_heads=4),
    "qwen2vl-small": lambda: _small(2, num_layers=5, max_len=2500, num_kv_heads=2),
    "video-small": lambda: _small(3, num_layers=3, max_len=3000, num_kv_heads=2),
    "ragged-small": lambda: _small(4, num_layers=5, max_len=3000, num_kv_heads=2),
}


def run_case(name, wl, gpu_kw=None, orc_kw=None, split=True, fused=True, make=None,
             supplied_lse=False, strict=False):
    import torch
    from paper_2606_14782_amd import bacon
    rtol = P.RTOL[wl.dtype]
    P.log(f"[{name}] {wl.name} B={wl.batch} L={wl.num_layers} Hq={wl.num_q_heads} "
          f"Hkv={wl.num_kv_heads} d={wl.head_dim} W={wl.window} lens={wl.seq_lens[:8]}")
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    orc = ref.Prompt.for_workload(wl, P.oracle_params(**(orc_kw or {})))
    ctx_s = P.make_ctx(wl, P.params_for(wl, **(gpu_kw or {}))) if split else None
    ctx_f = P.make_ctx(wl, P.params_for(wl, **(gpu_kw or {}))) if fused else None
    ctx_l = P.make_ctx(wl, P.params_for(wl, **(gpu_kw or {}))) if supplied_lse else None
    if split:
        ctx_s.bacon_begin_prompt(batch)
    if fused:
        ctx_f.bacon_begin_prompt(batch)
    if supplied_lse:
        ctx_l.bacon_begin_prompt(batch)
    worst = {}
    stats = {}
    pool_mean_s = (gpu_kw or {}).get("pool_mode", 0) == 0
    cap = None
    if fused:
        # the fused call's own B, V and lambda, per layer
        T, Hkv = wl.total_tokens, wl.num_kv_heads
        cap = (torch.zeros((wl.num_layers, Hkv, T), dtype=torch.float32, device="cuda"),
               torch.zeros((wl.num_layers, Hkv, T), dtype=torch.float32, device="cuda"),
               torch.zeros((wl.num_layers, wl.batch, Hkv), dtype=torch.float32, device="cuda"))
        ctx_f.bacon_debug_capture(*cap)
    cmask = P.candidate_mask(wl)
    lam_kw = {k: v for k, v in (orc_kw or {}).items() if k in ("gamma", "eps")}
    for layer in range(wl.num_layers):
        x = make(layer) if make else inputs.layer_inputs(wl, layer)
        r = orc.layer(layer, x["q_win"], x["k"])
        q, k, v = P.to_dev(x["q_win"], wl), P.to_dev(x["k"], wl), P.to_dev(x["v"], wl)
        kb, vb = P.as_bytes(x["k"], wl), P.as_bytes(x["v"], wl)
        P.log(f"[{name}] layer {layer}")
        idx_split = None
        if split:
            B, Q, lse = ctx_s.bacon_score(layer, batch, q, k, want_lse=True)
            cal = ctx_s.bacon_calibrate(layer, batch, B, Q, want_E=True, want_V=True)
            idx = ctx_s.bacon_select_topk(batch, cal["S"])
            ko, vo = ctx_s.bacon_compact(batch, k, v, idx)
            torch.cuda.synchronize()
            want = dict(r)
            if (gpu_kw or {}).get("pool_mode") == 2:
                # pooling before calibration: the candidates' score is pool(B) + lambda V
                want["S"] = np.where(P.candidate_mask(wl), r["S_pool"], r["S"])
            for key, got in (("lse", lse), ("B", B), ("Q", Q), ("E", cal["E"]), ("V", cal["V"]),
                             ("S", cal["S"])):
                w = P.close(f"{name} L{layer} {key}", got.cpu().numpy(), want[key], rtol)
                worst[key] = max(worst.get(key, 0.0), w)
            w = P.check_lambda(f"{name} L{layer} lambda", cal["lambda"].cpu().numpy(), r, wl, rtol,
                               B_gpu=B.cpu().numpy(), V_gpu=cal["V"].cpu().numpy(), **lam_kw)
            worst["lambda"] = max(worst.get("lambda", 0.0), w)
            idx_split = idx.cpu().numpy()
            P.check_idx(f"{name} L{layer} split", idx_split, r, wl, rtol, strict=strict)
            near_boundary(f"{name} L{layer} split", wl, r, B.cpu().numpy(),
                          cal["S"].cpu().numpy() if pool_mean_s else None, rtol, worst)
            assert np.array_equal(P.tensor_bytes(ko), P.gather_rows(kb, idx_split, wl))
            assert np.array_equal(P.tensor_bytes(vo), P.gather_rows(vb, idx_split, wl))
        if supplied_lse:
            # the window-row normalisers given (here the oracle's, in float32)
            lse = torch.from_numpy(np.ascontiguousarray(r["lse"], dtype=np.float32)).to(q.device)
            idx, ko, vo = ctx_l.bacon_compress_layer_lse(layer, batch, q, k, v, lse)
            torch.cuda.synchronize()
            gl = idx.cpu().numpy()
            P.check_idx(f"{name} L{layer} supplied-lse", gl, r, wl, rtol, strict=strict)
            assert np.array_equal(P.tensor_bytes(ko), P.gather_rows(kb, gl, wl)), "K gather"
            assert np.array_equal(P.tensor_bytes(vo), P.gather_rows(vb, gl, wl)), "V gather"
        if fused:
            idx, ko, vo = ctx_f.bacon_compress_layer(layer, batch, q, k, v)
            torch.cuda.synchronize()
            gi = idx.cpu().numpy()
            P.check_idx(f"{name} L{layer} fused", gi, r, wl, rtol, strict=strict, stats=stats)
            check_captured(f"{name} L{layer} fused", wl, r, cap, layer, cmask, rtol, worst, lam_kw)
            assert np.array_equal(P.tensor_bytes(ko), P.gather_rows(kb, gi, wl)), "K gather"
            assert np.array_equal(P.tensor_bytes(vo), P.gather_rows(vb, gi, wl)), "V gather"
            if idx_split is not None:
                # both paths are checked against the oracle above; they round
                # pooling differently (pool(S) against pool(B) + lambda pool(V)),
                # so they may swap keys whose scores tie within the tolerance
                stats["fused_split_diff"] = stats.get("fused_split_diff", 0) + int(
                    np.count_nonzero(gi != idx_split))
        del q, k, v
    if fused:
        ctx_f.bacon_debug_capture()
        assert ctx_f.bacon_debug_device_errors() == 0, "a meeting of the single-read pass ran out"
    P.log(f"[{name}] ok; worst rel err {worst}; fused kept sets exact {stats.get('strict', 0)}/"
          f"{stats.get('pairs', 0)} ({stats.get('gated', 0)} held to exactness by their gaps), "
          f"swaps {stats.get('swaps', 0)}, fused/split index differences "
          f"{stats.get('fused_split_diff', 0)}")
    return worst, stats


def near_boundary(name, wl, r, B_gpu, S_gpu, rtol, worst):
    """Plain relative error of B near each head's M-th boundary and of the
    pooled S near its K-th boundary (S_gpu: unpooled GPU score over [Hkv, T],
    pooled here; None skips it)."""
    bh = P._head_budgets(wl, None)
    for b, (s0, s1) in enumerate(P.seq_slices(wl)):
        nc = (s1 - s0) - wl.window
        if nc <= 0:
            continue
        for h in range(wl.num_kv_heads):
            M = int(r["m_count"][b, h])
            Bref = r["B"][h, s0:s0 + nc]
            w = P.check_near_boundary(f"{name} b{b} h{h} B near M", B_gpu[h, s0:s0 + nc], Bref,
                                      Bref, M, rtol)
            worst["B@M"] = max(worst.get("B@M", 0.0), w)
            if S_gpu is not None:
                Sp = P.box_pool(S_gpu[h, s0:s0 + nc], wl.pool_kernel)
                Pref = r["S_pool"][h, s0:s0 + nc]
                w = P.check_near_boundary(f"{name} b{b} h{h} pooled S near K", Sp, Pref, Pref,
                                          int(bh[b, h]), rtol)
                worst["S@K"] = max(worst.get("S@K", 0.0), w)


def check_captured(name, wl, r, cap, layer, cmask, rtol, worst, lam_kw=None):
    """The fused call's own window score B (every position), evidence V (the
    candidates) and lambda, read back through bacon_debug_capture, against the
    oracle element by element, and B near the M-th boundary."""
    B = cap[0][layer].cpu().numpy()
    w = P.close(f"{name} captured B", B, r["B"], rtol)
    worst["cap B"] = max(worst.get("cap B", 0.0), w)
    V = cap[1][layer].cpu().numpy()
    if cmask.any():
        w = P.close(f"{name} captured V", V[cmask], r["V"][cmask], rtol)
        worst["cap V"] = max(worst.get("cap V", 0.0), w)
    lam = cap[2][layer].cpu().numpy()
    w = P.check_lambda(f"{name} captured lambda", lam, r, wl, rtol, B_gpu=B, V_gpu=V,
                       **(lam_kw or {}))
    worst["cap lambda"] = max(worst.get("cap lambda", 0.0), w)
    near_boundary(name + " captured", wl, r, B, None, rtol, worst)


@pytest.mark.parametrize("name", list(CASES))
def test_workload_parity(name):
    run_case(name, CASES[name]())


@pytest.mark.parametrize("name", ["tiny-fp32", "video-n32768", "ragged-small", "llava-small"])
def test_supplied_normalisers(name):
    """bacon_compress_layer_lse with the window-row normalisers given matches
    the oracle like the fused call."""
    run_case(name + "/lse", CASES[name](), split=False, supplied_lse=True)


@pytest.mark.parametrize("name", ["video-small", "ragged-small", "llava-small", "qwen2vl-small",
                                  "tiny-fp32", "video-n32768", "ragged-b8"])
def test_prompt_call_equals_layer_calls(name):
    """bacon_compress_prompt (the measured path) gives the per-layer calls'
    outputs bit for bit, whole or split into two calls, and with the
    normalisers supplied; its own B, V and lambda (read back through
    bacon_debug_capture) and its kept sets match the oracle in every layer,
    past the wrap-around of the E history on the full-size cases."""
    import torch
    from paper_2606_14782_amd import bacon
    wl = CASES[name]()
    wl = wl.with_(num_layers=min(wl.num_layers, 7))
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    xs = [inputs.layer_inputs(wl, l) for l in range(wl.num_layers)]
    qs = [P.to_dev(x["q_win"], wl) for x in xs]
    ks = [P.to_dev(x["k"], wl) for x in xs]
    vs = [P.to_dev(x["v"], wl) for x in xs]
    P.log(f"[prompt {name}] {wl.num_layers} layers")
    ref_ctx = P.make_ctx(wl, P.params_for(wl))
    ref_ctx.bacon_begin_prompt(batch)
    want = [ref_ctx.bacon_compress_layer(l, batch, qs[l], ks[l], vs[l]) for l in range(wl.num_layers)]
    ctx = P.make_ctx(wl, P.params_for(wl))
    T, Hkv, L = wl.total_tokens, wl.num_kv_heads, wl.num_layers
    cap = (torch.zeros((L, Hkv, T), dtype=torch.float32, device="cuda"),
           torch.zeros((L, Hkv, T), dtype=torch.float32, device="cuda"),
           torch.zeros((L, wl.batch, Hkv), dtype=torch.float32, device="cuda"))
    ctx.bacon_debug_capture(*cap)
    ctx.bacon_begin_prompt(batch)
    got = ctx.bacon_compress_prompt(0, batch, qs, ks, vs)
    torch.cuda.synchronize()
    ctx.bacon_debug_capture()
    # the measured path against the oracle, every layer
    orc = ref.Prompt.for_workload(wl, P.oracle_params())
    rtol, worst, stats = P.RTOL[wl.dtype], {}, {}
    cmask = P.candidate_mask(wl)
    for l in range(L):
        r = orc.layer(l, xs[l]["q_win"], xs[l]["k"])
        check_captured(f"{name} L{l} prompt call", wl, r, cap, l, cmask, rtol, worst)
        P.check_idx(f"{name} L{l} prompt call", got[l][0].cpu().numpy(), r, wl, rtol, stats=stats)
    assert ctx.bacon_debug_device_errors() == 0, "a meeting of the single-read pass ran out"
    P.log(f"[prompt {name}] vs oracle: worst {worst}; kept sets exact {stats['strict']}/"
          f"{stats['pairs']} ({stats['gated']} held to exactness by their gaps)")
    ctx.bacon_begin_prompt(batch)
    cut = wl.num_layers // 2
    got2 = (ctx.bacon_compress_prompt(0, batch, qs[:cut], ks[:cut], vs[:cut]) +
            ctx.bacon_compress_prompt(cut, batch, qs[cut:], ks[cut:], vs[cut:]))
    torch.cuda.synchronize()
    for l in range(wl.num_layers):
        for i, what in enumerate(("idx", "k_out", "v_out")):
            assert torch.equal(got[l][i], want[l][i]), f"layer {l} {what}"
            assert torch.equal(got2[l][i], want[l][i]), f"layer {l} {what} (two calls)"
    # normalisers supplied: the prompt call equals bacon_compress_layer_lse
    lses = [ctx.bacon_window_lse(batch, qs[l], ks[l]) for l in range(wl.num_layers)]
    ref_ctx.bacon_begin_prompt(batch)
    want = [ref_ctx.bacon_compress_layer_lse(l, batch, qs[l], ks[l], vs[l], lses[l])
            for l in range(wl.num_layers)]
    ctx.bacon_begin_prompt(batch)
    got = ctx.bacon_compress_prompt(0, batch, qs, ks, vs, lses=lses)
    torch.cuda.synchronize()
    for l in range(wl.num_layers):
        for i, what in enumerate(("idx", "k_out", "v_out")):
            assert torch.equal(got[l][i], want[l][i]), f"layer {l} {what} (normalisers given)"


@pytest.mark.parametrize("name,per_head", [("ragged-small", False), ("video-small", False),
                                           ("ragged-small", True)])
def test_prompt_call_budget_schedule(name, per_head):
    """A per-layer budget schedule on the measured path: bacon_compress_prompt
    with one batch per layer (a shrinking per-sequence schedule, or random
    per-(sequence, KV head) budgets that change every layer) equals the
    per-layer calls with the same batches bit for bit, and matches the oracle
    run with the same budgets."""
    import torch
    from paper_2606_14782_amd import bacon, budgets as sched
    wl = CASES[name]()
    L = wl.num_layers
    rng = np.random.default_rng(77)
    if per_head:
        hbs = [rng.integers(1, 2 * max(wl.budgets) + 1, size=(wl.batch, wl.num_kv_heads)).astype(np.int32)
               for _ in range(L)]
        lbs = [bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr, head_budgets=hb) for hb in hbs]
    else:
        per = [sched.pyramid(int(k), L, 0.25) for k in wl.budgets]
        bls = [np.array([per[b][l] for b in range(wl.batch)], np.int32) for l in range(L)]
        lbs = [bacon.BatchLayout(wl.cu_seqlens, bl) for bl in bls]
    xs = [inputs.layer_inputs(wl, l) for l in range(L)]
    qs = [P.to_dev(x["q_win"], wl) for x in xs]
    ks = [P.to_dev(x["k"], wl) for x in xs]
    vs = [P.to_dev(x["v"], wl) for x in xs]
    a, b = P.make_ctx(wl), P.make_ctx(wl)
    a.bacon_begin_prompt(lbs[0])
    want = [a.bacon_compress_layer(l, lbs[l], qs[l], ks[l], vs[l]) for l in range(L)]
    b.bacon_begin_prompt(lbs[0])
    got = b.bacon_compress_prompt(0, lbs[0], qs, ks, vs, layer_batches=lbs)
    torch.cuda.synchronize()
    orc = ref.Prompt.for_workload(wl, P.oracle_params())
    for l in range(L):
        for i, what in enumerate(("idx", "k_out", "v_out")):
            assert torch.equal(got[l][i], want[l][i]), f"{name} L{l} {what}"
        if per_head:
            r = orc.layer(l, xs[l]["q_win"], xs[l]["k"], head_budgets=hbs[l])
            P.check_idx(f"{name}/schedule L{l}", got[l][0].cpu().numpy(), r, wl, P.RTOL[wl.dtype],
                        hb=hbs[l])
        else:
            r = orc.layer(l, xs[l]["q_win"], xs[l]["k"], budgets=bls[l])
            P.check_idx(f"{name}/schedule L{l}", got[l][0].cpu().numpy(), r,
                        wl.with_(budgets=tuple(int(x) for x in bls[l])), P.RTOL[wl.dtype])


def test_prompt_calls_mix_with_layer_calls():
    """Prompt calls and per-layer calls in one prompt (layers 0-1 in a prompt
    call, 2 alone, 3 alone in a prompt call, 4 per layer) give the per-layer
    outputs: the history and the parity buffers carry over between them."""
    import torch
    from paper_2606_14782_amd import bacon
    wl = CASES["video-small"]().with_(num_layers=5)
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    xs = [inputs.layer_inputs(wl, l) for l in range(wl.num_layers)]
    qs = [P.to_dev(x["q_win"], wl) for x in xs]
    ks = [P.to_dev(x["k"], wl) for x in xs]
    vs = [P.to_dev(x["v"], wl) for x in xs]
    a, b = P.make_ctx(wl), P.make_ctx(wl)
    a.bacon_begin_prompt(batch)
    want = [a.bacon_compress_layer(l, batch, qs[l], ks[l], vs[l]) for l in range(wl.num_layers)]
    b.bacon_begin_prompt(batch)
    got = b.bacon_compress_prompt(0, batch, qs[:2], ks[:2], vs[:2])
    got.append(b.bacon_compress_layer(2, batch, qs[2], ks[2], vs[2]))
    got += b.bacon_compress_prompt(3, batch, qs[3:4], ks[3:4], vs[3:4])
    got.append(b.bacon_compress_layer(4, batch, qs[4], ks[4], vs[4]))
    torch.cuda.synchronize()
    for l in range(wl.num_layers):
        for i, what in enumerate(("idx", "k_out", "v_out")):
            assert torch.equal(got[l][i], want[l][i]), f"layer {l} {what}"


def test_prompt_call_with_a_budget_too_large_to_overlap():
    """A budget whose row table does not fit beside the score kernel's LDS:
    the prompt call keeps each layer's select to its own launches, and still
    equals the per-layer calls and the oracle."""
    import torch
    from paper_2606_14782_amd import bacon
    wl = inputs.Workload("big-budget", 3, 8, 2, 128, 32, 7, "bf16", (16384, 5000), (11000, 4000),
                         ((32, 16000), (32, 4700)), 0, 31)
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    xs = [inputs.layer_inputs(wl, l) for l in range(wl.num_layers)]
    qs = [P.to_dev(x["q_win"], wl) for x in xs]
    ks = [P.to_dev(x["k"], wl) for x in xs]
    vs = [P.to_dev(x["v"], wl) for x in xs]
    a, b = P.make_ctx(wl), P.make_ctx(wl)
    a.bacon_begin_prompt(batch)
    want = [a.bacon_compress_layer(l, batch, qs[l], ks[l], vs[l]) for l in range(wl.num_layers)]
    b.bacon_begin_prompt(batch)
    got = b.bacon_compress_prompt(0, batch, qs, ks, vs)
    torch.cuda.synchronize()
    orc = ref.Prompt.for_workload(wl, P.oracle_params())
    for l in range(wl.num_layers):
        for i, what in enumerate(("idx", "k_out", "v_out")):
            assert torch.equal(got[l][i], want[l][i]), f"layer {l} {what}"
        r = orc.layer(l, xs[l]["q_win"], xs[l]["k"])
        P.check_idx(f"big-budget L{l}", got[l][0].cpu().numpy(), r, wl, P.RTOL[wl.dtype])


PROMPT_VARIANTS = [
    ("max of S", {"pool_mode": 1}),
    ("mean of B", {"pool_mode": 2}),
    ("S = B", {"use_last_query": 0}),
    ("radius 0, m 0", {"radius": 0, "persist_m": 0}),
    ("m 8, terms E+T", {"persist_m": 8, "terms": 5}),
]


@pytest.mark.parametrize("variant", range(len(PROMPT_VARIANTS)), ids=[v[0] for v in PROMPT_VARIANTS])
def test_prompt_call_variants(variant):
    """The prompt call equals the per-layer calls bit for bit under other
    pooling, evidence and persistence settings, and with a budget per
    (sequence, KV head); the variants read other buffers in the select."""
    import torch
    from paper_2606_14782_amd import bacon
    _, kw = PROMPT_VARIANTS[variant]
    wl = CASES["ragged-small"]().with_(num_layers=4)
    rng = np.random.default_rng(5 + variant)
    hb = rng.integers(1, 2 * max(wl.budgets) + 1, size=(wl.batch, wl.num_kv_heads)).astype(np.int32)
    for batch in (bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr),
                  bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr, head_budgets=hb)):
        xs = [inputs.layer_inputs(wl, l) for l in range(wl.num_layers)]
        qs = [P.to_dev(x["q_win"], wl) for x in xs]
        ks = [P.to_dev(x["k"], wl) for x in xs]
        vs = [P.to_dev(x["v"], wl) for x in xs]
        a, b = P.make_ctx(wl, P.params_for(wl, **kw)), P.make_ctx(wl, P.params_for(wl, **kw))
        a.bacon_begin_prompt(batch)
        want = [a.bacon_compress_layer(l, batch, qs[l], ks[l], vs[l]) for l in range(wl.num_layers)]
        b.bacon_begin_prompt(batch)
        got = b.bacon_compress_prompt(0, batch, qs, ks, vs)
        torch.cuda.synchronize()
        for l in range(wl.num_layers):
            for i, what in enumerate(("idx", "k_out", "v_out")):
                assert torch.equal(got[l][i], want[l][i]), f"{PROMPT_VARIANTS[variant][0]} L{l} {what}"


@pytest.mark.parametrize("name,streaming", [("tiny-fp32", False), ("ragged-small", False),
                                            ("video-n32768", False), ("ragged-small", True)])
def test_window_lse(name, streaming, monkeypatch):
    """bacon_window_lse: the window-row normalisers alone match the oracle's,
    and fed to bacon_compress_layer_lse they give the oracle's kept sets."""
    import torch
    from paper_2606_14782_amd import bacon
    if streaming:
        monkeypatch.setenv("BACON_KEY_REGISTERS", "0")
    wl = CASES[name]().with_(num_layers=2)
    rtol = P.RTOL[wl.dtype]
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    orc = ref.Prompt.for_workload(wl, P.oracle_params())
    ctx = P.make_ctx(wl, P.params_for(wl))
    ctx.bacon_begin_prompt(batch)
    for layer in range(wl.num_layers):
        x = inputs.layer_inputs(wl, layer)
        r = orc.layer(layer, x["q_win"], x["k"])
        q, k, v = P.to_dev(x["q_win"], wl), P.to_dev(x["k"], wl), P.to_dev(x["v"], wl)
        P.log(f"[window_lse {name}{' streaming' if streaming else ''}] layer {layer}")
        lse = ctx.bacon_window_lse(batch, q, k)
        torch.cuda.synchronize()
        P.close(f"{name} L{layer} window_lse", lse.cpu().numpy(), r["lse"], rtol)
        idx, ko, vo = ctx.bacon_compress_layer_lse(layer, batch, q, k, v, lse)
        torch.cuda.synchronize()
        gi = idx.cpu().numpy()
        P.check_idx(f"{name} L{layer} window_lse + compress_layer_lse", gi, r, wl, rtol)
        assert np.array_equal(P.tensor_bytes(ko), P.gather_rows(P.as_bytes(x["k"], wl), gi, wl))
        del q, k, v


@pytest.mark.parametrize("name", ["video-n32768", "llava-small", "ragged-small"])
def test_streaming_passes(name, monkeypatch):
    """The two streaming K passes (the path of fp32 keys and of more than 128
    window rows), forced on shapes that take the key-register passes."""
    monkeypatch.setenv("BACON_KEY_REGISTERS", "0")
    run_case(name + "/streaming", CASES[name](), split=False)
    run_case(name + "/streaming-lse", CASES[name](), split=False, fused=False, supplied_lse=True)


@pytest.mark.parametrize("name", ["video-n32768", "ragged-small", "llava-small"])
def test_two_pass_path(name, monkeypatch):
    """The two-K-pass path (normaliser pass, then the scoring pass; the
    prompt call's dual launches) forced on shapes that take the single-read
    pass: parity with the oracle, and the prompt call equal to the per-layer
    calls bit for bit."""
    import torch
    from paper_2606_14782_amd import bacon
    monkeypatch.setenv("BACON_SINGLE", "0")
    wl = CASES[name]().with_(num_layers=3)
    run_case(name + "/two-pass", wl, split=False)
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    xs = [inputs.layer_inputs(wl, l) for l in range(wl.num_layers)]
    qs = [P.to_dev(x["q_win"], wl) for x in xs]
    ks = [P.to_dev(x["k"], wl) for x in xs]
    vs = [P.to_dev(x["v"], wl) for x in xs]
    a, b = P.make_ctx(wl), P.make_ctx(wl)
    a.bacon_begin_prompt(batch)
    want = [a.bacon_compress_layer(l, batch, qs[l], ks[l], vs[l]) for l in range(wl.num_layers)]
    b.bacon_begin_prompt(batch)
    got = b.bacon_compress_prompt(0, batch, qs, ks, vs)
    torch.cuda.synchronize()
    for l in range(wl.num_layers):
        for i, what in enumerate(("idx", "k_out", "v_out")):
            assert torch.equal(got[l][i], want[l][i]), f"{name} L{l} {what}"


@pytest.mark.parametrize("name", ["ragged-small", "video-small"])
def test_per_layer_budget_schedule(name):
    """Budgets that change from layer to layer within a prompt (a shrinking
    per-layer schedule per sequence): the fused call matches the oracle run
    with the same schedule, and the compacted cache follows each layer's
    budgets."""
    import torch
    from paper_2606_14782_amd import bacon, budgets as sched
    wl = CASES[name]()
    per = [sched.pyramid(int(k), wl.num_layers, 0.25) for k in wl.budgets]
    orc = ref.Prompt.for_workload(wl, P.oracle_params())
    ctx = P.make_ctx(wl)
    ctx.bacon_begin_prompt(bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr))
    rtol = P.RTOL[wl.dtype]
    for layer in range(wl.num_layers):
        bl = tuple(per[b][layer] for b in range(wl.batch))
        wll = wl.with_(budgets=bl)
        x = inputs.layer_inputs(wl, layer)
        r = orc.layer(layer, x["q_win"], x["k"], budgets=np.array(bl, np.int32))
        batch = bacon.BatchLayout(wl.cu_seqlens, wll.budgets_arr)
        idx, ko, vo = ctx.bacon_compress_layer(layer, batch, P.to_dev(x["q_win"], wl),
                                               P.to_dev(x["k"], wl), P.to_dev(x["v"], wl))
        torch.cuda.synchronize()
        gi = idx.cpu().numpy()
        P.check_idx(f"{name}/schedule L{layer}", gi, r, wll, rtol)
        assert np.array_equal(P.tensor_bytes(ko), P.gather_rows(P.as_bytes(x["k"], wl), gi, wll))
        assert np.array_equal(P.tensor_bytes(vo), P.gather_rows(P.as_bytes(x["v"], wl), gi, wll))


@pytest.mark.parametrize("name", ["ragged-small", "video-small", "llava-small"])
def test_head_budgets(name):
    """A budget per (sequence, KV head), as a head-wise allocation gives it:
    the fused call and the split calls match the oracle, and the compacted
    cache pads every head to its sequence's largest budget."""
    import torch
    from paper_2606_14782_amd import bacon
    wl = CASES[name]()
    rng = np.random.default_rng(11)
    hb = rng.integers(1, 2 * max(wl.budgets) + 1, size=(wl.batch, wl.num_kv_heads)).astype(np.int32)
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr, head_budgets=hb)
    orc = ref.Prompt.for_workload(wl, P.oracle_params())
    ctx_f, ctx_s = P.make_ctx(wl), P.make_ctx(wl)
    ctx_f.bacon_begin_prompt(batch)
    ctx_s.bacon_begin_prompt(batch)
    rtol = P.RTOL[wl.dtype]
    for layer in range(wl.num_layers):
        x = inputs.layer_inputs(wl, layer)
        r = orc.layer(layer, x["q_win"], x["k"], head_budgets=hb)
        q, k, v = P.to_dev(x["q_win"], wl), P.to_dev(x["k"], wl), P.to_dev(x["v"], wl)
        kb, vb = P.as_bytes(x["k"], wl), P.as_bytes(x["v"], wl)
        idx, ko, vo = ctx_f.bacon_compress_layer(layer, batch, q, k, v)
        B, Q, _ = ctx_s.bacon_score(layer, batch, q, k)
        cal = ctx_s.bacon_calibrate(layer, batch, B, Q, want_V=True)
        idx_s = ctx_s.bacon_select_topk(batch, cal["S"])
        ko_s, vo_s = ctx_s.bacon_compact(batch, k, v, idx_s)
        torch.cuda.synchronize()
        P.check_lambda(f"{name}/heads L{layer} lambda", cal["lambda"].cpu().numpy(), r, wl, rtol,
                       B_gpu=B.cpu().numpy(), V_gpu=cal["V"].cpu().numpy())
        for tag, gi, kk, vv in (("fused", idx, ko, vo), ("split", idx_s, ko_s, vo_s)):
            g = gi.cpu().numpy()
            P.check_idx(f"{name}/heads L{layer} {tag}", g, r, wl, rtol, hb=hb)
            assert np.array_equal(P.tensor_bytes(kk), P.gather_rows(kb, g, wl, hb=hb)), tag
            assert np.array_equal(P.tensor_bytes(vv), P.gather_rows(vb, g, wl, hb=hb)), tag


def _batch64():
    rng = np.random.default_rng(64)
    lens = tuple(int(x) for x in rng.integers(40, 401, size=64))
    budgets = tuple(int(x) for x in rng.choice([1, 8, 64, 300], size=64))
    visual = tuple((2, n - 12) for n in lens)
    return inputs.Workload("edge", 2, 4, 2, 64, 8, 5, "bf16", lens, budgets, visual, 1, 22)


EDGE = {
    # generic row layout (G*W = 24, pad rows), d = 64, budget > |I|, budget = |I|
    "gqa3-w8-d64": dict(wl=inputs.Workload("edge", 3, 6, 2, 64, 8, 5, "bf16", (40, 300, 77),
                                           (5, 500, 69), ((0, 30), (10, 250), (5, 60)), 1, 7)),
    # fp32 path with d = 128 and a window that is not a multiple of 32
    "fp32-d128-w20": dict(wl=inputs.Workload("edge", 3, 4, 2, 128, 20, 3, "fp32", (333, 97),
                                             (40, 7), ((10, 300), (5, 60)), 2, 8)),
    # the window is the whole prompt: empty candidate set
    "window-only": dict(wl=inputs.Workload("edge", 2, 4, 4, 64, 8, 5, "fp32", (8, 50),
                                           (4, 4), ((0, 0), (0, 30)), 0, 9)),
    # single window row, budget 1, MHA bf16
    "w1-budget1": dict(wl=inputs.Workload("edge", 2, 2, 2, 128, 1, 1, "bf16", (129,), (1,),
                                          ((0, 100),), 1, 10)),
    # parameter variants on one workload
    "radius0-m0": dict(wl=inputs.Workload("edge", 3, 4, 2, 64, 16, 5, "bf16", (600,), (32,),
                                          ((40, 500),), 2, 11),
                       gpu=dict(radius=0, persist_m=0), orc=dict(radius=0, persist_m=0)),
    "m1-pool1-r9": dict(wl=inputs.Workload("edge", 4, 4, 2, 64, 16, 1, "bf16", (600,), (32,),
                                           ((40, 500),), 2, 12),
                        gpu=dict(radius=9, persist_m=1), orc=dict(radius=9, persist_m=1)),
    # the calibration kernel sums the neighbourhoods of three consecutive
    # window positions and the pools of two consecutive candidates per
    # thread: radius 1 runs its shared-tap loop once, radius 2 with pool 5
    # twice, on lengths whose segments end in a partial thread
    "radius1-pool3": dict(wl=inputs.Workload("edge", 3, 4, 2, 64, 16, 3, "bf16", (2500, 701), (48, 20),
                                             ((40, 2000), (10, 600)), 2, 34),
                          gpu=dict(radius=1), orc=dict(radius=1)),
    "radius2-pool5-ragged": dict(wl=inputs.Workload("edge", 3, 4, 2, 64, 16, 5, "bf16", (4099, 1030),
                                                    (64, 24), ((100, 3900), (0, 900)), 2, 35),
                                 gpu=dict(radius=2), orc=dict(radius=2)),
    "window-score-only": dict(wl=inputs.Workload("edge", 2, 8, 2, 128, 32, 7, "bf16", (1000,),
                                                 (64,), ((30, 800),), 3, 13),
                              gpu=dict(use_last_query=0), orc=dict(use_last_query=0)),
    "gamma0": dict(wl=inputs.Workload("edge", 2, 8, 2, 128, 32, 7, "bf16", (1000,), (64,),
                                      ((30, 800),), 3, 14),
                   gpu=dict(gamma=0.0), orc=dict(gamma=0.0)),
    "terms-E-T": dict(wl=inputs.Workload("edge", 3, 8, 2, 128, 32, 7, "bf16", (1000,), (64,),
                                         ((30, 800),), 3, 15),
                      gpu=dict(terms=5), orc=dict(terms=5)),
    "gamma-rho": dict(wl=inputs.Workload("edge", 3, 8, 2, 128, 32, 7, "bf16", (1000, 700),
                                         (64, 300), ((30, 800), (30, 600)), 3, 16),
                      gpu=dict(gamma=0.5, rho=3.0), orc=dict(gamma=0.5, rho=3.0)),
    # fractional rho: M = floor(rho K) formed in double on both sides
    # (1.3 * 90 gives 117, 0.7 * 90 gives 62 in binary double)
    "rho-1.3-budget-90": dict(wl=inputs.Workload("edge", 3, 8, 2, 128, 32, 7, "bf16", (1500, 900),
                                                 (90, 90), ((30, 1200), (30, 800)), 3, 26),
                              gpu=dict(rho=1.3), orc=dict(rho=1.3)),
    "rho-0.7-budget-90": dict(wl=inputs.Workload("edge", 3, 8, 2, 128, 32, 7, "bf16", (1500,),
                                                 (90,), ((30, 1200),), 3, 27),
                              gpu=dict(rho=0.7), orc=dict(rho=0.7)),
    # widest pool (33) and coherence radius (16) over several select segments,
    # sequence ends inside a segment and inside the pool halo
    "pool33-r16-segments": dict(wl=inputs.Workload("edge", 3, 8, 2, 128, 32, 33, "bf16",
                                                   (5000, 2070, 4111), (100, 40, 700),
                                                   ((30, 4000), (0, 2000), (100, 4000)), 4, 17),
                                gpu=dict(radius=16), orc=dict(radius=16)),
    # scale-matching set larger than a segment (every segment position is a
    # candidate) and a budget above half the candidate set
    "M-over-segment": dict(wl=inputs.Workload("edge", 3, 8, 2, 128, 32, 7, "bf16", (8000,),
                                              (1500,), ((30, 7000),), 4, 18)),
    # pooling variants: max of S, and mean of B before calibration, over
    # several segments with a pool halo that crosses them
    "pool-max-s": dict(wl=inputs.Workload("edge", 3, 8, 2, 128, 32, 9, "bf16", (5000, 2070),
                                          (100, 40), ((30, 4000), (0, 2000)), 4, 23),
                       gpu=dict(pool_mode=1), orc=dict(pool_mode=1)),
    "pool-mean-b": dict(wl=inputs.Workload("edge", 3, 8, 2, 128, 32, 9, "bf16", (5000, 2070),
                                           (100, 40), ((30, 4000), (0, 2000)), 4, 24),
                        gpu=dict(pool_mode=2), orc=dict(pool_mode=2)),
    "pool-max-s-fp32": dict(wl=inputs.Workload("edge", 2, 4, 2, 64, 20, 33, "fp32", (3000, 333),
                                               (64, 40), ((10, 2500), (5, 300)), 2, 25),
                            gpu=dict(pool_mode=1), orc=dict(pool_mode=1)),
    # the largest window-row block: G*W = 256 rows (eight row tiles)
    "rows256-g8-w32": dict(wl=inputs.Workload("edge", 3, 16, 2, 128, 32, 7, "bf16", (3000, 1500),
                                              (100, 40), ((30, 2500), (0, 1200)), 4, 20)),
    # a 256-query window with one head per group
    "w256-mha": dict(wl=inputs.Workload("edge", 2, 2, 2, 64, 256, 5, "bf16", (1200,), (50,),
                                        ((10, 800),), 3, 21)),
    # d = 64 with a 32-query window: two and four row tiles (G = 2 and 4)
    "d64-w32-g2": dict(wl=inputs.Workload("edge", 3, 4, 2, 64, 32, 7, "bf16", (1500, 700), (64, 32),
                                          ((20, 1200), (5, 500)), 2, 31)),
    "d64-w32-g4": dict(wl=inputs.Workload("edge", 3, 8, 2, 64, 32, 7, "bf16", (2100, 333), (90, 17),
                                          ((40, 1800), (0, 200)), 2, 32)),
    # G = 3 with a 32-query window: 96 window rows in four row tiles, the last
    # tile all pad rows (their weights are 0, also on the last-query row)
    "g3-w32-pad-rows": dict(wl=inputs.Workload("edge", 3, 6, 2, 128, 32, 7, "bf16", (1800, 650),
                                               (70, 24), ((30, 1500), (8, 400)), 2, 33)),
    # the largest batch: 64 sequences of ragged lengths and budgets
    "batch64": dict(wl=_batch64()),
    # large budgets: scale-matching set and kept set of thousands of positions
    "large-budget-whole-sequence": dict(wl=inputs.Workload("edge", 2, 8, 2, 128, 32, 7, "bf16",
                                                           (20000, 3000), (3000, 200),
                                                           ((30, 19000), (10, 2500)), 4, 19)),
}


@pytest.mark.parametrize("name", list(EDGE))
def test_edge_cases(name):
    c = EDGE[name]
    run_case(name, c["wl"], c.get("gpu"), c.get("orc"))


def test_fused_pass_is_deterministic():
    import torch
    from paper_2606_14782_amd import bacon
    wl = _small(4, num_layers=3, max_len=4000, num_kv_heads=2)
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    outs = []
    for rep in range(2):
        ctx = P.make_ctx(wl)
        ctx.bacon_begin_prompt(batch)
        got = []
        for layer in range(wl.num_layers):
            x = inputs.layer_inputs(wl, layer)
            idx, ko, vo = ctx.bacon_compress_layer(layer, batch, P.to_dev(x["q_win"], wl),
                                                   P.to_dev(x["k"], wl), P.to_dev(x["v"], wl))
            torch.cuda.synchronize()
            got.append((idx.cpu().numpy(), P.tensor_bytes(ko), P.tensor_bytes(vo)))
        outs.append(got)
    for a, b in zip(*outs):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


def test_outputs_stay_inside_their_buffers():
    """Guard regions around every output are left untouched."""
    import torch
    from paper_2606_14782_amd import bacon
    wl = _small(4, num_layers=2, max_len=2000, num_kv_heads=2)
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    ctx = P.make_ctx(wl)
    ctx.bacon_begin_prompt(batch)
    n_idx = batch.idx_count(wl.num_kv_heads)
    rows = batch.kept_rows(wl.window)
    G = 4096
    idx_buf = torch.full((n_idx + 2 * G,), 0x5A5A5A5A, dtype=torch.int32, device="cuda")
    row_elems = wl.num_kv_heads * wl.head_dim
    k_buf = torch.full((rows * row_elems + 2 * G,), 3.0, dtype=torch.bfloat16, device="cuda")
    v_buf = torch.full((rows * row_elems + 2 * G,), 5.0, dtype=torch.bfloat16, device="cuda")
    for layer in range(wl.num_layers):
        x = inputs.layer_inputs(wl, layer)
        out = (idx_buf[G:G + n_idx], k_buf[G:G + rows * row_elems].view(rows, wl.num_kv_heads, -1),
               v_buf[G:G + rows * row_elems].view(rows, wl.num_kv_heads, -1))
        ctx.bacon_compress_layer(layer, batch, P.to_dev(x["q_win"], wl), P.to_dev(x["k"], wl),
                                 P.to_dev(x["v"], wl), out=out)
    torch.cuda.synchronize()
    for buf, fill in ((idx_buf, 0x5A5A5A5A), (k_buf, 3.0), (v_buf, 5.0)):
        assert bool((buf[:G] == fill).all()) and bool((buf[-G:] == fill).all())


def test_ragged_batch_equals_single_sequences(monkeypatch):
    """Sequences of a packed batch are independent: a batch gives the same kept
    positions as each sequence run alone (same chunking forced for both)."""
    import torch
    from paper_2606_14782_amd import bacon
    monkeypatch.setenv("BACON_CHUNK_STAGES", "2")
    wl = _small(4, num_layers=3, max_len=2500, num_kv_heads=2)
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    ctx = P.make_ctx(wl)
    ctx.bacon_begin_prompt(batch)
    xs = [inputs.layer_inputs(wl, l) for l in range(wl.num_layers)]
    full = []
    for layer, x in enumerate(xs):
        idx, _, _ = ctx.bacon_compress_layer(layer, batch, P.to_dev(x["q_win"], wl),
                                             P.to_dev(x["k"], wl), P.to_dev(x["v"], wl))
        full.append(idx.cpu().numpy())
    cu = wl.cu_seqlens
    base = 0
    for b in range(wl.batch):
        one = wl.with_(seq_lens=(wl.seq_lens[b],), budgets=(wl.budgets[b],),
                       visual=(wl.visual[b],))
        bt = bacon.BatchLayout(one.cu_seqlens, one.budgets_arr)
        c1 = P.make_ctx(one)
        c1.bacon_begin_prompt(bt)
        K = wl.budgets[b]
        for layer, x in enumerate(xs):
            q = x["q_win"][b * wl.window:(b + 1) * wl.window]
            k = x["k"][cu[b]:cu[b + 1]]
            v = x["v"][cu[b]:cu[b + 1]]
            idx, _, _ = c1.bacon_compress_layer(layer, bt, P.to_dev(q, wl), P.to_dev(k, wl),
                                                P.to_dev(v, wl))
            got = idx.cpu().numpy()
            want = full[layer][base * wl.num_kv_heads:(base + K) * wl.num_kv_heads]
            assert np.array_equal(got, want), f"sequence {b} layer {layer}"
        base += K
    torch.cuda.synchronize()


def _tied_inputs(wl, distinct):
    """Keys drawn from `distinct` fixed vectors: the window scores of the
    candidates take only a few values, so every selection meets exact ties."""
    def make(layer):
        rng = np.random.default_rng(1000 + layer)
        T, Hkv, d = wl.total_tokens, wl.num_kv_heads, wl.head_dim
        q = inputs.round_bf16(rng.standard_normal((wl.batch * wl.window, wl.num_q_heads, d),
                                                  dtype=np.float32))
        base = inputs.round_bf16(rng.standard_normal((distinct, Hkv, d), dtype=np.float32))
        which = rng.integers(0, distinct, T) if distinct > 1 else np.zeros(T, np.int64)
        k = np.ascontiguousarray(base[which])
        v = inputs.round_bf16(rng.standard_normal((T, Hkv, d), dtype=np.float32))
        return {"q_win": q, "k": k, "v": v}
    return make


@pytest.mark.parametrize("n,K,distinct", [(600, 40, 1), (3000, 100, 1), (3000, 100, 3),
                                          (20000, 256, 2)])
def test_near_ties_with_pooling(n, K, distinct):
    """Identical or few distinct keys with the default calibration and a
    pool of 5: mathematically tied pooled scores that the truncated pool
    windows and the coherence sums round differently on the two sides (fp32
    against fp64), so the kept sets may swap such positions (within rtol of
    the K-th score, list and fallback select paths)."""
    wl = inputs.Workload("ties", 3, 4, 2, 64, 8, 5, "bf16", (n,), (K,), ((0, 0),), 0, 21)
    run_case(f"ties-n{n}-d{distinct}", wl, make=_tied_inputs(wl, distinct))


@pytest.mark.parametrize("n,K,distinct", [(600, 40, 1), (3000, 100, 3), (20000, 256, 2)])
def test_near_ties_single_pass(n, K, distinct, monkeypatch):
    """The near-tie cases on the single-read pass (forced): equal keys differ
    there in the last bits of B as well."""
    monkeypatch.setenv("BACON_SINGLE", "1")
    wl = inputs.Workload("ties", 3, 4, 2, 64, 8, 5, "bf16", (n,), (K,), ((0, 0),), 0, 21)
    run_case(f"ties-single-n{n}-d{distinct}", wl, make=_tied_inputs(wl, distinct), split=False)


def _constant_evidence_inputs(wl):
    """Layer 0: keys of one vector on [0, n/2) and another on the rest, the
    last window query aligned with the first and the other rows with the
    second, so E_0 is one positive constant over [0, n/2).  Layer 1: keys
    near a third vector (small noise) on [0, n/2), which the window queries
    favour, so the scale-matching set lies in [0, n/2) where B varies and
    V = T = E_0 is constant."""
    def make(layer):
        rng = np.random.default_rng(4000 + layer)
        n, W, d = wl.total_tokens, wl.window, wl.head_dim
        half = n // 2
        base = rng.standard_normal((3, d)).astype(np.float32)
        base /= np.linalg.norm(base, axis=1, keepdims=True)
        k = np.empty((n, 1, d), np.float32)
        q = np.empty((W, 1, d), np.float32)
        if layer == 0:
            k[:half, 0] = base[0]
            k[half:, 0] = base[1]
            q[:, 0] = 3.0 * base[1]
            q[W - 1, 0] = 3.0 * base[0]
        else:
            k[:half, 0] = base[2] + 0.05 * rng.standard_normal((half, d))
            k[half:, 0] = base[1]
            q[:, 0] = 3.0 * base[2] + 0.1 * rng.standard_normal((W, d))
        v = rng.standard_normal((n, 1, d)).astype(np.float32)
        return {"q_win": inputs.round_bf16(q), "k": inputs.round_bf16(k), "v": inputs.round_bf16(v)}
    return make


def test_constant_evidence_on_the_scale_matching_set():
    """V constant (and positive) over the scale-matching set while B varies,
    so lambda = gamma Std_M(B) / eps (Eq. lambda_solution).  The two-pass
    score (the split call, and the fused call on this small grid) gives
    identical keys bit-equal probabilities, so Std_M(V) is exactly 0 (moments
    of shifted values) and lambda agrees with the oracle's within rtol.  The
    single-read pass (forced for a second fused run) stores each probability
    relative to its tile's running maximum, so identical keys in tiles with
    different maxima round differently and its Std_M(V) is a rounding
    residue: its lambda is held to the interval its B and V allow, and its
    kept set to the oracle's."""
    from paper_2606_14782_amd import bacon
    kw = dict(terms=4, persist_m=1)
    wl = inputs.Workload("const-v", 2, 1, 1, 64, 8, 1, "bf16", (1000,), (32,), ((0, 0),), 0, 28)
    run_case("const-v", wl, gpu_kw=kw, orc_kw=kw, make=_constant_evidence_inputs(wl))
    with pytest.MonkeyPatch.context() as mp:
        mp.setenv("BACON_SINGLE", "1")
        run_case("const-v/single", wl, gpu_kw=kw, orc_kw=kw, make=_constant_evidence_inputs(wl),
                 split=False)
    orc = ref.Prompt.for_workload(wl, P.oracle_params(**kw))
    ctx = P.make_ctx(wl, P.params_for(wl, **kw))
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    ctx.bacon_begin_prompt(batch)
    mk = _constant_evidence_inputs(wl)
    for l in range(2):
        x = mk(l)
        r = orc.layer(l, x["q_win"], x["k"])
        q, k = P.to_dev(x["q_win"], wl), P.to_dev(x["k"], wl)
        B, Q, _ = ctx.bacon_score(l, batch, q, k)
        cal = ctx.bacon_calibrate(l, batch, B, Q)
        lam = float(cal["lambda"].cpu()[0, 0])
        want = float(r["lambda"][0, 0])
        assert abs(lam - want) <= P.RTOL[wl.dtype] * abs(want), (l, lam, want)
    assert r["sigma_V"][0, 0] == 0.0 and r["sigma_B"][0, 0] > 0.0
    assert r["lambda"][0, 0] > 1e3, "the case must reach the eps-dominated lambda"


TIE_PARAMS = {
    # S = B: the window score alone
    "window-score": dict(use_last_query=0),
    # S = B + lambda E: equal keys give bit-equal B, Q and E on both sides
    "residual-only": dict(radius=0, persist_m=0),
}


# (params, n, K, distinct).  With the evidence term, the scale-matching set
# (rho K positions) stays inside the top class of B: over two classes the
# variance-matched lambda is (B_1 - B_2) / (V_2 - V_1), which makes the two
# classes' scores equal in exact arithmetic (S_2 = B_2 + lambda V_2 = B_1 +
# lambda V_1), a tie that fp32 and fp64 rounding break differently.
TIE_CASES = [(p, n, K, d) for p in TIE_PARAMS for (n, K, d) in
             [(600, 40, 1), (3000, 100, 1), (3000, 100, 2), (20000, 256, 2), (20000, 3000, 1)]]
TIE_CASES += [("window-score", 3000, 700, 3), ("residual-only", 3000, 300, 3)]


@pytest.mark.parametrize("params,n,K,distinct", TIE_CASES)
def test_exact_ties_resolve_by_lowest_position(n, K, distinct, params, monkeypatch):
    """Exact ties by construction: keys drawn from a few fixed vectors, no
    pooling, and no term that mixes neighbouring positions, so on the
    two-K-pass path every key of a class has the same score bit for bit on
    the GPU and in the oracle.  Its kept set (split and fused calls) must
    then be exactly the oracle's: score descending, and among equal scores
    the lowest positions (Eqs. scale_matching_set and topk_selection with the
    tie rule), for the top-K and, through lambda, the scale-matching set.
    Covers the list path, boundary bins of thousands of tied entries, and
    the whole-sequence fallback.  The single-read pass stores each
    probability relative to its tile's running maximum, so equal keys in
    tiles with different maxima differ in the last bits of B: its kept set
    may resolve the tie differently, but only among positions whose oracle
    score is within rtol of the K-th."""
    kw = TIE_PARAMS[params]
    wl = inputs.Workload("ties", 3, 4, 2, 64, 8, 1, "bf16", (n,), (K,), ((0, 0),), 0, 21)
    monkeypatch.setenv("BACON_SINGLE", "0")
    worst, stats = run_case(f"exact-ties-{params}-n{n}-d{distinct}", wl, gpu_kw=kw, orc_kw=kw,
                            make=_tied_inputs(wl, distinct), strict=True)
    assert stats["strict"] == stats["pairs"]
    monkeypatch.setenv("BACON_SINGLE", "1")
    run_case(f"exact-ties-{params}-n{n}-d{distinct}/single", wl, gpu_kw=kw, orc_kw=kw,
             make=_tied_inputs(wl, distinct), split=False)


LONG_CASES = {
    # one GPU's share of the paper's extreme contexts (budget 1024): the
    # single-read pass (every chunk of the sequence fits on the GPU at once)
    "long-n65536": lambda: inputs.Workload(
        "long", 3, 16, 4, 128, 32, 7, "bf16", (65536,), (1024,), ((32, 65000),), 8, 41,
        frame_rank=8, frame_len=256),
    "long-n131072": lambda: inputs.Workload(
        "long", 3, 8, 2, 128, 32, 7, "bf16", (131072,), (1024,), ((32, 130000),), 8, 42,
        frame_rank=8, frame_len=256),
    # more chunks than the GPU holds at once: the two-K-pass path
    "long-n65536-h8": lambda: inputs.Workload(
        "long", 3, 32, 8, 128, 32, 7, "bf16", (65536,), (512,), ((32, 65000),), 8, 43),
    # a long sequence among short ones
    "long-ragged": lambda: inputs.Workload(
        "long", 3, 8, 2, 128, 32, 7, "bf16", (3000, 98304, 20000), (256, 1024, 128),
        ((32, 2800), (32, 98000), (32, 19000)), 8, 44),
}


@pytest.mark.parametrize("name", list(LONG_CASES))
def test_long_sequences(name):
    """Sequences beyond 32768 tokens (up to 131072) through the fused call:
    64 select segments per sequence, scores and kept sets against the oracle.
    (The split calls' block select holds at most 32768 positions.)"""
    run_case(name, LONG_CASES[name](), split=False)


@pytest.mark.parametrize("name", ["long-n131072", "long-ragged"])
def test_long_prompt_call_equals_layer_calls(name):
    import torch
    from paper_2606_14782_amd import bacon
    wl = LONG_CASES[name]()
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    xs = [inputs.layer_inputs(wl, l) for l in range(wl.num_layers)]
    qs = [P.to_dev(x["q_win"], wl) for x in xs]
    ks = [P.to_dev(x["k"], wl) for x in xs]
    vs = [P.to_dev(x["v"], wl) for x in xs]
    a, b = P.make_ctx(wl), P.make_ctx(wl)
    a.bacon_begin_prompt(batch)
    want = [a.bacon_compress_layer(l, batch, qs[l], ks[l], vs[l]) for l in range(wl.num_layers)]
    b.bacon_begin_prompt(batch)
    got = b.bacon_compress_prompt(0, batch, qs, ks, vs)
    torch.cuda.synchronize()
    for l in range(wl.num_layers):
        for i, what in enumerate(("idx", "k_out", "v_out")):
            assert torch.equal(got[l][i], want[l][i]), f"{name} L{l} {what}"


@pytest.mark.parametrize("n,K,params", [(65536, 300, "residual-only"),
                                        (131072, 1024, "window-score")])
def test_long_exact_ties_take_the_streamed_select(n, K, params, monkeypatch):
    """Identical keys over a sequence beyond 32768 tokens: every candidate
    falls in one histogram bin, so the scale-matching set (with the evidence
    term) and the top-K take the select that streams the sequence from memory
    (no register copy fits); on the two-K-pass path the equal scores are
    bit-equal and the kept set must be the lowest positions exactly."""
    monkeypatch.setenv("BACON_SINGLE", "0")
    kw = TIE_PARAMS[params]
    wl = inputs.Workload("ties", 2, 4, 2, 64, 8, 1, "bf16", (n,), (K,), ((0, 0),), 0, 23)
    worst, stats = run_case(f"long-ties-n{n}", wl, gpu_kw=kw, orc_kw=kw, make=_tied_inputs(wl, 1),
                            strict=True, split=False)
    assert stats["strict"] == stats["pairs"]


SINGLE_FORCED = ["llava-n2048", "ragged-b8", "llava-small", "ragged-small", "video-small",
                 "batch64", "gqa3-w8-d64", "w1-budget1", "pool33-r16-segments", "M-over-segment",
                 "pool-max-s", "pool-mean-b", "large-budget-whole-sequence", "window-score-only",
                 "gamma0", "radius0-m0", "d64-w32-g2", "d64-w32-g4", "g3-w32-pad-rows"]


@pytest.mark.parametrize("name", SINGLE_FORCED)
def test_single_pass_forced(name, monkeypatch):
    """The single-read pass forced (BACON_SINGLE=1) where the library would
    take the two-K-pass path: small grids, and batches whose grid runs in
    rounds (every sequence's chunks still fit on the GPU at once)."""
    monkeypatch.setenv("BACON_SINGLE", "1")
    if name in CASES:
        wl = CASES[name]()
        run_case(name + "/single", wl.with_(num_layers=min(wl.num_layers, 5)), split=False)
    else:
        c = EDGE[name]
        run_case(name + "/single", c["wl"], c.get("gpu"), c.get("orc"), split=False)


@pytest.mark.parametrize("name", ["ragged-b8", "llava-n2048"])
def test_single_pass_forced_prompt_call(name, monkeypatch):
    import torch
    from paper_2606_14782_amd import bacon
    monkeypatch.setenv("BACON_SINGLE", "1")
    wl = CASES[name]().with_(num_layers=3)
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    xs = [inputs.layer_inputs(wl, l) for l in range(wl.num_layers)]
    qs = [P.to_dev(x["q_win"], wl) for x in xs]
    ks = [P.to_dev(x["k"], wl) for x in xs]
    vs = [P.to_dev(x["v"], wl) for x in xs]
    a, b = P.make_ctx(wl), P.make_ctx(wl)
    a.bacon_begin_prompt(batch)
    want = [a.bacon_compress_layer(l, batch, qs[l], ks[l], vs[l]) for l in range(wl.num_layers)]
    b.bacon_begin_prompt(batch)
    got = b.bacon_compress_prompt(0, batch, qs, ks, vs)
    torch.cuda.synchronize()
    for l in range(wl.num_layers):
        for i, what in enumerate(("idx", "k_out", "v_out")):
            assert torch.equal(got[l][i], want[l][i]), f"{name} L{l} {what}"
    assert a.bacon_debug_device_errors() == 0 and b.bacon_debug_device_errors() == 0
