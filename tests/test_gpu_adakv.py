"""GPU parity of the AdaKV head-wise allocation (App. B: BACON on the AdaKV
backbone keeps its budgets and changes only the score within each head).

The allocation decides integers (K_{b,h}) from floating-point comparisons of
the pooled window score A: where the oracle's union boundary (the slot of the
layer's last union entry) is separated from the next entry by more than the
score tolerance, the GPU's budgets must be the oracle's exactly; otherwise
each head's budget must lie between the counts that entries clearly above and
clearly below the boundary fix, and the budgets must still fill the
sequence's H K slots.  The kept sets are then checked against the oracle run
with the GPU's own budgets, and the compacted cache (one head per row) must
be a bit copy of the rows the GPU's indices name.
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
    "video-n32768": lambda: inputs.workload(3).with_(num_layers=3),
    "qwen2vl-n8192": lambda: inputs.workload(2).with_(num_layers=3),
    "llava-n2048": lambda: inputs.workload(1).with_(num_layers=3),   # 32 KV heads
    "ragged-small": lambda: _small(4, num_layers=4, max_len=3000, num_kv_heads=4),
    # budget 2 with alpha 0.2: no floor, so a head may get no slot at all
    "tiny-budget": lambda: _small(4, num_layers=3, max_len=900, num_kv_heads=4).with_(
        budgets=(2,) * 8),
}


def pooled_scores(r, wl, b, pool_kernel):
    s0, s1 = P.seq_slices(wl)[b]
    nc = (s1 - s0) - wl.window
    return np.stack([ref.pool(r["B"][h, s0:s0 + nc], pool_kernel) for h in range(wl.num_kv_heads)])


def check_alloc(name, got, A_of, wl, alpha, rtol, gap_tol=None):
    """got [batch, Hkv] against the oracle's allocation of A_of(b) [Hkv, n_c]:
    exact where the union boundary's relative gap exceeds gap_tol (GAP_TOL by
    default), else within the counts the entries clearly (rtol) above and
    below the boundary fix."""
    gap_tol = P.GAP_TOL if gap_tol is None else gap_tol
    got = np.asarray(got, np.int64).reshape(wl.batch, wl.num_kv_heads)
    exact = 0
    for b in range(wl.batch):
        K = int(wl.budgets[b])
        A = A_of(b)
        H, nc = A.shape
        want = ref.adaptive_budgets(A, K, alpha)
        if K >= nc:
            assert got[b].tolist() == [K] * H, (name, b, got[b])
            continue
        f = int(np.floor(alpha * K))
        R = H * (K - f)
        if R == 0:                     # the floor takes every slot: uniform budgets
            assert got[b].tolist() == [f] * H, (name, b, got[b])
            exact += 1
            continue
        rest = np.sort(np.concatenate([np.sort(A[h])[::-1][f:] for h in range(H)]))[::-1]
        vR, vN = rest[R - 1], rest[R] if R < len(rest) else -np.inf
        assert got[b].sum() == H * K, (name, b, got[b].sum(), H * K)
        if vR - vN > gap_tol * abs(vR):
            assert got[b].tolist() == want.tolist(), (name, b, got[b], want)
            exact += 1
            continue
        band = rtol * abs(vR)
        for h in range(H):
            lo = max(f, int(np.count_nonzero(A[h] > vR + band)))
            hi = max(f, int(np.count_nonzero(A[h] >= vR - band)))
            assert lo <= got[b, h] <= hi, (name, b, h, got[b, h], lo, hi, want[h])
    return exact


def gather_rows_flat(x_bytes, idx, wl, kh):
    """Expected compacted cache with one head per row: sequence b's H (K_b + W)
    rows, head h's block its K_{b,h} kept rows (zero rows for -1 entries), then
    its W window rows."""
    W, Hkv = wl.window, wl.num_kv_heads
    row_b = x_bytes.shape[-1]
    out = np.zeros((int(np.sum(np.asarray(wl.budgets) + W)) * Hkv, row_b), np.uint8)
    off, r0 = 0, 0
    for b, (s0, s1) in enumerate(P.seq_slices(wl)):
        n = s1 - s0
        for h in range(Hkv):
            K = int(kh[b, h])
            g = np.asarray(idx[off:off + K])
            off += K
            for j, p in enumerate(g):
                if p >= 0:
                    out[r0 + j] = x_bytes[s0 + p, h]
            out[r0 + K:r0 + K + W] = x_bytes[s0 + n - W:s0 + n, h]
            r0 += K + W
    return out


def run_adaptive(name, wl, alpha):
    import torch
    from paper_2606_14782_amd import bacon
    rtol = P.RTOL[wl.dtype]
    P.log(f"[{name}] adaptive alpha={alpha} B={wl.batch} Hkv={wl.num_kv_heads} "
          f"lens={wl.seq_lens[:8]} budgets={wl.budgets[:8]}")
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    ctx = P.make_ctx(wl, P.params_for(wl, head_alloc=bacon.ALLOC_ADAPTIVE, alloc_floor=alpha))
    kh_all = torch.full((wl.num_layers, wl.batch, wl.num_kv_heads), -7, dtype=torch.int32,
                        device="cuda")
    ctx.bacon_alloc_output(kh_all)
    # the fused call's own B, to check the allocation on the scores it saw
    T, Hkv = wl.total_tokens, wl.num_kv_heads
    cap = (torch.zeros((wl.num_layers, Hkv, T), dtype=torch.float32, device="cuda"),
           torch.zeros((wl.num_layers, Hkv, T), dtype=torch.float32, device="cuda"),
           torch.zeros((wl.num_layers, wl.batch, Hkv), dtype=torch.float32, device="cuda"))
    ctx.bacon_debug_capture(*cap)
    ctx.bacon_begin_prompt(batch)
    orc = ref.Prompt.for_workload(wl)
    stats, exact, self_exact = {}, 0, 0
    outs = []
    for layer in range(wl.num_layers):
        x = inputs.layer_inputs(wl, layer)
        q, k, v = P.to_dev(x["q_win"], wl), P.to_dev(x["k"], wl), P.to_dev(x["v"], wl)
        kb, vb = P.as_bytes(x["k"], wl), P.as_bytes(x["v"], wl)
        P.log(f"[{name}] layer {layer}")
        idx, ko, vo = ctx.bacon_compress_layer(layer, batch, q, k, v)
        torch.cuda.synchronize()
        kh = kh_all[layer].cpu().numpy()
        r = orc.layer_adaptive(layer, x["q_win"], x["k"], alpha)
        exact += check_alloc(f"{name} L{layer}", kh, lambda b: pooled_scores(r, wl, b, wl.pool_kernel),
                             wl, alpha, rtol)
        # on the GPU's own B the allocation is the rule's up to the fp32 pool
        Bg = {"B": cap[0][layer].cpu().numpy().astype(np.float64)}
        self_exact += check_alloc(f"{name} L{layer} own B", kh,
                                  lambda b: pooled_scores(Bg, wl, b, wl.pool_kernel), wl, alpha,
                                  1e-5, gap_tol=1e-5)
        # the selection under the GPU's own budgets
        r2 = orc.layer(layer, x["q_win"], x["k"], head_budgets=kh)
        gi = idx.cpu().numpy()
        P.check_idx(f"{name} L{layer} adaptive", gi, r2, wl, rtol, hb=kh, stats=stats)
        kflat = P.tensor_bytes(ko).reshape(-1, kb.shape[-1])
        vflat = P.tensor_bytes(vo).reshape(-1, vb.shape[-1])
        assert np.array_equal(kflat, gather_rows_flat(kb, gi, wl, kh)), "K gather"
        assert np.array_equal(vflat, gather_rows_flat(vb, gi, wl, kh)), "V gather"
        outs.append((idx, ko, vo))
    ctx.bacon_alloc_output(None)
    ctx.bacon_debug_capture()
    assert ctx.bacon_debug_device_errors() == 0
    P.log(f"[{name}] ok; budgets exact on {exact} sequence-layers ({self_exact} on the GPU's own "
          f"B); kept sets exact "
          f"{stats.get('strict', 0)}/{stats.get('pairs', 0)}, swaps {stats.get('swaps', 0)}")
    return kh_all, outs


@pytest.mark.parametrize("name", list(CASES))
def test_adaptive_allocation(name):
    run_adaptive(name, CASES[name](), 0.2)


@pytest.mark.parametrize("alpha", [0.0, 0.5, 1.0])
def test_adaptive_floor_values(alpha):
    """No floor (a head may get nothing), half, and the full floor (uniform
    budgets: the compacted rows are the uniform layout's, head by head)."""
    kh, _ = run_adaptive(f"ragged-a{alpha}", CASES["ragged-small"]().with_(num_layers=2), alpha)
    if alpha == 1.0:
        wl = CASES["ragged-small"]()
        assert (kh.cpu().numpy() == np.asarray(wl.budgets)[None, :, None]).all()


def test_allocate_heads_entry_point():
    """bacon_allocate_heads on the oracle's own B (as float32): the pooled
    scores differ from the oracle's only by fp32 rounding."""
    import torch
    from paper_2606_14782_amd import bacon
    wl = CASES["ragged-small"]()
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    orc = ref.Prompt.for_workload(wl)
    x = inputs.layer_inputs(wl, 0)
    r = orc.layer(0, x["q_win"], x["k"])
    B32 = np.ascontiguousarray(r["B"], np.float32)
    ctx = P.make_ctx(wl)
    for alpha in (0.0, 0.2, 0.7):
        ctx = P.make_ctx(wl, P.params_for(wl, alloc_floor=alpha))
        kh = ctx.bacon_allocate_heads(batch, torch.from_numpy(B32).cuda())
        torch.cuda.synchronize()

        def A_of(b):
            s0, s1 = P.seq_slices(wl)[b]
            nc = (s1 - s0) - wl.window
            return np.stack([ref.pool(B32[h, s0:s0 + nc].astype(np.float64), wl.pool_kernel)
                             for h in range(wl.num_kv_heads)])
        check_alloc(f"entry a{alpha}", kh.cpu().numpy(), A_of, wl, alpha, 1e-5)


@pytest.mark.parametrize("name", ["ragged-small", "video-n32768"])
def test_adaptive_prompt_call_equals_layer_calls(name):
    import torch
    from paper_2606_14782_amd import bacon
    wl = CASES[name]()
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    xs = [inputs.layer_inputs(wl, l) for l in range(wl.num_layers)]
    qs = [P.to_dev(x["q_win"], wl) for x in xs]
    ks = [P.to_dev(x["k"], wl) for x in xs]
    vs = [P.to_dev(x["v"], wl) for x in xs]
    prm = P.params_for(wl, head_alloc=bacon.ALLOC_ADAPTIVE, alloc_floor=0.2)
    a, b = P.make_ctx(wl, prm), P.make_ctx(wl, prm)
    ka = torch.zeros((wl.num_layers, wl.batch, wl.num_kv_heads), dtype=torch.int32, device="cuda")
    kb = torch.zeros_like(ka)
    a.bacon_alloc_output(ka)
    b.bacon_alloc_output(kb)
    a.bacon_begin_prompt(batch)
    want = [a.bacon_compress_layer(l, batch, qs[l], ks[l], vs[l]) for l in range(wl.num_layers)]
    b.bacon_begin_prompt(batch)
    got = b.bacon_compress_prompt(0, batch, qs, ks, vs)
    torch.cuda.synchronize()
    assert torch.equal(ka, kb)
    for l in range(wl.num_layers):
        for i, what in enumerate(("idx", "k_out", "v_out")):
            assert torch.equal(got[l][i], want[l][i]), f"{name} L{l} {what}"


def test_adaptive_with_a_per_layer_budget_schedule():
    """The adaptive allocation on a per-layer budget schedule (the backbone's
    layer-wise budgets, each layer's H K_l slots allocated across its heads):
    the prompt call with one batch per layer equals the per-layer calls bit
    for bit, and each layer's budgets fill its own slots."""
    import torch
    from paper_2606_14782_amd import bacon
    wl = CASES["ragged-small"]()
    rng = np.random.default_rng(31)
    sched = [tuple(int(x) for x in rng.choice([16, 64, 200], size=wl.batch))
             for _ in range(wl.num_layers)]
    batches = [bacon.BatchLayout(wl.cu_seqlens, np.asarray(s, np.int32)) for s in sched]
    xs = [inputs.layer_inputs(wl, l) for l in range(wl.num_layers)]
    qs = [P.to_dev(x["q_win"], wl) for x in xs]
    ks = [P.to_dev(x["k"], wl) for x in xs]
    vs = [P.to_dev(x["v"], wl) for x in xs]
    prm = P.params_for(wl, head_alloc=bacon.ALLOC_ADAPTIVE, alloc_floor=0.2)
    a, b = P.make_ctx(wl, prm), P.make_ctx(wl, prm)
    ka = torch.zeros((wl.num_layers, wl.batch, wl.num_kv_heads), dtype=torch.int32, device="cuda")
    kb = torch.zeros_like(ka)
    a.bacon_alloc_output(ka)
    b.bacon_alloc_output(kb)
    a.bacon_begin_prompt(batches[0])
    want = [a.bacon_compress_layer(l, batches[l], qs[l], ks[l], vs[l]) for l in range(wl.num_layers)]
    b.bacon_begin_prompt(batches[0])
    got = b.bacon_compress_prompt(0, batches[0], qs, ks, vs, layer_batches=batches)
    torch.cuda.synchronize()
    assert torch.equal(ka, kb)
    for l in range(wl.num_layers):
        for i, what in enumerate(("idx", "k_out", "v_out")):
            assert torch.equal(got[l][i], want[l][i]), f"L{l} {what}"
        kh = ka[l].cpu().numpy()
        for bb, (s0, s1) in enumerate(P.seq_slices(wl)):
            K = sched[l][bb]
            if (s1 - s0) - wl.window > K:
                assert kh[bb].sum() == wl.num_kv_heads * K, (l, bb)
    assert a.bacon_debug_device_errors() == 0 and b.bacon_debug_device_errors() == 0


def test_adaptive_on_a_long_sequence(monkeypatch):
    """131072 tokens, budget 1024, two KV heads (the single-read pass): the
    allocation and the kept sets against the oracle."""
    wl = inputs.Workload("long", 2, 8, 2, 128, 32, 7, "bf16", (131072,), (1024,), ((32, 130000),),
                         8, 45, frame_rank=8, frame_len=256)
    run_adaptive("long-adaptive", wl, 0.2)
