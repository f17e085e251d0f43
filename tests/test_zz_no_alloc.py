"""The allocation-free entry point bacon_window_lse_static (static device
scratch, no context, no workspace) against bacon_window_lse of a context on
the same inputs: bit-equal normalisers on consecutive calls that reuse the
same scratch, each smaller than the one before, on both pass families, and
within the score tolerance of the oracle's."""
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


def test_static_scratch_matches_the_context_call():
    import torch
    from paper_2606_14782_amd import bacon
    cases = [
        inputs.workload(3).with_(num_layers=1),                                  # 32K video, 8 KV heads
        inputs.shrink(inputs.workload(4), num_layers=1, max_len=3000, num_kv_heads=2),   # ragged, smaller
        inputs.workload(0).with_(num_layers=1),                                  # tiny fp32: streaming pass
    ]
    for wl in cases:
        P.log(f"[no-alloc] {wl.name} B={wl.batch} T={wl.total_tokens} Hkv={wl.num_kv_heads} {wl.dtype}")
        batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
        x = inputs.layer_inputs(wl, 0)
        q, k = P.to_dev(x["q_win"], wl), P.to_dev(x["k"], wl)
        ctx = P.make_ctx(wl)
        want = ctx.bacon_window_lse(batch, q, k)
        got = bacon.bacon_window_lse_static(ctx.shape, batch, q, k)
        torch.cuda.synchronize()
        assert torch.equal(got, want), f"{wl.name}: static-scratch normalisers differ"
        r = ref.Prompt.for_workload(wl).layer(0, x["q_win"], x["k"])
        P.close(f"{wl.name} static lse", got.cpu().numpy(), r["lse"], P.RTOL[wl.dtype])
        del q, k, ctx
