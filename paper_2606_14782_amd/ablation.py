"""Ablation and sensitivity sweeps of the calibration on the synthetic workloads.

Runs the fused per-layer call (``bacon_compress_layer``) through the C ABI for a
default configuration and a set of variants on the same seeded inputs, and
reports how far each variant's kept set moves from the default one and how
many planted evidence keys each keeps.  The variants are the evidence terms of
V (Sec. 4.3, Eq. structurally_calibrated_evidence: E, L, T and their subsets),
the coherence radius r (Eqs. neighbor_matrix, intra_layer_coherence), the
persistence depth m (Eq. inter_layer_persistence), the calibration strength
gamma (Eq. lambda_solution), and the pooling of the score before the top-K.
The window score alone (no last-query evidence, S = B) is the SnapKV baseline.

Every statistic is over (layer, sequence, KV head):
  overlap   |kept_variant & kept_default| / budget, mean
  changed   share of (layer, sequence, head) whose kept set differs at all
  planted   share of the planted evidence keys kept (workloads that plant them)

Usage (needs a GPU):  python -m paper_2606_14782_amd.ablation [--workloads 2,4]
                      [--layers 8] [--out table.md]
"""
from __future__ import annotations

import argparse
import sys

import numpy as np

from . import bacon, inputs

# name -> bacon_params overrides
VARIANTS = [
    ("default (E+L+T, r 5, m 4, mean of S)", {}),
    ("window score only (S = B)", {"use_last_query": 0}),
    ("terms E", {"terms": 1}),
    ("terms E+L", {"terms": 3}),
    ("terms E+T", {"terms": 5}),
    ("terms L+T", {"terms": 6}),
    ("radius 0", {"radius": 0}),
    ("radius 2", {"radius": 2}),
    ("radius 10", {"radius": 10}),
    ("radius 16", {"radius": 16}),
    ("persistence m 0", {"persist_m": 0}),
    ("persistence m 1", {"persist_m": 1}),
    ("persistence m 8", {"persist_m": 8}),
    ("persistence m 16", {"persist_m": 16}),
    ("gamma 0.5", {"gamma": 0.5}),
    ("gamma 2", {"gamma": 2.0}),
    ("pool off (width 1)", {"pool_kernel": 1}),
    ("pool width 15", {"pool_kernel": 15}),
    ("max of S", {"pool_mode": bacon.POOL_MAX_S}),
    ("mean of B before calibration", {"pool_mode": bacon.POOL_MEAN_B}),
]


def sweep(wl: inputs.Workload, layers: int, log=print) -> list[dict]:
    """Kept sets of every variant on the first ``layers`` layers of ``wl``."""
    import torch
    wl = wl.with_(num_layers=layers)
    batch = bacon.BatchLayout(wl.cu_seqlens, wl.budgets_arr)
    ctxs = []
    for _, kw in VARIANTS:
        p = bacon.default_params(**{"pool_kernel": wl.pool_kernel, **kw})
        ctx = bacon.Context(wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim,
                            wl.window, wl.batch, wl.total_tokens, wl.dtype, p)
        ctx.bacon_begin_prompt(batch)
        ctxs.append(ctx)
    planted = inputs.planted_positions(wl) if wl.n_planted else None
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    kept = [[] for _ in VARIANTS]          # per variant, per layer: idx array
    for layer in range(layers):
        x = inputs.layer_inputs(wl, layer)
        q = torch.from_numpy(x["q_win"]).cuda().to(tdt)
        k = torch.from_numpy(x["k"]).cuda().to(tdt)
        v = torch.from_numpy(x["v"]).cuda().to(tdt)
        for vi, ctx in enumerate(ctxs):
            idx, _, _ = ctx.bacon_compress_layer(layer, batch, q, k, v)
            kept[vi].append(idx)
        torch.cuda.synchronize()
        kept_np = [kv[-1].cpu().numpy() for kv in kept]
        for vi in range(len(VARIANTS)):
            kept[vi][-1] = kept_np[vi]
        log(f"  {wl.name}: layer {layer} done")
        del q, k, v
    rows = []
    off = np.concatenate([[0], np.cumsum(wl.budgets_arr * wl.num_kv_heads)])
    for vi, (name, _) in enumerate(VARIANTS):
        ov, changed, pk, ptot = [], 0, 0, 0
        for layer in range(layers):
            for b in range(wl.batch):
                K = int(wl.budgets_arr[b])
                for h in range(wl.num_kv_heads):
                    s0 = int(off[b]) + h * K
                    a = set(int(i) for i in kept[vi][layer][s0:s0 + K] if i >= 0)
                    d = set(int(i) for i in kept[0][layer][s0:s0 + K] if i >= 0)
                    ov.append(len(a & d) / K)
                    changed += a != d
                    if planted is not None:
                        pk += sum(int(p) in a for p in planted[b][h])
                        ptot += len(planted[b][h])
        n = layers * wl.batch * wl.num_kv_heads
        rows.append({"variant": name, "overlap": float(np.mean(ov)), "changed": changed / n,
                     "planted": (pk / ptot) if ptot else None})
    return rows


def table(wl_rows: list[tuple[inputs.Workload, int, list[dict]]]) -> str:
    heads = [f"{wl.name} ({layers} layers)" for wl, layers, _ in wl_rows]
    lines = ["| variant | " + " | ".join(f"{h}: overlap / changed / planted" for h in heads) + " |",
             "|---|" + "---|" * len(heads)]
    for i, (name, _) in enumerate(VARIANTS):
        cells = []
        for _, _, rows in wl_rows:
            r = rows[i]
            pl = "–" if r["planted"] is None else f"{100 * r['planted']:.1f}%"
            cells.append(f"{100 * r['overlap']:.1f}% / {100 * r['changed']:.0f}% / {pl}")
        lines.append(f"| {name} | " + " | ".join(cells) + " |")
    return "\n".join(lines)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--workloads", default="2,4,1,3", help="workload indices (inputs.workload)")
    ap.add_argument("--layers", type=int, default=8)
    ap.add_argument("--out")
    args = ap.parse_args(argv)
    import torch
    if not torch.cuda.is_available():
        raise SystemExit("the ablation sweep runs the GPU path: no GPU")
    bacon.lib()
    results = []
    for w in (int(x) for x in args.workloads.split(",")):
        wl = inputs.workload(w)
        layers = min(args.layers, wl.num_layers)
        print(f"workload {wl.name}: {layers} layers, {len(VARIANTS)} variants", file=sys.stderr,
              flush=True)
        results.append((wl, layers, sweep(wl, layers, log=lambda *a: print(*a, file=sys.stderr,
                                                                          flush=True))))
    md = table(results)
    print(md)
    if args.out:
        with open(args.out, "w") as fh:
            fh.write(md + "\n")


if __name__ == "__main__":
    main()
