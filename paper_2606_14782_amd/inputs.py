"""Seeded synthetic inputs for the prefill KV-compression pass.

This module only draws numbers: it holds none of the method's arithmetic
(no attention, no scores, no selection).  Both the fp64 CPU oracle and the
HIP path consume the bytes produced here, so a given (workload, seed, layer)
always yields identical tensors on every machine and for any thread count.

Tensor layouts (packed, padding-free, ``cu_seqlens`` offsets):

* ``q_win`` ``[B*W, H_q, d]``: the last ``W`` prompt queries of every sequence
  (row ``b*W + w`` is position ``N_b - W + w`` of sequence ``b``), post-RoPE.
* ``k``, ``v`` ``[T, H_kv, d]`` with ``T = sum_b N_b``: the layer's cache.

Workload shapes follow the multimodal settings of the paper (Sec. 5, Tables 1-4):
a LLaVA-style MHA model with 576 visual tokens, a Qwen2-VL-style GQA model with
thousands of visual tokens, a 32K-token video prompt (the paper's efficiency
runs use 32000 tokens) and a ragged serving batch.  No benchmark item is used:
every value is drawn from the seeded distributions below.
"""
from __future__ import annotations

import concurrent.futures as _cf
import os
from dataclasses import dataclass, replace

import numpy as np

_BLOCK = 1 << 22          # elements per independently seeded RNG block
_T_Q, _T_K, _T_V, _T_OUT, _T_LOWRANK, _T_PLANT = 1, 2, 3, 4, 5, 6
PLANT_MAG = 4.0           # planted key = PLANT_MAG * unit(last query) + noise
PLANT_NOISE = 0.1         # std of the per-entry noise on planted keys
PLANT_SPACING_RADIUS = 5  # planted keys are >= 2r+1 apart, r = default radius


@dataclass(frozen=True)
class Workload:
    """A synthetic prompt batch: model shape, per-sequence lengths and budgets."""

    name: str
    num_layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    window: int
    pool_kernel: int
    dtype: str                       # "fp32" or "bf16"
    seq_lens: tuple[int, ...]
    budgets: tuple[int, ...]         # per sequence, per KV head
    visual: tuple[tuple[int, int], ...]  # per sequence [start, end) of visual tokens
    n_planted: int                   # planted evidence keys per (sequence, KV head)
    seed: int
    value_scale: float = 1.0         # Q, K, V are N(0,1) * value_scale
    k_outlier_channels: int = 0      # K channels multiplied by k_outlier_scale
    k_outlier_scale: float = 1.0
    frame_rank: int = 0              # rank of a frame-periodic component added to K
    frame_len: int = 256

    @property
    def batch(self) -> int:
        return len(self.seq_lens)

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def total_tokens(self) -> int:
        return int(sum(self.seq_lens))

    @property
    def cu_seqlens(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.seq_lens)]).astype(np.int32)

    @property
    def budgets_arr(self) -> np.ndarray:
        return np.asarray(self.budgets, dtype=np.int32)

    @property
    def elem_size(self) -> int:
        return 4 if self.dtype == "fp32" else 2

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# --------------------------------------------------------------------------
# The five workloads.  Index 0 is the tiny fp32 case the oracle runs in
# seconds; 1-4 are the model-shaped bf16 cases.
# --------------------------------------------------------------------------

def _ragged(seed: int, batch: int, lo: int, hi: int, budget_choices) -> tuple:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 99])))
    lens = rng.integers(lo, hi + 1, size=batch)
    buds = rng.choice(np.asarray(budget_choices), size=batch)
    return tuple(int(x) for x in lens), tuple(int(x) for x in buds)


def workload(idx: int) -> Workload:
    """Return workload ``idx`` (0..4) at its full size."""
    seed = 0xBAC0 + idx
    if idx == 0:
        return Workload("tiny-fp32", 2, 4, 4, 64, 8, 5, "fp32", (512,), (64,),
                        ((64, 320),), 3, seed)
    if idx == 1:
        return Workload("llava-mha-n2048", 32, 32, 32, 128, 32, 7, "bf16", (2048,), (64,),
                        ((35, 611),), 8, seed, value_scale=128 ** -0.5)
    if idx == 2:
        return Workload("qwen2vl-gqa-n8192", 28, 28, 4, 128, 32, 7, "bf16", (8192,), (128,),
                        ((35, 6435),), 16, seed, k_outlier_channels=4, k_outlier_scale=8.0)
    if idx == 3:
        return Workload("video-gqa-n32768", 32, 32, 8, 128, 32, 7, "bf16", (32768,), (256,),
                        ((32, 30752),), 0, seed, frame_rank=8, frame_len=256)
    if idx == 4:
        lens, buds = _ragged(seed, 8, 1024, 16384, (64, 128, 512))
        return Workload("ragged-b8-gqa", 32, 32, 8, 128, 32, 7, "bf16", lens, buds,
                        tuple((32, n - 256) for n in lens), 8, seed)
    raise ValueError(f"no workload {idx}")


def shrink(wl: Workload, num_layers: int | None = None, max_len: int | None = None,
           num_kv_heads: int | None = None) -> Workload:
    """A smaller copy of ``wl`` with the same structure, for fast oracle runs.

    Sequence lengths are capped at ``max_len`` (visual spans clipped to match)
    and the KV head count reduced keeping the GQA group size.
    """
    kw = {}
    if num_layers is not None:
        kw["num_layers"] = num_layers
    if num_kv_heads is not None:
        kw["num_kv_heads"] = num_kv_heads
        kw["num_q_heads"] = num_kv_heads * wl.group
    if max_len is not None:
        lens = tuple(min(n, max_len) for n in wl.seq_lens)
        vis = tuple((min(s, n), min(e, n)) for (s, e), n in zip(wl.visual, lens))
        kw["seq_lens"] = lens
        kw["visual"] = vis
    return wl.with_(**kw)


# --------------------------------------------------------------------------
# Drawing
# --------------------------------------------------------------------------

def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def _threads() -> int:
    return max(1, min(16, int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))))


def _normal(shape, *key: int) -> np.ndarray:
    """N(0,1) float32 array; each 4M-element block has its own seed key."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)
    blocks = [(i, min(n, i + _BLOCK)) for i in range(0, n, _BLOCK)]

    def fill(bi):
        lo, hi = blocks[bi]
        out[lo:hi] = _rng(*key, bi).standard_normal(hi - lo, dtype=np.float32)

    if len(blocks) > 1:
        with _cf.ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(len(blocks))))
    elif blocks:
        fill(0)
    return out.reshape(shape)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); float32 result."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """The uint16 bfloat16 encoding of bf16-exact float32 values."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def planted_positions(wl: Workload) -> list[np.ndarray]:
    """Per sequence, an int array ``[H_kv, n_planted]`` of planted key positions.

    Positions lie inside the visual span, outside the last ``W + r`` prompt
    positions, pairwise at least ``2r + 1`` apart, and are the same at every
    layer (persistent evidence).
    """
    r = PLANT_SPACING_RADIUS
    out = []
    for b, (n, (vs, ve)) in enumerate(zip(wl.seq_lens, wl.visual)):
        hi = min(ve, n - wl.window - r)
        pos = np.zeros((wl.num_kv_heads, wl.n_planted), dtype=np.int64)
        for h in range(wl.num_kv_heads):
            rng = _rng(wl.seed, _T_PLANT, b, h)
            chosen: list[int] = []
            tries = 0
            while len(chosen) < wl.n_planted:
                if tries > 100000 or hi <= vs:
                    raise ValueError("visual span too small for planted keys")
                c = int(rng.integers(vs, hi))
                tries += 1
                if all(abs(c - p) >= 2 * r + 1 for p in chosen):
                    chosen.append(c)
            pos[h] = np.sort(np.asarray(chosen, dtype=np.int64))
        out.append(pos)
    return out


def layer_inputs(wl: Workload, layer: int) -> dict[str, np.ndarray]:
    """Draw one layer: ``q_win``, ``k``, ``v`` as float32 (bf16-exact for bf16).

    * Q, K, V ~ N(0, 1) * value_scale.
    * K: optional outlier channels (seed-chosen per layer and KV head) scaled
      up, and an optional frame-periodic low-rank component on visual tokens,
      ``K[i] += U[(i - vs) mod frame_len] @ R`` with ``U`` N(0,1) and ``R``
      N(0,1)/sqrt(rank) per layer and KV head, producing near-ties.
    * Planted evidence keys: ``PLANT_MAG * q_hat/|q_hat| + N(0, PLANT_NOISE^2)``
      with ``q_hat`` the group mean of the last query of the KV head's group.
    """
    B, W, Hq, Hkv, d = wl.batch, wl.window, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    T = wl.total_tokens
    cu = wl.cu_seqlens
    s = wl.value_scale
    q = _normal((B * W, Hq, d), wl.seed, _T_Q, layer)
    k = _normal((T, Hkv, d), wl.seed, _T_K, layer)
    v = _normal((T, Hkv, d), wl.seed, _T_V, layer)
    if s != 1.0:
        q *= np.float32(s)
        k *= np.float32(s)
        v *= np.float32(s)
    if wl.k_outlier_channels:
        for h in range(Hkv):
            ch = _rng(wl.seed, _T_OUT, layer, h).choice(d, wl.k_outlier_channels, replace=False)
            k[:, h, ch] *= np.float32(wl.k_outlier_scale)
    if wl.frame_rank:
        rank = wl.frame_rank
        for h in range(Hkv):
            g = _rng(wl.seed, _T_LOWRANK, layer, h)
            U = g.standard_normal((wl.frame_len, rank), dtype=np.float32)
            R = (g.standard_normal((rank, d), dtype=np.float32) / np.float32(np.sqrt(rank)))
            comp = U @ R                                  # [frame_len, d]
            for b in range(B):
                vs, ve = wl.visual[b]
                if ve <= vs:
                    continue
                phase = (np.arange(vs, ve) - vs) % wl.frame_len
                k[cu[b] + vs:cu[b] + ve, h, :] += comp[phase]
    if wl.n_planted:
        G = wl.group
        for b, pos in enumerate(planted_positions(wl)):
            last = q[b * W + W - 1]                       # [Hq, d]
            for h in range(Hkv):
                qh = last[h * G:(h + 1) * G].astype(np.float64).mean(axis=0)
                unit = qh / np.linalg.norm(qh)
                noise = _rng(wl.seed, _T_PLANT, 1000 + layer, b, h).standard_normal(
                    (pos.shape[1], d))
                k[cu[b] + pos[h], h, :] = (PLANT_MAG * unit[None, :] + PLANT_NOISE * noise
                                           ).astype(np.float32)
    if wl.dtype == "bf16":
        q, k, v = round_bf16(q), round_bf16(k), round_bf16(v)
    return {"q_win": q, "k": k, "v": v}
