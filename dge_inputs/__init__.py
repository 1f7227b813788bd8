"""Seeded synthetic inputs for the eviction step, shared by the GPU path and the oracle.

This module holds no arithmetic of the eviction method itself: it draws Gaussian
query/key/value tensors, plants attention-attracting spans the way the workload
recipes below state, rounds to bfloat16 storage, and records the geometry.
Both sides read the *stored* values: ``bits`` (uint16 bfloat16 patterns or the
float32 array itself) and an exact float32 copy of them.

Workload recipes (Llama-3-8B KV geometry: 32 query / 8 KV heads, head dim 128,
the paper's backbone table (Llama-3-8B); lengths cover LongBench's input range, Sec. 6):

* ``c1`` tiny fp32 case: 4q/2kv heads, d 64, L 512, window 8, k 2, B 64, pool 5,
  eight candidate keys per KV head scaled x4.
* ``c2`` one Llama-3-8B-shaped layer: L 4096, window 32, k 2, B 512, pool 7, bf16,
  three 16-token spans per KV head pulled toward the group's mean query.
* ``c3`` the same geometry at L 16384 over 32 layers with PyramidKV-style layer
  budgets falling linearly 2048 -> 256, eleven spans per layer.
* ``c4`` batch of 8 ragged sequences, L_b ~ U[16384, 32768], 32 layers, B 2048.
* ``c5`` H2O: one layer, L 8192 + k 2 rows all scored, B 1024 = 512 heavy + 512
  recent; StreamingLLM 4 sinks + 1020 recent as the closed-form check.

RNG: ``numpy.random.default_rng(SeedSequence([cfg_id, layer, seq, tensor]))``
with tensor ids Q=0, K=1, V=2, plant=3, standard normal float32 draws.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from typing import Optional

import numpy as np

T_Q, T_K, T_V, T_PLANT, T_QALL, T_LEN = 0, 1, 2, 3, 4, 5


# --------------------------------------------------------------------------------------
# bfloat16 storage (round to nearest even), used only to produce stored input bits.
# --------------------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    return r


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------------------
# Workload geometry
# --------------------------------------------------------------------------------------
@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    prompt_lens: tuple          # L_b per sequence
    window: int
    k_draft: int
    budget: int                 # per-head budget B (window included)
    pool: int                   # max-pool kernel (odd)
    dtype: str                  # "bf16" or "f32"
    n_layers: int = 1
    plant: str = "none"         # "none" | "scale_rows" | "spans"
    plant_rows: int = 0         # c1: candidate rows scaled per KV head
    plant_scale: float = 4.0
    layer_budgets: Optional[tuple] = None   # per-layer B_l (c3)
    h2o: bool = False           # c5: all rows are scored (H2O accumulator)
    n_recent: int = 0           # c5: recent rows kept by H2O
    slm_sinks: int = 0
    slm_recent: int = 0

    @property
    def batch(self) -> int:
        return len(self.prompt_lens)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def cached_lens(self) -> tuple:
        return tuple(L + self.k_draft for L in self.prompt_lens)

    @property
    def kv_offsets(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.cached_lens)]).astype(np.int64)

    @property
    def total_rows(self) -> int:
        return int(sum(self.cached_lens))

    @property
    def n_rows(self) -> int:
        return self.window + self.k_draft

    def budget_of_layer(self, layer: int) -> int:
        if self.layer_budgets is not None:
            return int(self.layer_budgets[layer])
        return self.budget


def _c3_budgets(n_layers: int = 32, hi: int = 2048, lo: int = 256) -> tuple:
    # Endpoints kept as stated (2048 at layer 0, 256 at the last layer), linear between.
    return tuple(int(hi - round(l * (hi - lo) / (n_layers - 1))) for l in range(n_layers))


def _c4_lengths(batch: int = 8) -> tuple:
    rng = np.random.default_rng(np.random.SeedSequence([4, 0, 0, T_LEN]))
    return tuple(int(x) for x in rng.integers(16384, 32768 + 1, size=batch))


WORKLOADS = {
    "c1": Workload("c1", 1, 4, 2, 64, (512,), 8, 2, 64, 5, "f32",
                   plant="scale_rows", plant_rows=8, plant_scale=4.0),
    "c2": Workload("c2", 2, 32, 8, 128, (4096,), 32, 2, 512, 7, "bf16", plant="spans"),
    "c3": Workload("c3", 3, 32, 8, 128, (16384,), 32, 2, 2048, 7, "bf16", n_layers=32,
                   plant="spans", layer_budgets=_c3_budgets()),
    "c4": Workload("c4", 4, 32, 8, 128, _c4_lengths(), 32, 2, 2048, 7, "bf16", n_layers=32),
    "c5": Workload("c5", 5, 32, 8, 128, (8192,), 0, 2, 1024, 1, "bf16", h2o=True,
                   n_recent=512, slm_sinks=4, slm_recent=1020),
}


def small_variant(base: str, prompt_lens, name: Optional[str] = None, **kw) -> Workload:
    """A reduced copy of a named workload (same heads/dtype/recipe, other lengths)."""
    w = WORKLOADS[base]
    return replace(w, name=name or f"{base}_small", prompt_lens=tuple(prompt_lens), **kw)


# --------------------------------------------------------------------------------------
# Generators
# --------------------------------------------------------------------------------------
def _rng(cfg_id: int, layer: int, seq: int, tensor: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([cfg_id, layer, seq, tensor]))


@dataclass
class LayerInputs:
    """One layer's stored inputs in the packed, head-major layouts of the library.

    q:     [H_q][batch * (w + k)][d]  scoring rows (window then draft), ascending position
    k, v:  [H_kv][sum N_b][d]
    q_all: [H_q][sum N_b][d]          every cached row's query (H2O only)
    ``*_bits`` hold what is stored on the device (uint16 for bf16, float32 for f32);
    the float32 arrays are the exact values of those bits.
    """
    wl: Workload
    layer: int
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    q_bits: np.ndarray
    k_bits: np.ndarray
    v_bits: np.ndarray
    q_all: Optional[np.ndarray] = None
    q_all_bits: Optional[np.ndarray] = None
    planted: dict = field(default_factory=dict)


def _store(x: np.ndarray, dtype: str):
    if dtype == "bf16":
        bits = f32_to_bf16_bits(x)
        return bf16_bits_to_f32(bits).reshape(x.shape), bits.reshape(x.shape)
    x = np.ascontiguousarray(x, dtype=np.float32)
    return x, x


def make_layer(wl: Workload, layer: int = 0, with_v: bool = True) -> LayerInputs:
    Hq, Hkv, d, G = wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.group
    nr = wl.n_rows
    T = wl.total_rows
    offs = wl.kv_offsets
    q = np.empty((Hq, wl.batch * nr, d), np.float32)
    k = np.empty((Hkv, T, d), np.float32)
    v = np.empty((Hkv, T, d), np.float32) if with_v else np.zeros((Hkv, 0, d), np.float32)
    q_all = np.empty((Hq, T, d), np.float32) if wl.h2o else None
    planted = {}
    for b in range(wl.batch):
        N = wl.cached_lens[b]
        s0 = int(offs[b])
        k[:, s0:s0 + N] = _rng(wl.cfg_id, layer, b, T_K).standard_normal((Hkv, N, d), np.float32)
        if with_v:
            v[:, s0:s0 + N] = _rng(wl.cfg_id, layer, b, T_V).standard_normal((Hkv, N, d), np.float32)
        if wl.h2o:
            q_all[:, s0:s0 + N] = _rng(wl.cfg_id, layer, b, T_QALL).standard_normal((Hq, N, d), np.float32)
            # the scoring rows of the window/draft modes are the last w + k rows of q_all
            q[:, b * nr:(b + 1) * nr] = q_all[:, s0 + N - nr:s0 + N]
        else:
            q[:, b * nr:(b + 1) * nr] = _rng(wl.cfg_id, layer, b, T_Q).standard_normal((Hq, nr, d), np.float32)
        C = N - nr  # candidate rows (the tail is protected)
        prng = _rng(wl.cfg_id, layer, b, T_PLANT)
        if wl.plant == "scale_rows":
            for h in range(Hkv):
                rows = prng.choice(C, size=wl.plant_rows, replace=False)
                k[h, s0 + rows] *= wl.plant_scale
                planted[(b, h)] = np.sort(rows)
        elif wl.plant == "spans":
            L = wl.prompt_lens[b]
            n_spans = int(math.ceil(0.01 * L / 16))
            for h in range(Hkv):
                qg = q[h * G:(h + 1) * G, b * nr:(b + 1) * nr].reshape(-1, d).astype(np.float64)
                u = qg.mean(axis=0)
                u /= np.linalg.norm(u)
                # non-overlapping 16-token spans at random candidate starts: one span
                # inside each of n_spans distinct 32-row slots, at a random offset
                n_slots = C // 32
                n_spans = min(n_spans, n_slots)
                slots = np.sort(prng.choice(max(n_slots, 1), size=n_spans, replace=False))
                starts = slots * 32 + prng.integers(0, 17, size=n_spans)
                rows = (starts[:, None] + np.arange(16)[None, :]).reshape(-1)
                k[h, s0 + rows] += np.float32(wl.plant_scale * math.sqrt(d)) * u.astype(np.float32)
                planted[(b, h)] = rows
    q, qb = _store(q, wl.dtype)
    k, kb = _store(k, wl.dtype)
    v, vb = _store(v, wl.dtype)
    qa = qab = None
    if q_all is not None:
        qa, qab = _store(q_all, wl.dtype)
    return LayerInputs(wl, layer, q, k, v, qb, kb, vb, qa, qab, planted)


def random_scores(shape, seed: int, kind: str = "continuous") -> np.ndarray:
    """Non-negative float32 score arrays for selection tests.

    ``continuous`` is tie-free with probability ~1; ``plateau`` repeats values in
    short runs (as max-pooling does); ``ints`` draws small integers (many ties);
    ``ulps`` draws values a few thousand units in the last place above 1.0, so that
    distinct values share every leading bit but the last dozen (and some repeat).
    """
    rng = np.random.default_rng(np.random.SeedSequence([99, seed]))
    if kind == "continuous":
        return rng.random(shape, dtype=np.float32) + np.float32(1e-6)
    if kind == "ints":
        return rng.integers(0, 6, size=shape).astype(np.float32)
    if kind == "plateau":
        base = rng.random(shape, dtype=np.float32)
        n = shape[-1]
        runs = rng.integers(1, 6, size=n)
        idx = np.repeat(np.arange(n), runs)[:n]
        return np.ascontiguousarray(base[..., idx])
    if kind == "ulps":
        off = rng.integers(0, 3000, size=shape).astype(np.uint32)
        return (np.uint32(0x3F800000) + off).view(np.float32)
    raise ValueError(kind)


def device_layer(wl: Workload, layer: int, device: str):
    """One layer of a workload without planted structure (c4), drawn on the GPU: the same
    distribution as make_layer (standard normal float32, rounded to nearest even bf16),
    from torch's Philox generator seeded by (cfg_id, layer).  For benchmark layers beyond
    the one the oracle checks, where drawing tens of GB on the host would take minutes.
    Returns device tensors (q [H_q][batch*(w+k)][d], k, v [H_kv][T][d])."""
    import torch
    if wl.plant != "none" or wl.h2o:
        raise ValueError("device_layer draws unplanted layers only")
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    gen = torch.Generator(device=device)
    out = []
    for tensor, shape in ((T_Q, (wl.n_q_heads, wl.batch * wl.n_rows, wl.head_dim)),
                          (T_K, (wl.n_kv_heads, wl.total_rows, wl.head_dim)),
                          (T_V, (wl.n_kv_heads, wl.total_rows, wl.head_dim))):
        gen.manual_seed(int(np.random.SeedSequence([wl.cfg_id, layer, tensor]).generate_state(1)[0]))
        out.append(torch.randn(shape, generator=gen, device=device, dtype=torch.float32).to(dt))
    return tuple(out)
