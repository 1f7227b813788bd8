"""GPU parity: the HIP path through the C ABI against the float64 oracle.

Tolerances (written here, derived in the design notes):
* scores: |gpu - oracle| <= 1e-3 * |oracle| + 1e-20 elementwise (bf16 inputs, fp32
  products/softmax/accumulation; the absolute floor only covers entries that
  underflow fp32);
* selection in isolation (identical fp32 scores on both sides): bit-exact indices;
* selection end to end: every candidate whose oracle pooled score exceeds the oracle's
  B'-th value t by more than 1e-3 relative is kept, every one below t by more than
  1e-3 is dropped, and the counts agree;
* compaction: byte-exact given the GPU's own indices.
"""
import math
import sys

import numpy as np
import pytest
import torch

import dge_inputs as di
import oracle
import paper_2609_33334_amd as dge

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
RTOL, ATOL = 1e-3, 1e-20


def _log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(bits, dtype):
    t = torch.from_numpy(np.ascontiguousarray(bits))
    if dtype == "bf16":
        t = t.view(torch.int16).view(torch.bfloat16)
    return t.to(DEV)


def geom_of(wl, **kw):
    dt = dge.DGE_BF16 if wl.dtype == "bf16" else dge.DGE_F32
    return dge.Geometry(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.window, wl.k_draft,
                        wl.cached_lens, dtype=dt, device=DEV, **kw)


def mode_rows(x, wl, mode):
    """The scoring rows of a mode, packed per sequence (taken from the w+k block)."""
    nr = wl.window + wl.k_draft
    sl = {oracle.ROWS_WINDOW_DRAFT: slice(0, nr), oracle.ROWS_DRAFT: slice(wl.window, nr),
          oracle.ROWS_WINDOW: slice(0, wl.window)}[mode]
    def pick(a):
        a = a.reshape(a.shape[0], wl.batch, nr, a.shape[-1])[:, :, sl]
        return np.ascontiguousarray(a.reshape(a.shape[0], -1, a.shape[-1]))
    return pick(x.q), pick(x.q_bits)


def check_scores(got, want, what):
    got = np.asarray(got, np.float64)
    err = np.abs(got - want)
    bad = err > RTOL * np.abs(want) + ATOL
    worst = float((err / (np.abs(want) + ATOL)).max())
    _log(f"  {what}: max rel err {worst:.2e}")
    assert not bad.any(), f"{what}: {int(bad.sum())} scores out of tolerance (worst rel {worst:.3g})"


def oracle_select_compact(scores, k_bits, v_bits, lens, H, pool, n_tail, n_sel):
    """The oracle's pool -> top-B' -> compact for every (sequence, KV head) of one layer,
    on the given fp32 scores [H][T] and stored K/V element bits [H][T][d]:
    {(b, h): (idx, k rows, v rows)}."""
    offs = np.concatenate([[0], np.cumsum(lens)])
    out = {}
    for b, N in enumerate(lens):
        C = N - n_tail
        seg = slice(offs[b], offs[b + 1])
        for h in range(H):
            pooled = oracle.maxpool(np.asarray(scores[h, seg], np.float64), C, pool)
            sel = oracle.select_topb(pooled, n_sel)
            out[(b, h)] = (sel,) + oracle.compact(k_bits[h, seg], v_bits[h, seg], sel, C)
    return out


def check_select_compact(idx, n_kept, k_out, v_out, want, n_sel, n_tail, what):
    """GPU idx [batch][H][n_sel], n_kept [batch], K/V [batch][H][n_sel + n_tail][d] against
    oracle_select_compact: bit-exact indices (-1 padded), exact counts, byte-exact rows
    followed by zero rows."""
    idx = idx.cpu().numpy()
    n_kept = n_kept.cpu().numpy()
    iv = torch.int16 if k_out.dtype == torch.bfloat16 else torch.int32
    kg = k_out.cpu().view(iv).numpy()
    vg = v_out.cpu().view(iv).numpy()
    assert kg.shape[2] == n_sel + n_tail, what
    for (b, h), (sel, ko, vo) in want.items():
        assert n_kept[b] == len(sel), (what, b)
        assert np.array_equal(idx[b, h, :len(sel)], sel), (what, b, h)
        assert (idx[b, h, len(sel):] == -1).all(), (what, b, h)
        m = ko.shape[0]
        assert np.array_equal(kg[b, h, :m], ko.view(kg.dtype)), (what, b, h, "k")
        assert np.array_equal(vg[b, h, :m], vo.view(vg.dtype)), (what, b, h, "v")
        assert (kg[b, h, m:] == 0).all() and (vg[b, h, m:] == 0).all(), (what, b, h)


def check_threshold_rule(pooled, got_idx, n_sel, what):
    """End-to-end selection rule: with t the oracle's B'-th largest pooled score, every
    candidate above t by more than 1e-3 relative is kept, every one below by more than
    1e-3 dropped, and the count is B' = min(n_sel, C)."""
    C = pooled.shape[0]
    n = min(n_sel, C)
    got = set(int(i) for i in got_idx if i >= 0)
    assert len(got) == n, (what, len(got), n)
    if n == 0 or n == C:
        assert got == set(range(n)), what
        return
    t = np.sort(pooled)[::-1][n - 1]
    must = set(np.nonzero(pooled > t * (1 + 1e-3))[0].tolist())
    never = set(np.nonzero(pooled < t * (1 - 1e-3))[0].tolist())
    assert must <= got, (what, "missing", sorted(must - got)[:8])
    assert not (never & got), (what, "extra", sorted(never & got)[:8])


def run_score(wl, x, mode=oracle.ROWS_WINDOW_DRAFT):
    g = geom_of(wl)
    q, qb = mode_rows(x, wl, mode)
    raw = dge.score(g, mode, to_dev(qb, wl.dtype), to_dev(x.k_bits, wl.dtype))
    torch.cuda.synchronize()
    want = oracle.window_scores(q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads, wl.window,
                                wl.k_draft, mode)
    return raw.cpu().numpy(), want


SCORE_CASES = {
    "c1": di.WORKLOADS["c1"],
    "c2_700": di.small_variant("c2", [700]),
    "c2_ragged": di.small_variant("c2", [300, 517, 1029, 70]),
    "f32_d128": di.small_variant("c2", [333], dtype="f32", plant="none"),
    "bf16_d64": di.small_variant("c1", [400, 129], dtype="bf16"),
    "big_M": di.small_variant("c2", [260], n_q_heads=64, window=64, k_draft=8, plant="none"),
    "w0": di.small_variant("c2", [96], window=0, k_draft=3, plant="none"),
    # row-tile splits across the 4 wavefronts: 7 tiles (1 own + 3 shared), 14 tiles
    # (3 own + 2 shared), fp32 with 13 tiles (3 + 1), and 52 tiles in two row groups
    "t7": di.small_variant("c2", [611, 130], window=24, k_draft=4, plant="none"),
    "t14": di.small_variant("c2", [777], window=48, k_draft=8, plant="none"),
    "f32_t13": di.small_variant("c2", [300], dtype="f32", window=46, k_draft=6, plant="none"),
    "groups2": di.small_variant("c2", [450, 200], n_q_heads=64, window=96, k_draft=8,
                                plant="none"),
}


@pytest.mark.parametrize("case", list(SCORE_CASES))
def test_score_parity(case):
    wl = SCORE_CASES[case]
    _log(f"score parity {case} lens={wl.prompt_lens}")
    x = di.make_layer(wl)
    got, want = run_score(wl, x)
    check_scores(got, want, case)
    # each sequence's scores sum to its number of scoring rows
    for b in range(wl.batch):
        s0, s1 = wl.kv_offsets[b], wl.kv_offsets[b + 1]
        assert np.allclose(got[:, s0:s1].sum(1), wl.n_rows, rtol=1e-4)


@pytest.mark.parametrize("mode", [oracle.ROWS_DRAFT, oracle.ROWS_WINDOW])
def test_score_modes(mode):
    wl = di.small_variant("c2", [450, 1100])
    _log(f"score mode {mode}")
    x = di.make_layer(wl)
    got, want = run_score(wl, x, mode)
    check_scores(got, want, f"mode{mode}")


def test_score_full_c2():
    wl = di.WORKLOADS["c2"]
    _log("score parity c2 full")
    x = di.make_layer(wl)
    got, want = run_score(wl, x)
    check_scores(got, want, "c2")


def test_score_c3_layer():
    wl = di.WORKLOADS["c3"]
    _log("score parity c3 layer 5 (L=16384)")
    x = di.make_layer(wl, layer=5, with_v=False)
    got, want = run_score(wl, x)
    check_scores(got, want, "c3/l5")
    # selection of that layer under its own budget, end to end by the threshold rule
    g = geom_of(wl)
    n_tail = wl.window + wl.k_draft
    nsel = wl.budget_of_layer(5) - wl.window
    idx, nk = dge.select_topb(g, torch.from_numpy(np.ascontiguousarray(got)).to(DEV), wl.pool,
                              n_tail, nsel)
    torch.cuda.synchronize()
    idx = idx.cpu().numpy()
    C = wl.cached_lens[0] - n_tail
    for h in range(wl.n_kv_heads):
        pooled = oracle.maxpool(want[h], C, wl.pool)
        t = np.sort(pooled)[::-1][nsel - 1]
        sel = set(idx[0, h].tolist())
        assert len(sel) == nsel
        must = set(np.nonzero(pooled > t * (1 + 1e-3))[0].tolist())
        never = set(np.nonzero(pooled < t * (1 - 1e-3))[0].tolist())
        assert must <= sel and not (never & sel), h


def test_score_and_select_c4_layer_sampled():
    # the full ragged c4 layer (8 sequences of 16K-32K rows, 64-tile walks as in the
    # 32-layer launch) on the GPU; the oracle scores two of its sequences, and the
    # selection of those sequences must pass the end-to-end threshold rule
    wl = di.WORKLOADS["c4"]
    _log("score + select parity: c4 layer, sequences 0 and 7 sampled")
    x = di.make_layer(wl, with_v=False)
    g = geom_of(wl)
    raw = dge.score(g, oracle.ROWS_WINDOW_DRAFT, to_dev(x.q_bits, "bf16"), to_dev(x.k_bits, "bf16"))
    n_tail = wl.window + wl.k_draft
    nsel = wl.budget - wl.window
    idx, nk = dge.select_topb(g, raw, wl.pool, n_tail, nsel)
    torch.cuda.synchronize()
    raw, idx, nk = raw.cpu().numpy(), idx.cpu().numpy(), nk.cpu().numpy()
    nr = n_tail
    for b in (0, 7):
        s0, s1 = int(wl.kv_offsets[b]), int(wl.kv_offsets[b + 1])
        want = oracle.window_scores(x.q[:, b * nr:(b + 1) * nr], x.k[:, s0:s1], [0, s1 - s0],
                                    wl.n_q_heads, wl.n_kv_heads, wl.window, wl.k_draft)
        check_scores(raw[:, s0:s1], want, f"c4 sequence {b}")
        C = s1 - s0 - n_tail
        assert nk[b] == min(nsel, C)
        for h in range(wl.n_kv_heads):
            pooled = oracle.maxpool(want[h], C, wl.pool)
            t = np.sort(pooled)[::-1][nsel - 1]
            got = set(idx[b, h].tolist())
            assert len(got) == nsel
            must = set(np.nonzero(pooled > t * (1 + 1e-3))[0].tolist())
            never = set(np.nonzero(pooled < t * (1 - 1e-3))[0].tolist())
            assert must <= got and not (never & got), (b, h)


def test_score_layer_major_long_walks():
    # eight copies of a c3 layer scored as one layer-major geometry (64 KV heads): every
    # workgroup walks the longest chunk (64 tiles of 64 keys); each copy must match the
    # oracle of the layer
    wl = di.WORKLOADS["c3"]
    _log("score parity: 8 stacked c3 layers in one call")
    x = di.make_layer(wl, layer=2, with_v=False)
    nl = 8
    g = dge.Geometry(wl.n_q_heads * nl, wl.n_kv_heads * nl, wl.head_dim, wl.window, wl.k_draft,
                     wl.cached_lens, device=DEV)
    q = to_dev(x.q_bits, "bf16").repeat(nl, 1, 1)
    k = to_dev(x.k_bits, "bf16").repeat(nl, 1, 1)
    raw = dge.score(g, oracle.ROWS_WINDOW_DRAFT, q, k)
    torch.cuda.synchronize()
    raw = raw.cpu().numpy()
    want = oracle.window_scores(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads, wl.window,
                                wl.k_draft, oracle.ROWS_WINDOW_DRAFT)
    H = wl.n_kv_heads
    for l in range(nl):
        check_scores(raw[l * H:(l + 1) * H], want, f"layer copy {l}")


@pytest.mark.parametrize("mode", [oracle.ROWS_WINDOW_DRAFT, oracle.ROWS_WINDOW])
def test_score_long_walks_short_last_chunks(mode):
    # eight stacked copies of a ragged three-sequence layer (64 KV heads): the launch walks
    # 64 tiles per workgroup, which takes the stats pass with one K stream per wavefront
    # (9 or 8 row tiles); two sequences end 20 and 70 keys into their last 4096-key chunk,
    # whose 2 and 5 subtiles of 16 keys leave some wavefronts of the workgroup no keys
    wl = di.small_variant("c3", [16382, 12306, 8260])
    assert tuple(wl.cached_lens) == (16384, 12308, 8262)
    _log(f"score parity: long walks, short last chunks, mode {mode}")
    x = di.make_layer(wl, layer=3, with_v=False)
    nl = 8
    g = dge.Geometry(wl.n_q_heads * nl, wl.n_kv_heads * nl, wl.head_dim, wl.window, wl.k_draft,
                     wl.cached_lens, device=DEV)
    q, qb = mode_rows(x, wl, mode)
    raw = dge.score(g, mode, to_dev(qb, "bf16").repeat(nl, 1, 1),
                    to_dev(x.k_bits, "bf16").repeat(nl, 1, 1))
    torch.cuda.synchronize()
    raw = raw.cpu().numpy()
    want = oracle.window_scores(q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads, wl.window,
                                wl.k_draft, mode)
    H = wl.n_kv_heads
    for l in range(nl):
        check_scores(raw[l * H:(l + 1) * H], want, f"layer copy {l}")


@pytest.mark.parametrize("case", ["g8_w16_k2", "g2_w64_k4"])
def test_score_long_walks_other_group_sizes(case):
    # the per-wavefront passes serve any 8 or 9 row tiles: 8 query heads per KV head with
    # 18 scoring rows (144 rows, no padding row) and 2 heads with 68 rows (136 rows, 8
    # padding rows), eight stacked layers so that the walks are long
    kw = {"g8_w16_k2": dict(n_q_heads=64, window=16, k_draft=2),
          "g2_w64_k4": dict(n_q_heads=16, window=64, k_draft=4)}[case]
    wl = di.small_variant("c3", [16382, 8260], plant="none", **kw)
    _log(f"score parity: long walks, {case}")
    x = di.make_layer(wl, layer=1, with_v=False)
    nl = 8
    g = dge.Geometry(wl.n_q_heads * nl, wl.n_kv_heads * nl, wl.head_dim, wl.window, wl.k_draft,
                     wl.cached_lens, device=DEV)
    raw = dge.score(g, oracle.ROWS_WINDOW_DRAFT, to_dev(x.q_bits, "bf16").repeat(nl, 1, 1),
                    to_dev(x.k_bits, "bf16").repeat(nl, 1, 1))
    torch.cuda.synchronize()
    raw = raw.cpu().numpy()
    want = oracle.window_scores(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads, wl.window,
                                wl.k_draft)
    H = wl.n_kv_heads
    for l in range(nl):
        check_scores(raw[l * H:(l + 1) * H], want, f"{case} layer copy {l}")


def test_score_lse_long_walks_short_last_chunks():
    # the single pass with the rows' LSE supplied, on the stacked ragged layers above: 64-tile
    # walks take the colsum pass with one K stream per wavefront, the normalisers entering
    # as its products' initial accumulators
    wl = di.small_variant("c3", [16382, 12306, 8260])
    _log("score with supplied row LSE: long walks, short last chunks")
    x = di.make_layer(wl, layer=3, with_v=False)
    nl = 8
    g = dge.Geometry(wl.n_q_heads * nl, wl.n_kv_heads * nl, wl.head_dim, wl.window, wl.k_draft,
                     wl.cached_lens, device=DEV)
    lse = oracle.scoring_row_lse(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads, wl.window,
                                 wl.k_draft)
    lse_d = torch.from_numpy(lse.astype(np.float32)).to(DEV).repeat(nl, 1).contiguous()
    raw = dge.score_lse(g, dge.ROWS_WINDOW_DRAFT, to_dev(x.q_bits, "bf16").repeat(nl, 1, 1),
                        to_dev(x.k_bits, "bf16").repeat(nl, 1, 1), lse_d)
    torch.cuda.synchronize()
    raw = raw.cpu().numpy()
    want = oracle.window_scores(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads, wl.window,
                                wl.k_draft)
    H = wl.n_kv_heads
    for l in range(nl):
        check_scores(raw[l * H:(l + 1) * H], want, f"score_lse layer copy {l}")


@pytest.mark.parametrize("case", ["c2", "c2_ragged", "c1"])
def test_score_lse_single_pass(case):
    wl = {"c2": di.WORKLOADS["c2"], "c2_ragged": SCORE_CASES["c2_ragged"], "c1": di.WORKLOADS["c1"]}[case]
    _log(f"score with supplied row LSE {case}")
    x = di.make_layer(wl, with_v=False)
    g = geom_of(wl)
    lse = oracle.scoring_row_lse(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads, wl.window,
                                 wl.k_draft)
    q, k = to_dev(x.q_bits, wl.dtype), to_dev(x.k_bits, wl.dtype)
    raw = dge.score_lse(g, dge.ROWS_WINDOW_DRAFT, q, k, torch.from_numpy(lse.astype(np.float32)).to(DEV))
    torch.cuda.synchronize()
    want = oracle.window_scores(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads, wl.window,
                                wl.k_draft)
    check_scores(raw.cpu().numpy(), want, f"score_lse {case}")


def test_score_deterministic():
    wl = di.small_variant("c2", [2000, 900])
    x = di.make_layer(wl, with_v=False)
    g = geom_of(wl)
    q, k = to_dev(x.q_bits, wl.dtype), to_dev(x.k_bits, wl.dtype)
    a = dge.score(g, 0, q, k).clone()
    b = dge.score(g, 0, q, k)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))



# ------------------------------------------------------------------------------------------
# Selection
# ------------------------------------------------------------------------------------------
SELECT_CASES = [
    # (lens, kind, pool, n_tail, n_select)
    ((4098,), "continuous", 7, 34, 480),
    ((4098,), "plateau", 7, 34, 480),
    ((700, 1500, 33, 4000), "ints", 5, 10, 200),
    ((700, 1500, 33, 4000), "plateau", 1, 10, 64),
    ((1000,), "continuous", 3, 34, 5000),       # budget covers every candidate
    ((1000,), "continuous", 7, 34, 0),          # budget equal to the window
    ((50, 34), "continuous", 7, 34, 10),        # a sequence with no candidates
    ((32770,), "plateau", 7, 34, 2016),         # largest per-sequence length of the c4 mix
    ((9000,), "ints", 1, 512, 512),             # H2O-like split
    ((40000, 300), "plateau", 7, 34, 2016),     # beyond the register path: global fallback
    ((3000, 700), "continuous", 19, 34, 300),   # pool wider than the register halo
    ((32768 + 34, 5000), "ints", 17, 34, 2016), # largest register-path candidate set
    # values that differ only in their lowest bits: the last radix digit decides
    ((4098, 1200), "ulps", 7, 34, 480),
    ((16418,), "ulps", 1, 34, 2016),
    ((30000, 9000), "ulps", 5, 34, 1500),
]


@pytest.mark.parametrize("case", range(len(SELECT_CASES)))
def test_select_isolated_bit_exact(case):
    lens, kind, pool, n_tail, n_select = SELECT_CASES[case]
    _log(f"select {lens} {kind} pool={pool} tail={n_tail} sel={n_select}")
    H = 4
    T = sum(lens)
    scores = di.random_scores((H, T), seed=case, kind=kind)
    g = dge.Geometry(8, H, 128, 0, 0, lens, device=DEV)
    idx, nk = dge.select_topb(g, torch.from_numpy(scores).to(DEV), pool, n_tail, n_select)
    torch.cuda.synchronize()
    idx, nk = idx.cpu().numpy(), nk.cpu().numpy()
    offs = np.concatenate([[0], np.cumsum(lens)])
    for b, N in enumerate(lens):
        C = N - n_tail
        assert nk[b] == min(n_select, C)
        for h in range(H):
            pooled = oracle.maxpool(scores[h, offs[b]:offs[b + 1]], C, pool)
            want = oracle.select_topb(pooled, n_select)
            got = idx[b, h]
            assert np.array_equal(got[:len(want)], want), (b, h)
            assert (got[len(want):] == -1).all()


def test_select_end_to_end_c2():
    wl = di.WORKLOADS["c2"]
    _log("select end-to-end c2")
    x = di.make_layer(wl)
    g = geom_of(wl)
    out = dge.evict_layer(g, to_dev(x.q_bits, "bf16"), to_dev(x.k_bits, "bf16"),
                          to_dev(x.v_bits, "bf16"), wl.budget, wl.pool)
    torch.cuda.synchronize()
    raw_ref, ref = oracle.evict_layer(x.q, x.k, x.v, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads,
                                      wl.window, wl.k_draft, wl.budget, wl.pool)
    idx = out["idx"].cpu().numpy()
    nsel = wl.budget - wl.window
    for h in range(wl.n_kv_heads):
        pooled = ref[(0, h)]["pooled"]
        t = np.sort(pooled)[::-1][nsel - 1]
        got = set(idx[0, h].tolist())
        assert len(got) == nsel
        must = set(np.nonzero(pooled > t * (1 + 1e-3))[0].tolist())
        never = set(np.nonzero(pooled < t * (1 - 1e-3))[0].tolist())
        assert must <= got and not (never & got), h
        # planted spans are found
        hits = np.isin(x.planted[(0, h)], idx[0, h]).mean()
        assert hits > 0.5, hits


def test_compact_bit_exact():
    wl = di.small_variant("c2", [600, 1200, 40])
    _log("compact bit-exact")
    x = di.make_layer(wl)
    g = geom_of(wl)
    k, v = to_dev(x.k_bits, "bf16"), to_dev(x.v_bits, "bf16")
    out = dge.evict_layer(g, to_dev(x.q_bits, "bf16"), k, v, wl.budget, wl.pool)
    torch.cuda.synchronize()
    idx, nk = out["idx"].cpu().numpy(), out["n_kept"].cpu().numpy()
    ko = out["k"].cpu().view(torch.int16).numpy()
    vo = out["v"].cpu().view(torch.int16).numpy()
    kb, vb = x.k_bits.view(np.int16), x.v_bits.view(np.int16)
    n_tail = wl.window + wl.k_draft
    n_out = wl.budget - wl.window + n_tail
    assert ko.shape == (wl.batch, wl.n_kv_heads, n_out, wl.head_dim)
    for b in range(wl.batch):
        s0, N = wl.kv_offsets[b], wl.cached_lens[b]
        C = N - n_tail
        assert nk[b] == min(wl.budget - wl.window, C)
        for h in range(wl.n_kv_heads):
            rows = np.concatenate([idx[b, h, :nk[b]], np.arange(C, N)]) + s0
            m = len(rows)
            assert np.array_equal(ko[b, h, :m], kb[h, rows]) and np.array_equal(vo[b, h, :m], vb[h, rows])
            assert (ko[b, h, m:] == 0).all() and (vo[b, h, m:] == 0).all()


FUSED_CASES = {
    "c2": (di.WORKLOADS["c2"], None),
    "ragged": (di.small_variant("c2", [600, 1200, 40, 3000]), None),
    "c1_f32": (di.WORKLOADS["c1"], None),
    "keep_all": (di.small_variant("c2", [300, 90]), 1000),
    "window_only_budget": (di.small_variant("c2", [500]), 32),
    "fallback_40k": (di.small_variant("c2", [40000], plant="none"), 2048),
}


@pytest.mark.parametrize("case", list(FUSED_CASES))
def test_select_compact_fused_and_separate_vs_oracle(case):
    """dge_select_compact (one launch) and dge_select_topb + dge_compact against the
    oracle's pool -> top-B' -> compact on the GPU's own fp32 scores: indices bit-exact,
    n_kept exact, compacted K/V byte-exact with zero padding (Alg. 1 steps B-C)."""
    wl, budget = FUSED_CASES[case]
    budget = wl.budget if budget is None else budget
    _log(f"select+compact vs oracle {case}")
    x = di.make_layer(wl)
    g = geom_of(wl)
    q, k, v = to_dev(x.q_bits, wl.dtype), to_dev(x.k_bits, wl.dtype), to_dev(x.v_bits, wl.dtype)
    n_tail, n_sel = wl.window + wl.k_draft, budget - wl.window
    for fused in (True, False):
        out = dge.evict_layer(g, q, k, v, budget, wl.pool, fused=fused)
        torch.cuda.synchronize()
        want = oracle_select_compact(out["raw"].cpu().numpy(), x.k_bits, x.v_bits,
                                     wl.cached_lens, wl.n_kv_heads, wl.pool, n_tail, n_sel)
        check_select_compact(out["idx"], out["n_kept"], out["k"], out["v"], want, n_sel,
                             n_tail, f"{case} fused={fused}")


def test_compact_keep_all_is_identity():
    wl = di.small_variant("c1", [60], budget=1000)
    x = di.make_layer(wl)
    g = geom_of(wl)
    k, v = to_dev(x.k_bits, "f32"), to_dev(x.v_bits, "f32")
    out = dge.evict_layer(g, to_dev(x.q_bits, "f32"), k, v, wl.budget, wl.pool)
    torch.cuda.synchronize()
    N = wl.cached_lens[0]
    assert torch.equal(out["k"][0, :, :N].cpu(), k.cpu()) and torch.equal(out["v"][0, :, :N].cpu(), v.cpu())
    assert out["idx"][0, :, :N - 10].cpu().numpy().tolist() == [list(range(N - 10))] * wl.n_kv_heads


def test_streaming_closed_form():
    wl = di.WORKLOADS["c5"]
    _log("streaming c5 + ragged")
    for lens in [wl.cached_lens, (1022, 1030, 3000, 1020)]:   # C_b = 2, 10, 1980, 0
        g = dge.Geometry(32, 8, 128, 0, 2, lens, device=DEV)
        idx, nk = dge.select_streaming(g, wl.slm_sinks, wl.slm_recent)
        torch.cuda.synchronize()
        for b, N in enumerate(lens):
            want = oracle.streaming_select(N, wl.slm_sinks, wl.slm_recent)
            assert nk[b].item() == len(want)
            for h in range(8):
                got = idx[b, h].cpu().numpy()
                assert got[:len(want)].tolist() == want.tolist() and (got[len(want):] == -1).all()


# ------------------------------------------------------------------------------------------
# H2O accumulated attention
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("supply_lse", [False, True])
@pytest.mark.parametrize("lens", [(300, 77, 1000), (5, 640, 129)])
def test_h2o_parity_small(supply_lse, lens):
    wl = di.small_variant("c5", list(lens))
    _log(f"h2o small lens={lens} supply_lse={supply_lse}")
    x = di.make_layer(wl, with_v=False)
    g = geom_of(wl)
    lse = None
    if supply_lse:
        lse_ref = oracle.h2o_row_lse(x.q_all, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads)
        lse = torch.from_numpy(lse_ref.astype(np.float32)).to(DEV)
    col = dge.h2o_colsum(g, to_dev(x.q_all_bits, "bf16"), to_dev(x.k_bits, "bf16"), lse=lse)
    torch.cuda.synchronize()
    want = oracle.h2o_colsum(x.q_all, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads)
    got = col.cpu().numpy()
    check_scores(got, want, "h2o_small")
    for b in range(wl.batch):
        s0, s1 = wl.kv_offsets[b], wl.kv_offsets[b + 1]
        assert np.allclose(got[:, s0:s1].sum(1), s1 - s0, rtol=1e-4)


def _wide_logit_layer(kind, lens):
    """A small H2O-shaped layer (every row has a query) whose logits span hundreds of
    log2 units along the keys, so that the row sums' reference must move mid-stream:
    every query is a * (1, ..., 1) plus noise and key j is r_j * (1, ..., 1) plus noise,
    giving logits of about a * r_j * sqrt(d).  "ramp": r_j grows linearly to 8.8 (a
    single new key exceeds the running reference by far more than 2^7); "step": r_j = 0
    for the first 64 keys of a sequence and 1.9 after them (every later term is ~2^124
    times the first tile's, so the sums overflow by accumulation)."""
    wl = di.small_variant("c5", list(lens))
    x = di.make_layer(wl, with_v=False)
    d = wl.head_dim
    k = 0.1 * x.k.astype(np.float32)
    q = 0.1 * x.q_all.astype(np.float32) + np.float32(4.0)
    for b in range(wl.batch):
        s0, N = int(wl.kv_offsets[b]), wl.cached_lens[b]
        j = np.arange(N, dtype=np.float32)
        r = 8.8 * j / max(N - 1, 1) if kind == "ramp" else np.where(j < 64, 0.0, 1.9)
        k[:, s0:s0 + N] += r.astype(np.float32)[None, :, None]
    kb = di.f32_to_bf16_bits(k)
    qab = di.f32_to_bf16_bits(q)
    x.k, x.k_bits = di.bf16_bits_to_f32(kb).reshape(k.shape), kb.reshape(k.shape)
    x.q_all, x.q_all_bits = di.bf16_bits_to_f32(qab).reshape(q.shape), qab.reshape(q.shape)
    nr = wl.n_rows
    qs = np.empty((wl.n_q_heads, wl.batch * nr, d), np.float32)
    qsb = np.empty(qs.shape, np.uint16)
    for b in range(wl.batch):
        s0, N = int(wl.kv_offsets[b]), wl.cached_lens[b]
        qs[:, b * nr:(b + 1) * nr] = x.q_all[:, s0 + N - nr:s0 + N]
        qsb[:, b * nr:(b + 1) * nr] = x.q_all_bits[:, s0 + N - nr:s0 + N]
    x.q, x.q_bits = qs, qsb
    return wl, x


@pytest.mark.parametrize("kind", ["ramp", "step"])
def test_wide_logit_range_scores_and_h2o_vs_oracle(kind):
    wl, x = _wide_logit_layer(kind, (700, 130))
    _log(f"wide logit range {kind}: lens={wl.cached_lens}")
    got, want = run_score(wl, x)
    check_scores(got, want, f"scores {kind}")
    g = geom_of(wl)
    # the merged row normalisers: logits of a few hundred carry fp32 accumulation error
    # proportional to their size, hence the relative term
    _, row_lse = dge.score_with_lse(g, dge.ROWS_WINDOW_DRAFT, to_dev(x.q_bits, "bf16"),
                                    to_dev(x.k_bits, "bf16"))
    torch.cuda.synchronize()
    want_lse = oracle.scoring_row_lse(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads,
                                      wl.window, wl.k_draft)
    lerr = np.abs(row_lse.cpu().numpy().astype(np.float64) - want_lse)
    _log(f"  row log-partitions in [{want_lse.min():.1f}, {want_lse.max():.1f}]: max |err| {lerr.max():.2e}")
    assert (lerr <= 1e-4 + 1e-6 * np.abs(want_lse)).all()
    col = dge.h2o_colsum(g, to_dev(x.q_all_bits, "bf16"), to_dev(x.k_bits, "bf16"))
    torch.cuda.synchronize()
    want_h = oracle.h2o_colsum(x.q_all, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads)
    got_h = col.cpu().numpy()
    check_scores(got_h, want_h, f"h2o {kind}")
    for b in range(wl.batch):
        s0, s1 = wl.kv_offsets[b], wl.kv_offsets[b + 1]
        assert np.allclose(got_h[:, s0:s1].sum(1), s1 - s0, rtol=1e-4)


def test_h2o_c5_two_heads_and_select():
    wl = di.WORKLOADS["c5"]
    _log("h2o c5 full size, oracle on KV heads 0 and 5")
    x = di.make_layer(wl, with_v=False)
    g = geom_of(wl)
    col = dge.h2o_colsum(g, to_dev(x.q_all_bits, "bf16"), to_dev(x.k_bits, "bf16"))
    idx, nk = dge.select_topb(g, col, 1, wl.n_recent, wl.budget - wl.n_recent)
    torch.cuda.synchronize()
    got = col.cpu().numpy()
    N = wl.cached_lens[0]
    assert np.allclose(got.sum(1), N, rtol=1e-4)
    G = wl.group
    for h in (0, 5):
        qs = x.q_all[h * G:(h + 1) * G]
        want = oracle.h2o_colsum(qs, x.k[h:h + 1], wl.kv_offsets, G, 1)[0]
        check_scores(got[h], want, f"h2o c5 head {h}")
        ref_idx = oracle.h2o_select(want, wl.budget, wl.n_recent)
        t = np.sort(want[:N - wl.n_recent])[::-1][len(ref_idx) - 1]
        gi = set(idx[0, h].cpu().numpy().tolist())
        assert len(gi) == wl.budget - wl.n_recent
        must = set(np.nonzero(want[:N - wl.n_recent] > t * (1 + 1e-3))[0].tolist())
        never = set(np.nonzero(want[:N - wl.n_recent] < t * (1 - 1e-3))[0].tolist())
        assert must <= gi and not (never & gi)


# ------------------------------------------------------------------------------------------
# Attention over the compacted cache (continuation check, Eq. 1 / eviction-mass equation)
# ------------------------------------------------------------------------------------------
def _evicted_cache(wl, x, g):
    """GPU eviction of one layer: (idx, n_kept, k_c, v_c) on the device."""
    n_tail = wl.window + wl.k_draft
    n_sel = wl.budget - wl.window
    q, k, v = to_dev(x.q_bits, wl.dtype), to_dev(x.k_bits, wl.dtype), to_dev(x.v_bits, wl.dtype)
    raw = dge.score(g, dge.ROWS_WINDOW_DRAFT, q, k)
    idx, nk, kc, vc = dge.select_compact(g, raw, wl.pool, n_tail, n_sel, k, v)
    torch.cuda.synchronize()
    return idx, nk, kc, vc, k, v, n_sel, n_tail


def _host_f64(t, dtype):
    t = t.cpu()
    if dtype == "bf16":
        return di.bf16_bits_to_f32(t.view(torch.int16).numpy().view(np.uint16)).astype(np.float64)
    return t.numpy().astype(np.float64)


def _check_att(got_o, got_l, want_o, want_l, what):
    got_o, got_l = got_o.cpu().numpy().astype(np.float64), got_l.cpu().numpy().astype(np.float64)
    fin = np.isfinite(want_l)
    assert np.array_equal(fin, np.isfinite(got_l)), f"{what}: attended-nothing rows differ"
    lerr = float(np.abs(got_l[fin] - want_l[fin]).max()) if fin.any() else 0.0
    oerr = float(np.abs(got_o - want_o).max())
    _log(f"  {what}: max |lse err| {lerr:.2e}, max |out err| {oerr:.2e}")
    assert lerr <= 1e-4, f"{what}: lse error {lerr}"
    assert np.all(np.abs(got_o - want_o) <= 1e-4 + 1e-3 * np.abs(want_o)), f"{what}: output error {oerr}"


ATT_CASES = {
    "c2_700": di.small_variant("c2", [700]),
    "ragged": di.small_variant("c2", [300, 517, 1029, 70]),
    "f32_d64": di.WORKLOADS["c1"],
}


@pytest.mark.parametrize("case", list(ATT_CASES))
def test_cache_attention_parity(case):
    wl = ATT_CASES[case]
    _log(f"cache attention parity {case} lens={wl.prompt_lens}")
    x = di.make_layer(wl)
    g = geom_of(wl)
    idx, nk, kc, vc, _, _, n_sel, n_tail = _evicted_cache(wl, x, g)
    kc64, vc64 = _host_f64(kc, wl.dtype), _host_f64(vc, wl.dtype)
    n_kept = nk.cpu().numpy()[:wl.batch]
    # decode queries (positions N_b, N_b + 1, N_b + 2: every kept row visible)
    rng = np.random.default_rng(77)
    qd = rng.standard_normal((wl.n_q_heads, wl.batch * 3, wl.head_dim)).astype(np.float32)
    qd_bits = di.f32_to_bf16_bits(qd) if wl.dtype == "bf16" else qd
    qd64 = di.bf16_bits_to_f32(qd_bits).astype(np.float64) if wl.dtype == "bf16" else qd.astype(np.float64)
    out, lse = dge.cache_attention(g, to_dev(qd_bits, wl.dtype), 3, 0, kc, vc, n_sel, n_tail, nk)
    torch.cuda.synchronize()
    wo, wlse = oracle.cache_attention(qd64, kc64, vc64, n_kept, n_tail, 0, wl.n_q_heads, wl.n_kv_heads)
    _check_att(out, lse, wo, wlse, f"{case} decode")
    # the scoring rows themselves (causal inside the tail)
    out, lse = dge.cache_attention(g, to_dev(x.q_bits, wl.dtype), n_tail, n_tail, kc, vc, n_sel,
                                   n_tail, nk)
    torch.cuda.synchronize()
    wo, wlse = oracle.cache_attention(x.q, kc64, vc64, n_kept, n_tail, n_tail, wl.n_q_heads,
                                      wl.n_kv_heads)
    _check_att(out, lse, wo, wlse, f"{case} scoring rows")


def test_cache_attention_eq1_and_evicted_mass():
    """Eq. 1 on GPU outputs alone (keep-all, kept and evicted compactions of the same
    layer), and the scoring rows' evicted mass rho_q against the oracle's."""
    wl = di.small_variant("c2", [900, 1400])
    _log("cache attention Eq. 1 decomposition and evicted mass")
    x = di.make_layer(wl)
    g = geom_of(wl)
    idx, nk, kc, vc, k, v, n_sel, n_tail = _evicted_cache(wl, x, g)
    C = [n - n_tail for n in wl.cached_lens]
    n_kept = nk.cpu().numpy()[:wl.batch]
    idx_h = idx.cpu().numpy()
    # keep-all compaction and the complement (evicted rows only, no tail)
    n_all = max(C)
    idx_all = np.full((wl.batch, wl.n_kv_heads, n_all), -1, np.int32)
    n_ev = max(C[b] - int(n_kept[b]) for b in range(wl.batch))
    idx_ev = np.full((wl.batch, wl.n_kv_heads, n_ev), -1, np.int32)
    for b in range(wl.batch):
        for h in range(wl.n_kv_heads):
            idx_all[b, h, :C[b]] = np.arange(C[b])
            ev = np.setdiff1d(np.arange(C[b]), idx_h[b, h, :n_kept[b]])
            idx_ev[b, h, :len(ev)] = ev
    nk_all = torch.tensor(C, dtype=torch.int32, device=DEV)
    nk_ev = torch.tensor([C[b] - int(n_kept[b]) for b in range(wl.batch)], dtype=torch.int32,
                         device=DEV)
    kf, vf = dge.compact(g, torch.from_numpy(idx_all).to(DEV), nk_all, n_all, n_tail, k, v)
    ke, ve = dge.compact(g, torch.from_numpy(idx_ev).to(DEV), nk_ev, n_ev, 0, k, v)
    rng = np.random.default_rng(78)
    qd = di.f32_to_bf16_bits(rng.standard_normal((wl.n_q_heads, wl.batch * 2, wl.head_dim)).astype(np.float32))
    qdd = to_dev(qd, "bf16")
    o_f, l_f = dge.cache_attention(g, qdd, 2, 0, kf, vf, n_all, n_tail, nk_all)
    o_r, l_r = dge.cache_attention(g, qdd, 2, 0, kc, vc, n_sel, n_tail, nk)
    o_e, l_e = dge.cache_attention(g, qdd, 2, 0, ke, ve, n_ev, 0, nk_ev)
    torch.cuda.synchronize()
    o_f, l_f, o_r, l_r, o_e, l_e = (t.cpu().double().numpy() for t in (o_f, l_f, o_r, l_r, o_e, l_e))
    m = 1.0 - np.exp(l_r - l_f)
    recon = (1 - m)[..., None] * o_r + m[..., None] * o_e
    err_o = float(np.abs(o_f - recon).max())
    err_l = float(np.abs(l_f - np.logaddexp(l_r, l_e)).max())
    _log(f"  Eq. 1: max |o_full - ((1-m) o_R + m o_E)| {err_o:.2e}; log-partition {err_l:.2e}; "
         f"evicted mass of the decode queries in [{m.min():.3g}, {m.max():.3g}]")
    assert err_o < 1e-4 and err_l < 1e-4
    # evicted mass rho_q of the scoring rows (observation queries of the matching loss)
    qs = to_dev(x.q_bits, "bf16")
    _, lf_s = dge.cache_attention(g, qs, n_tail, n_tail, kf, vf, n_all, n_tail, nk_all)
    _, lr_s = dge.cache_attention(g, qs, n_tail, n_tail, kc, vc, n_sel, n_tail, nk)
    torch.cuda.synchronize()
    rho = 1.0 - np.exp(lr_s.cpu().double().numpy() - lf_s.cpu().double().numpy())
    kc64, vc64 = _host_f64(kc, "bf16"), _host_f64(vc, "bf16")
    _, w_r = oracle.cache_attention(x.q, kc64, vc64, n_kept, n_tail, n_tail, wl.n_q_heads, wl.n_kv_heads)
    w_f = oracle.scoring_row_lse(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads, wl.window,
                                 wl.k_draft)
    rho_want = 1.0 - np.exp(w_r - w_f)
    err = float(np.abs(rho - rho_want).max())
    _log(f"  scoring rows: evicted mass max |err| {err:.2e}; matching loss "
         f"{float(np.mean(-np.log1p(-rho))):.4f} (oracle {float(np.mean(-np.log1p(-rho_want))):.4f})")
    assert err < 2e-4


MASS_CASES = {
    "c2_two_seqs": (di.small_variant("c2", [900, 1400]), None),
    "c1_f32_d64": (di.WORKLOADS["c1"], None),
    "c4_length": (di.small_variant("c4", [32768 - 2]), None),
    "keep_all": (di.small_variant("c2", [300, 500]), 2000),
}


@pytest.mark.parametrize("case", list(MASS_CASES))
def test_score_with_lse_and_evicted_mass_vs_oracle(case):
    """dge_score_with_lse's row normalisers against the oracle's log-partitions, its raw
    scores bit-identical to dge_score's; dge_evicted_mass on the GPU's own compaction
    against the oracle's rho_q, beta and attention-matching loss (Eq. match) computed
    directly from the evicted keys of the full cache."""
    wl, budget = MASS_CASES[case]
    budget = wl.budget if budget is None else budget
    _log(f"score_with_lse + evicted_mass {case}: lens={wl.prompt_lens} B={budget}")
    x = di.make_layer(wl)
    g = geom_of(wl)
    q, k, v = to_dev(x.q_bits, wl.dtype), to_dev(x.k_bits, wl.dtype), to_dev(x.v_bits, wl.dtype)
    n_tail, n_sel = wl.window + wl.k_draft, budget - wl.window
    raw, row_lse = dge.score_with_lse(g, dge.ROWS_WINDOW_DRAFT, q, k)
    raw_ref = dge.score(g, dge.ROWS_WINDOW_DRAFT, q, k)
    idx, nk, kc, vc = dge.select_compact(g, raw, wl.pool, n_tail, n_sel, k, v)
    rho, beta, lm = dge.evicted_mass(g, q, n_tail, n_tail, kc, n_sel, n_tail, nk, row_lse)
    torch.cuda.synchronize()
    assert torch.equal(raw.view(torch.int32), raw_ref.view(torch.int32))
    want_lse = oracle.scoring_row_lse(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads,
                                      wl.window, wl.k_draft)
    lerr = float(np.abs(row_lse.cpu().numpy().astype(np.float64) - want_lse).max())
    _log(f"  row log-partitions: max |err| {lerr:.2e}")
    assert lerr <= 1e-4
    idx_h, nk_h = idx.cpu().numpy(), nk.cpu().numpy()
    kept = {(b, h): idx_h[b, h, :nk_h[b]] for b in range(wl.batch) for h in range(wl.n_kv_heads)}
    w_rho, w_beta, w_lm = oracle.eviction_diagnostics(x.q, x.k, wl.kv_offsets, wl.n_q_heads,
                                                      wl.n_kv_heads, kept, n_tail, n_tail)
    g_rho = rho.cpu().numpy().astype(np.float64)
    g_beta, g_lm = beta.cpu().numpy().astype(np.float64), lm.cpu().numpy().astype(np.float64)
    e_rho = float(np.abs(g_rho - w_rho).max())
    e_beta = float(np.abs(g_beta - w_beta).max())
    e_lm = float(np.abs(g_lm - w_lm).max())
    _log(f"  rho max |err| {e_rho:.2e}, beta {e_beta:.2e}, L_match {e_lm:.2e}; "
         f"beta in [{w_beta.min():.3g}, {w_beta.max():.3g}], L_match mean {w_lm.mean():.4f}")
    # rho is a difference of two float32 log-partitions: absolute bound, plus 1e-3 relative
    # on the loss (which grows as rho approaches 1)
    assert e_rho <= 1e-4 and e_beta <= 1e-4
    assert (np.abs(g_lm - w_lm) <= 1e-4 + 1e-3 * np.abs(w_lm)).all()
    if case == "keep_all":
        assert w_rho.max() == 0 and g_rho.max() <= 1e-5


# ----------------------------------------------------------------------------------
# Retained-set contiguity (dge_retained_runs) against the oracle: exact counts, and the
# float32 mean n_kept / runs
# ----------------------------------------------------------------------------------
def _runs_check(geom, idx, n_kept, what):
    runs, mean = dge.retained_runs(geom, torch.from_numpy(idx).to(DEV),
                                   torch.from_numpy(n_kept).to(DEV))
    torch.cuda.synchronize()
    runs, mean = runs.cpu().numpy(), mean.cpu().numpy()
    for b in range(idx.shape[0]):
        for h in range(idx.shape[1]):
            n = int(min(max(n_kept[b], 0), idx.shape[2]))
            want_runs, want_mean = oracle.retained_runs(idx[b, h, :n])
            assert runs[b, h] == want_runs, (what, b, h, runs[b, h], want_runs)
            assert mean[b, h] == np.float32(n / want_runs if want_runs else 0.0), (what, b, h)
    return runs, mean


def test_retained_runs_synthetic():
    _log("retained runs: synthetic index sets")
    rng = np.random.default_rng(29)
    n_select = 700
    g = dge.Geometry(8, 4, 128, 8, 2, [900, 1000, 800, 1200], device=DEV)
    idx = np.full((4, 4, n_select), -1, np.int32)
    n_kept = np.array([n_select, 0, 350, 1], np.int32)
    for h in range(4):
        idx[0, h] = np.arange(n_select) + 5 * h                       # one run
        idx[2, h, :350] = np.arange(0, 700, 2)                         # 350 runs of one
        idx[3, h, :1] = 17 + h
    # random ascending subsets, including a row whose kept prefix is shorter than the row
    for h in range(4):
        pick = np.sort(rng.choice(1100, n_select, replace=False)).astype(np.int32)
        idx[1, h] = pick
    _runs_check(g, idx, n_kept, "structured")
    n_kept2 = np.array([n_select, 600, 350, 1], np.int32)
    _runs_check(g, idx, n_kept2, "random subsets")


@pytest.mark.parametrize("pool", [1, 7])
def test_retained_runs_on_gpu_selection(pool):
    wl = di.WORKLOADS["c2"]
    _log(f"retained runs on the c2 selection, pool {pool}")
    x = di.make_layer(wl)
    g = geom_of(wl)
    out = dge.evict_layer(g, to_dev(x.q_bits, "bf16"), to_dev(x.k_bits, "bf16"),
                          to_dev(x.v_bits, "bf16"), wl.budget, pool)
    torch.cuda.synchronize()
    idx = out["idx"].cpu().numpy().astype(np.int32)
    n_kept = out["n_kept"].cpu().numpy().astype(np.int32)[: g.batch]
    runs, mean = _runs_check(g, idx, n_kept, f"pool {pool}")
    _log(f"  mean run length per head: {np.round(mean[0], 2).tolist()}")


# ----------------------------------------------------------------------------------
# Select + compact over several layers in one launch: bit-identical to one
# dge_select_compact call per layer slice
# ----------------------------------------------------------------------------------
LAYER_CASES = {
    # name: (lens, H_kv, head_dim, dtype, n_select per layer, pool, n_tail, score kind)
    "ragged_budgets": ((3000, 700), 4, 128, "bf16", [600, 64, 0, 2000], 7, 34, "plateau"),
    "pool5_f32": ((1500, 260, 900), 2, 64, "f32", [100, 250, 17], 5, 10, "ints"),
    "no_pool_ulps": ((5000,), 8, 128, "bf16", [480, 2016, 1000], 1, 34, "ulps"),
    "wide_pool": ((2000,), 2, 128, "bf16", [300, 40], 19, 34, "continuous"),     # per-layer launches
    "beyond_register_path": ((33000, 400), 2, 128, "bf16", [100, 2016], 7, 34, "plateau"),
    "many_layers": ((200, 90), 1, 64, "f32", [(7 * l) % 150 for l in range(130)], 3, 8, "continuous"),
}


@pytest.mark.parametrize("case", list(LAYER_CASES))
def test_select_compact_layers_vs_oracle(case):
    """dge_select_compact_layers (every layer's pool, top-B'_l and gather in one launch)
    against the oracle layer by layer: indices bit-exact given the same fp32 scores,
    n_kept exact, compacted K/V byte-exact (Alg. 1 steps B-C for all layers)."""
    lens, H, d, dtype, n_sel, pool, n_tail, kind = LAYER_CASES[case]
    _log(f"select_compact_layers vs oracle {case}: lens={lens} H={H} layers={len(n_sel)}")
    nl, T = len(n_sel), sum(lens)
    rng = np.random.default_rng(np.random.SeedSequence([7, len(case)]))
    scores_h = di.random_scores((nl * H, T), seed=len(case), kind=kind)
    if dtype == "bf16":
        kb = rng.integers(0, 1 << 16, size=(nl * H, T, d), dtype=np.uint16)
        vb = rng.integers(0, 1 << 16, size=(nl * H, T, d), dtype=np.uint16)
    else:
        kb = rng.standard_normal((nl * H, T, d), dtype=np.float32)
        vb = rng.standard_normal((nl * H, T, d), dtype=np.float32)
    g = dge.Geometry(2 * H, H, d, 0, 0, lens, dtype=dge.DGE_BF16 if dtype == "bf16" else dge.DGE_F32,
                     device=DEV)
    idx_l, nk, k_l, v_l = dge.select_compact_layers(g, torch.from_numpy(scores_h).to(DEV), pool,
                                                    n_tail, n_sel, to_dev(kb, dtype),
                                                    to_dev(vb, dtype))
    torch.cuda.synchronize()
    for l in range(nl):
        sl = slice(l * H, (l + 1) * H)
        want = oracle_select_compact(scores_h[sl], kb[sl], vb[sl], lens, H, pool, n_tail, n_sel[l])
        check_select_compact(idx_l[l], nk[l], k_l[l], v_l[l], want, n_sel[l], n_tail,
                             f"{case} layer {l}")


def test_c3_layers_score_select_compact_vs_oracle():
    """Four c3-shaped layers (32q/8kv, d 128, L 16384, each generated with its own seeds
    and planted spans) scored by one dge_score call over the layer-major cache and
    evicted by one dge_select_compact_layers launch with distinct budgets: the PyramidKV
    maximum (2048), the window only (B' = 0), keep-all, and an interior value.  Scores
    within 1e-3 of the oracle; selection by the threshold rule against the oracle's own
    scores and bit-exact given the GPU's scores; K/V byte-exact."""
    wl = di.WORKLOADS["c3"]
    budgets = [wl.budget_of_layer(0), wl.window, 20000, wl.budget_of_layer(20)]
    nl, Hq, H = len(budgets), wl.n_q_heads, wl.n_kv_heads
    _log(f"c3 layers vs oracle: budgets {budgets}")
    xs = [di.make_layer(wl, layer=l) for l in range(nl)]
    g1 = geom_of(wl)
    ga = dge.Geometry(Hq * nl, H * nl, wl.head_dim, wl.window, wl.k_draft, wl.cached_lens,
                      device=DEV)
    q = to_dev(np.concatenate([x.q_bits for x in xs]), "bf16")
    k = to_dev(np.concatenate([x.k_bits for x in xs]), "bf16")
    v = to_dev(np.concatenate([x.v_bits for x in xs]), "bf16")
    raw = dge.score(ga, dge.ROWS_WINDOW_DRAFT, q, k)
    n_tail = wl.window + wl.k_draft
    n_sel = [B - wl.window for B in budgets]
    idx_l, nk, k_l, v_l = dge.select_compact_layers(g1, raw, wl.pool, n_tail, n_sel, k, v)
    torch.cuda.synchronize()
    raw_h = raw.cpu().numpy()
    N = wl.cached_lens[0]
    C = N - n_tail
    for l, x in enumerate(xs):
        sl = slice(l * H, (l + 1) * H)
        want_raw = oracle.window_scores(x.q, x.k, wl.kv_offsets, Hq, H, wl.window, wl.k_draft)
        check_scores(raw_h[sl], want_raw, f"c3 layer {l} scores")
        want = oracle_select_compact(raw_h[sl], x.k_bits, x.v_bits, wl.cached_lens, H, wl.pool,
                                     n_tail, n_sel[l])
        check_select_compact(idx_l[l], nk[l], k_l[l], v_l[l], want, n_sel[l], n_tail,
                             f"c3 layer {l}")
        gi = idx_l[l].cpu().numpy()
        for h in range(H):
            pooled = oracle.maxpool(want_raw[h], C, wl.pool)
            check_threshold_rule(pooled, gi[0, h], n_sel[l], f"c3 layer {l} head {h}")


# ----------------------------------------------------------------------------------
# In-place compaction: the first n_kept + n_tail rows of every segment equal the
# out-of-place compaction, the rest of the segment is untouched
# ----------------------------------------------------------------------------------
INPLACE_CASES = {
    # name: (lens, H_kv, head_dim, dtype, n_select, n_tail, pool, selector)
    "ragged_bf16": ((3000, 700, 90), 4, 128, "bf16", 480, 34, 7, "topb"),
    "keep_all": ((600, 1200), 2, 128, "bf16", 5000, 34, 7, "topb"),
    "tail_only": ((800,), 2, 128, "bf16", 0, 34, 7, "topb"),
    "f32_d64": ((2500, 333), 2, 64, "f32", 300, 8, 5, "topb"),
    "streaming": ((4098, 2000), 8, 128, "bf16", 4, 1020, 1, "streaming"),
    "c4_length": ((32802,), 1, 128, "bf16", 2016, 34, 7, "topb"),
    # kept keys packed at the front: long chains of rows whose sources are other rows'
    # destinations (every second candidate from 100 on, or the first ones shifted by one)
    "near_every_second": ((9000, 5000), 2, 128, "bf16", 2016, 34, 1, "front2"),
    "near_shift_one": ((6000,), 2, 128, "bf16", 3000, 34, 1, "shift1"),
    "near_f32_d64": ((7000, 300), 2, 64, "f32", 1500, 8, 1, "front2"),
}


@pytest.mark.parametrize("case", list(INPLACE_CASES))
def test_compact_inplace_vs_oracle(case):
    """dge_compact_inplace (Alg. 1 step C as one in-place edit, temporal order kept)
    against the oracle: the selection bit-exact to the oracle's rule on the same scores
    (or the StreamingLLM closed form), the first n_kept + n_tail rows of every segment
    byte-equal to oracle.compact, the rest of the segment untouched."""
    lens, H, d, dtype, n_select, n_tail, pool, selector = INPLACE_CASES[case]
    _log(f"compact_inplace vs oracle {case}: lens={lens} H={H} sel={n_select} tail={n_tail}")
    T = sum(lens)
    rng = np.random.default_rng(np.random.SeedSequence([11, len(case)]))
    g = dge.Geometry(2 * H, H, d, 0, 0, lens, dtype=dge.DGE_BF16 if dtype == "bf16" else dge.DGE_F32,
                     device=DEV)
    if dtype == "bf16":
        kb = rng.integers(0, 1 << 16, size=(H, T, d), dtype=np.uint16)
        vb = rng.integers(0, 1 << 16, size=(H, T, d), dtype=np.uint16)
        bits = np.int16
    else:
        kb = rng.standard_normal((H, T, d), dtype=np.float32)
        vb = rng.standard_normal((H, T, d), dtype=np.float32)
        bits = np.int32
    k, v = to_dev(kb, dtype), to_dev(vb, dtype)
    offs = np.concatenate([[0], np.cumsum(lens)])
    if selector in ("topb", "front2", "shift1"):
        scores_h = di.random_scores((H, T), seed=len(case), kind="plateau")
        for b, N in enumerate(lens):
            seg = scores_h[:, offs[b]:offs[b + 1]]
            if selector == "front2":      # the kept keys: 100, 102, 104, ...
                seg[:, 100:100 + 2 * n_select:2] += 10.0
            elif selector == "shift1":    # the kept keys: 1 .. n_select
                seg[:, 1:1 + n_select] += 10.0
        idx, nk = dge.select_topb(g, torch.from_numpy(scores_h).to(DEV), pool, n_tail, n_select)
        want = oracle_select_compact(scores_h, kb, vb, lens, H, pool, n_tail, n_select)
    else:
        idx, nk = dge.select_streaming(g, n_select, n_tail)
        want = {}
        for b, N in enumerate(lens):
            sel = oracle.streaming_select(N, n_select, n_tail)
            for h in range(H):
                seg = slice(offs[b], offs[b + 1])
                want[(b, h)] = (sel,) + oracle.compact(kb[h, seg], vb[h, seg], sel, N - n_tail)
    dge.compact_inplace(g, idx, nk, n_select, n_tail, k, v)
    torch.cuda.synchronize()
    idx, nk = idx.cpu().numpy(), nk.cpu().numpy()
    kg = k.cpu().view(torch.int16 if dtype == "bf16" else torch.int32).numpy()
    vg = v.cpu().view(torch.int16 if dtype == "bf16" else torch.int32).numpy()
    for b, N in enumerate(lens):
        for h in range(H):
            sel, ko, vo = want[(b, h)]
            assert nk[b] == len(sel), (case, b)
            assert np.array_equal(idx[b, h, :len(sel)], sel), (case, b, h)
            m = len(sel) + n_tail
            s0 = offs[b]
            assert np.array_equal(kg[h, s0:s0 + m], ko.view(bits)), (case, b, h, "k")
            assert np.array_equal(vg[h, s0:s0 + m], vo.view(bits)), (case, b, h, "v")
            assert np.array_equal(kg[h, s0 + m:s0 + N], kb[h, s0 + m:s0 + N].view(bits)), (case, b, h)
            assert np.array_equal(vg[h, s0 + m:s0 + N], vb[h, s0 + m:s0 + N].view(bits)), (case, b, h)


# ----------------------------------------------------------------------------------
# More sequences than travel inline in the kernel arguments (16): every kernel reads the
# device offsets array
# ----------------------------------------------------------------------------------
BIG_BATCH = tuple(int(n) for n in np.random.default_rng(np.random.SeedSequence([18, 0])).integers(40, 700, size=18))


def test_batch_of_18_sequences_vs_oracle():
    """18 ragged sequences through every entry point that takes the sequence offsets:
    dge_score, dge_select_compact, dge_select_topb + dge_compact, dge_compact_inplace,
    dge_select_streaming, dge_retained_runs, dge_cache_attention and dge_h2o_colsum,
    each against the oracle."""
    wl = di.small_variant("c2", BIG_BATCH)
    _log(f"batch of {wl.batch} sequences, lens {BIG_BATCH}")
    x = di.make_layer(wl)
    g = geom_of(wl)
    q, k, v = to_dev(x.q_bits, "bf16"), to_dev(x.k_bits, "bf16"), to_dev(x.v_bits, "bf16")
    n_tail, n_sel = wl.window + wl.k_draft, 100
    raw = dge.score(g, dge.ROWS_WINDOW_DRAFT, q, k)
    torch.cuda.synchronize()
    raw_h = raw.cpu().numpy()
    want_raw = oracle.window_scores(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads,
                                    wl.window, wl.k_draft)
    check_scores(raw_h, want_raw, "batch 18 scores")
    want = oracle_select_compact(raw_h, x.k_bits, x.v_bits, wl.cached_lens, wl.n_kv_heads,
                                 wl.pool, n_tail, n_sel)
    idx, nk, kc, vc = dge.select_compact(g, raw, wl.pool, n_tail, n_sel, k, v)
    torch.cuda.synchronize()
    check_select_compact(idx, nk, kc, vc, want, n_sel, n_tail, "batch 18 fused")
    gi = idx.cpu().numpy()
    offs = wl.kv_offsets
    for b, N in enumerate(wl.cached_lens):
        for h in range(wl.n_kv_heads):
            pooled = oracle.maxpool(want_raw[h, offs[b]:offs[b + 1]], N - n_tail, wl.pool)
            check_threshold_rule(pooled, gi[b, h], n_sel, f"batch 18 seq {b} head {h}")
    idx2, nk2 = dge.select_topb(g, raw, wl.pool, n_tail, n_sel)
    kc2, vc2 = dge.compact(g, idx2, nk2, n_sel, n_tail, k, v)
    torch.cuda.synchronize()
    check_select_compact(idx2, nk2, kc2, vc2, want, n_sel, n_tail, "batch 18 separate")
    # in place, on copies of the cache
    kw, vw = k.clone(), v.clone()
    dge.compact_inplace(g, idx2, nk2, n_sel, n_tail, kw, vw)
    torch.cuda.synchronize()
    kg = kw.cpu().view(torch.int16).numpy()
    vg = vw.cpu().view(torch.int16).numpy()
    for (b, h), (sel, ko, vo) in want.items():
        m = len(sel) + n_tail
        assert np.array_equal(kg[h, offs[b]:offs[b] + m], ko.view(np.int16)), (b, h)
        assert np.array_equal(vg[h, offs[b]:offs[b] + m], vo.view(np.int16)), (b, h)
    # StreamingLLM and the run-length diagnostic
    sidx, snk = dge.select_streaming(g, 4, 40)
    torch.cuda.synchronize()
    for b, N in enumerate(wl.cached_lens):
        s_want = oracle.streaming_select(N, 4, 40)
        assert snk[b].item() == len(s_want)
        for h in range(wl.n_kv_heads):
            assert sidx[b, h, :len(s_want)].cpu().numpy().tolist() == s_want.tolist()
    _runs_check(g, gi.astype(np.int32), nk.cpu().numpy().astype(np.int32)[:wl.batch], "batch 18")
    # attention over the compacted caches: decode queries and the scoring rows
    kc64, vc64 = _host_f64(kc, "bf16"), _host_f64(vc, "bf16")
    n_kept = nk.cpu().numpy()[:wl.batch]
    out, lse = dge.cache_attention(g, q, n_tail, n_tail, kc, vc, n_sel, n_tail, nk)
    torch.cuda.synchronize()
    wo, wlse = oracle.cache_attention(x.q, kc64, vc64, n_kept, n_tail, n_tail, wl.n_q_heads,
                                      wl.n_kv_heads)
    _check_att(out, lse, wo, wlse, "batch 18 scoring rows")
    # H2O accumulated attention over every cached row of the 18 sequences
    wh = di.small_variant("c5", BIG_BATCH)
    xh = di.make_layer(wh, with_v=False)
    gh = geom_of(wh)
    col = dge.h2o_colsum(gh, to_dev(xh.q_all_bits, "bf16"), to_dev(xh.k_bits, "bf16"))
    torch.cuda.synchronize()
    want_col = oracle.h2o_colsum(xh.q_all, xh.k, wh.kv_offsets, wh.n_q_heads, wh.n_kv_heads)
    check_scores(col.cpu().numpy(), want_col, "batch 18 h2o colsum")


MANY_SEQS = tuple(int(n) for n in np.random.default_rng(np.random.SeedSequence([520, 0])).integers(100, 300, size=520))


def test_score_launch_of_many_workgroups_vs_oracle():
    """A launch with more than 4096 colsum workgroups (520 ragged sequences x 8 KV heads,
    one chunk each), which takes the colsum instance compiled for three wavefronts per
    SIMD: dge_score, dge_score_with_lse and dge_score_lse (the oracle's row LSEs) against
    the oracle on every sequence."""
    wl = di.small_variant("c2", MANY_SEQS)
    _log(f"score launch of {wl.batch} sequences x {wl.n_kv_heads} heads, lens {min(MANY_SEQS)}..{max(MANY_SEQS)}")
    x = di.make_layer(wl, with_v=False)
    g = geom_of(wl)
    q, k = to_dev(x.q_bits, "bf16"), to_dev(x.k_bits, "bf16")
    want_raw = oracle.window_scores(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads,
                                    wl.window, wl.k_draft)
    want_lse = oracle.scoring_row_lse(x.q, x.k, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads,
                                      wl.window, wl.k_draft)
    raw = dge.score(g, dge.ROWS_WINDOW_DRAFT, q, k)
    torch.cuda.synchronize()
    check_scores(raw.cpu().numpy(), want_raw, "many workgroups, score")
    raw2, lse = dge.score_with_lse(g, dge.ROWS_WINDOW_DRAFT, q, k)
    torch.cuda.synchronize()
    check_scores(raw2.cpu().numpy(), want_raw, "many workgroups, score_with_lse")
    lse_h = lse.cpu().numpy().astype(np.float64)
    lerr = np.abs(lse_h - want_lse)
    _log(f"  row lse: max abs err {lerr.max():.2e}")
    assert (lerr <= 1e-4 + 1e-6 * np.abs(want_lse)).all()
    raw3 = dge.score_lse(g, dge.ROWS_WINDOW_DRAFT, q, k,
                         torch.from_numpy(want_lse.astype(np.float32)).to(DEV))
    torch.cuda.synchronize()
    check_scores(raw3.cpu().numpy(), want_raw, "many workgroups, score_lse")


# ----------------------------------------------------------------------------------
# Repeated-KV layout (every KV head copied to the G query heads of its group, scored and
# selected per query head, no group mean): the geometry with G = 1 over the repeated cache
# ----------------------------------------------------------------------------------
def test_repeated_kv_layout_per_query_head():
    wl = di.small_variant("c2", [700, 1300])
    _log("repeated-KV layout: per-query-head scores and selection")
    x = di.make_layer(wl, with_v=True)
    G = wl.n_q_heads // wl.n_kv_heads
    k_rep = np.repeat(x.k_bits, G, axis=0)
    v_rep = np.repeat(x.v_bits, G, axis=0)
    g1 = dge.Geometry(wl.n_q_heads, wl.n_q_heads, wl.head_dim, wl.window, wl.k_draft,
                      wl.cached_lens, device=DEV)
    kd, vd = to_dev(k_rep, "bf16"), to_dev(v_rep, "bf16")
    raw = dge.score(g1, oracle.ROWS_WINDOW_DRAFT, to_dev(x.q_bits, "bf16"), kd)
    torch.cuda.synchronize()
    want = oracle.window_scores(x.q, np.repeat(x.k, G, axis=0), wl.kv_offsets, wl.n_q_heads,
                                wl.n_q_heads, wl.window, wl.k_draft)
    got = raw.cpu().numpy()
    check_scores(got, want, "per-query-head scores")
    # per-query-head top-B' and compaction on the repeated cache, bit-exact given the scores
    n_tail = wl.window + wl.k_draft
    n_sel = wl.budget - wl.window
    idx, nk, k_out, v_out = dge.select_compact(g1, raw, wl.pool, n_tail, n_sel, kd, vd)
    torch.cuda.synchronize()
    idx = idx.cpu().numpy()
    offs = wl.kv_offsets
    for b, N in enumerate(wl.cached_lens):
        C = N - n_tail
        for h in range(wl.n_q_heads):
            pooled = oracle.maxpool(got[h, offs[b]:offs[b + 1]].astype(np.float64), C, wl.pool)
            sel = oracle.select_topb(pooled, n_sel)
            assert np.array_equal(idx[b, h, :len(sel)], sel), (b, h)
            rows = np.concatenate([sel, np.arange(C, N)])
            ref_k = k_rep[h, offs[b] + rows]
            assert np.array_equal(k_out[b, h, :len(rows)].view(torch.int16).cpu().numpy(),
                                  ref_k.view(np.int16)), (b, h)


# ----------------------------------------------------------------------------------
# Rotary position embedding of the query/key rows (dge_rope) against the oracle
# ----------------------------------------------------------------------------------
@pytest.mark.parametrize("case", ["bf16_d128", "f32_d64", "bf16_long_positions"])
def test_rope_parity(case):
    _log(f"rope parity {case}")
    rng = np.random.default_rng(np.random.SeedSequence([31, len(case)]))
    H, n, d, dt = {"bf16_d128": (8, 300, 128, "bf16"), "f32_d64": (4, 257, 64, "f32"),
                   "bf16_long_positions": (2, 130, 128, "bf16")}[case]
    x = rng.standard_normal((H, n, d), dtype=np.float32) * 2.0
    if case == "bf16_long_positions":
        pos = np.sort(rng.integers(0, 1 << 20, size=n)).astype(np.int32)
    else:
        pos = np.arange(n, dtype=np.int32) + 17
    if dt == "bf16":
        xt = torch.from_numpy(x).to(torch.bfloat16)
        x_in = xt.float().numpy().astype(np.float64)      # the stored bf16 values
        xd = xt.to(DEV)
    else:
        x_in = x.astype(np.float64)
        xd = torch.from_numpy(x).to(DEV)
    dge.rope(xd, torch.from_numpy(pos).to(DEV))
    torch.cuda.synchronize()
    got = xd.float().cpu().numpy().astype(np.float64)
    want = oracle.rope(x_in, pos)
    # one rounding to the stored type: half an ulp, plus the double-to-float step for bf16
    ulp = 2.0 ** -8 if dt == "bf16" else 2.0 ** -23
    tol = ulp * np.maximum(np.abs(want), 2.0 ** -126)
    bad = np.abs(got - want) > tol
    assert not bad.any(), (case, int(bad.sum()), float(np.abs(got - want).max()))
    # rotations keep every pair's length
    half = d // 2
    r_in = np.hypot(x_in[..., :half], x_in[..., half:])
    r_out = np.hypot(got[..., :half], got[..., half:])
    assert np.allclose(r_out, r_in, rtol=2 * ulp, atol=1e-6)


# ----------------------------------------------------------------------------------
# Query/key capture from the layer input: RoPE(x W^T) (dge_project_rope)
# ----------------------------------------------------------------------------------
PROJ_CASES = {
    # name: (n_rows, hidden, n_heads, head_dim, first position, rows checked)
    "llama_q_scoring_rows": (34, 4096, 32, 128, 26507, None),
    "llama_k_scoring_rows": (34, 4096, 8, 128, 26507, None),
    "fused_qk_weight": (34, 4096, 40, 128, 26507, None),
    "hidden_384_rows_70": (70, 384, 6, 128, 100, None),
    "split_d64_rows_10": (10, 2048, 6, 64, 3, None),
    "split_rows_64": (64, 4096, 4, 128, 1000, None),
    "d64_ragged_rows": (130, 1024, 4, 64, 0, None),
    "tiles_and_122_rows": (250, 1024, 4, 128, 5, None),
    "tiles_256_128_and_16_rows": (400, 1024, 4, 128, 7, None),
    "tiles_256_d64": (300, 512, 8, 64, 11, None),
    "one_row": (1, 128, 1, 64, 7, None),
    "h2o_all_rows_sampled": (8194, 4096, 32, 128, 0, 48),
}


@pytest.mark.parametrize("case", list(PROJ_CASES))
def test_project_rope_vs_oracle(case):
    """dge_project_rope against the float64 composition RoPE(x W^T): each output within half
    a bf16 ulp of the exact value plus the float32 accumulation bound (2^-8 |o| +
    8e-5 * sum_k |x_k| (|w_lo,k| + |w_hi,k|), the rotation mixing the two columns of a pair);
    on the 8194-row case sampled rows only."""
    n, hidden, H, d, p0, n_check = PROJ_CASES[case]
    _log(f"project_rope {case}: rows={n} hidden={hidden} heads={H} d={d}")
    rng = np.random.default_rng(np.random.SeedSequence([61, n, hidden, H]))
    xb = di.f32_to_bf16_bits(rng.standard_normal((n, hidden), dtype=np.float32))
    wb = di.f32_to_bf16_bits((rng.standard_normal((H * d, hidden)) / math.sqrt(hidden)).astype(np.float32))
    pos = (p0 + np.arange(n)).astype(np.int32)
    if case == "d64_ragged_rows":
        pos = np.sort(rng.integers(0, 1 << 17, size=n)).astype(np.int32)
    out = dge.project_rope(to_dev(xb, "bf16"), to_dev(wb, "bf16"), torch.from_numpy(pos).to(DEV), H, d)
    torch.cuda.synchronize()
    got = di.bf16_bits_to_f32(out.cpu().view(torch.int16).numpy().view(np.uint16)).astype(np.float64)
    # sampled rows: a random set plus the edges of the 128-row tiles and the last rows (the
    # rows past the last whole tile take another kernel)
    rows = np.arange(n) if n_check is None else np.unique(np.concatenate(
        [rng.choice(n, size=n_check, replace=False), [0, 127, 128, n - 131, n - 130, n - 3, n - 2, n - 1]]))
    x64 = di.bf16_bits_to_f32(xb).astype(np.float64)[rows]
    w64 = di.bf16_bits_to_f32(wb).astype(np.float64)
    want = oracle.project_rope(x64, w64, pos[rows], H, d)
    s = (np.abs(x64) @ np.abs(w64).T).reshape(len(rows), H, d).transpose(1, 0, 2)
    s_pair = np.concatenate([s[..., :d // 2] + s[..., d // 2:]] * 2, axis=-1)
    err = np.abs(got[:, rows] - want)
    tol = 2.0 ** -8 * np.abs(want) + 8e-5 * s_pair
    _log(f"  max |err| {err.max():.3e}, max err/tol {float((err / tol).max()):.3f}")
    assert (err <= tol).all(), (case, int((err > tol).sum()))
