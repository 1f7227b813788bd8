"""Pins of the float64 oracle against facts that do not come from the oracle itself.

Each test names what fixes the expected value: a worked example the paper prints,
a closed form, an invariant, a library routine that computes the same definition
independently (torch SDPA, max_pool1d, topk, logsumexp), or brute force.
CPU only.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import dge_inputs as di
import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


# ----------------------------------------------------------------------------------
# PyramidKV: the paper's five worked examples (App. "Additional analysis")
# ----------------------------------------------------------------------------------
def test_pyramid_worked_examples():
    cases = json.load(open(os.path.join(GOLDEN, "pyramidkv_worked_examples.json")))["cases"]
    for c in cases:
        Bl = oracle.pyramid_budgets(c["B"], c["w"], c["n_layers"])
        past = Bl - c["w"]
        assert len(past) == c["n_layers"]
        steps = set((past[:-1] - past[1:]).tolist())
        assert steps == {c["steps"]}, (c, past)
        if "last_layers_past" in c:
            tail = c["last_layers_past"]
            assert past[-len(tail):].tolist() == tail, (c, past)
        if "every_layer_past" in c:
            assert (past == c["every_layer_past"]).all()


# ----------------------------------------------------------------------------------
# Scoring: closed forms, invariants and an independent library implementation
# ----------------------------------------------------------------------------------
def test_score_hand_example_scale_and_mask():
    # d = 4, sqrt(d) = 2.  One draft row at position 1 sees keys 0 and 1:
    # logits 0 and (2 * ln 3) / 2 = ln 3  ->  softmax (1/4, 3/4).  A dropped 1/sqrt(d)
    # gives (1/10, 9/10); a flipped sign gives (3/4, 1/4).
    q = np.zeros((1, 1, 4)); q[0, 0, 0] = 2.0
    k = np.zeros((1, 2, 4)); k[0, 1, 0] = math.log(3.0)
    raw = oracle.window_scores(q, k, [0, 2], 1, 1, w=0, k_draft=1, mode=oracle.ROWS_DRAFT)
    assert np.allclose(raw[0], [0.25, 0.75], rtol=0, atol=1e-15)
    # A window row at position 0 (the last prompt row, L = 1) sees key 0 only.
    raw = oracle.window_scores(q, k, [0, 2], 1, 1, w=1, k_draft=1, mode=oracle.ROWS_WINDOW)
    assert raw[0].tolist() == [1.0, 0.0]


@pytest.mark.parametrize("mode", [oracle.ROWS_WINDOW_DRAFT, oracle.ROWS_DRAFT, oracle.ROWS_WINDOW])
def test_score_mass_equals_rows(mode):
    # every softmax row sums to 1, so each head's total mass is the number of scoring rows
    Hq, Hkv, d, w, kd = 8, 2, 16, 5, 3
    offs = [0, 40, 97]
    nr = oracle.scoring_rows(10, w, kd, mode)[1]
    q = _rand((Hq, 2 * nr, d), 1, 2.0)
    k = _rand((Hkv, offs[-1], d), 2, 2.0)
    raw = oracle.window_scores(q, k, offs, Hq, Hkv, w, kd, mode)
    for b in range(2):
        tot = raw[:, offs[b]:offs[b + 1]].sum(axis=1)
        assert np.allclose(tot, nr, rtol=1e-12, atol=0)


def test_repeated_kv_scores_average_to_group_scores():
    # App. "Complexity and overheads": the prototype repeats every KV head to the G query
    # heads of its group and scores per query head; the native GQA score of a KV head is
    # the mean of those G per-query-head scores (a dropped 1/G, a wrong head-to-group map
    # or a transposed repeat fails here)
    Hq, Hkv, d, w, kd = 12, 3, 16, 4, 2
    G = Hq // Hkv
    offs = [0, 37, 90]
    nr = w + kd
    q = _rand((Hq, 2 * nr, d), 5, 2.0)
    k = _rand((Hkv, offs[-1], d), 6, 2.0)
    per_head = oracle.window_scores(q, np.repeat(k, G, axis=0), offs, Hq, Hq, w, kd)
    grouped = oracle.window_scores(q, k, offs, Hq, Hkv, w, kd)
    assert per_head.shape == (Hq, offs[-1])
    assert np.allclose(per_head.reshape(Hkv, G, -1).mean(axis=1), grouped, rtol=1e-12, atol=1e-300)
    # and the per-query-head rows keep their own softmax mass (n_rows per head)
    for b in range(2):
        assert np.allclose(per_head[:, offs[b]:offs[b + 1]].sum(axis=1), nr, rtol=1e-12)


def _brute_scores(q, k, offs, Hq, Hkv, w, kd, h2o=False):
    # the definitions written out as plain Python loops with math.exp: for each scoring
    # row (or, for H2O, every cached row) a causal softmax over the sequence's keys,
    # summed into the keys' columns and divided by the group size
    G = Hq // Hkv
    d = len(k[0][0])
    T = offs[-1]
    out = [[0.0] * T for _ in range(Hkv)]
    for b in range(len(offs) - 1):
        s0, N = offs[b], offs[b + 1] - offs[b]
        if h2o:
            rows = [(p, s0 + p) for p in range(N)]            # (position, row of q)
        else:
            nr = w + kd
            rows = [(N - nr + r, b * nr + r) for r in range(nr)]
        for hq in range(Hq):
            h = hq // G
            for p, qi in rows:
                logits = [sum(q[hq][qi][e] * k[h][s0 + j][e] for e in range(d)) / math.sqrt(d)
                          for j in range(p + 1)]
                top = max(logits)
                ex = [math.exp(x - top) for x in logits]
                z = sum(ex)
                for j in range(p + 1):
                    out[h][s0 + j] += ex[j] / z / G
    return np.array(out)


def test_scores_match_plain_python_loops():
    Hq, Hkv, d, w, kd = 4, 2, 5, 3, 2
    offs = [0, 9, 23]
    q = _rand((Hq, 2 * (w + kd), d), 11, 1.5)
    k = _rand((Hkv, offs[-1], d), 12, 1.5)
    want = _brute_scores(q.tolist(), k.tolist(), offs, Hq, Hkv, w, kd)
    got = oracle.window_scores(q, k, offs, Hq, Hkv, w, kd)
    assert np.allclose(got, want, rtol=1e-12, atol=1e-15)


def test_h2o_colsum_matches_plain_python_loops():
    Hq, Hkv, d = 4, 2, 5
    offs = [0, 11, 20]
    q = _rand((Hq, offs[-1], d), 13, 1.5)
    k = _rand((Hkv, offs[-1], d), 14, 1.5)
    want = _brute_scores(q.tolist(), k.tolist(), offs, Hq, Hkv, 0, 0, h2o=True)
    got = oracle.h2o_colsum(q, k, offs, Hq, Hkv)
    assert np.allclose(got, want, rtol=1e-12, atol=1e-15)


def test_score_uniform_closed_form():
    # identical keys: a row at position p spreads 1/(p+1) over keys 0..p, so
    # raw[j] = sum_{p = max(j, p0)}^{N-1} 1/(p+1)  (the group mean of equal heads)
    Hq, Hkv, d, w, kd, N = 4, 1, 8, 6, 2, 30
    q = _rand((Hq, w + kd, d), 3)
    k = np.tile(_rand((1, 1, d), 4), (Hkv, N, 1))
    raw = oracle.window_scores(q, k, [0, N], Hq, Hkv, w, kd)
    p0 = N - w - kd
    want = [sum(1.0 / (p + 1) for p in range(max(j, p0), N)) for j in range(N)]
    assert np.allclose(raw[0], want, rtol=1e-13, atol=0)


def _sdpa_probs(qrows, keys, positions):
    # torch's SDPA with V = identity returns the attention probabilities themselves,
    # with its own default scale 1/sqrt(d) and the boolean mask j <= p.
    Q = torch.tensor(qrows)[None, None]
    K = torch.tensor(keys)[None, None]
    V = torch.eye(keys.shape[0], dtype=torch.float64)[None, None]
    mask = torch.arange(keys.shape[0])[None, :] <= torch.tensor(positions)[:, None]
    return torch.nn.functional.scaled_dot_product_attention(Q, K, V, attn_mask=mask)[0, 0].numpy()


@pytest.mark.parametrize("mode", [oracle.ROWS_WINDOW_DRAFT, oracle.ROWS_DRAFT, oracle.ROWS_WINDOW])
def test_score_matches_torch_sdpa(mode):
    Hq, Hkv, d, w, kd = 6, 3, 32, 7, 2
    offs = [0, 23, 64]
    G = Hq // Hkv
    nr = oracle.scoring_rows(10, w, kd, mode)[1]
    q = _rand((Hq, 2 * nr, d), 5, 1.5)
    k = _rand((Hkv, offs[-1], d), 6, 1.5)
    raw = oracle.window_scores(q, k, offs, Hq, Hkv, w, kd, mode)
    for b in range(2):
        s0, N = offs[b], offs[b + 1] - offs[b]
        p0, _ = oracle.scoring_rows(N, w, kd, mode)
        pos = np.arange(p0, p0 + nr)
        for h in range(Hkv):
            cols = [_sdpa_probs(q[h * G + g, b * nr:(b + 1) * nr], k[h, s0:s0 + N], pos).sum(0)
                    for g in range(G)]
            assert np.allclose(raw[h, s0:s0 + N], np.mean(cols, axis=0), rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("mode", [oracle.ROWS_WINDOW_DRAFT, oracle.ROWS_DRAFT, oracle.ROWS_WINDOW])
def test_scoring_row_lse_matches_torch_logsumexp(mode):
    Hq, Hkv, d, w, kd = 4, 2, 16, 5, 2
    offs = [0, 20, 51]
    G = Hq // Hkv
    nr = oracle.scoring_rows(10, w, kd, mode)[1]
    q = _rand((Hq, 2 * nr, d), 24, 2.0)
    k = _rand((Hkv, offs[-1], d), 25, 2.0)
    lse = oracle.scoring_row_lse(q, k, offs, Hq, Hkv, w, kd, mode)
    for b in range(2):
        s0, N = offs[b], offs[b + 1] - offs[b]
        p0, _ = oracle.scoring_rows(N, w, kd, mode)
        for hq in range(Hq):
            Q = torch.tensor(q[hq, b * nr:(b + 1) * nr])
            K = torch.tensor(k[hq // G, s0:s0 + N])
            x = (Q @ K.T) / math.sqrt(d)
            mask = torch.arange(N)[None, :] > (p0 + torch.arange(nr))[:, None]
            want = torch.logsumexp(x.masked_fill(mask, float("-inf")), dim=1).numpy()
            assert np.allclose(lse[hq, b * nr:(b + 1) * nr], want, rtol=1e-13)


def test_dgew_timing_invariance():
    # DGE-W keeps the window scorer and only moves the eviction step: the window rows'
    # scores of the prompt keys do not change when k draft rows are appended to the cache
    Hq, Hkv, d, w, L, kd = 4, 2, 16, 8, 50, 3
    q = _rand((Hq, w, d), 7)
    k_prompt = _rand((Hkv, L, d), 8)
    k_full = np.concatenate([k_prompt, _rand((Hkv, kd, d), 9)], axis=1)
    a = oracle.window_scores(q, k_prompt, [0, L], Hq, Hkv, w, 0, oracle.ROWS_WINDOW)
    b = oracle.window_scores(q, k_full, [0, L + kd], Hq, Hkv, w, kd, oracle.ROWS_WINDOW)
    assert np.array_equal(a, b[:, :L])
    assert (b[:, L:] == 0).all()


# ----------------------------------------------------------------------------------
# Pooling and selection
# ----------------------------------------------------------------------------------
@pytest.mark.parametrize("kappa", [1, 3, 5, 7])
def test_maxpool_matches_torch(kappa):
    x = np.random.default_rng(10 + kappa).random(57)
    C = 50
    want = torch.nn.functional.max_pool1d(torch.tensor(x[:C])[None, None], kappa, 1, kappa // 2)[0, 0]
    assert np.array_equal(oracle.maxpool(x, C, kappa), want.numpy())


def test_select_matches_torch_topk_tie_free():
    rng = np.random.default_rng(11)
    for C, n in [(100, 10), (257, 64), (64, 64), (30, 100)]:
        s = rng.random(C)
        idx = oracle.select_topb(s, n)
        want = torch.topk(torch.tensor(s), min(n, C)).indices.numpy()
        assert set(idx.tolist()) == set(want.tolist())
        assert (np.diff(idx) > 0).all()


def test_select_bruteforce_with_ties():
    # max-sum subsets of size n, lexicographically smallest ascending tuple on ties
    rng = np.random.default_rng(12)
    for trial in range(40):
        C = int(rng.integers(1, 11))
        n = int(rng.integers(1, C + 1))
        s = rng.integers(0, 4, size=C).astype(np.float64)   # exact sums, many ties
        best = None
        for sub in itertools.combinations(range(C), n):
            key = (-sum(s[list(sub)]), sub)
            if best is None or key < best:
                best = key
        assert oracle.select_topb(s, n).tolist() == list(best[1]), (s, n)


def test_keep_all_when_budget_exceeds_candidates():
    # B >= L keeps every token; compaction is then the identity
    Hq, Hkv, d, w, kd, L = 4, 2, 8, 4, 2, 20
    N = L + kd
    q = _rand((Hq, w + kd, d), 13)
    k = _rand((Hkv, N, d), 14)
    v = _rand((Hkv, N, d), 15)
    raw, out = oracle.evict_layer(q, k, v, [0, N], Hq, Hkv, w, kd, budget=L + 5, kappa=3)
    for h in range(Hkv):
        assert out[(0, h)]["idx"].tolist() == list(range(N - w - kd))
        assert np.array_equal(out[(0, h)]["k"], k[h]) and np.array_equal(out[(0, h)]["v"], v[h])


def test_streaming_closed_form_c5():
    wl = di.WORKLOADS["c5"]
    N = wl.cached_lens[0]
    idx = oracle.streaming_select(N, wl.slm_sinks, wl.slm_recent)
    kept = np.concatenate([idx, np.arange(N - wl.slm_recent, N)])
    want = np.concatenate([np.arange(4), np.arange(N - 1020, N)])
    assert np.array_equal(kept, want)
    assert oracle.streaming_select(10, 4, 8).tolist() == [0, 1]     # sinks clipped to C
    assert oracle.streaming_select(5, 4, 8).tolist() == []


# ----------------------------------------------------------------------------------
# Compaction: exact identities of Eq. 1, the eviction-mass equation and the attention-matching-loss equation
# ----------------------------------------------------------------------------------
def test_compaction_attention_identities():
    Hq, Hkv, d, w, kd, L = 4, 1, 16, 4, 2, 60
    N = L + kd
    q = _rand((Hq, w + kd, d), 16, 1.5)
    k = _rand((Hkv, N, d), 17, 1.5)
    v = _rand((Hkv, N, d), 18)
    raw, out = oracle.evict_layer(q, k, v, [0, N], Hq, Hkv, w, kd, budget=20, kappa=3)
    o = out[(0, 0)]
    C = N - w - kd
    kept = np.concatenate([o["idx"], np.arange(C, N)])
    E = np.setdiff1d(np.arange(N), kept)
    assert len(E) == N - (20 - w) - w - kd
    for t in range(3):
        qt = _rand((d,), 100 + t, 1.5)
        full = oracle.attention_output(qt, k[0], v[0])
        comp = oracle.attention_output(qt, o["k"], o["v"])      # renormalized over R
        m = oracle.evicted_mass(qt, k[0], E)
        a = np.exp(k[0] @ qt / math.sqrt(d)); a /= a.sum()
        mu_E = (a[E] @ v[0][E]) / m
        assert np.allclose(full, (1 - m) * comp + m * mu_E, rtol=1e-12, atol=1e-13)
        dlogz = oracle.log_partition(qt, k[0]) - oracle.log_partition(qt, o["k"])
        assert abs(dlogz - (-math.log(1 - m))) < 1e-12


# ----------------------------------------------------------------------------------
# Evicted mass of the observation rows and the attention-matching loss (Eq. match)
# ----------------------------------------------------------------------------------
def _diag_case(seed, lens=(40, 57), Hq=4, Hkv=2, d=16, n_tail=6):
    q = _rand((Hq, len(lens) * n_tail, d), seed, 1.5)
    k = _rand((Hkv, sum(lens), d), seed + 1, 1.5)
    offs = np.concatenate([[0], np.cumsum(lens)])
    return q, k, offs, Hq, Hkv, n_tail, lens


def test_eviction_diagnostics_against_torch_softmax():
    """rho_q against torch's float64 softmax mass on the evicted keys, and the loss against
    torch's logsumexp over the full and the retained keys (the two sides of Eq. match)."""
    q, k, offs, Hq, Hkv, n_tail, lens = _diag_case(41)
    rng = np.random.default_rng(5)
    kept = {(b, h): np.sort(rng.choice(N - n_tail, size=(N - n_tail) // 3, replace=False))
            for b, N in enumerate(lens) for h in range(Hkv)}
    rho, beta, lm = oracle.eviction_diagnostics(q, k, offs, Hq, Hkv, kept, n_tail, n_tail)
    G = Hq // Hkv
    for b, N in enumerate(lens):
        C = N - n_tail
        for h in range(Hkv):
            keep = torch.zeros(N, dtype=torch.bool)
            keep[torch.from_numpy(kept[(b, h)])] = True
            keep[C:] = True
            rows, losses = [], []
            for g in range(G):
                for r in range(n_tail):
                    p = C + r
                    x = torch.from_numpy(k[h, offs[b]:offs[b] + p + 1]) @ torch.from_numpy(q[h * G + g, b * n_tail + r])
                    x = x / math.sqrt(k.shape[2])
                    a = torch.softmax(x, dim=0)
                    want = float(a[~keep[:p + 1]].sum())
                    assert abs(rho[h * G + g, b * n_tail + r] - want) < 1e-13
                    rows.append(want)
                    losses.append(float(torch.logsumexp(x, 0) - torch.logsumexp(x[keep[:p + 1]], 0)))
            assert abs(beta[b, h] - np.mean(rows)) < 1e-13
            assert abs(lm[b, h] - np.mean(losses)) < 1e-12


def test_eviction_diagnostics_match_loss_identity_and_special_cases():
    q, k, offs, Hq, Hkv, n_tail, lens = _diag_case(43)
    G = Hq // Hkv
    rng = np.random.default_rng(6)
    kept = {(b, h): np.sort(rng.choice(N - n_tail, size=5, replace=False))
            for b, N in enumerate(lens) for h in range(Hkv)}
    rho, beta, lm = oracle.eviction_diagnostics(q, k, offs, Hq, Hkv, kept, n_tail, n_tail)
    # Eq. match: E_q[-log(1 - rho_q)] equals the mean log-partition deficit
    for b in range(len(lens)):
        for h in range(Hkv):
            r = rho[h * G:(h + 1) * G, b * n_tail:(b + 1) * n_tail]
            assert abs(lm[b, h] - np.mean(-np.log1p(-r))) < 1e-12
            assert 0 < beta[b, h] < 1
    # keep-all: nothing evicted
    all_kept = {(b, h): np.arange(N - n_tail) for b, N in enumerate(lens) for h in range(Hkv)}
    rho0, beta0, lm0 = oracle.eviction_diagnostics(q, k, offs, Hq, Hkv, all_kept, n_tail, n_tail)
    assert (rho0 == 0).all() and (beta0 == 0).all() and np.abs(lm0).max() < 1e-12
    # uniform attention (q = 0), nothing kept but the tail: a row at position p spreads
    # 1/(p+1) over its keys, so rho = C/(p+1) and the loss is log((p+1)/(p+1-C))
    none = {(b, h): np.zeros(0, np.int64) for b in range(len(lens)) for h in range(Hkv)}
    rho1, beta1, lm1 = oracle.eviction_diagnostics(np.zeros_like(q), k, offs, Hq, Hkv, none,
                                                   n_tail, n_tail)
    for b, N in enumerate(lens):
        C = N - n_tail
        want = np.array([C / (C + r + 1) for r in range(n_tail)])
        for hq in range(Hq):
            assert np.allclose(rho1[hq, b * n_tail:(b + 1) * n_tail], want, rtol=1e-14)
        for h in range(Hkv):
            assert abs(beta1[b, h] - want.mean()) < 1e-14
            assert abs(lm1[b, h] - np.mean([math.log((C + r + 1) / (r + 1)) for r in range(n_tail)])) < 1e-12


# ----------------------------------------------------------------------------------
# Attention over a compacted cache (continuation check)
# ----------------------------------------------------------------------------------
def _compacted(k, v, idx_per_seq, n_tail, offs, n_out):
    """[batch][H_kv][n_out][d] caches: retained rows || tail || zero padding."""
    Hkv, _, d = k.shape
    batch = len(offs) - 1
    kc = np.zeros((batch, Hkv, n_out, d))
    vc = np.zeros((batch, Hkv, n_out, d))
    for b in range(batch):
        s0, N = offs[b], offs[b + 1] - offs[b]
        rows = np.concatenate([idx_per_seq[b], np.arange(N - n_tail, N)]).astype(int)
        kc[b, :, :len(rows)] = k[:, s0 + rows]
        vc[b, :, :len(rows)] = v[:, s0 + rows]
    return kc, vc


def test_cache_attention_matches_sdpa_with_explicit_mask():
    # torch SDPA (float64, CPU) with a boolean mask built independently from positions
    Hq, Hkv, d, n_tail, n_q, q_from_end = 6, 2, 16, 5, 7, 5
    offs = [0, 40, 71]
    k = _rand((Hkv, 71, d), 31, 1.3)
    v = _rand((Hkv, 71, d), 32)
    idx = [np.array([1, 4, 9, 20, 33]), np.array([0, 2, 3, 17])]
    n_kept = [5, 4]
    kc, vc = _compacted(k, v, idx, n_tail, offs, 12)
    q = _rand((Hq, 2 * n_q, d), 33, 1.3)
    out, lse = oracle.cache_attention(q, kc, vc, n_kept, n_tail, q_from_end, Hq, Hkv)
    G = Hq // Hkv
    for b in range(2):
        N = offs[b + 1] - offs[b]
        pos_rows = np.concatenate([idx[b], np.arange(N - n_tail, N)])       # original positions
        pos_rows = np.concatenate([pos_rows, np.full(12 - len(pos_rows), 10 ** 9)])  # padding never seen
        qpos = N - q_from_end + np.arange(n_q)
        mask = torch.from_numpy(pos_rows[None, :] <= qpos[:, None])
        for hq in range(Hq):
            Q = torch.from_numpy(q[hq, b * n_q:(b + 1) * n_q])[None]
            K = torch.from_numpy(kc[b, hq // G])[None]
            V = torch.from_numpy(vc[b, hq // G])[None]
            ref = torch.nn.functional.scaled_dot_product_attention(Q, K, V, attn_mask=mask)[0].numpy()
            assert np.allclose(out[hq, b * n_q:(b + 1) * n_q], ref, rtol=1e-10, atol=1e-12)
            x = (Q[0] @ K[0].T) / math.sqrt(d)
            ref_lse = torch.logsumexp(x.masked_fill(~mask, float("-inf")), dim=1).numpy()
            assert np.allclose(lse[hq, b * n_q:(b + 1) * n_q], ref_lse, rtol=1e-12, atol=1e-12)


def test_cache_attention_keep_all_reproduces_scoring_row_lse():
    # keep-all compaction + the scoring rows (q_from_end = w + k) sees exactly the causal
    # keys of each scoring row: its log-partition is the scoring pass's row LSE
    Hq, Hkv, d, w, kd = 4, 2, 8, 5, 2
    offs = [0, 30, 47]
    k = _rand((Hkv, 47, d), 34, 1.2)
    v = _rand((Hkv, 47, d), 35)
    q = _rand((Hq, 2 * (w + kd), d), 36, 1.2)
    n_tail = w + kd
    idx = [np.arange(30 - n_tail), np.arange(17 - n_tail)]
    kc, vc = _compacted(k, v, idx, n_tail, offs, 30)
    _, lse = oracle.cache_attention(q, kc, vc, [len(i) for i in idx], n_tail, n_tail, Hq, Hkv)
    want = oracle.scoring_row_lse(q, k, offs, Hq, Hkv, w, kd)
    assert np.allclose(lse, want, rtol=1e-12, atol=1e-12)


def test_cache_attention_decomposes_over_keep_and_evict():
    # Eq. 1: a decode query's full output is (1 - m) * output over R + m * output over E,
    # with m = 1 - exp(lse_R - lse_full); and lse_full = logaddexp(lse_R, lse_E)
    Hq, Hkv, d, n_tail, N = 4, 2, 8, 3, 25
    k = _rand((Hkv, N, d), 37, 1.5)
    v = _rand((Hkv, N, d), 38)
    q = _rand((Hq, 2, d), 39, 1.5)
    C = N - n_tail
    keep = np.array([0, 3, 7, 8, 15])
    ev = np.setdiff1d(np.arange(C), keep)
    full_k, full_v = _compacted(k, v, [np.arange(C)], n_tail, [0, N], N)
    r_k, r_v = _compacted(k, v, [keep], n_tail, [0, N], N)
    e_k, e_v = _compacted(k, v, [ev], 0, [0, N], N)
    o_f, l_f = oracle.cache_attention(q, full_k, full_v, [C], n_tail, 0, Hq, Hkv)
    o_r, l_r = oracle.cache_attention(q, r_k, r_v, [len(keep)], n_tail, 0, Hq, Hkv)
    o_e, l_e = oracle.cache_attention(q, e_k, e_v, [len(ev)], 0, 0, Hq, Hkv)
    m = 1.0 - np.exp(l_r - l_f)
    assert np.allclose(o_f, (1 - m)[..., None] * o_r + m[..., None] * o_e, rtol=1e-12, atol=1e-13)
    assert np.allclose(l_f, np.logaddexp(l_r, l_e), rtol=1e-13, atol=1e-13)
    assert np.all((m > 0) & (m < 1))


# ----------------------------------------------------------------------------------
# H2O accumulated attention
# ----------------------------------------------------------------------------------
def test_h2o_uniform_is_harmonic():
    # identical keys: colsum[j] = sum_{p=j}^{N-1} 1/(p+1) = H_N - H_j
    Hq, Hkv, d, N = 4, 2, 8, 37
    q = _rand((Hq, N, d), 19)
    k = np.tile(_rand((1, 1, d), 20), (Hkv, N, 1))
    col = oracle.h2o_colsum(q, k, [0, N], Hq, Hkv, block=8)
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, N + 1))])
    assert np.allclose(col, (H[N] - H[:N])[None, :], rtol=1e-13, atol=0)
    assert np.allclose(col.sum(axis=1), N, rtol=1e-13)


def test_h2o_matches_causal_sdpa():
    Hq, Hkv, d = 4, 2, 16
    offs = [0, 33, 70]
    G = Hq // Hkv
    q = _rand((Hq, offs[-1], d), 21, 1.5)
    k = _rand((Hkv, offs[-1], d), 22, 1.5)
    col = oracle.h2o_colsum(q, k, offs, Hq, Hkv, block=16)
    lse = oracle.h2o_row_lse(q, k, offs, Hq, Hkv, block=16)
    for b in range(2):
        s0, N = offs[b], offs[b + 1] - offs[b]
        for h in range(Hkv):
            acc = np.zeros(N)
            for g in range(G):
                Q = torch.tensor(q[h * G + g, s0:s0 + N])[None, None]
                K = torch.tensor(k[h, s0:s0 + N])[None, None]
                P = torch.nn.functional.scaled_dot_product_attention(
                    Q, K, torch.eye(N, dtype=torch.float64)[None, None], is_causal=True)[0, 0]
                acc += P.sum(0).numpy()
                x = (Q[0, 0] @ K[0, 0].T) / math.sqrt(d)
                x = x.masked_fill(torch.ones(N, N, dtype=torch.bool).triu(1), float("-inf"))
                assert np.allclose(lse[h * G + g, s0:s0 + N], torch.logsumexp(x, 1).numpy(), rtol=1e-13)
            assert np.allclose(col[h, s0:s0 + N], acc / G, rtol=1e-12, atol=1e-15)


def test_h2o_select_splits_heavy_and_recent():
    s = np.array([5, 1, 4, 4, 0, 9, 9, 9], np.float64)
    # budget 5 = 3 heavy among the first 5 + 3 recent (positions 5..7)
    assert oracle.h2o_select(s, 6, 3).tolist() == [0, 2, 3]


# ----------------------------------------------------------------------------------
# Input storage (the shared generator's bf16 rounding vs torch's own conversion)
# ----------------------------------------------------------------------------------
def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(23).standard_normal(10000).astype(np.float32) * 7
    x[:4] = [0.0, -0.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8]   # ties to even both ways
    bits = di.f32_to_bf16_bits(x)
    want = torch.tensor(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bits, want)
    assert np.array_equal(di.bf16_bits_to_f32(bits), torch.tensor(x).to(torch.bfloat16).float().numpy())


def test_byte_accounting_pins_bf16_storage():
    # App. "Complexity and overheads": 3.79 GiB (KV repeated to 32 heads) vs 0.95 GiB (8 KV heads) at L = 7762;
    # intro: ~16 GiB for an 8B model at 128K; App. "Draft-guided eviction implementation": ~60 MB of prompt queries per layer
    def kv_bytes(layers, H, L, d=128, elt=2):
        return layers * 2 * H * L * d * elt
    assert round(kv_bytes(32, 32, 7762) / 2 ** 30, 2) == 3.79
    assert round(kv_bytes(32, 8, 7762) / 2 ** 30, 2) == 0.95
    assert round(kv_bytes(32, 8, 128 * 1024) / 2 ** 30) == 16
    assert round(32 * 7762 * 128 * 2 / 2 ** 20, 1) == 60.6


def test_c1_planted_keys_survive():
    # the eight x4-scaled keys per KV head attract attention and survive eviction
    wl = di.WORKLOADS["c1"]
    x = di.make_layer(wl)
    raw, out = oracle.evict_layer(x.q, x.k, x.v, wl.kv_offsets, wl.n_q_heads, wl.n_kv_heads,
                                  wl.window, wl.k_draft, wl.budget, wl.pool)
    for h in range(wl.n_kv_heads):
        kept = set(out[(0, h)]["idx"].tolist())
        hits = sum(int(r) in kept for r in x.planted[(0, h)])
        assert hits >= 6, (h, hits)


# ----------------------------------------------------------------------------------
# Retained-set contiguity (Sec. 4; Table "Selection decomposition", "run len.")
# ----------------------------------------------------------------------------------
def test_retained_runs_closed_forms():
    # one block of n consecutive positions; every other position; the empty set
    for n in (1, 5, 64):
        assert oracle.retained_runs(range(7, 7 + n)) == (1, float(n))
        assert oracle.retained_runs(range(0, 2 * n, 2)) == (n, 1.0)
    assert oracle.retained_runs([]) == (0, 0.0)
    # order and duplicates do not matter
    assert oracle.retained_runs([9, 3, 4, 10, 3, 11]) == (2, 2.5)


def test_retained_runs_match_rising_edges_of_the_mask():
    # an independent count: runs are the 0 -> 1 transitions of the retained 0/1 mask
    rng = np.random.default_rng(17)
    for trial in range(200):
        C = int(rng.integers(1, 60))
        keep = rng.random(C) < rng.random()
        idx = np.flatnonzero(keep)
        mask = np.concatenate([[0], keep.astype(int)])
        edges = int(np.sum((mask[1:] == 1) & (mask[:-1] == 0)))
        runs, mean = oracle.retained_runs(idx)
        assert runs == edges
        assert (mean == 0.0) if edges == 0 else math.isclose(mean, keep.sum() / edges)


def test_maxpool_plateau_is_one_run():
    # a single positive raw score at position j spreads, after max-pooling with an odd
    # kernel kappa, over the kappa candidates around j (clipped at the ends); selecting
    # exactly that many keeps one run of that length -- the contiguity the paper credits
    # to SnapKV's pooling
    for C, j, kappa in ((40, 20, 7), (40, 1, 7), (40, 39, 5), (12, 6, 1)):
        raw = np.zeros(C + 3)
        raw[j] = 1.0
        pooled = oracle.maxpool(raw, C, kappa)
        width = min(C - 1, j + kappa // 2) - max(0, j - kappa // 2) + 1
        idx = oracle.select_topb(pooled, width)
        assert oracle.retained_runs(idx) == (1, float(width))


def test_rope_hand_example_pairs_and_frequencies():
    # d = 4, theta = 10000, p = 1: pair (x0, x2) turns by 1 rad, pair (x1, x3) by
    # 10000^(-2/4) = 0.01 rad (rotate-half pairing; the lowest index has the fastest turn)
    got = oracle.rope(np.array([[1.0, 2.0, 3.0, 4.0]]), [1], theta=10000.0)[0]
    c1, s1, c2, s2 = math.cos(1.0), math.sin(1.0), math.cos(0.01), math.sin(0.01)
    want = [1 * c1 - 3 * s1, 2 * c2 - 4 * s2, 3 * c1 + 1 * s1, 4 * c2 + 2 * s2]
    assert np.allclose(got, want, rtol=0, atol=1e-15)


def test_rope_is_a_complex_phase_and_keeps_relative_positions():
    rng = np.random.default_rng(21)
    d, n = 128, 6
    x = rng.standard_normal((3, n, d))
    pos = np.array([0, 1, 7, 300, 4097, 32767])
    got = oracle.rope(x, pos)
    # as complex numbers z = x_i + i x_{i+d/2}, each pair is multiplied by exp(i p theta_i)
    z = x[..., :d // 2] + 1j * x[..., d // 2:]
    ph = np.exp(1j * pos[:, None] * 500000.0 ** (-np.arange(d // 2) * 2.0 / d))
    w = z * ph
    assert np.allclose(got, np.concatenate([w.real, w.imag], axis=-1), rtol=0, atol=1e-9)
    assert np.array_equal(got[:, 0], x[:, 0])                      # position 0: identity
    assert np.allclose(np.linalg.norm(got, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-12)
    # the logit of a rotated query/key pair depends on the position difference only
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    def logit(p, s):
        return float(oracle.rope(q[None], [p])[0] @ oracle.rope(k[None], [s])[0])
    assert math.isclose(logit(50, 20), logit(1050, 1020), rel_tol=1e-10)
    assert math.isclose(logit(7, 7), float(q @ k), rel_tol=1e-10)


# ----------------------------------------------------------------------------------
# Query/key capture: RoPE(x W^T) per head
# ----------------------------------------------------------------------------------
def test_project_rope_against_torch_linear_and_complex_phase():
    """The composition against torch's float64 Linear (head split [n][H*d] -> [H][n][d])
    and the rotation written as a complex phase (an implementation independent of
    oracle.rope); at position 0 the output is the plain projection."""
    rng = np.random.default_rng(23)
    n, hidden, H, d = 7, 48, 3, 16
    x = rng.standard_normal((n, hidden))
    w = rng.standard_normal((H * d, hidden)) / math.sqrt(hidden)
    pos = np.array([0, 3, 17, 255, 4096, 30000, 2])
    got = oracle.project_rope(x, w, pos, H, d)
    y = torch.nn.functional.linear(torch.from_numpy(x), torch.from_numpy(w))
    y = y.view(n, H, d).permute(1, 0, 2).numpy()
    z = y[..., :d // 2] + 1j * y[..., d // 2:]
    z = z * np.exp(1j * pos[:, None] * 500000.0 ** (-np.arange(d // 2) * 2.0 / d))
    assert np.allclose(got, np.concatenate([z.real, z.imag], axis=-1), rtol=0, atol=1e-12)
    assert np.allclose(got[:, 0], y[:, 0], rtol=0, atol=1e-13)      # position 0: identity
    assert got.shape == (H, n, d)


def test_project_rope_logits_depend_on_position_difference():
    rng = np.random.default_rng(29)
    hidden, d = 32, 8
    xq, xk = rng.standard_normal((1, hidden)), rng.standard_normal((1, hidden))
    wq, wk = rng.standard_normal((d, hidden)), rng.standard_normal((d, hidden))
    def logit(p, s):
        q = oracle.project_rope(xq, wq, [p], 1, d)[0, 0]
        k = oracle.project_rope(xk, wk, [s], 1, d)[0, 0]
        return float(q @ k)
    assert math.isclose(logit(40, 10), logit(1040, 1010), rel_tol=1e-10)
    assert math.isclose(logit(9, 9), float((xq @ wq.T)[0] @ (xk @ wk.T)[0]), rel_tol=1e-10)
