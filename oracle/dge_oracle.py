"""Float64 CPU oracle for the Draft-Guided Eviction (DGE) eviction step.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with the
GPU library (no kernels, helpers, tables or constants) and never imports it.

Every function is the plain definition of one step, written from the paper
(arxiv 2609.33334, "Draft-Guided Eviction"), in float64, with no blocking or
fusion.  Notation, per layer, KV head h and sequence b:

* G = H_q / H_kv query heads share KV head h (native GQA layout, App. "Complexity and overheads");
* L prompt rows, w window rows, k draft rows, N = L + k cached rows;
* the protected tail is the last n_tail = w + k cached rows (window + draft tail,
  Alg. 1 step C and App. "Draft-guided eviction implementation", implementation notes);
* C = N - n_tail candidate rows, B' = min(B - w, C) selected rows.

Readings of points the paper leaves open (each also listed with its evidence in
the design notes): softmax runs causally over every cached key j <= p, tail
included; the score is the SUM over scoring rows (App. "Diagnostic details", "score sum"),
which ranks identically to Alg. 1's 1/k mean; the GQA group MEAN is taken before
max-pooling; pooling only spans the candidates, out-of-range counting as -inf;
top-B ties go to the lower position; selected indices are returned ascending.
"""
from __future__ import annotations

import math

import numpy as np

# scoring-row modes (Alg. 1 step B): window+draft (default), draft only (DGE), window only (DGE-W)
ROWS_WINDOW_DRAFT, ROWS_DRAFT, ROWS_WINDOW = 0, 1, 2


def as_f64(x) -> np.ndarray:
    """Exact up-cast of stored float32 values (bf16 inputs arrive already widened)."""
    return np.asarray(x, dtype=np.float64)


def scoring_rows(N: int, w: int, k: int, mode: int):
    """First position p0 and count of the scoring rows for one sequence.

    Alg. 1 step B (DGE): the k draft rows, positions [N-k, N).
    Alg. 1 step B alternative (DGE-W, SnapKV's window): the last w prompt rows,
    positions [L-w, L) with L = N - k.  Default here: window and draft rows together.
    """
    if mode == ROWS_WINDOW_DRAFT:
        return N - w - k, w + k
    if mode == ROWS_DRAFT:
        return N - k, k
    if mode == ROWS_WINDOW:
        return N - k - w, w
    raise ValueError(mode)


def causal_probs(qrows: np.ndarray, keys: np.ndarray, positions: np.ndarray) -> np.ndarray:
    """softmax_j(q_r . k_j / sqrt(d)) over keys j <= position of row r, 0 beyond.

    Alg. 1 step B (the softmax of q K^T / sqrt(d)); fp32 softmax in the paper
    (App. "Diagnostic details"), float64 here.  qrows [R][d], keys [N][d] -> [R][N].
    """
    d = keys.shape[1]
    x = (qrows @ keys.T) / math.sqrt(d)
    j = np.arange(keys.shape[0])[None, :]
    valid = j <= positions[:, None]
    x = np.where(valid, x, -np.inf)
    m = x.max(axis=1, keepdims=True)
    e = np.where(valid, np.exp(x - m), 0.0)
    return e / e.sum(axis=1, keepdims=True)


def window_scores(q, k, kv_offsets, n_q_heads: int, n_kv_heads: int, w: int, k_draft: int,
                  mode: int = ROWS_WINDOW_DRAFT) -> np.ndarray:
    """Per-KV-head attention mass each cached key receives from the scoring rows.

    raw[h][j] = (1/G) * sum_{g in group h} sum_{r} softmax_j(q_{g,r} K^T / sqrt(d)),
    i.e. the score sum over past keys of App. "Diagnostic details", from the rows Alg. 1 step B
    names, averaged over the query heads of the GQA group (App. "Complexity and overheads",
    gqa_score_agg).  q [H_q][batch*n_rows][d] holds the mode's rows in ascending
    position; k [H_kv][T][d] -> raw [H_kv][T].
    """
    q = as_f64(q)
    k = as_f64(k)
    G = n_q_heads // n_kv_heads
    offs = [int(o) for o in kv_offsets]
    T = offs[-1]
    raw = np.zeros((n_kv_heads, T), np.float64)
    for b in range(len(offs) - 1):
        s0, N = offs[b], offs[b + 1] - offs[b]
        p0, nr = scoring_rows(N, w, k_draft, mode)
        pos = p0 + np.arange(nr)
        r0 = b * nr  # q holds exactly this mode's n_rows rows per sequence
        for h in range(n_kv_heads):
            acc = np.zeros(N, np.float64)
            for g in range(G):
                P = causal_probs(q[h * G + g, r0:r0 + nr], k[h, s0:s0 + N], pos)
                acc += P.sum(axis=0)
            raw[h, s0:s0 + N] = acc / G
    return raw


def scoring_row_lse(q, k, kv_offsets, n_q_heads: int, n_kv_heads: int, w: int, k_draft: int,
                    mode: int = ROWS_WINDOW_DRAFT) -> np.ndarray:
    """log sum_{j <= p_r} exp(q_r . k_j / sqrt(d)) of every scoring row (the softmax
    normaliser of Alg. 1 step B), [H_q][batch * n_rows] in the row order of q."""
    q = as_f64(q)
    k = as_f64(k)
    G = n_q_heads // n_kv_heads
    offs = [int(o) for o in kv_offsets]
    d = k.shape[2]
    out = np.zeros((n_q_heads, q.shape[1]), np.float64)
    for b in range(len(offs) - 1):
        s0, N = offs[b], offs[b + 1] - offs[b]
        p0, nr = scoring_rows(N, w, k_draft, mode)
        for hq in range(n_q_heads):
            x = (q[hq, b * nr:(b + 1) * nr] @ k[hq // G, s0:s0 + N].T) / math.sqrt(d)
            x = np.where(np.arange(N)[None, :] <= (p0 + np.arange(nr))[:, None], x, -np.inf)
            m = x.max(axis=1)
            out[hq, b * nr:(b + 1) * nr] = m + np.log(np.exp(x - m[:, None]).sum(axis=1))
    return out


def maxpool(raw_row: np.ndarray, C: int, kappa: int) -> np.ndarray:
    """SnapKV 1-D max-pool (kernel kappa, stride 1, same length) over candidates [0, C).

    pooled[j] = max{raw[i] : |i - j| <= kappa // 2, 0 <= i < C} (App. "Diagnostic details",
    Sec. 6 compression settings: kernel 7).  Keys outside the candidate range do
    not take part.
    """
    r = kappa // 2
    x = np.asarray(raw_row[:C], np.float64)
    out = np.empty(C, np.float64)
    for j in range(C):
        out[j] = x[max(0, j - r):min(C, j + r + 1)].max()
    return out


def select_topb(pooled: np.ndarray, n_select: int) -> np.ndarray:
    """Indices of the n_select largest pooled scores, ties to the lower index, ascending.

    Alg. 1 step B: I <- R_E(s, B - w) with per-head top-B; App. "Draft-guided eviction
    implementation": indices are sorted to keep temporal order.  Keeps everything when
    n_select >= C.
    """
    C = pooled.shape[0]
    n = min(int(n_select), C)
    order = np.lexsort((np.arange(C), -np.asarray(pooled, np.float64)))
    return np.sort(order[:n]).astype(np.int64)


def compact(k_rows: np.ndarray, v_rows: np.ndarray, idx: np.ndarray, C: int):
    """[retained past, ascending] || [window + draft tail] (App. "Draft-guided eviction implementation", implementation notes)."""
    N = k_rows.shape[0]
    keep = np.concatenate([np.asarray(idx, np.int64), np.arange(C, N)])
    return k_rows[keep].copy(), v_rows[keep].copy()


def evict_layer(q, k, v, kv_offsets, n_q_heads, n_kv_heads, w, k_draft, budget, kappa,
                mode=ROWS_WINDOW_DRAFT, n_tail=None):
    """Whole eviction step for one layer: score -> pool -> top-(B-w) -> compact.

    Returns raw [H_kv][T], and per (b, h): pooled, idx, compacted K and V.
    """
    raw = window_scores(q, k, kv_offsets, n_q_heads, n_kv_heads, w, k_draft, mode)
    n_tail = w + k_draft if n_tail is None else n_tail
    offs = [int(o) for o in kv_offsets]
    out = {}
    for b in range(len(offs) - 1):
        s0, N = offs[b], offs[b + 1] - offs[b]
        C = N - n_tail
        for h in range(n_kv_heads):
            pooled = maxpool(raw[h, s0:s0 + N], C, kappa)
            idx = select_topb(pooled, budget - w)
            ko, vo = compact(np.asarray(k)[h, s0:s0 + N], np.asarray(v)[h, s0:s0 + N], idx, C)
            out[(b, h)] = dict(pooled=pooled, idx=idx, k=ko, v=vo)
    return raw, out


# ---------------------------------------------------------------------------------------
# Alternative retention rules
# ---------------------------------------------------------------------------------------
def h2o_row_lse(q_all, k, kv_offsets, n_q_heads: int, n_kv_heads: int, block: int = 1024):
    """log sum_{j <= p} exp(q_p . k_j / sqrt(d)) for every cached row p and query head."""
    q_all = as_f64(q_all)
    k = as_f64(k)
    G = n_q_heads // n_kv_heads
    offs = [int(o) for o in kv_offsets]
    lse = np.zeros((n_q_heads, offs[-1]), np.float64)
    d = k.shape[2]
    for b in range(len(offs) - 1):
        s0, N = offs[b], offs[b + 1] - offs[b]
        for hq in range(n_q_heads):
            K = k[hq // G, s0:s0 + N]
            for p0 in range(0, N, block):
                p1 = min(N, p0 + block)
                x = (q_all[hq, s0 + p0:s0 + p1] @ K[:p1].T) / math.sqrt(d)
                valid = np.arange(p1)[None, :] <= np.arange(p0, p1)[:, None]
                x = np.where(valid, x, -np.inf)
                m = x.max(axis=1)
                lse[hq, s0 + p0:s0 + p1] = m + np.log(np.where(valid, np.exp(x - m[:, None]), 0).sum(axis=1))
    return lse


def h2o_colsum(q_all, k, kv_offsets, n_q_heads: int, n_kv_heads: int, block: int = 1024):
    """H2O accumulated attention, kept running through the draft rows.

    colsum[h][j] = (1/G) * sum_g sum_{p = j}^{N-1} softmax_j(q_{g,p} K^T / sqrt(d)):
    the causal attention every cached row (all prefill rows plus the k draft rows)
    pays to key j (Table "Complexity and measured overhead", footnote a), meaned over the GQA group.
    """
    q_all = as_f64(q_all)
    k = as_f64(k)
    G = n_q_heads // n_kv_heads
    offs = [int(o) for o in kv_offsets]
    col = np.zeros((n_kv_heads, offs[-1]), np.float64)
    for b in range(len(offs) - 1):
        s0, N = offs[b], offs[b + 1] - offs[b]
        for h in range(n_kv_heads):
            K = k[h, s0:s0 + N]
            acc = np.zeros(N, np.float64)
            for g in range(G):
                qh = q_all[h * G + g, s0:s0 + N]
                for p0 in range(0, N, block):
                    p1 = min(N, p0 + block)
                    P = causal_probs(qh[p0:p1], K[:p1], np.arange(p0, p1))
                    acc[:p1] += P.sum(axis=0)
            col[h, s0:s0 + N] = acc / G
    return col


def h2o_select(colsum_row: np.ndarray, budget: int, n_recent: int) -> np.ndarray:
    """H2O retention: heavy hitters = top-(B - n_recent) accumulated scores among the
    non-recent rows, plus the n_recent most recent rows (kept as the tail)."""
    N = colsum_row.shape[0]
    C = N - n_recent
    return select_topb(colsum_row[:C], budget - n_recent)


def streaming_select(N: int, n_sink: int, n_recent: int) -> np.ndarray:
    """StreamingLLM: keep the first n_sink rows (attention sinks) and the last n_recent
    rows; no scores (Sec. 6 baselines; App. "Additional analysis": four sinks and a recency window).
    Returns the kept sink indices; the recent rows are the protected tail."""
    C = max(N - n_recent, 0)
    return np.arange(min(n_sink, C), dtype=np.int64)


def pyramid_budgets(B: int, w: int, n_layers: int, beta: int = 20) -> np.ndarray:
    """PyramidKV per-layer total budgets B_l (App. "Additional analysis", discrete schedule).

    c = B - w past tokens; the ramp starts at max = 2c - floor(c/beta) on layer 0 and
    falls by steps = floor((max - min) / (n_layers - 1)) per layer, min = floor(c/beta)
    (the paper states max and steps; this min reproduces its five worked examples).
    B_l = c_l + w.
    """
    c = B - w
    mx = 2 * c - c // beta
    mn = c // beta
    steps = (mx - mn) // (n_layers - 1) if n_layers > 1 else 0
    return np.array([mx - l * steps + w for l in range(n_layers)], np.int64)


# ---------------------------------------------------------------------------------------
# Identities used to check compaction (Eq. 1 / the eviction-mass equation / the attention-matching loss)
# ---------------------------------------------------------------------------------------
def attention_output(qrow: np.ndarray, keys: np.ndarray, vals: np.ndarray) -> np.ndarray:
    """o = sum_j softmax_j(q . k_j / sqrt(d)) v_j over the given keys."""
    d = keys.shape[1]
    x = keys @ as_f64(qrow) / math.sqrt(d)
    a = np.exp(x - x.max())
    a /= a.sum()
    return a @ vals


def evicted_mass(qrow: np.ndarray, keys: np.ndarray, evicted: np.ndarray) -> float:
    """m(E) = sum_{j in E} softmax_j(q . k_j / sqrt(d)) (the eviction-mass equation; rho_q of the attention-matching loss)."""
    d = keys.shape[1]
    x = keys @ as_f64(qrow) / math.sqrt(d)
    a = np.exp(x - x.max())
    a /= a.sum()
    return float(a[evicted].sum())


def log_partition(qrow: np.ndarray, keys: np.ndarray) -> float:
    """log Z(q) = log sum_j exp(q . k_j / sqrt(d)) (attention-matching loss, App. "Attention-matching loss")."""
    d = keys.shape[1]
    x = keys @ as_f64(qrow) / math.sqrt(d)
    m = x.max()
    return float(m + np.log(np.exp(x - m).sum()))


def eviction_diagnostics(q, k, kv_offsets, n_q_heads: int, n_kv_heads: int, kept, n_tail: int,
                         q_from_end: int):
    """Evicted mass of the observation rows and the attention-matching loss of a selection.

    App. "Attention-matching loss", Eq. match: for an observation query q,
    rho_q = sum_{j in E} e^{q.k_j/sqrt d} / sum_{j in R u E} e^{q.k_j/sqrt d}, and the loss
    is E_q[-log(1 - rho_q)] = E_q |log Z - log Z_R|.  Sec. 3 Eq. 1 calls the same quantity
    for a query the missed mass beta.  Here, for sequence b and KV head h, the rows are
    q[hq][b * n_q + r] at positions p = N_b - q_from_end + r (inside the tail, so every
    candidate precedes them), each attending keys j <= p of the full cache; R is the kept
    past keys kept[(b, h)] plus the tail [N_b - n_tail, N_b), E the other candidates.

    Returns rho [H_q][batch * n_q], beta [batch][H_kv] (mean rho over the group's G heads
    and n_q rows) and l_match [batch][H_kv] (mean of -log(1 - rho) over the same rows).
    rho is computed directly as the softmax mass on E; l_match from the two log-partitions.
    """
    q = as_f64(q)
    k = as_f64(k)
    G = n_q_heads // n_kv_heads
    offs = [int(o) for o in kv_offsets]
    batch = len(offs) - 1
    n_q = q.shape[1] // batch
    d = k.shape[2]
    rho = np.zeros((n_q_heads, batch * n_q), np.float64)
    beta = np.zeros((batch, n_kv_heads), np.float64)
    l_match = np.zeros((batch, n_kv_heads), np.float64)
    for b in range(batch):
        s0, N = offs[b], offs[b + 1] - offs[b]
        C = N - n_tail
        for h in range(n_kv_heads):
            keep = np.zeros(N, bool)
            keep[np.asarray(kept[(b, h)], np.int64)] = True
            keep[C:] = True
            losses = []
            for g in range(G):
                hq = h * G + g
                for r in range(n_q):
                    p = N - q_from_end + r
                    x = k[h, s0:s0 + p + 1] @ q[hq, b * n_q + r] / math.sqrt(d)
                    m = x.max()
                    e = np.exp(x - m)
                    kp = keep[:p + 1]
                    rho[hq, b * n_q + r] = e[~kp].sum() / e.sum()
                    log_z = m + np.log(e.sum())
                    log_zr = m + np.log(e[kp].sum())
                    losses.append(log_z - log_zr)
            rows = [rho[h * G + g, b * n_q + r] for g in range(G) for r in range(n_q)]
            beta[b, h] = np.mean(rows)
            l_match[b, h] = np.mean(losses)
    return rho, beta, l_match


def cache_attention(q, k_c, v_c, n_kept, n_tail: int, q_from_end: int, n_q_heads: int,
                    n_kv_heads: int):
    """Attention of query rows over compacted caches: the check of a continuation on the
    evicted cache (Alg. 1 step C's output; Sec. 3 Eq. 1; the eviction-mass equation of
    App. "Why deferral can recover FullKV").

    q: [H_q][batch * n_q][d]; k_c, v_c: [batch][H_kv][n_out][d], laid out as
    [retained past rows (n_kept[b])] || [tail (n_tail)] || padding.  Query row r of
    sequence b sits at position N_b - q_from_end + r; it attends every retained past row
    (all precede the tail) and the tail rows t <= n_tail - q_from_end + r, i.e. the tail
    rows at positions not after its own.  Returns out [H_q][batch * n_q][d] and the
    natural-log partition lse [H_q][batch * n_q] over the attended rows.
    """
    q = as_f64(q)
    k_c = as_f64(k_c)
    v_c = as_f64(v_c)
    G = n_q_heads // n_kv_heads
    batch = k_c.shape[0]
    n_q = q.shape[1] // batch
    d = q.shape[2]
    out = np.zeros((n_q_heads, batch * n_q, d), np.float64)
    lse = np.full((n_q_heads, batch * n_q), -np.inf, np.float64)
    for b in range(batch):
        nk = int(n_kept[b])
        for hq in range(n_q_heads):
            keys, vals = k_c[b, hq // G], v_c[b, hq // G]
            for r in range(n_q):
                n_vis_tail = min(n_tail, max(0, n_tail - q_from_end + r + 1))
                rows = np.concatenate([np.arange(nk), nk + np.arange(n_vis_tail)]).astype(np.int64)
                if rows.size == 0:
                    continue
                qr = q[hq, b * n_q + r]
                out[hq, b * n_q + r] = attention_output(qr, keys[rows], vals[rows])
                lse[hq, b * n_q + r] = log_partition(qr, keys[rows])
    return out, lse


def retained_runs(idx) -> tuple:
    """Contiguity of a retained set: (number of runs, mean run length).

    The selection diagnostics (Sec. 4, "Selection trades coverage for contiguity";
    Table "Selection decomposition", column "run len."; App. "Diagnostic details") report
    how contiguous a retention rule's kept positions are: a run is a maximal block of
    consecutive retained positions, the run length the mean block size.  Measured over the
    selected past keys: the protected window/draft tail is one block under every rule and
    is not counted.  idx: selected positions (any order; duplicates count once).  An empty
    set gives (0, 0.0).
    """
    pos = sorted({int(i) for i in idx})
    if not pos:
        return 0, 0.0
    runs = 1
    for a, b in zip(pos, pos[1:]):
        if b != a + 1:
            runs += 1
    return runs, len(pos) / runs


def rope(x, positions, theta: float = 500000.0) -> np.ndarray:
    """Rotary position embedding of the query/key rows, the step that produces the
    post-RoPE Q and K the scoring reads (App. "Draft-guided eviction implementation":
    queries recomputed post-RoPE from each layer's input; App. on the compensation token:
    rotate-half pairs (i, i + d/2); Table "Backbones": theta = 500,000).

    x: [..., n_rows, d] (any leading dims), positions: [n_rows].  Pair i of a row at
    position p, i < d/2, is rotated by the angle p * theta^(-2i/d):
        x_i'       = x_i cos - x_{i+d/2} sin
        x_{i+d/2}' = x_{i+d/2} cos + x_i sin
    Returns float64.
    """
    x = as_f64(x)
    d = x.shape[-1]
    half = d // 2
    pos = np.asarray(positions, np.float64)
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / d)
    ang = pos[:, None] * inv[None, :]                 # [n_rows, d/2]
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)



def project_rope(x, w, positions, n_heads: int, head_dim: int, theta: float = 500000.0) -> np.ndarray:
    """Query/key capture from a layer's input: the Linear projection x W^T split into heads,
    then the rotary embedding of each row at its position (App. "Draft-guided eviction
    implementation": post-RoPE queries recomputed from the layer input).

    x [n_rows][hidden], w [n_heads * head_dim][hidden] (rows = output features) ->
    [n_heads][n_rows][head_dim], float64.
    """
    y = as_f64(x) @ as_f64(w).T
    y = y.reshape(y.shape[0], n_heads, head_dim).transpose(1, 0, 2)
    return rope(y, positions, theta)
