"""CPU oracle for one SeKV decode step.  TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this module; the product path (the HIP library and its Python binding)
never does.  It shares no code with that path and imports nothing from it.

It is a plain, slow, float64 NumPy rendering of the paper's decode step
(Sec. 3.3, "Trained Zoom-In Mechanism", with the routing gate and the
reconstruction of Sec. 3.2):

1. routing score of every span for every query head (eq. routing_gate),
2. per-KV-head selection of the top-k spans (the budget rule of Sec. 3.3:
   keep spans in decreasing routing-score order until the budget is filled),
3. reconstruction of the selected spans from their factors
   (eq. key_reconstruction; the same decomposition for the value matrix),
4. one softmax over the mixed-resolution memory: anchors at full resolution,
   one coarse entry per unexpanded span with ln|S| added to its score, and
   the reconstructed tokens of the expanded spans (Sec. 3.3).

The end of the module adds the paper's own selection rule (learned routing
projection, sigmoid gate, per-head thresholds and the budget cap), which
replaces steps 1-2 and keeps steps 3-4.

Readings taken where the paper leaves the decode step open (each is listed
with its reason in the design notes):

* Routing uses the coarse mean key k_bar_S itself as the summary, with an
  identity projection (d' = d_h), no normalisation and scale 1/sqrt(d_h).  The
  routing score then equals the coarse entry's attention score, ln|S| included.
* The zoom rule is top-k on that score (the sigmoid is monotone, so ranking the
  pre-sigmoid score ranks the gate).  A KV head's key for span S is the maximum
  of its query heads' scores: the union of per-head decisions under one shared
  threshold.  Ties go to the lower span index.
* The rank gates are folded into sigma (m_i = 1 for the stored components).
  Per-span retained ranks (the deployment-time drop of Sec. 3.2) come as a
  table of (r_K, r_V) per block; without one, every block has the common rank.
* ln is the natural logarithm; an expanded span's coarse entry is replaced by
  its tokens, never kept beside them.

Floating point.  The routing score is defined bit for bit so that selection is
exact: s = sum_j q[j] * k_bar[j] accumulated left to right in float64 (every
product of two bfloat16 or two float32 values is exact in float64), then
score = (s * scale) + ln|S| as two separately rounded float64 operations.
Everything else is float64 with no particular order.

Stored inputs are bfloat16 bit patterns (uint16) or float32; they are widened
exactly to float64 before use.
"""

from __future__ import annotations

import numpy as np

SOFTMAX_SUM_TOL = 1e-12


# ---------------------------------------------------------------------------
# stored values -> float64
# ---------------------------------------------------------------------------

def widen(a, dtype: str) -> np.ndarray:
    """Exact float64 value of a stored array ('bf16' bit patterns or 'f32')."""
    if dtype == "bf16":
        bits = np.asarray(a, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return bits.view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    raise ValueError(f"unknown storage dtype {dtype!r}")


def _elem(dtype: str):
    return {"bf16": (np.uint16, 2), "f32": (np.float32, 4)}[dtype]


def read_span_block(factors: np.ndarray, offset: int, length: int, rank: int,
                    head_dim: int, dtype: str, rank_v: int | None = None) -> dict:
    """Factors of one span: U_K[|S|][r_K], sigma_K[r_K], Vt_K[r_K][d], then the same
    for V with r_V (rank_v, default rank).

    This is the per-span storage of Sec. 3.2 (U of |S| x r_S, Sigma of r_S
    values, V of d_h x r_S, for keys and for values, each with its own retained
    rank), one contiguous block.
    """
    np_t, e = _elem(dtype)
    if offset % e:
        raise ValueError("misaligned block offset")
    L, d = int(length), int(head_dim)
    ranks = {"K": int(rank), "V": int(rank if rank_v is None else rank_v)}
    n = sum(L * r + r + r * d for r in ranks.values())
    raw = np.frombuffer(np.asarray(factors, dtype=np.uint8).data, dtype=np_t,
                        count=n, offset=int(offset))
    x = widen(raw, dtype)
    out = {}
    pos = 0
    for side in ("K", "V"):
        r = ranks[side]
        out["U" + side] = x[pos:pos + L * r].reshape(L, r)
        pos += L * r
        out["s" + side] = x[pos:pos + r].copy()
        pos += r
        out["Vt" + side] = x[pos:pos + r * d].reshape(r, d)
        pos += r * d
    return out


def block_ranks(block_rank, b: int, g: int, S: int, rank: int):
    """(r_K, r_V) of block (b, g, S): from the packed table (r_K | r_V << 16), or the
    common rank when there is no table."""
    if block_rank is None:
        return int(rank), int(rank)
    w = int(np.asarray(block_rank)[b, g, S])
    return w & 0xFFFF, w >> 16


# ---------------------------------------------------------------------------
# the steps
# ---------------------------------------------------------------------------

def gated_reconstruct(U: np.ndarray, sigma: np.ndarray, Vt: np.ndarray, gates) -> np.ndarray:
    """sum_i m_i sigma_i u_i v_i^T (eq. key_reconstruction with the gates of eq. rank_gates)."""
    return U @ np.diag(np.asarray(gates, dtype=np.float64) * sigma) @ Vt


def deploy_factors(U: np.ndarray, sigma: np.ndarray, Vt: np.ndarray, gates, keep):
    """The stored factors at deployment (Sec. 3.2): the components whose gate is kept,
    with the gate folded into sigma; the others are dropped.  Returns (U, sigma, Vt)
    of rank r_S = number kept."""
    idx = np.flatnonzero(np.asarray(keep, dtype=bool))
    g = np.asarray(gates, dtype=np.float64)
    return U[:, idx], (g * sigma)[idx], Vt[idx]


def reconstruct(U: np.ndarray, sigma: np.ndarray, Vt: np.ndarray) -> np.ndarray:
    """Token-level matrix of a span, sum_i sigma_i u_i v_i^T (eq. key_reconstruction).

    The rank gates m_i are folded into sigma, so the stored components are
    used as they are.
    """
    return U @ np.diag(sigma) @ Vt


def routing_logits(q, sum_k, span_logsize, n_spans, scale: float) -> np.ndarray:
    """Pre-sigmoid routing score of every span for every query head.

    eq. routing_gate with the summary read as the coarse mean key and an
    identity projection: score[b,h,S] = (q_h . k_bar_S) * scale + ln|S|.
    The dot product is summed left to right in float64; padding spans get -inf.
    Returns float64 [B][Hq][M_max].
    """
    q = np.asarray(q, dtype=np.float64)
    sum_k = np.asarray(sum_k, dtype=np.float64)
    B, Hq, d = q.shape
    Hkv, M = sum_k.shape[1], sum_k.shape[2]
    G = Hq // Hkv
    out = np.full((B, Hq, M), -np.inf)
    for b in range(B):
        m = int(n_spans[b])
        for h in range(Hq):
            kb = sum_k[b, h // G, :m, :]
            s = np.zeros(m)
            for j in range(d):
                s = s + q[b, h, j] * kb[:, j]
            out[b, h, :m] = s * scale + span_logsize[b, :m]
    return out


def group_keys(logits: np.ndarray, n_kv_heads: int) -> np.ndarray:
    """Selection key of each span for a KV head: the largest score over its query heads."""
    B, Hq, M = logits.shape
    G = Hq // n_kv_heads
    return logits.reshape(B, n_kv_heads, G, M).max(axis=2)


def select_topk(keys: np.ndarray, n_spans, k: int) -> np.ndarray:
    """Spans to expand per (b, KV head): the k highest keys, ties to the lower index.

    This is the budget rule of Sec. 3.3 (keep spans in decreasing routing
    score until the budget is filled) with a budget of k spans.  Listed in
    that order; slots past the number of spans hold -1.
    """
    B, Hkv, M = keys.shape
    sel = np.full((B, Hkv, k), -1, dtype=np.int32)
    for b in range(B):
        m = int(n_spans[b])
        for g in range(Hkv):
            order = sorted(range(m), key=lambda S: (-keys[b, g, S], S))
            chosen = order[:min(k, m)]
            sel[b, g, :len(chosen)] = chosen
    return sel


def softmax_weights(logits: np.ndarray) -> np.ndarray:
    z = np.exp(logits - logits.max())
    return z / z.sum()


def mixed_attention_head(qh, scale, anchor_k, anchor_v, coarse_logits, coarse_v, zoom):
    """One softmax over anchors, coarse span entries and zoomed tokens (Sec. 3.3).

    qh: [d]; anchor_k/v: [A][d]; coarse_logits: [n_c] (ln|S| already in);
    coarse_v: [n_c][d]; zoom: list of (K_hat [L][d], V_hat [L][d]).
    Returns (out [d], weights [n]) with the weights ordered anchors, coarse, zoom.
    """
    logit_parts = [scale * (anchor_k @ qh), np.asarray(coarse_logits, dtype=np.float64)]
    value_parts = [anchor_v, coarse_v]
    for K_hat, V_hat in zoom:
        logit_parts.append(scale * (K_hat @ qh))
        value_parts.append(V_hat)
    logits = np.concatenate(logit_parts)
    values = np.concatenate(value_parts, axis=0)
    if logits.size == 0:
        raise ValueError("empty attention set: no anchors and no spans")
    p = softmax_weights(logits)
    if abs(p.sum() - 1.0) > SOFTMAX_SUM_TOL:
        raise AssertionError("softmax weights do not sum to one")
    return p @ values, p


def zoom_attend(q, anchor_k, anchor_v, n_anchors, sum_v, n_spans, span_len, factors,
                block_off, sel, logits, *, rank: int, softmax_scale: float,
                dtype: str, block_rank=None) -> np.ndarray:
    """Mixed-resolution decode attention given the selection and routing scores.

    q and the cache arrays are stored values (widened here); logits are the
    float64 routing scores from routing_logits.  block_rank: per-block retained
    ranks (r_K | r_V << 16, [B][Hkv][M]) or None for the common rank.  Returns
    float64 [B][Hq][d].
    """
    qf = widen(q, dtype)
    ak, av, sv = widen(anchor_k, dtype), widen(anchor_v, dtype), widen(sum_v, dtype)
    B, Hq, d = qf.shape
    Hkv = ak.shape[1]
    G = Hq // Hkv
    out = np.zeros((B, Hq, d))
    for b in range(B):
        A, m = int(n_anchors[b]), int(n_spans[b])
        for g in range(Hkv):
            chosen = [int(S) for S in sel[b, g] if S >= 0]
            zoom = []
            for S in chosen:
                rk, rv = block_ranks(block_rank, b, g, S, rank)
                f = read_span_block(factors, int(block_off[b, g, S]), int(span_len[b, S]),
                                    rk, d, dtype, rank_v=rv)
                zoom.append((reconstruct(f["UK"], f["sK"], f["VtK"]),
                             reconstruct(f["UV"], f["sV"], f["VtV"])))
            coarse = [S for S in range(m) if S not in set(chosen)]
            for h in range(g * G, (g + 1) * G):
                out[b, h], _ = mixed_attention_head(
                    qf[b, h], softmax_scale, ak[b, g, :A], av[b, g, :A],
                    logits[b, h, coarse], sv[b, g, coarse], zoom)
    return out


def decode_step(q, anchor_k, anchor_v, n_anchors, sum_k, sum_v, n_spans, span_len,
                span_logsize, factors, block_off, *, rank: int, top_k: int,
                softmax_scale: float, dtype: str, block_rank=None) -> dict:
    """Route, select, reconstruct and attend: one SeKV decode step for one layer."""
    qf = widen(q, dtype)
    logits = routing_logits(qf, widen(sum_k, dtype), np.asarray(span_logsize, np.float64),
                            n_spans, softmax_scale)
    keys = group_keys(logits, np.asarray(sum_k).shape[1])
    sel = select_topk(keys, n_spans, top_k)
    out = zoom_attend(q, anchor_k, anchor_v, n_anchors, sum_v, n_spans, span_len, factors,
                      block_off, sel, logits, rank=rank, softmax_scale=softmax_scale,
                      dtype=dtype, block_rank=block_rank)
    return {"sel": sel, "out": out, "logits": logits, "keys": keys}


# ---------------------------------------------------------------------------
# split softmax algebra and the factored identity (test aids)
# ---------------------------------------------------------------------------

def softmax_partial(logits: np.ndarray, values: np.ndarray):
    """(max, sum of exp(logit - max), sum of exp(logit - max) * value) over one chunk."""
    logits = np.asarray(logits, dtype=np.float64)
    if logits.size == 0:
        return -np.inf, 0.0, np.zeros(values.shape[1])
    mx = logits.max()
    w = np.exp(logits - mx)
    return mx, w.sum(), w @ values


def merge_partials(parts) -> np.ndarray:
    """Combine chunk partials into the output of the one softmax over their union."""
    M = max(p[0] for p in parts)
    l = sum(p[1] * np.exp(p[0] - M) for p in parts if p[1] > 0)
    o = sum(p[2] * np.exp(p[0] - M) for p in parts if p[1] > 0)
    return o / l


def zoom_scores_factored(qh, scale, U, sigma, Vt):
    """scale * q . K_hat_t for every token without forming K_hat: U (sigma * (Vt q))."""
    return scale * (U @ (sigma * (Vt @ qh)))


def zoom_values_factored(p, U, sigma, Vt):
    """sum_t p_t V_hat_t without forming V_hat: ((p^T U) * sigma) Vt."""
    return ((p @ U) * sigma) @ Vt


# ---------------------------------------------------------------------------
# learned routing: the paper's own selection rule
# (Sec. 3.2 eqs. surprisal_weight, summary_key, query_projection, routing_gate;
#  Sec. 3.3 eq. zoom_decision and the budget cap)
# ---------------------------------------------------------------------------
#
# Readings (each listed with its reason in the design notes):
#
# * Indices.  The projections are per query head (Sec. 3.3, learnable-parameters
#   paragraph: L x H x d' x d_h with H the 32 query heads): W[h] is d' x d_h, and query
#   head h routes against summaries built from its KV head's keys with its own
#   W[h], so the routing summaries are [B][Hq][M][d'].  Thresholds are per
#   query head.
# * Union per KV head.  z[h,S] decides per query head; the factors belong to
#   the KV head, so a span is expanded for a (sequence, KV head) pair when any
#   of its query heads votes for it, and the expanded tokens serve every query
#   head of the group (a span whose tokens are on hand is not also kept coarse).
# * Budget cap.  Candidates (spans with at least one vote) are ordered by the
#   largest pre-sigmoid gate among the voting heads, descending, ties to the
#   lower span index (the sigmoid is strictly increasing, so this is the order
#   of alpha~).  The longest prefix of that order whose token count stays within
#   the budget and whose length stays within the count cap is expanded.
# * The threshold is applied in logit space: alpha~ > tau is the same event as
#   x > ln(tau / (1 - tau)), and the threshold enters as that logit.
#
# Floating point (selection must be bit exact, as for the identity routing):
# q' = W q is summed left to right over d_h in float64 (products of stored
# values are exact) and rounded once to float32; the gate's dot product
# q' . Kbar is summed left to right over d' in float64 (float32 x stored
# products are exact); then x = (s * (1/sqrt(d'))) + ln|S| as two separately
# rounded float64 operations.  1/sqrt(d') is 1.0 / sqrt(float(d')) in float64.

def surprisal_weights(H) -> np.ndarray:
    """Span-local token weights w_t = H_t / sum_k H_k (eq. surprisal_weight)."""
    H = np.asarray(H, dtype=np.float64)
    return H / H.sum()


def summary_key(K_tokens, weights, W) -> np.ndarray:
    """Normalised, weighted, projected routing summary of one span (eq. summary_key).

    K_tokens [|S|][d_h], weights [|S|], W [d'][d_h]; returns [d'] of unit norm.
    """
    K = np.asarray(K_tokens, dtype=np.float64)
    w = np.asarray(weights, dtype=np.float64)
    Wm = np.asarray(W, dtype=np.float64)
    x = np.zeros(Wm.shape[0])
    for t in range(K.shape[0]):
        x = x + w[t] * (Wm @ K[t])
    return x / np.linalg.norm(x)


def project_queries(q, W) -> np.ndarray:
    """q'[b,h] = W[h] q[b,h] for every query head (eq. query_projection).

    q [B][Hq][d_h] and W [Hq][d'][d_h] as float64 values of stored numbers.
    Summed left to right over d_h in float64, then rounded to float32.
    Returns the float32 values as float64, [B][Hq][d'].
    """
    q = np.asarray(q, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    B, Hq, d = q.shape
    out = np.zeros((B, Hq, W.shape[1]))
    for j in range(d):
        out = out + W[None, :, :, j] * q[:, :, None, j]
    return out.astype(np.float32).astype(np.float64)


def gate_logits(q_proj, sum_route, span_logsize, n_spans) -> np.ndarray:
    """Pre-sigmoid routing gate x[b,h,S] = q'.Kbar[b,h,S] / sqrt(d') + ln|S| (eq. routing_gate).

    q_proj [B][Hq][d'] (from project_queries), sum_route [B][Hq][M][d'].  The
    dot product is summed left to right in float64; padding spans get -inf.
    """
    qp = np.asarray(q_proj, dtype=np.float64)
    kr = np.asarray(sum_route, dtype=np.float64)
    B, Hq, dr = qp.shape
    M = kr.shape[2]
    scale = 1.0 / np.sqrt(float(dr))
    out = np.full((B, Hq, M), -np.inf)
    for b in range(B):
        m = int(n_spans[b])
        for h in range(Hq):
            s = np.zeros(m)
            for i in range(dr):
                s = s + qp[b, h, i] * kr[b, h, :m, i]
            out[b, h, :m] = s * scale + span_logsize[b, :m]
    return out


def gate(x) -> np.ndarray:
    """The routing gate alpha~ = sig(x) of eq. routing_gate."""
    x = np.asarray(x, dtype=np.float64)
    return 1.0 / (1.0 + np.exp(-x))


def threshold_logit(tau) -> np.ndarray:
    """x-space threshold of eq. zoom_decision: sig(x) > tau exactly when x > ln(tau / (1 - tau))."""
    tau = np.asarray(tau, dtype=np.float64)
    return np.log(tau) - np.log1p(-tau)


def gated_selection(x, thresholds, span_len, n_spans, n_kv_heads: int, max_zoom: int,
                    budget_tokens: int) -> np.ndarray:
    """Spans to expand per (b, KV head): eq. zoom_decision, then the budget cap of Sec. 3.3.

    x [B][Hq][M] pre-sigmoid gates, thresholds [Hq] in x space.  Listed in
    expansion order; unused slots hold -1.  Returns int32 [B][Hkv][max_zoom].
    """
    B, Hq, M = x.shape
    G = Hq // n_kv_heads
    sel = np.full((B, n_kv_heads, max_zoom), -1, dtype=np.int32)
    for b in range(B):
        m = int(n_spans[b])
        for g in range(n_kv_heads):
            heads = range(g * G, (g + 1) * G)
            cands = []
            for S in range(m):
                votes = [x[b, h, S] for h in heads if x[b, h, S] > thresholds[h]]
                if votes:
                    cands.append((max(votes), S))
            cands.sort(key=lambda c: (-c[0], c[1]))
            used, chosen = 0, []
            for _, S in cands:
                if len(chosen) == max_zoom or used + int(span_len[b, S]) > budget_tokens:
                    break
                chosen.append(S)
                used += int(span_len[b, S])
            sel[b, g, :len(chosen)] = chosen
    return sel


def decode_step_gated(q, anchor_k, anchor_v, n_anchors, sum_k, sum_v, n_spans, span_len,
                      span_logsize, factors, block_off, proj, sum_route, thresholds, *,
                      rank: int, max_zoom: int, budget_tokens: int, softmax_scale: float,
                      dtype: str, block_rank=None) -> dict:
    """One decode step under the learned selection rule.

    The routing (projection, gate, threshold, budget) decides which spans are
    expanded; the attention is the same mixed-resolution softmax as for the
    identity routing, with unexpanded spans entering as their coarse mean key
    and value, score scale * q . k_bar + ln|S| (Sec. 3.3).
    """
    qf = widen(q, dtype)
    qp = project_queries(qf, widen(proj, dtype))
    x = gate_logits(qp, widen(sum_route, dtype), np.asarray(span_logsize, np.float64), n_spans)
    Hkv = np.asarray(sum_k).shape[1]
    sel = gated_selection(x, np.asarray(thresholds, np.float64), span_len, n_spans, Hkv,
                          max_zoom, budget_tokens)
    coarse = routing_logits(qf, widen(sum_k, dtype), np.asarray(span_logsize, np.float64),
                            n_spans, softmax_scale)
    out = zoom_attend(q, anchor_k, anchor_v, n_anchors, sum_v, n_spans, span_len, factors,
                      block_off, sel, coarse, rank=rank, softmax_scale=softmax_scale,
                      dtype=dtype, block_rank=block_rank)
    return {"sel": sel, "out": out, "gate_logits": x, "q_proj": qp}


# ---------------------------------------------------------------------------
# prefill-side builder: segmentation, surprisal-weighted summaries, factors
# (Sec. 3.1; Sec. 3.2 eqs. surprisal_weight, key_svd and the summary paragraph)
# ---------------------------------------------------------------------------
#
# Readings (listed with their reasons in the design notes):
#
# * mu and sigma are the mean and the population standard deviation of the
#   sequence's n surprisal values.  So that the boundary decisions are exact,
#   both sums have one fixed order: 1024 partial sums, partial j adding tokens
#   j, j + 1024, j + 2048, ... in increasing order (float64), then the partials
#   combined by halving (partial j += partial j + h for h = 512, 256, ..., 1).
#   mu = S1 / n; sigma = sqrt(S2 / n) with S2 over (H_t - mu)^2, each product
#   and difference rounded on its own (no fused multiply-add); the threshold is
#   mu + (alpha * sigma) in float64, and H_t (float32) is compared in float64.
# * Anchors: the boundary tokens, the last `window` tokens (the local window),
#   and the tokens of any run between neighbouring anchors shorter than
#   `min_span` (short spans stay at full resolution).  The sequence start and
#   end act as neighbours for the first and last run.  Spans: the remaining
#   runs, in token order.
# * A span whose surprisal sums to zero (or less) gets uniform weights.
# * The factors of a span are its truncated SVD of rank min(|S|, d, R_max)
#   (eq. key_svd); stored with the rank rounded up to the 16-byte granule, the
#   extra components zero.

_SEG_LANES = 1024


def _fixed_order_sum(x) -> float:
    """Sum in the fixed order of the segmentation reading (1024 strided partials, halving)."""
    x = np.asarray(x, dtype=np.float64)
    part = np.zeros(_SEG_LANES)
    for j in range(_SEG_LANES):
        acc = 0.0
        for v in x[j::_SEG_LANES]:
            acc = acc + v
        part[j] = acc
    h = _SEG_LANES // 2
    while h >= 1:
        part[:h] = part[:h] + part[h:2 * h]
        h //= 2
    return float(part[0])


def surprisal_threshold(H, n: int, alpha: float):
    """(mu, sigma, mu + alpha sigma) of the first n surprisal values (Sec. 3.1)."""
    h = np.asarray(H, dtype=np.float32)[:n].astype(np.float64)
    mu = _fixed_order_sum(h) / n
    dev = h - mu
    sq = dev * dev
    sigma = float(np.sqrt(_fixed_order_sum(sq) / n))
    return mu, sigma, mu + alpha * sigma


def segment(H, n: int, alpha: float, min_span: int, window: int):
    """Anchors and spans of one sequence (Sec. 3.1).

    Returns (anchors: sorted token indices, spans: list of (start, length))."""
    if n <= 0:
        return [], []
    _, _, thr = surprisal_threshold(H, n, alpha)
    h = np.asarray(H, dtype=np.float32)[:n].astype(np.float64)
    anchor = h > thr
    anchor[max(0, n - window):n] = True
    spans = []
    t = 0
    while t < n:
        if anchor[t]:
            t += 1
            continue
        s = t
        while t < n and not anchor[t]:
            t += 1
        if t - s >= min_span:
            spans.append((s, t - s))
        else:
            anchor[s:t] = True
    return [int(i) for i in np.flatnonzero(anchor)], spans


def weighted_summary(X, H):
    """sum_t w_t X_t with w_t = H_t / sum_k H_k over the span (eq. surprisal_weight)."""
    X = np.asarray(X, dtype=np.float64)
    h = np.asarray(H, dtype=np.float32).astype(np.float64)
    tot = h.sum()
    w = h / tot if tot > 0 else np.full(h.shape, 1.0 / h.size)
    return w @ X


def truncated_svd(X, r_max: int):
    """Rank min(|S|, d, R_max) truncated SVD of a span matrix (eq. key_svd): (U, sigma, Vt)."""
    X = np.asarray(X, dtype=np.float64)
    U, s, Vt = np.linalg.svd(X, full_matrices=False)
    r = min(X.shape[0], X.shape[1], int(r_max))
    return U[:, :r], s[:r], Vt[:r]


def narrow(x, dtype: str) -> np.ndarray:
    """float64 -> stored values: float32 by round-to-nearest-even, then for 'bf16' the
    upper 16 bits after round-to-nearest-even (returned as uint16 bit patterns)."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    if dtype == "f32":
        return f
    if dtype != "bf16":
        raise ValueError(f"unknown storage dtype {dtype!r}")
    u = f.view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def build_layer_cache(keys, values, surprisal, n_tokens, *, alpha: float, min_span: int,
                      window: int, r_max: int, dtype: str) -> dict:
    """One layer's stored cache from its token keys/values and surprisal (Sec. 3.1, 3.2).

    keys/values [B][Hkv][N][d] stored values, surprisal [B][N] float32.  Segments each
    sequence, copies the anchor rows, forms the surprisal-weighted span summaries and
    each span's truncated SVD, and lays the factors out one block per (b, g, S), both
    sides of stored rank ceil(r / granule) * granule, blocks 256-byte aligned.  Returns
    the cache arrays (the decode step's inputs, q excepted) and the segmentation."""
    B, Hkv, _, d = np.asarray(keys).shape
    _, e = _elem(dtype)
    gran = 16 // e
    segs = [segment(surprisal[b], int(n_tokens[b]), alpha, min_span, window) for b in range(B)]
    A = max([len(a) for a, _ in segs] + [1])
    M = max([len(s) for _, s in segs] + [1])
    st = np.uint16 if dtype == "bf16" else np.float32
    out = {"anchor_k": np.zeros((B, Hkv, A, d), st), "anchor_v": np.zeros((B, Hkv, A, d), st),
           "sum_k": np.zeros((B, Hkv, M, d), st), "sum_v": np.zeros((B, Hkv, M, d), st),
           "n_anchors": np.array([len(a) for a, _ in segs], np.int32),
           "n_spans": np.array([len(s) for _, s in segs], np.int32),
           "span_len": np.ones((B, M), np.int32), "span_logsize": np.zeros((B, M)),
           "block_off": np.zeros((B, Hkv, M), np.int64), "block_rank": np.zeros((B, Hkv, M), np.int32)}
    chunks, pos = [], 0
    for b, (anchors, spans) in enumerate(segs):
        h = np.asarray(surprisal[b], dtype=np.float32)
        for S, (s0, L) in enumerate(spans):
            out["span_len"][b, S] = L
            out["span_logsize"][b, S] = np.log(L)
        for g in range(Hkv):
            out["anchor_k"][b, g, :len(anchors)] = np.asarray(keys)[b, g, anchors]
            out["anchor_v"][b, g, :len(anchors)] = np.asarray(values)[b, g, anchors]
            for S, (s0, L) in enumerate(spans):
                block = []
                r = min(L, d, r_max)
                rs = -(-r // gran) * gran
                for src, name in ((keys, "k"), (values, "v")):
                    X = widen(np.asarray(src)[b, g, s0:s0 + L], dtype)
                    out["sum_" + name][b, g, S] = narrow(weighted_summary(X, h[s0:s0 + L]), dtype)
                    U, sig, Vt = truncated_svd(X, r_max)
                    Up = np.zeros((L, rs)); Up[:, :r] = U
                    sp = np.zeros(rs); sp[:r] = sig
                    Vp = np.zeros((rs, d)); Vp[:r] = Vt
                    block += [Up.ravel(), sp, Vp.ravel()]
                raw = narrow(np.concatenate(block), dtype).tobytes()
                raw += b"\0" * (-len(raw) % 256)
                out["block_off"][b, g, S] = pos
                out["block_rank"][b, g, S] = rs | (rs << 16)
                chunks.append(raw)
                pos += len(raw)
    out["factors"] = np.frombuffer(b"".join(chunks) or b"\0" * 256, dtype=np.uint8).copy()
    out["segments"] = segs
    return out
