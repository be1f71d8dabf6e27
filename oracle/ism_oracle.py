"""fp64 CPU oracle of ISM attention (arXiv 2408.00539). TEST INFRASTRUCTURE.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
use this module; the product path never does. Numpy only; no blocking, fusion
or reordering beyond what the definitions below state.

Readings of the paper fixed here (each is also listed in the design notes):

* Eq. 5 gives, for 1-indexed token j, the last key f(j) it may see. In the
  0-indexed packed layout used throughout, token j of segment g = [a_g, c_g)
  has the inclusive bound ``lim(j) = c_g - 1`` if g is a query segment and
  ``lim(j) = j`` if it is an answer segment; key i is visible to j iff
  ``s_b <= i <= lim(j)`` where s_b is the start of j's dialogue.
  (``f(j) = lim(j) + 1`` with ``j_paper = j + 1``.)
* The prompt P has no case of its own: Eq. 5's first case covers P and Q_1
  together, so the caller passes P followed by Q_1 as one query segment.
* Segments that are not strictly alternating are allowed; each query-flagged
  segment is its own bidirectional block (adjacent query segments are not
  merged), an answer segment is causal. All-answer gives the causal mask.
* Several dialogues packed along one token axis never see each other.
* The analysed update of Eq. 4 is the linear surrogate; the method as
  integrated (Sec. 2.3) is ordinary softmax attention with the ISM mask, so the
  oracle computes softmax(scale * Q K^T + M) V with M = 0 / -inf.
* Multi-head: heads are independent; with Hq query heads and Hkv key/value
  heads, query head h reads key/value head h // (Hq // Hkv).
* LSE is the natural-log log-sum-exp of the scaled, masked scores.

Array conventions: q [T, Hq, d], k and v [T, Hkv, d], o [T, Hq, d],
lse [Hq, T]; segment metadata ``cu_seqlens`` [B+1], ``cu_segs`` [S+1],
``seg_is_query`` [S]; every cu_seqlens entry is also a cu_segs entry.
"""

from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_ROW_BLOCK = 1024


# --------------------------------------------------------------------------
# The mask rule (Eq. 5)
# --------------------------------------------------------------------------

def lim(cu_seqlens, cu_segs, seg_is_query):
    """Inclusive visibility bound per token, from Eq. 5 (0-indexed).

    For a query segment [a, c) every token gets c - 1 (first two cases of
    Eq. 5: f(j) = m_{q_k}, the end of the current query); for an answer
    segment every token j gets j (third case, f(j) = j).
    """
    cu_segs = np.asarray(cu_segs, dtype=np.int64)
    isq = np.asarray(seg_is_query).astype(bool)
    T = int(cu_segs[-1])
    out = np.empty(T, dtype=np.int64)
    for g in range(len(isq)):
        a, c = int(cu_segs[g]), int(cu_segs[g + 1])
        if isq[g]:
            out[a:c] = c - 1
        else:
            out[a:c] = np.arange(a, c)
    return out


def seq_index(cu_seqlens, T=None):
    """Dialogue index of every token of the packed axis."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    T = int(cu[-1]) if T is None else T
    out = np.empty(T, dtype=np.int64)
    for b in range(len(cu) - 1):
        out[cu[b]:cu[b + 1]] = b
    return out


def mask_dense(cu_seqlens, cu_segs, seg_is_query, b):
    """Dense boolean mask of dialogue b: M[j, i] = (s_b <= i <= lim(j)).

    Indices are local to the dialogue (row j - s_b, column i - s_b).
    """
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    s, e = int(cu[b]), int(cu[b + 1])
    L = lim(cu_seqlens, cu_segs, seg_is_query)[s:e] - s
    cols = np.arange(e - s)
    return cols[None, :] <= L[:, None]


def mask_eq5(m_p, q_lens, a_lens):
    """Literal transcription of Eq. 5 for ONE dialogue, 1-indexed.

    The dialogue is [P, Q_1, A_1, ..., Q_N, (A_N)] with |P| = m_p,
    |Q_k| = q_lens[k-1] and |A_k| = a_lens[k-1]; ``a_lens`` may be one
    shorter than ``q_lens`` (dialogue ending with a query). Boundaries follow
    the paper's definitions: m_{a_0} := m_p, m_{q_k} = m_{a_{k-1}} + |Q_k|,
    m_{a_k} = m_{q_k} + |A_k|. Returns mask[j-1, i-1] = (i <= f(j)).
    """
    N = len(q_lens)
    assert len(a_lens) in (N, N - 1)
    m_q = [None] * (N + 1)
    m_a = [None] * (N + 1)
    m_a[0] = m_p
    for k in range(1, N + 1):
        m_q[k] = m_a[k - 1] + q_lens[k - 1]
        m_a[k] = m_q[k] + (a_lens[k - 1] if k - 1 < len(a_lens) else 0)
    n = m_a[N]

    def f(j):
        if 1 <= j <= m_q[1]:
            return m_q[1]
        for k in range(2, N + 1):
            if m_a[k - 1] < j <= m_q[k]:
                return m_q[k]
        for k in range(1, N + 1):
            if m_q[k] < j <= m_a[k]:
                return j
        raise ValueError(f"token {j} is in no case of Eq. 5")

    M = np.zeros((n, n), dtype=bool)
    for j in range(1, n + 1):
        fj = f(j)
        for i in range(1, n + 1):
            M[j - 1, i - 1] = i <= fj
    return M


def visible_pairs(cu_seqlens, cu_segs, seg_is_query):
    """|vis| = number of visible (query row, key) pairs per query head."""
    L = lim(cu_seqlens, cu_segs, seg_is_query)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    s = cu[seq_index(cu_seqlens, len(L))]
    return int(np.sum(L - s + 1))


# --------------------------------------------------------------------------
# Forward: softmax(scale Q K^T + M) V, per (dialogue, query head)
# --------------------------------------------------------------------------

def _softmax_attend(qh, kh, vh, vis, scale):
    """Masked softmax attention of query rows qh over keys kh/vh (fp64).

    vis[r, i] tells whether key i is visible to row r. Returns (o, lse).
    """
    S = scale * (qh @ kh.T)
    S = np.where(vis, S, -np.inf)
    m = S.max(axis=1, keepdims=True)
    E = np.exp(S - m)
    l = E.sum(axis=1, keepdims=True)
    P = E / l
    return P @ vh, (m + np.log(l))[:, 0]


def _group(hq, hkv):
    assert hq % hkv == 0, "Hq must be a multiple of Hkv"
    return hq // hkv


def fwd_rows(q, k, v, cu_seqlens, cu_segs, seg_is_query, scale, b, h,
             rows=None):
    """Forward of dialogue b, query head h, for local row range ``rows``.

    Returns (o [r, d], lse [r]) in fp64 for local rows r0..r1-1.
    """
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    s, e = int(cu[b]), int(cu[b + 1])
    r0, r1 = (0, e - s) if rows is None else rows
    g = h // _group(q.shape[1], k.shape[1])
    L = lim(cu_seqlens, cu_segs, seg_is_query)[s:e] - s
    kh = np.asarray(k[s:e, g], dtype=np.float64)
    vh = np.asarray(v[s:e, g], dtype=np.float64)
    cols = np.arange(e - s)
    o = np.empty((r1 - r0, q.shape[2]))
    lse = np.empty(r1 - r0)
    for a in range(r0, r1, _ROW_BLOCK):
        c = min(a + _ROW_BLOCK, r1)
        qh = np.asarray(q[s + a:s + c, h], dtype=np.float64)
        vis = cols[None, :] <= L[a:c, None]
        o[a - r0:c - r0], lse[a - r0:c - r0] = _softmax_attend(
            qh, kh, vh, vis, scale)
    return o, lse


def fwd(q, k, v, cu_seqlens, cu_segs, seg_is_query, scale, pairs=None,
        workers=1):
    """Full forward (or the listed (dialogue, head) pairs), fp64.

    Returns (o [T, Hq, d], lse [Hq, T]); entries of pairs not computed are NaN.
    """
    T, hq, d = q.shape
    nb = len(cu_seqlens) - 1
    if pairs is None:
        pairs = [(b, h) for b in range(nb) for h in range(hq)]
    o = np.full((T, hq, d), np.nan)
    lse = np.full((hq, T), np.nan)
    cu = np.asarray(cu_seqlens, dtype=np.int64)

    def one(bh):
        b, h = bh
        ob, lb = fwd_rows(q, k, v, cu_seqlens, cu_segs, seg_is_query, scale,
                          b, h)
        s, e = int(cu[b]), int(cu[b + 1])
        o[s:e, h] = ob
        lse[h, s:e] = lb

    _run(one, pairs, workers)
    return o, lse


def _run(fn, items, workers):
    if workers <= 1:
        for it in items:
            fn(it)
    else:
        with ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(fn, items))


# --------------------------------------------------------------------------
# Backward: textbook softmax-attention gradients
# --------------------------------------------------------------------------

def _bwd_one(q, k, v, do, L, s, e, hs, g, scale):
    """Gradients of one dialogue [s, e) for query heads hs sharing kv head g.

    Follows the chain rule of o = softmax(scale q k^T + M) v step by step:
    dV = P^T dO; dP = dO V^T; D_j = sum_i P_ji dP_ji; dS = P o (dP - D);
    dQ = scale dS K; dK = scale dS^T Q. Returns (dq [n, len(hs), d], dk, dv).
    """
    n = e - s
    kh = np.asarray(k[s:e, g], dtype=np.float64)
    vh = np.asarray(v[s:e, g], dtype=np.float64)
    cols = np.arange(n)
    dq = np.zeros((n, len(hs), q.shape[2]))
    dk = np.zeros((n, q.shape[2]))
    dv = np.zeros((n, q.shape[2]))
    for t, h in enumerate(hs):
        for a in range(0, n, _ROW_BLOCK):
            c = min(a + _ROW_BLOCK, n)
            qh = np.asarray(q[s + a:s + c, h], dtype=np.float64)
            doh = np.asarray(do[s + a:s + c, h], dtype=np.float64)
            vis = cols[None, :] <= L[a:c, None]
            S = np.where(vis, scale * (qh @ kh.T), -np.inf)
            E = np.exp(S - S.max(axis=1, keepdims=True))
            P = E / E.sum(axis=1, keepdims=True)
            dv += P.T @ doh
            dP = doh @ vh.T
            D = np.sum(P * dP, axis=1, keepdims=True)
            dS = P * (dP - D)
            dq[a:c, t] = scale * (dS @ kh)
            dk += scale * (dS.T @ qh)
    return dq, dk, dv


def bwd(q, k, v, do, cu_seqlens, cu_segs, seg_is_query, scale, pairs=None,
        workers=1):
    """Gradients (dq [T,Hq,d], dk [T,Hkv,d], dv [T,Hkv,d]) in fp64.

    ``pairs`` lists (dialogue, kv head) to compute; the rest is NaN.
    """
    T, hq, d = q.shape
    hkv = k.shape[1]
    G = _group(hq, hkv)
    nb = len(cu_seqlens) - 1
    if pairs is None:
        pairs = [(b, g) for b in range(nb) for g in range(hkv)]
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    Lall = lim(cu_seqlens, cu_segs, seg_is_query)
    dq = np.full((T, hq, d), np.nan)
    dk = np.full((T, hkv, d), np.nan)
    dv = np.full((T, hkv, d), np.nan)

    def one(bg):
        b, g = bg
        s, e = int(cu[b]), int(cu[b + 1])
        hs = list(range(g * G, (g + 1) * G))
        a, kk, vv = _bwd_one(q, k, v, do, Lall[s:e] - s, s, e, hs, g, scale)
        dq[s:e, g * G:(g + 1) * G] = a
        dk[s:e, g] = kk
        dv[s:e, g] = vv

    _run(one, pairs, workers)
    return dq, dk, dv


# --------------------------------------------------------------------------
# Inference with KV-cache reuse (Sec. 2.3)
# --------------------------------------------------------------------------

def prefill_cached(k_hist, v_hist, q_new, k_new, v_new, scale,
                   new_is_query=True):
    """One dialogue's new segment against the cached history C_h.

    Sec. 2.3: reuse C_h, compute C_q from the new tokens, concatenate
    [C_h; C_q]. For a query segment Q_n (Eq. 5 first two cases, f = m_{q_n}
    for every token of Q_n) each new row sees every key of the concatenation.
    For an answer segment (``new_is_query=False``; Eq. 5 third case,
    f(j) = j) new row r sees the history and the new rows 0..r: the causal
    mask of Eq. 2 restricted to these rows. Shapes: k_hist/v_hist
    [C, Hkv, d], q_new [L, Hq, d], k_new/v_new [L, Hkv, d]. Returns
    (o [L, Hq, d], lse [Hq, L], k_cat, v_cat).
    """
    k_cat = np.concatenate([k_hist, k_new], axis=0).astype(np.float64)
    v_cat = np.concatenate([v_hist, v_new], axis=0).astype(np.float64)
    L, hq, d = q_new.shape
    G = _group(hq, k_cat.shape[1])
    o = np.empty((L, hq, d))
    lse = np.empty((hq, L))
    C = k_hist.shape[0]
    if new_is_query:
        vis = np.ones((L, C + L), dtype=bool)
    else:
        vis = np.arange(C + L)[None, :] <= C + np.arange(L)[:, None]
    for h in range(hq):
        qh = np.asarray(q_new[:, h], dtype=np.float64)
        o[:, h], lse[h] = _softmax_attend(qh, k_cat[:, h // G],
                                          v_cat[:, h // G], vis, scale)
    return o, lse, k_cat, v_cat


def decode_step(k_cache, v_cache, q, k, v, scale):
    """One answer token: append its key/value, then attend to every cached
    key including its own (Eq. 5 third case, f(j) = j).

    Shapes: k_cache/v_cache [p, Hkv, d] (the p earlier tokens), q [Hq, d],
    k/v [Hkv, d]. Returns (o [Hq, d], lse [Hq], k_cache', v_cache').
    """
    k2 = np.concatenate([k_cache, k[None]], axis=0).astype(np.float64)
    v2 = np.concatenate([v_cache, v[None]], axis=0).astype(np.float64)
    hq, d = q.shape
    G = _group(hq, k2.shape[1])
    o = np.empty((hq, d))
    lse = np.empty(hq)
    vis = np.ones((1, k2.shape[0]), dtype=bool)
    for h in range(hq):
        oh, lh = _softmax_attend(np.asarray(q[h:h + 1], dtype=np.float64),
                                 k2[:, h // G], v2[:, h // G], vis, scale)
        o[h], lse[h] = oh[0], lh[0]
    return o, lse, k2, v2


# --------------------------------------------------------------------------
# Who sees a key, and closed forms at Q = 0
# --------------------------------------------------------------------------

def seer(cu_seqlens, cu_segs, seg_is_query):
    """First token of each key's dialogue that sees the key under Eq. 5:
    seer(i) = min { j in i's dialogue : i <= lim(j) }.

    lim is non-decreasing inside a dialogue (a query segment's tokens all map
    to the segment end, which is below the next token; an answer token maps
    to itself), so the minimum is the first j whose lim reaches i; the
    monotonicity is asserted, not assumed.
    """
    L = lim(cu_seqlens, cu_segs, seg_is_query)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    out = np.empty_like(L)
    for b in range(len(cu) - 1):
        s, e = int(cu[b]), int(cu[b + 1])
        Lb = L[s:e]
        assert np.all(np.diff(Lb) >= 0), "lim must be non-decreasing in a dialogue"
        out[s:e] = s + np.searchsorted(Lb, np.arange(s, e), side="left")
    return out


def _visible_counts(cu_seqlens, cu_segs, seg_is_query):
    """n_j = lim(j) - s_b + 1 visible keys per token, and s_b per token."""
    L = lim(cu_seqlens, cu_segs, seg_is_query)
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    sb = cu[seq_index(cu_seqlens, len(L))]
    return L - sb + 1, sb, L


def _range_sums(x, sb, L):
    """sum_{i = sb[j]}^{L[j]} x[i] for every j, through fp64 prefix sums."""
    c = np.concatenate([np.zeros((1,) + x.shape[1:]), np.cumsum(x, axis=0)])
    return c[L + 1] - c[sb]


def uniform_fwd(v, cu_seqlens, cu_segs, seg_is_query):
    """Forward at Q = 0 (any scale): every visible score is 0, so row j's
    softmax weights are 1 / n_j on its n_j = lim(j) - s_b + 1 visible keys
    (Eq. 5) and the outputs are O_j = mean(V[s_b .. lim(j)]),
    LSE_j = ln n_j. v [T, Hkv, d]; returns (o [T, Hkv, d], lse [T]): query
    head h takes o[:, h // (Hq / Hkv)], every head the same lse.
    """
    n, sb, L = _visible_counts(cu_seqlens, cu_segs, seg_is_query)
    v = np.asarray(v, dtype=np.float64)
    o = _range_sums(v, sb, L) / n[:, None, None]
    return o, np.log(n.astype(np.float64))


def uniform_bwd(k, v, hq, scale, cu_seqlens, cu_segs, seg_is_query,
                row_weight=None):
    """Gradients at Q = 0 and dO = 1 (all ones), from the chain rule of the
    backward with P_ji = 1 / n_j on the visible keys:
    dP_ji = dO_j . V_i = r_i (the row sum of V_i); D_j = mean of r over j's
    keys; dS_ji = (r_i - D_j) / n_j; dQ_j = scale sum_i dS_ji K_i;
    dK = scale dS^T Q = 0; dV_i = sum over the G query heads of kv head g and
    the rows j that see i (seer(i) <= j < e_b) of P_ji.

    ``row_weight`` [T] replaces the weight 1 / n_j in dV only (a test may
    pass the weights rounded as a device rounds them). Returns
    (dq [T, Hq, d], dk [T, Hkv, d], dv [T, Hkv, d]).
    """
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    T, hkv, d = k.shape
    G = _group(hq, hkv)
    n, sb, L = _visible_counts(cu_seqlens, cu_segs, seg_is_query)
    r = v.sum(axis=2)                                   # [T, hkv]
    D = _range_sums(r, sb, L) / n[:, None]              # [T, hkv]
    sum_rk = _range_sums(r[:, :, None] * k, sb, L)      # [T, hkv, d]
    sum_k = _range_sums(k, sb, L)
    dq_kv = scale * (sum_rk - D[:, :, None] * sum_k) / n[:, None, None]
    dq = np.repeat(dq_kv, G, axis=1)
    w = 1.0 / n if row_weight is None else np.asarray(row_weight, np.float64)
    # dV_i = G * sum_{j = seer(i)}^{e_b - 1} w_j: suffix sums inside each dialogue
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    se = seer(cu_seqlens, cu_segs, seg_is_query)
    eb = cu[seq_index(cu_seqlens, T) + 1]
    c = np.concatenate([[0.0], np.cumsum(w)])
    dv1 = G * (c[eb] - c[se])
    dv = np.repeat(dv1[:, None, None], hkv, axis=1) * np.ones((1, 1, d))
    return dq, np.zeros_like(k), dv


# --------------------------------------------------------------------------
# Brute force (tiny inputs): per-element loops of Eq. 4 with softmax
# --------------------------------------------------------------------------

def brute_force_fwd(q, k, v, cu_seqlens, cu_segs, seg_is_query, scale):
    """Pure-Python loops: for every token j, find its segment and dialogue,
    apply Eq. 5 directly, and form the softmax-weighted sum of values.
    Independent of :func:`lim` and of numpy's vector ops. Tiny inputs only.
    """
    T, hq, d = q.shape
    G = hq // k.shape[1]
    cu = [int(x) for x in cu_seqlens]
    cs = [int(x) for x in cu_segs]
    isq = [bool(x) for x in seg_is_query]
    o = [[[0.0] * d for _ in range(hq)] for _ in range(T)]
    lse = [[0.0] * T for _ in range(hq)]
    for j in range(T):
        b = max(x for x in range(len(cu) - 1) if cu[x] <= j)
        g = max(x for x in range(len(isq)) if cs[x] <= j)
        bound = cs[g + 1] - 1 if isq[g] else j
        keys = list(range(cu[b], bound + 1))
        for h in range(hq):
            kv = h // G
            sc = []
            for i in keys:
                dot = 0.0
                for t in range(d):
                    dot += float(q[j][h][t]) * float(k[i][kv][t])
                sc.append(scale * dot)
            mx = max(sc)
            w = [math.exp(x - mx) for x in sc]
            tot = sum(w)
            for t in range(d):
                acc = 0.0
                for wi, i in zip(w, keys):
                    acc += wi * float(v[i][kv][t])
                o[j][h][t] = acc / tot
            lse[h][j] = mx + math.log(tot)
    return np.array(o), np.array(lse)
