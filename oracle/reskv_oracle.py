"""ResKV oracle: a plain, slow, fp64 statement of what the hot path computes.

This module is TEST INFRASTRUCTURE. Only the test suite, the package smoke
check and the CPU-baseline leg of the benchmark may import it. The product
path (the HIP library and its Python binding) never calls it and shares no
code with it: no kernels, headers, helpers, tables or pre/post-processing.
Inputs come from the seeded generators, which hold none of the method's
arithmetic; everything below is written from the paper's definitions.

Every floating-point step runs in float64. Inputs stored in bf16 or fp32 are
exactly representable in float64, so they are upcast without loss.

Paper map (section / equation / algorithm):
  full attention ............ Sec. 3.1, attention equation
  eviction attention ........ Sec. 3.2, eviction equation
  Z / N statistics .......... Sec. 4.2, (Z, N) definition; App. A.1 decomposition
  main selection ............ Sec. 5.2, main-selection equation
  observation-window scores . App. B.2.2 (SnapKV rule: observation window,
                              average pooling with kernel 5, recent protection)
  residual partition ........ Sec. 5.3, key-space partition objective, solved
                              with Lloyd iterations seeded from the
                              highest-scored evicted tokens (App. B.3)
  residual summary .......... Sec. 5.3, summary equation (mean key, mean value,
                              count); App. B.3 (count exponent beta)
  shared-softmax decode ..... Sec. 5.4, residual-logit, denominator, numerator
                              and output equations; App. D, Algorithm 2
  dynamic gate .............. Sec. 5.5.2, gate equation; App. A.3
  validation proxy .......... Sec. 5.5.1, validation-loss and margin
                              equations; App. D, Algorithm 1; App. B.3
                              (grid, 96 fit / 32 validation queries, delta)
  two-branch decode ......... Sec. 6.1 (main branch and residual branch
                              merged through log-sum-exp statistics);
                              Sec. 6.6 ablation table (separate
                              normalisations, reading R25)
  AdaKV allocation .......... App. B.2.2 compared methods (cross-head budget
                              allocation from SnapKV scores, safeguard 0.2;
                              reading R26)
  alternative scorers ....... App. B.2.2 compared methods: H2O (accumulated
                              attention of the observation queries, recent
                              64) and TOVA (last-token window, recent 1),
                              feeding the same selection and residual path

Readings taken where the paper is silent (each also listed in the design
notes of the repository):
  R1  window scores use causal masking inside the observation window and each
      window row is normalised over every key it can see;
  R2  scores of the query heads that share a KV head are summed;
  R3  pooling is a centred 5-tap sum with zero padding over the scored range;
  R4  the protected recent window is |P| = min(recent_window, m) last tokens and
      only the positions before it are scored;
  R6  score ties are broken by the lower position;
  R7  Lloyd seeds are the evicted tokens of rank k_top .. k_top+r-1 in the
      selection order; centre j is the j-th seed by ascending position;
      assignment ties go to the lower centre index;
  R8  one Lloyd iteration is one assignment plus one update; the entries come
      from the T-th assignment;
  R9  an empty cluster keeps its centre; a final count of 0 marks the entry
      empty (log-count -inf, value 0) and it contributes nothing at decode;
  R10 mean key and mean value are stored in the cache dtype, rounded once to
      nearest-even; log-counts are fp32;
  R12 single-token residual entries reproduce full attention only with the
      gate held at 1 (g_min = 1);
  R13 p_max covers every main slot, including tokens appended during decode;
  R19 a grid fraction f gives the candidate count r = floor(f * b + 1/2);
  R20 the validation queries are the last `val_rows` window positions of
      every query head of the group, the fit queries the leading ones (96/32
      at G = 4, w = 32, val_rows = 8); the fit queries alone score the tokens;
  R21 validation queries are evaluated like decode queries: o_S attends to
      the whole prefix [0, s), the candidate output to the whole compressed
      cache, with the decode gate at the scalar threshold tau;
  R22 the loss is the mean over validation queries of the squared L2 error;
      among r > 0 the smallest loss wins, ties to the smaller r;
  R23 H2O's accumulated attention of the observation queries is the raw
      window score (R1, R2) without pooling (kernel 1), with 64 protected
      recent tokens;
  R24 TOVA's last-token window is w = 1 (the last prefill query of every
      head of the group, summed by R2), without pooling, with 1 protected
      recent token;
  R25 the ablation with separate main and residual normalisations mixes the
      two separately normalised branch outputs by the gate,
      (1 - g) o_main + g o_res (g = 0 without populated entries); the paper
      does not print its formula, so this variant is parity unpinned against
      the paper and pinned only to its own limits;
  R26 AdaKV reallocates the top-k (scored) part of the main budgets of the KV
      heads of one (layer, sequence): every head keeps floor(alpha * k) of
      its own best tokens (alpha = the safeguard), the remaining slots follow
      one ranking of all heads' other tokens (score, then head, then
      position), each head capped by its slot capacity; recent protection
      and residual counts stay per head as in the uniform split.
"""

import math

import numpy as np

__all__ = [
    "round_to_dtype", "full_attention", "evict_attention", "zn_stats",
    "decode_branches", "merge_branches", "adakv_allocate", "build_heads_adakv",
    "window_raw_scores", "pool", "pool5", "scored_length", "select_main", "select_top",
    "lloyd", "lloyd_objective", "assign_nearest", "residual_entries",
    "build_head", "build_cache", "gate_value", "decode_head", "decode",
    "candidate_counts", "proxy_choice", "validation_proxy",
]

_F64 = np.float64


# --------------------------------------------------------------------------
# storage rounding of the oracle's own outputs (R10)
# --------------------------------------------------------------------------

def _round_bf16(x):
    """Round float64 values to the nearest bf16 value, ties to even.

    bf16 keeps 8 significant bits; the quantum of a value with binary exponent
    e (x = f * 2**e, 0.5 <= |f| < 1) is 2**(e-8), floored at the subnormal
    quantum 2**-133. Dividing by a power of two is exact in float64, and
    np.rint rounds halves to even.
    """
    x = np.asarray(x, dtype=_F64)
    out = np.zeros_like(x)
    nz = (x != 0) & np.isfinite(x)
    _, e = np.frexp(x[nz])
    q = np.maximum(e - 8, -133).astype(_F64)
    scale = np.exp2(q)
    out[nz] = np.rint(x[nz] / scale) * scale
    out[~np.isfinite(x)] = x[~np.isfinite(x)]
    big = np.abs(out) > 3.3895313892515355e38  # largest finite bf16
    out[big] = np.sign(out[big]) * np.inf
    return out


def round_to_dtype(x, dtype):
    """Value of float64 `x` after storage in `dtype` ('bf16' or 'f32')."""
    if dtype == "bf16":
        return _round_bf16(x)
    if dtype == "f32":
        return np.asarray(x, dtype=_F64).astype(np.float32).astype(_F64)
    raise ValueError(dtype)


# --------------------------------------------------------------------------
# plain attention definitions (Sec. 3.1, Sec. 3.2, Sec. 4.2)
# --------------------------------------------------------------------------

def _logits(q, K):
    d = K.shape[-1]
    return (np.asarray(K, _F64) @ np.asarray(q, _F64)) / math.sqrt(d)


def full_attention(q, K, V):
    """o = softmax(q K^T / sqrt(d)) V  (Sec. 3.1, attention equation)."""
    a = _logits(q, K)
    w = np.exp(a - a.max())
    return (w @ np.asarray(V, _F64)) / w.sum()


def evict_attention(q, K, V, kept):
    """Attention over the kept rows only (Sec. 3.2, eviction equation)."""
    kept = np.asarray(kept, dtype=np.int64)
    return full_attention(q, np.asarray(K)[kept], np.asarray(V)[kept])


def zn_stats(q, K, V, subset):
    """(log Z_T, N_T / Z_T-free form) for a token subset T (Sec. 4.2).

    Returns (Z, N) with Z = sum_{p in T} e^{a_p}, N = sum_{p in T} e^{a_p} v_p,
    both scaled by e^{-c} for the shift c returned as the third item, so that
    Z * e^c and N * e^c are the paper's statistics without overflow.
    """
    subset = np.asarray(subset, dtype=np.int64)
    a = _logits(q, np.asarray(K)[subset])
    c = a.max() if a.size else 0.0
    w = np.exp(a - c)
    return w.sum(), w @ np.asarray(V, _F64)[subset], c


# --------------------------------------------------------------------------
# observation-window scoring (App. B.2.2, SnapKV rule; readings R1-R4)
# --------------------------------------------------------------------------

def scored_length(s, m, recent_window):
    """Number of scored positions: everything before the protected window."""
    p = min(recent_window, m, s)
    return s - p


def window_raw_scores(K, Qw, fit_rows=None):
    """Per-key attention mass from the observation window.

    K  : [s, d] prefill keys of one KV head.
    Qw : [G, w, d] window queries of the G query heads sharing that KV head;
         row i of each head sits at position s - w + i.
    fit_rows : if given, only the leading `fit_rows` positions of each head
         take part (the fit queries of the validation proxy, R20).
    Returns raw[s]: raw[p] = sum over window rows t that can see p (p <= pos(t))
    of softmax_t[p], where softmax_t normalises over every key row t can see
    (R1), summed over the G heads of the group (R2).
    """
    K = np.asarray(K, _F64)
    Qw = np.asarray(Qw, _F64)
    s, d = K.shape
    G, w, _ = Qw.shape
    nr = w if fit_rows is None else fit_rows
    raw = np.zeros(s, dtype=_F64)
    for h in range(G):
        a = (Qw[h, :nr] @ K.T) / math.sqrt(d)         # [nr, s]
        pos = s - w + np.arange(nr)
        visible = np.arange(s)[None, :] <= pos[:, None]
        a = np.where(visible, a, -np.inf)
        a = a - a.max(axis=1, keepdims=True)
        e = np.exp(a)
        soft = e / e.sum(axis=1, keepdims=True)
        raw += soft.sum(axis=0)
    return raw


def pool(raw, kernel=5):
    """Centred `kernel`-tap sum (odd kernel) with zero padding (R3):
    out[p] = sum_{|i| <= kernel // 2} raw[p+i]; kernel 1 returns the raw
    scores (the H2O and TOVA rules, R23, R24)."""
    assert kernel >= 1 and kernel % 2 == 1
    raw = np.asarray(raw, _F64)
    n = raw.shape[0]
    out = np.zeros(n, dtype=_F64)
    h = kernel // 2
    for off in range(-h, h + 1):
        lo = max(0, -off)
        hi = min(n, n - off)
        if lo < hi:  # a shift of n or more positions leaves nothing inside
            out[lo:hi] += raw[lo + off:hi + off]
    return out


def pool5(raw):
    """The SnapKV pooling of App. B.2.2: pool(raw, 5)."""
    return pool(raw, 5)


# --------------------------------------------------------------------------
# main selection (Sec. 5.2, main-selection equation; R4, R6, R7)
# --------------------------------------------------------------------------

def select_main(scores, s, m, recent_window, r):
    """M = P  U  Top_{m-|P|}(s),  E = S \\ M, plus the Lloyd seeds.

    scores : [n] pooled scores of positions 0..n-1, n = scored_length(...).
    Returns (main_idx ascending, evicted ascending, seeds ascending).
    When s <= m every token is kept and nothing is evicted.
    """
    if s <= m:
        return np.arange(s), np.zeros(0, np.int64), np.zeros(0, np.int64)
    p = min(recent_window, m, s)
    return select_top(scores, s, s - p, m - p, r)


def select_top(scores, s, n, k_top, r):
    """The k_top best of the scored positions [0, n) (score descending, then
    position ascending), plus the protected positions [n, s), are main; the
    rest is evicted; the next r in that order seed the Lloyd groups.
    Returns (main_idx ascending, evicted ascending, seeds ascending)."""
    scores = np.asarray(scores, _F64)
    assert scores.shape[0] == n
    order = np.lexsort((np.arange(n), -scores))
    top = order[:k_top]
    main = np.sort(np.concatenate([top, np.arange(n, s)]))
    evicted = np.sort(order[k_top:])
    seeds = np.sort(order[k_top:k_top + r])
    return main, evicted, seeds


# --------------------------------------------------------------------------
# residual partition by Lloyd iterations (Sec. 5.3; App. B.3; R7-R9)
# --------------------------------------------------------------------------

def assign_nearest(KE, centers):
    """argmin_j ||k_p - mu_j||^2 in direct-difference form; ties -> lowest j.

    Returns (assignment [n], squared distances [n, r]).
    """
    KE = np.asarray(KE, _F64)
    centers = np.asarray(centers, _F64)
    n = KE.shape[0]
    r = centers.shape[0]
    dist = np.empty((n, r), dtype=_F64)
    step = max(1, (1 << 22) // max(1, r * KE.shape[1]))
    for lo in range(0, n, step):
        diff = KE[lo:lo + step, None, :] - centers[None, :, :]
        dist[lo:lo + step] = np.einsum("prd,prd->pr", diff, diff)
    return np.argmin(dist, axis=1), dist


def lloyd_objective(KE, assign, r):
    """sum_j sum_{p in C_j} ||k_p - kbar_j||^2 (Sec. 5.3, partition objective)."""
    KE = np.asarray(KE, _F64)
    tot = 0.0
    for j in range(r):
        mem = KE[assign == j]
        if mem.shape[0]:
            tot += float(((mem - mem.mean(axis=0)) ** 2).sum())
    return tot


def lloyd(KE, init_centers, iters):
    """`iters` rounds of (assign, update) from the given centres (R8, R9).

    Returns (final assignment, final centres, per-iteration history of
    (assignment, centres before that assignment)).
    """
    mu = np.array(init_centers, dtype=_F64, copy=True)
    KE = np.asarray(KE, _F64)
    history = []
    assign = np.zeros(KE.shape[0], dtype=np.int64)
    for _ in range(iters):
        prev = mu.copy()
        assign, _ = assign_nearest(KE, mu)
        for j in range(mu.shape[0]):
            mem = KE[assign == j]
            if mem.shape[0]:
                mu[j] = mem.mean(axis=0)
        history.append((assign.copy(), prev))
    return assign, mu, history


def residual_entries(KE, VE, assign, centers, r, d):
    """Mean key, mean value and count per group (Sec. 5.3, summary equation).

    Entries j >= number of centres, and groups with no member, are empty:
    count 0, mean value 0, mean key = the centre (or 0), log-count -inf (R9).
    """
    kbar = np.zeros((r, d), _F64)
    vbar = np.zeros((r, d), _F64)
    cnt = np.zeros(r, dtype=np.int64)
    KE = np.asarray(KE, _F64)
    VE = np.asarray(VE, _F64)
    for j in range(len(centers)):
        kbar[j] = centers[j]
        mem = assign == j
        c = int(mem.sum())
        cnt[j] = c
        if c:
            vbar[j] = VE[mem].mean(axis=0)
    with np.errstate(divide="ignore"):
        logc = np.where(cnt > 0, np.log(np.maximum(cnt, 1).astype(_F64)), -np.inf)
    return kbar, vbar, cnt, logc


# --------------------------------------------------------------------------
# construction of one (layer, KV head) (App. D, Algorithm 1 with r given)
# --------------------------------------------------------------------------

def build_head(K, V, Qw, m, r, recent_window, lloyd_iters, dtype="bf16", fit_rows=None, pool_kernel=5):
    """Construct the main + residual layout for one (layer, KV head).

    K, V : [s, d] prefill keys/values (values already in the storage dtype).
    Qw   : [G, w, d] window queries (only the leading `fit_rows` positions of
           each head score the tokens when given).
    pool_kernel : taps of the score pooling (5: SnapKV; 1: H2O and TOVA).
    Returns a dict with the scores, selection, Lloyd record and the cache
    rows in slot order: residual entries in slots [0, r), main tokens in
    slots [r, r + main_len).
    """
    K = np.asarray(K, _F64)
    V = np.asarray(V, _F64)
    s = K.shape[0]
    out = {}
    if s <= m:
        main = np.arange(s)
        evicted = np.zeros(0, np.int64)
        seeds = np.zeros(0, np.int64)
        out["scores"] = np.zeros(0)
    else:
        n = scored_length(s, m, recent_window)
        raw = window_raw_scores(K, Qw, fit_rows)
        out["raw"] = raw
        scores = pool(raw[:n], pool_kernel)
        out["scores"] = scores
        main, evicted, seeds = select_main(scores, s, m, recent_window, r)
    return _residual_layout(out, K, V, main, evicted, seeds, r, lloyd_iters, dtype)


def _residual_layout(out, K, V, main, evicted, seeds, r, lloyd_iters, dtype):
    """Lloyd partition of the evicted rows, the r entries and the cache rows
    in slot order (shared by the uniform and the AdaKV construction)."""
    out["main_idx"], out["evicted"], out["seeds"] = main, evicted, seeds
    KE, VE = K[evicted], V[evicted]
    centers0 = K[seeds]
    if r > 0 and evicted.size > 0:
        assign, mu, hist = lloyd(KE, centers0, lloyd_iters)
    else:
        assign, mu, hist = np.zeros(evicted.size, np.int64), centers0, []
    out["assign"], out["centers"], out["lloyd_history"] = assign, mu, hist
    kbar, vbar, cnt, logc = residual_entries(KE, VE, assign, mu, r, K.shape[1])
    out["counts"], out["logc"] = cnt, logc
    out["kbar64"], out["vbar64"] = kbar, vbar
    kres = round_to_dtype(kbar, dtype)
    vres = round_to_dtype(vbar, dtype)
    out["kc"] = np.concatenate([kres, K[main]], axis=0)
    out["vc"] = np.concatenate([vres, V[main]], axis=0)
    out["res_len"] = r
    out["main_len"] = main.size
    return out


# --------------------------------------------------------------------------
# AdaKV cross-head budget allocation (App. B.2.2 compared methods; R26)
# --------------------------------------------------------------------------

def adakv_allocate(scores, k_top, safeguard, cap):
    """Top-k budgets of the KV heads of one (layer, sequence) under AdaKV.

    scores    : per head, the pooled scores of its scored positions;
    k_top     : per head, its top-k budget under the uniform split;
    safeguard : alpha; head h keeps at least floor(alpha * k_top[h]) of its
                own best tokens;
    cap       : per head, the most top-k tokens it may hold.
    The other sum(k_top) - sum(floors) slots go down one ranking of every
    head's remaining tokens, by score descending, then head, then position
    ascending; a head takes its next token only while under its cap.
    Returns the per-head top-k counts.
    """
    H = len(scores)
    floors = [int(math.floor(safeguard * k)) for k in k_top]
    total = sum(k_top)
    kk = list(floors)
    ranking = []
    for h in range(H):
        sc = np.asarray(scores[h], _F64)
        order = np.lexsort((np.arange(sc.size), -sc))
        for p in order[floors[h]:]:
            ranking.append((-sc[p], h, int(p)))
    ranking.sort()
    taken = sum(floors)
    for _, h, _ in ranking:
        if taken >= total:
            break
        if kk[h] < cap[h]:
            kk[h] += 1
            taken += 1
    return kk


def build_heads_adakv(Ks, Vs, Qws, budget, res, recent_window, lloyd_iters, safeguard, slot_cap,
                      dtype="bf16", pool_kernel=5):
    """AdaKV allocation followed by ResKV construction for the KV heads of
    one (layer, sequence). Per head the uniform split gives m = b - r, the
    protected |P| = min(recent_window, m, s) and the scored range [0, s-|P|);
    heads with s <= m keep every token and take no part. The others share
    their top-k budgets through adakv_allocate with cap = min(s - |P|,
    slot_cap - r - |P|); each keeps its |P| recent tokens and its top-k'
    scored tokens, and builds its r residual entries from the rest as in
    build_head. Returns one record per head.
    """
    H = len(Ks)
    s = np.asarray(Ks[0]).shape[0]
    recs, live, sc, kt, cap, prot = [None] * H, [], [], [], [], []
    for h in range(H):
        m = budget - res[h]
        if s <= m:
            recs[h] = build_head(Ks[h], Vs[h], Qws[h], m, res[h], recent_window, lloyd_iters, dtype,
                                 pool_kernel=pool_kernel)
            continue
        P = min(recent_window, m, s)
        n = s - P
        raw = window_raw_scores(np.asarray(Ks[h], _F64), Qws[h])
        live.append(h)
        sc.append(pool(raw[:n], pool_kernel))
        kt.append(m - P)
        cap.append(min(n, slot_cap - res[h] - P))
        prot.append(P)
    kk = adakv_allocate(sc, kt, safeguard, cap)
    for i, h in enumerate(live):
        K = np.asarray(Ks[h], _F64)
        V = np.asarray(Vs[h], _F64)
        k = kk[i]
        main, evicted, seeds = select_top(sc[i], s, s - prot[i], k, res[h])
        out = {"scores": sc[i], "k_top": k, "protected": prot[i]}
        recs[h] = _residual_layout(out, K, V, main, evicted, seeds, res[h], lloyd_iters, dtype)
    return recs


def build_cache(K, V, Qobs, seq_len, budget, res_count, recent_window,
                lloyd_iters, dtype, slot_cap, res_cap, heads=None):
    """Run build_head over (batch, KV head) and lay the result out as the
    library's cache tensors.

    K, V     : [B, Hkv, S, d]; Qobs : [B, Hq, w, d]; seq_len, budget : [B];
    res_count : [B, Hkv]. `heads` optionally restricts to a list of
    (b, kvh) pairs; other rows stay zero.
    Returns kc, vc [B, Hkv, C, d], logc [B, Hkv, Rcap], main_idx [B, Hkv, C],
    res_len, main_len [B, Hkv], plus per-head records.
    """
    K = np.asarray(K)
    B, Hkv, S, d = K.shape
    Hq = Qobs.shape[1]
    G = Hq // Hkv
    kc = np.zeros((B, Hkv, slot_cap, d))
    vc = np.zeros((B, Hkv, slot_cap, d))
    logc = np.full((B, Hkv, res_cap), -np.inf)
    main_idx = np.full((B, Hkv, slot_cap), -1, dtype=np.int64)
    res_len = np.zeros((B, Hkv), np.int64)
    main_len = np.zeros((B, Hkv), np.int64)
    recs = {}
    todo = heads if heads is not None else [(b, h) for b in range(B) for h in range(Hkv)]
    for b, h in todo:
        s = int(seq_len[b])
        r = int(res_count[b][h])
        m = int(budget[b]) - r
        rec = build_head(K[b, h, :s], V[b, h, :s], Qobs[b, h * G:(h + 1) * G],
                         m, r, recent_window, lloyd_iters, dtype)
        n = rec["kc"].shape[0]
        kc[b, h, :n] = rec["kc"]
        vc[b, h, :n] = rec["vc"]
        logc[b, h, :r] = rec["logc"]
        main_idx[b, h, :rec["main_len"]] = rec["main_idx"]
        res_len[b, h] = r
        main_len[b, h] = rec["main_len"]
        recs[(b, h)] = rec
    return dict(kc=kc, vc=vc, logc=logc, main_idx=main_idx, res_len=res_len,
                main_len=main_len, records=recs)


# --------------------------------------------------------------------------
# shared-softmax decode with the dynamic gate (Sec. 5.4, Sec. 5.5.2, Alg. 2)
# --------------------------------------------------------------------------

def gate_value(p_max, tau, alpha, g_min):
    """g = max(g_min, sigmoid((tau - p_max) / T_g)) with T_g = 1/alpha."""
    x = (tau - p_max) * alpha
    with np.errstate(over="ignore"):
        sig = 1.0 / (1.0 + math.exp(-x)) if x > -700 else 0.0
    return max(g_min, sig)


def decode_head(q, Kmain, Vmain, Kres, Vres, logc, tau, alpha, g_min, beta):
    """One query against one KV head's cache, in Algorithm 2's order.

    Returns (output [d], debug dict with lse_main, lse_res, gate, p_max).
    lse_res is log sum_j exp(<q, kbar_j>/sqrt(d) + beta*log c_j) before the
    gate shift (-inf when no entry is populated).
    """
    q = np.asarray(q, _F64)
    d = q.shape[0]
    Kmain = np.asarray(Kmain, _F64)
    Vmain = np.asarray(Vmain, _F64)
    # main logits a_p = <q, k_p>/sqrt(d)
    a = (Kmain @ q) / math.sqrt(d)
    amax = a.max()
    wm = np.exp(a - amax)
    # p_max = max_p e^{a_p} / sum_p' e^{a_p'}
    p_max = float(wm.max() / wm.sum())
    g = gate_value(p_max, tau, alpha, g_min)
    log_g = math.log(g) if g > 0 else -np.inf
    # residual logits: <q, kbar_j>/sqrt(d) + beta*log c_j + log g; empty
    # entries (log c = -inf) are left out entirely.
    logc = np.asarray(logc, _F64)
    live = np.isfinite(logc)
    Kres = np.asarray(Kres, _F64)[live]
    Vres = np.asarray(Vres, _F64)[live]
    ares_nogate = (Kres @ q) / math.sqrt(d) + beta * logc[live]
    ares = ares_nogate + log_g
    # one shared softmax over main logits and residual logits
    all_a = np.concatenate([a, ares])
    top = all_a.max()
    w = np.exp(all_a - top)
    num = w[:a.size] @ Vmain + (w[a.size:] @ Vres if Kres.shape[0] else 0.0)
    den = w.sum()
    out = num / den
    lse_main = amax + math.log(wm.sum())
    if ares_nogate.size:
        t = ares_nogate.max()
        lse_res = t + math.log(np.exp(ares_nogate - t).sum())
    else:
        lse_res = -np.inf
    return out, dict(lse_main=lse_main, lse_res=lse_res, gate=g, p_max=p_max)


def decode_branches(q, Kmain, Vmain, Kres, Vres, logc, beta):
    """The two branches of one decode query, each under its own softmax
    (Sec. 6.1: a fused main-branch kernel returns its output and per-query
    log-sum-exp; the residual branch is evaluated over the entries):
      o_main = softmax(a) V_main,  lse_main = log sum_p e^{a_p};
      o_res  = softmax(at) Vbar,   lse_res  = log sum_j e^{at_j},
    with at_j = <q, kbar_j>/sqrt(d) + beta log c_j (no gate). Empty entries
    are left out; with none populated o_res = 0 and lse_res = -inf.
    """
    q = np.asarray(q, _F64)
    d = q.shape[0]
    a = (np.asarray(Kmain, _F64) @ q) / math.sqrt(d)
    top = a.max()
    w = np.exp(a - top)
    o_main = (w @ np.asarray(Vmain, _F64)) / w.sum()
    lse_main = top + math.log(w.sum())
    logc = np.asarray(logc, _F64)
    live = np.isfinite(logc)
    if not live.any():
        return o_main, lse_main, np.zeros(d), -np.inf
    at = (np.asarray(Kres, _F64)[live] @ q) / math.sqrt(d) + beta * logc[live]
    t = at.max()
    u = np.exp(at - t)
    o_res = (u @ np.asarray(Vres, _F64)[live]) / u.sum()
    return o_main, lse_main, o_res, t + math.log(u.sum())


def merge_branches(o_main, lse_main, o_res, lse_res, g, mode):
    """Combine the two branches.

    "shared": the log-sum-exp merge with the residual mass scaled by the
    gate, (e^{lse_main} o_main + g e^{lse_res} o_res) / (e^{lse_main} +
    g e^{lse_res}) -- the shared softmax of Sec. 5.4 written over branch
    statistics (Sec. 6.1).
    "separate": the ablation without the shared softmax (Sec. 6.6, ablation
    table): each branch keeps its own normalisation and the gate mixes the
    two, (1 - g) o_main + g o_res, with g taken as 0 when no entry is
    populated (reading R25).
    """
    o_main = np.asarray(o_main, _F64)
    o_res = np.asarray(o_res, _F64)
    if mode == "separate":
        gg = g if np.isfinite(lse_res) else 0.0
        return (1.0 - gg) * o_main + gg * o_res
    assert mode == "shared"
    lr = lse_res + math.log(g) if (g > 0 and np.isfinite(lse_res)) else -np.inf
    top = max(lse_main, lr)
    wm = math.exp(lse_main - top)
    wr = math.exp(lr - top) if np.isfinite(lr) else 0.0
    return (wm * o_main + wr * o_res) / (wm + wr)


def decode(q, kc, vc, logc, res_len, main_len, tau, alpha, g_min, beta, heads=None):
    """Decode one step for every (batch, query head).

    q : [B, Hq, d]; kc, vc : [B, Hkv, C, d]; logc : [B, Hkv, Rcap];
    res_len, main_len : [B, Hkv]; tau : scalar or [B, Hq].
    Returns out [B, Hq, d], lse_main, lse_res, gate [B, Hq].
    """
    q = np.asarray(q, _F64)
    B, Hq, d = q.shape
    Hkv = kc.shape[1]
    G = Hq // Hkv
    out = np.zeros((B, Hq, d))
    lse_m = np.zeros((B, Hq))
    lse_r = np.zeros((B, Hq))
    gate = np.zeros((B, Hq))
    tau = np.broadcast_to(np.asarray(tau, _F64), (B, Hq))
    todo = heads if heads is not None else [(b, h) for b in range(B) for h in range(Hq)]
    for b, h in todo:
        kv = h // G
        r = int(res_len[b, kv])
        n = int(main_len[b, kv])
        o, dbg = decode_head(q[b, h], kc[b, kv, r:r + n], vc[b, kv, r:r + n],
                             kc[b, kv, :r], vc[b, kv, :r], logc[b, kv, :r],
                             float(tau[b, h]), alpha, g_min, beta)
        out[b, h] = o
        lse_m[b, h] = dbg["lse_main"]
        lse_r[b, h] = dbg["lse_res"]
        gate[b, h] = dbg["gate"]
    return out, lse_m, lse_r, gate


# --------------------------------------------------------------------------
# construction-time validation proxy (Sec. 5.5.1; App. D, Algorithm 1)
# --------------------------------------------------------------------------

def candidate_counts(budget, grid):
    """Residual counts of the budget grid: r = floor(f * b + 1/2) (R19)."""
    return [int(math.floor(f * budget + 0.5)) for f in grid]


def proxy_choice(losses, counts, delta):
    """r* = argmin over r > 0 of the validation loss (ties to the smaller r,
    R22); it is chosen only if L_{r*} < (1 - delta) L_0 (margin equation),
    else r = 0. `losses[i]` belongs to `counts[i]`; one count must be 0."""
    i0 = counts.index(0)
    best = None
    for i, r in enumerate(counts):
        if r <= 0:
            continue
        if best is None or losses[i] < losses[best] or (losses[i] == losses[best] and r < counts[best]):
            best = i
    if best is not None and losses[best] < (1.0 - delta) * losses[i0]:
        return counts[best], best
    return 0, i0


def validation_proxy(K, V, Qw, budget, grid, recent_window, lloyd_iters, val_rows, delta,
                     tau, alpha, g_min, beta, dtype="bf16"):
    """Algorithm 1 for one (layer, KV head).

    The fit queries (leading window positions) score the tokens once; for
    each grid count r the cache is built with m = b - r, the validation
    queries (trailing `val_rows` positions of every head) are decoded against
    it with the gated shared softmax, and the loss is their mean squared
    error against full attention over the whole prefix (R21, R22). Returns the
    chosen r, the per-candidate losses and counts, and the chosen candidate's
    build record.
    """
    K = np.asarray(K, _F64)
    V = np.asarray(V, _F64)
    Qw = np.asarray(Qw, _F64)
    G, w, d = Qw.shape
    fit = w - val_rows
    counts = candidate_counts(budget, grid)
    vq = Qw[:, fit:].reshape(-1, d)
    target = [full_attention(q, K, V) for q in vq]
    losses, recs = [], []
    for r in counts:
        rec = build_head(K, V, Qw, budget - r, r, recent_window, lloyd_iters, dtype, fit_rows=fit)
        n = rec["main_len"]
        kc, vc = rec["kc"], rec["vc"]
        err = 0.0
        for q, o in zip(vq, target):
            out, _ = decode_head(q, kc[r:r + n], vc[r:r + n], kc[:r], vc[:r], rec["logc"],
                                 tau, alpha, g_min, beta)
            err += float(((out - o) ** 2).sum())
        losses.append(err / len(vq))
        recs.append(rec)
    r_star, i = proxy_choice(losses, counts, delta)
    return dict(r=r_star, losses=losses, counts=counts, record=recs[i], records=recs)
