"""Plain fp64 CPU oracle for the per-position scoring of the method.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call or link
this module: only the test suite, the package smoke check and the benchmark's
CPU-baseline leg use it. It shares no code with the HIP path.

What it computes (for every packed position of a batch of stitched rollouts):
  * z_X[v] = s_X * sum_k h_X[k] * W_X[k, v]     -- the vocabulary projection of
    each model X in {student S, teacher T} (the language-model parameterisation of
    pi_theta and pi_T used throughout Sec. 3.1; s_X = 1/temperature, and the
    configuration table of App. A (Table 3) fixes the training temperature at 1.0);
  * lse_X = M_X + ln sum_v exp(z_X[v] - M_X), M_X = max_v z_X[v]   -- the
    normaliser of the softmax over the full vocabulary;
  * logp_X = z_X[y] - lse_X for the realised token y   -- the per-token log-prob
    whose negative sum over the teacher continuation is the loss of Eq. 1;
  * KL(p_T || p_S) = sum_v p_T[v] (log p_T[v] - log p_S[v])   -- the full
    vocabulary divergence between teacher and student (knowledge distillation
    minimises it, Sec. 6; OPD scores student tokens with the teacher, Sec. 1);
  * KL(p_S || p_T) = sum_v p_S[v] (log p_S[v] - log p_T[v])   -- the reverse
    direction, the per-token objective of on-policy distillation (Sec. 1);
  * JSD(p_S, p_T) = 1/2 KL(p_S || m) + 1/2 KL(p_T || m), m = (p_S + p_T) / 2  -- the
    symmetric divergence between the two, bounded by ln 2 (the paper names only the
    reverse KL for OPD; the Jensen-Shannon form is offered beside it);
  * argmax_X = lowest v attaining M_X   -- the greedy token (the K = 1 case of the
    top-K overlap statistic of Sec. 4.1);
  * TopK_X = the K largest logits of model X, ties broken towards the lower index;
    overlap = |TopK_S & TopK_T| / K (the top-K overlap ratio of Sec. 4.1) and the
    top-K KL approximation sum_{v in TopK_T} p_T[v] (log p_T[v] - log p_S[v]) with
    full-vocabulary normalisers (OPD's LogProb top-K = 16, App. A Table 3);
  * the gradient of L = w_ce * sum_b CE_b + w_kl * sum_t KL(p_T || p_S)[t] (Eq. 1's
    loss, and the distillation divergence, over the in-region positions) with respect
    to the student's hidden states and LM-head weight, for the backward pass the
    student's update step on the masked CE loss needs (the update of Alg. 1 with
    Eq. 1, Sec. 3.1): per in-region position, dL/dz_S = w_ce (p_S - onehot(y)) +
    w_kl (p_S - p_T) for the scaled logits z_S, then dh = s_S W dL/dz_S and
    dW = s_S sum_t h_t (dL/dz_S)_t^T;
  * masks: a position is valid when it precedes the sequence's valid length, and
    in-region (scored) for the teacher region when it is at or past the cut, the
    prompt and student prefix being masked out of Eq. 1's loss (Sec. 3.1).

Everything is the plain two-pass definition in float64 over the exact values of
the (bf16- or fp32-) rounded inputs: one library matmul per row chunk, then max,
exp, an exactly rounded sum (math.fsum), log. No online rescaling, no vocabulary
splitting, no fusion.
"""
from __future__ import annotations

import math
from typing import Optional

import numpy as np

REGION_TEACHER = 0   # t >= cut: the teacher continuation (Eq. 1's scored tokens)
REGION_STUDENT = 1   # t <  cut: the student prefix (OPD's scored tokens)
REGION_ALL = 2       # every valid position
REGION_SPANS = 3     # the given scored spans of each sequence (multi-turn: teacher actions)


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def masks(cu_seqlens, cut, valid_len=None, region: int = REGION_TEACHER, spans=None) -> dict:
    """Position masks and counts (Sec. 3.1, Eq. 1 and the sentence after it;
    Sec. 3.2 for span masks).

    Sequence b occupies packed rows [cu[b], cu[b+1]); local index t = row - cu[b].
    valid(t) = t < valid_len[b] (valid_len defaults to the sequence length);
    in-region(t) = valid(t) and (t >= cut[b] | t < cut[b] | true) for the
    teacher / student / all regions. With `spans` (REGION_SPANS; one list of
    (start, end) pairs per sequence, local and half-open) in-region(t) = valid(t)
    and t lies in one of the sequence's spans: in the multi-turn form of the method
    only the teacher's action tokens are scored, while the student's turns and every
    environment observation stay in the context.
    """
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    B = len(cu) - 1
    T = int(cu[-1])
    lengths = cu[1:] - cu[:-1]
    vl = lengths.copy() if valid_len is None else np.asarray(valid_len, dtype=np.int64)
    if region == REGION_SPANS:
        if spans is None or len(spans) != B:
            raise ValueError("REGION_SPANS needs one span list per sequence")
    else:
        cut = np.asarray(cut, dtype=np.int64)
    seq_id = np.empty(T, dtype=np.int64)
    local_t = np.empty(T, dtype=np.int64)
    valid = np.zeros(T, dtype=bool)
    inreg = np.zeros(T, dtype=bool)
    for b in range(B):
        t = np.arange(lengths[b], dtype=np.int64)
        rows = slice(cu[b], cu[b + 1])
        seq_id[rows] = b
        local_t[rows] = t
        v = t < vl[b]
        valid[rows] = v
        if region == REGION_TEACHER:
            r = t >= cut[b]
        elif region == REGION_STUDENT:
            r = t < cut[b]
        elif region == REGION_ALL:
            r = np.ones_like(v)
        elif region == REGION_SPANS:
            r = np.zeros_like(v)
            for (a, e) in spans[b]:
                r |= (t >= a) & (t < e)
        else:
            raise ValueError("unknown region %r" % (region,))
        inreg[rows] = v & r
    return dict(seq_id=seq_id, local_t=local_t, valid=valid, in_region=inreg,
                n_scored=int(inreg.sum()), t_valid=int(valid.sum()))


def project(h_rows, w, scale: float = 1.0) -> np.ndarray:
    """z = scale * (h @ W): the vocabulary logits of a model, [n, V] in float64.

    h_rows: [n, d]; w: [d, V] (the layout of the workloads). The product of two
    bf16 values is exact in float64; the d-term sum is one library matmul.
    """
    return float(scale) * (_f64(h_rows) @ _f64(w))


def log_softmax_stats(z_row) -> dict:
    """Max, log-normaliser, greedy index and top-2 gap of one logit row (fp64)."""
    z = _f64(z_row)
    M = float(z.max())
    lse = M + math.log(math.fsum(np.exp(z - M).tolist()))
    am = int(np.argmax(z))                      # first index attaining the max
    if z.shape[0] >= 2:
        second = float(np.partition(z, -2)[-2])
        gap = M - second
    else:
        gap = math.inf
    return dict(max=M, lse=lse, argmax=am, gap=gap)


def kl_teacher_student(z_t, lse_t: float, z_s, lse_s: float) -> tuple:
    """KL(p_T || p_S) of one row, two ways (fp64, exactly rounded sums).

    direct: sum_v p_T (log p_T - log p_S).
    nonneg: sum_v p_T (expm1(d) - d), d = log p_S - log p_T, whose every term is
            >= 0; it equals the direct form because sum p_S = sum p_T = 1.
    """
    lp_t = _f64(z_t) - lse_t
    lp_s = _f64(z_s) - lse_s
    p_t = np.exp(lp_t)
    direct = math.fsum((p_t * (lp_t - lp_s)).tolist())
    d = lp_s - lp_t
    with np.errstate(over="ignore", invalid="ignore"):
        term = p_t * (np.expm1(d) - d)
    big = ~np.isfinite(term)
    if big.any():   # p_T * e^d = p_S exactly; use it where expm1 overflows
        term[big] = np.exp(lp_s[big]) - p_t[big] * (1.0 + d[big])
    nonneg = math.fsum(term.tolist())
    return direct, nonneg


def kl_student_teacher(z_s, lse_s: float, z_t, lse_t: float) -> tuple:
    """Reverse KL(p_S || p_T) of one row: sum_v p_S (log p_S - log p_T), the
    divergence on-policy distillation minimises on student tokens (Sec. 1).

    The same definition as kl_teacher_student with the roles of the two
    distributions exchanged (the first argument is the one the sum weights by);
    returns the direct and the pointwise non-negative forms.
    """
    return kl_teacher_student(z_s, lse_s, z_t, lse_t)


def jsd(z_s, lse_s: float, z_t, lse_t: float) -> float:
    """Jensen-Shannon divergence of one row's two distributions (fp64, exactly rounded
    sums): 1/2 sum_v p_S (log p_S - log m) + 1/2 sum_v p_T (log p_T - log m) with the
    mixture m = (p_S + p_T) / 2, whose log is formed as logaddexp(log p_S, log p_T) -
    ln 2 so that it stays finite where one probability underflows."""
    lp_s = _f64(z_s) - lse_s
    lp_t = _f64(z_t) - lse_t
    log_m = np.logaddexp(lp_s, lp_t) - math.log(2.0)
    a = math.fsum((np.exp(lp_s) * (lp_s - log_m)).tolist())
    b = math.fsum((np.exp(lp_t) * (lp_t - log_m)).tolist())
    return 0.5 * a + 0.5 * b


TOPK = 16   # LogProb top-K of the OPD baseline (App. A, Table 3)


def topk_set(z_row, k: int) -> np.ndarray:
    """Indices of the k largest entries, ordered by (value descending, index
    ascending): ties at the boundary go to the lower vocabulary indices. One library
    sort on the key (value descending, index ascending)."""
    z = _f64(z_row)
    order = np.lexsort((np.arange(len(z)), -z))
    return order[:k].astype(np.int64)


def topk_overlap(set_s, set_t, k: int = TOPK) -> float:
    """|TopK(student) & TopK(teacher)| / k (Sec. 4.1's top-K overlap ratio), from
    the two index sets."""
    return len(set(np.asarray(set_s).tolist()) & set(np.asarray(set_t).tolist())) / float(k)


def kl_topk(z_t, lse_t: float, z_s, lse_s: float, set_t) -> float:
    """KL(teacher || student) restricted to the teacher's top-k tokens (set_t), with
    the full-vocabulary normalisers (not renormalised): the top-K approximation of
    the OPD baseline (abstract; App. A, Table 3: LogProb top-K = 16)."""
    zt, zs = _f64(z_t), _f64(z_s)
    idx = np.asarray(set_t, dtype=np.int64)
    lp_t = zt[idx] - lse_t
    lp_s = zs[idx] - lse_s
    return math.fsum((np.exp(lp_t) * (lp_t - lp_s)).tolist())


def row_scores(h_student_rows, w_student, targets_rows, scale_student: float = 1.0,
               h_teacher_rows=None, w_teacher=None, scale_teacher: float = 1.0,
               chunk: Optional[int] = None, extras: bool = True) -> dict:
    """Unmasked per-row quantities for a set of rows (every row treated as valid).

    Returns float64 / int64 arrays of length n: z_y_s, lse_s, logp_s, argmax_s,
    gap_s, max_s, and with a teacher the same for t plus kl (direct) and
    kl_nonneg (KL(teacher || student)), kl_rev and kl_rev_nonneg (KL(student ||
    teacher)), jsd (Jensen-Shannon), overlap and kl_topk (top-K statistics, K = TOPK)
    and the top-K index sets topk_s / topk_t ([n, TOPK]).

    extras=False leaves out the reverse KL, the Jensen-Shannon divergence and the top-K
    statistics (their keys are then absent); every value that is returned is computed
    exactly as with extras=True.
    """
    hs = _f64(h_student_rows)
    n = hs.shape[0]
    y = np.asarray(targets_rows, dtype=np.int64)
    ws = _f64(w_student)
    V = ws.shape[1]
    has_t = h_teacher_rows is not None
    if has_t:
        ht = _f64(h_teacher_rows)
        wt = _f64(w_teacher)
        assert wt.shape[1] == V, "student and teacher share one vocabulary"
    if chunk is None:
        chunk = max(1, min(256, (1 << 22) // max(V, 1)))
    out = {k: np.zeros(n) for k in ("z_y_s", "lse_s", "logp_s", "gap_s", "max_s")}
    out["argmax_s"] = np.zeros(n, dtype=np.int64)
    if has_t:
        for k in ("z_y_t", "lse_t", "logp_t", "gap_t", "max_t", "kl", "kl_nonneg"):
            out[k] = np.zeros(n)
        if extras:
            for k in ("kl_rev", "kl_rev_nonneg", "jsd", "overlap", "kl_topk"):
                out[k] = np.zeros(n)
            out["topk_s"] = np.zeros((n, min(TOPK, V)), dtype=np.int64)
            out["topk_t"] = np.zeros((n, min(TOPK, V)), dtype=np.int64)
        out["argmax_t"] = np.zeros(n, dtype=np.int64)
    for r0 in range(0, n, chunk):
        r1 = min(n, r0 + chunk)
        zs = project(hs[r0:r1], ws, scale_student)
        zt = project(ht[r0:r1], wt, scale_teacher) if has_t else None
        for i in range(r1 - r0):
            g = r0 + i
            st = log_softmax_stats(zs[i])
            out["z_y_s"][g] = zs[i, y[g]]
            out["lse_s"][g] = st["lse"]
            out["logp_s"][g] = zs[i, y[g]] - st["lse"]
            out["argmax_s"][g] = st["argmax"]
            out["gap_s"][g] = st["gap"]
            out["max_s"][g] = st["max"]
            if has_t:
                tt = log_softmax_stats(zt[i])
                out["z_y_t"][g] = zt[i, y[g]]
                out["lse_t"][g] = tt["lse"]
                out["logp_t"][g] = zt[i, y[g]] - tt["lse"]
                out["argmax_t"][g] = tt["argmax"]
                out["gap_t"][g] = tt["gap"]
                out["max_t"][g] = tt["max"]
                kl, klp = kl_teacher_student(zt[i], tt["lse"], zs[i], st["lse"])
                out["kl"][g] = kl
                out["kl_nonneg"][g] = klp
                if not extras:
                    continue
                klr, klrp = kl_student_teacher(zs[i], st["lse"], zt[i], tt["lse"])
                out["kl_rev"][g] = klr
                out["kl_rev_nonneg"][g] = klrp
                out["jsd"][g] = jsd(zs[i], st["lse"], zt[i], tt["lse"])
                kk = min(TOPK, V)
                set_s, set_t = topk_set(zs[i], kk), topk_set(zt[i], kk)
                out["overlap"][g] = topk_overlap(set_s, set_t, kk)
                out["kl_topk"][g] = kl_topk(zt[i], tt["lse"], zs[i], st["lse"], set_t)
                out["topk_s"][g] = set_s
                out["topk_t"][g] = set_t
    return out


def score(h_student, w_student, targets, cu_seqlens, cut, valid_len=None,
          h_teacher=None, w_teacher=None, scale_student: float = 1.0,
          scale_teacher: float = 1.0, region: int = REGION_TEACHER,
          rows=None, spans=None) -> dict:
    """The whole scoring of a packed batch, masked.

    Outputs per packed position (length T): logp_s, logp_t, argmax_s, argmax_t,
    kl (KL(teacher || student) in-region, exactly +0.0 elsewhere), kl_rev
    (KL(student || teacher)) and jsd (Jensen-Shannon), masked the same way; at positions
    past the valid length logp = 0 and argmax = -1. Per sequence: ce (Eq. 1's
    loss, minus the sum of the student's log-probs over the in-region positions).
    Counts: n_scored (in-region positions) and t_valid (valid positions).

    rows: optional subset of packed rows to evaluate (the others are left at the
    masked values and reported in `evaluated`); masks and counts are always full.
    """
    m = masks(cu_seqlens, cut, valid_len, region, spans)
    T = m["valid"].shape[0]
    B = len(np.asarray(cu_seqlens)) - 1
    has_t = h_teacher is not None
    sel = np.arange(T) if rows is None else np.unique(np.asarray(rows, dtype=np.int64))
    sel = sel[m["valid"][sel]]
    y = np.asarray(targets, dtype=np.int64)
    if sel.size:
        r = row_scores(np.asarray(h_student)[sel], w_student, y[sel], scale_student,
                       None if not has_t else np.asarray(h_teacher)[sel], w_teacher,
                       scale_teacher)
    out = dict(logp_s=np.zeros(T), argmax_s=np.full(T, -1, dtype=np.int64),
               lse_s=np.zeros(T), gap_s=np.full(T, math.inf), kl=np.zeros(T),
               kl_nonneg=np.zeros(T), kl_rev=np.zeros(T), jsd=np.zeros(T), overlap=np.zeros(T),
               kl_topk=np.zeros(T), evaluated=np.zeros(T, dtype=bool))
    if has_t:
        out.update(logp_t=np.zeros(T), argmax_t=np.full(T, -1, dtype=np.int64),
                   lse_t=np.zeros(T), gap_t=np.full(T, math.inf))
    if sel.size:
        out["evaluated"][sel] = True
        for k in ("logp_s", "argmax_s", "lse_s", "gap_s"):
            out[k][sel] = r[k]
        if has_t:
            for k in ("logp_t", "argmax_t", "lse_t", "gap_t"):
                out[k][sel] = r[k]
            inr = m["in_region"][sel]
            out["kl"][sel[inr]] = r["kl"][inr]
            out["kl_nonneg"][sel[inr]] = r["kl_nonneg"][inr]
            out["kl_rev"][sel[inr]] = r["kl_rev"][inr]
            out["jsd"][sel[inr]] = r["jsd"][inr]
            out["overlap"][sel[inr]] = r["overlap"][inr]
            out["kl_topk"][sel[inr]] = r["kl_topk"][inr]
    # Eq. 1: the loss of sequence b is minus the sum of the student's log-probs of
    # its in-region tokens; an empty region gives 0.
    ce = np.zeros(B)
    seq = m["seq_id"]
    for b in range(B):
        idx = np.nonzero((seq == b) & m["in_region"] & out["evaluated"])[0]
        ce[b] = -math.fsum(out["logp_s"][idx].tolist()) if idx.size else 0.0
    out["ce"] = ce
    out["n_scored"] = m["n_scored"]
    out["t_valid"] = m["t_valid"]
    out["valid"] = m["valid"]
    out["in_region"] = m["in_region"]
    return out


def grad_logits(z_s, lse_s: float, y: int, w_ce: float = 1.0, z_t=None, lse_t=None,
                w_kl: float = 0.0) -> np.ndarray:
    """dL/dz_S of one in-region row, for L = w_ce (-log p_S[y]) + w_kl KL(p_T || p_S)
    and the scaled student logits z_S: the derivative of -log p_S[y] is
    p_S - onehot(y); that of KL(p_T || p_S) = sum p_T log p_T - sum p_T log p_S is
    p_S - p_T (sum p_T = 1)."""
    p_s = np.exp(_f64(z_s) - lse_s)
    g = (w_ce + w_kl) * p_s
    g[int(y)] -= w_ce
    if w_kl != 0.0:
        g -= w_kl * np.exp(_f64(z_t) - lse_t)
    return g


def backward(h_student, w_student, targets, cu_seqlens, cut, valid_len=None,
             h_teacher=None, w_teacher=None, scale_student: float = 1.0,
             scale_teacher: float = 1.0, region: int = REGION_TEACHER, spans=None,
             w_ce: float = 1.0, w_kl: float = 0.0, rows=None, cols=None,
             keep_g: bool = True) -> dict:
    """Gradient of L = w_ce * sum_b CE_b + w_kl * sum_{t in region} KL(p_T || p_S)[t]
    (CE_b: Eq. 1's loss of sequence b) with respect to the student's hidden states
    h_S [T, d] and LM-head weight W_S [d, V] (the layout of the workloads).

    z_S = s_S h W, so dL/dh_t = s_S W g_t and dL/dW = s_S sum_t h_t g_t^T with
    g_t = dL/dz_S at row t (grad_logits) for in-region t and 0 elsewhere.

    Returns grad_h [T, d] (rows outside the region are 0), grad_w [d, V] and the
    per-row g for the evaluated rows. rows: optional subset of packed rows whose
    grad_h is formed (grad_w is then None: it needs every in-region row). cols:
    optional vocabulary columns of grad_w to keep (grad_w is then [d, len(cols)]).
    keep_g: keep the per-row g (off for large batches).
    """
    m = masks(cu_seqlens, cut, valid_len, region, spans)
    T = m["valid"].shape[0]
    hs = _f64(h_student)
    ws = _f64(w_student)
    d, V = ws.shape
    y = np.asarray(targets, dtype=np.int64)
    inr = np.nonzero(m["in_region"])[0]
    sel = inr if rows is None else np.intersect1d(np.asarray(rows, dtype=np.int64), inr)
    grad_h = np.zeros((T, d))
    cols = None if cols is None else np.asarray(cols, dtype=np.int64)
    grad_w = None if rows is not None else np.zeros((d, V if cols is None else len(cols)))
    g_rows = np.zeros((len(sel), V)) if keep_g else None
    if w_kl != 0.0:
        ht, wt = _f64(h_teacher), _f64(w_teacher)
    chunk = max(1, min(256, (1 << 22) // max(V, 1)))
    for r0 in range(0, len(sel), chunk):
        idx = sel[r0:r0 + chunk]
        zs = project(hs[idx], ws, scale_student)
        zt = project(ht[idx], wt, scale_teacher) if w_kl != 0.0 else None
        gb = np.zeros((len(idx), V))
        for i, t in enumerate(idx):
            lse_s = log_softmax_stats(zs[i])["lse"]
            if w_kl != 0.0:
                lse_t = log_softmax_stats(zt[i])["lse"]
                gb[i] = grad_logits(zs[i], lse_s, y[t], w_ce, zt[i], lse_t, w_kl)
            else:
                gb[i] = grad_logits(zs[i], lse_s, y[t], w_ce)
        if g_rows is not None:
            g_rows[r0:r0 + len(idx)] = gb
        grad_h[idx] = scale_student * (gb @ ws.T)
        if grad_w is not None:
            grad_w += scale_student * (hs[idx].T @ (gb if cols is None else gb[:, cols]))
    return dict(grad_h=grad_h, grad_w=grad_w, g=g_rows, rows=sel, in_region=m["in_region"])


def loss(h_student, w_student, targets, cu_seqlens, cut, valid_len=None, h_teacher=None,
         w_teacher=None, scale_student: float = 1.0, scale_teacher: float = 1.0,
         region: int = REGION_TEACHER, spans=None, w_ce: float = 1.0,
         w_kl: float = 0.0) -> float:
    """L = w_ce * sum_b CE_b + w_kl * sum_t KL(p_T || p_S)[t] from the forward scoring
    (the function whose gradient `backward` forms)."""
    r = score(h_student, w_student, targets, cu_seqlens, cut, valid_len,
              h_teacher if w_kl != 0.0 else None, w_teacher if w_kl != 0.0 else None,
              scale_student, scale_teacher, region, spans=spans)
    total = w_ce * math.fsum(r["ce"].tolist())
    if w_kl != 0.0:
        total += w_kl * math.fsum(r["kl"].tolist())
    return total
