"""Shared helpers of the GPU tests: run the HIP path through the C ABI and the fp64
oracle on the same seeded workload, and compare them at the acceptance tolerances.

Tolerances: per-token log-prob within 2e-3 absolute; per-position KL (either
direction, and the top-K KL) within 1e-3 + 1e-3 |KL|; masked counts, valid counts and
greedy argmax bit-exact; Eq. 1's per-sequence loss within 1e-3 relative (plus 1e-3
absolute for tiny sums). Top-K sets are decided on exact logits on both sides (fp64
sums of exact bf16 products): equal to the oracle's, in rank order, wherever the
fp64 logits separate the entries by more than twice the fp64 summation bound (every
row but exact-tie rows of crafted inputs), and otherwise a valid top-16 of logits
moved by at most that bound; the overlap ratio exact.
"""
import math
import sys
import time

import numpy as np
import torch

from oracle import olive_oracle as O
from paper_2609_36246_amd import _lib as L
from tests import oracle_pool

LOGP_ATOL = 2e-3
KL_ATOL = 1e-3
KL_RTOL = 1e-3
CE_RTOL = 1e-3


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


def to_np(t):
    if t is None:
        return None
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.detach().cpu().numpy()


TOPK_OUTPUTS = ("overlap", "kl_topk", "tk_s", "tk_t")


def run_hip(wl, region=L.OLIVE_REGION_TEACHER, simple=False, student_only=False,
            outputs=("kl", "counts", "logp_s", "logp_t", "am_s", "am_t", "ce"),
            poison=False, ctx=None, keep_ctx=False, timing=False, repeat=1, out_flags=0,
            topk_ctx=None, narrow=False):
    """Score a workload on the GPU; returns numpy outputs (and stats).

    Top-K outputs ("overlap", "kl_topk", "tk_s", "tk_t") make the context reserve
    the top-K workspace (topk_ctx overrides that choice)."""
    dev = wl["h_student"].device
    spec = wl["spec"]
    T = wl["total_positions"]
    B = wl["cu_seqlens"].shape[0] - 1
    own = ctx is None
    if own:
        if topk_ctx is None:
            topk_ctx = any(k in outputs for k in TOPK_OUTPUTS)
        flags = (L.OLIVE_FLAG_SIMPLE_KERNEL if simple else 0) | \
                (L.OLIVE_FLAG_KERNEL_TIMING if timing else 0) | \
                (L.OLIVE_FLAG_TOPK if topk_ctx else 0) | \
                (L.OLIVE_FLAG_NARROW_TILE if narrow else 0)
        desc = L.make_desc(spec.vocab, spec.d_student, 0 if student_only else spec.d_teacher,
                           L.OLIVE_BF16 if spec.dtype == "bf16" else L.OLIVE_F32, L.OLIVE_W_DV,
                           wl["scale_student"], wl["scale_teacher"], max_positions=T,
                           max_seqs=B, flags=flags)
        ctx = L.olive_score_init(desc, wl["w_student"],
                                 None if student_only else wl["w_teacher"])
    fill = float("nan") if poison else 0.0

    def f32():
        return torch.full((T,), fill, dtype=torch.float32, device=dev)

    def i32():
        return torch.full((T,), -7, dtype=torch.int32, device=dev)
    out = {}
    out["kl"] = f32() if "kl" in outputs and not student_only else None
    out["kl_rev"] = f32() if "kl_rev" in outputs and not student_only else None
    out["jsd"] = f32() if "jsd" in outputs and not student_only else None
    out["counts"] = torch.full((2,), -1, dtype=torch.int64, device=dev) \
        if "counts" in outputs else None
    out["logp_s"] = f32() if "logp_s" in outputs else None
    out["logp_t"] = f32() if "logp_t" in outputs and not student_only else None
    out["am_s"] = i32() if "am_s" in outputs else None
    out["am_t"] = i32() if "am_t" in outputs and not student_only else None
    out["ce"] = torch.full((B,), fill, dtype=torch.float32, device=dev) \
        if "ce" in outputs and not student_only else None
    out["overlap"] = f32() if "overlap" in outputs else None
    out["kl_topk"] = f32() if "kl_topk" in outputs else None
    for k in ("tk_s", "tk_t"):
        out[k] = torch.full((T, L.OLIVE_TOPK), -7, dtype=torch.int32, device=dev) \
            if k in outputs else None
    any_topk = any(out[k] is not None for k in TOPK_OUTPUTS)
    spans = wl.get("spans") if region == L.OLIVE_REGION_SPANS else None
    batch = L.make_batch(wl["cu_seqlens"], None if spans is not None else wl["cut"],
                         wl["targets"], wl["h_student"],
                         None if student_only else wl["h_teacher"], wl["valid_len"], region)
    for _ in range(repeat):
        if spans is not None or out["kl_rev"] is not None or out["jsd"] is not None or \
                out_flags or any_topk:
            o = L.make_outputs(kl=out["kl"], kl_reverse=out["kl_rev"], counts=out["counts"],
                               logp_student=out["logp_s"], logp_teacher=out["logp_t"],
                               argmax_student=out["am_s"], argmax_teacher=out["am_t"],
                               ce_per_seq=out["ce"], topk_overlap=out["overlap"],
                               kl_topk=out["kl_topk"], topk_student=out["tk_s"],
                               topk_teacher=out["tk_t"], jsd=out["jsd"], flags=out_flags)
            if spans is not None:
                sp = L.make_spans(wl["span_offsets"], wl["span_pairs"])
                L.olive_score_batch_spans(ctx, batch, sp, o)
            else:
                L.olive_score_batch(ctx, batch, o)
        elif student_only or out["kl"] is None:
            L.olive_token_logprobs(ctx, batch, out["logp_s"], out["logp_t"], out["am_s"],
                                   out["am_t"])
        else:
            L.olive_kl_masked(ctx, batch, out["kl"], out["counts"], out["logp_s"], out["logp_t"],
                              out["am_s"], out["am_t"], out["ce"])
    torch.cuda.synchronize()
    res = {k: to_np(v) for k, v in out.items() if v is not None}
    res["stats"] = L.olive_score_last_stats(ctx)
    res["err"] = L.olive_score_last_error(ctx)
    if keep_ctx:
        res["ctx"] = ctx
    elif own:
        L.olive_score_free(ctx)
    return res


def oracle_rows(wl, rows, student_only=False, extras=True):
    """fp64 oracle on a subset of packed rows (all rows treated as valid). Large row
    sets run in the worker pool of tests/oracle_pool.py (the same oracle function,
    over chunks of rows). extras=False leaves out the reverse KL and top-K values."""
    rows = np.asarray(rows, dtype=np.int64)
    idx = torch.from_numpy(rows).to(wl["h_student"].device)
    hs = to_np(wl["h_student"][idx])
    ht = None if student_only else to_np(wl["h_teacher"][idx])
    y = to_np(wl["targets"][idx])
    ws = to_np(wl["w_student"])
    wt = None if student_only else to_np(wl["w_teacher"])
    t0 = time.time()
    if len(rows) >= POOL_MIN_ROWS:
        r = oracle_pool.row_scores(hs, ws, y, wl["scale_student"], ht, wt, wl["scale_teacher"],
                                   extras=extras, log=say)
        how = "%d worker processes" % oracle_pool.workers()
    else:
        r = O.row_scores(hs, ws, y, wl["scale_student"], ht, wt, wl["scale_teacher"],
                         extras=extras)
        how = "one process"
    say("oracle on %d rows took %.1fs (%s)" % (len(rows), time.time() - t0, how))
    return r


POOL_MIN_ROWS = 64


def structure_np(wl):
    return (to_np(wl["cu_seqlens"]), to_np(wl["cut"]),
            None if wl["valid_len"] is None else to_np(wl["valid_len"]))


def masks_of(wl, region):
    cu, cut, vl = structure_np(wl)
    return O.masks(cu, cut, vl, region, wl.get("spans") if region == O.REGION_SPANS else None)


def parity_rows(wl, frac=0.01, n_whole=2, seed=1):
    """The row sample of a workload too large for the oracle in full: every row of the
    n_whole sequences with the fewest valid rows, the rows around every cut (cut-1,
    cut, cut+1) and end of the valid prefix (valid_len-1, valid_len), the first and
    last row of every sequence, every outlier row, and random valid rows until the
    sample holds at least `frac` of the valid rows. Returns (rows, whole sequences)."""
    cu, cut, vl = structure_np(wl)
    B = len(cu) - 1
    lengths = np.diff(cu)
    vlen = lengths if vl is None else vl
    whole = [int(b) for b in np.argsort(vlen, kind="stable")[:n_whole]]
    picks = set()
    for b in whole:
        picks.update(range(int(cu[b]), int(cu[b] + vlen[b])))
    base = stratified_rows(wl, n_random=0)
    picks.update(int(x) for x in base)
    valid = masks_of(wl, O.REGION_TEACHER)["valid"]
    t_valid = int(valid.sum())
    want = int(np.ceil(frac * t_valid))
    rng = np.random.default_rng(seed)
    have = sum(1 for r in picks if valid[r])
    for x in rng.permutation(np.nonzero(valid)[0]):
        if have >= want:
            break
        if int(x) not in picks:
            picks.add(int(x))
            have += 1
    rows = np.array(sorted(picks), dtype=np.int64)
    n_valid = int(valid[rows].sum())
    assert n_valid >= want, (n_valid, want)
    return rows, whole


def stratified_rows(wl, n_random=128, seed=1):
    """Rows of a large workload the oracle evaluates: around every cut and end of
    sequence, first/last rows, every outlier row, and random rows."""
    cu, cut, vl = structure_np(wl)
    B = len(cu) - 1
    lengths = np.diff(cu)
    vlen = lengths if vl is None else vl
    picks = set()
    for b in range(B):
        for t in (0, cut[b] - 1, cut[b], cut[b] + 1, vlen[b] - 1, vlen[b], lengths[b] - 1):
            if 0 <= t < lengths[b]:
                picks.add(int(cu[b] + t))
    for r in wl.get("outlier_rows", []):
        picks.add(int(r))
    for b, sp in enumerate(wl.get("spans") or []):
        for (a0, e0) in sp:
            for t in (a0 - 1, a0, e0 - 1, e0):
                if 0 <= t < lengths[b]:
                    picks.add(int(cu[b] + t))
    rng = np.random.default_rng(seed)
    T = int(cu[-1])
    if n_random > 0:
        picks.update(int(x) for x in rng.choice(T, size=min(n_random, T), replace=False))
    return np.array(sorted(picks), dtype=np.int64)


def compare(hip, wl, region=O.REGION_TEACHER, rows=None, student_only=False, check_ce=True,
            label="", region_only=False, whole_seqs=None):
    """Compare HIP outputs with the oracle, element by element, at the acceptance bar.

    region_only: the call scored only the region; every output outside it must hold
    the fixed values of unscored positions, and the region is compared as usual.
    rows: the packed rows to compare (default all); whole_seqs: sequences every row of
    which is among them, whose per-sequence loss is then compared too (every sequence
    when rows is None)."""
    cu, cut, vl = structure_np(wl)
    m = masks_of(wl, region)
    T = len(m["valid"])
    if region_only:
        m = dict(m)
        m["valid"] = m["in_region"].copy()
    if "counts" in hip:
        assert int(hip["counts"][0]) == m["n_scored"], (label, hip["counts"], m["n_scored"])
        assert int(hip["counts"][1]) == m["t_valid"], (label, hip["counts"], m["t_valid"])
    if region_only:
        m["t_valid"] = int(m["valid"].sum())
    valid, inr = m["valid"], m["in_region"]
    # fixed values outside the valid prefix, bit-exact
    inval = ~valid
    assert np.all(hip["logp_s"][inval] == 0.0), label
    if "am_s" in hip:
        assert np.all(hip["am_s"][inval] == -1), label
    for key in ("kl", "kl_rev", "jsd"):
        if not student_only and key in hip:
            assert np.all(hip[key][~inr] == 0.0) and not np.any(np.signbit(hip[key][~inr])), \
                (label, key)
    sel = np.arange(T) if rows is None else np.asarray(rows)
    sel = sel[valid[sel]]
    r = oracle_rows(wl, sel, student_only, extras="kl_rev" in hip or "jsd" in hip)
    worst = {}

    def chk(name, got, want, atol, rtol=0.0):
        err = np.abs(got - want)
        bound = atol + rtol * np.abs(want)
        bad = np.nonzero(~(err <= bound))[0]
        worst[name] = float(err.max()) if err.size else 0.0
        assert bad.size == 0, "%s %s: %d/%d rows off, first row %d got %r want %r" % (
            label, name, bad.size, err.size, sel[bad[0]], got[bad[0]], want[bad[0]])
    chk("logp_s", hip["logp_s"][sel], r["logp_s"], LOGP_ATOL)
    if "am_s" in hip:
        mism = np.nonzero(hip["am_s"][sel] != r["argmax_s"])[0]
        assert mism.size == 0, "%s argmax_s mismatch at rows %s (gap %s)" % (
            label, sel[mism[:5]], r["gap_s"][mism[:5]])
    if not student_only:
        if "logp_t" in hip:
            chk("logp_t", hip["logp_t"][sel], r["logp_t"], LOGP_ATOL)
        if "am_t" in hip:
            mism = np.nonzero(hip["am_t"][sel] != r["argmax_t"])[0]
            assert mism.size == 0, "%s argmax_t mismatch at rows %s (gap %s)" % (
                label, sel[mism[:5]], r["gap_t"][mism[:5]])
        if "kl" in hip:
            want = np.where(inr[sel], r["kl"], 0.0)
            chk("kl", hip["kl"][sel], want, KL_ATOL, KL_RTOL)
        if "kl_rev" in hip:
            want = np.where(inr[sel], r["kl_rev"], 0.0)
            chk("kl_rev", hip["kl_rev"][sel], want, KL_ATOL, KL_RTOL)
        if "jsd" in hip:
            want = np.where(inr[sel], r["jsd"], 0.0)
            chk("jsd", hip["jsd"][sel], want, KL_ATOL, KL_RTOL)
        if check_ce and "ce" in hip and (rows is None or whole_seqs):
            B = len(cu) - 1
            seqs = range(B) if rows is None else whole_seqs
            for b in seqs:
                idx = np.nonzero((m["seq_id"] == b) & inr)[0]
                pos = np.searchsorted(sel, idx)
                assert np.all(sel[np.minimum(pos, sel.size - 1)] == idx), \
                    (label, "sequence %d is not whole in the sample" % b)
                want = -math.fsum(r["logp_s"][pos].tolist()) if idx.size else 0.0
                assert abs(hip["ce"][b] - want) <= CE_RTOL * abs(want) + 1e-3, \
                    (label, b, hip["ce"][b], want)
    n_valid = int(valid.sum())
    line = "%s parity ok on %d of %d valid rows (%.2f%%)%s; worst %s" % (
        label, sel.size, n_valid, 100.0 * sel.size / max(1, n_valid),
        "" if not whole_seqs else "; whole sequences %s (%d rows, CE compared)" % (
            list(whole_seqs), int(np.isin(m["seq_id"][sel], whole_seqs).sum())),
        {k: "%.2e" % v for k, v in worst.items()})
    say(line)
    if label in COVERAGE_LABELS:
        COVERAGE.append(line)
    return r


# Parity lines of the named workloads, printed in the run's terminal summary.
COVERAGE = []
COVERAGE_LABELS = ("tiny", "small", "large_vocab", "long_rollout", "ragged", "multi_turn")


def exact_logit_bound(h_rows, w, scale):
    """Per row, a bound on how far two fp64 evaluations of an exact logit (exact bf16
    products, fp64 sums in any order) can be apart: each errs by at most
    d 2^-53 sum |h_k w_k| <= d 2^-53 |h| |w_v| (taken with an 8x margin)."""
    h = np.asarray(h_rows, dtype=np.float64)
    wn = np.sqrt((np.asarray(w, dtype=np.float64) ** 2).sum(axis=0)).max()
    d = h.shape[1]
    return scale * d * 2.0 ** -50 * np.sqrt((h ** 2).sum(axis=1)) * wn


def check_topk_set(got, z, delta, label):
    """got: 16 vocabulary indices in rank order; z: exact (fp64) logits of the row;
    delta: the rounding bound of one logit. Returns True when the oracle's set is
    unique at this resolution (then got must equal it in rank order wherever the
    ranking is unique); else checks got is a valid top-16 of logits moved by <= delta."""
    K = len(got)
    want = O.topk_set(z, K)
    zs = z[want]
    rest = np.ones(len(z), dtype=bool)
    rest[want] = False
    z17 = z[rest].max() if rest.any() else -np.inf
    assert len(set(got.tolist())) == K and got.min() >= 0 and got.max() < len(z), \
        (label, got)
    gz = z[got]
    # every returned entry at least as large as every other, up to 2 delta
    others = np.ones(len(z), dtype=bool)
    others[got] = False
    top_other = z[others].max() if others.any() else -np.inf
    assert gz.min() >= top_other - 2 * delta, (label, gz.min(), top_other, delta)
    # rank order: non-increasing up to 2 delta, ties (within 2 delta) in any order
    assert np.all(gz[:-1] >= gz[1:] - 2 * delta), (label, gz)
    unique = (zs[-1] - z17) > 2 * delta
    if unique:
        assert set(got.tolist()) == set(want.tolist()), (label, got, want)
        # where neighbouring values are separated, the order is the oracle's
        sep = np.diff(zs) < -2 * delta
        for k in range(K):
            lo_ok = k == 0 or sep[k - 1]
            hi_ok = k == K - 1 or sep[k]
            if lo_ok and hi_ok:
                assert got[k] == want[k], (label, k, got, want)
    return unique


def compare_topk(hip, wl, region=O.REGION_TEACHER, rows=None, label="", region_only=False,
                 max_ambiguous_frac=0.0):
    """Top-K outputs against the oracle: fixed values at unscored positions, sets
    equal to the oracle's where the exact logits rank them uniquely (and valid where
    they tie), overlap exact (equal to the oracle's where both sets are unique),
    kl_topk at the KL tolerance against the oracle's (on the returned teacher set
    where the oracle's is not unique)."""
    m = masks_of(wl, region)
    valid, inr = m["valid"], m["in_region"]
    T = len(valid)
    K = L.OLIVE_TOPK
    uns = ~inr
    if "overlap" in hip:
        assert np.all(hip["overlap"][uns] == 0.0) and not np.any(np.signbit(hip["overlap"][uns]))
    if "kl_topk" in hip:
        assert np.all(hip["kl_topk"][uns] == 0.0) and not np.any(np.signbit(hip["kl_topk"][uns]))
    for k in ("tk_s", "tk_t"):
        if k in hip:
            assert np.all(hip[k][uns] == -1), (label, k)
    sel = np.nonzero(inr)[0] if rows is None else np.asarray(rows)
    sel = sel[inr[sel]]
    if sel.size == 0:
        return
    idx = torch.from_numpy(sel).to(wl["h_student"].device)
    hs, ht = to_np(wl["h_student"][idx]), to_np(wl["h_teacher"][idx])
    ws = to_np(wl["w_student"]).astype(np.float64)
    wt = to_np(wl["w_teacher"]).astype(np.float64)
    sS, sT = wl["scale_student"], wl["scale_teacher"]
    ds = exact_logit_bound(hs, ws, sS)
    dt = exact_logit_bound(ht, wt, sT)
    n_amb = 0
    worst = 0.0
    t0 = time.time()
    for r0 in range(0, sel.size, 64):
        zs_all = O.project(hs[r0:r0 + 64], ws, sS)
        zt_all = O.project(ht[r0:r0 + 64], wt, sT)
        for i in range(zs_all.shape[0]):
            g = int(sel[r0 + i])
            zs, zt = zs_all[i], zt_all[i]
            tag = "%s row %d" % (label, g)
            us = check_topk_set(hip["tk_s"][g], zs, ds[r0 + i], tag + " S") \
                if "tk_s" in hip else True
            ut = check_topk_set(hip["tk_t"][g], zt, dt[r0 + i], tag + " T") \
                if "tk_t" in hip else True
            n_amb += (not us) or (not ut)
            set_s = hip["tk_s"][g] if "tk_s" in hip else None
            set_t = hip["tk_t"][g] if "tk_t" in hip else None
            if "overlap" in hip:
                if us and ut:
                    want = O.topk_overlap(O.topk_set(zs, K), O.topk_set(zt, K), K)
                    assert hip["overlap"][g] == want, (tag, hip["overlap"][g], want)
                if set_s is not None and set_t is not None:
                    own = len(set(set_s.tolist()) & set(set_t.tolist())) / K
                    assert hip["overlap"][g] == own, (tag, hip["overlap"][g], own)
            if "kl_topk" in hip:
                st, tt = O.log_softmax_stats(zs), O.log_softmax_stats(zt)
                tset = O.topk_set(zt, K) if ut or set_t is None else set_t
                want = O.kl_topk(zt, tt["lse"], zs, st["lse"], tset)
                err = abs(hip["kl_topk"][g] - want)
                worst = max(worst, err)
                assert err <= KL_ATOL + KL_RTOL * abs(want), (tag, hip["kl_topk"][g], want)
    assert n_amb <= max_ambiguous_frac * sel.size + 1, (label, n_amb, sel.size)
    say("%s top-K ok on %d rows (%d with a near-tie at the 16th entry); worst kl_topk err "
        "%.2e; oracle %.1fs" % (label, sel.size, n_amb, worst, time.time() - t0))
