"""GPU parity of the backward pass (dL/dh_S, dL/dW_S of w_ce sum_b CE_b + w_kl sum_t
KL(p_T || p_S) over the region) against the fp64 oracle, through the C ABI.

Tolerance per element, from the arithmetic: the logit gradient g is held in bf16
(round to nearest even: error <= 2^-9 |g|, taken as 2^-8 to cover the fp32
exponentials and normalisers it is formed from) and the products accumulate K terms
in fp32 (error <= K 2^-24 of the magnitude sum). With the magnitude sums
S_h[t,k] = sum_v |g_tv| |W_kv| and S_w[k,v] = sum_t |h_tk| |g_tv| (oracle values):
  |dh - dh*| <= s (2^-8 + V 2^-24) S_h + 1e-6,   |dW - dW*| <= s (2^-8 + R 2^-24) S_w + 1e-6
with R the number of scored rows.
"""
import numpy as np
import pytest
import torch

from oracle import olive_oracle as O
from paper_2609_36246_amd import _lib as L
from paper_2609_36246_amd import workloads as W
from tests.gpu_harness import masks_of, say, structure_np, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    L.load()


def custom(name, seed=0, **kw):
    spec = W.custom_spec(name=name, **kw)
    return W.make_workload(name, seed, device="cuda", spec=spec)


def run_backward(wl, w_ce=1.0, w_kl=0.0, region=L.OLIVE_REGION_TEACHER, want=("h", "w"),
                 layout=L.OLIVE_W_DV, ctx=None, keep_ctx=False, narrow=False):
    spec = wl["spec"]
    T = wl["total_positions"]
    B = wl["cu_seqlens"].shape[0] - 1
    dev = wl["h_student"].device
    own = ctx is None
    if own:
        ws, wt = wl["w_student"], wl["w_teacher"]
        if layout == L.OLIVE_W_VD:
            ws, wt = ws.t().contiguous(), wt.t().contiguous()
        desc = L.make_desc(spec.vocab, spec.d_student, spec.d_teacher, L.OLIVE_BF16, layout,
                           wl["scale_student"], wl["scale_teacher"], max_positions=T,
                           max_seqs=B, flags=L.OLIVE_FLAG_BACKWARD |
                           (L.OLIVE_FLAG_NARROW_TILE if narrow else 0))
        ctx = L.olive_score_init(desc, ws, wt)
    gh = torch.full((T, spec.d_student), float("nan"), dtype=torch.float32, device=dev) \
        if "h" in want else None
    gw = torch.full((spec.d_student * spec.vocab,), float("nan"), dtype=torch.float32,
                    device=dev) if "w" in want else None
    spans = wl.get("spans") if region == L.OLIVE_REGION_SPANS else None
    batch = L.make_batch(wl["cu_seqlens"], None if spans is not None else wl["cut"],
                         wl["targets"], wl["h_student"], wl["h_teacher"], wl["valid_len"],
                         region)
    sp = L.make_spans(wl["span_offsets"], wl["span_pairs"]) if spans is not None else None
    counts = torch.full((2,), -1, dtype=torch.int64, device=dev)
    g = L.make_grad_outputs(w_ce, w_kl, gh, gw, counts)
    L.olive_score_backward(ctx, batch, g, spans=sp)
    torch.cuda.synchronize()
    out = {"err": L.olive_score_last_error(ctx), "counts": counts.cpu().numpy()}
    if gh is not None:
        out["h"] = to_np(gh)
    if gw is not None:
        gwn = to_np(gw)
        out["w"] = gwn.reshape(spec.d_student, spec.vocab) if layout == L.OLIVE_W_DV \
            else gwn.reshape(spec.vocab, spec.d_student).T
    if keep_ctx:
        out["ctx"] = ctx
    elif own:
        L.olive_score_free(ctx)
    return out


def oracle_backward(wl, w_ce, w_kl, region, rows=None, cols=None):
    cu, cut, vl = structure_np(wl)
    spans = wl.get("spans") if region == O.REGION_SPANS else None
    hs, ws = to_np(wl["h_student"]), to_np(wl["w_student"])
    ht = to_np(wl["h_teacher"]) if w_kl else None
    wt = to_np(wl["w_teacher"]) if w_kl else None
    return O.backward(hs, ws, to_np(wl["targets"]), cu, cut, vl, ht, wt, wl["scale_student"],
                      wl["scale_teacher"], region, spans, w_ce, w_kl, rows=rows, cols=cols,
                      keep_g=True)


def check_grads(hip, ref, wl, label, rows=None, cols=None):
    s = wl["scale_student"]
    ws = to_np(wl["w_student"]).astype(np.float64)
    hs = to_np(wl["h_student"]).astype(np.float64)
    V = ws.shape[1]
    g = ref["g"]
    sel = ref["rows"]
    worst = {}
    if "h" in hip:
        inr = ref["in_region"]
        out = np.nonzero(~inr)[0]
        assert np.all(hip["h"][out] == 0.0), (label, "grad_h outside the region")
        check_rows = sel if rows is None else np.intersect1d(rows, sel)
        pos = np.searchsorted(sel, check_rows)
        S_h = np.abs(g[pos]) @ np.abs(ws.T)
        tol = s * (2.0 ** -8 + V * 2.0 ** -24) * S_h + 1e-6
        err = np.abs(hip["h"][check_rows] - ref["grad_h"][check_rows])
        bad = np.argwhere(err > tol)
        worst["h"] = float((err / tol).max()) if err.size else 0.0
        assert bad.size == 0, "%s grad_h off at %s: got %r want %r tol %r" % (
            label, bad[:3], hip["h"][check_rows][tuple(bad[0])],
            ref["grad_h"][check_rows][tuple(bad[0])], tol[tuple(bad[0])])
    if "w" in hip and ref["grad_w"] is not None:
        R = len(sel)
        gc = g if cols is None else g[:, cols]
        S_w = np.abs(hs[sel].T) @ np.abs(gc)
        tol = s * (2.0 ** -8 + R * 2.0 ** -24) * S_w + 1e-6
        got = hip["w"] if cols is None else hip["w"][:, cols]
        err = np.abs(got - ref["grad_w"])
        bad = np.argwhere(err > tol)
        worst["w"] = float((err / tol).max()) if err.size else 0.0
        assert bad.size == 0, "%s grad_w off at %s: got %r want %r tol %r" % (
            label, bad[:3], got[tuple(bad[0])], ref["grad_w"][tuple(bad[0])], tol[tuple(bad[0])])
    say("%s backward ok; worst err/tol %s" % (label, worst))


CASES = {
    "ragged_v1000": dict(num_seqs=3, ragged_len=(40, 300), vocab=1000, d_student=128,
                         d_teacher=256, cut_rule=("frac", 0.1, 0.9), eos=True),
    "multi_tile": dict(num_seqs=5, ragged_len=(700, 1300), vocab=5000, d_student=256,
                       d_teacher=128, logit_scale=4.0, target_source="student",
                       cut_rule=("frac", 0.1, 0.9)),
    "narrow_k": dict(num_seqs=2, ragged_len=(100, 250), vocab=700, d_student=64,
                     d_teacher=192, cut_rule=("frac", 0.2, 0.8)),
    "even_v": dict(num_seqs=2, seq_len=200, vocab=2048, d_student=384, d_teacher=512,
                   target_source="teacher", cut_rule=("abs", 1, 199), outlier_frac=0.05,
                   outlier_mul=8.0),
    # V % 4 != 0: the shifted last vocabulary tile starts off 4-row alignment (at 1 and
    # at 745), so its first new row sits inside a 4-row group of the tile's lanes
    "v257": dict(num_seqs=2, seq_len=150, vocab=257, d_student=64, d_teacher=64,
                 logit_scale=2.0, cut_rule=("abs", 1, 149)),
    "v1001": dict(num_seqs=3, ragged_len=(60, 200), vocab=1001, d_student=128,
                  d_teacher=64, target_source="student", cut_rule=("frac", 0.1, 0.9)),
    # wider hidden states over several 256-row position tiles and a ragged vocabulary
    "d512": dict(num_seqs=4, ragged_len=(300, 700), vocab=3001, d_student=512,
                 d_teacher=256, logit_scale=2.0, cut_rule=("frac", 0.1, 0.9)),
}


@pytest.mark.parametrize("w_kl", [0.0, 0.5], ids=["ce", "ce+kl"])
@pytest.mark.parametrize("case", list(CASES))
def test_backward_full(case, w_kl):
    say("backward", case, "w_kl", w_kl)
    wl = custom(case, **CASES[case])
    hip = run_backward(wl, 1.0, w_kl)
    assert hip["err"] == 0
    m = masks_of(wl, O.REGION_TEACHER)
    assert list(hip["counts"]) == [m["n_scored"], m["t_valid"]]
    ref = oracle_backward(wl, 1.0, w_kl, O.REGION_TEACHER)
    check_grads(hip, ref, wl, "%s-%s" % (case, w_kl))


# The cross-entropy's normaliser and logit-gradient passes run on the 256 x 256 kernel by
# default; OLIVE_FLAG_NARROW_TILE keeps them on the 256 x 128 one.
@pytest.mark.parametrize("case", ["ragged_v1000", "v257"])
def test_backward_narrow_tile(case):
    say("backward, 256 x 128 kernel", case)
    wl = custom(case, **CASES[case])
    hip = run_backward(wl, 1.0, 0.0, narrow=True)
    assert hip["err"] == 0
    ref = oracle_backward(wl, 1.0, 0.0, O.REGION_TEACHER)
    check_grads(hip, ref, wl, "narrow-%s" % case)


@pytest.mark.parametrize("region", [O.REGION_STUDENT, O.REGION_ALL])
def test_backward_regions_and_kl_only(region):
    say("backward region", region)
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    hip = run_backward(wl, 0.0, 1.0, region)
    ref = oracle_backward(wl, 0.0, 1.0, region)
    check_grads(hip, ref, wl, "region%d" % region)


# w_kl = 0: the cross-entropy alone takes the 256 x 256 logit-gradient pass
@pytest.mark.parametrize("w_kl", [0.25, 0.0], ids=["ce+kl", "ce"])
def test_backward_spans_and_vd_layout(w_kl):
    say("backward with span masks, weights in the [V][d] layout, w_kl", w_kl)
    wl = custom("turns", num_seqs=3, vocab=1000, d_student=128, d_teacher=256,
                target_source="teacher", turns=(4, 16, 3, 2, 4, 24, 4, 40))
    hip = run_backward(wl, 1.0, w_kl, O.REGION_SPANS, layout=L.OLIVE_W_VD)
    assert hip["err"] == 0
    ref = oracle_backward(wl, 1.0, w_kl, O.REGION_SPANS)
    check_grads(hip, ref, wl, "turns-vd-%s" % w_kl)


def test_backward_chunks_and_repeat():
    """More scored rows than one gradient chunk (8192): the dW product accumulates
    over chunks. A second call on the same context gives the same bits."""
    say("backward over two chunks")
    wl = custom("chunks", num_seqs=3, seq_len=3200, vocab=600, d_student=64, d_teacher=64,
                cut_rule=("abs", 1, 10))
    a = run_backward(wl, 1.0, 0.0, keep_ctx=True)
    b = run_backward(wl, 1.0, 0.0, ctx=a["ctx"])
    L.olive_score_free(a["ctx"])
    np.testing.assert_array_equal(a["h"], b["h"])
    np.testing.assert_array_equal(a["w"], b["w"])
    m = masks_of(wl, O.REGION_TEACHER)
    assert m["n_scored"] > 8192
    ref = oracle_backward(wl, 1.0, 0.0, O.REGION_TEACHER)
    check_grads(a, ref, wl, "chunks")


def test_backward_second_chunk_with_wider_rows():
    """d_S = 256 (whole 256-row blocks of dL/dh) on the second gradient chunk's rows."""
    say("backward over two chunks, d_S = 256")
    wl = custom("chunks256", num_seqs=3, seq_len=3200, vocab=600, d_student=256,
                d_teacher=64, cut_rule=("abs", 1, 10))
    hip = run_backward(wl, 1.0, 0.0)
    m = masks_of(wl, O.REGION_TEACHER)
    assert m["n_scored"] > 8192
    ref = oracle_backward(wl, 1.0, 0.0, O.REGION_TEACHER)
    check_grads(hip, ref, wl, "chunks256")


def test_backward_empty_region_gives_zero():
    say("backward, empty region")
    wl = custom("empty", num_seqs=2, seq_len=64, vocab=1000, d_student=128, d_teacher=128,
                cut_rule=("abs", 64, 64))
    hip = run_backward(wl, 1.0, 0.5)
    assert np.all(hip["h"] == 0.0) and np.all(hip["w"] == 0.0)


def test_backward_on_long_rollout_sampled():
    """The long-rollout workload (CE only, the loss of Eq. 1): dL/dh on sampled scored
    rows and dL/dW on sampled vocabulary columns (each needs every scored row)."""
    say("backward, long_rollout sampled")
    wl = W.make_workload("long_rollout", 0, device="cuda")
    hip = run_backward(wl, 1.0, 0.0)
    assert hip["err"] == 0
    m = masks_of(wl, O.REGION_TEACHER)
    inr = np.nonzero(m["in_region"])[0]
    rng = np.random.default_rng(7)
    rows = np.sort(rng.choice(inr, size=24, replace=False))
    y = to_np(wl["targets"])
    cols = np.unique(np.concatenate([y[rows[:8]], rng.choice(wl["spec"].vocab, 16,
                                                             replace=False)]))
    ref_h = oracle_backward(wl, 1.0, 0.0, O.REGION_TEACHER, rows=rows)
    check_grads({"h": hip["h"]}, ref_h, wl, "long_rollout-h", rows=rows)
    cu, cut, vl = structure_np(wl)
    ref_w = O.backward(to_np(wl["h_student"]), to_np(wl["w_student"]), y, cu, cut, vl,
                       scale_student=wl["scale_student"], w_ce=1.0, w_kl=0.0, cols=cols,
                       keep_g=False)
    # the magnitude sums of the tolerance need g at the kept columns for every row:
    # recompute them per chunk from the oracle's own logit gradient
    hs = to_np(wl["h_student"]).astype(np.float64)
    ws = to_np(wl["w_student"]).astype(np.float64)
    S_w = np.zeros((hs.shape[1], len(cols)))
    sel = ref_w["rows"]
    for r0 in range(0, len(sel), 256):
        idx = sel[r0:r0 + 256]
        zs = O.project(hs[idx], ws, wl["scale_student"])
        gb = np.stack([O.grad_logits(zs[i], O.log_softmax_stats(zs[i])["lse"], y[t])[cols]
                       for i, t in enumerate(idx)])
        S_w += np.abs(hs[idx].T) @ np.abs(gb)
    tol = wl["scale_student"] * (2.0 ** -8 + len(sel) * 2.0 ** -24) * S_w + 1e-6
    err = np.abs(hip["w"][:, cols] - ref_w["grad_w"])
    assert np.all(err <= tol), ("grad_w", float((err / tol).max()))
    say("long_rollout dW columns ok; worst err/tol %.3f" % float((err / tol).max()))
    del wl
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode", ["ce", "ce+kl", "ce+kl-topk", "ce+kl-reverse"])
def test_backward_reuses_forward_normalisers(mode):
    """OLIVE_GRAD_REUSE_FORWARD: the normalisers of the preceding forward call on the same
    batch stand in for the backward's own pass (from the top-K workspace when that call
    asked for top-K outputs; from the student-first 256 x 256 kernel when it asked for
    the reverse KL alone). The gradients meet the same bar and repeat bit for bit; the
    flag is refused once no matching forward call holds them."""
    say("backward reusing the forward normalisers", mode)
    w_kl = 0.0 if mode == "ce" else 0.5
    topk = mode.endswith("topk")
    rev = mode.endswith("reverse")
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    spec = wl["spec"]
    T = wl["total_positions"]
    B = wl["cu_seqlens"].shape[0] - 1
    dev = wl["h_student"].device
    flags = L.OLIVE_FLAG_BACKWARD | (L.OLIVE_FLAG_TOPK if topk else 0)
    desc = L.make_desc(spec.vocab, spec.d_student, spec.d_teacher, L.OLIVE_BF16, L.OLIVE_W_DV,
                       wl["scale_student"], wl["scale_teacher"], max_positions=T,
                       max_seqs=B, flags=flags)
    ctx = L.olive_score_init(desc, wl["w_student"], wl["w_teacher"])

    def batch_of(region):
        return L.make_batch(wl["cu_seqlens"], wl["cut"], wl["targets"], wl["h_student"],
                            wl["h_teacher"], wl["valid_len"], region)

    def forward(batch):
        kl = torch.empty(T, dtype=torch.float32, device=dev)
        ov = torch.empty(T, dtype=torch.float32, device=dev) if topk else None
        L.olive_score_batch(ctx, batch, L.make_outputs(kl=None if rev else kl,
                                                       kl_reverse=kl if rev else None,
                                                       topk_overlap=ov))
        if rev:
            assert L.olive_score_last_stats(ctx)["tile"] == "256x256"

    def backward(batch, reuse, check=True):
        gh = torch.full((T, spec.d_student), float("nan"), dtype=torch.float32, device=dev)
        gw = torch.full((spec.d_student * spec.vocab,), float("nan"), dtype=torch.float32,
                        device=dev)
        g = L.make_grad_outputs(1.0, w_kl, gh, gw, reuse_forward=reuse)
        st = L.olive_score_backward(ctx, batch, g, check=check)
        torch.cuda.synchronize()
        return st, {"h": to_np(gh), "w": to_np(gw).reshape(spec.d_student, spec.vocab)}

    batch = batch_of(L.OLIVE_REGION_TEACHER)
    forward(batch)
    _, a = backward(batch, True)
    _, b = backward(batch, True)
    np.testing.assert_array_equal(a["h"], b["h"])
    np.testing.assert_array_equal(a["w"], b["w"])
    ref = oracle_backward(wl, 1.0, w_kl, O.REGION_TEACHER)
    check_grads(a, ref, wl, "reuse-" + mode)
    # a backward without the flag replaces the normalisers
    backward(batch, False)
    assert backward(batch, True, check=False)[0] == L.OLIVE_E_RANGE
    # the last forward call was on another batch (another region)
    forward(batch)
    forward(batch_of(L.OLIVE_REGION_ALL))
    assert backward(batch, True, check=False)[0] == L.OLIVE_E_RANGE
    if w_kl:
        # a student-only forward call holds no teacher normalisers
        lp = torch.empty(T, dtype=torch.float32, device=dev)
        L.olive_token_logprobs(ctx, batch, lp)
        assert backward(batch, True, check=False)[0] == L.OLIVE_E_RANGE
    assert L.olive_score_last_error(ctx) == 0
    L.olive_score_free(ctx)


def test_backward_reuse_after_a_region_only_span_forward():
    """OLIVE_GRAD_REUSE_FORWARD after a region-only forward call with span masks, weights
    in the [V][d] layout: the region-only compaction gives the scored rows the indices the
    backward uses."""
    say("backward reusing a region-only span forward, [V][d] weights")
    wl = custom("turns", num_seqs=3, vocab=1000, d_student=128, d_teacher=256,
                target_source="teacher", turns=(4, 16, 3, 2, 4, 24, 4, 40))
    spec = wl["spec"]
    T = wl["total_positions"]
    B = wl["cu_seqlens"].shape[0] - 1
    dev = wl["h_student"].device
    desc = L.make_desc(spec.vocab, spec.d_student, spec.d_teacher, L.OLIVE_BF16, L.OLIVE_W_VD,
                       wl["scale_student"], wl["scale_teacher"], max_positions=T,
                       max_seqs=B, flags=L.OLIVE_FLAG_BACKWARD)
    ctx = L.olive_score_init(desc, wl["w_student"].t().contiguous(),
                             wl["w_teacher"].t().contiguous())
    batch = L.make_batch(wl["cu_seqlens"], None, wl["targets"], wl["h_student"],
                         wl["h_teacher"], wl["valid_len"], L.OLIVE_REGION_SPANS)
    sp = L.make_spans(wl["span_offsets"], wl["span_pairs"])
    kl = torch.empty(T, dtype=torch.float32, device=dev)
    L.olive_score_batch_spans(ctx, batch, sp,
                              L.make_outputs(kl=kl, flags=L.OLIVE_OUT_REGION_ONLY))
    gh = torch.full((T, spec.d_student), float("nan"), dtype=torch.float32, device=dev)
    gw = torch.full((spec.vocab * spec.d_student,), float("nan"), dtype=torch.float32,
                    device=dev)
    g = L.make_grad_outputs(1.0, 0.25, gh, gw, reuse_forward=True)
    L.olive_score_backward(ctx, batch, g, spans=sp)
    torch.cuda.synchronize()
    assert L.olive_score_last_error(ctx) == 0
    L.olive_score_free(ctx)
    hip = {"h": to_np(gh), "w": to_np(gw).reshape(spec.vocab, spec.d_student).T}
    ref = oracle_backward(wl, 1.0, 0.25, O.REGION_SPANS)
    check_grads(hip, ref, wl, "reuse-spans-vd")


def test_backward_argument_errors():
    say("backward argument errors")
    wl = custom("narrow_k", **CASES["narrow_k"])
    spec = wl["spec"]
    T = wl["total_positions"]
    dev = wl["h_student"].device
    gh = torch.zeros((T, spec.d_student), dtype=torch.float32, device=dev)
    batch = L.make_batch(wl["cu_seqlens"], wl["cut"], wl["targets"], wl["h_student"],
                         wl["h_teacher"], wl["valid_len"], L.OLIVE_REGION_TEACHER)
    # a context without the backward workspace
    desc = L.make_desc(spec.vocab, spec.d_student, spec.d_teacher, L.OLIVE_BF16, L.OLIVE_W_DV,
                       1.0, 1.0, max_positions=T, max_seqs=4)
    ctx = L.olive_score_init(desc, wl["w_student"], wl["w_teacher"])
    g = L.make_grad_outputs(1.0, 0.0, gh)
    assert L.olive_score_backward(ctx, batch, g, check=False) == L.OLIVE_E_UNSUPPORTED
    L.olive_score_free(ctx)
    desc.flags = L.OLIVE_FLAG_BACKWARD
    ctx = L.olive_score_init(desc, wl["w_student"], wl["w_teacher"])
    bad = L.make_grad_outputs(1.0, 0.0, gh)
    bad.size = 8
    assert L.olive_score_backward(ctx, batch, bad, check=False) == L.OLIVE_E_RANGE
    assert L.olive_score_backward(ctx, batch, L.make_grad_outputs(float("nan"), 0.0, gh),
                                  check=False) == L.OLIVE_E_RANGE
    assert L.olive_score_backward(ctx, batch, L.make_grad_outputs(1.0, 0.0),
                                  check=False) == L.OLIVE_E_NULL
    L.olive_score_free(ctx)
    # KL weight on a student-only context
    desc0 = L.make_desc(spec.vocab, spec.d_student, 0, L.OLIVE_BF16, L.OLIVE_W_DV, 1.0, 1.0,
                        max_positions=T, max_seqs=4, flags=L.OLIVE_FLAG_BACKWARD)
    ctx = L.olive_score_init(desc0, wl["w_student"], None)
    assert L.olive_score_backward(ctx, batch, L.make_grad_outputs(1.0, 0.5, gh),
                                  check=False) == L.OLIVE_E_UNSUPPORTED
    assert L.olive_score_backward(ctx, batch, L.make_grad_outputs(1.0, 0.0, gh)) == L.OLIVE_OK
    L.olive_score_free(ctx)
    # an fp32 context cannot take the flag
    desc32 = L.make_desc(spec.vocab, spec.d_student, spec.d_teacher, L.OLIVE_F32, L.OLIVE_W_DV,
                         1.0, 1.0, max_positions=T, max_seqs=4, flags=L.OLIVE_FLAG_BACKWARD)
    w32 = torch.zeros(spec.d_teacher * spec.vocab, dtype=torch.float32, device=dev)
    status, handle = L.olive_score_init(desc32, w32, w32, check=False)
    assert status == L.OLIVE_E_UNSUPPORTED and handle is None


@pytest.mark.parametrize("narrow", [False, True], ids=["one_pass", "narrow_tile"])
def test_backward_bad_target_row(narrow):
    """A realised token out of range in one scored row: the error word's target bit is
    set, that row's normaliser and so its gradient row are NaN, and every other row of
    dL/dh is what it is without the bad row (rows do not mix in dL/dh). The cross-entropy
    backward of a context with the 256 x 256 kernel forms its normalisers in its own
    logit-gradient pass; with OLIVE_FLAG_NARROW_TILE it runs the separate normaliser
    pass: both treat the row alike."""
    say("backward with a bad target", "narrow" if narrow else "one pass")
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    ref = oracle_backward(wl, 1.0, 0.0, O.REGION_TEACHER)
    inr = masks_of(wl, O.REGION_TEACHER)["in_region"]
    r = int(np.nonzero(inr)[0][7])
    wl["targets"][r] = wl["spec"].vocab
    hip = run_backward(wl, 1.0, 0.0, want=("h",), narrow=narrow)
    assert hip["err"] & 1
    assert np.all(np.isnan(hip["h"][r]))
    # every other row at the bar of the backward tests (the bad row stands in for itself)
    rest = {"h": hip["h"].copy()}
    rest["h"][r] = ref["grad_h"][r]
    check_grads(rest, ref, wl, "bad-target-%s" % ("narrow" if narrow else "one-pass"))
