"""GPU parity of the HIP scoring path against the fp64 oracle (through the C ABI).

Small workloads are compared on every position (they span several vocabulary and
position tiles and end in ragged tails); of the five named workloads, tiny, small and
large_vocab are compared on every row, long_rollout and ragged on at least 1% of their
valid rows including two whole sequences, at the launch configuration the benchmark
times. Masks and counts are always compared in full.
"""
import numpy as np
import pytest
import torch

from oracle import olive_oracle as O
from paper_2609_36246_amd import _lib as L
from paper_2609_36246_amd import workloads as W
from tests.gpu_harness import (CE_RTOL, KL_ATOL, KL_RTOL, LOGP_ATOL, compare, masks_of,
                               oracle_rows, parity_rows, run_hip, say, stratified_rows,
                               to_np)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    L.load()


def custom(name, seed=0, **kw):
    spec = W.custom_spec(name=name, **kw)
    return W.make_workload(name, seed, device="cuda", spec=spec)


CASES = {
    # ragged lengths, V not a multiple of 256, EOS cut-off, 3 position tiles
    "ragged_v1000": dict(num_seqs=3, ragged_len=(40, 300), vocab=1000, d_student=128,
                         d_teacher=256, cut_rule=("frac", 0.1, 0.9), eos=True),
    # several vocabulary tiles per split, many position tiles, peaked (scale 4)
    "multi_tile": dict(num_seqs=5, ragged_len=(700, 1300), vocab=5000, d_student=256,
                       d_teacher=128, logit_scale=4.0, target_source="student",
                       cut_rule=("frac", 0.1, 0.9)),
    # one K step for the student, an odd count (3) for the teacher: short unit pipelines
    "narrow_k": dict(num_seqs=2, ragged_len=(100, 250), vocab=700, d_student=64,
                     d_teacher=192, cut_rule=("frac", 0.2, 0.8)),
    # last vocabulary tile with a single valid row: whole lanes see only masked rows
    "v257": dict(num_seqs=2, seq_len=150, vocab=257, d_student=64, d_teacher=64,
                 logit_scale=2.0, cut_rule=("abs", 1, 149)),
    # vocabulary a multiple of 256, teacher-sampled targets, outlier rows
    "even_v": dict(num_seqs=2, seq_len=200, vocab=2048, d_student=384, d_teacher=512,
                   target_source="teacher", cut_rule=("abs", 1, 199), outlier_frac=0.05,
                   outlier_mul=8.0),
}


@pytest.mark.parametrize("kernel", ["wide", "narrow", "generic"])
@pytest.mark.parametrize("case", list(CASES))
def test_custom_parity_full(case, kernel):
    say("custom parity", case, kernel)
    wl = custom(case, **CASES[case])
    hip = run_hip(wl, simple=kernel == "generic", narrow=kernel == "narrow")
    assert hip["stats"]["kernel"] == ("generic" if kernel == "generic" else "mfma")
    if kernel != "generic":
        assert hip["stats"]["tile"] == ("256x128" if kernel == "narrow" else "256x256")
    assert hip["err"] == 0
    compare(hip, wl, label="%s/%s" % (case, kernel))


def _weighted_mad(wl, rows, under="teacher"):
    """Per row: the mean absolute deviation of the scaled logit difference z_T - z_S
    under p_T (or under p_S with under="student"), fp64, from the oracle's
    projections."""
    f = lambda t: (t.float() if t.dtype == torch.bfloat16 else t).cpu().numpy()
    hs, ht = f(wl["h_student"])[rows], f(wl["h_teacher"])[rows]
    zs = O.project(hs, f(wl["w_student"]), wl["scale_student"])
    zt = O.project(ht, f(wl["w_teacher"]), wl["scale_teacher"])
    zw = zt if under == "teacher" else zs
    out = []
    for i in range(len(rows)):
        lw = O.log_softmax_stats(zw[i])["lse"]
        pw = np.exp(zw[i] - lw)
        d = zt[i] - zs[i]
        dbar = float(np.sum(pw * d))
        out.append(float(np.sum(pw * np.abs(d - dbar))))
    return np.array(out)


@pytest.mark.parametrize("case", ["multi_tile", "even_v"])
def test_wide_kl_error_within_its_weight_rounding_bound(case):
    # The 256 x 256 kernel forms KL's cross term with the teacher's softmax weights in
    # fp16, normalised by their own sum: the rounding (relative error <= 2^-11) moves a
    # KL value by at most 2^-11 / (1 - 2^-11) times the teacher-weighted mean absolute
    # deviation of the logit difference. Beyond that, the kernel may differ from the
    # oracle only as the 256 x 128 kernel (fp32 weights) does.
    say("wide KL bound", case)
    wl = custom(case, **CASES[case])
    wide = run_hip(wl)
    narrow = run_hip(wl, narrow=True)
    assert wide["stats"]["tile"] == "256x256" and narrow["stats"]["tile"] == "256x128"
    rows = np.nonzero(masks_of(wl, O.REGION_TEACHER)["in_region"])[0]
    assert rows.size > 100
    ref = oracle_rows(wl, rows, extras=False)["kl"]
    mad = _weighted_mad(wl, rows)
    u = 2.0 ** -11
    err_w = np.abs(wide["kl"][rows] - ref)
    err_n = np.abs(narrow["kl"][rows] - ref)
    bound = u / (1 - u) * mad + 2 * err_n + 1e-6 * (1 + np.abs(ref))
    worst = np.max(err_w / bound)
    say("  rows %d  max |dKL| wide %.2e narrow %.2e  worst error / bound %.3f"
        % (rows.size, err_w.max(), err_n.max(), worst))
    assert np.all(err_w <= bound)


@pytest.mark.parametrize("region", [O.REGION_TEACHER, O.REGION_STUDENT, O.REGION_ALL])
def test_regions(region):
    say("regions", region)
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    hip = run_hip(wl, region=region)
    compare(hip, wl, region=region, label="region%d" % region)


def test_widths_off_the_mfma_step_take_the_generic_kernel():
    say("hidden widths not multiples of 64")
    wl = custom("w96", num_seqs=2, ragged_len=(60, 140), vocab=900, d_student=96,
                d_teacher=160, cut_rule=("frac", 0.2, 0.8))
    hip = run_hip(wl)
    assert hip["stats"]["kernel"] == "generic"
    compare(hip, wl, label="w96")


def test_misaligned_hidden_states_take_the_generic_kernel():
    say("hidden states not 16-byte aligned")
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    for key in ("h_student", "h_teacher"):
        h = wl[key]
        buf = torch.empty(h.numel() + 1, dtype=h.dtype, device=h.device)
        view = buf[1:].view(h.shape)          # 2-byte offset from the allocation
        view.copy_(h)
        assert view.data_ptr() % 16 != 0
        wl[key] = view
    hip = run_hip(wl)
    assert hip["stats"]["kernel"] == "generic"
    compare(hip, wl, label="misaligned")


def test_different_scales_general_difference_path():
    say("different logit scales")
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    wl["scale_student"], wl["scale_teacher"] = 1.0, 2.5
    for simple in (False, True):
        hip = run_hip(wl, simple=simple)
        compare(hip, wl, label="scales-%s" % ("generic" if simple else "mfma"))


ALL_OUT = ("kl", "kl_rev", "counts", "logp_s", "logp_t", "am_s", "am_t", "ce")
# One KL direction: the 256 x 256 kernel (teacher block first for the forward KL, the
# student's for the reverse KL alone); both directions: the 256 x 128 kernel.
FWD_OUT = tuple(k for k in ALL_OUT if k != "kl_rev")
REV_OUT = tuple(k for k in ALL_OUT if k != "kl")
OUTSETS = {"both": ALL_OUT, "forward": FWD_OUT, "reverse": REV_OUT}


def tile_of(outs):
    return "256x128" if outs == "both" else "256x256"


@pytest.mark.parametrize("simple", [False, True], ids=["mfma", "generic"])
@pytest.mark.parametrize("case", ["ragged_v1000", "multi_tile", "narrow_k", "v257"])
def test_reverse_kl_full(case, simple):
    say("reverse KL", case, "generic" if simple else "mfma")
    wl = custom(case, **CASES[case])
    hip = run_hip(wl, simple=simple, outputs=ALL_OUT)
    assert hip["stats"]["kernel"] == ("generic" if simple else "mfma")
    compare(hip, wl, label="rev-" + case)


@pytest.mark.parametrize("region", [O.REGION_STUDENT, O.REGION_ALL])
def test_reverse_kl_regions_and_scales(region):
    say("reverse KL region", region)
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    wl["scale_student"], wl["scale_teacher"] = 2.0, 0.5
    for simple in (False, True):
        hip = run_hip(wl, region=region, simple=simple, outputs=ALL_OUT)
        compare(hip, wl, region=region, label="rev-scales-%d" % region)


@pytest.mark.parametrize("both", [True, False], ids=["both_directions", "reverse_only"])
def test_reverse_kl_on_long_rollout_sampled(both):
    say("reverse KL, long_rollout sampled", "both" if both else "reverse only")
    wl = W.make_workload("long_rollout", 0, device="cuda")
    hip = run_hip(wl, outputs=ALL_OUT if both else REV_OUT)
    assert hip["stats"]["kernel"] == "mfma"
    assert hip["stats"]["tile"] == ("256x128" if both else "256x256")
    compare(hip, wl, rows=stratified_rows(wl, n_random=64), label="rev-long_rollout")
    del wl
    torch.cuda.empty_cache()



@pytest.mark.parametrize("case", list(CASES))
def test_reverse_kl_alone_on_the_wide_kernel(case):
    say("reverse KL alone", case)
    wl = custom(case, **CASES[case])
    hip = run_hip(wl, outputs=REV_OUT)
    assert hip["stats"]["kernel"] == "mfma" and hip["stats"]["tile"] == "256x256"
    assert hip["err"] == 0 and "kl" not in hip
    compare(hip, wl, label="rev-wide-" + case)
    # the narrow tile still takes the same call
    nar = run_hip(wl, outputs=REV_OUT, narrow=True)
    assert nar["stats"]["tile"] == "256x128"
    compare(nar, wl, label="rev-narrow-" + case)


@pytest.mark.parametrize("region", [O.REGION_TEACHER, O.REGION_STUDENT, O.REGION_ALL])
@pytest.mark.parametrize("scales", [(2.0, 0.5), (1.5, 1.5)], ids=["scales_differ", "scales_equal"])
def test_reverse_kl_alone_regions_and_scales(region, scales):
    say("reverse KL alone region", region, scales)
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    wl["scale_student"], wl["scale_teacher"] = scales
    hip = run_hip(wl, region=region, outputs=REV_OUT)
    assert hip["stats"]["tile"] == "256x256"
    compare(hip, wl, region=region, label="rev-wide-scales-%d" % region)


@pytest.mark.parametrize("direction", ["forward", "reverse"])
def test_wide_kl_of_equal_models_is_zero_to_rounding(direction):
    # Identical weights and hidden rows: the cross term (the first model's fp16 weights
    # times its own logits, minus the same weights times the other model's bit-identical
    # logits) is exactly 0. The two log-normalisers come from different fold orders (the
    # first model's sums are rescaled once per tile, the second's once per block), so
    # the KL is their difference: zero up to the rounding of a log-normaliser.
    say("wide kernel, teacher == student", direction)
    wl = custom("multi_tile", **dict(CASES["multi_tile"], d_teacher=256))
    wl["w_teacher"], wl["h_teacher"] = wl["w_student"], wl["h_student"]
    wl["scale_teacher"] = wl["scale_student"]
    key = "kl" if direction == "forward" else "kl_rev"
    outs = ("kl", "counts", "logp_s", "logp_t", "am_s", "am_t") if direction == "forward" \
        else REV_OUT
    hip = run_hip(wl, region=O.REGION_ALL, outputs=outs)
    assert hip["stats"]["tile"] == "256x256"
    lse_mag = np.max(np.abs(hip["logp_s"]))
    say("  max |%s| %.2e  max |logp_s - logp_t| %.2e  max |logp| %.1f"
        % (key, np.max(np.abs(hip[key])), np.max(np.abs(hip["logp_s"] - hip["logp_t"])),
           lse_mag))
    assert np.max(np.abs(hip[key])) <= 1e-5
    np.testing.assert_allclose(hip["logp_s"], hip["logp_t"], rtol=0, atol=1e-5)
    np.testing.assert_array_equal(hip["am_s"], hip["am_t"])


@pytest.mark.parametrize("case", ["multi_tile", "even_v"])
def test_wide_reverse_kl_error_within_its_weight_rounding_bound(case):
    # As for the forward KL, with the student's fp16 weights: the rounding moves a
    # reverse-KL value by at most 2^-11 / (1 - 2^-11) times the student-weighted mean
    # absolute deviation of the logit difference, beyond the 256 x 128 kernel's error.
    say("wide reverse KL bound", case)
    wl = custom(case, **CASES[case])
    wide = run_hip(wl, outputs=REV_OUT)
    narrow = run_hip(wl, outputs=REV_OUT, narrow=True)
    assert wide["stats"]["tile"] == "256x256" and narrow["stats"]["tile"] == "256x128"
    rows = np.nonzero(masks_of(wl, O.REGION_TEACHER)["in_region"])[0]
    assert rows.size > 100
    ref = oracle_rows(wl, rows)["kl_rev"]
    mad = _weighted_mad(wl, rows, under="student")
    u = 2.0 ** -11
    err_w = np.abs(wide["kl_rev"][rows] - ref)
    err_n = np.abs(narrow["kl_rev"][rows] - ref)
    bound = u / (1 - u) * mad + 2 * err_n + 1e-6 * (1 + np.abs(ref))
    worst = np.max(err_w / bound)
    say("  rows %d  max |dKL_rev| wide %.2e narrow %.2e  worst error / bound %.3f"
        % (rows.size, err_w.max(), err_n.max(), worst))
    assert np.all(err_w <= bound)


# ----------------------------------------------------------------------------- span masks
TURNS_CASE = dict(num_seqs=3, vocab=1000, d_student=128, d_teacher=256, target_source="teacher",
                  turns=(4, 16, 3, 2, 4, 24, 4, 40))


@pytest.mark.parametrize("outs", list(OUTSETS))
@pytest.mark.parametrize("simple", [False, True], ids=["mfma", "generic"])
def test_span_masks_full(simple, outs):
    say("span masks", "generic" if simple else "mfma", outs)
    wl = custom("turns", **TURNS_CASE)
    hip = run_hip(wl, region=L.OLIVE_REGION_SPANS, simple=simple, outputs=OUTSETS[outs])
    assert hip["err"] == 0
    if not simple:
        assert hip["stats"]["tile"] == tile_of(outs)
    compare(hip, wl, region=O.REGION_SPANS, label="spans-" + outs)


@pytest.mark.parametrize("outs", list(OUTSETS))
def test_spans_equal_to_the_cut_region_reproduce_it(outs):
    say("spans [cut, len) == teacher region", outs)
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    cu = wl["cu_seqlens"].cpu().numpy()
    cut = wl["cut"].cpu().numpy()
    lens = np.diff(cu)
    wl["spans"] = [[(int(c), int(n))] for c, n in zip(cut, lens)]
    wl["span_offsets"] = torch.arange(len(lens) + 1, dtype=torch.int32, device="cuda")
    wl["span_pairs"] = torch.tensor([[int(c), int(n)] for c, n in zip(cut, lens)],
                                    dtype=torch.int32, device="cuda")
    a = run_hip(wl, region=L.OLIVE_REGION_SPANS, outputs=OUTSETS[outs])
    b = run_hip(wl, region=L.OLIVE_REGION_TEACHER, outputs=OUTSETS[outs])
    assert a["stats"]["tile"] == b["stats"]["tile"] == tile_of(outs)
    for k in OUTSETS[outs]:
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)


def test_empty_spans_score_nothing():
    say("no spans")
    wl = custom("turns", **TURNS_CASE)
    B = wl["cu_seqlens"].shape[0] - 1
    wl["spans"] = [[] for _ in range(B)]
    wl["span_offsets"] = torch.zeros(B + 1, dtype=torch.int32, device="cuda")
    wl["span_pairs"] = torch.zeros((0, 2), dtype=torch.int32, device="cuda")
    hip = run_hip(wl, region=L.OLIVE_REGION_SPANS, outputs=ALL_OUT)
    assert int(hip["counts"][0]) == 0 and hip["err"] == 0
    assert np.all(hip["kl"] == 0.0) and np.all(hip["kl_rev"] == 0.0) and np.all(hip["ce"] == 0.0)
    compare(hip, wl, region=O.REGION_SPANS, label="no-spans")


def test_malformed_spans_set_the_error_word():
    say("malformed spans")
    wl = custom("turns", **TURNS_CASE)
    pairs = wl["span_pairs"].clone()
    # overlap the first two spans of sequence 1 (entries 2 and 3)
    pairs[3, 0] = pairs[2, 1] - 1
    wl["span_pairs"] = pairs
    hip = run_hip(wl, region=L.OLIVE_REGION_SPANS, outputs=ALL_OUT)
    assert hip["err"] & 16
    cu = wl["cu_seqlens"].cpu().numpy()
    assert np.all(np.isnan(hip["logp_s"][cu[1]:cu[2]]))
    assert np.isnan(hip["ce"][1]) and not np.isnan(hip["ce"][0]) and not np.isnan(hip["ce"][2])
    assert not np.any(np.isnan(hip["logp_s"][cu[0]:cu[1]]))
    # offsets that do not end at S: every sequence is rejected
    wl2 = custom("turns", **TURNS_CASE)
    off = wl2["span_offsets"].clone()
    off[-1] += 1
    wl2["span_offsets"] = off
    hip2 = run_hip(wl2, region=L.OLIVE_REGION_SPANS, outputs=ALL_OUT)
    assert hip2["err"] & 16 and np.all(np.isnan(hip2["logp_s"]))


@pytest.mark.parametrize("outs", list(OUTSETS))
@pytest.mark.parametrize("simple", [False, True], ids=["mfma", "generic"])
@pytest.mark.parametrize("case", ["ragged_v1000", "turns"])
def test_region_only_scores_just_the_region(case, simple, outs):
    say("region only", case, "generic" if simple else "mfma", outs)
    if case == "turns":
        wl, region = custom("turns", **TURNS_CASE), O.REGION_SPANS
    else:
        wl, region = custom(case, **CASES[case]), O.REGION_TEACHER
    hip = run_hip(wl, region=region, simple=simple, outputs=OUTSETS[outs],
                  out_flags=L.OLIVE_OUT_REGION_ONLY)
    assert hip["err"] == 0
    if not simple:
        assert hip["stats"]["tile"] == tile_of(outs)
    compare(hip, wl, region=region, region_only=True, label="region-only-%s-%s" % (case, outs))
    # the compacted rows are the scored ones
    full = run_hip(wl, region=region, simple=simple, outputs=OUTSETS[outs])
    np.testing.assert_array_equal(hip["counts"], full["counts"])


@pytest.mark.parametrize("outs", ["both", "forward"])
def test_multi_turn_workload_sampled(outs):
    say("multi_turn workload sampled", outs)
    wl = W.make_workload("multi_turn", 0, device="cuda")
    hip = run_hip(wl, region=L.OLIVE_REGION_SPANS, outputs=OUTSETS[outs])
    say("multi_turn stats", hip["stats"])
    assert hip["stats"]["kernel"] == "mfma" and hip["err"] == 0
    assert hip["stats"]["tile"] == tile_of(outs)
    compare(hip, wl, region=O.REGION_SPANS, rows=stratified_rows(wl, n_random=48),
            label="multi_turn-" + outs)
    del wl
    torch.cuda.empty_cache()


# student-only contexts: every block of a unit is a student block (one K step each in
# narrow_k and v257), so each block end moves to the next vocabulary tile; both MFMA
# kernels take them (the 256 x 256 one by default)
@pytest.mark.parametrize("narrow", [False, True], ids=["wide", "narrow"])
@pytest.mark.parametrize("case", ["ragged_v1000", "multi_tile", "narrow_k", "v257"])
def test_student_only_token_logprobs(case, narrow):
    say("student only", case, "narrow" if narrow else "wide")
    wl = custom(case, **CASES[case])
    hip = run_hip(wl, student_only=True, outputs=("logp_s", "am_s"), narrow=narrow)
    assert hip["stats"]["kernel"] == "mfma"
    assert hip["stats"]["tile"] == ("256x128" if narrow else "256x256")
    compare(hip, wl, student_only=True, label="student-only-" + case)


def test_tiny_workload_full():
    say("tiny workload (fp32, generic kernel)")
    wl = W.make_workload("tiny", 0, device="cuda")
    hip = run_hip(wl)
    assert hip["stats"]["kernel"] == "generic"
    compare(hip, wl, label="tiny")


def test_small_workload_full():
    say("small workload full parity")
    wl = W.make_workload("small", 0, device="cuda")
    hip = run_hip(wl)
    assert hip["stats"]["kernel"] == "mfma"
    say("small stats", hip["stats"])
    compare(hip, wl, label="small")


def test_large_vocab_workload_full():
    say("large_vocab workload, full parity on every row")
    wl = W.make_workload("large_vocab", 0, device="cuda")
    hip = run_hip(wl)
    say("large_vocab stats", hip["stats"])
    assert hip["stats"]["kernel"] == "mfma" and hip["err"] == 0
    compare(hip, wl, label="large_vocab")
    del wl
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["long_rollout", "ragged"])
def test_large_workload_sampled(name):
    """At least 1% of the valid rows: every row of the two sequences with the fewest
    valid rows (their per-sequence loss compared too), the rows around every cut and
    end of the valid prefix, and random valid rows; masks and counts in full."""
    say("workload", name, "sampled parity")
    wl = W.make_workload(name, 0, device="cuda")
    hip = run_hip(wl)
    say(name, "stats", hip["stats"])
    assert hip["stats"]["kernel"] == "mfma" and hip["err"] == 0
    rows, whole = parity_rows(wl, frac=0.01, n_whole=2)
    compare(hip, wl, rows=rows, whole_seqs=whole, label=name)
    del wl
    torch.cuda.empty_cache()


# ----------------------------------------------------------------------------- properties
def test_vocabulary_permutation_permutes_the_outputs():
    """Metamorphic: relabel the vocabulary (W columns permuted, targets mapped the same
    way). Log-probs, both KLs and the per-sequence loss are functions of the logit
    multiset and keep their values up to fp32 summation order (held to the acceptance
    bar); greedy tokens map through the permutation (random logits have no exact
    ties)."""
    say("vocabulary permutation")
    wl = custom("multi_tile", **CASES["multi_tile"])
    a = run_hip(wl, outputs=ALL_OUT)
    V = wl["spec"].vocab
    perm = torch.from_numpy(np.random.default_rng(5).permutation(V)).cuda()   # v -> perm[v]
    inv = torch.argsort(perm)
    for key in ("w_student", "w_teacher"):
        wl[key] = wl[key][:, inv].contiguous()          # new column perm[v] = old column v
    wl["targets"] = perm[wl["targets"].long()].to(torch.int32)
    b = run_hip(wl, outputs=ALL_OUT)
    p = perm.cpu().numpy()
    valid = a["am_s"] >= 0
    for k in ("am_s", "am_t"):
        np.testing.assert_array_equal(b[k][valid], p[a[k][valid]], err_msg=k)
        np.testing.assert_array_equal(b[k][~valid], a[k][~valid], err_msg=k)
    np.testing.assert_array_equal(a["counts"], b["counts"])
    for k in ("logp_s", "logp_t"):
        assert np.max(np.abs(a[k] - b[k])) <= LOGP_ATOL, k
    for k in ("kl", "kl_rev"):
        assert np.all(np.abs(a[k] - b[k]) <= KL_ATOL + KL_RTOL * np.abs(a[k])), k
        assert np.all((a[k] == 0.0) == (b[k] == 0.0)), k
    assert np.all(np.abs(a["ce"] - b["ce"]) <= CE_RTOL * np.abs(a["ce"]) + 1e-3)
    compare(b, wl, label="permuted-vocab")


@pytest.mark.parametrize("case,order", [("ragged_v1000", [2, 0, 1]),
                                        ("multi_tile", [4, 3, 2, 1, 0])])
def test_sequence_reordering_permutes_the_outputs(case, order):
    """Metamorphic: reorder the sequences of the packed batch (cu_seqlens, cuts, valid
    lengths, hidden rows and targets moved together). Rows are scored independently,
    with the same vocabulary splits and fixed merge orders, so every per-position output
    moves with its row bit for bit, and the per-sequence losses are permuted."""
    say("sequence reordering", case, order)
    wl = custom(case, **CASES[case])
    a = run_hip(wl, outputs=ALL_OUT)
    cu = wl["cu_seqlens"].cpu().numpy().astype(np.int64)
    src = np.concatenate([np.arange(cu[b], cu[b + 1]) for b in order])   # new row -> old row
    lens = np.diff(cu)[order]
    ncu = np.zeros(len(order) + 1, dtype=np.int32)
    np.cumsum(lens, out=ncu[1:])
    idx = torch.from_numpy(src).cuda()
    wl2 = dict(wl)
    for key in ("h_student", "h_teacher"):
        wl2[key] = wl[key][idx].contiguous()
    wl2["targets"] = wl["targets"][idx].contiguous()
    wl2["cu_seqlens"] = torch.from_numpy(ncu).cuda()
    o = torch.tensor(order, dtype=torch.long).cuda()
    wl2["cut"] = wl["cut"][o].contiguous()
    wl2["valid_len"] = None if wl["valid_len"] is None else wl["valid_len"][o].contiguous()
    b = run_hip(wl2, outputs=ALL_OUT)
    for k in ("kl", "kl_rev", "logp_s", "logp_t", "am_s", "am_t"):
        np.testing.assert_array_equal(b[k], a[k][src], err_msg=k)
    np.testing.assert_array_equal(b["ce"], a["ce"][order])
    np.testing.assert_array_equal(b["counts"], a["counts"])


def test_identical_teacher_gives_exact_zero_kl():
    say("teacher == student")
    wl = custom("multi_tile", **CASES["multi_tile"])
    wl["h_teacher"] = wl["h_student"]
    wl["w_teacher"] = wl["w_student"]
    spec = wl["spec"]
    wl["spec"] = W.custom_spec(name="same", num_seqs=spec.num_seqs, ragged_len=spec.ragged_len,
                               vocab=spec.vocab, d_student=spec.d_student,
                               d_teacher=spec.d_student, logit_scale=spec.logit_scale)
    for simple in (False, True):
        hip = run_hip(wl, simple=simple, region=O.REGION_ALL, outputs=ALL_OUT)
        assert np.all(hip["kl"] == 0.0)
        assert np.all(hip["kl_rev"] == 0.0)
        np.testing.assert_array_equal(hip["logp_s"], hip["logp_t"])
        np.testing.assert_array_equal(hip["am_s"], hip["am_t"])


def plant_ulp_pair(w, h, a, b, k, scale=4.0):
    """Make columns a < b of w [d, V] the two largest logits of every row, one bf16 ulp
    apart in row k: both get w[0] = scale (h[:, 0] = scale lifts them by scale^2), equal
    entries elsewhere, and w[k, b] = w[k, a] + ulp with w[k, a] = 2^-10. The exact
    winner is then b where h[:, k] > 0 and a (the lower index) where h[:, k] <= 0, with a
    gap of |h[:, k]| 2^-17 -- far inside the fp32 near-tie window."""
    w[:, b] = w[:, a]
    w[0, a] = w[0, b] = scale
    w[k, a] = 2.0 ** -10
    w[k, b] = 2.0 ** -10 + 2.0 ** -17
    h[:, 0] = scale


@pytest.mark.parametrize("simple", [False, True], ids=["mfma", "generic"])
def test_more_near_ties_than_one_window(simple):
    """Every one of 20,000 rows has its two best logits one bf16 ulp apart (both
    models): each row is flagged, queued and re-decided exactly -- more than the 8192
    rows one window of the generic path's re-decision holds -- and every greedy token
    equals the oracle's."""
    say("20k near-tied rows", "generic" if simple else "mfma")
    wl = custom("ulp_pairs", num_seqs=4, seq_len=5000, vocab=512, d_student=64, d_teacher=64,
                cut_rule=("abs", 1, 4999))
    plant_ulp_pair(wl["w_student"], wl["h_student"], 100, 140, 3)
    plant_ulp_pair(wl["w_teacher"], wl["h_teacher"], 7, 300, 5)
    hip = run_hip(wl, simple=simple)
    T = wl["total_positions"]
    say("stats", hip["stats"])
    assert hip["stats"]["flagged"] == T > 8192, hip["stats"]
    hk_s = wl["h_student"][:, 3].float().cpu().numpy()
    hk_t = wl["h_teacher"][:, 5].float().cpu().numpy()
    np.testing.assert_array_equal(hip["am_s"], np.where(hk_s > 0, 140, 100))
    np.testing.assert_array_equal(hip["am_t"], np.where(hk_t > 0, 300, 7))
    compare(hip, wl, label="ulp-pairs-" + ("generic" if simple else "mfma"))


def test_duplicate_best_column_takes_lowest_index():
    say("duplicate best column")
    wl = custom("even_v", **CASES["even_v"])
    hip = run_hip(wl)
    # copy the winning column of row 0 to a lower index: every row whose greedy token
    # was that column now ties, and must report the lower index
    j = int(hip["am_s"][0])
    lo = j // 3
    wl["w_student"][:, lo] = wl["w_student"][:, j]
    hip2 = run_hip(wl)
    tied = hip["am_s"] == j
    assert tied.any()
    assert np.all(hip2["am_s"][tied] == lo)
    compare(hip2, wl, label="dup-column")


# Exact greedy ties placed in the winner's own 256-row tile (its split must be read
# again) and/or in another split (decided from the per-split maximum and argmax alone).
# narrow_k's widths (64 and 192: one and three K steps) take the filter's odd tail.
@pytest.mark.parametrize("partner", ["same_tile", "other_split", "both"])
@pytest.mark.parametrize("case", ["even_v", "multi_tile", "narrow_k"])
def test_greedy_ties_within_and_across_splits(case, partner):
    say("greedy ties", case, partner)
    wl = custom(case, **CASES[case])
    hip = run_hip(wl)
    V = wl["spec"].vocab
    for key, am in (("w_student", hip["am_s"]), ("w_teacher", hip["am_t"])):
        j = int(am[am >= 0][0])
        near = j ^ 1 if (j ^ 1) < V else j - 1
        far = (j + V // 2) % V
        partners = {"same_tile": [near], "other_split": [far], "both": [near, far]}[partner]
        for p in partners:
            wl[key][:, p] = wl[key][:, j]
        tied = am == j
        assert tied.any()
        expect = min([j] + partners)
        hip2 = run_hip(wl)
        got = hip2["am_s"] if key == "w_student" else hip2["am_t"]
        assert np.all(got[tied] == expect), (key, j, partners)
    compare(hip2, wl, label="ties-%s-%s" % (case, partner))


def test_one_context_across_batches_of_different_sizes():
    """Per-call state (counts, near-tie lists, filter queues and split masks) starts
    afresh on every call: one context scores a batch with a planted greedy tie, a
    smaller batch of the same weights, and the first batch again."""
    say("one context, three calls")
    big = custom("multi_tile", **CASES["multi_tile"])
    kw = dict(CASES["multi_tile"])
    kw.update(num_seqs=2, ragged_len=(60, 200))
    small = custom("multi_tile_small", **kw)
    assert torch.equal(small["w_student"], big["w_student"])
    assert torch.equal(small["w_teacher"], big["w_teacher"])
    # a tie in the winner's own tile: the greedy filter must read that split again
    am = run_hip(big)["am_s"]
    j = int(am[am >= 0][0])
    p = j ^ 1 if (j ^ 1) < big["spec"].vocab else j - 1
    for w in (big, small):
        w["w_student"][:, p] = w["w_student"][:, j]
    first = run_hip(big, outputs=ALL_OUT, keep_ctx=True)
    ctx = first["ctx"]
    try:
        compare(first, big, label="ctx-call1")
        second = run_hip(small, outputs=ALL_OUT, ctx=ctx)
        compare(second, small, label="ctx-call2")
        third = run_hip(big, outputs=ALL_OUT, ctx=ctx)
        compare(third, big, label="ctx-call3")
        for k in ("kl", "kl_rev", "logp_s", "logp_t", "am_s", "am_t", "ce", "counts"):
            np.testing.assert_array_equal(first[k], third[k], err_msg=k)
    finally:
        L.olive_score_free(ctx)


def test_deterministic_and_fully_written():
    say("determinism / poisoned outputs")
    wl = custom("multi_tile", **CASES["multi_tile"])
    a = run_hip(wl, poison=True)
    b = run_hip(wl, poison=True)
    for k in ("kl", "logp_s", "logp_t", "ce"):
        assert not np.isnan(a[k]).any(), k
        np.testing.assert_array_equal(a[k], b[k])
    for k in ("am_s", "am_t"):
        np.testing.assert_array_equal(a[k], b[k])


def test_concurrent_calls_on_two_streams_match_calls_alone():
    """Two contexts score two batches at once on two streams, with tiles long enough
    (d_S + d_T = 1024) for the 256 x 256 kernel's phase lock. Both launches then read
    and write the one device array of tile start times; those steer timing only, so
    every output equals, bit for bit, the same call made alone."""
    say("two streams at once, phase-locked kernels")
    kw = dict(num_seqs=4, ragged_len=(400, 900), vocab=6000, d_student=512, d_teacher=512,
              cut_rule=("frac", 0.1, 0.9))
    wls = [custom("conc%d" % i, seed=i, **kw) for i in range(2)]
    alone = [run_hip(wl) for wl in wls]
    assert all(r["stats"]["tile"] == "256x256" for r in alone)
    ctxs, outs, batches = [], [], []
    for wl in wls:
        spec, T = wl["spec"], wl["total_positions"]
        B = wl["cu_seqlens"].shape[0] - 1
        desc = L.make_desc(spec.vocab, spec.d_student, spec.d_teacher, L.OLIVE_BF16,
                           L.OLIVE_W_DV, wl["scale_student"], wl["scale_teacher"],
                           max_positions=T, max_seqs=B)
        ctxs.append(L.olive_score_init(desc, wl["w_student"], wl["w_teacher"]))
        dev = wl["h_student"].device
        outs.append(dict(kl=torch.full((T,), float("nan"), device=dev),
                         counts=torch.full((2,), -1, dtype=torch.int64, device=dev),
                         logp_s=torch.full((T,), float("nan"), device=dev),
                         logp_t=torch.full((T,), float("nan"), device=dev),
                         am_s=torch.full((T,), -7, dtype=torch.int32, device=dev),
                         am_t=torch.full((T,), -7, dtype=torch.int32, device=dev),
                         ce=torch.full((B,), float("nan"), device=dev)))
        batches.append(L.make_batch(wl["cu_seqlens"], wl["cut"], wl["targets"],
                                    wl["h_student"], wl["h_teacher"], wl["valid_len"]))
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for _ in range(3):
        for i in range(2):
            o = outs[i]
            L.olive_kl_masked(ctxs[i], batches[i], o["kl"], o["counts"], o["logp_s"],
                              o["logp_t"], o["am_s"], o["am_t"], o["ce"], streams[i])
    torch.cuda.synchronize()
    for i in range(2):
        assert L.olive_score_last_error(ctxs[i]) == 0
        for k in ("kl", "logp_s", "logp_t", "am_s", "am_t", "ce", "counts"):
            np.testing.assert_array_equal(to_np(outs[i][k]), alone[i][k], err_msg=k)
        L.olive_score_free(ctxs[i])


def test_cut_extremes():
    say("cut = 0 and cut = len")
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    cu = wl["cu_seqlens"].cpu().numpy()
    lens = np.diff(cu)
    wl["valid_len"] = None
    wl["cut"] = torch.zeros_like(wl["cut"])
    h0 = run_hip(wl)
    assert int(h0["counts"][0]) == int(h0["counts"][1]) == int(cu[-1])
    compare(h0, wl, label="cut0")
    wl["cut"] = torch.from_numpy(lens.astype(np.int32)).cuda()
    hl = run_hip(wl)
    assert int(hl["counts"][0]) == 0
    assert np.all(hl["kl"] == 0.0) and np.all(hl["ce"] == 0.0)


def test_bad_target_sets_error_word_and_nan():
    say("bad target")
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    wl["valid_len"] = None
    wl["targets"][5] = wl["spec"].vocab + 3
    hip = run_hip(wl)
    assert hip["err"] & 1
    assert np.isnan(hip["logp_s"][5])
    assert not np.isnan(hip["logp_s"][6])
