"""Plant plausible mistakes in the oracle (on the CPU) and check that the pins fail.

Each mutant replaces one oracle function with a version carrying a single, plausible
slip (a dropped term, a wrong sign or direction, a wrong tie-break, an off-by-one
mask, a lost scale). The pin tests of test_oracle_pins.py are then run against the
mutant and at least one of them must fail.
"""
import math

import numpy as np
import pytest

from oracle import olive_oracle as O
from tests import test_oracle_pins as P

_orig_lss = O.log_softmax_stats
_orig_kl = O.kl_teacher_student
_orig_klr = O.kl_student_teacher
_orig_topk = O.topk_set
_orig_kltk = O.kl_topk
_orig_masks = O.masks
_orig_project = O.project
_orig_glog = O.grad_logits
_orig_backward = O.backward
_orig_jsd = O.jsd


def _jsd_parts(z_s, lse_s, z_t, lse_t):
    lp_s = np.asarray(z_s, dtype=np.float64) - lse_s
    lp_t = np.asarray(z_t, dtype=np.float64) - lse_t
    return lp_s, lp_t


def jsd_geometric_mixture(z_s, lse_s, z_t, lse_t):
    # the mixture taken as the geometric mean of the two distributions
    lp_s, lp_t = _jsd_parts(z_s, lse_s, z_t, lse_t)
    log_m = 0.5 * (lp_s + lp_t)
    return 0.5 * math.fsum((np.exp(lp_s) * (lp_s - log_m)).tolist()) + \
        0.5 * math.fsum((np.exp(lp_t) * (lp_t - log_m)).tolist())


def jsd_mixture_not_halved(z_s, lse_s, z_t, lse_t):
    # log(p_S + p_T) in place of log((p_S + p_T) / 2)
    lp_s, lp_t = _jsd_parts(z_s, lse_s, z_t, lse_t)
    log_m = np.logaddexp(lp_s, lp_t)
    return 0.5 * math.fsum((np.exp(lp_s) * (lp_s - log_m)).tolist()) + \
        0.5 * math.fsum((np.exp(lp_t) * (lp_t - log_m)).tolist())


def jsd_one_sided(z_s, lse_s, z_t, lse_t):
    # KL(p_S || m) alone
    lp_s, lp_t = _jsd_parts(z_s, lse_s, z_t, lse_t)
    log_m = np.logaddexp(lp_s, lp_t) - math.log(2.0)
    return math.fsum((np.exp(lp_s) * (lp_s - log_m)).tolist())


def jsd_not_halved(z_s, lse_s, z_t, lse_t):
    return 2.0 * _orig_jsd(z_s, lse_s, z_t, lse_t)


def lss_dropped_max(z_row):
    r = _orig_lss(z_row)
    z = np.asarray(z_row, dtype=np.float64)
    r["lse"] = math.log(math.fsum(np.exp(z - r["max"]).tolist()))
    return r


def lss_last_index(z_row):
    r = _orig_lss(z_row)
    z = np.asarray(z_row, dtype=np.float64)
    r["argmax"] = int(len(z) - 1 - np.argmax(z[::-1]))
    return r


def lss_plain_sum_of_logits(z_row):
    r = _orig_lss(z_row)
    z = np.asarray(z_row, dtype=np.float64)
    r["lse"] = r["max"] + math.log(math.fsum(np.exp(z - r["max"]).tolist()) + 1.0 / len(z))
    return r


def kl_reversed(z_t, lse_t, z_s, lse_s):
    return _orig_kl(z_s, lse_s, z_t, lse_t)


def kl_wrong_sign(z_t, lse_t, z_s, lse_s):
    a, b = _orig_kl(z_t, lse_t, z_s, lse_s)
    return -a, -b


def klr_forward(z_s, lse_s, z_t, lse_t):
    return _orig_klr(z_t, lse_t, z_s, lse_s)


def klr_dropped_cross_term(z_s, lse_s, z_t, lse_t):
    # sum p_S log p_S only (the entropy part): forgets the teacher term
    a, b = _orig_klr(z_s, lse_s, z_s, lse_s)
    lp = np.asarray(z_s, dtype=np.float64) - lse_s
    ent = -math.fsum((np.exp(lp) * lp).tolist())
    return a - ent, b - ent


def topk_ties_high_index(z_row, k):
    z = np.asarray(z_row, dtype=np.float64)
    order = np.lexsort((-np.arange(len(z)), -z))
    return order[:k].astype(np.int64)


def kl_topk_renormalised(z_t, lse_t, z_s, lse_s, set_t):
    idx = np.asarray(set_t, dtype=np.int64)
    zt = np.asarray(z_t, dtype=np.float64)[idx]
    zs = np.asarray(z_s, dtype=np.float64)[idx]
    lt = zt - (zt.max() + math.log(np.exp(zt - zt.max()).sum()))
    ls = zs - (zs.max() + math.log(np.exp(zs - zs.max()).sum()))
    return math.fsum((np.exp(lt) * (lt - ls)).tolist())


def overlap_jaccard(set_s, set_t, k=O.TOPK):
    a, b = set(np.asarray(set_s).tolist()), set(np.asarray(set_t).tolist())
    return len(a & b) / float(len(a | b))


def masks_off_by_one(cu_seqlens, cut, valid_len=None, region=O.REGION_TEACHER, spans=None):
    return _orig_masks(cu_seqlens, np.asarray(cut) + 1, valid_len, region, spans)


def masks_ignore_valid(cu_seqlens, cut, valid_len=None, region=O.REGION_TEACHER, spans=None):
    return _orig_masks(cu_seqlens, cut, None, region, spans)


def masks_span_end_inclusive(cu_seqlens, cut, valid_len=None, region=O.REGION_TEACHER,
                             spans=None):
    if spans is not None:
        spans = [[(a, e + 1) for (a, e) in sp] for sp in spans]
    return _orig_masks(cu_seqlens, cut, valid_len, region, spans)


def project_no_scale(h_rows, w, scale=1.0):
    return _orig_project(h_rows, w, 1.0)


def project_dropped_last_k(h_rows, w, scale=1.0):
    h = np.asarray(h_rows, dtype=np.float64).copy()
    if h.shape[1] > 1:
        h[:, -1] = 0.0
    return _orig_project(h, w, scale)


def glog_kl_sign(z_s, lse_s, y, w_ce=1.0, z_t=None, lse_t=None, w_kl=0.0):
    # the KL part as p_T - p_S
    g = _orig_glog(z_s, lse_s, y, w_ce, z_t, lse_t, 0.0)
    if w_kl != 0.0:
        g -= w_kl * (np.exp(np.asarray(z_s, dtype=np.float64) - lse_s) -
                     np.exp(np.asarray(z_t, dtype=np.float64) - lse_t))
    return g


def glog_target_off_by_one(z_s, lse_s, y, w_ce=1.0, z_t=None, lse_t=None, w_kl=0.0):
    V = len(z_s)
    return _orig_glog(z_s, lse_s, (int(y) + 1) % V, w_ce, z_t, lse_t, w_kl)


def glog_ce_weight_on_softmax_dropped(z_s, lse_s, y, w_ce=1.0, z_t=None, lse_t=None, w_kl=0.0):
    g = _orig_glog(z_s, lse_s, y, w_ce, z_t, lse_t, w_kl)
    return g - w_ce * np.exp(np.asarray(z_s, dtype=np.float64) - lse_s)


def backward_no_scale(*args, **kw):
    r = _orig_backward(*args, **kw)
    s = kw.get("scale_student", args[8] if len(args) > 8 else 1.0)
    r["grad_h"] = r["grad_h"] / s
    return r


def backward_grad_w_unscaled_rows(*args, **kw):
    # dW formed from the logit gradient without the hidden states' scale
    r = _orig_backward(*args, **kw)
    if r["grad_w"] is not None:
        s = kw.get("scale_student", args[8] if len(args) > 8 else 1.0)
        r["grad_w"] = r["grad_w"] / s
    return r


MUTANTS = [
    ("log_softmax_stats", lss_dropped_max),
    ("log_softmax_stats", lss_last_index),
    ("log_softmax_stats", lss_plain_sum_of_logits),
    ("kl_teacher_student", kl_reversed),
    ("kl_teacher_student", kl_wrong_sign),
    ("kl_student_teacher", klr_forward),
    ("kl_student_teacher", klr_dropped_cross_term),
    ("masks", masks_off_by_one),
    ("masks", masks_ignore_valid),
    ("masks", masks_span_end_inclusive),
    ("topk_set", topk_ties_high_index),
    ("kl_topk", kl_topk_renormalised),
    ("topk_overlap", overlap_jaccard),
    ("project", project_no_scale),
    ("project", project_dropped_last_k),
    ("grad_logits", glog_kl_sign),
    ("grad_logits", glog_target_off_by_one),
    ("grad_logits", glog_ce_weight_on_softmax_dropped),
    ("backward", backward_no_scale),
    ("backward", backward_grad_w_unscaled_rows),
    ("jsd", jsd_geometric_mixture),
    ("jsd", jsd_mixture_not_halved),
    ("jsd", jsd_one_sided),
    ("jsd", jsd_not_halved),
]

PINS = [
    lambda: [P.test_decimal_brute_force(s) for s in range(6)],
    P.test_golden_worked_examples,
    lambda: [P.test_equal_columns_give_uniform(V) for V in (1, 2, 7, 1000)],
    P.test_two_token_softplus_and_bernoulli_kl,
    P.test_probabilities_sum_to_one_and_lse_bounds,
    P.test_kl_nonnegative_and_two_forms_agree,
    P.test_kl_cross_entropy_identity,
    P.test_kl_zero_for_identical_models_and_row_shift,
    P.test_peaked_student_limit_of_reverse_kl,
    P.test_argmax_exact_ties_take_lowest_index,
    P.test_mask_counts_enumerated,
    P.test_eq1_masks_prefix_and_scores_continuation,
    P.test_span_masks_reduce_to_the_cut_regions_and_add_up,
    P.test_topk_set_ties_take_lower_indices,
    P.test_topk_worked_example,
    P.test_topk_reduces_to_argmax_and_to_the_full_kl,
    P.test_masked_outputs_exact_values,
    lambda: [P.test_backward_matches_finite_differences(r, sp) for r, sp in
             ((O.REGION_TEACHER, None), (O.REGION_SPANS, [[(0, 2), (3, 5)], [(1, 4)]]))],
    P.test_backward_invariants,
    lambda: [P.test_jsd_decimal_entropy_form(s) for s in range(4)],
    P.test_jsd_bounds_symmetry_and_limits,
    P.test_jsd_two_tokens_closed_form,
]


@pytest.mark.parametrize("target,mutant", MUTANTS, ids=[m.__name__ for _, m in MUTANTS])
def test_pins_catch_mutant(monkeypatch, target, mutant):
    monkeypatch.setattr(O, target, mutant)
    caught = 0
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            caught += 1
    assert caught >= 1, "no pin caught mutant %s" % mutant.__name__
