"""The seeded workload generator: structure, ranges and the target-sampling law.

Target sampling is input synthesis, not part of the scoring; its only check is
distributional ("parity unpinned" for the draw itself): the mean log-prob of
sampled tokens must match minus the entropy of the law they were drawn from.
"""
import math

import numpy as np
import torch

from oracle import olive_oracle as O
from paper_2609_36246_amd import workloads as W


def test_structure_ranges_all_workloads():
    for name in W.WORKLOAD_ORDER:
        spec = W.WORKLOADS[name]
        s = W.draw_structure(spec, 0)
        cu, cut, vl = s["cu_seqlens"].astype(np.int64), s["cut"], s["valid_len"]
        lengths = np.diff(cu)
        assert cu[0] == 0 and np.all(lengths >= 0) and len(cut) == spec.num_seqs
        kind, lo, hi = spec.cut_rule
        if spec.turns is not None:
            check_turns(spec, s)
        elif kind == "abs":
            assert np.all(cut >= lo) and np.all(cut <= hi)
            assert np.all(lengths == spec.seq_len)
        else:
            assert np.all(cut >= np.ceil(lo * lengths)) and np.all(cut <= np.floor(hi * lengths))
            a, b = spec.ragged_len
            assert np.all(lengths >= a) and np.all(lengths <= b)
        if spec.eos:
            assert np.all(vl > cut) and np.all(vl <= lengths)
        else:
            assert vl is None
        assert len(s["outlier_rows"]) == int(round(spec.outlier_frac * cu[-1]))
        # same seed, same structure
        s2 = W.draw_structure(spec, 0)
        np.testing.assert_array_equal(s2["cut"], cut)


def check_turns(spec, s):
    """Multi-turn structure: the cut is the first teacher turn, one span per teacher
    action, spans inside the sequence, increasing and disjoint, lengths within the
    per-turn ranges."""
    p_lo, p_hi, k, m, a_lo, a_hi, o_lo, o_hi = spec.turns
    lengths = np.diff(s["cu_seqlens"].astype(np.int64))
    off = s["span_offsets"]
    assert off[0] == 0 and off[-1] == len(s["span_pairs"])
    for b, sp in enumerate(s["spans"]):
        assert len(sp) == m and off[b + 1] - off[b] == m
        np.testing.assert_array_equal(s["span_pairs"][off[b]:off[b + 1]], np.array(sp))
        assert sp[0][0] == s["cut"][b]
        assert p_lo + k * (a_lo + o_lo) <= s["cut"][b] <= p_hi + k * (a_hi + o_hi)
        prev = 0
        for (a, e) in sp:
            assert prev <= a and a_lo <= e - a <= a_hi
            prev = e + o_lo
        assert prev - o_lo + o_lo <= lengths[b] <= sp[-1][1] + o_hi
    assert s["valid_len"] is None


def test_ragged_total_positions_near_expectation():
    s = W.draw_structure(W.WORKLOADS["ragged"], 0)
    T = s["total_positions"]
    assert 64 * 128 <= T <= 64 * 8192
    assert abs(T - 64 * (128 + 8192) / 2) < 6 * math.sqrt(64 * (8064 ** 2) / 12)


def test_tiny_workload_shapes_and_dtypes():
    w = W.make_workload("tiny", 0)
    assert w["h_student"].shape == (64, 64) and w["h_teacher"].shape == (64, 96)
    assert w["w_student"].shape == (64, 1000) and w["w_teacher"].shape == (96, 1000)
    assert w["h_student"].dtype == torch.float32
    assert w["targets"].dtype == torch.int32
    assert int(w["targets"].min()) >= 0 and int(w["targets"].max()) < 1000
    w2 = W.make_workload("tiny", 0)
    assert torch.equal(w["h_student"], w2["h_student"])
    assert torch.equal(w["targets"], w2["targets"])


def test_gumbel_targets_follow_the_softmax():
    spec = W.custom_spec(num_seqs=4, seq_len=500, vocab=64, d_student=16, d_teacher=16,
                         dtype="bf16", logit_scale=2.0, target_source="student",
                         cut_rule=("abs", 1, 499))
    w = W.make_workload("custom", 3, spec=spec)
    h = w["h_student"].float().numpy()
    ws = w["w_student"].float().numpy()
    y = w["targets"].numpy()
    r = O.row_scores(h, ws, y, 2.0)
    z = O.project(h, ws, 2.0)
    lp = z - r["lse_s"][:, None]
    ent = -(np.exp(lp) * lp).sum(axis=1)
    var = (np.exp(lp) * lp ** 2).sum(axis=1) - ent ** 2
    n = len(y)
    dev = (r["logp_s"].sum() + ent.sum()) / math.sqrt(var.sum())
    assert abs(dev) < 5.0, dev
