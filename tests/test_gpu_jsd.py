"""GPU parity of the Jensen-Shannon divergence output (olive_score_outputs.jsd): the
second MFMA pass over the scored positions, against the fp64 oracle through the C ABI,
at the KL tolerance (1e-3 + 1e-3 |JSD|), exactly +0.0 outside the region."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import olive_oracle as O
from paper_2609_36246_amd import _lib as L
from paper_2609_36246_amd import workloads as W
from tests.gpu_harness import compare, run_hip, say, stratified_rows
from tests.test_gpu_parity import CASES, TURNS_CASE, custom

pytestmark = pytest.mark.gpu

OUT = ("kl", "kl_rev", "jsd", "counts", "logp_s", "logp_t", "am_s", "am_t", "ce")


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    L.load()


@pytest.mark.parametrize("case", list(CASES))
def test_jsd_full(case):
    say("jsd", case)
    wl = custom(case, **CASES[case])
    hip = run_hip(wl, outputs=OUT)
    assert hip["stats"]["kernel"] == "mfma" and hip["err"] == 0
    assert np.all(hip["jsd"] <= np.log(2.0) + 1e-6) and np.all(hip["jsd"] >= -1e-6)
    compare(hip, wl, label="jsd-" + case)


@pytest.mark.parametrize("region", [O.REGION_STUDENT, O.REGION_ALL])
def test_jsd_regions_and_scales(region):
    say("jsd region", region)
    wl = custom("multi_tile", **CASES["multi_tile"])
    wl["scale_student"], wl["scale_teacher"] = 2.0, 0.5
    hip = run_hip(wl, region=region, outputs=OUT)
    compare(hip, wl, region=region, label="jsd-scales-%d" % region)


def test_jsd_spans_and_region_only():
    say("jsd spans, region only")
    wl = custom("turns", **TURNS_CASE)
    full = run_hip(wl, region=L.OLIVE_REGION_SPANS, outputs=OUT)
    compare(full, wl, region=O.REGION_SPANS, label="jsd-spans")
    ro = run_hip(wl, region=L.OLIVE_REGION_SPANS, outputs=OUT, out_flags=L.OLIVE_OUT_REGION_ONLY)
    compare(ro, wl, region=O.REGION_SPANS, region_only=True, label="jsd-spans-region-only")


# Calls with one KL direction or none: the normalisers come from the 256 x 256 kernel
# (teacher block first, or the student's for the reverse KL alone).
ONE_DIR = {
    "forward": ("kl", "jsd", "counts", "logp_s", "logp_t", "am_s", "am_t", "ce"),
    "reverse": ("kl_rev", "jsd", "counts", "logp_s", "logp_t", "am_s", "am_t", "ce"),
    "jsd_alone": ("jsd", "counts", "logp_s", "am_s"),
}


@pytest.mark.parametrize("which", list(ONE_DIR))
@pytest.mark.parametrize("case", ["ragged_v1000", "multi_tile", "v257"])
def test_jsd_after_the_wide_kernel(case, which):
    say("jsd after the 256 x 256 kernel", case, which)
    wl = custom(case, **CASES[case])
    hip = run_hip(wl, outputs=ONE_DIR[which])
    assert hip["stats"]["tile"] == "256x256" and hip["err"] == 0
    assert np.all(hip["jsd"] <= np.log(2.0) + 1e-6) and np.all(hip["jsd"] >= -1e-6)
    compare(hip, wl, label="jsd-wide-%s-%s" % (case, which))


@pytest.mark.parametrize("which", list(ONE_DIR))
def test_jsd_of_identical_models_after_the_wide_kernel(which):
    # The 256 x 256 kernel forms the two log-normalisers in different fold orders, so
    # for identical models they may differ by a rounding step and the JSD is 0 up to
    # its square (exactly 0 after the 256 x 128 kernel, below).
    say("jsd, teacher == student, after the 256 x 256 kernel", which)
    wl = custom("multi_tile", **dict(CASES["multi_tile"], d_teacher=256))
    wl["w_teacher"], wl["h_teacher"] = wl["w_student"], wl["h_student"]
    wl["scale_teacher"] = wl["scale_student"]
    hip = run_hip(wl, region=O.REGION_ALL, outputs=ONE_DIR[which])
    assert hip["stats"]["tile"] == "256x256"
    assert np.max(np.abs(hip["jsd"])) <= 1e-6


def test_jsd_of_identical_models_is_exactly_zero():
    say("jsd, teacher == student")
    wl = custom("multi_tile", **CASES["multi_tile"])
    wl["h_teacher"] = wl["h_student"]
    wl["w_teacher"] = wl["w_student"]
    spec = wl["spec"]
    wl["spec"] = W.custom_spec(name="same", num_seqs=spec.num_seqs, ragged_len=spec.ragged_len,
                               vocab=spec.vocab, d_student=spec.d_student,
                               d_teacher=spec.d_student, logit_scale=spec.logit_scale)
    hip = run_hip(wl, region=O.REGION_ALL, outputs=OUT)
    assert np.all(hip["jsd"] == 0.0) and not np.any(np.signbit(hip["jsd"]))


def test_jsd_request_leaves_the_other_outputs_unchanged():
    say("jsd on / off")
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    a = run_hip(wl, outputs=OUT)
    b = run_hip(wl, outputs=tuple(k for k in OUT if k != "jsd"))
    for k in b:
        if k not in ("stats", "err"):
            np.testing.assert_array_equal(a[k], b[k], err_msg=k)


def test_jsd_on_long_rollout_sampled():
    say("jsd, long_rollout sampled")
    wl = W.make_workload("long_rollout", 0, device="cuda")
    hip = run_hip(wl, outputs=OUT)
    assert hip["stats"]["kernel"] == "mfma" and hip["err"] == 0
    compare(hip, wl, rows=stratified_rows(wl, n_random=64), label="jsd-long_rollout")
    del wl
    torch.cuda.empty_cache()


def test_jsd_needs_the_mfma_path_and_old_output_structs_still_work():
    say("jsd: generic path refused; the output struct without the jsd field")
    wl = custom("ragged_v1000", **CASES["ragged_v1000"])
    spec = wl["spec"]
    T, B = wl["total_positions"], spec.num_seqs
    dev = wl["h_student"].device
    batch = L.make_batch(wl["cu_seqlens"], wl["cut"], wl["targets"], wl["h_student"],
                         wl["h_teacher"], wl["valid_len"])
    jsd = torch.full((T,), 7.0, device=dev)
    kl = torch.full((T,), 7.0, device=dev)
    for simple, expect in ((True, L.OLIVE_E_UNSUPPORTED), (False, L.OLIVE_OK)):
        desc = L.make_desc(spec.vocab, spec.d_student, spec.d_teacher, L.OLIVE_BF16,
                           L.OLIVE_W_DV, 1.0, 1.0, max_positions=T, max_seqs=B,
                           flags=L.OLIVE_FLAG_SIMPLE_KERNEL if simple else 0)
        ctx = L.olive_score_init(desc, wl["w_student"], wl["w_teacher"])
        try:
            o = L.make_outputs(kl=kl, jsd=jsd)
            assert L.olive_score_batch(ctx, batch, o, check=False) == expect
            # the layout before the jsd field: accepted, and jsd is not touched
            jsd.fill_(7.0)
            o.size = L.olive_score_outputs.jsd.offset
            assert L.olive_score_batch(ctx, batch, o, check=False) == L.OLIVE_OK
            torch.cuda.synchronize()
            assert bool(torch.all(jsd == 7.0))
            o.size = L.olive_score_outputs.jsd.offset - 8
            assert L.olive_score_batch(ctx, batch, o, check=False) == L.OLIVE_E_RANGE
        finally:
            L.olive_score_free(ctx)
    assert ctypes.sizeof(L.olive_score_outputs) == L.olive_score_outputs.jsd.offset + 8
