"""GPU parity over seeded random shapes: vocabulary sizes, hidden widths (multiples of the
MFMA step or not), ragged lengths, cut points, EOS, logit scales (equal or not), regions
and output sets (one KL direction, the other, or both), each call through the C ABI
against the fp64 oracle on every row at the acceptance bar. The draws are fixed by the
test's seed, so a failure names a reproducible case.
"""
import numpy as np
import pytest
import torch

from oracle import olive_oracle as O
from paper_2609_36246_amd import _lib as L
from paper_2609_36246_amd import workloads as W
from tests.gpu_harness import compare, run_hip, say

pytestmark = pytest.mark.gpu

N_CASES = 40
OUTSETS = {
    "forward": ("kl", "counts", "logp_s", "logp_t", "am_s", "am_t", "ce"),
    "reverse": ("kl_rev", "counts", "logp_s", "logp_t", "am_s", "am_t", "ce"),
    "both": ("kl", "kl_rev", "counts", "logp_s", "logp_t", "am_s", "am_t", "ce"),
}
REGIONS = (O.REGION_TEACHER, O.REGION_STUDENT, O.REGION_ALL)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    L.load()


def draw_case(i):
    rng = np.random.default_rng(1000 + i)
    width = lambda: int(64 * rng.integers(1, 9)) if rng.random() < 0.85 \
        else int(32 * rng.integers(1, 16) + 32)
    lo = int(rng.integers(8, 300))
    hi = lo + int(rng.integers(1, 600))
    case = dict(num_seqs=int(rng.integers(1, 5)), ragged_len=(lo, hi),
                vocab=int(rng.integers(200, 4097)), d_student=width(), d_teacher=width(),
                logit_scale=float(rng.choice([1.0, 2.5, 4.0])),
                target_source=str(rng.choice(["uniform", "student", "teacher"])),
                cut_rule=("frac", float(rng.uniform(0.0, 0.5)), float(rng.uniform(0.5, 1.0))),
                eos=bool(rng.random() < 0.5))
    scales = None
    if rng.random() < 0.3:
        scales = (float(rng.choice([0.5, 1.0, 2.0])), float(rng.choice([0.75, 1.5, 3.0])))
    region = int(rng.choice(REGIONS))
    outs = str(rng.choice(list(OUTSETS)))
    return case, scales, region, outs


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_shape_parity(i):
    case, scales, region, outs = draw_case(i)
    say("random case", i, case, "scales", scales, "region", region, "outputs", outs)
    wl = W.make_workload("rand%d" % i, i, device="cuda",
                         spec=W.custom_spec(name="rand%d" % i, **case))
    if scales is not None:
        wl["scale_student"], wl["scale_teacher"] = scales
    hip = run_hip(wl, region=region, outputs=OUTSETS[outs])
    st = hip["stats"]
    mfma_ok = case["d_student"] % 64 == 0 and case["d_teacher"] % 64 == 0 and case["vocab"] >= 256
    assert st["kernel"] == ("mfma" if mfma_ok else "generic"), st
    if mfma_ok:
        assert st["tile"] == ("256x128" if outs == "both" else "256x256"), st
    assert hip["err"] == 0
    compare(hip, wl, region=region, label="rand%d-%s" % (i, outs))
