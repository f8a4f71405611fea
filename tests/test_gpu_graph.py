"""HIP-graph capture of the scoring calls, through the C ABI.

The call path of every entry point only enqueues kernels on the caller's stream: it
allocates nothing, records no memset and never synchronises (its workspace is the
context's, or the library's fixed scratch array for the no-allocation entry point).
A caller can therefore capture a call into a graph once and replay it on new contents
of the same input buffers. Each test captures one call, then for several input sets
writes them into the captured buffers, makes an eager call on them into other output
buffers, synchronises, replays the graph into its own (poisoned) output buffers and
compares the two bit for bit: the kernels are the same and deterministic.
"""
import numpy as np
import pytest
import torch

from paper_2609_36246_amd import _lib as L
from paper_2609_36246_amd import workloads as W
from tests.gpu_harness import say, to_np
from tests.test_gpu_parity import TURNS_CASE

pytestmark = pytest.mark.gpu

# fixed lengths, so that every seed gives buffers of the same shapes (cuts, targets
# and hidden states differ)
SPEC = dict(num_seqs=3, seq_len=700, vocab=5000, d_student=256, d_teacher=128,
            logit_scale=4.0, target_source="student", cut_rule=("frac", 0.1, 0.9))
SEEDS = (0, 1, 2)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    L.load()


def draw(seed, name="graph", **spec):
    return W.make_workload(name, seed, device="cuda", spec=W.custom_spec(name=name, **spec))


INPUT_KEYS = ("h_student", "h_teacher", "targets", "cut", "cu_seqlens")


def write_inputs(dst, src):
    for k in INPUT_KEYS:
        assert dst[k].shape == src[k].shape, k
        dst[k].copy_(src[k])


def new_outputs(T, B, d_s=None, V=None, grads=False):
    dev = "cuda"
    nan = float("nan")
    if grads:
        return dict(h=torch.full((T, d_s), nan, device=dev),
                    w=torch.full((d_s * V,), nan, device=dev),
                    counts=torch.full((2,), -1, dtype=torch.int64, device=dev))
    return dict(kl=torch.full((T,), nan, device=dev), kl_rev=torch.full((T,), nan, device=dev),
                counts=torch.full((2,), -1, dtype=torch.int64, device=dev),
                logp_s=torch.full((T,), nan, device=dev), logp_t=torch.full((T,), nan, device=dev),
                am_s=torch.full((T,), -7, dtype=torch.int32, device=dev),
                am_t=torch.full((T,), -7, dtype=torch.int32, device=dev),
                ce=torch.full((B,), nan, device=dev))


def poison(out):
    for v in out.values():
        v.fill_(-7 if v.dtype in (torch.int32, torch.int64) else float("nan"))


def snapshot(out, keys):
    return {k: to_np(out[k]) for k in keys}


def capture(call, out):
    """Capture call(out) into a graph on a side stream of default priority (a warm-up
    call on that stream first)."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        call(out)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        call(out)
    torch.cuda.synchronize()
    return g


def replays_match_eager(wl, call, keys, grads=False, spec=SPEC, seeds=SEEDS, name="graph"):
    T, B = wl["total_positions"], wl["cu_seqlens"].shape[0] - 1
    mk = lambda: new_outputs(T, B, spec["d_student"], spec["vocab"], grads)
    out_g, out_e = mk(), mk()
    g = capture(call, out_g)
    for seed in seeds:
        write_inputs(wl, draw(seed, name, **spec))
        poison(out_e)
        call(out_e)                 # eager, on the current stream
        torch.cuda.synchronize()
        ref = snapshot(out_e, keys)
        poison(out_g)
        g.replay()
        torch.cuda.synchronize()
        got = snapshot(out_g, keys)
        for k in keys:
            np.testing.assert_array_equal(got[k], ref[k], err_msg="seed %d: %s" % (seed, k))
        assert not np.all(np.isnan(ref[keys[0]])), "the eager call wrote nothing"
        say("  seed %d: replay == eager on %s" % (seed, ", ".join(keys)))
    return g


def context(wl, flags=0, spec=SPEC):
    desc = L.make_desc(spec["vocab"], spec["d_student"], spec["d_teacher"], L.OLIVE_BF16,
                       L.OLIVE_W_DV, wl["scale_student"], wl["scale_teacher"],
                       max_positions=wl["total_positions"],
                       max_seqs=wl["cu_seqlens"].shape[0] - 1, flags=flags)
    return L.olive_score_init(desc, wl["w_student"], wl["w_teacher"])


def batch_of(wl, region=L.OLIVE_REGION_TEACHER):
    return L.make_batch(wl["cu_seqlens"], wl["cut"], wl["targets"], wl["h_student"],
                        wl["h_teacher"], wl["valid_len"], region)


BATCH_OUTPUTS = {
    # one KL direction: the 256 x 256 kernel; both: the 256 x 128 kernel
    "forward": ("kl",),
    "reverse_only": ("kl_rev",),
    "both_directions": ("kl", "kl_rev"),
}


def test_graph_of_kl_masked():
    say("graph: olive_kl_masked")
    wl = draw(SEEDS[0], **SPEC)
    ctx = context(wl)
    b = batch_of(wl)

    def call(o):
        L.olive_kl_masked(ctx, b, o["kl"], o["counts"], o["logp_s"], o["logp_t"], o["am_s"],
                          o["am_t"], o["ce"])
    try:
        replays_match_eager(wl, call, ("kl", "counts", "logp_s", "logp_t", "am_s", "am_t", "ce"))
        assert L.olive_score_last_stats(ctx)["tile"] == "256x256"
    finally:
        L.olive_score_free(ctx)


@pytest.mark.parametrize("which", list(BATCH_OUTPUTS))
def test_graph_of_score_batch(which):
    say("graph: olive_score_batch", which)
    wl = draw(SEEDS[0], **SPEC)
    ctx = context(wl)
    b = batch_of(wl)
    kls = BATCH_OUTPUTS[which]

    def call(o):
        outs = L.make_outputs(kl=o["kl"] if "kl" in kls else None,
                              kl_reverse=o["kl_rev"] if "kl_rev" in kls else None,
                              counts=o["counts"], logp_student=o["logp_s"],
                              logp_teacher=o["logp_t"], argmax_student=o["am_s"],
                              argmax_teacher=o["am_t"], ce_per_seq=o["ce"])
        L.olive_score_batch(ctx, b, outs)
    try:
        replays_match_eager(wl, call, kls + ("counts", "logp_s", "logp_t", "am_s", "am_t", "ce"))
        want = "256x128" if which == "both_directions" else "256x256"
        assert L.olive_score_last_stats(ctx)["tile"] == want
    finally:
        L.olive_score_free(ctx)


def test_graph_of_span_scoring():
    # the spans stay (their count is captured with the call); hidden states and targets
    # change between replays
    say("graph: olive_score_batch_spans")
    spec = dict(TURNS_CASE)
    wl = draw(0, "turns", **spec)
    ctx = context(wl, spec=spec)
    b = batch_of(wl, L.OLIVE_REGION_SPANS)
    b.cut = None
    sp = L.make_spans(wl["span_offsets"], wl["span_pairs"])

    def call(o):
        outs = L.make_outputs(kl=o["kl"], counts=o["counts"], logp_student=o["logp_s"],
                              argmax_student=o["am_s"], ce_per_seq=o["ce"])
        L.olive_score_batch_spans(ctx, b, sp, outs)
    try:
        T, B = wl["total_positions"], wl["cu_seqlens"].shape[0] - 1
        out_g, out_e = new_outputs(T, B), new_outputs(T, B)
        g = capture(call, out_g)
        keys = ("kl", "counts", "logp_s", "am_s", "ce")
        orig = {k: wl[k].clone() for k in ("h_student", "h_teacher", "targets")}
        for seed in SEEDS:
            # new contents of the same shapes: rows moved by a seed-dependent shift
            for k, v in orig.items():
                wl[k].copy_(torch.roll(v, shifts=37 * seed, dims=0))
            poison(out_e)
            call(out_e)
            torch.cuda.synchronize()
            ref = snapshot(out_e, keys)
            poison(out_g)
            g.replay()
            torch.cuda.synchronize()
            got = snapshot(out_g, keys)
            for k in keys:
                np.testing.assert_array_equal(got[k], ref[k], err_msg="seed %d: %s" % (seed, k))
        assert L.olive_score_last_stats(ctx)["tile"] == "256x256"
    finally:
        L.olive_score_free(ctx)


def test_graph_of_the_no_allocation_entry_point():
    say("graph: olive_kl_masked_static")
    wl = draw(SEEDS[0], **SPEC)
    ws, wt = wl["w_student"].t().contiguous(), wl["w_teacher"].t().contiguous()
    desc = L.make_desc(SPEC["vocab"], SPEC["d_student"], SPEC["d_teacher"], L.OLIVE_BF16,
                       L.OLIVE_W_VD, wl["scale_student"], wl["scale_teacher"],
                       max_positions=wl["total_positions"], max_seqs=SPEC["num_seqs"])
    b = batch_of(wl)

    def call(o):
        L.olive_kl_masked_static(desc, ws, wt, b, o["kl"], o["counts"], o["logp_s"],
                                 o["logp_t"], o["am_s"], o["am_t"], o["ce"])
    replays_match_eager(wl, call, ("kl", "counts", "logp_s", "logp_t", "am_s", "am_t", "ce"))


@pytest.mark.parametrize("w_kl", [0.0, 0.5], ids=["ce", "ce_kl"])
def test_graph_of_the_backward(w_kl):
    say("graph: olive_score_backward", w_kl)
    wl = draw(SEEDS[0], **SPEC)
    ctx = context(wl, flags=L.OLIVE_FLAG_BACKWARD)
    b = batch_of(wl)

    def call(o):
        g = L.make_grad_outputs(1.0, w_kl, o["h"], o["w"], o["counts"])
        L.olive_score_backward(ctx, b, g)
    try:
        replays_match_eager(wl, call, ("h", "w", "counts"), grads=True)
    finally:
        L.olive_score_free(ctx)
