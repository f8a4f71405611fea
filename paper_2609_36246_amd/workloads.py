"""Seeded synthetic workloads for the per-position scoring path.

This module only draws inputs. It holds none of the scoring arithmetic and is
shared, as plain input data, by the HIP path, the fp64 oracle, the tests and the
benchmark. It imports neither of them.

The five workloads mirror the stitched student-prefix / teacher-continuation
rollouts of the method (Sec. 3.1, Alg. 1, Eq. 1): every sequence is a student
prefix followed by a teacher continuation, split at a per-sequence cut point,
with a shared vocabulary. The paper's own data (RLVE problems, AgentGym
environments, Qwen3 weights) is not available, so random hidden states and
random projection weights of the stated shapes stand in for it; the trace
geometry follows the paper's configuration table (App. A: prefix 4096,
continuation 1024, batch 64) and a Qwen-family vocabulary of 151,936 tokens.

Recipe (all draws seeded; integer structure is drawn with NumPy on the host so it
is identical on every device; float tensors are drawn with a seeded torch
generator on the device that will hold them):
  * hidden states h ~ N(0, 1) as [T, d] row-major, rounded to bf16 (RNE) unless
    the workload is fp32;
  * projection weights W ~ N(0, 1/d) (variance 1/d) as [d, V] row-major;
  * cut points, valid lengths (EOS), outlier rows and ragged lengths as integers;
  * realised tokens either uniform, or sampled at temperature 1 (times the
    workload's logit scale) from the named model's softmax by the Gumbel-max
    rule: y = argmax_v (s * z_v + g_v), g = -log(-log u), u ~ U(0, 1), where
    z = h @ W is a library matmul in fp32 accumulation.  The sampled tokens are
    plain integer inputs to both sides; nothing downstream depends on how they
    were drawn.
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import Optional

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class WorkloadSpec:
    name: str
    num_seqs: int
    seq_len: Optional[int]          # fixed length, or None for ragged lengths
    ragged_len: Optional[tuple]     # (lo, hi) inclusive when ragged
    vocab: int
    d_student: int
    d_teacher: int
    dtype: str                      # "f32" or "bf16"
    logit_scale: float              # applied to both models (1/temperature)
    target_source: str              # "uniform" | "student" | "teacher"
    cut_rule: tuple                 # ("abs", lo, hi) or ("frac", lo, hi)
    eos: bool                       # draw a valid length past the cut
    outlier_frac: float             # fraction of rows scaled by outlier_mul
    outlier_mul: float
    # Multi-turn structure (Sec. 3.2), or None: (prompt_lo, prompt_hi, student_turns,
    # teacher_turns, action_lo, action_hi, obs_lo, obs_hi). Each turn is an action
    # followed by an environment observation; lengths are drawn per turn, the cut is
    # the first teacher turn and the scored spans are the teacher's actions.
    turns: Optional[tuple] = None


# The five workloads the scoring path is measured and checked on.
WORKLOADS = {
    "tiny": WorkloadSpec("tiny", 2, 32, None, 1000, 64, 96, "f32", 1.0,
                         "uniform", ("abs", 1, 31), False, 0.0, 1.0),
    "small": WorkloadSpec("small", 8, 512, None, 32000, 1024, 2048, "bf16", 1.0,
                          "student", ("abs", 16, 512 - 16), False, 0.0, 1.0),
    "large_vocab": WorkloadSpec("large_vocab", 4, 2048, None, 151936, 1536, 3584, "bf16",
                                1.0, "teacher", ("abs", 64, 2048 - 64), False, 0.01, 8.0),
    "long_rollout": WorkloadSpec("long_rollout", 8, 4096, None, 151936, 2048, 4096, "bf16",
                                 4.0, "student", ("abs", 256, 4096 - 256), True, 0.0, 1.0),
    "ragged": WorkloadSpec("ragged", 64, None, (128, 8192), 151936, 2048, 5120, "bf16", 1.0,
                           "teacher", ("frac", 0.1, 0.9), False, 0.0, 1.0),
    # Agentic rollouts (Sec. 3.2, Sec. 4.2): 10 student turns then 5 teacher turns;
    # only the teacher's action tokens are scored.
    "multi_turn": WorkloadSpec("multi_turn", 8, None, None, 151936, 2048, 5120, "bf16", 1.0,
                               "teacher", ("abs", 0, 0), False, 0.0, 1.0,
                               turns=(128, 512, 10, 5, 32, 192, 32, 384)),
}
WORKLOAD_ORDER = ["tiny", "small", "large_vocab", "long_rollout", "ragged", "multi_turn"]

# Fixed order of the per-tensor random streams spawned from the seed.
_STREAMS = ["h_student", "h_teacher", "w_student", "w_teacher", "lengths", "cuts",
            "eos", "outliers", "targets", "turns"]


def _streams(seed: int):
    kids = np.random.SeedSequence(seed).spawn(len(_STREAMS))
    return dict(zip(_STREAMS, kids))


def _torch_gen(seq: np.random.SeedSequence, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seq.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1)))
    return g


def draw_structure(spec: WorkloadSpec, seed: int = 0):
    """Integer structure of a workload: lengths, cuts, valid lengths, outlier rows.

    Returns host int32/int64 NumPy arrays, identical on every machine for a seed.
    """
    st = _streams(seed)
    B = spec.num_seqs
    if spec.turns is not None:
        return _draw_turns(spec, st)
    if spec.seq_len is not None:
        lengths = np.full(B, spec.seq_len, dtype=np.int64)
    else:
        lo, hi = spec.ragged_len
        lengths = np.random.default_rng(st["lengths"]).integers(lo, hi + 1, size=B)
    rng_cut = np.random.default_rng(st["cuts"])
    kind, lo, hi = spec.cut_rule
    if kind == "abs":
        cuts = rng_cut.integers(lo, hi + 1, size=B)
    else:
        lo_b = np.ceil(lo * lengths).astype(np.int64)
        hi_b = np.floor(hi * lengths).astype(np.int64)
        cuts = np.array([rng_cut.integers(a, b + 1) for a, b in zip(lo_b, hi_b)], dtype=np.int64)
    if spec.eos:
        rng_eos = np.random.default_rng(st["eos"])
        valid = np.array([rng_eos.integers(c + 1, n + 1) for c, n in zip(cuts, lengths)],
                         dtype=np.int64)
    else:
        valid = None
    cu = np.zeros(B + 1, dtype=np.int64)
    np.cumsum(lengths, out=cu[1:])
    T = int(cu[-1])
    n_out = int(round(spec.outlier_frac * T))
    if n_out > 0:
        outliers = np.sort(np.random.default_rng(st["outliers"]).choice(T, size=n_out,
                                                                          replace=False))
    else:
        outliers = np.zeros(0, dtype=np.int64)
    return dict(
        cu_seqlens=cu.astype(np.int32),
        cut=cuts.astype(np.int32),
        valid_len=None if valid is None else valid.astype(np.int32),
        outlier_rows=outliers.astype(np.int64),
        total_positions=T,
    )


def _draw_turns(spec: WorkloadSpec, st: dict) -> dict:
    """Multi-turn structure: prompt, student turns, teacher turns (action + observation
    each); cut = start of the first teacher turn; spans = the teacher's actions."""
    p_lo, p_hi, k, m, a_lo, a_hi, o_lo, o_hi = spec.turns
    rng = np.random.default_rng(st["turns"])
    B = spec.num_seqs
    lengths = np.zeros(B, dtype=np.int64)
    cuts = np.zeros(B, dtype=np.int64)
    spans = []
    for b in range(B):
        t = int(rng.integers(p_lo, p_hi + 1))
        seq_spans = []
        for turn in range(k + m):
            if turn == k:
                cuts[b] = t
            a = int(rng.integers(a_lo, a_hi + 1))
            o = int(rng.integers(o_lo, o_hi + 1))
            if turn >= k:
                seq_spans.append((t, t + a))
            t += a + o
        lengths[b] = t
        spans.append(seq_spans)
    cu = np.zeros(B + 1, dtype=np.int64)
    np.cumsum(lengths, out=cu[1:])
    off = np.zeros(B + 1, dtype=np.int64)
    np.cumsum([len(x) for x in spans], out=off[1:])
    flat = np.array([list(x) for sp in spans for x in sp], dtype=np.int32).reshape(-1, 2)
    return dict(
        cu_seqlens=cu.astype(np.int32),
        cut=cuts.astype(np.int32),
        valid_len=None,
        outlier_rows=np.zeros(0, dtype=np.int64),
        total_positions=int(cu[-1]),
        spans=spans,
        span_offsets=off.astype(np.int32),
        span_pairs=flat,
    )


def _randn(shape, gen, device, std=1.0, chunk_rows=8192):
    """N(0, std^2) fp32 draws, produced in row chunks to bound temporary memory."""
    out = torch.empty(shape, dtype=torch.float32, device=device)
    rows = shape[0]
    for r0 in range(0, rows, chunk_rows):
        r1 = min(rows, r0 + chunk_rows)
        out[r0:r1] = torch.randn((r1 - r0,) + tuple(shape[1:]), generator=gen, device=device)
    if std != 1.0:
        out.mul_(std)
    return out


def _to_dtype(x: torch.Tensor, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        return x.to(torch.bfloat16)  # round-to-nearest-even
    return x


def sample_targets_gumbel(h: torch.Tensor, w: torch.Tensor, scale: float,
                          gen: torch.Generator, chunk_rows: int = 1024) -> torch.Tensor:
    """Realised tokens drawn from softmax(scale * h @ w) by the Gumbel-max rule.

    h: [T, d], w: [d, V] (same device). The logits are a library matmul with fp32
    accumulation, used only to draw integer inputs.
    """
    T = h.shape[0]
    V = w.shape[1]
    out = torch.empty(T, dtype=torch.int32, device=h.device)
    wf = w if w.is_cuda else w.float()
    for r0 in range(0, T, chunk_rows):
        r1 = min(T, r0 + chunk_rows)
        hc = h[r0:r1]
        if h.is_cuda:
            z = torch.matmul(hc, wf).float()
        else:
            z = torch.matmul(hc.float(), wf)
        u = torch.rand((r1 - r0, V), generator=gen, device=h.device, dtype=torch.float32)
        u.clamp_(min=torch.finfo(torch.float32).tiny)
        g = -torch.log(-torch.log(u))
        out[r0:r1] = torch.argmax(z * scale + g, dim=1).to(torch.int32)
        del z, u, g
    return out


def make_workload(name: str, seed: int = 0, device="cpu", spec: Optional[WorkloadSpec] = None,
                  with_targets: bool = True) -> dict:
    """Draw one full workload.

    Returns a dict of torch tensors on `device` (hidden states [T,d], weights [d,V],
    targets [T] int32, cu_seqlens [B+1] int32, cut [B] int32, valid_len [B] int32 or
    None) plus the spec and the integer structure.
    """
    spec = spec or WORKLOADS[name]
    st = _streams(seed)
    s = draw_structure(spec, seed)
    T = s["total_positions"]
    dev = torch.device(device)
    g_hs = _torch_gen(st["h_student"], dev)
    g_ht = _torch_gen(st["h_teacher"], dev)
    g_ws = _torch_gen(st["w_student"], dev)
    g_wt = _torch_gen(st["w_teacher"], dev)

    h_s = _randn((T, spec.d_student), g_hs, dev)
    h_t = _randn((T, spec.d_teacher), g_ht, dev)
    if len(s["outlier_rows"]):
        idx = torch.from_numpy(s["outlier_rows"]).to(dev)
        h_s[idx] *= spec.outlier_mul
        h_t[idx] *= spec.outlier_mul
    h_s = _to_dtype(h_s, spec.dtype)
    h_t = _to_dtype(h_t, spec.dtype)
    w_s = _to_dtype(_randn((spec.d_student, spec.vocab), g_ws, dev,
                           std=1.0 / math.sqrt(spec.d_student), chunk_rows=256), spec.dtype)
    w_t = _to_dtype(_randn((spec.d_teacher, spec.vocab), g_wt, dev,
                           std=1.0 / math.sqrt(spec.d_teacher), chunk_rows=256), spec.dtype)

    targets = None
    if with_targets:
        g_y = _torch_gen(st["targets"], dev)
        if spec.target_source == "uniform":
            targets = torch.randint(0, spec.vocab, (T,), generator=g_y, device=dev,
                                    dtype=torch.int64).to(torch.int32)
        elif spec.target_source == "student":
            targets = sample_targets_gumbel(h_s, w_s, spec.logit_scale, g_y)
        else:
            targets = sample_targets_gumbel(h_t, w_t, spec.logit_scale, g_y)

    def t32(a):
        return None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    return dict(
        spec=spec,
        seed=seed,
        h_student=h_s.contiguous(),
        h_teacher=h_t.contiguous(),
        w_student=w_s.contiguous(),
        w_teacher=w_t.contiguous(),
        targets=targets,
        cu_seqlens=t32(s["cu_seqlens"]),
        cut=t32(s["cut"]),
        valid_len=t32(s["valid_len"]),
        outlier_rows=s["outlier_rows"],
        total_positions=T,
        scale_student=spec.logit_scale,
        scale_teacher=spec.logit_scale,
        structure=s,
        spans=s.get("spans"),
        span_offsets=t32(s.get("span_offsets")),
        span_pairs=t32(s.get("span_pairs")),
    )


def custom_spec(num_seqs=2, seq_len=32, vocab=1000, d_student=64, d_teacher=96, dtype="bf16",
                logit_scale=1.0, target_source="uniform", cut_rule=("abs", 1, 31), eos=False,
                ragged_len=None, outlier_frac=0.0, outlier_mul=1.0, name="custom", turns=None):
    """A workload spec of arbitrary size, for tests (same recipe as the named ones)."""
    return WorkloadSpec(name, num_seqs, None if (ragged_len or turns) else seq_len, ragged_len,
                        vocab, d_student, d_teacher, dtype, logit_scale, target_source, cut_rule,
                        eos, outlier_frac, outlier_mul, turns)


def tensor_digest(t: torch.Tensor) -> str:
    """Short content hash of a tensor (for logs and result caches)."""
    a = t.detach().cpu().contiguous()
    if a.dtype == torch.bfloat16:
        a = a.view(torch.int16)
    return hashlib.sha256(a.numpy().tobytes()).hexdigest()[:16]
