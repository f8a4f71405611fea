"""Writes worked_examples.json: small scoring cases whose answers are closed forms.

The paper prints no numeric example of the scoring, so each case here is chosen so
that its answer follows by hand from the definitions the scoring uses: the softmax
log-prob of a realised token (the summand of Eq. 1, Sec. 3.1), the full-vocabulary
KL(teacher || student) (the divergence distillation minimises, Sec. 6) and its
reverse KL(student || teacher) (on-policy distillation's objective, Sec. 1), the cut
mask of Eq. 1 (prompt and prefix excluded, continuation scored) and the greedy
(lowest-index) argmax. The expected values are evaluated from those closed forms
with the standard `math` module only; nothing here calls the oracle or the GPU
path. Run: python tests/golden/make_worked_examples.py
"""
import json
import math
import os

L2, L3 = math.log(2.0), math.log(3.0)

cases = []

# 1. Logits (0, ln 2, ln 3) from d = 1, h = 1: p = (1/6, 2/6, 3/6), lse = ln 6.
#    Teacher uses these logits, the student is uniform (all-zero logits):
#    KL = sum p log(3 p) = (1/6) ln(1/2) + (1/3) ln 1 + (1/2) ln(3/2).
cases.append(dict(
    name="three_token_softmax",
    d_student=1, d_teacher=1, vocab=3,
    h_student=[[1.0]], w_student=[[0.0, 0.0, 0.0]],
    h_teacher=[[1.0]], w_teacher=[[0.0, L2, L3]],
    targets=[2], cu_seqlens=[0, 1], cut=[0], valid_len=None,
    expect=dict(
        lse_t=[math.log(6.0)], lse_s=[math.log(3.0)],
        logp_t=[math.log(0.5)], logp_s=[-math.log(3.0)],
        kl=[(1.0 / 6.0) * math.log(0.5) + 0.5 * math.log(1.5)],
        kl_rev=[math.log(4.0 / 3.0) / 3.0],
        argmax_t=[2], argmax_s=[0], n_scored=1, t_valid=1,
        ce=[math.log(3.0)]),
    derivation="p_T = (1,2,3)/6; p_S = (1,1,1)/3; KL = sum p_T ln(p_T/p_S); "
               "reverse KL = sum p_S ln(p_S/p_T) = (1/3)(ln 2 + ln 1 + ln(2/3)); "
               "student argmax is the lowest of three tied zeros"))

# 2. A stitched sequence of length 7, cut 4, valid length 6 (one token past EOS):
#    teacher-region positions are local t = 4, 5; uniform logits over V = 4 give
#    logp = -ln 4 at every valid position, so Eq. 1's loss is 2 ln 4.
cases.append(dict(
    name="stitched_cut_and_eos",
    d_student=2, d_teacher=2, vocab=4,
    h_student=[[1.0, -1.0]] * 7, w_student=[[0.5] * 4, [0.25] * 4],
    h_teacher=[[1.0, -1.0]] * 7, w_teacher=[[0.5] * 4, [0.25] * 4],
    targets=[0, 1, 2, 3, 0, 1, 2], cu_seqlens=[0, 7], cut=[4], valid_len=[6],
    expect=dict(
        logp_s=[-math.log(4.0)] * 6 + [0.0], logp_t=[-math.log(4.0)] * 6 + [0.0],
        kl=[0.0] * 7, kl_rev=[0.0] * 7, argmax_s=[0] * 6 + [-1], argmax_t=[0] * 6 + [-1],
        n_scored=2, t_valid=6, ce=[2.0 * math.log(4.0)]),
    derivation="equal logits -> p = 1/4; scored t in {4,5}; t = 6 is past the valid length"))

# 3. V = 2: the log-prob of the realised token is -softplus(z_other - z_y) and the
#    KL between two Bernoulli laws has the textbook closed form.
zs = (0.75, -0.5)       # student logits from h = 1, W = [[0.75, -0.5]]
zt = (-1.25, 2.0)
def softplus(x):
    return math.log1p(math.exp(x))
ps1 = 1.0 / (1.0 + math.exp(zs[0] - zs[1]))
pt1 = 1.0 / (1.0 + math.exp(zt[0] - zt[1]))
kl_bern = pt1 * math.log(pt1 / ps1) + (1 - pt1) * math.log((1 - pt1) / (1 - ps1))
kl_bern_rev = ps1 * math.log(ps1 / pt1) + (1 - ps1) * math.log((1 - ps1) / (1 - pt1))
cases.append(dict(
    name="two_token_closed_form",
    d_student=1, d_teacher=1, vocab=2,
    h_student=[[1.0]], w_student=[list(zs)],
    h_teacher=[[1.0]], w_teacher=[list(zt)],
    targets=[0], cu_seqlens=[0, 1], cut=[0], valid_len=None,
    expect=dict(
        logp_s=[-softplus(zs[1] - zs[0])], logp_t=[-softplus(zt[1] - zt[0])],
        kl=[kl_bern], kl_rev=[kl_bern_rev], argmax_s=[0], argmax_t=[1], n_scored=1, t_valid=1,
        ce=[softplus(zs[1] - zs[0])]),
    derivation="Bernoulli: p(1) = sigmoid(z1 - z0); KL = p ln(p/q) + (1-p) ln((1-p)/(1-q)); "
               "the reverse exchanges p and q"))

# 4. Multi-turn (Sec. 3.2): prompt [0,3), student action/observation turns [3,5)/[5,7)
#    and [7,9)/[9,11), teacher turns [11,14)/[14,15) and [15,18)/[18,19); only the
#    teacher actions are scored. EOS after local t = 16 (valid length 17) drops the
#    last action's final token: 3 + 2 = 5 scored positions, each with logp = -ln 4
#    under uniform logits over V = 4, so Eq. 1's loss is 5 ln 4.
cases.append(dict(
    name="multi_turn_teacher_actions",
    d_student=1, d_teacher=1, vocab=4,
    h_student=[[1.0]] * 19, w_student=[[0.5] * 4],
    h_teacher=[[1.0]] * 19, w_teacher=[[0.5] * 4],
    targets=[t % 4 for t in range(19)], cu_seqlens=[0, 19], cut=[11], valid_len=[17],
    region="spans", spans=[[[11, 14], [15, 18]]],
    expect=dict(
        logp_s=[-math.log(4.0)] * 17 + [0.0, 0.0], kl=[0.0] * 19,
        argmax_s=[0] * 17 + [-1, -1], n_scored=5, t_valid=17, ce=[5.0 * math.log(4.0)]),
    derivation="scored = teacher action tokens inside the valid length: {11,12,13,15,16}"))

out = dict(
    source="closed forms of the scoring definitions (Sec. 3.1 Eq. 1; Sec. 3.2 multi-turn masks; "
           "Sec. 6 KL; Sec. 1 reverse KL); "
           "the paper prints no numeric worked example",
    cases=cases)
path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "worked_examples.json")
with open(path, "w") as f:
    json.dump(out, f, indent=1)
print("wrote", path)
