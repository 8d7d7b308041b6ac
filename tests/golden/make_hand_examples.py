"""Writes hand_examples.json: closed-form single- and two-step SwiLA cases.

Every expected value below is a closed-form evaluation, by hand, of the
recurrence, E-step and retrieval of Sec. 3.2 (eq. recurrence, eq.
responsibility, eq. retrieval) with beta and the priors from logits as App. B.2
states.  Nothing here runs the oracle or the GPU library; the paper itself
prints no numeric worked example.  Run: python tests/golden/make_hand_examples.py
"""
import json
import math
import os


def main():
    r1 = 1 / (1 + math.exp(0.5))
    case1 = dict(
        name="one_step_two_components", J=2, Dk=1, Dv=1,
        W0=[[[0.0]], [[1.0]]], k=[[1.0]], q=[[1.0]], v=[[1.0]],
        beta_logit=[[[40.0], [40.0]]], prior_k_logit=[[[0.0], [0.0]]],
        prior_q_logit=[[[0.0], [0.0]]],
        derivation=("sigmoid(40) rounds to 1 in fp64; delta=(1-0,1-1)=(1,0); pi^k=(1/2,1/2); "
                    "r_1=e^{-1/2}/(e^{-1/2}+1)=1/(1+e^{1/2}), r_2=1-r_1; "
                    "w_1=0+1*r_1*1*1=r_1, w_2=1+r_2*0=1; o=(w_1+w_2)/2 with the updated state"),
        expect=dict(resp=[[[r1], [1 - r1]]], state=[[[r1]], [[1.0]]], o=[[(r1 + 1) / 2]]))

    # two steps, Dk=2, Dv=1; beta=1/2, pi^k=(3/4,1/4), pi^q=(1/4,3/4)
    e = math.exp(0.39)             # e^{(1.45^2 - 1.15^2)/2}
    d1, d2 = -1.45, -1.15
    R1, R2 = 3 / (3 + e), e / (3 + e)
    c1, c2 = 0.5 * R1 * d1, 0.5 * R2 * d2
    w1 = [0.75 + c1 * 0.6, c1 * 0.8]
    w2 = [0.25 + c2 * 0.6, c2 * 0.8]
    o2 = 0.25 * (w1[0] - w1[1]) + 0.75 * (w2[0] - w2[1])
    case2 = dict(
        name="two_steps_unequal_priors", J=2, Dk=2, Dv=1, W0=None,
        k=[[1.0, 0.0], [0.6, 0.8]], q=[[1.0, 1.0], [1.0, -1.0]], v=[[2.0], [-1.0]],
        beta_logit=[[[0.0], [0.0]], [[0.0], [0.0]]],
        prior_k_logit=[[[math.log(3.0)], [0.0]], [[math.log(3.0)], [0.0]]],
        prior_q_logit=[[[0.0], [math.log(3.0)]], [[0.0], [math.log(3.0)]]],
        derivation=("beta=1/2, pi^k=(3/4,1/4), pi^q=(1/4,3/4). Step 1: zero state so delta=(2,2), "
                    "r=pi^k, c=beta*r*delta=(3/4,1/4), w_1=(3/4,0), w_2=(1/4,0), "
                    "o_1=1/4*3/4+3/4*1/4=3/8. Step 2: k=(0.6,0.8): pred=(0.45,0.15), "
                    "delta=(-1.45,-1.15), r_1=3e^{-1.45^2/2}/(3e^{-1.45^2/2}+e^{-1.15^2/2})"
                    "=3/(3+e^{0.39}), r_2=1-r_1; c_j=beta*r_j*delta_j; w_j+=c_j*k; "
                    "o_2=sum_j pi^q_j w_j.q with q=(1,-1)"),
        expect=dict(resp=[[[0.75], [0.25]], [[R1], [R2]]],
                    state=[[[w1[0]], [w1[1]]], [[w2[0]], [w2[1]]]], o=[[0.375], [o2]]))
    doc = {
        "citation": ("Sec. 3.2 (eq. recurrence, eq. responsibility, eq. retrieval) and App. B.2 "
                     "(beta = sigmoid of a logit, priors = softmax over components of logits). "
                     "The paper prints no numeric worked example; each case is a closed-form "
                     "evaluation of those equations derived by hand, written out in 'derivation'."),
        "layout": ("k,q: [T][Dk]; v: [T][Dv]; logits: [T][J][Dv]; W0/state: [J][Dk][Dv] "
                   "(element j,i,d is weight i of component j for output dim d); "
                   "resp: [T][J][Dv]; o: [T][Dv]"),
        "cases": [case1, case2],
    }
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "hand_examples.json")
    with open(path, "w") as f:
        json.dump(doc, f, indent=1)


if __name__ == "__main__":
    main()
