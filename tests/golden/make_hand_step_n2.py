"""Writes hand_step_n2.json: one NLR iteration worked out by hand (no oracle code).

n=2, d=1, K=r=1.  Every value below is a closed form from the derivation in
the JSON's "source" field (Section 3, eqs. gradient / dualnormalized /
projected-primal-step / movement-estimate, Algorithm 1), evaluated with plain
float arithmetic.  Run:  python tests/golden/make_hand_step_n2.py
"""
import json
import math
import os

s122 = math.sqrt(1.22)
U1 = [1.1 / s122, 0.1 / s122]
q1 = [1.32 / 1.22 - 1.0, 0.12 / 1.22 - 1.0]
g = {
    "source": (
        "Worked by hand for n=2, d=1, K=r=1. X=[[-1],[3]] -> xbar=1, X_c=[[-2],[2]], "
        "a=||X_c||_2=2*sqrt(2), Xhat=[[-1/sqrt2],[1/sqrt2]] (Section 3). U0=[[1],[0]] is in Omega. "
        "y=0, beta=4, alpha=0.1. p=U^T1=1, q=Up-1=[0,-1], Theta=Xhat^T U=-1/sqrt2, "
        "Xhat Theta=[1/2,-1/2], ybar=y/sqrt(n)+(beta/n)q=[0,-2] (eq. dualnormalized), s=U^T ybar=0, "
        "grad=-2 Xhat Theta+ybar p^T+1 s^T=[-1,-1] (eq. gradient), W=(U-alpha grad)_+=[1.1,0.1], "
        "a=||W||^2=1.22, b=||U||^2=1, h=<W,U>=1.1, c=sqrt(K/a), U1=cW (eq. projected-primal-step), "
        "delta^2=c^2 a+b-2ch=2-2.2/sqrt(1.22) (eq. movement-identity), p1=1.2/sqrt(1.22), "
        "q1=U1 p1-1=[1.32/1.22-1, 0.12/1.22-1], f(U0)=-Theta^2+beta/2*||q/sqrt2||^2=1/2 "
        "(eq. normalized), gated dual step y1=(beta/sqrt2) q1 (Algorithm 1); the stored dual "
        "ytilde=y/sqrt(n) takes (beta/n) q1 = 2 q1 (Section 3, storage convention)."),
    "X": [[-1.0], [3.0]], "U0": [[1.0], [0.0]], "K": 1, "alpha": 0.1, "beta": 4.0,
    "a_norm": 2.0 * math.sqrt(2.0),
    "Xhat": [[-1 / math.sqrt(2)], [1 / math.sqrt(2)]],
    "grad": [[-1.0], [-1.0]],
    "W": [[1.1], [0.1]],
    "stats": {"a": 1.22, "b": 1.0, "h": 1.1, "c": 1.0 / s122},
    "U1": [[U1[0]], [U1[1]]],
    "delta": math.sqrt((U1[0] - 1.0) ** 2 + U1[1] ** 2),
    "delta_sq_identity": 2.0 - 2.2 / s122,
    "q1": q1,
    "rho1": math.sqrt(q1[0] ** 2 + q1[1] ** 2) / math.sqrt(2.0),
    "objective0": 0.5,
    "y1_if_gated": [4.0 / math.sqrt(2.0) * q1[0], 4.0 / math.sqrt(2.0) * q1[1]],
    "ytilde1_if_gated": [2.0 * q1[0], 2.0 * q1[1]],
}
with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "hand_step_n2.json"), "w") as f:
    json.dump(g, f, indent=1)
