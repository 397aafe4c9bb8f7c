"""Writes the hand-derived fixtures in this folder (no library, no oracle).

attend_hand.json -- Algorithm 2 / Equations 8-9 on grids small enough to do by
hand: each key gets the score ln(w), so the softmax weights are the integers w
and the expected output is sum(w * v) / sum(w).

propagation_hand.json -- one and two propagation sweeps of Algorithm 1 on a
1x6 grid, worked by hand (reasoning in the file's "how_derived").
"""
import json
import math
import os

HERE = os.path.dirname(os.path.abspath(__file__))
ln = math.log


def attend_cases():
    k3 = [[ln(2)], [0.0], [ln(3)]]
    v3 = [[6.0], [12.0], [18.0]]
    k9 = [[ln(j + 1)] for j in range(9)]
    v9 = [[j + 1.0, 1.0] for j in range(9)]
    one = dict(Hq=1, Wq=1, q=[1.0])
    return [
        dict(one, note="1x3 key grid, d=1, scores ln2, 0, ln3 -> weights 2:1:3; window 3 around the middle key "
                       "covers all three: (2*6+1*12+3*18)/6 = 13",
             Hk=1, Wk=3, k=k3, v=v3, J=[1], window=3, scale=1.0, expected=[[13.0]]),
        dict(one, note="same grid, b = 0 (window 1): the output is the value of the match itself "
                       "(the kappa = 1, b = 0 special case)",
             Hk=1, Wk=3, k=k3, v=v3, J=[2], window=1, scale=1.0, expected=[[18.0]]),
        dict(one, note="same grid, window 3 around the first key: only keys 0 and 1 are in the grid, "
                       "weights 2:1 -> (12+12)/3 = 8",
             Hk=1, Wk=3, k=k3, v=v3, J=[0], window=3, scale=1.0, expected=[[8.0]]),
        dict(one, note="3x3 key grid, key j (row-major) has score ln(j+1), value (j+1, 1). Window 3 at the centre "
                       "covers all nine: sum (j+1)^2 / 45 = 285/45; the constant second channel stays 1",
             Hk=3, Wk=3, k=k9, v=v9, J=[4], window=3, scale=1.0, expected=[[285.0 / 45.0, 1.0]]),
        dict(one, note="same 3x3 grid, window 3 at the corner (0,0): keys 0,1,3,4 with weights 1,2,4,5 -> "
                       "(1+4+16+25)/12 = 23/6",
             Hk=3, Wk=3, k=k9, v=v9, J=[0], window=3, scale=1.0, expected=[[23.0 / 6.0, 1.0]]),
        dict(one, note="scale enters the exponent: key scores 2 ln(j+1) with scale 1/2 give the same weights as "
                       "above; window 5 at the corner covers the whole 3x3 grid",
             Hk=3, Wk=3, k=[[2.0 * ln(j + 1)] for j in range(9)], v=v9, J=[0], window=5, scale=0.5,
             expected=[[285.0 / 45.0, 1.0]]),
    ]


def main():
    attend = {
        "citation": "Algorithm 2 (window expansion around the match, sparse softmax, glimpse output) and "
                    "Equations 8-9; keys outside the key grid are dropped from the window",
        "how_derived": "by hand: each key is given a score ln(w) so the softmax weights are the integers w; "
                       "expected = sum(w*v)/sum(w)",
        "tolerance": 1e-12,
        "cases": attend_cases(),
    }
    with open(os.path.join(HERE, "attend_hand.json"), "w") as f:
        json.dump(attend, f, indent=1)

    th = [0.5 * j for j in range(6)]
    pm = {
        "citation": "Algorithm 1, propagation step, read as: the neighbour at p + o offers its match shifted back "
                    "by o (Section 4.1, assumption (1)); candidates outside the key grid are skipped; reads come "
                    "from the previous iteration's field",
        "how_derived": "by hand. 1x6 grid, key j = (cos 0.5j, sin 0.5j), Q = K, so q_p.k_j = cos(0.5|p-j|) is "
                       "largest at j = p and falls with |p-j|. Random search off. With J0 = [3,5,2,0,1,4]: query 0 "
                       "takes 2-2=0 from offset +2; query 1 takes 2-1=1 from offset +1; query 2 keeps 2; query 3 "
                       "takes 2+1=3 from offset -1; query 4 takes 2+2=4 from offset -2; query 5 is offered "
                       "1+1=2, 0+2=2 (and 5+4=9 is off-grid) and keeps its own 4. Iteration 2: query 5 takes "
                       "4+1=5 from offset -1.",
        "flags": "no_random_search",
        "Hq": 1, "Wq": 6, "Hk": 1, "Wk": 6, "d": 2,
        "k": [[math.cos(a), math.sin(a)] for a in th],
        "J0": [3, 5, 2, 0, 1, 4],
        "expected": {"1": [0, 1, 2, 3, 4, 4], "2": [0, 1, 2, 3, 4, 5]},
    }
    with open(os.path.join(HERE, "propagation_hand.json"), "w") as f:
        json.dump(pm, f, indent=1)


if __name__ == "__main__":
    main()
