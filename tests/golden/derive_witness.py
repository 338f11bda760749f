"""Write the derived values of the -24 witness fixture from the oracle.

The fixture's "printed_by_paper" block holds the values the paper prints for
its four-key example (Section 3.4; appendix A, the exact -24 witness).  The
"derived_by_oracle" block holds values the paper does not print, computed here
only by `oracle/` from the printed inputs:
  exact_dq, exact_dv      the FP64 exact VJP (oracle.exact) at the witness row
  plain_dq_bf16           the BF16 model of Algorithm 1 (oracle.algo_model),
  gproj_dq_bf16           plain and GProj modes, at the witness row
  gproj_dq_before_cast    alpha (A - lambda B) before the final BF16 cast
  lambda                  rho / m at the witness row
Run:  python tests/golden/derive_witness.py   (rewrites the file in place).
"""
from __future__ import annotations

import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
PATH = os.path.join(HERE, "witness_minus24.json")


def embed(pb, d: int = 64):
    """The witness as row 3 of an N = 4 causal head, zero-padded to d."""
    N = 4
    q = np.zeros((N, d), np.float32)
    k = np.zeros((N, d), np.float32)
    v = np.zeros((N, d), np.float32)
    u = np.zeros((N, d), np.float32)
    k[:, :2] = pb["k"]
    v[:, :2] = pb["v"]
    u[3, :2] = pb["u"]
    return q, k, v, u


def derive(pb) -> dict:
    sys.path.insert(0, ROOT)
    import oracle
    from oracle import algo_model as M
    q, k, v, u = embed(pb)
    alpha = pb["alpha"]
    ex = oracle.exact(q[None].astype(np.float64), k[None].astype(np.float64),
                      v[None].astype(np.float64), u[None].astype(np.float64), True, alpha)
    out = {"exact_dq": [float(t) for t in ex["dQ"][0, 3, :2]],
           "exact_dv": [float(t) for t in ex["dV"][0, 0, :2]],
           "exact_dk_max_abs": float(np.abs(ex["dK"]).max())}
    for mode in ("plain", "gproj"):
        O, LSE, dQ, dK, dV, st = M.forward_backward(q, k, v, u, True, alpha, mode)
        out[f"{mode}_dq_bf16"] = [float(t) for t in dQ[3, :2]]
        if mode == "gproj":
            a = np.float32(alpha)
            lam = st["lam"][3]
            corr = (lam * st["B"][3, :2]).astype(np.float32)
            out["gproj_dq_before_cast"] = [float(t) for t in
                                           (a * (st["A"][3, :2] - corr).astype(np.float32))]
            out["lambda"] = float(lam)
            out["A"] = [float(t) for t in st["A"][3, :2]]
            out["B"] = [float(t) for t in st["B"][3, :2]]
    return out


def main():
    with open(PATH) as f:
        w = json.load(f)
    w.pop("derived_by_hand_from_printed_values", None)
    w["derived_by_oracle"] = {"note": "written by tests/golden/derive_witness.py from the printed "
                                      "inputs with oracle.exact and oracle.algo_model only",
                              **derive(w["printed_by_paper"])}
    with open(PATH, "w") as f:
        json.dump(w, f, indent=2)
        f.write("\n")
    print(json.dumps(w["derived_by_oracle"], indent=2))


if __name__ == "__main__":
    main()
