"""Write tests/golden/c1_step.json from the oracle (test infrastructure only).

Calls only the oracle and the seeded input generator; nothing here touches the
HIP library.  Run from the repository root: python tests/golden/make_golden.py
"""
import hashlib
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import qcfuse as Q  # noqa: E402
from paper_2606_05875_amd.workloads import make_workload  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c1_step.json")
SAMPLE = [0, 75, 151, 152, 183]  # positions in R: first, middle and last context row, first and last query row


def input_digest(w):
    h = hashlib.sha256()
    for f in ("k_pic", "v_pic", "q_new", "k_new", "v_new"):
        h.update(np.ascontiguousarray(getattr(w, f), np.float32).tobytes())
    for a in w.anchor_local:
        h.update(np.ascontiguousarray(a, np.int64).tobytes())
    return h.hexdigest()


def golden():
    w = make_workload("c1")
    res = Q.fusion_step(w)
    R = np.asarray(res["R"][0], np.int64)
    rows = [int(R[i]) for i in SAMPLE]
    return {
        "workload": "c1 (seed 0): 4 x 128 chunks + 32 query tokens, 8/2/64 heads, float32, rho 30%",
        "input_sha256": input_digest(w),
        "P": [int(x) for x in res["P"][0]],
        "R": [int(x) for x in R],
        "scores": [float(x) for x in np.asarray(res["scores"], np.float64)[: int(w.ctx_len[0])]],
        "sample_rows": rows,
        "o_sample": [np.asarray(res["o"][r], np.float64).ravel().tolist() for r in rows],
    }


if __name__ == "__main__":
    g = golden()
    with open(OUT, "w") as f:
        json.dump(g, f)
    print(f"wrote {OUT}: |P| = {len(g['P'])}, |R| = {len(g['R'])}")
