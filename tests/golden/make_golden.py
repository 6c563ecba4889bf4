"""Write tiny_l2k_oracle.json from the oracle (run: python tests/golden/make_golden.py)."""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

from oracle import cosa_oracle as O  # noqa: E402
from paper_2607_25291_amd.inputs import WORKLOADS, make_inputs  # noqa: E402


def compute():
    w = WORKLOADS["tiny_l2k"]
    q, k, v = make_inputs(w)
    sc, hr = O.kap_score(q, k, n_kv_heads=1, block=w.block, stride=w.stride)
    order, count = O.kap_select(sc, hr, mode=O.SELECT_FRACTION, value=w.kap_budget)
    base = O.osk_attention(q, k, v, order, count, block=w.block)
    margins = base["margin"][~np.isnan(base["margin"])]
    total = O.causal_blocks(w.seq_len, w.block)
    delta, n_skip = O.calibrate_delta(margins, listed=int(count.sum()), total_causal=total,
                                      target_budget=w.osk_budget, seq_len=w.seq_len)
    r = O.osk_attention(q, k, v, order, count, block=w.block, skip_mode=O.SKIP_ROWMAX, delta=delta)
    nb = w.n_blocks
    return {
        "workload": w.name,
        "count": count[0, 0].tolist(),
        "order": [order[0, 0, i, :count[0, 0, i]].tolist() for i in range(nb)],
        "hrm": [np.nonzero(hr[0, 0, i, :i + 1])[0].tolist() for i in range(nb)],
        "score": [[float(x) for x in sc[0, 0, i, :i + 1]] for i in range(nb)],
        "margin": [[float(x) for x in base["margin"][0, 0, i, :count[0, 0, i]]] for i in range(nb)],
        "delta": delta,
        "visit": [r["visit"][0, 0, i, :count[0, 0, i]].tolist() for i in range(nb)],
        "o_row_sums": [float(x) for x in r["o"][0, 0].sum(axis=1)[::64]],
    }


if __name__ == "__main__":
    with open(os.path.join(HERE, "tiny_l2k_oracle.json"), "w") as f:
        json.dump(compute(), f)
