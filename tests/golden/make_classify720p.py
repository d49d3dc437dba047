"""Writes tests/golden/classify720p.json: the oracle's head labels and Eq. 3-4
statistics for every layer of the planted 720P classification workload
(30 layers x 12 heads, classification at the block where the 7-block window
first fills).  Calls only oracle/ and the seeded input generator.

    python tests/golden/make_classify720p.py [first_layer last_layer]

Layers already present in the file are kept, so the script can be resumed.
"""
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import headcast_oracle as O  # noqa: E402
from synth import inputs as S  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "classify720p.json")


def main():
    w = S.WORKLOADS["classify720p"]
    lo, hi = (int(sys.argv[1]), int(sys.argv[2])) if len(sys.argv) > 2 else (0, w.n_layers - 1)
    data = json.load(open(OUT)) if os.path.exists(OUT) else {
        "workload": "classify720p", "cur_block": w.window_blocks - 1, "layers": {}}
    cur = w.window_blocks - 1
    for layer in range(lo, hi + 1):
        if str(layer) in data["layers"]:
            continue
        t0 = time.time()
        q, k, v = S.gen_layer(w, layer, cur, classify_block=cur)
        labels, stats = O.classify_layer(q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                                         w.proxy_radius)
        data["layers"][str(layer)] = {"labels": [int(x) for x in labels],
                                      "stats": [[float(x) for x in row] for row in stats],
                                      "planted": [int(x) for x in S.head_types(w)[layer]]}
        json.dump(data, open(OUT + ".tmp", "w"), indent=0)
        os.replace(OUT + ".tmp", OUT)
        print(f"layer {layer}: {list(labels)} in {time.time() - t0:.0f}s", flush=True)


if __name__ == "__main__":
    main()
