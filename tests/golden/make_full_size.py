"""Writes <workload>_seed0.npz: the oracle's per-token log-sum-exp and loss for the full-size
workloads (Llama-3-8B, Qwen2.5-7B and Mistral-Large output-layer shapes), and for the Llama-3-8B
shape with the final RMSNorm in front (llama3_8b_rmsnorm: pre-norm rows and a gain from
workloads.make_rmsnorm_inputs).

Only `workloads` (the seeded inputs) and `oracle` (float64 CPU) are used. The GPU tests read these
files to check the HIP path at full size: the loss directly, and sampled rows of dH and dW, which
the oracle recomputes row by row from the stored lse.

    python tests/golden/make_full_size.py [workload ...]
"""
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
import workloads  # noqa: E402
from oracle import rmsnorm_lce  # noqa: E402

FULL = ("llama3_8b", "qwen25_7b", "mistral_large", "llama3_8b_rmsnorm")


def main(names):
    for name in names:
        t = time.time()
        if name.endswith("_rmsnorm"):
            d = workloads.make_rmsnorm_inputs(name[:-len("_rmsnorm")], seed=0)
            x, _ = rmsnorm_lce.rms_normalise(d["hidden"], d["gamma"], d["eps"])
        else:
            d = workloads.make_inputs(name, seed=0)
            x = d["hidden"]
        fp = workloads.fingerprint(d)
        r = oracle.forward(x, d["weight"], d["labels"], d["ignore_index"], d["reduction"], rows_per_block=512)
        np.savez_compressed(os.path.join(HERE, f"{name}_seed0.npz"), lse=r["lse"], token_loss=r["token_loss"])
        meta = {"workload": name, "seed": 0, "fingerprint": fp, "loss": r["loss"], "n_valid": r["n_valid"],
                "reduction": d["reduction"], "N": d["N"], "H": d["H"], "V": d["V"], "eps": d.get("eps"),
                "written_by": "tests/golden/make_full_size.py (oracle.forward, float64)"}
        with open(os.path.join(HERE, f"{name}_seed0.json"), "w") as f:
            json.dump(meta, f, indent=1)
        print(name, f"{time.time() - t:.1f}s", meta["loss"], flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or FULL)
