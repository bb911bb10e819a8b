"""Write fulldepth_spread.json: how far the oracle's float32-BLAS mode lies from its float64 mode
at the full depth of the 7B (32 layers), 13B (40 layers) and 7B batch-4 workloads.

Both runs use the bf16 storage roundings of a bf16 model and the same prompt chunking; they differ
only in float32 vs float64 accumulation.  At these depths a storage rounding that flips in one
layer changes every later layer's inputs, so the two modes' logits drift apart by far more than
float32 rounding itself; the parity tests of the whole models bound the GPU's distance from the
float32 oracle by this spread.  Records, per workload, the largest and the mean |logit difference|
of the first block (draft step 1 after the prompt) over all its rows and sequences.

Calls only the oracle and the seeded input generator.  Needs about 160 GB of host memory (the 13B
weights in float32 and float64); run it on a machine that has it:
    python tests/golden/make_fulldepth_spread.py
"""
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import decode as D  # noqa: E402
from oracle import model as M  # noqa: E402
from paper_2403_18647_amd import synth  # noqa: E402

PREFILL_CHUNK = 256
OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "fulldepth_spread.json")


def first_block_logits(sh, W, prompt, k, adaptive, b, mode, temperature, top_p, top_k, seed):
    tr = D.Trace()
    D.generate_sdsat(sh, W, prompt, k, 1, adaptive, mode=mode, temperature=temperature, top_p=top_p,
                     top_k=top_k, seed=seed, b=b, bf16=True, trace=tr, prefill_chunk=PREFILL_CHUNK,
                     on_prefill_chunk=lambda n: print(f"    prefill rows {n}", flush=True))
    return tr.blocks[0]["logits"].astype(np.float64)


def main():
    res = {"what": "oracle float32-BLAS vs float64 mode, first block, bf16 storage roundings",
           "prefill_chunk": PREFILL_CHUNK, "numpy": np.__version__, "machine": platform.machine(),
           "workloads": {}}
    for name in ("7b", "13b", "7b_bs4_nucleus"):
        wl = synth.workload(name)
        sh = wl.shape
        t0 = time.time()
        host = {}
        for n in synth.tensor_names(sh):
            t = synth.tensor(wl, n)
            host[n] = synth.bf16_bits_to_f32(t) if t.dtype == np.uint16 else t
        print(f"{name}: weights {time.time() - t0:.0f}s", flush=True)
        prompts = synth.prompts(wl)
        ad = synth.adaptive_ids(sh, wl.k)
        kw = dict(mode=wl.mode, temperature=wl.temperature if wl.mode == "nucleus" else 0.0, top_p=wl.top_p,
                  top_k=wl.top_k, seed=wl.seed)
        logits = {}
        for dt in (np.float32, np.float64):
            W = M.Weights(sh, host, dtype=dt)
            logits[dt] = []
            for b in range(wl.batch):
                t0 = time.time()
                logits[dt].append(first_block_logits(sh, W, prompts[b], wl.k, ad, b, **kw))
                print(f"{name}: {np.dtype(dt).name} sequence {b} {time.time() - t0:.0f}s", flush=True)
            del W
        d = np.abs(np.stack(logits[np.float32]) - np.stack(logits[np.float64]))
        res["workloads"][name] = {"layers": sh.n_layers, "batch": wl.batch, "rows": wl.k + 1,
                                  "max_abs": float(d.max()), "mean_abs": float(d.mean()),
                                  "frac_above_3e-2": float(np.mean(d > 3e-2))}
        print(name, res["workloads"][name], flush=True)
        del host, logits
    with open(OUT, "w") as f:
        json.dump(res, f, indent=1)
        f.write("\n")
    print(f"wrote {OUT}")


if __name__ == "__main__":
    main()
