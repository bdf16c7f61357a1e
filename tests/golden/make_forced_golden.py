"""Write tests/golden/forced_<config>.npz: the oracle's values for the
teacher-forced parity test of a large configuration.  Calls only oracle/ (and
workload/ for the seeded inputs); nothing here comes from the HIP path.

Subset: prompts 0 and 1 of the batch and their 2*m trajectories, the whole
prompt prefill, and the first S = 64 generated tokens of every trajectory
(20 for the reduced full-width MoE shape of the parity tests),
teacher-forced with workload.gen.teacher_forcing_tokens (the forced
end-of-sequence lengths still apply).  Per (trajectory, generated index):
log-prob of the taken token, entropy, the oracle's own Gumbel-max sample and
its top-2 perturbed-score margin, the log-sum-exp, the row's largest logit
(value, index and magnitude) and the logits at 256 fixed vocabulary ids.  For
MoE models, per row and layer: the routed expert ids, their softmax
probabilities and the k / k+1 probability margin.

    python tests/golden/make_forced_golden.py qwen3-8b [--jobs 8]
    python tests/golden/make_forced_golden.py qwen3-30b-a3b
    python tests/golden/make_forced_golden.py moe-full-width
"""
import argparse
import multiprocessing as mp
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle.forced import reference_values                   # noqa: E402
from workload import get_config, rollout_inputs              # noqa: E402
from workload.gen import teacher_forcing_tokens              # noqa: E402

PROMPTS = (0, 1)
STEPS = {"moe-full-width": 20}      # generated tokens per trajectory (default 64)
N_IDX = {"moe-full-width": 512}     # fixed vocabulary ids stored per row (default 256)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("config")
    ap.add_argument("--jobs", type=int, default=os.cpu_count() or 1)
    ap.add_argument("--out", default=None)
    args = ap.parse_args()
    t0 = time.time()
    cfg, run = get_config(args.config)
    prompts, forced = rollout_inputs(cfg, run)
    steps = STEPS.get(args.config, 64)
    tokens = teacher_forcing_tokens(cfg, run, steps)
    log = lambda msg: print(f"{time.time() - t0:6.0f} s  {msg}", flush=True)
    with mp.get_context("fork").Pool(args.jobs) as pool:
        out = reference_values(cfg, run, prompts, forced, tokens, PROMPTS, steps, pool=pool,
                               n_idx=N_IDX.get(args.config, 256), log=log)
    out["config"] = np.array(args.config)
    path = args.out or os.path.join(HERE, f"forced_{args.config}.npz")
    np.savez_compressed(path, **out)
    log(f"wrote {path} ({os.path.getsize(path) / 1e6:.1f} MB)")


if __name__ == "__main__":
    main()
