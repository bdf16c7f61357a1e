"""Write tests/golden/forced_<config>.npz: the oracle's values for the
teacher-forced parity test of a large configuration.  Calls only oracle/ (and
workload/ for the seeded inputs); nothing here comes from the HIP path.

Subset: prompts 0 and 1 of the batch and their 2*m trajectories, the whole
prompt prefill, and the first S = 64 generated tokens of every trajectory,
teacher-forced with workload.gen.teacher_forcing_tokens (the forced
end-of-sequence lengths still apply).  Per (trajectory, generated index):
log-prob of the taken token, entropy, the oracle's own Gumbel-max sample and
its top-2 perturbed-score margin, the log-sum-exp, the row's largest logit
(value, index and magnitude) and the logits at 256 fixed vocabulary ids.  For
MoE models, per row and layer: the routed expert ids, their softmax
probabilities and the k / k+1 probability margin.

    python tests/golden/make_forced_golden.py qwen3-8b [--jobs 8]
    python tests/golden/make_forced_golden.py qwen3-30b-a3b
"""
import argparse
import multiprocessing as mp
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import model as M                               # noqa: E402
from oracle.forced import forced_forward, taken_tokens      # noqa: E402
from oracle.sampler import sample_row, top2_margin          # noqa: E402
from workload import get_config, rollout_inputs              # noqa: E402
from workload.gen import teacher_forcing_tokens              # noqa: E402

PROMPTS = (0, 1)
STEPS = 64
N_IDX = 256


def _score(args):
    logits, temperature, g, s, seed, force = args
    tok, lp, ent = sample_row(logits, temperature, g, s, seed, force)
    z = np.asarray(logits, dtype=np.float64) / float(temperature)
    mx = z.max()
    lse = mx + np.log(np.exp(z - mx).sum())
    return tok, lp, ent, top2_margin(logits.astype(np.float32), temperature, g, s, seed), lse


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("config")
    ap.add_argument("--jobs", type=int, default=os.cpu_count() or 1)
    ap.add_argument("--out", default=None)
    args = ap.parse_args()
    t0 = time.time()
    cfg, run = get_config(args.config)
    prompts, forced = rollout_inputs(cfg, run)
    m, eos = run.m, cfg.vocab - 1
    traj = np.array([p * m + j for p in PROMPTS for j in range(m)])
    traj_prompt = np.repeat(np.arange(len(PROMPTS)), m)
    tokens = teacher_forcing_tokens(cfg, run, STEPS)[traj]
    taken, n_gen = taken_tokens(forced[traj], tokens, run.cap, eos)
    consumed = taken[:, :STEPS - 1]
    sub_prompts = prompts[list(PROMPTS)]
    seed, d, dt = cfg.weight_seed, cfg.d_model, cfg.dtype
    routing = {}
    with mp.get_context("fork").Pool(args.jobs) as pool:
        def get_layer(l):
            t = time.time()
            lw = M.init_layer(cfg, l, pool=pool)
            print(f"layer {l}: weights {time.time() - t:.0f} s", flush=True)
            return lw
        emb = lambda tk: M.init_rows(seed, M.T_EMBED, 0, tk, d, 1, dt)
        last, dec = forced_forward(cfg, sub_prompts, traj_prompt, consumed, get_layer, emb, routing=routing)
        print(f"forward done {time.time() - t0:.0f} s", flush=True)
        head = M.init_tensor(seed, M.T_LM, 0, cfg.vocab, d, d, dt, pool=pool)
        T = len(traj)
        hid = np.concatenate([last[traj_prompt][:, None, :], dec], axis=1)      # [T, S, d]
        logits = (hid.reshape(T * STEPS, d) @ head.T).reshape(T, STEPS, cfg.vocab)
        del head
        print(f"logits done {time.time() - t0:.0f} s", flush=True)
        jobs = [(logits[t, s], run.temperature, int(traj[t]), s, run.sample_seed, int(taken[t, s]))
                for t in range(T) for s in range(STEPS)]
        res = pool.map(_score, jobs, chunksize=8)
    idx = np.sort(np.random.default_rng(2605).choice(cfg.vocab, N_IDX, replace=False))
    res = np.array(res, dtype=np.float64).reshape(T, STEPS, 5)
    out = dict(
        config=np.array(args.config), prompts=np.array(PROMPTS), traj=traj.astype(np.int32),
        steps=np.int32(STEPS), tokens=tokens.astype(np.int32), taken=taken.astype(np.int32),
        n_gen=n_gen.astype(np.int32), idx=idx.astype(np.int32),
        logits_at_idx=logits[:, :, idx].astype(np.float32),
        zmax=logits.max(axis=-1), zabs=np.abs(logits).max(axis=-1),
        argmax=logits.argmax(axis=-1).astype(np.int32),
        sampled=res[..., 0].astype(np.int32), logprob=res[..., 1], entropy=res[..., 2],
        margin=res[..., 3], lse=res[..., 4])
    if cfg.n_experts:
        out["route_ids"] = routing["ids"].astype(np.uint8)
        out["route_p"] = routing["p"].astype(np.float32)
        out["route_margin"] = routing["margin"].astype(np.float32)
    path = args.out or os.path.join(HERE, f"forced_{args.config}.npz")
    np.savez_compressed(path, **out)
    print(f"wrote {path} ({os.path.getsize(path) / 1e6:.1f} MB) in {time.time() - t0:.0f} s", flush=True)


if __name__ == "__main__":
    main()
