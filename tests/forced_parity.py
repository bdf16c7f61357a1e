"""Shared GPU runner and checks of the teacher-forced parity tests (not a test
module): the GPU decodes a whole batch through the C ABI while a subset of
trajectories takes a forced token table (and, for MoE models, the oracle's
experts); every generated token of the subset is compared with the oracle's
values (oracle.forced.reference_values)."""
import sys

import numpy as np
import torch

from oracle.sampler import sample_row

DEV = "cuda"
STRICT_STEPS = (0, 1, 2, 31, 32, 62, 63)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_forced(model, run, prompts, forced, g, label, strict_all=False):
    """The GPU side: the whole batch decodes through the C ABI while the
    trajectories of g["traj"] take g["taken"] (and, for MoE models, combine
    the oracle's experts, g["route_ids"]); returns per-(trajectory, step)
    GPU values, the rows kept for the strict sampler check and the router's
    own decisions.  Rows the GPU no longer decodes (trajectories aborted by
    the early stop) are left out; a subset trajectory the GPU still decodes
    after the oracle's window ended it is an error."""
    from paper_2605_30859_amd import binding as B
    B.load_library()
    P, m, Lp = run.n_prompts, run.m, run.prompt_len
    traj, taken, n_gen, S = g["traj"], g["taken"], g["n_gen"], int(g["steps"])
    sub_p = [int(p) for p in g["prompts"]]
    T, n_traj = len(traj), P * m
    n_pre = len(sub_p) * Lp
    say(f"{label}: GPU context (full batch {n_traj} trajectories, {P} x {Lp} prompt tokens)")
    ro = B.Rollout(model, run)
    pr = torch.from_numpy(np.ascontiguousarray(prompts.reshape(-1))).to(DEV)
    fl = torch.from_numpy(forced.astype(np.int32)).to(DEV)
    moe = model.is_moe
    route = None
    if moe:
        L, k = model.n_layers, model.top_k
        n_keys = max(P * Lp, n_traj)
        r_force = torch.full((n_keys, L, k), -1, dtype=torch.int32, device=DEV)
        r_own = torch.full((n_keys, L, k), -1, dtype=torch.int32, device=DEV)
        r_used = torch.zeros((n_keys, L, k), dtype=torch.float32, device=DEV)
        rid = torch.from_numpy(g["route_ids"].astype(np.int32)).to(DEV)
        ro.debug_moe_routing(r_force, r_own, r_used)
        # prefill keys are prompt positions: the subset prompts' oracle rows
        for i, p in enumerate(sub_p):
            r_force[p * Lp:(p + 1) * Lp] = rid[i * Lp:(i + 1) * Lp]
        route = {"own": np.full((n_pre + T * (S - 1), L, k), -1, dtype=np.int64),
                 "used": np.zeros((n_pre + T * (S - 1), L, k))}
    rec = {key: np.full((T, S), np.nan) for key in ("lp", "ent", "zmax", "lse", "dz_idx")}
    rec["sampled"] = np.full((T, S), -1, dtype=np.int64)
    rec["seen"] = np.zeros((T, S), dtype=bool)
    strict = []
    for s in range(S):
        want = np.nonzero(n_gen > s)[0]
        f = np.full(n_traj, -1, dtype=np.int32)
        f[traj[want]] = taken[want, s]
        ft = torch.from_numpy(f).to(DEV)
        if s == 0:
            rows = ro.darts_prefill(pr, fl, ft)
        else:
            if moe:
                r_force[:n_traj] = -1
                keys = torch.from_numpy(traj[want].astype(np.int64)).to(DEV)
                src = torch.from_numpy((n_pre + want * (S - 1) + s - 1).astype(np.int64)).to(DEV)
                r_force[keys] = rid[src]
            rows = ro.darts_decode_step(ft)
        h = {key: v.cpu().numpy() for key, v in rows.items()}
        n = len(h["traj"])
        pos = {int(x): r for r, x in enumerate(h["traj"])}
        late = [int(traj[t]) for t in range(T) if n_gen[t] <= s and int(traj[t]) in pos]
        assert not late, (label, s, "decoded after the oracle's termination", late)
        act = np.array([t for t in want if int(traj[t]) in pos], dtype=np.int64)
        if len(act) == 0:
            ro.darts_select_and_prune()
            if ro.n_done >= P:
                break
            continue
        rec["seen"][act, s] = True
        r_of = np.array([pos[int(traj[t])] for t in act], dtype=np.int64)
        lrow_i = np.array([sub_p[t // m] for t in act]) if s == 0 else r_of
        lg = ro.debug_logits(max(n, P))[torch.from_numpy(lrow_i).to(DEV)].cpu().numpy()
        z = lg.astype(np.float64)
        mx = z.max(axis=1)
        rec["zmax"][act, s] = mx
        rec["lse"][act, s] = mx + np.log(np.exp(z - mx[:, None]).sum(axis=1))
        rec["dz_idx"][act, s] = np.max(np.abs(z[:, g["idx"]] - g["logits_at_idx"][act, s]), axis=1)
        rec["lp"][act, s] = h["logprob"][r_of]
        rec["ent"][act, s] = h["entropy"][r_of]
        rec["sampled"][act, s] = h["sampled"][r_of]
        if strict_all or s in STRICT_STEPS:
            for j, t in enumerate(act):
                strict.append((t, s, int(h["sampled"][r_of[j]]), lg[j].copy(),
                               float(h["logprob"][r_of[j]]), float(h["entropy"][r_of[j]])))
        if moe:
            if s == 0:
                for i, p in enumerate(sub_p):
                    route["own"][i * Lp:(i + 1) * Lp] = r_own[p * Lp:(p + 1) * Lp].cpu().numpy()
                    route["used"][i * Lp:(i + 1) * Lp] = r_used[p * Lp:(p + 1) * Lp].cpu().numpy()
            else:
                keys = torch.from_numpy(traj[act].astype(np.int64)).to(DEV)
                dst = n_pre + act * (S - 1) + s - 1
                route["own"][dst] = r_own[keys].cpu().numpy()
                route["used"][dst] = r_used[keys].cpu().numpy()
        ro.darts_select_and_prune()
        if s % 16 == 0 or s == S - 1:
            say(f"{label}: step {s}, {n} rows")
        if ro.n_done >= P:       # every kept set complete: the rollout is over
            say(f"{label}: rollout complete after step {s}")
            break
    ro.close()
    return rec, strict, route


def check_forced(model, run, g, rec, strict, route, label):
    """Compare the GPU values with the oracle's (see the test modules).
    Returns the number of rows compared."""
    config = label
    valid = (np.arange(int(g["steps"]))[None, :] < g["n_gen"][:, None]) & rec["seen"]
    zabs = g["zabs"]
    tol = 2e-2 * zabs
    n_rows = int(valid.sum())
    dz = rec["dz_idx"][valid]
    dmax = np.abs(rec["zmax"] - g["zmax"])[valid]
    dlse = np.abs(rec["lse"] - g["lse"])[valid]
    dlp = np.abs(rec["lp"] - g["logprob"])[valid]
    dent = np.abs(rec["ent"] - g["entropy"])[valid]
    say(f"{config}: {n_rows} rows; logit dev at 256 ids: worst {np.max(dz / zabs[valid]):.2e} "
        f"of max|z| (max|z| {zabs[valid].min():.1f}-{zabs[valid].max():.1f}); row max worst "
        f"{np.max(dmax):.3e}; LSE worst {np.max(dlse):.3e}")
    say(f"{config}: |d logprob| worst {dlp.max():.3e} mean {dlp.mean():.3e}; |d entropy| worst "
        f"{dent.max():.3e} mean {dent.mean():.3e}")
    assert (dz <= tol[valid]).all()
    assert (dmax <= tol[valid]).all() and (dlse <= tol[valid]).all()
    # log-prob = z_taken - LSE and entropy = LSE - E_p[z]: each moves by at most
    # twice the largest logit deviation
    assert (dlp <= 2 * tol[valid]).all() and (dent <= 2 * tol[valid]).all()
    # the GPU's sample is the oracle sampler's choice on the GPU's own logits,
    # and its log-prob (of the token taken) and entropy are the oracle's values
    # on those logits within the 1e-3 of the specification
    dlp_own, dent_own = [], []
    for t, s, tok, lrow, lp_g, ent_g in strict:
        want, lp_o, ent_o = sample_row(lrow, run.temperature, int(g["traj"][t]), s, run.sample_seed,
                                       force=int(g["taken"][t, s]))
        assert tok == want, (config, t, s, tok, want)
        dlp_own.append(abs(lp_g - lp_o))
        dent_own.append(abs(ent_g - ent_o))
    if strict:
        say(f"{config}: on the GPU's own logits ({len(strict)} rows): |d logprob| worst "
            f"{max(dlp_own):.3e}, |d entropy| worst {max(dent_own):.3e}")
        assert max(dlp_own) <= 1e-3 and max(dent_own) <= 1e-3
    # and the oracle's own sample wherever the margin exceeds twice the tolerance
    clear = valid & (g["margin"] > 2 * tol)
    mism = clear & (rec["sampled"] != g["sampled"])
    excused = int((valid & ~clear & (rec["sampled"] != g["sampled"])).sum())
    say(f"{config}: sampled tokens: {len(strict)} bit-exact on the GPU's logits; "
        f"{int(clear.sum())} rows with a clear margin, {int(mism.sum())} differ; "
        f"{excused} near-tie rows differ (excused)")
    assert not mism.any()
    if model.is_moe:
        rows = np.concatenate([np.arange(len(g["prompts"]) * run.prompt_len),
                               len(g["prompts"]) * run.prompt_len +
                               (np.nonzero(valid[:, 1:])[0] * (int(g["steps"]) - 1) + np.nonzero(valid[:, 1:])[1])])
        ref_ids = g["route_ids"][rows].astype(np.int64)
        ref_p = g["route_p"][rows].astype(np.float64)
        dp = np.abs(route["used"][rows] - ref_p)
        delta = float(dp.max())
        say(f"{config}: router probabilities at the oracle's experts: worst |dp| {delta:.3e} "
            f"(relative {np.max(dp / ref_p):.3e}) over {len(rows)} rows x {model.n_layers} layers")
        # bf16 operands through 48 layers: the router's probabilities stay
        # within 5% of the oracle's
        assert np.max(dp / ref_p) < 5e-2
        own = np.sort(route["own"][rows], axis=-1)
        same = (own == np.sort(ref_ids, axis=-1)).all(axis=-1)
        clear_r = g["route_margin"][rows] > 2 * delta
        say(f"{config}: own top-{model.top_k}: {int(clear_r.sum())} (row, layer) decisions with a "
            f"margin above 2x the measured deviation, {int((clear_r & ~same).sum())} differ; "
            f"{int((~clear_r).sum())} near ties, {int((~clear_r & ~same).sum())} of them differ")
        assert (same | ~clear_r).all()
    return n_rows


