"""The parity statistics of bench.py's JSON line, on the CPU: the oracle's own rounded outputs pass
with no mismatch, and single planted errors (a theta~ two bf16 ulps off on a strict element, a
changed dropped gradient, a kept gradient off by 1e-5 relative) are each counted."""
import argparse

import numpy as np
import torch

import bench
import oracle
import workloads


def _setup():
    cfg = workloads.config("mini")
    inp = workloads.make_inputs(cfg, device="cpu")
    step = 11
    params = workloads.step_params(cfg, inp.settings, step)
    _, wins = bench.sample_windows(cfg, cfg.numel // 3)
    g_pre = [inp.grad_theta[i].view(-1)[a:a + m].numpy().copy() for i, a, m in wins]
    tasks = bench.window_tasks(wins, inp, g_pre, torch, np, piece=4096)
    # the "GPU" outputs: the oracle's rounded theta~ and its accumulated gradient
    tt, gg = [], []
    for i, off, th, t0, gs, gp in tasks:
        tt.append(oracle.simulate(th, t0, cfg.theta0_dtype, cfg.out_dtype, params[i], cfg.smat_seed, step, i, off))
        gg.append(oracle.backward_accum(gs, cfg.grad_dtype, gp, params[i], cfg.lam, cfg.smat_seed, step, i, off))
    rec, outs = bench.cpu_baseline(cfg, tasks, params, step, budget_s=600.0)
    return cfg, tasks, outs, tt, gg, params, rec


def test_parity_of_the_oracle_with_itself_and_planted_errors():
    cfg, tasks, outs, tt, gg, params, rec = _setup()
    assert rec["kind"] == "oracle" and rec["cores"] >= 1 and rec["cores"] <= rec["affinity_cores"]
    assert len(outs) == len(tasks)
    st = bench.parity_stats(cfg, tasks, outs, tt, gg, params, np)
    assert st["elements"] == sum(t[2].size for t in tasks)
    assert st["theta_tilde"]["mismatches"] == 0 and st["theta_tilde"]["max_ulp"] == 0
    assert st["grad_theta"]["mismatches"] == 0 and st["grad_theta"]["dropped_changed"] == 0
    # plant one error of each kind in copies of the outputs
    k = max(range(len(tasks)), key=lambda j: tasks[j][2].size)
    _, y, kept, _, _ = next(r for r in outs if r[0] == k)
    tt2 = [x.copy() for x in tt]
    gg2 = [x.copy() for x in gg]
    e = int(np.flatnonzero(np.abs(y) > 1e-3)[0])          # far from zero: a strict element
    tt2[k][e] = np.uint16(int(tt2[k][e]) + 2)               # two bf16 ulps off
    dropped = np.flatnonzero(~kept)
    keptix = np.flatnonzero(kept)
    gg2[k][int(dropped[0])] = np.float32(gg2[k][int(dropped[0])]) * np.float32(1.5) + np.float32(1e-3)
    gg2[k][int(keptix[0])] = np.float32(gg2[k][int(keptix[0])] * (1 + 1e-5))
    st2 = bench.parity_stats(cfg, tasks, outs, tt2, gg2, params, np)
    assert st2["theta_tilde"]["mismatches"] == 1 and st2["theta_tilde"]["max_ulp"] == 2
    assert st2["grad_theta"]["dropped_changed"] == 1
    assert st2["grad_theta"]["mismatches"] >= 1 and st2["grad_theta"]["max_rel_err"] > 1e-6


def test_default_steps_scale_with_the_list():
    a = argparse.Namespace(steps=None, warmup=None)
    assert bench.default_steps(a, workloads.config("c4")) == (20, 5)
    k2, w2 = bench.default_steps(a, workloads.config("c2"))
    assert k2 * workloads.config("c2").numel >= 20 * workloads.config("c4").numel and w2 == k2 // 4
    assert bench.default_steps(a, workloads.config("c1"))[0] == 2000
    assert bench.default_steps(argparse.Namespace(steps=7, warmup=2), workloads.config("c2")) == (7, 2)
