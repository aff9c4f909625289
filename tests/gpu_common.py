"""Shared fixtures of the GPU tests (test infrastructure)."""
import numpy as np
import torch

from paper_2609_16206_amd import rt_router as R


def run_sim(points, trace_np, device="cuda", check_status=True):
    """Run the HIP simulation over a numpy trace; returns numpy outputs,
    goodput, met and the data-flag word."""
    sim = R.Simulator(points)
    try:
        tr = R.to_device(trace_np, device)
        out = sim.run(tr)
        g, met = sim.goodput(tr, out)
        flags = sim.data_status()
        res = {k: v.cpu().numpy() for k, v in out.items()}
        g, met = g.cpu().numpy(), met.cpu().numpy()
    finally:
        sim.close()
    return res, g, met, flags


def log(msg):
    print(msg, flush=True)
