"""Staleness profiles of the PS policies (Fig. 1 left of arXiv 1410.8043), measured on the GPU.

The paper plots, for matrix factorization with a 1% minibatch per clock, the share of
parameter reads per clock differential (parameter age - local clock): BSP is always -1,
SSP spreads reads nearly uniformly over the window, ESSP concentrates them at -2
(staleness 1 regardless of s).  This script runs the library on seeded synthetic ratings
with the laws of a configured workload, scaled down, for each policy and staleness, and
prints the normalized profiles (PS_MF_IDX_STALENESS) as a markdown table.

    python -m paper_1410_8043_amd.staleness_profile [--config full] [--scale 0.1] [--B 100]
        [--clocks 300] [--s 1 3 7] [--policies lazy ssp_row essp_row essp vap] [--value-bound 0.01]
        [--seq]

--seq runs the sequential step (each worker applies its ratings one by one to its own rows);
the profile counts the view versions the workers start from.  vap is the value-bounded
policy with v_t = v0 / sqrt(t).
"""
from __future__ import annotations

import argparse

import numpy as np

POLICY_IDS = {"lazy": 0, "worst": 1, "essp": 2, "ssp_row": 3, "essp_row": 4, "vap": 5}


def profile(spec, w, policy: int, s: int, B: int, clocks: int, value_bound=None, seq=False) -> np.ndarray:
    import torch

    from paper_1410_8043_amd import ps_mf

    with ps_mf.PsMf(spec.N, spec.M, spec.K, spec.P, s, spec.eta, spec.lam, policy=policy, B=B, mb_seed=spec.seed,
                    stream=torch.cuda.current_stream(), value_bound=value_bound if policy == 5 else None,
                    step=ps_mf.STEP_SEQ if seq else ps_mf.STEP_ROWMEAN) as g:
        g.load_ratings(w.user, w.item, w.val)
        g.set_factors(w.L0, w.R0)
        g.clock(clocks)
        return g.export_index(ps_mf.IDX_STALENESS)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", default="full")
    ap.add_argument("--scale", type=float, default=0.1)
    ap.add_argument("--B", type=int, default=100, help="minibatch blocks (100: 1%% of the ratings per clock)")
    ap.add_argument("--clocks", type=int, default=300)
    ap.add_argument("--s", type=int, nargs="+", default=[1, 3, 7])
    ap.add_argument("--policies", nargs="+", default=["lazy", "ssp_row", "essp_row", "essp"])
    ap.add_argument("--value-bound", type=float, default=0.01, help="v0 of the vap policy")
    ap.add_argument("--seq", action="store_true", help="the sequential step instead of one fixed view")
    args = ap.parse_args(argv)
    import torch

    from paper_1410_8043_amd import synth

    torch.cuda.set_device(0)
    spec = synth.scaled(synth.CONFIGS[args.config], args.scale)
    w = synth.generate(spec)
    smax = max(args.s)
    print(f"{args.config} at {args.scale:g}: {spec.N} users x {spec.M} items, {w.nnz} ratings, K={spec.K}, "
          f"P={spec.P}, B={args.B}, {args.clocks} clocks" + (", sequential step" if args.seq else "") +
          "; share of reads per clock differential")
    print()
    print("| policy | s | " + " | ".join(str(-(d + 1)) for d in range(smax + 1)) + " | mean |")
    print("|---|---|" + "---|" * (smax + 2))
    for s in args.s:
        for name in args.policies:
            h = profile(spec, w, POLICY_IDS[name], s, args.B, args.clocks, args.value_bound, args.seq)
            h = h.astype(np.float64)
            share = h / max(1.0, h.sum())
            mean = -float(np.dot(np.arange(1, s + 2), share))
            cells = [f"{share[d]:.3f}" if d <= s else "" for d in range(smax + 1)]
            label = f"vap (v0={args.value_bound:g})" if name == "vap" else name
            print(f"| {label} | {s} | " + " | ".join(cells) + f" | {mean:.2f} |", flush=True)


if __name__ == "__main__":
    main()
