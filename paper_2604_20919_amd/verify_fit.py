"""The edge server's verify latency on this GPU, fitted to the affine model
of eq. 6, and the DiP-SD schedule it implies.

The paper profiles its verifier on an A100 and fits
G^v(b, F) = c^v b F^v(L, I) + beta^v (eq. 4, 6; Table II: c^v = 1.2077e-11,
beta^v = 95.1 ms).  Here the pass is timed through the library
(sd_verify_batch + sd_accept, host wall time from first enqueue to the
accept's return) on a grid of batch size b, draft length L and prefix I of
the Qwen3-32B shape, the same least-squares fit is taken, and Algorithm 1
(paper_2604_20919_amd.scheduler) runs with the fitted (c^v, beta^v) and the
paper's device-side parameters.

Usage:  python -m paper_2604_20919_amd.verify_fit [--model qwen3-32b] [--out file.json]

Inputs are synthetic: random-init weights, drafts uniform over the
vocabulary, q a softmax of Gaussian logits; the cached keys and values are
the zero-filled pool (the pass reads the same bytes whatever they hold).
"""
from __future__ import annotations

import argparse
import json
import sys
import time

import numpy as np


def measure(model: str = "qwen3-32b", bs=(1, 2, 4, 8, 16), Ls=(1, 4, 8), Is=(512, 2048),
            steps: int = 10, warmup: int = 3, seed: int = 11):
    """Median ms per verify pass (enqueue to sd_accept return) per (b, L, I)."""
    import torch
    import workload as wl
    from workload.device import DeviceWeights
    from . import sdverify as sv
    from .verifier import Verifier

    assert torch.cuda.is_available(), "the fit needs a GPU"
    sv.lib()
    m = wl.MODELS[model]
    dw = DeviceWeights(m, seed)
    names = {"wq": wl.W_Q, "wk": wl.W_K, "wv": wl.W_V, "wo": wl.W_O, "wg": wl.W_G, "wu": wl.W_U,
             "wd": wl.W_D, "norm1": wl.N_1, "norm2": wl.N_2, "qnorm": wl.N_Q, "knorm": wl.N_K}
    ptrs = {"embed": dw.ptr(wl.EMBED), "lm_head": dw.ptr(wl.LM_HEAD), "norm_f": dw.ptr(wl.NORM_F),
            "layers": [{f: dw.ptr(k, l) for f, k in names.items()} for l in range(m.n_layers)]}
    B, Lmax, Imax = max(bs), max(Ls), max(Is)
    pages = B * ((Imax + Lmax + 1 + 15) // 16) + 16
    v = Verifier(m, ptrs, n_pages=pages, max_users=B, max_draft=Lmax, max_batch_users=B,
                 max_batch_tokens=B * (Lmax + 1), max_ctx=Imax + Lmax + 1, max_pending=1)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    samples = []
    for I in Is:
        for b in bs:
            for L in Ls:
                for u in range(B):
                    v.reset_user(u, I, 0)
                assign = [0 if u < b else -1 for u in range(B)]
                dl = [L if u < b else 0 for u in range(B)]
                d = torch.randint(0, m.vocab, (b * L,), generator=g, device="cuda", dtype=torch.int32)
                q = torch.softmax(torch.randn((b * L, m.vocab), generator=g, device="cuda"), dim=1)
                ts = []
                for k in range(warmup + steps):
                    torch.cuda.synchronize()
                    t0 = time.perf_counter()
                    v.verify(0, assign, dl, d, q, "stochastic", seed=seed, round_=k)
                    v.accept(0, B)
                    ts.append((time.perf_counter() - t0) * 1e3)
                ms = float(np.median(ts[warmup:]))
                samples.append((b, L, I, ms))
                print(f"[fit] b={b:2d} L={L} I={I}: {ms:.3f} ms", file=sys.stderr, flush=True)
    v.close()
    return samples


def main():
    from . import scheduler as sch
    ap = argparse.ArgumentParser()
    ap.add_argument("--model", default="qwen3-32b")
    ap.add_argument("--out", default=None)
    args = ap.parse_args()
    samples = measure(args.model)
    verify = sch.ModelDims(64, 5120, 25600)
    c, beta = sch.fit_verify_latency(samples, verify)
    xs = np.array([b * sch.cost_verify(verify, L, I) for b, L, I, _ in samples])
    ys = np.array([t for *_, t in samples])
    pred = c * xs + beta
    r2 = 1.0 - float(np.sum((ys - pred) ** 2) / np.sum((ys - ys.mean()) ** 2))
    out = {"model": args.model, "samples": [list(s) for s in samples],
           "fit": {"c_v": c, "beta_v_ms": beta, "r2": r2,
                   "max_abs_err_ms": float(np.max(np.abs(ys - pred)))},
           "paper_fit_a100": {"c_v": 1.2077e-11, "beta_v_ms": 95.1074},
           "schedules": []}
    for M, alpha in ((6, 0.78), (6, 0.95), (14, 0.78)):
        row = {"M": M, "alpha": alpha}
        for label, (cv, bv) in (("a100_paper", (1.2077e-11, 95.1074)), ("this_gpu", (c, beta))):
            p = sch.paper_defaults(M, alpha)
            p.c_v, p.beta_v = cv, bv
            t0 = time.perf_counter()
            s = sch.solve(p)
            row[label] = {"R_tok_s": round(s.R, 2), "N": s.N, "assign": s.assign, "l": s.l,
                          "S_ms": round(s.S, 3), "solve_s": round(time.perf_counter() - t0, 3)}
        out["schedules"].append(row)
    text = json.dumps(out)
    if args.out:
        open(args.out, "w").write(text + "\n")
    print(text, flush=True)


if __name__ == "__main__":
    main()
