"""Calibrate the cross-Gram route model on the GPU it runs on.

The route between the factorized form (Eq. 4) and dense gradients for a
layer's cross-Gram contribution (Sec. 3.2 "FLOP-aware routing"; App. A.4) is
chosen from exact operation counts and eight effective rates
(``dattri_crossgram_cost_model``).  This script:

1. times, for a sweep of layer shapes (transformer-sized and narrow layers,
   T from 16 to 2048, 8 x 1, 16 x 16 and 8 x 8 example batches), the forced
   factorized route, both forms of the forced materialized route (DW staged
   in the workspace, and the one-pass kernel; each form is forced by making
   the other one's rate negligible in the context's model), and the gradient
   build alone (``dattri_materialize_gradient`` over both batches).  Each
   measurement captures LAYERS layers of the shape, as a model's layer stack
   would, so that the factorized route runs as one grouped launch; times are
   reported per layer;
2. fits the eight rates by minimising the squared log error of the predicted
   times (the same formula as the library's model: whole 128 x 128 tiles of
   the padded token Gram for the factorized kernel; gradient build (rounds of
   512 workgroups of tile builds), products and four launches for the staged
   form; rounds of 512 workgroups of tile builds for the one-pass form);
3. prints one JSON object with the fitted model and, per shape, the measured
   and predicted times, the route AUTO picks and its regret.

Usage:  python -m paper_2609_38767_amd.calibrate_crossgram [--quick] [--out FILE]
        python -m paper_2609_38767_amd.calibrate_crossgram --refit FILE  (fit saved measurements)
"""
import argparse
import json
import math
import sys

import torch

from . import (DATTRI_ROUTE_FACTORED, DATTRI_ROUTE_MATERIALIZED, dattri_cross_gram_costs,
               dattri_get_crossgram_cost_model, dattri_materialize_gradient, dattri_set_crossgram_cost_model,
               load)
from .session import ProjectionSession, cross_gram

# (d_in, d_out, T, n_a, n_b)
SWEEP = [(di, dq, T, 8, 1) for (di, dq) in ((1024, 1024), (1024, 4096), (4096, 1024), (1024, 3072))
         for T in (16, 64, 256, 1024, 2048)]
SWEEP += [(1024, 1024, T, 16, 16) for T in (32, 128, 512)]
SWEEP += [(128, 128, T, 8, 8) for T in (64, 512, 2048)]
SWEEP += [(1024, 4096, 512, 8, 1), (1024, 4096, 128, 8, 1)]
QUICK = [SWEEP[i] for i in (0, 2, 4, 5, 7, 9, 15, 20, 23)]

FIELDS = ["ghost_tflops", "ghost_gbs", "ghost_layer_us", "build_tflops", "build_gbs", "dot_gbs",
          "launch_us", "onepass_tflops"]
TILE = 128
SLOTS = 512  # resident one-pass workgroups
MAX_RUN = 4  # examples of batch a per one-pass workgroup, at most
LAYERS = 24


def _time_ms(fn, stream, warmup=2, reps=5):
    for _ in range(warmup):
        fn()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(reps)]
    for a, b in evs:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return sorted(a.elapsed_time(b) for a, b in evs)[reps // 2]


def _session(d_in, d_out, n, T, device, seed):
    sess = ProjectionSession([dict(d_in=d_in, d_out=d_out, k_in=1, k_out=1)] * LAYERS, dtype="bf16",
                             seed=0, device=device)
    g = torch.Generator(device=device).manual_seed(seed)
    for li in range(LAYERS):
        A = torch.randn((n, T, d_in), generator=g, device=device).to(torch.bfloat16)
        B = torch.randn((n, T, d_out), generator=g, device=device).to(torch.bfloat16)
        sess.capture(li, A, B)
    return sess


def measure(shape, device):
    d_in, d_out, T, na, nb = shape
    sa = _session(d_in, d_out, na, T, device, 1)
    sb = _session(d_in, d_out, nb, T, device, 2)
    stream = torch.cuda.current_stream()
    K = torch.empty((na, nb), dtype=torch.float32, device=device)
    t_f = _time_ms(lambda: cross_gram(sa, sb, DATTRI_ROUTE_FACTORED, K=K), stream) / LAYERS
    model = dattri_get_crossgram_cost_model(sa.ctx)
    dattri_set_crossgram_cost_model(sa.ctx, dict(model, onepass_tflops=1e-9))  # staged form only
    t_m = _time_ms(lambda: cross_gram(sa, sb, DATTRI_ROUTE_MATERIALIZED, K=K), stream) / LAYERS
    dattri_set_crossgram_cost_model(sa.ctx, dict(model, dot_gbs=1e-9))  # one-pass form only
    t_o = _time_ms(lambda: cross_gram(sa, sb, DATTRI_ROUTE_MATERIALIZED, K=K), stream) / LAYERS
    dattri_set_crossgram_cost_model(sa.ctx, model)
    G = torch.empty((max(na, nb), d_out, d_in), dtype=torch.float32, device=device)

    def build():
        for li in range(LAYERS):
            dattri_materialize_gradient(sa.ctx, li, 0, na, G)
            dattri_materialize_gradient(sb.ctx, li, 0, nb, G)
    t_b = _time_ms(build, stream) / LAYERS
    sa.close()
    sb.close()
    return {"shape": {"d_in": d_in, "d_out": d_out, "T": T, "n_a": na, "n_b": nb},
            "factored_ms": t_f, "materialized_ms": t_m, "onepass_ms": t_o, "build_ms": t_b,
            "counts": dattri_cross_gram_costs(na, nb, T, T, d_in, d_out, 2)}


def _r16(T):
    return (T + 15) // 16 * 16


def _r32(T):
    return (T + 31) // 32 * 32


def onepass_us(model, tiles, na, nb, T):
    """Predicted one-pass time (without launches): the run length (at most
    MAX_RUN examples) with the fewest rounds of SLOTS workgroups times the
    workgroup's tile builds."""
    per = 2.0 * TILE * TILE * _r32(T) / (model["onepass_tflops"] * 1e6 / SLOTS)
    best = math.inf
    for nz in range(-(-na // MAX_RUN), na + 1):
        ipw = -(-na // nz)
        if -(-na // ipw) != nz:
            continue
        best = min(best, -(-(tiles * nb * nz) // SLOTS) * (ipw * per + per))
    return best


def predict_us(model, s):
    """(factorized, staged materialized, build, one-pass materialized)
    microseconds; mirrors the library."""
    sh = s["shape"]
    di, dq, T, na, nb = sh["d_in"], sh["d_out"], sh["T"], sh["n_a"], sh["n_b"]
    tiles = math.ceil(na * _r16(T) / TILE) * math.ceil(nb * _r16(T) / TILE)
    tflops = tiles * 2.0 * TILE * TILE * (di + dq + 1)
    tbytes = tiles * 2.0 * TILE * (di + dq) * 2
    f = max(tflops / (model["ghost_tflops"] * 1e6), tbytes / (model["ghost_gbs"] * 1e3)) + model["ghost_layer_us"]
    f_bytes = (na * T + nb * T) * (di + dq) * 2
    build_bytes = f_bytes + 4 * (na + nb) * di * dq
    dot_bytes = 4 * (na + nb) * di * dq
    dtiles = math.ceil(dq / TILE) * math.ceil(di / TILE)
    per = 2.0 * TILE * TILE * _r32(T) / (model["build_tflops"] * 1e6 / SLOTS)
    rounds = (-(-(dtiles * na) // SLOTS) + -(-(dtiles * nb) // SLOTS)) * per
    b = max(rounds, build_bytes / (model["build_gbs"] * 1e3))
    m = b + dot_bytes / (model["dot_gbs"] * 1e3) + 4 * model["launch_us"]
    o = onepass_us(model, dtiles, na, nb, T) + 2 * model["launch_us"]
    return f, m, b + 2 * model["launch_us"], o


def fit(samples, start):
    from scipy.optimize import minimize

    def loss(x):
        model = {k: math.exp(v) for k, v in zip(FIELDS, x)}
        err = 0.0
        for s in samples:
            f, m, b, o = predict_us(model, s)
            pairs = [(f, s["factored_ms"]), (m, s["materialized_ms"]), (b, s["build_ms"])]
            if s.get("onepass_ms") is not None:
                pairs.append((o, s["onepass_ms"]))
            for pred, meas in pairs:
                err += (math.log(pred) - math.log(meas * 1e3)) ** 2
        return err

    x0 = [math.log(max(start[k], 1e-3)) for k in FIELDS]
    res = minimize(loss, x0, method="Nelder-Mead", options={"maxiter": 20000, "xatol": 1e-4, "fatol": 1e-8})
    return {k: math.exp(v) for k, v in zip(FIELDS, res.x)}


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--quick", action="store_true")
    ap.add_argument("--out")
    ap.add_argument("--refit", help="fit the samples of a saved output instead of measuring")
    args = ap.parse_args(argv)
    load()
    if args.refit:
        with open(args.refit) as f:
            saved = json.load(f)
        samples = [{k: s.get(k) for k in ("shape", "factored_ms", "materialized_ms", "onepass_ms", "build_ms",
                                          "counts")} for s in saved["samples"]]
        start = {k: saved["model"].get(k, 2.0) for k in FIELDS}
    else:
        device = torch.device("cuda:0")
        samples = []
        for shape in (QUICK if args.quick else SWEEP):
            samples.append(measure(shape, device))
            print(f"[calibrate_crossgram] {shape}: factored {samples[-1]['factored_ms']:.3f} ms, "
                  f"staged {samples[-1]['materialized_ms']:.3f} ms, one-pass {samples[-1]['onepass_ms']:.3f} ms, "
                  f"build {samples[-1]['build_ms']:.3f} ms", file=sys.stderr, flush=True)
        probe = ProjectionSession([dict(d_in=16, d_out=16, k_in=1, k_out=1)], dtype="bf16", device=device)
        start = dattri_get_crossgram_cost_model(probe.ctx)
        probe.close()
    model = fit(samples, start)
    rows, regrets = [], []
    for s in samples:
        f, m, _, o = predict_us(model, s)
        meas = {"factored": s["factored_ms"], "staged": s["materialized_ms"]}
        pred = {"factored": f, "staged": m}
        if s.get("onepass_ms") is not None:
            meas["one-pass"], pred["one-pass"] = s["onepass_ms"], o
        auto = min(pred, key=lambda k: (pred[k], k != "factored"))
        regrets.append(meas[auto] / min(meas.values()) - 1.0)
        rows.append({**s, "pred_factored_ms": f / 1e3, "pred_materialized_ms": m / 1e3, "pred_onepass_ms": o / 1e3,
                     "auto": auto, "auto_regret": regrets[-1]})
    out = {"model": model, "start": start, "samples": rows,
           "mean_regret": sum(regrets) / len(regrets), "max_regret": max(regrets),
           "auto_is_fastest": sum(r <= 1e-9 for r in regrets), "n": len(regrets)}
    text = json.dumps(out)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)
    print(text)


if __name__ == "__main__":
    main()
