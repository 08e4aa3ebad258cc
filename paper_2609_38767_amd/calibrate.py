"""Calibrate the routing cost model on the GPU it runs on.

The route choice between the factored and the materialized form (Sec. 3.2,
FLOP-aware routing; App. A.4) is made from exact FLOP and byte counts and a
small table of effective rates: for each kernel class, an MFMA rate and an HBM
bandwidth, plus a per-launch overhead.  This script measures those rates:

1. for a sweep of single-layer shapes it times, with HIP events on the launch
   stream, the forced factored route, the forced materialized route, and the
   materialized route's first kernel alone (G = B^T A, through
   ``dattri_materialize_gradient``);
2. it fits the seven rates of ``dattri_cost_model`` by minimising the squared
   log error between predicted and measured times (Nelder-Mead on log rates);
3. it prints one JSON object: the fitted model, and per shape the measured and
   predicted times of both routes, the route AUTO picks with the fitted model
   and its regret against the faster forced route.

Usage:  python -m paper_2609_38767_amd.calibrate [--quick] [--out FILE]
The fitted rates can be installed on a context with ``dattri_set_cost_model``.
"""
import argparse
import json
import math
import sys
import time

import torch

from . import (DATTRI_ROUTE_AUTO, DATTRI_ROUTE_FACTORED, DATTRI_ROUTE_MATERIALIZED,
               dattri_get_cost_model, dattri_layer_costs, dattri_layer_route,
               dattri_materialize_gradient, dattri_set_cost_model, load)
from .session import ProjectionSession

# (d_in, d_out, k_in, k_out, T, n): transformer layer shapes from small to
# wide, short and long sequences, adapter-shaped and narrow layers
SWEEP = [
    (1024, 1024, 64, 64, 32, 8), (1024, 1024, 64, 64, 128, 8), (1024, 1024, 64, 64, 512, 8),
    (1024, 1024, 64, 64, 2048, 8),
    (1024, 4096, 64, 64, 32, 8), (1024, 4096, 64, 64, 512, 8), (1024, 4096, 64, 64, 2048, 8),
    (4096, 1024, 64, 64, 32, 8), (4096, 1024, 64, 64, 512, 8),
    (4096, 4096, 32, 32, 16, 16), (4096, 4096, 32, 32, 64, 16), (4096, 4096, 32, 32, 256, 16),
    (4096, 14336, 32, 32, 2048, 2),
    (8192, 28672, 64, 64, 32, 64),
    (8, 4096, 8, 64, 32, 64), (16, 4096, 16, 64, 64, 64), (4096, 8, 64, 8, 32, 64),
    (128, 128, 64, 64, 2048, 8), (128, 128, 64, 64, 256, 64), (256, 256, 64, 64, 512, 64),
    (64, 1024, 64, 64, 128, 64), (512, 512, 32, 32, 64, 64),
]
QUICK = [SWEEP[i] for i in (0, 3, 5, 9, 13, 14, 17, 19)]

FIELDS = ["factored_tflops", "factored_gbs", "gradient_tflops", "gradient_gbs",
          "gproject_tflops", "gproject_gbs", "launch_us"]


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


def measure(shape, device, seed=0):
    d_in, d_out, k_in, k_out, T, n = shape
    layer = {"d_in": d_in, "d_out": d_out, "k_in": k_in, "k_out": k_out}
    sess = ProjectionSession([layer], dtype="bf16", seed=seed, device=device)
    g = torch.Generator(device=device).manual_seed(seed)
    A = torch.randn((n, T, d_in), generator=g, device=device).to(torch.bfloat16)
    B = torch.randn((n, T, d_out), generator=g, device=device).to(torch.bfloat16)
    sess.capture(0, A, B)
    stream = torch.cuda.current_stream()
    phi = torch.empty((n, sess.F), dtype=torch.float32, device=device)
    t_f = _time_ms(lambda: sess.project(n, route=DATTRI_ROUTE_FACTORED, phi=phi), stream)
    t_m = _time_ms(lambda: sess.project(n, route=DATTRI_ROUTE_MATERIALIZED, phi=phi), stream)
    # the G = B^T A kernel alone, over the same examples, in chunks of at most 1 GiB
    per_ex = 4 * d_in * d_out
    chunk = max(1, min(n, (1 << 30) // per_ex))
    G = torch.empty((chunk, d_out, d_in), dtype=torch.float32, device=device)

    def grad_only():
        for e0 in range(0, n, chunk):
            dattri_materialize_gradient(sess.ctx, 0, e0, min(chunk, n - e0), G)
    t_g = _time_ms(grad_only, stream)
    costs = dattri_layer_costs(sess.ctx, 0, T)
    sess.close()
    del A, B, G, phi
    return {"shape": {"d_in": d_in, "d_out": d_out, "k_in": k_in, "k_out": k_out, "T": T, "n": n},
            "factored_ms": t_f, "materialized_ms": t_m, "gradient_ms": t_g,
            "launches_gradient": (n + chunk - 1) // chunk, "counts": costs}


def _counts(s):
    """Per-kernel-class (flops, bytes) totals for n examples; the same exact
    counts the library's cost model uses (dattri_layer_costs)."""
    sh = s["shape"]
    di, dq, ki, ko, T, n = sh["d_in"], sh["d_out"], sh["k_in"], sh["k_out"], sh["T"], sh["n"]
    f_flops, m_flops, f_bytes, m_bytes = s["counts"]
    g_flops = 2 * T * di * dq
    g_bytes = f_bytes + 4 * dq * di
    return {"f": (n * f_flops, n * f_bytes), "g": (n * g_flops, n * g_bytes),
            "p": (n * (m_flops - g_flops), n * (m_bytes - g_bytes))}


def predict_us(model, s):
    c = _counts(s)

    def t(flops, nbytes, tflops, gbs):
        return max(flops / (tflops * 1e6), nbytes / (gbs * 1e3))
    f = t(*c["f"], model["factored_tflops"], model["factored_gbs"]) + model["launch_us"]
    g = t(*c["g"], model["gradient_tflops"], model["gradient_gbs"]) + model["launch_us"]
    p = t(*c["p"], model["gproject_tflops"], model["gproject_gbs"]) + model["launch_us"]
    return f, g + p + model["launch_us"], g


def fit(samples, start):
    from scipy.optimize import minimize

    def loss(x):
        m = dict(zip(FIELDS, map(math.exp, x)))
        err = 0.0
        for s in samples:
            f, mt, g = predict_us(m, s)
            err += math.log(f / (1e3 * s["factored_ms"])) ** 2
            err += math.log(mt / (1e3 * s["materialized_ms"])) ** 2
            err += math.log(g / (1e3 * s["gradient_ms"])) ** 2
        return err
    x0 = [math.log(max(start[k], 1e-3)) for k in FIELDS]
    best = minimize(loss, x0, method="Nelder-Mead",
                    options={"maxiter": 20000, "maxfev": 20000, "xatol": 1e-4, "fatol": 1e-8})
    return dict(zip(FIELDS, map(math.exp, best.x))), best.fun


def decisions(model, samples, device):
    rows = []
    for s in samples:
        sh = s["shape"]
        sess = ProjectionSession([sh], dtype="bf16", device=device)
        dattri_set_cost_model(sess.ctx, model)
        A = torch.empty((sh["n"], sh["T"], sh["d_in"]), dtype=torch.bfloat16, device=device)
        B = torch.empty((sh["n"], sh["T"], sh["d_out"]), dtype=torch.bfloat16, device=device)
        sess.capture(0, A, B)
        route, pf, pm = dattri_layer_route(sess.ctx, 0)
        sess.close()
        best = min(s["factored_ms"], s["materialized_ms"])
        picked = s["factored_ms"] if route == DATTRI_ROUTE_FACTORED else s["materialized_ms"]
        rows.append({**sh, "factored_ms": round(s["factored_ms"], 4),
                     "materialized_ms": round(s["materialized_ms"], 4),
                     "pred_factored_ms": round(pf / 1e3, 4), "pred_materialized_ms": round(pm / 1e3, 4),
                     "auto": "factored" if route == DATTRI_ROUTE_FACTORED else "materialized",
                     "faster": "factored" if s["factored_ms"] <= s["materialized_ms"] else "materialized",
                     "regret": round(picked / best - 1.0, 4)})
    return rows


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--quick", action="store_true", help="a shorter sweep")
    ap.add_argument("--out", default=None, help="also write the JSON to this file")
    args = ap.parse_args(argv)
    load()
    device = torch.device("cuda:0")
    torch.cuda.set_device(device)
    samples = []
    for shape in (QUICK if args.quick else SWEEP):
        t0 = time.perf_counter()
        samples.append(measure(shape, device))
        s = samples[-1]
        print(f"[calibrate] {shape}: factored {s['factored_ms']:.4f} ms, materialized "
              f"{s['materialized_ms']:.4f} ms, gradient {s['gradient_ms']:.4f} ms "
              f"({time.perf_counter() - t0:.1f} s)", file=sys.stderr, flush=True)
    probe = ProjectionSession([{"d_in": 16, "d_out": 16, "k_in": 16, "k_out": 16}], device=device)
    start = dattri_get_cost_model(probe.ctx)
    probe.close()
    model, loss = fit(samples, start)
    rows = decisions(model, samples, device)
    out = {"model": model, "rms_log_error": math.sqrt(loss / (3 * len(samples))),
           "device": torch.cuda.get_device_name(device), "shapes": rows,
           "max_regret": max(r["regret"] for r in rows),
           "mean_regret": sum(r["regret"] for r in rows) / len(rows)}
    text = json.dumps(out)
    print(text, flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text + "\n")


if __name__ == "__main__":
    main()
