"""Calibrate the routing cost model on the GPU it runs on.

The route choice between the factored and the materialized form (Sec. 3.2,
FLOP-aware routing; App. A.4) is made from exact FLOP and byte counts, the
number of kernel launches each form runs, and a small table of effective
rates (``dattri_cost_model``): per kernel class an MFMA rate and an HBM
bandwidth, a cost per launch and a cost per call.  This script measures them:

1. for a sweep of single-layer shapes it times, with HIP events on the launch
   stream, the forced factored route, the forced materialized route, and the
   materialized route's first kernel alone (G = B^T A, through
   ``dattri_materialize_gradient``); launch plans stay on the device between
   calls (the session binds a plan buffer), as in any repeated use;
2. it asks the library how many launches each form runs for each shape (its
   own planner, through the predictions of ``dattri_layer_route`` under a
   model whose launch cost dwarfs everything else);
3. it fits the eight fields, every rate held below a physical bound (the
   measured HBM read rate for bandwidths, the published MFMA peaks for
   FLOP rates), by minimising the squared log error of the predicted times
   plus a penalty on every shape whose predicted faster route is the
   measured slower one, weighted by the time that choice would lose; of fits
   from several starting points, the one with the least mean regret wins;
4. it prints one JSON object: the fitted model, and per shape the measured and
   predicted times of both routes, the route AUTO picks with the fitted model
   and its regret against the faster forced route.

Usage:  python -m paper_2609_38767_amd.calibrate [--quick] [--out FILE]
Load the file into a context with ``dattri_set_cost_calibration(ctx, FILE)``.
"""
import argparse
import json
import math
import sys
import time

import torch

from . import (DATTRI_ROUTE_FACTORED, DATTRI_ROUTE_MATERIALIZED,
               dattri_capture_layer, dattri_create, dattri_destroy, dattri_get_cost_model, dattri_layer_costs,
               dattri_layer_route, dattri_materialize_gradient, dattri_register_layer, dattri_set_cost_model,
               DATTRI_BF16, load)
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
    # more narrow and adapter-shaped layers, where the two routes are close
    (128, 128, 64, 64, 512, 32), (64, 64, 32, 32, 2048, 16), (256, 128, 64, 64, 1024, 32),
    (128, 512, 32, 32, 256, 64), (96, 96, 32, 32, 4096, 8), (256, 256, 32, 32, 128, 64),
]
QUICK = [SWEEP[i] for i in (0, 3, 5, 9, 13, 14, 17, 19)]

FIELDS = ["factored_tflops", "factored_gbs", "gradient_tflops", "gradient_gbs",
          "gproject_tflops", "gproject_gbs", "launch_us", "call_us", "round_us"]
# Upper bounds of the effective rates: the HBM read rate measured on MI355X
# (a streaming probe; below the 8 TB/s peak) and the published MFMA peaks
# (bf16 for the factored and G kernels, float32 for the G projection).
READ_GBS = 6450.0
CAPS = {"factored_tflops": 2500.0, "factored_gbs": READ_GBS, "gradient_tflops": 2500.0,
        "gradient_gbs": READ_GBS, "gproject_tflops": 157.3, "gproject_gbs": READ_GBS}


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


def launch_counts(shape):
    """(factored launches, materialized launches) the library plans for the
    shape alone, read from its predictions under a model in which one launch
    costs 10^6 us and all work is at peak rate (host-only, no GPU)."""
    d_in, d_out, k_in, k_out, T, n = shape
    ctx = dattri_create(DATTRI_BF16, 0)
    try:
        dattri_register_layer(ctx, d_in, d_out, k_in, k_out)
        fake = 1 << 40
        dattri_capture_layer(ctx, 0, fake, fake + (1 << 38), n, T, None)
        probe = {"factored_tflops": 2500.0, "factored_gbs": 8000.0, "gradient_tflops": 2500.0,
                 "gradient_gbs": 8000.0, "gproject_tflops": 157.3, "gproject_gbs": 8000.0,
                 "launch_us": 1e6, "call_us": 0.0, "round_us": 0.0}
        dattri_set_cost_model(ctx, probe)
        _, pf, pm = dattri_layer_route(ctx, 0)
    finally:
        dattri_destroy(ctx)
    return round(pf / 1e6), round(pm / 1e6)


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
    lf, lm = launch_counts(shape)
    return {"shape": {"d_in": d_in, "d_out": d_out, "k_in": k_in, "k_out": k_out, "T": T, "n": n},
            "factored_ms": t_f, "materialized_ms": t_m, "gradient_ms": t_g,
            "launches_gradient": (n + chunk - 1) // chunk, "launches_factored": lf,
            "launches_materialized": lm, "counts": costs}


class LibraryPredictor:
    """The library's own predictions (``dattri_layer_route``) for every sampled
    shape under a candidate model: one host-only context per shape with the
    shape captured at 16-byte aligned placeholder addresses (the alignment the
    sweep's tensors have); nothing is launched."""

    def __init__(self, samples):
        self.ctx = []
        fake = 1 << 40
        for s in samples:
            sh = s["shape"]
            c = dattri_create(DATTRI_BF16, 0)
            dattri_register_layer(c, sh["d_in"], sh["d_out"], sh["k_in"], sh["k_out"])
            dattri_capture_layer(c, 0, fake, fake + (1 << 38), sh["n"], sh["T"], None)
            self.ctx.append(c)

    def __call__(self, model):
        out = []
        for c in self.ctx:
            dattri_set_cost_model(c, model)
            _, pf, pm = dattri_layer_route(c, 0)
            out.append((pf, pm))
        return out

    def close(self):
        for c in self.ctx:
            dattri_destroy(c)
        self.ctx = []


# Fitted fields: gproject_tflops and gproject_gbs only enter the staged G
# route (float32 or unaligned blocks, k_in > 128), which the bf16 sweep does
# not run, so they keep their values.
FIT_FIELDS = [k for k in FIELDS if k not in ("gproject_tflops", "gproject_gbs")]


def _model_of(x, base):
    m = dict(base)
    for i, k in enumerate(FIT_FIELDS):
        if k in CAPS:  # (0, cap) through a logistic map
            m[k] = CAPS[k] / (1.0 + math.exp(-max(min(x[i], 50.0), -50.0)))
        else:
            m[k] = math.exp(max(min(x[i], 50.0), -50.0))
    return m


def _x_of(m):
    x = []
    for k in FIT_FIELDS:
        if k in CAPS:
            r = min(max(m[k] / CAPS[k], 1e-9), 1 - 1e-9)
            x.append(math.log(r / (1 - r)))
        else:
            x.append(math.log(max(m[k], 1e-3)))
    return x


def regret_of(preds, samples):
    """Per shape: time lost by the route predicted faster, relative to the
    faster measured route (0 when it picks that one)."""
    out = []
    for (f, m), s in zip(preds, samples):
        picked = s["factored_ms"] if f <= m else s["materialized_ms"]
        out.append(picked / min(s["factored_ms"], s["materialized_ms"]) - 1.0)
    return out


def fit(samples, starts, weight=4.0, margin=0.05, maxfev=4000):
    """Least squares on log predicted time plus a smooth penalty on wrong
    choices (a hinge on the predicted log-time gap, weighted by the measured
    gap); of the fits from `starts`, the one with the least mean regret."""
    from scipy.optimize import minimize
    predict = LibraryPredictor(samples)

    def loss(x):
        preds = predict(_model_of(x, starts[0]))
        err = 0.0
        for (f, mt), s in zip(preds, samples):
            lf, lm = math.log(1e3 * s["factored_ms"]), math.log(1e3 * s["materialized_ms"])
            err += (math.log(f) - lf) ** 2 + (math.log(mt) - lm) ** 2
            gap = lm - lf  # > 0 when the factored route is faster
            sign = 1.0 if gap >= 0 else -1.0
            err += weight * abs(gap) * max(0.0, margin - sign * (math.log(mt) - math.log(f))) ** 2 / margin
        return err
    best = None
    try:
        for start in starts:
            r = minimize(loss, _x_of(start), method="Nelder-Mead",
                         options={"maxfev": maxfev, "xatol": 1e-4, "fatol": 1e-7, "adaptive": True})
            m = _model_of(r.x, starts[0])
            reg = regret_of(predict(m), samples)
            key = (sum(reg) / len(reg), max(reg), r.fun)
            if best is None or key < best[0]:
                best = (key, m, r.fun)
    finally:
        predict.close()
    return best[1], best[2]


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
                     "gradient_ms": round(s["gradient_ms"], 4),
                     "launches_factored": s["launches_factored"],
                     "launches_materialized": s["launches_materialized"],
                     "pred_factored_ms": round(pf / 1e3, 4), "pred_materialized_ms": round(pm / 1e3, 4),
                     "auto": "factored" if route == DATTRI_ROUTE_FACTORED else "materialized",
                     "faster": "factored" if s["factored_ms"] <= s["materialized_ms"] else "materialized",
                     "regret": round(picked / best - 1.0, 4)})
    return rows


def _starts(default):
    return [default,
            dict(default, launch_us=2.0, call_us=20.0),
            dict(default, launch_us=10.0, call_us=5.0, factored_gbs=2000.0),
            dict(default, gproject_tflops=100.0, gradient_tflops=300.0)]


def _summary(model, loss, samples, rows, device_name):
    reg = [r["regret"] for r in rows]
    preds = [(1e3 * r["pred_factored_ms"], 1e3 * r["pred_materialized_ms"]) for r in rows]
    rms = math.sqrt(sum((math.log(p) - math.log(1e3 * m)) ** 2
                        for (pf, pm), s in zip(preds, samples)
                        for p, m in ((pf, s["factored_ms"]), (pm, s["materialized_ms"]))) / (2 * len(samples)))
    return {"model": model, "objective": loss, "rms_log_error": rms, "device": device_name, "shapes": rows,
            "picked_faster": sum(1 for r in rows if r["auto"] == r["faster"]), "n_shapes": len(rows),
            "max_regret": max(reg), "mean_regret": sum(reg) / len(reg)}


def _host_decisions(model, samples):
    """decisions() without a GPU: the library's route and predictions for
    each measured shape under `model`."""
    predict = LibraryPredictor(samples)
    try:
        preds = predict(model)
    finally:
        predict.close()
    rows = []
    for (pf, pm), s in zip(preds, samples):
        sh = s["shape"]
        best = min(s["factored_ms"], s["materialized_ms"])
        auto = "factored" if pf <= pm else "materialized"
        picked = s["factored_ms"] if auto == "factored" else s["materialized_ms"]
        rows.append({**sh, "factored_ms": s["factored_ms"], "materialized_ms": s["materialized_ms"],
                     "pred_factored_ms": round(pf / 1e3, 4), "pred_materialized_ms": round(pm / 1e3, 4),
                     "auto": auto, "faster": "factored" if s["factored_ms"] <= s["materialized_ms"] else "materialized",
                     "regret": round(picked / best - 1.0, 4)})
    return rows


def refit(path, out_path=None):
    """Refit the rates to the measured times in an earlier calibration JSON."""
    with open(path) as f:
        prev = json.load(f)
    keys = ("d_in", "d_out", "k_in", "k_out", "T", "n")
    samples = [{"shape": {k: r[k] for k in keys}, "factored_ms": r["factored_ms"],
                "materialized_ms": r["materialized_ms"]} for r in prev["shapes"]]
    ctx = dattri_create(DATTRI_BF16, 0)
    default = dattri_get_cost_model(ctx)
    dattri_destroy(ctx)
    model, loss = fit(samples, _starts(default))
    out = _summary(model, loss, samples, _host_decisions(model, samples), prev.get("device", ""))
    out["refit_of"] = path
    text = json.dumps(out)
    print(text, flush=True)
    if out_path:
        with open(out_path, "w") as f:
            f.write(text + "\n")


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--quick", action="store_true", help="a shorter sweep")
    ap.add_argument("--out", default=None, help="also write the JSON to this file")
    ap.add_argument("--refit", default=None, metavar="FILE",
                    help="refit the measurements of an earlier run's JSON on the host (no GPU)")
    args = ap.parse_args(argv)
    load()
    if args.refit:
        return refit(args.refit, args.out)
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
    default = dattri_get_cost_model(probe.ctx)
    probe.close()
    model, loss = fit(samples, _starts(default))
    rows = decisions(model, samples, device)
    out = _summary(model, loss, samples, rows, torch.cuda.get_device_name(device))
    # the library's built-in model on the same measurements (out of sample
    # when the defaults came from an earlier sweep)
    d_rows = decisions(default, samples, device)
    d_reg = [r["regret"] for r in d_rows]
    out["default_model"] = {"model": default, "picked_faster": sum(1 for r in d_rows if r["auto"] == r["faster"]),
                            "mean_regret": sum(d_reg) / len(d_reg), "max_regret": max(d_reg),
                            "shapes": [{k: r[k] for k in ("d_in", "d_out", "k_in", "k_out", "T", "n", "auto",
                                                          "faster", "regret")} for r in d_rows]}
    text = json.dumps(out)
    print(text, flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text + "\n")


if __name__ == "__main__":
    main()
