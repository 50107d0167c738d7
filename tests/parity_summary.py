"""Per-workload parity summary: every full-size workload through the HIP path and the oracle.

    python tests/parity_summary.py --out profiles/parity_summary.md [--json stats.json] [--only NAME]

For each workload and dtype it prints and tabulates, per layer, the normwise
error of row 0 and of rows >= 1 (each at its own scale), the elementwise error
with a floor of 1e-3 of the largest value, and the discrete decisions (pool
argmax, rectifier branch) that differ from the oracle's with their band
statistics, exactly as the GPU parity tests check them (``gpu_harness``).
Not collected by pytest; needs the GPU.
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

from tests import gpu_harness as H  # noqa: E402
from workloads import CONFIGS, get_config, he_params, make_batch, random_labels  # noqa: E402


def config_case(cfg, index=0):
    if cfg.generator == "paths":  # inputs from the oracle's encoding of the pen paths
        from oracle.strokes import encode_strokes
        from workloads import Batch, make_paths
        p = make_paths(cfg, index)
        coords, feats = encode_strokes(p.points, p.stroke_begin, p.stroke_sample, p.batch, p.grid)
        b = Batch(coords=coords.astype(np.int32), feats=feats, batch=cfg.batch, grid=cfg.grid)
    else:
        b = make_batch(cfg, index)
    Ws, bs = he_params(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, cfg.weight_seed, cfg.arch)
    labels = random_labels(cfg.batch, cfg.n_classes, cfg.label_seed)
    return b, Ws, bs, labels


def run_one(cfg, dtype):
    b, Ws, bs, labels = config_case(cfg)
    H.log(f"[summary] {cfg.name} {dtype} n={b.n} batch={cfg.batch}")
    t0 = time.perf_counter()
    pair = H.Pair(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, cfg.batch, b.coords, b.feats, Ws, bs, labels, dtype,
                  max_active=int(b.n * 1.25), arch=cfg.arch, rates=list(cfg.dropout) or None,
                  dseed=cfg.dropout_seed).run_gpu()
    H.check_structure(pair)
    pair.report, pair.stats, pair.failures = {}, {}, []
    check_grads = cfg.mode != "infer"
    if not check_grads:
        pass
    H._check_values(pair, None, check_grads)
    H.log(f"  {time.perf_counter() - t0:.1f} s, failures: {pair.failures or 'none'}")
    return pair.stats, pair.failures


def fmt(x):
    return "–" if x is None else (f"{x:.2e}" if isinstance(x, float) else str(x))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=None)
    ap.add_argument("--json", default=None)
    ap.add_argument("--only", default=None)
    args = ap.parse_args()
    assert torch.cuda.is_available(), "needs a GPU"
    from paper_1409_6070_amd import sscn
    sscn.load_library()
    results = {}
    for cfg in CONFIGS:
        if args.only and cfg.name != args.only:
            continue
        if cfg.mode == "infer":
            continue  # forward-only: its logits test covers it
        for dtype in cfg.dtypes:
            stats, failures = run_one(cfg, dtype)
            results[f"{cfg.name}/{dtype}"] = {"stats": stats, "failures": failures}
    if args.json:
        with open(args.json, "w") as f:
            json.dump(results, f, indent=1)
    lines = ["# GPU parity summary (full-size workloads)", "",
             f"Command: `python tests/parity_summary.py --out {args.out}`", "",
             "Per workload: the worst normwise error over all feature (X) and gradient (G) matrices, for row 0 "
             "and for rows >= 1 each at its own scale; the worst elementwise error (floor 1e-3 of the largest "
             "value) over rows >= 1; the worst parameter-gradient error; and the discrete decisions that differ "
             "from the oracle's (count / decisions, and in brackets the worst of: the oracle's gap between the two "
             "window values, or |Z| at a differing rectifier branch, in units of eps x the magnitude sum "
             "sum|w x| + |b| of the deciding convolution rows; eps = 2^-24 (f32), 2^-8 (bf16); the band is 1). "
             "Tolerances: f32 1e-4, bf16 2e-2 normwise; the elementwise figure is reported.", "",
             "| workload | dtype | X row 0 | X rows≥1 | X elem | G row 0 | G rows≥1 | G elem | dW/db | logits | "
             "argmax flips (max ulps) | rectifier flips (max) | failures |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for key, r in results.items():
        st = r["stats"]
        name, dtype = key.split("/")

        def worst(prefix, field):
            vals = [v[field] for k, v in st.items() if k.startswith(prefix) and k[len(prefix):].isdigit()
                    and field in v]
            return max(vals) if vals else None

        pg = [v["rows"] for k, v in st.items() if k.startswith(("dW", "db"))]
        af = sum(v["flips"] for k, v in st.items() if k.startswith("argmax"))
        ad = sum(v["decisions"] for k, v in st.items() if k.startswith("argmax"))
        ag = max([v.get("max_band", 0.0) for k, v in st.items() if k.startswith("argmax")] + [0.0])
        rf = sum(v["flips"] for k, v in st.items() if k.startswith("relu"))
        rd = sum(v["decisions"] for k, v in st.items() if k.startswith("relu"))
        rz = max([v.get("max_band", 0.0) for k, v in st.items() if k.startswith("relu")] + [0.0])
        lines.append(f"| {name} | {dtype} | {fmt(worst('X', 'row0'))} | {fmt(worst('X', 'rows'))} | "
                     f"{fmt(worst('X', 'elem'))} | {fmt(worst('G', 'row0'))} | {fmt(worst('G', 'rows'))} | "
                     f"{fmt(worst('G', 'elem'))} | {fmt(max(pg) if pg else None)} | "
                     f"{fmt(st.get('logits', {}).get('rows'))} | {af}/{ad} ({ag:.2f}) | {rf}/{rd} ({rz:.2f}) | "
                     f"{'; '.join(r['failures']) or 'none'} |")
    text = "\n".join(lines) + "\n"
    print(text)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)
    sys.exit(1 if any(r["failures"] for r in results.values()) else 0)


if __name__ == "__main__":
    main()
