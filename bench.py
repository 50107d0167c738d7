"""Benchmark: DeepCNet(5,50) sparse-convolution forward + backward, samples/s on one MI355X.

One step = rulebook build + forward + backward (every stage, the softmax layer
and its loss, all parameter gradients) for one batch of 100 synthetic
pen-stroke samples on a 96x96 grid; the inputs of 8 pre-generated batches are
resident in HBM before timing starts.  Prints one JSON line on stdout.

    python bench.py [--steps K] [--warmup W] [--dtype bf16|f32] [--workload NAME]
    python bench.py --workload deepcnet5_10_digits_b1000   # forward-only inference, characters/s
    python bench.py --calibrate-copy      # plain device copy, for counter scaling

Measurement: W untimed steps, then K steps between two device synchronisations
give `value`.  The same K steps are then run again with every launch of the
gather-GEMM kernel class bracketed by HIP events on the stream it runs on; the
roofline object divides that class's algorithmic FLOPs by its event-measured
time.  A second,
shorter pass times every kernel class for the breakdown.  The CPU baseline is
the oracle (test infrastructure) timed on this host on batch 0.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

from workloads import get_config, he_params, make_batches, make_paths, random_labels  # noqa: E402

DEFAULT_WORKLOAD = "deepcnet5_50_strokes_b100"
MFMA_PEAK = {"bf16": 2.5e15, "f32": 157.3e12}  # dense MFMA FLOP/s, MI355X
HBM_PEAK = 8.0e12  # bytes/s
PAPER_DIGITS_PER_S = 3000.0  # Section 3.2: DeepCNet(5,10) test-time classification rate, GTX 680
PROFILES = os.path.join(ROOT, "profiles")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def layer_shapes(cfg):
    """(kind, A, C_in, C_out) per stage of DeepCNet(ell, k) (Section 2.1) or DeepCNiN(ell, k)
    (Section 2.2: a 1x1 convolution after every pool and after the last convolution)."""
    nin = cfg.arch == "deepcnin"
    st = [("conv", 9, cfg.c_in, cfg.k)]
    c = cfg.k
    for n in range(2, cfg.ell + 2):
        st.append(("pool", 4, c, c))
        if nin:
            st.append(("conv", 1, c, c))
        st.append(("conv", 4, c, n * cfg.k))
        c = n * cfg.k
    if nin:
        st.append(("conv", 1, c, c))
    return st


def gemm_work(cfg, sizes, infer=False, e=2, routed=True):
    """Algorithmic FLOPs of one step, per kernel class, and the compulsory bytes of the
    gather-GEMM launches (e bytes per stored element).

    gather_gemm: convolution forward 2(n_s+1)A C_in C_out per stage (except a
    layer with at most 32 products per output and one 16-byte vector of input
    channels, the first layer of a one- or three-channel input: conv_narrow,
    the vector-ALU kernel), convolution
    input gradient 2 n_{s-1} A C_out C_in per stage s > 1 (the first layer's
    input gradient is not part of a training step), softmax layer forward and
    dh, 2 B C_last classes each.
    wgrad: 2(n_s+1)A C_in C_out per stage plus 2 B C_last classes.

    Compulsory bytes of a gather-GEMM launch (each operand moved once, channel
    padding not counted): forward (n_{s-1}+1)C_in e + (n_s+1)A*4 (window list,
    none for 1x1) + (n_s+1)C_out e + A C_in C_out e; input gradient
    (n_s+1)C_out e + (n_{s-1}+1)A*4 + n_{s-1}C_in e (+ the same again for the
    rectifier mask when a convolution lies below) + the weights; softmax layer
    forward B C e + 4B + 4B classes + C classes e, dh B classes e + 4 B C + the
    weights.  With ``routed`` an input-gradient GEMM whose output is a pooling
    layer also runs that layer's backward in its epilogue: + the convolution
    below's output read and delta written (n_c C e each), the argmax bytes
    (n_{s-1} C), the pooling windows (16 n_{s-1}) and, above the first layer,
    the convolution's window lists (n_c A_c 4).  A convolution with a pooling
    layer above computes that layer in its epilogue (even grid sides): + the
    pooling windows read (16 (n_p + 1)), the pooled rows and argmax written
    (n_p C_out (e + 1)).
    """
    fwd = dgrad = narrow = 0.0
    fbytes = dbytes = 0.0
    shapes = layer_shapes(cfg)
    ve = 16 // e
    for s, (kind, A, ci, co) in enumerate(shapes, start=1):
        if kind != "conv":
            continue
        n, nb = sizes[s], sizes[s - 1]
        w = A * ci * co * e
        if A > 1 and ci <= ve and A * ci <= 32:  # few input channels: the vector-ALU kernel, not a GEMM
            narrow += 2.0 * (n + 1) * A * ci * co
        else:
            fwd += 2.0 * (n + 1) * A * ci * co
            fbytes += (nb + 1) * ci * e + (n + 1) * (A * 4 if A > 1 else 0) + (n + 1) * co * e + w
            if s < len(shapes) and shapes[s][0] == "pool":  # the pooling layer above, in the epilogue
                npool = sizes[s + 1]
                fbytes += 16 * (npool + 1) + npool * co * (e + 1)
        if s > 1:
            dgrad += 2.0 * nb * A * co * ci
            mask = nb * ci * e if shapes[s - 2][0] == "conv" else 0
            dbytes += (n + 1) * co * e + (nb + 1) * (A * 4 if A > 1 else 0) + nb * ci * e + mask + w
            if routed and shapes[s - 2][0] == "pool" and A > 1:
                nc, Ac = sizes[s - 2], shapes[s - 3][1]
                dbytes += 2 * nc * ci * e + nb * ci + 16 * nb + (nc * Ac * 4 if s - 2 > 1 else 0)
    C = (cfg.ell + 1) * cfg.k
    B, K = cfg.batch, cfg.n_classes
    head = 2.0 * B * C * K
    hf_bytes = B * C * e + 4 * B + 4 * B * K + C * K * e
    hd_bytes = B * K * e + 4 * B * C + C * K * e
    if infer:  # forward only: conv forward and the logits
        return {"gather_gemm": fwd + head, "wgrad": 0.0, "conv_narrow": narrow, "conv_total": fwd + narrow,
                "gather_gemm_bytes": fbytes + hf_bytes}
    return {"gather_gemm": fwd + dgrad + 2 * head, "wgrad": fwd + narrow + head, "conv_narrow": narrow,
            "conv_total": 2 * (fwd + narrow) + dgrad, "gather_gemm_bytes": fbytes + dbytes + hf_bytes + hd_bytes}


def flops_8d(cfg, sizes):
    """Per convolution stage s: 2 (n_s + 1) A C_in C_out, the unit of algorithmic work that each of the
    forward, the input gradient and the weight gradient of that stage does (the per-stage figure of the
    measurement plan; the input gradient is counted over the stage's output rows like the others)."""
    out = {}
    for s, (kind, A, ci, co) in enumerate(layer_shapes(cfg), start=1):
        if kind == "conv":
            out[s] = 2.0 * (sizes[s] + 1) * A * ci * co
    return out


def rulebook_bytes(cfg, sizes):
    """Algorithmic bytes of the rulebook per step: n_in (8 + 8A) + n_out (8 + 4A) per stage."""
    tot = 0.0
    for s, (kind, A, ci, co) in enumerate(layer_shapes(cfg), start=1):
        tot += sizes[s - 1] * (8 + 8 * A) + sizes[s] * (8 + 4 * A)
    return tot


def narrow_bytes(cfg, sizes, e):
    """Algorithmic bytes of the first-layer vector-ALU kernel (with the pooling layer above it fused):
    per convolution row (ground row included) its window list 4A, its inputs A C_in e and its output C_out e;
    per pooling row its window 16 and its pooled value and argmax C_out (e + 1)."""
    kind, A, ci, co = layer_shapes(cfg)[0]
    n1, n2 = sizes[1], sizes[2]
    return (n1 + 1) * (4 * A + A * ci * e + co * e) + (n2 + 1) * 16 + n2 * co * (e + 1)


ROLE_NAMES = {0: "forward", 1: "input gradient", 2: "softmax logits", 3: "softmax dh", 4: "other"}
PLAN_NAMES = {0: "k_gemm_gather 128x128", 1: "k_gemm_gather 128x64", 2: "k_gemm_gather 64x64",
              3: "k_gemm_gather 32x64", 4: "k_gemm_direct 32x64", 15: ""}


def decode_tag(tag):
    return {"stage": tag & 0xFF, "role": (tag >> 8) & 0xF, "plan": (tag >> 12) & 0xF,
            "routed": bool((tag >> 16) & 1), "pooled": bool((tag >> 17) & 1)}


def group_key(kc, t):
    """A kernel instantiation: class, role, tile plan and fused epilogue."""
    if kc == "conv_narrow":
        return "k_conv_narrow (first layer, pooling forward fused; bf16 on the matrix cores, f32 on the vector ALUs)"
    if kc == "wgrad":
        return "k_wgrad (all weight gradients, grouped)"
    name = PLAN_NAMES.get(t["plan"], f"plan {t['plan']}")
    extra = " + pooling backward" if t["routed"] else (" + pooling forward" if t["pooled"] else "")
    return f"{name}: {ROLE_NAMES[t['role']]}{extra}"


def read_traffic(kernel, dtype, workload):
    """HBM bytes per launch from the committed counter summary, if it matches the current kernel source,
    the dtype and the workload."""
    path = os.path.join(PROFILES, f"{kernel}_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    h = hashlib.sha256()
    for name in kv.get("source", "gemm.hip").split():
        src = os.path.join(ROOT, "paper_1409_6070_amd", "csrc", name)
        if not os.path.exists(src):
            return None
        h.update(open(src, "rb").read())
    sha = h.hexdigest()[:16]
    if kv.get("source_sha256_16") != sha or kv.get("dtype") != dtype or kv.get("workload") != workload:
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _oracle_reps(cfg, batch, Ws, bs, labels, dtype, budget_s, infer, paths):
    """Repeats the oracle's step on batch 0 for about budget_s seconds; returns (reps, seconds)."""
    from oracle import SparseDeepCNet as Oracle
    from oracle.sgd import sgd_step
    from oracle.strokes import encode_strokes

    def storage(x):
        t = torch.tensor(np.asarray(x, np.float64), dtype=torch.float32)
        return (t.to(torch.bfloat16) if dtype == "bf16" else t).double().numpy()

    feats = storage(batch.feats) if batch is not None else None
    Wn = [storage(W) for W in Ws]
    if paths is not None:
        vW = [np.zeros_like(w) for w in Wn]
        vb = [np.zeros_like(np.asarray(x, np.float64)) for x in bs]
    reps, t0 = 0, time.perf_counter()
    while True:
        o = Oracle(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, dtype, cfg.arch)
        if paths is not None:
            coords, f = encode_strokes(paths.points, paths.stroke_begin, paths.stroke_sample, paths.batch, paths.grid)
            feats = storage(f)
            o.build(coords, paths.batch)
        else:
            o.build(batch.coords, batch.batch)
        if cfg.dropout and not infer:
            o.set_dropout(cfg.dropout, cfg.dropout_seed + reps)
        o.forward(feats, Wn, bs, labels)
        if not infer:
            dW, db, _ = o.backward()
            if cfg.sgd:
                Wn, _, bs, vW, vb = sgd_step(Wn, bs, dW, db, vW, vb, *cfg.sgd, mode=dtype)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 50:
            return reps, el


def cpu_baseline(cfg, batch, Ws, bs, labels, dtype, budget_s=12.0, infer=False, paths=None):
    """The oracle, as it stands, on batch 0: build + forward (+ backward unless infer), repeated for
    ~budget_s with the host's BLAS threads, then for ~budget_s / 2 on one thread.

    With pen paths (``paths``) each repetition is a whole training step: the oracle's encoding,
    build, forward, backward and SGD update."""
    try:
        from threadpoolctl import threadpool_info, threadpool_limits

        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threadpool_limits, threads = None, 1
    reps, el = _oracle_reps(cfg, batch, Ws, bs, labels, dtype, budget_s, infer, paths)
    single = None
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            r1, e1 = _oracle_reps(cfg, batch, Ws, bs, labels, dtype, budget_s / 2, infer, paths)
        single = round(r1 * cfg.batch / e1, 3)
    cpu = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    what = "build + forward" if infer else "build + forward + backward"
    if paths is not None:
        what = "encode + " + what
    if cfg.sgd:
        what += " + SGD update"
    return {"value": round(reps * cfg.batch / el, 3), "unit": "characters/s" if infer else "samples/s",
            "cores": threads, "kind": "oracle", "value_1_thread": single,
            "sample": f"batch 0 of {cfg.name} ({cfg.batch} samples), {reps} x ({what}), "
                      f"mode {dtype}, {el:.1f} s; NumPy float64, BLAS threads {threads} "
                      f"(value_1_thread: the same on one thread); host CPU: {cpu}"}


def calibrate_copy():
    """A plain device-to-device copy of known size (for scaling FETCH_SIZE / WRITE_SIZE)."""
    n = 256 << 20  # bytes
    a = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 3}))


TIMED = ["gather_gemm", "conv_narrow", "wgrad", "wgrad_reduce", "rulebook"]


def measure(cfg, dtype, steps, warmup, nbatches, cpu=True):
    """Times one workload; returns the JSON record (see the module docstring)."""
    from paper_1409_6070_amd.sscn import KERNEL_CLASSES, SparseDeepCNet, StrokeEncoder

    dev = torch.device("cuda:0")
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    log(f"[bench] {cfg.name} {dtype}: generating {nbatches} batches")
    paths = cfg.generator == "paths"
    Ws, bs = he_params(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, cfg.weight_seed, cfg.arch)
    labels = random_labels(cfg.batch, cfg.n_classes, cfg.label_seed)
    W32_d = [torch.tensor(W, dtype=torch.float32).to(dev).contiguous() for W in Ws]
    Ws_d = [w.to(tdt).contiguous() for w in W32_d] if dtype == "bf16" else W32_d
    bs_d = [torch.tensor(b, dtype=torch.float32).to(dev).contiguous() for b in bs]
    vW_d = [torch.zeros_like(w) for w in W32_d]
    vb_d = [torch.zeros_like(b) for b in bs_d]
    lab_d = torch.tensor(labels, dtype=torch.int32, device=dev)
    inputs, raw, path_batches, enc = [], [], [], None
    if paths:
        # raw pen paths: every step encodes them on the device (Section 2.4); one
        # untimed pass learns the site counts that size the encoder and the net
        path_batches = [make_paths(cfg, i) for i in range(nbatches)]
        raw = [tuple(torch.tensor(a, dtype=torch.int32, device=dev).contiguous()
                     for a in (p.points, p.stroke_begin, p.stroke_sample)) for p in path_batches]
        probe = StrokeEncoder(cfg.grid, cfg.batch, cfg.batch * cfg.grid * cfg.grid, dtype)
        counts = [int(probe.encode(*r, cfg.batch)[0].shape[0]) for r in raw]
        del probe
        max_active = max(counts)
        enc = StrokeEncoder(cfg.grid, cfg.batch, max_active, dtype)
        batches = []
    else:
        batches = make_batches(cfg, nbatches)
        for b in batches:
            # sites listed sample by sample (as the stroke and picture generators emit them): the
            # grouped rulebook build, given the per-sample offsets
            grouped = len(b.coords) == 0 or bool(np.all(np.diff(b.coords[:, 0]) >= 0))
            sb = (torch.tensor(np.searchsorted(b.coords[:, 0], np.arange(cfg.batch + 1)), dtype=torch.int32,
                               device=dev).contiguous() if grouped else None)
            inputs.append((torch.tensor(b.coords, dtype=torch.int32, device=dev).contiguous(),
                           torch.tensor(b.feats, dtype=torch.float32).to(tdt).to(dev).contiguous(), sb))
        max_active = max(b.n for b in batches)
    net = SparseDeepCNet(cfg.ell, cfg.k, cfg.c_in, cfg.n_classes, batch_max=cfg.batch, max_active=max_active,
                         dtype=dtype, arch=cfg.arch, dropout=bool(cfg.dropout))

    def inputs_of(i):
        if paths:  # synchronises: the site count goes to the host
            return (*enc.encode(*raw[i % len(raw)], cfg.batch), None)
        return inputs[i % len(inputs)]

    sizes = []
    for i in range(len(raw) if paths else len(inputs)):
        c, _, sb = inputs_of(i)
        net.rulebook_build(c, cfg.batch, sample_begin=sb)
        sizes.append(net.layer_sizes())
    torch.cuda.synchronize()

    infer = cfg.mode == "infer"

    def step(i):
        c, f, sb = inputs_of(i)
        net.rulebook_build(c, cfg.batch, sample_begin=sb)
        if infer:
            net.forward(f, Ws_d, bs_d, None)
        else:
            if cfg.dropout:  # fresh masks every step (a host-side call)
                net.set_dropout(cfg.dropout, cfg.dropout_seed + i)
            net.forward(f, Ws_d, bs_d, lab_d)
            net.backward()
            if cfg.sgd:
                net.sgd_step(W32_d, Ws_d if dtype == "bf16" else None, bs_d, vW_d, vb_d, *cfg.sgd)

    log(f"[bench] warmup {warmup} steps")
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    log(f"[bench] timing {steps} steps")
    t0 = time.perf_counter()
    for i in range(steps):
        step(i)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    sec = (t1 - t0) / steps
    value = cfg.batch / sec
    log(f"[bench] {sec * 1e3:.3f} ms/step, {value:.1f} samples/s")

    # The same K steps again with the launches of the convolution kernels and the
    # rulebook bracketed by HIP events on the stream they run on (the GEMM kernels
    # record their own start and end); the brackets slow the step, so `value`
    # above comes from the unbracketed pass.
    for kc in KERNEL_CLASSES:
        net.timing_launches(kc)  # drop anything recorded so far
    net.timing(TIMED)
    for i in range(steps):
        step(i)
    torch.cuda.synchronize()
    recs = {kc: net.timing_launches(kc) for kc in TIMED}
    net.timing([])

    # algorithmic work of the timed steps (batches cycle in order)
    step_sizes = [sizes[i % len(sizes)] for i in range(steps)]
    esz = 2 if dtype == "bf16" else 4
    peak = MFMA_PEAK[dtype]
    conv_fl = [flops_8d(cfg, sz) for sz in step_sizes]
    head_fl = 2.0 * cfg.batch * layer_shapes(cfg)[-1][3] * cfg.n_classes
    # each launch's algorithmic FLOPs from the sizes of its own step: in launch order a
    # step's forward launches precede its softmax logits, its input gradients follow them
    groups = {}  # key -> [launches, ms, flops]

    def add(key, ms, fl):
        g = groups.setdefault(key, [0, 0.0, 0.0])
        g[0] += 1
        g[1] += ms
        g[2] += fl

    conv_ms = conv_flops = 0.0
    for kc in ("gather_gemm", "conv_narrow"):
        nlog = 0
        for j, (tag, ms) in enumerate(recs[kc]):
            t = decode_tag(tag)
            if kc == "conv_narrow":
                si = j  # one launch per step
            elif t["role"] == 2:
                si, nlog = nlog, nlog + 1
            else:
                si = nlog if t["role"] == 0 else nlog - 1
            fl_step = conv_fl[min(max(si, 0), len(conv_fl) - 1)]
            if t["role"] in (0, 1):
                fl = fl_step.get(t["stage"], 0.0)
                conv_ms += ms
                conv_flops += fl
            else:
                fl = head_fl
            add(group_key(kc, t), ms, fl)
    wg_ms = sum(ms for _, ms in recs["wgrad"])
    wr_ms = sum(ms for _, ms in recs["wgrad_reduce"])
    if recs["wgrad"]:
        wg_fl = sum(sum(f.values()) for f in conv_fl)  # the softmax layer's weight gradient not counted
        g = groups.setdefault(group_key("wgrad", None), [0, 0.0, 0.0])
        g[0] += len(recs["wgrad"])
        g[1] += wg_ms
        g[2] += wg_fl
        conv_ms += wg_ms + wr_ms
        conv_flops += wg_fl
    table = []
    for key, (n, ms, fl) in groups.items():
        if "softmax" in key:
            continue
        table.append({"kernel": key, "launches_per_step": n / steps, "us_per_step": round(ms * 1e3 / steps, 2),
                      "avg_launch_us": round(ms * 1e3 / n, 3), "gflop_per_launch": round(fl / n / 1e9, 4),
                      "tflops": round(fl / (ms / 1e3) / 1e12, 3) if ms else 0.0,
                      "frac": round(fl / (ms / 1e3) / peak, 5) if ms else 0.0})
    table.sort(key=lambda r: -r["us_per_step"])
    dom = table[0]
    roofline = {
        "kernel": dom["kernel"], "bound": "mfma", "achieved": dom["tflops"], "peak": peak / 1e12,
        "unit": "TFLOP/s", "frac": dom["frac"],
        "traffic": read_traffic(traffic_key(dom["kernel"]), dtype, cfg.name),
        "launches_per_step": dom["launches_per_step"], "avg_launch_us": dom["avg_launch_us"],
        "algorithmic_gflop_per_launch": dom["gflop_per_launch"],
        "flop_convention": "2 (n_s + 1) A C_in C_out per convolution stage, for each of forward, input gradient "
                           "and weight gradient",
    }
    conv_frac = conv_flops / (conv_ms / 1e3) / peak if conv_ms else 0.0

    # memory-bound kernels against HBM bandwidth
    def hbm(kc, bytes_per_step):
        n = len(recs[kc])
        if not n:
            return None
        ms = sum(m for _, m in recs[kc])
        gbps = bytes_per_step * steps / (ms / 1e3) / 1e9
        return {"kernel_class": kc, "launches_per_step": n / steps, "us_per_step": round(ms * 1e3 / steps, 2),
                "algorithmic_mb_per_step": round(bytes_per_step / 1e6, 3), "achieved": round(gbps, 1),
                "peak": HBM_PEAK / 1e9, "unit": "GB/s", "frac": round(gbps * 1e9 / HBM_PEAK, 4)}

    mean_sizes = np.mean(np.array(step_sizes, dtype=np.float64), axis=0)
    hbm_objs = {"rulebook": hbm("rulebook", float(np.mean([rulebook_bytes(cfg, sz) for sz in step_sizes])))}
    if recs["conv_narrow"]:
        hbm_objs["conv_narrow"] = hbm("conv_narrow", float(np.mean([narrow_bytes(cfg, sz, esz)
                                                                    for sz in step_sizes])))

    # breakdown of one pass over a few steps with every class timed
    net.timing(KERNEL_CLASSES)
    nb = min(5, steps)
    for i in range(nb):
        step(i)
    breakdown = {}
    for kc in KERNEL_CLASSES:
        n, ms = net.timing_collect(kc)
        breakdown[kc] = {"launches_per_step": n / nb, "us_per_step": round(ms * 1e3 / nb, 2)}
    net.timing([])

    if infer:
        metric = f"DeepCNet({cfg.ell},{cfg.k}) forward-only characters/sec (digit pictures in a {cfg.grid}x{cfg.grid} grid)"
        unit = "characters/s"
    else:
        metric = "DeepCNet(5,50) sparse-conv fwd+bwd samples/sec; GEMM % MFMA peak"
        if cfg.arch != "deepcnet" or (cfg.ell, cfg.k) != (5, 50):
            metric = (f"{'DeepCNiN' if cfg.arch == 'deepcnin' else 'DeepCNet'}({cfg.ell},{cfg.k}) "
                      "sparse-conv fwd+bwd samples/sec; GEMM % MFMA peak")
        if cfg.dropout:
            metric = metric.replace("fwd+bwd", "fwd+bwd with dropout per level")
        if paths:
            metric = (f"DeepCNet({cfg.ell},{cfg.k}) M=9 training step (8-direction histogram encoding + "
                      "fwd + bwd + SGD) samples/sec; GEMM % MFMA peak")
        unit = "samples/s"
    out = {
        "metric": metric,
        "value": round(value, 2),
        "unit": unit,
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(sec * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name,
                   "net": f"{'DeepCNiN' if cfg.arch == 'deepcnin' else 'DeepCNet'}({cfg.ell},{cfg.k})",
                   "grid": cfg.grid,
                   "c_in": cfg.c_in, "classes": cfg.n_classes, "batch": cfg.batch,
                   "input_active_fraction": round(float(mean_sizes[0]) / (cfg.batch * cfg.grid ** 2), 4),
                   "step": ("rulebook build + forward (logits)" if infer else
                            ("pen-path encoding + " if paths else "") + "rulebook build + forward + backward" +
                            (" + SGD update" if cfg.sgd else "")),
                   **({"dropout": list(cfg.dropout)} if cfg.dropout else {})},
        "conv_gemm_gflop_per_step": round(float(np.mean([sum(f.values()) for f in conv_fl])) *
                                          (1 if infer else 3) / 1e9, 3),
        "roofline": roofline,
        "conv_gemm": {"frac": round(conv_frac, 5), "achieved": round(conv_flops / (conv_ms / 1e3) / 1e12, 3)
                      if conv_ms else 0.0, "peak": peak / 1e12, "unit": "TFLOP/s",
                      "us_per_step": round(conv_ms * 1e3 / steps, 2),
                      "kernels": "every convolution launch: forward (GEMM and vector-ALU), input gradient, "
                                 "weight gradient and its reduce; the softmax layer excluded"},
        "kernels": table,
        "hbm": hbm_objs,
        "kernel_breakdown": breakdown,
        "cpu_baseline": None,
    }
    if infer and cfg.ell == 5 and cfg.k == 10:
        # the paper's one speed figure is this workload: 3000 characters/s classified
        # by DeepCNet(5,10) on a GTX 680 (Section 3.2) -- another machine, context only
        out["vs_baseline"] = round(value / PAPER_DIGITS_PER_S, 2)
        out["baseline_context"] = "paper: 3000 characters/s, DeepCNet(5,10) forward on digit pictures, GTX 680 (Section 3.2)"
    if cpu:
        log("[bench] cpu baseline (oracle)")
        out["cpu_baseline"] = cpu_baseline(cfg, batches[0] if batches else None, Ws, bs, labels, dtype,
                                           infer=infer, paths=path_batches[0] if paths else None)
    del net
    torch.cuda.synchronize()
    return out


def traffic_key(kernel_name):
    """File-name key of a kernel group's counter summary in profiles/."""
    k = kernel_name.lower()
    for a, b in ((":", ""), ("+", ""), ("(", ""), (")", ""), (",", ""), (" ", "_")):
        k = k.replace(a, b)
    while "__" in k:
        k = k.replace("__", "_")
    return k


# rocprofv3 kernel names of each kernel group of the bench line (template arguments
# of the direct kernel: <waves per tile, epilogue>, 0 and 4 the pooling backward),
# and the sources whose hash a counter summary records
COUNTER_GROUPS = {
    "k_gemm_direct 32x64: input gradient + pooling backward": (
        r"k_gemm_direct<\d+, [04]>", "gemm_direct.hip epilogue.h pool_route.h ground_tasks.h kernels.h common.h"),
    "k_wgrad (all weight gradients, grouped)": (
        r"k_wgrad_trI|k_wgradI|k_wgrad<", "gemm.hip kernels.h common.h ground_tasks.h"),
    "k_gemm_gather 64x64: input gradient + pooling backward": (
        r"k_gemm_gatherIDF16bNS_4GCfgIDF16bLi2ELi2ELi2ELi2EEELi[04]EEE|k_gemm_gather<.*, [04]>\(sscn::GemmArgs\)",
        "gemm.hip epilogue.h pool_route.h ground_tasks.h kernels.h common.h"),
}


def _counter_rows(d):
    """(kernel name, counter, value) of every dispatch in a rocprofv3 --pmc csv directory."""
    import csv
    import glob
    rows = []
    for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                rows.append((r["Kernel_Name"], r["Counter_Name"], float(r["Counter_Value"]), r.get("Dispatch_Id")))
    return rows


def counter_summary(group, fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, workload, dtype, commands):
    """Writes profiles/<group>_traffic.txt: HBM bytes per launch of a kernel group from FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch), scaled by what the same counters read for a 256 MiB device copy."""
    import re
    pat, sources = COUNTER_GROUPS[group]
    n_copy = 256 << 20

    def per_dispatch(d, counter, name_re):
        vals = {}
        for name, c, v, disp in _counter_rows(d):
            if c.startswith(counter) and re.search(name_re, name):
                vals[disp] = vals.get(disp, 0.0) + v  # summed over the counter's instances
        return list(vals.values())

    cf = max(per_dispatch(copy_fetch_dir, "FETCH_SIZE", r"copy|Copy"))
    cw = max(per_dispatch(copy_write_dir, "WRITE_SIZE", r"copy|Copy"))
    fs, ws = n_copy / (cf * 1024.0), n_copy / (cw * 1024.0)
    f = per_dispatch(fetch_dir, "FETCH_SIZE", pat)
    w = per_dispatch(write_dir, "WRITE_SIZE", pat)
    rd, wr = float(np.mean(f)) * 1024 * fs, float(np.mean(w)) * 1024 * ws
    h = hashlib.sha256()
    for name in sources.split():
        h.update(open(os.path.join(ROOT, "paper_1409_6070_amd", "csrc", name), "rb").read())
    path = os.path.join(PROFILES, f"{traffic_key(group)}_traffic.txt")
    lines = [f"# HBM traffic per launch of {group}, {workload} {dtype} (one MI355X)",
             "# Commands (repository root):"] + [f"#   {c}" for c in commands] + [
             f"# Calibration: a 256 MiB device copy reads {fs:.4f} x FETCH_SIZE KiB x 1024 bytes and writes "
             f"{ws:.4f} x WRITE_SIZE KiB x 1024 bytes.",
             f"# {len(f)} FETCH_SIZE and {len(w)} WRITE_SIZE dispatches of the group (rocprofv3 names matching "
             f"{pat}), averaged per launch.",
             f"kernel: {group}", f"source: {sources}", f"workload: {workload}",
             f"source_sha256_16: {h.hexdigest()[:16]}", f"dtype: {dtype}",
             f"fetch_scale: {fs:.4f}", f"write_scale: {ws:.4f}",
             f"read_bytes_per_launch: {rd:.0f}", f"write_bytes_per_launch: {wr:.0f}",
             f"hbm_bytes_per_launch: {rd + wr:.0f}"]
    with open(path, "w") as fo:
        fo.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def traffic_table(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, trace_dir, out, title, commands):
    """A markdown table of every kernel's HBM traffic: FETCH_SIZE and WRITE_SIZE per dispatch (scaled by
    what the counters read for a 256 MiB device copy) averaged per kernel, launches per step (dispatches
    relative to the weight packing's, which runs once a step; rounded), and the average duration from a
    kernel trace of the same build, so bytes over time per launch."""
    import csv
    import glob
    n_copy = 256 << 20

    def per_kernel(d, counter):
        disp = {}
        for name, c, v, di in _counter_rows(d):
            if c.startswith(counter):
                key = (name, di)
                disp[key] = disp.get(key, 0.0) + v  # summed over the counter's instances
        out_ = {}
        for (name, _), v in disp.items():
            out_.setdefault(name, []).append(v)
        return out_

    cf = max(per_kernel(copy_fetch_dir, "FETCH_SIZE").items(), key=lambda kv: max(kv[1]) if "opy" in kv[0] else 0)
    cw = max(per_kernel(copy_write_dir, "WRITE_SIZE").items(), key=lambda kv: max(kv[1]) if "opy" in kv[0] else 0)
    fs, ws = n_copy / (max(cf[1]) * 1024.0), n_copy / (max(cw[1]) * 1024.0)
    fetch, write = per_kernel(fetch_dir, "FETCH_SIZE"), per_kernel(write_dir, "WRITE_SIZE")
    dur = {}
    for path in glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True):
        with open(path) as f:
            for r in csv.DictReader(f):
                dur[r["Name"]] = float(r["AverageNs"]) / 1e3
    ref = [k for k in fetch if "k_pack_all" in k]
    steps = len(fetch[ref[0]]) if ref else 1
    rows = []
    for name in fetch:
        if name not in write or "rocclr" in name or "at::native" in name:
            continue
        per_step = len(fetch[name]) // steps  # (the rulebook also runs once per resident batch to size them)
        if per_step < 1:
            continue
        rd = float(np.mean(fetch[name])) * 1024 * fs
        wr = float(np.mean(write[name])) * 1024 * ws
        us = dur.get(name)
        rows.append((name, per_step, rd, wr, us))
    tot = sum(n * (rd + wr) for _, n, rd, wr, _ in rows)
    rows.sort(key=lambda r: -r[1] * (r[2] + r[3]))
    lines = [f"# {title}", "", "Commands (repository root):", "```"] + list(commands) + ["```", "",
             f"FETCH_SIZE scale {fs:.4f}, WRITE_SIZE scale {ws:.4f} (bytes per KiB-count x 1024 that a 256 MiB "
             f"device copy reads and writes); {steps} steps in the counter runs; durations from the kernel "
             "trace of the same build (every launch of the kernel averaged).", "",
             "| kernel | launches per step | MB read per launch | MB written per launch | MB per step | "
             "avg us | GB/s | % of step traffic |", "|---|---:|---:|---:|---:|---:|---:|---:|"]
    for name, n, rd, wr, us in rows:
        nm = name.replace("|", "/")
        if len(nm) > 90:
            nm = nm[:34] + "..." + nm[-53:]
        gbs = f"{(rd + wr) / (us * 1e3):.0f}" if us else "–"
        lines.append(f"| `{nm}` | {n} | {rd / 1e6:.2f} | {wr / 1e6:.2f} | {n * (rd + wr) / 1e6:.2f} | "
                     f"{us:.2f} | {gbs} | {100 * n * (rd + wr) / tot:.1f} |" if us else
                     f"| `{nm}` | {n} | {rd / 1e6:.2f} | {wr / 1e6:.2f} | {n * (rd + wr) / 1e6:.2f} | – | – | "
                     f"{100 * n * (rd + wr) / tot:.1f} |")
    lines += ["", f"Total per step: {tot / 1e6:.1f} MB.", "",
              "Names: `k_gemm_gather` modes -1 plain, -2 with the pooling forward, 0 and 4 with the pooling "
              "backward (4: the children's ground pattern from the rulebook's masks); `GCfg<T, WM, WN, TM, TN>` "
              "is a (16 WM TM) x (16 WN TN) tile, `k_gemm_direct<SK, mode>` the 32 x 64 direct kernel with SK "
              "waves per tile; the demangler drops the template values of the two routed 64 x 64 "
              "`k_gemm_gather` instantiations, which differ in their last value (the mode)."]
    with open(out, "w") as fo:
        fo.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def trace_summary(trace_dir, out, title, command, top=30):
    """A markdown table of a rocprofv3 --kernel-trace --stats run's per-kernel statistics."""
    import csv
    import glob
    paths = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)
    rows = []
    for path in paths:
        with open(path) as f:
            rows += list(csv.DictReader(f))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    tot = sum(float(r["TotalDurationNs"]) for r in rows)
    lines = [f"# {title}", "", "Command (repository root):", "```", command, "```", "",
             "| kernel | calls | avg us | min us | max us | % of kernel time |", "|---|---:|---:|---:|---:|---:|"]
    for r in rows[:top]:
        name = r["Name"].replace("|", "/")
        if len(name) > 90:
            name = name[:87] + "..."
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{100 * float(r['TotalDurationNs']) / tot:.1f} |")
    with open(out, "w") as fo:
        fo.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def wave_summary(dirs, out, title, commands, top=20):
    """Per-kernel wave counters from several rocprofv3 --pmc runs (one counter set each): the mean per
    dispatch of every counter, and the derived columns of the table."""
    per = {}  # kernel -> counter -> [values per dispatch]
    for d in dirs:
        acc = {}
        for name, c, v, disp in _counter_rows(d):
            acc.setdefault((name, c), {}).setdefault(disp, 0.0)
            acc[(name, c)][disp] += v
        for (name, c), dd in acc.items():
            per.setdefault(name, {})[c] = float(np.mean(list(dd.values())))
    rows = []
    for name, c in per.items():
        w = c.get("SQ_WAVES", 0.0)
        if w <= 0:
            continue
        cyc = c.get("SQ_WAVE_CYCLES", 0.0)
        hits, miss = c.get("TCC_HIT_sum", 0.0), c.get("TCC_MISS_sum", 0.0)

        def f(key, scale=1.0):
            return c[key] * scale if key in c else None

        rows.append((cyc * 4 / w * w, name, {
            "VMEM lat": f("VmemLatency"), "waves/SIMD": f("MeanOccupancyPerActiveCU"),
            "L2 hit": hits / (hits + miss) if hits + miss else None,
            "wait": c["SQ_WAIT_ANY"] / cyc if cyc and "SQ_WAIT_ANY" in c else None,
            "issue": c["SQ_ACTIVE_INST_ANY"] / cyc if cyc and "SQ_ACTIVE_INST_ANY" in c else None,
            "VALU/wave": f("SQ_INSTS_VALU", 1 / w), "SALU": f("SQ_INSTS_SALU", 1 / w),
            "MFMA": f("SQ_INSTS_MFMA", 1 / w), "VMEM": f("SQ_INSTS_VMEM", 1 / w), "LDS": f("SQ_INSTS_LDS", 1 / w),
            "wave life (cycles)": cyc * 4 / w if cyc else None}))
    rows.sort(key=lambda r: -r[0])
    cols = ["VMEM lat", "waves/SIMD", "L2 hit", "wait", "issue", "VALU/wave", "SALU", "MFMA", "VMEM", "LDS",
            "wave life (cycles)"]
    lines = [f"# {title}", "", "Commands (repository root), one rocprofv3 pass per counter set:", "```"] + \
        list(commands) + ["```", "",
                          "Columns: VMEM latency (cycles, derived `VmemLatency`); mean waves per SIMD "
                          "(`MeanOccupancyPerActiveCU`); L2 hit rate; fractions of wave time waiting on anything "
                          "(`SQ_WAIT_ANY`) and issuing (`SQ_ACTIVE_INST_ANY`) out of `SQ_WAVE_CYCLES`; instructions "
                          "per wave; wave lifetime in cycles (4 x `SQ_WAVE_CYCLES` / `SQ_WAVES`). Means per "
                          "dispatch; kernels ordered by total wave time.", "",
                          "| kernel | " + " | ".join(cols) + " |", "|---|" + "---:|" * len(cols)]
    for _, name, v in rows[:top]:
        nm = name.replace("|", "/")
        nm = nm[:70] + "..." if len(nm) > 73 else nm

        def fmt(x, k):
            if x is None:
                return "–"
            return f"{x:.2f}" if k in ("L2 hit", "wait", "issue", "waves/SIMD") else f"{x:.0f}"
        lines.append(f"| `{nm}` | " + " | ".join(fmt(v[k], k) for k in cols) + " |")
    with open(out, "w") as fo:
        fo.write("\n".join(lines) + "\n")
    print("\n".join(lines))


TABLE_ORDER = ["deepcnet4_20_strokes_b8", "deepcnet5_50_strokes_b100", "deepcnet5_50_strokes_m8_b100",
               "deepcnet5_100_rgbpatch_b128", "deepcnet6_100_strokes_b64"]


def write_table(path, rows, steps, warmup):
    lines = ["# Throughput and roofline of every workload (one MI355X)", "",
             f"Command: `python bench.py --table {os.path.relpath(path, ROOT)} --steps {steps} --warmup {warmup}`",
             "", "samples/s from an unbracketed loop of the timed steps; the fractions from a second loop of the "
             "same steps with every convolution launch, the weight gradients and the rulebook bracketed by HIP "
             "events. Convolution GEMM fraction: 2 (n_s + 1) A C_in C_out per stage for each of forward, input "
             "gradient and weight gradient, over the time of every convolution launch (softmax layer excluded), "
             "against the dense MFMA peak of the dtype (bf16 2.5 PFLOP/s, f32 157.3 TFLOP/s). HBM fractions: "
             "algorithmic bytes over event time, against 8 TB/s.", "",
             "| workload | dtype | samples/s | ms/step | conv GEMM frac | dominant kernel | its frac | "
             "rulebook µs, HBM frac | first layer µs, HBM frac |",
             "|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        rb = r["hbm"].get("rulebook") or {}
        cn = r["hbm"].get("conv_narrow") or {}
        lines.append(
            f"| {r['config']['workload']} | {r['dtype']} | {r['value']:,.0f} | {r['ms_per_step']:.3f} | "
            f"{r['conv_gemm']['frac']:.4f} | {r['roofline']['kernel']} ({r['roofline']['avg_launch_us']:.1f} µs × "
            f"{r['roofline']['launches_per_step']:g}) | {r['roofline']['frac']:.4f} | "
            f"{rb.get('us_per_step', '–')}, {rb.get('frac', '–')} | {cn.get('us_per_step', '–')}, "
            f"{cn.get('frac', '–')} |")
    lines += ["", "Per kernel (µs per step, achieved fraction of the MFMA peak):", ""]
    for r in rows:
        lines.append(f"* {r['config']['workload']} {r['dtype']}: " + "; ".join(
            f"{k['kernel']} {k['us_per_step']} µs, {k['frac']:.4f}" for k in r["kernels"]))
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def write_batch_sweep(path, rows, steps, warmup, base):
    """Throughput and roofline fractions of one workload at several batch sizes (context for the
    fixed-batch headline: how far the same kernels go when each launch has more work)."""
    lines = [f"# Batch sweep: {base} (one MI355X)", "",
             f"Command: `python bench.py --workload {base} --batch-sweep {' '.join(str(r['config']['batch']) for r in rows)} "
             f"--sweep-out {os.path.relpath(path, ROOT)} --steps {steps} --warmup {warmup}`", "",
             "The same workload generator and network at other batch sizes (the headline is the batch of the "
             "measurement plan). Fractions as in the bench line: the dominant kernel group's algorithmic FLOPs over "
             "its event time, every convolution launch likewise (softmax layer excluded), against the dense MFMA "
             "peak of the dtype; the rulebook's algorithmic bytes over its event time against 8 TB/s.", "",
             "| batch | samples/s | ms/step | conv GEMM frac | dominant kernel | its frac | its µs per launch | "
             "rulebook µs, HBM frac |", "|---|---|---|---|---|---|---|---|"]
    for r in rows:
        rb = r["hbm"].get("rulebook") or {}
        lines.append(f"| {r['config']['batch']} | {r['value']:,.0f} | {r['ms_per_step']:.3f} | "
                     f"{r['conv_gemm']['frac']:.4f} | {r['roofline']['kernel']} | {r['roofline']['frac']:.4f} | "
                     f"{r['roofline']['avg_launch_us']:.1f} | {rb.get('us_per_step', '–')}, {rb.get('frac', '–')} |")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--dtype", default="bf16", choices=["bf16", "f32"])
    ap.add_argument("--batches", type=int, default=8)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true")
    ap.add_argument("--table", default=None, help="time every workload of the measurement plan, write a table")
    ap.add_argument("--counter-summary", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR"),
                    help="write profiles/<group>_traffic.txt from rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs of "
                         "this benchmark and of --calibrate-copy (no GPU needed)")
    ap.add_argument("--group", default="k_gemm_direct 32x64: input gradient + pooling backward")
    ap.add_argument("--commands", nargs="*", default=[], help="the commands that made the counter runs")
    ap.add_argument("--traffic-table", nargs=6,
                    metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR", "TRACE_DIR", "OUT_MD"),
                    help="per-kernel HBM traffic of a step from rocprofv3 FETCH_SIZE / WRITE_SIZE runs")
    ap.add_argument("--trace-summary", nargs=2, metavar=("TRACE_DIR", "OUT_MD"),
                    help="a markdown table of a rocprofv3 --kernel-trace --stats run (no GPU needed)")
    ap.add_argument("--title", default="Kernel trace")
    ap.add_argument("--batch-sweep", nargs="+", type=int, default=None,
                    help="time the workload at these batch sizes (context only), write --sweep-out")
    ap.add_argument("--sweep-out", default=None)
    ap.add_argument("--wave-summary", nargs="+", metavar="DIR",
                    help="per-kernel wave counters from rocprofv3 --pmc runs; the last argument is the output .md")
    args = ap.parse_args()
    if args.wave_summary:
        wave_summary(args.wave_summary[:-1], args.wave_summary[-1], args.title, args.commands)
        return
    if args.counter_summary:
        counter_summary(args.group, *args.counter_summary, args.workload, args.dtype, args.commands)
        return
    if args.traffic_table:
        traffic_table(*args.traffic_table, args.title, args.commands)
        return
    if args.trace_summary:
        trace_summary(args.trace_summary[0], args.trace_summary[1], args.title,
                      " ".join(args.commands) if args.commands else "")
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported here "
              "(the path would shard over samples with one all-reduce of dW/db per step)", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.batch_sweep:
        import dataclasses
        base = get_config(args.workload)
        rows = []
        for b in args.batch_sweep:
            cfg = dataclasses.replace(base, batch=b, name=f"{base.name}@{b}")
            rows.append(measure(cfg, args.dtype, args.steps, args.warmup, args.batches, cpu=False))
            rows[-1]["config"]["batch"] = b
            print(json.dumps(rows[-1]), flush=True)
        if args.sweep_out:
            write_batch_sweep(args.sweep_out, rows, args.steps, args.warmup, base.name)
        return
    if args.table:
        rows = []
        for name in TABLE_ORDER:
            cfg = get_config(name)
            for dt in cfg.dtypes:
                rows.append(measure(cfg, dt, args.steps, args.warmup, args.batches, cpu=False))
                print(json.dumps(rows[-1]), flush=True)
        write_table(args.table, rows, args.steps, args.warmup)
        return
    out = measure(get_config(args.workload), args.dtype, args.steps, args.warmup, args.batches,
                  cpu=not args.no_cpu_baseline)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
