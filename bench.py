"""Benchmark of the fused MAP pruning stage (map_prune) on one MI355X.

Workload: the LLaVA-NeXT-7B shape -- one image of 2880 visual tokens x 4096
(bf16), a 64-token question, keep 160 (K0 = 80) -- from the seeded synthetic
generator (random-init predictor weights).  A step is one map_prune call:
predictor scoring, cosine similarity, selection and gather, inputs resident
in HBM.  Prints one JSON line: the headline (exactly K timed steps, plus
the median / p10 / p90 of individually timed steps), its kernels and
rooflines, and objects for the rest:
* `assembly`: map_assemble, the layer-0 input built from the same image's
  kept rows;
* `training_step`: map_train_step, the predictor's KL step on the same
  image against a Dirichlet(1) teacher;
* `decoder_layer_context`: one random-init 7B-shaped decoder layer built
  from PyTorch-ROCm ops (not this library) over the unpruned 2944-token and
  the pruned 224-token sequence, and the pruning time as a fraction of the
  first;
* `teacher_selection`: map_teacher, Eq. (1)-(2), on synthetic attention of
  LLaVA-NeXT-7B's shape (32 layers x 32 heads x 2880 tokens), with its own
  oracle CPU baseline;
* `configs`: the other workloads (the small fp32 image, the 16-image sweep
  at each K, the 8-image multi-frame batch), each with its rooflines;
* `cpu_baseline`: the oracle on this host, all BLAS threads and one.

    python bench.py [--steps K] [--warmup W] [--no-cpu-baseline] [--no-teacher]
                    [--no-configs] [--no-context] [--no-train]
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "pruned images/sec + µs/image at N=2880,d=4096,K=160; % MFMA/HBM roofline"
PEAK_MFMA_BF16 = 2500.0   # TFLOP/s, dense
PEAK_MFMA_F32 = 157.3     # TFLOP/s
PEAK_HBM = 8000.0         # GB/s


R0_FACTOR_MAX = 128  # largest K0 the selection places by one factorisation (its own kernel)


def subset_tokens(cfg, setting=0):
    """Size of map_prune's candidate subset per image (0: the full path); the
    library's rule, restated (setting as for --subset)."""
    if setting < 0 or cfg.dtype != "bf16" or cfg.pred.D % 256 or cfg.N > 8192:
        return 0
    nc = setting
    if setting == 0:
        if 12 * cfg.K > cfg.N:
            return 0
        nc = (cfg.K0 + max(2 * (cfg.K - cfg.K0), cfg.N // 4) + 63) // 64 * 64
        if 4 * nc > 3 * cfg.N:
            return 0
    nc = max(nc, cfg.K)
    return nc if nc < cfg.N else 0


def norms_in_prep(cfg, sumM, nc, cus=256):
    """Whether map_prune's prep launch reads V for the row norms, restated
    from the library: on the subset path (bf16) the first-layer launch forms
    them, by its 256 x 256 tiles when those take fewer waves (a wave of them
    costs about 2.3 waves of 128 x 128 tiles), else by workgroups on the
    compute units its last wave of 128 x 128 tiles leaves idle (at least 16,
    at most 128 rows each); otherwise prep does."""
    if not nc or cfg.dtype != "bf16":
        return True
    H, dp = cfg.pred.D_h, cfg.pred.d_p

    def tiles(t):
        c = lambda a: -(-a // t)  # noqa: E731
        return c(cfg.B * cfg.N) * c(H) + c(sumM) * c(H) + 2 * c(dp) * c(H)
    t128, t256 = tiles(128), tiles(256)
    if 23 * -(-t256 // cus) < 10 * -(-t128 // cus):
        return False
    idle = (cus - t128 % cus) % cus
    return not (idle >= 16 and idle * 128 >= cfg.B * cfg.N)


def algorithmic_work(cfg, sumM, gathered=True, nc=0, chunks=None):
    """Per-launch algorithmic work of each kernel: (bound, amount, unit).
    `gathered`: the selection launch also gathers the kept rows (no gather launch).
    `nc`: tokens per image of the candidate subset the selection runs on (0: all N).
    `chunks`: the images' chunks of 16 question tokens (default: one image)."""
    if chunks is None:
        chunks = -(-sumM // 16)
    B, N, K, K0 = cfg.B, cfg.N, cfg.K, cfg.K0
    K0f = K0 if 0 < K0 <= R0_FACTOR_MAX else 0  # picks placed by the R0 kernel
    D, H, dp = cfg.pred.D, cfg.pred.D_h, cfg.pred.d_p
    el = 2 if cfg.dtype == "bf16" else 4
    rows = B * N + sumM
    Ns = nc if nc else N  # tokens the selection works on
    ks = D // 512 if D % 512 == 0 else D // 256
    tiles = ((nc + 127) // 128) * ((nc + 127) // 128 + 1) // 2
    return {
        # layer 1 of f_V and f_T, the folded weights W_K W2 and W_Q W2, and the
        # unique half (with the diagonal) of each Gram matrix
        "gemm_layer1_gram": ("mfma", 2.0 * rows * D * H + 2.0 * 2 * dp * H * H + B * N * (N + 1) * D, "flop"),
        # the same without the Gram matrix (candidate subset)
        "gemm_layer1": ("mfma", 2.0 * rows * D * H + 2.0 * 2 * dp * H * H, "flop"),
        # the subset: p, the norms and their reciprocals in; the subset's
        # tokens, p, norms and reciprocals out
        "subset": ("hbm", B * (12.0 * N + 16.0 * nc), "byte"),
        # the unique half (with the diagonal) of the subset's Gram matrix
        "gemm_subset": ("mfma", 1.0 * B * nc * (nc + 1) * D, "flop"),
        # the K-range partial sums in, the subset's cosine matrix out
        "gram_reduce": ("hbm", 4.0 * B * tiles * ks * 128 * 128 + 4.0 * B * nc * nc, "byte"),
        # second layer and projection as one product with the folded weights
        "gemm_proj_rope": ("mfma", 2.0 * rows * H * dp, "flop"),
        # read V, write norms, 1/norms and the cos/sin table; transpose the two
        # second-layer weights and fold the biases
        # (on the subset path the layer-1 launch usually forms the norms: no V here)
        "prep": ("hbm", (B * N * D * el + 8.0 * B * N if norms_in_prep(cfg, sumM, nc) else 0.0)
                 + 8.0 * rows * dp / 2 + 2 * 2.0 * H * H * el
                 + 2 * (dp * H + H) * el + 8.0 * dp, "byte"),
        # read the selection order and the kept rows, write the rows, indices and positions
        "gather": ("hbm", 2.0 * B * K * D * el + 16.0 * B * K, "byte"),
        # read keys and queries, write logits and per-block (max, sum of exp)
        "logits": ("hbm", 4.0 * (B * N + sumM) * dp + 4.0 * sumM * N + 8.0 * sumM * ((N + 63) // 64), "byte"),
        # read logits and partials, write p
        "softmax_mean": ("hbm", 4.0 * sumM * N + 8.0 * sumM * ((N + 63) // 64) + 4.0 * B * N, "byte"),
        # both in one launch: read keys and queries; the per-block (max, sum of
        # exp) pairs and each question chunk's share of p written and read once;
        # write p
        "score": ("hbm", 4.0 * (B * N + sumM) * dp + 16.0 * sumM * ((N + 63) // 64) + 8.0 * chunks * N
                  + 4.0 * B * N, "byte"),
        # R0 (K0 <= 128): p, the norms and the K0 similarity rows of R0 in; the
        # K0 coefficient rows of every token, r^2, order and gain out
        "select_r0": ("hbm", B * (12.0 * Ns + 8.0 * K0 * Ns + 8.0 * K0), "byte"),
        # the greedy picks of Eq. (4): p, the norms, r^2 and the coefficient rows
        # so far in, the similarity rows of the picks; order, gain and indices
        # out; and, gathered in the same launch, the kept rows and positions
        "select": ("hbm", B * (12.0 * Ns + 4.0 * K0f * Ns + 4.0 * (K - K0f) * Ns + 12.0 * (K - K0f))
                   + (2.0 * B * K * D * el + 16.0 * B * K if gathered and not nc else 0.0), "byte"),
        # behind a subset: the full path's launches work only for images the
        # subset cannot certify; the selection launch gathers the kept rows of
        # the others
        "select_full": ("hbm", 2.0 * B * K * D * el + 16.0 * B * K if gathered else 0.0, "byte"),
    }


# Source files whose kernels each traffic record covers; a record whose
# hash no longer matches the sources is stale and reported as null.
KERNEL_SOURCES = {
    "prep": ("prep.hip", "internal.h"),
    "gemm_layer1_gram": ("gemm.hip", "internal.h"),
    "gemm_layer1": ("gemm.hip", "internal.h"),
    "gemm_subset": ("gemm.hip", "internal.h"),
    "gram_reduce": ("gemm.hip", "internal.h"),
    "subset": ("subset.hip", "internal.h"),
    "gemm_gram_full": ("gemm.hip", "internal.h"),
    "select_full": ("select.hip", "internal.h"),
    "gemm_proj_rope": ("gemm.hip", "internal.h"),
    "logits": ("score.hip", "internal.h"),
    "softmax_mean": ("score.hip", "internal.h"),
    "score": ("score.hip", "internal.h"),
    "select_r0": ("select.hip", "internal.h"),
    "select": ("select.hip", "internal.h"),
    "gather": ("gather.hip", "internal.h"),
    "attn_colsum": ("teacher.hip", "internal.h"),
    "layer_sum": ("teacher.hip", "internal.h"),
    "layer_js": ("teacher.hip", "internal.h"),
    "teacher": ("teacher.hip", "internal.h"),
    "assemble": ("gather.hip", "internal.h"),
}


def sources_sha(kernel):
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2608_06411_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, calibrated on a plain copy), or None when there
    is none or the kernel's sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.txt")
    if kernel not in KERNEL_SOURCES or not os.path.exists(path):
        return None
    for line in open(path):
        f = line.split()
        if len(f) > 1 and f[0] == "kernel" and f[1] == kernel:
            kv = dict(x.split("=", 1) for x in f[2:])
            if kv.get("sha") == sources_sha(kernel):
                return float(kv["traffic_bytes"])
    return None


def roofline(kernel, work, kern, cfg, workload):
    bound, amount, unit = work[kernel]
    avg_s = kern[kernel]["avg_us"] * 1e-6
    if bound == "mfma":
        peak = PEAK_MFMA_BF16 if cfg.dtype == "bf16" else PEAK_MFMA_F32
        roof = {"bound": "mfma", "achieved": amount / avg_s / 1e12, "peak": peak, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": amount / avg_s / 1e9, "peak": PEAK_HBM, "unit": "GB/s"}
    roof.update({"frac": roof["achieved"] / roof["peak"], "traffic": measured_traffic(workload, kernel),
                 "kernel": kernel, "avg_us": kern[kernel]["avg_us"],
                 "algorithmic_per_launch": amount, "algorithmic_unit": unit})
    return roof


TEACHER_SHAPE = dict(L=32, H=32, M=64, M_ref=8, N=2880, n_top=1)  # LLaVA-NeXT-7B (Vicuna-7B: 32 layers x 32 heads)


def teacher_slices(B, L, N):
    """The library's slice count for the column sums, restated."""
    wgs = 2 * B * L * ((N + 511) // 512)
    return min(16, max(1, -(-4096 // wgs)))


def teacher_bench(args, mp, torch, dev):
    """Teacher selection (Eq. (1)-(2)) for one training sample of the
    LLaVA-NeXT shape, bf16 attention resident in HBM: samples/s, per-kernel
    times and the HBM roofline of the column-sum launch (algorithmic bytes:
    every attention element read once, plus the float32 partial rows)."""
    from workloads import make_attention
    sh = TEACHER_SHAPE
    L, H, M, M_ref, N = sh["L"], sh["H"], sh["M"], sh["M_ref"], sh["N"]
    A_f, A_s = make_attention(L, H, M, N, dtype="bf16", seed=40)
    R_f, R_s = make_attention(L, H, M_ref, N, dtype="bf16", seed=40, reference=True)
    A = torch.from_numpy(A_s.reshape(-1).view(np.int16)).to(dev).view(torch.bfloat16)
    R = torch.from_numpy(R_s.reshape(-1).view(np.int16)).to(dev).view(torch.bfloat16)
    m_off = [0, M]
    out = mp.map_teacher(A, R, m_off, L, H, N, M_ref, sh["n_top"])
    for _ in range(args.warmup):
        mp.map_teacher(A, R, m_off, L, H, N, M_ref, sh["n_top"], out=out)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        mp.map_teacher(A, R, m_off, L, H, N, M_ref, sh["n_top"], out=out)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    mp.timing_reset()
    mp.timing_enable(True)
    for _ in range(args.steps):
        mp.map_teacher(A, R, m_off, L, H, N, M_ref, sh["n_top"], out=out)
    torch.cuda.synchronize()
    per = mp.timing_read()
    mp.timing_enable(False)
    mp.timing_reset()
    kern = {k: {"avg_us": 1e3 * v[0] / v[1], "launches_per_step": v[1] / args.steps} for k, v in per.items()}
    S = teacher_slices(1, L, N)
    colsum_bytes = 2 * L * H * (M + M_ref) * N + 2 * L * S * N * 4
    avg_s = kern["attn_colsum"]["avg_us"] * 1e-6
    roof = {"bound": "hbm", "achieved": colsum_bytes / avg_s / 1e9, "peak": PEAK_HBM, "unit": "GB/s",
            "frac": colsum_bytes / avg_s / 1e9 / PEAK_HBM, "traffic": measured_traffic(args.workload, "attn_colsum"),
            "kernel": "attn_colsum", "avg_us": kern["attn_colsum"]["avg_us"],
            "algorithmic_per_launch": colsum_bytes, "algorithmic_unit": "bytes"}
    res = {"metric": "teacher-selected samples/s", "value": 1000.0 / ms, "unit": "samples/s", "ms_per_step": ms,
           "workload": f"teacher selection, LLaVA-NeXT-7B shape: L={L} H={H} N={N} M={M} M_ref={M_ref} "
                       f"n_top={sh['n_top']} bf16 attention (synthetic), one sample per step",
           "kernels": kern, "roofline": roof, "layers": out["layers"][0].tolist()}
    if not args.no_cpu_baseline:
        import oracle
        t0 = time.perf_counter()
        ref = oracle.teacher_selection(A_f, R_f, sh["n_top"])
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": 1.0 / dt, "unit": "samples/s", "cores": 1, "kind": "oracle",
                               "sample": "one sample of the same workload (fp64 numpy reductions, one thread)"}
        res["oracle_layers"] = ref.layers.tolist()
    return res


def assembly_bench(args, mp, torch, dev, out, T, pos_t, t_off, cfg):
    """map_assemble after the timed map_prune steps: the layer-0 input of the
    language model (kept rows, then question rows) for the same image.  HBM
    roofline on its algorithmic bytes: every row read once and written once,
    plus 4 B of position each way per row."""
    X, pos = mp.map_assemble(out["V_out"], out["pos_out"], T, pos_t, t_off)
    mp.timing_reset()
    mp.timing_enable(True)
    for _ in range(args.steps):
        mp.map_assemble(out["V_out"], out["pos_out"], T, pos_t, t_off)
    torch.cuda.synchronize()
    per = mp.timing_read()
    mp.timing_enable(False)
    mp.timing_reset()
    avg_us = 1e3 * per["assemble"][0] / per["assemble"][1]
    rows = X.shape[0]
    nbytes = 2 * rows * (X.shape[1] * X.element_size() + 4)
    return {"workload": f"layer-0 input of {cfg.name}: {cfg.B} x ({cfg.K} kept + question) rows x {X.shape[1]} "
                        f"{cfg.dtype}", "rows": rows, "avg_us": avg_us,
            "roofline": {"bound": "hbm", "achieved": nbytes / (avg_us * 1e-6) / 1e9, "peak": PEAK_HBM, "unit": "GB/s",
                         "frac": nbytes / (avg_us * 1e-6) / 1e9 / PEAK_HBM,
                         "traffic": measured_traffic(args.workload, "assemble"), "kernel": "assemble",
                         "algorithmic_per_launch": nbytes, "algorithmic_unit": "bytes"}}


def _oracle_weights(x):
    names = ("w1_v", "b1_v", "w2_v", "b2_v", "w_k", "w1_t", "b1_t", "w2_t", "b2_t", "w_q")
    return {n: x[n + "_f32"] for n in names}


def _oracle_prune_one(x, cfg):
    import oracle
    lo, hi = int(x["t_off"][0]), int(x["t_off"][1])
    return oracle.prune(x["V_f32"][:1], x["T_f32"][lo:hi], np.array([0, hi - lo]), x["pos_v"][:1],
                        x["pos_t"][lo:hi], _oracle_weights(x), cfg.K, cfg.K0, cfg.tau, cfg.pred.rope_theta)


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(x, cfg, tiny_x=None, tiny_cfg=None, min_seconds=10.0, max_runs=8):
    """The oracle as it stands, timed on this host: the workload's first image,
    run again until at least `min_seconds` of CPU work (at most `max_runs`),
    with every BLAS thread; then once on one thread; and the small fp32
    workload's image both ways.  `value` is the all-thread rate."""
    from threadpoolctl import threadpool_info, threadpool_limits
    runs, t0 = 0, time.perf_counter()
    while True:
        _oracle_prune_one(x, cfg)
        runs += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds or runs >= max_runs:
            break
    threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    with threadpool_limits(limits=1, user_api="blas"):
        t1 = time.perf_counter()
        _oracle_prune_one(x, cfg)
        single = time.perf_counter() - t1
    per_config = {cfg.name: {"all_threads_s_per_image": dt / runs, "single_thread_s_per_image": single}}
    if tiny_x is not None:
        t2 = time.perf_counter()
        _oracle_prune_one(tiny_x, tiny_cfg)
        a = time.perf_counter() - t2
        with threadpool_limits(limits=1, user_api="blas"):
            t3 = time.perf_counter()
            _oracle_prune_one(tiny_x, tiny_cfg)
            b = time.perf_counter() - t3
        per_config[tiny_cfg.name] = {"all_threads_s_per_image": a, "single_thread_s_per_image": b}
    return {"value": runs / dt, "unit": "images/s", "cores": int(threads or 1), "kind": "oracle",
            "sample": f"{runs} run(s) of one image of the workload (N={cfg.N}, D={cfg.pred.D}, "
                      f"M={int(x['t_off'][1])}, K={cfg.K}, K0={cfg.K0}): float64 predictor, literal Eq. (4) "
                      f"greedy, gather; {dt:.2f} s with {threads} BLAS threads on {os.cpu_count()} visible CPUs",
            "single_thread": {"value": 1.0 / single, "unit": "images/s", "cores": 1,
                              "sample": "one run of the same image on one BLAS thread"},
            "cpu_model": _cpu_model(), "per_config": per_config}


def _to_dev(torch, dev, a, dtype):
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


WEIGHT_NAMES = ("w1_v", "b1_v", "w2_v", "b2_v", "w_k", "w1_t", "b1_t", "w2_t", "b2_t", "w_q")


def _upload(mp, torch, dev, x, cfg):
    w = mp.PredictorWeights(**{n: _to_dev(torch, dev, x[n + "_store"], cfg.dtype) for n in WEIGHT_NAMES},
                            rope_theta=cfg.pred.rope_theta)
    return dict(w=w, V=_to_dev(torch, dev, x["V_store"], cfg.dtype), T=_to_dev(torch, dev, x["T_store"], cfg.dtype),
                pos_v=torch.from_numpy(x["pos_v"]).to(dev), pos_t=torch.from_numpy(x["pos_t"]).to(dev))


def _kernel_table(mp, torch, run, steps):
    """Per-kernel average durations over `steps` calls of run(), measured with
    HIP events on the launch stream by the library's timing registry."""
    mp.timing_reset()
    mp.timing_enable(True)
    for _ in range(steps):
        run()
    torch.cuda.synchronize()
    per = mp.timing_read()
    mp.timing_enable(False)
    mp.timing_reset()
    return {k: {"avg_us": 1e3 * v[0] / v[1], "launches_per_step": v[1] / steps} for k, v in per.items()}


def _time_steps(torch, dev, run, steps, warmup, per_step=0):
    """ms per call over exactly `steps` timed calls (events bracketing the
    region, synchronised on both sides), and optionally the median, p10 and
    p90 of `per_step` individually timed calls."""
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    e0.record(stream)
    for _ in range(steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    res = {"ms_per_step": e0.elapsed_time(e1) / steps, "wall_s_timed": wall}
    if per_step:
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(per_step)]
        for a, b in ev:
            a.record(stream)
            run()
            b.record(stream)
        torch.cuda.synchronize()
        us = np.array([1e3 * a.elapsed_time(b) for a, b in ev])
        res["step_us"] = {"median": float(np.median(us)), "p10": float(np.percentile(us, 10)),
                          "p90": float(np.percentile(us, 90)), "samples": per_step}
    return res


def cold_steps(torch, dev, run, n, evict_mib=512):
    """Median, p10 and p90 of n individually timed calls, each after a write
    of evict_mib MiB of scratch memory (outside the timed region) that evicts
    the inputs from the Infinity Cache and the L2s: the step as it runs when
    its image arrives fresh in HBM."""
    scratch = torch.empty(evict_mib << 18, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for a, b in ev:
        scratch.fill_(1.0)
        a.record(stream)
        run()
        b.record(stream)
    torch.cuda.synchronize()
    us = np.array([1e3 * a.elapsed_time(b) for a, b in ev])
    del scratch
    return {"median": float(np.median(us)), "p10": float(np.percentile(us, 10)),
            "p90": float(np.percentile(us, 90)), "samples": n, "evict_mib_between_steps": evict_mib}


def concurrent_streams(mp, torch, dev, cfg, x, d, steps, warmup, n):
    """Images/s when n streams each run map_prune calls on the workload back
    to back (same batch size, own workspaces and outputs): one call's
    selection, which keeps a few compute units busy, runs beside another
    call's matrix products.  A serving context for the headline, not
    `value`; the outputs are checked equal to the single-stream ones."""
    t_off = x["t_off"]
    streams = [torch.cuda.Stream(dev) for _ in range(n)]
    wss = [mp.PruneWorkspace(d["w"], d["V"], t_off, cfg.K) for _ in streams]
    outs = []
    for st, ws in zip(streams, wss):
        with torch.cuda.stream(st):
            outs.append(mp.map_prune(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], t_off, cfg.K, cfg.K0, cfg.tau,
                                     workspace=ws))

    def run(i):
        with torch.cuda.stream(streams[i]):
            mp.map_prune(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], t_off, cfg.K, cfg.K0, cfg.tau,
                         out=outs[i], workspace=wss[i])

    for _ in range(warmup):
        for i in range(n):
            run(i)
    torch.cuda.synchronize()
    main = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(main)
    for st in streams:
        st.wait_event(e0)
    for _ in range(steps):
        for i in range(n):
            run(i)
    for st in streams:
        done = torch.cuda.Event()
        done.record(st)
        main.wait_event(done)
    e1.record(main)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    ref = mp.map_prune(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], t_off, cfg.K, cfg.K0, cfg.tau)
    torch.cuda.synchronize()
    same = all(torch.equal(o["idx"], ref["idx"]) and torch.equal(o["V_out"].view(torch.int16),
                                                                  ref["V_out"].view(torch.int16)) for o in outs)
    images = n * steps * cfg.B
    return {"streams": n, "value": images / (ms * 1e-3), "unit": "images/s", "us_per_image": 1e3 * ms / images,
            "calls_per_stream": steps, "outputs_equal_single_stream": bool(same)}


def measure_prune(mp, torch, dev, cfg, x, d, steps, warmup, subset=0, per_step=0, workload_key=None, cold=0):
    """One workload's map_prune: throughput, per-kernel times and rooflines.
    Returns (result dict, output tensors)."""
    t_off = x["t_off"]
    mp.set_subset_tokens(subset)
    ws = mp.PruneWorkspace(d["w"], d["V"], t_off, cfg.K)
    out = mp.map_prune(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], t_off, cfg.K, cfg.K0, cfg.tau, workspace=ws)

    def step():
        mp.map_prune(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], t_off, cfg.K, cfg.K0, cfg.tau, out=out,
                     workspace=ws)

    tm = _time_steps(torch, dev, step, steps, warmup, per_step)
    if cold:
        tm["step_us_cold"] = cold_steps(torch, dev, step, cold)
    kern = _kernel_table(mp, torch, step, steps)
    sumM = int(t_off[-1])
    nc = subset_tokens(cfg, subset) if "subset" in kern else 0
    chunks = sum(-(-(int(t_off[b + 1]) - int(t_off[b])) // 16) for b in range(cfg.B))
    work = algorithmic_work(cfg, sumM, gathered="gather" not in kern, nc=nc, chunks=chunks)
    # (the full-path launches behind a subset do work only for images the
    # subset cannot certify: they are never the dominant kernel)
    dominant = max((k for k in kern if not k.endswith("_full")),
                   key=lambda k: kern[k]["avg_us"] * kern[k]["launches_per_step"])
    key = workload_key or cfg.name
    roof = roofline(dominant, work, kern, cfg, key)
    gemm = max((k for k in kern if work.get(k, ("",))[0] == "mfma"), key=lambda k: kern[k]["avg_us"])
    roof_mfma = roofline(gemm, work, kern, cfg, key)
    if dominant == "select":
        # a chain of dependent picks: per-pick latency, not bandwidth, sets its time
        greedy = cfg.K - (cfg.K0 if 0 < cfg.K0 <= R0_FACTOR_MAX else 0)
        roof["note"] = (f"latency-bound: {greedy} sequential greedy picks per image, "
                        f"{kern[dominant]['avg_us'] / max(greedy, 1):.2f} us per pick (all images at once)")
    hbm = {}
    for k in kern:
        if work.get(k, ("",))[0] == "hbm" and k not in ("select", "select_r0", "subset"):
            r = roofline(k, work, kern, cfg, key)
            hbm[k] = {"achieved": r["achieved"], "frac": r["frac"], "avg_us": r["avg_us"],
                      "algorithmic_per_launch": r["algorithmic_per_launch"]}
    ms = tm["ms_per_step"]
    res = {"value": cfg.B * 1000.0 / ms, "unit": "images/s", "us_per_image": 1000.0 * ms / cfg.B,
           "dtype": cfg.dtype,
           "workload": f"{cfg.name}: B={cfg.B} N={cfg.N} D={cfg.pred.D} M={sumM} K={cfg.K} K0={cfg.K0} "
                       f"tau={cfg.tau} D_h={cfg.pred.D_h} d_p={cfg.pred.d_p} {cfg.dtype}",
           "subset_tokens": nc, **tm, "kernels": kern, "dominant_kernel": dominant, "roofline": roof,
           "roofline_mfma": roof_mfma, "hbm_stages": hbm}
    mp.set_subset_tokens(0)
    return res, out


def train_flops(cfg, sumM):
    """Algorithmic flops of one training step's matrix products: the forward
    (layer 1, the folded weights, the projection) and the backward (X = dz^T h
    and dL/da per branch; dW1 of f_V in one launch; dW1 of f_T, dW_K, dW2 in
    another)."""
    D, H, dp = cfg.pred.D, cfg.pred.D_h, cfg.pred.d_p
    rows = cfg.B * cfg.N + sumM
    fwd = 2.0 * rows * D * H + 4.0 * dp * H * H + 2.0 * rows * H * dp
    bwd = 4.0 * dp * H * rows + 2.0 * H * D * rows + 8.0 * dp * H * H
    return {"gemm_layer1": 2.0 * rows * D * H + 4.0 * dp * H * H, "gemm_proj_rope": 2.0 * rows * H * dp,
            "gemm_train_x_da": 4.0 * dp * H * rows, "gemm_train_dw": 2.0 * H * D * cfg.B * cfg.N,
            "gemm_train_dw_small": 2.0 * H * D * sumM + 8.0 * dp * H * H,
            "total": fwd + bwd}


def train_bench(mp, torch, dev, cfg, x, d, steps, warmup):
    """One predictor training step (KL from a teacher to p_hat, forward and
    backward) on the workload: steps/s, per-kernel times, and the matrix-core
    roofline of the whole step and of its largest product."""
    rng = np.random.default_rng(5)
    p_star = torch.from_numpy(rng.dirichlet(np.ones(cfg.N), size=cfg.B).astype(np.float32)).to(dev)
    ws = mp.TrainWorkspace(d["w"], d["V"], x["t_off"])
    loss, p, g = mp.map_train_step(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"], p_star, workspace=ws)

    def step():
        mp.map_train_step(d["w"], d["V"], d["pos_v"], d["T"], d["pos_t"], x["t_off"], p_star, grads=g, p_out=p,
                          workspace=ws)

    tm = _time_steps(torch, dev, step, steps, warmup)
    kern = _kernel_table(mp, torch, step, steps)
    fl = train_flops(cfg, int(x["t_off"][-1]))
    ms = tm["ms_per_step"]
    peak = PEAK_MFMA_BF16 if cfg.dtype == "bf16" else PEAK_MFMA_F32
    big = max((k for k in kern if k in fl), key=lambda k: kern[k]["avg_us"])
    ach = fl[big] / (kern[big]["avg_us"] * 1e-6) / 1e12
    return {"metric": "predictor training steps/s", "value": 1000.0 / ms, "unit": "steps/s", **tm,
            "workload": f"training step on {cfg.name}: B={cfg.B} N={cfg.N} D={cfg.pred.D} "
                        f"M={int(x['t_off'][-1])} D_h={cfg.pred.D_h} d_p={cfg.pred.d_p} {cfg.dtype}, "
                        f"Dirichlet(1) teacher",
            "loss": float(loss.mean().item()), "kernels": kern,
            "roofline_step": {"bound": "mfma", "achieved": fl["total"] / (ms * 1e-3) / 1e12, "peak": peak,
                              "unit": "TFLOP/s", "frac": fl["total"] / (ms * 1e-3) / 1e12 / peak,
                              "algorithmic_per_step": fl["total"], "algorithmic_unit": "flop"},
            "roofline_mfma": {"bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s", "frac": ach / peak,
                              "traffic": None, "kernel": big, "avg_us": kern[big]["avg_us"],
                              "algorithmic_per_launch": fl[big], "algorithmic_unit": "flop"}}


def decoder_layer_context(torch, dev, prune_us, steps=20, warmup=5):
    """One random-init 7B-shaped decoder layer (d 4096, 32 heads x 128, SwiGLU
    11008, RMSNorm, RoPE, causal attention; bf16) built from PyTorch-ROCm
    ops, outside the library, timed over the unpruned (2944) and pruned
    (224) sequences of the LLaVA-NeXT workload: the context for the pruning
    stage's own time."""
    import torch.nn.functional as F
    from torch.nn.attention import SDPBackend, sdpa_kernel
    d, H, hd, ff = 4096, 32, 128, 11008
    g = torch.Generator(device=dev).manual_seed(0)

    def W(o, i):
        return (0.02 * torch.randn(o, i, generator=g, device=dev)).to(torch.bfloat16)

    Wqkv, Wo, Wg, Wu, Wd = W(3 * d, d), W(d, d), W(ff, d), W(ff, d), W(d, ff)
    n1 = torch.ones(d, device=dev, dtype=torch.bfloat16)
    n2 = torch.ones(d, device=dev, dtype=torch.bfloat16)

    def rms(x, wt):
        xf = x.float()
        return (xf * torch.rsqrt(xf.pow(2).mean(-1, keepdim=True) + 1e-6)).to(torch.bfloat16) * wt

    def rope_tab(S):
        inv = 1.0 / (10000.0 ** (torch.arange(0, hd, 2, device=dev, dtype=torch.float32) / hd))
        ang = torch.arange(S, device=dev, dtype=torch.float32)[:, None] * inv[None, :]
        return torch.cat([ang.cos()] * 2, 1).to(torch.bfloat16), torch.cat([ang.sin()] * 2, 1).to(torch.bfloat16)

    def rot(x, c, s):
        x1, x2 = x[..., :hd // 2], x[..., hd // 2:]
        return x * c + torch.cat([-x2, x1], -1) * s

    def layer(x, c, s, backend):
        S = x.shape[0]
        qkv = F.linear(rms(x, n1), Wqkv).view(S, 3, H, hd).permute(1, 2, 0, 3).contiguous()  # [3, H, S, hd]
        q, k, v = rot(qkv[0], c, s)[None], rot(qkv[1], c, s)[None], qkv[2][None].contiguous()
        with sdpa_kernel([backend]):
            a = F.scaled_dot_product_attention(q.contiguous(), k.contiguous(), v, is_causal=True)
        x = x + F.linear(a[0].transpose(0, 1).reshape(S, d), Wo)
        h = rms(x, n2)
        return x + F.linear(F.silu(F.linear(h, Wg)) * F.linear(h, Wu), Wd)

    res = {"layer": "random-init 7B-shaped decoder layer: d=4096, 32 heads x 128, SwiGLU 11008, RMSNorm, RoPE, "
                    "causal attention, bf16, batch 1 (PyTorch-ROCm ops, not this library)"}
    backend = None
    for b in (SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION):
        try:
            c, s = rope_tab(64)
            layer(torch.zeros(64, d, device=dev, dtype=torch.bfloat16), c, s, b)
            torch.cuda.synchronize()
            backend = b
            break
        except RuntimeError:
            continue
    if backend is None:
        res["error"] = "no fused SDPA backend available (the bf16 math path is not used here)"
        return res
    res["sdpa_backend"] = str(backend).split(".")[-1]
    # the same layer in this library's kernels (map_decoder_layer), same weights
    import paper_2608_06411_amd as mp
    wl = mp.DecoderWeights(attn_norm=n1, w_qkv=Wqkv, w_o=Wo, ffn_norm=n2, w_gate_up=torch.cat([Wg, Wu]).contiguous(),
                           w_down=Wd, n_heads=H)
    weight_bytes = 2.0 * (4 * d * d + 3 * d * ff + 2 * d)
    ours = {}
    for S in (2944, 224):
        x = (0.5 * torch.randn(S, d, generator=g, device=dev)).to(torch.bfloat16)
        c, s = rope_tab(S)
        tm = _time_steps(torch, dev, lambda: layer(x, c, s, backend), steps, warmup)
        us = 1e3 * tm["ms_per_step"]
        flops = 2.0 * S * d * (3 * d + d + 3 * ff) + 2.0 * S * S * d  # causal attention: half of 4 S^2 d
        res[f"prefill_us_S{S}"] = us
        res[f"achieved_tflops_S{S}"] = flops / (us * 1e-6) / 1e12
        pos = torch.arange(S, device=dev, dtype=torch.int32)
        ws = mp.decoder_workspace(wl, S, dev)
        y = torch.empty_like(x)
        mine = _time_steps(torch, dev, lambda: mp.map_decoder_layer(wl, x, pos, [0, S], out=y, workspace=ws),
                           steps, warmup)
        ref = layer(x, c, s, backend).float()
        upd = (y.float() - x.float()) - (ref - x.float())
        kern = _kernel_table(mp, torch, lambda: mp.map_decoder_layer(wl, x, pos, [0, S], out=y, workspace=ws), steps)
        mus = 1e3 * mine["ms_per_step"]
        ours[f"S{S}"] = {"us": mus, "achieved_tflops": flops / (mus * 1e-6) / 1e12,
                         "hbm_weight_stream_frac": weight_bytes / (mus * 1e-6) / 1e9 / PEAK_HBM,
                         "speedup_vs_pytorch": us / mus,
                         "update_rel_diff_vs_pytorch": float(upd.norm() / (ref - x.float()).norm()),
                         "kernels": kern}
    res["map_decoder_layer"] = ours
    res["prune_us_per_image"] = prune_us
    res["prune_over_layer_prefill_2944"] = prune_us / res["prefill_us_S2944"]
    res["layer_prefill_2944_over_224"] = res["prefill_us_S2944"] / res["prefill_us_S224"]
    # a 32-layer model's prefill, unpruned in PyTorch against pruning plus the
    # pruned prefill in this library's layer (context: the paper's prefill
    # figures also cover the vision encoder, which is not here)
    res["prefill_32_layers_unpruned_pytorch_ms"] = 32 * res["prefill_us_S2944"] / 1e3
    res["prune_plus_prefill_32_layers_pruned_ms"] = (prune_us + 32 * ours["S224"]["us"]) / 1e3
    res["prefill_speedup_32_layers"] = res["prefill_32_layers_unpruned_pytorch_ms"] / \
        res["prune_plus_prefill_32_layers_pruned_ms"]
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llava_next")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-teacher", action="store_true", help="skip the teacher-selection measurement")
    ap.add_argument("--no-configs", action="store_true", help="skip the other workloads' lines")
    ap.add_argument("--no-context", action="store_true", help="skip the decoder-layer context timing")
    ap.add_argument("--no-train", action="store_true", help="skip the training-step measurement")
    ap.add_argument("--percentile-steps", type=int, default=200,
                    help="individually timed steps for the median / p10 / p90 (0: none)")
    ap.add_argument("--no-streams", action="store_true", help="skip the concurrent-stream throughput")
    ap.add_argument("--cold-steps", type=int, default=50,
                    help="individually timed steps after a 512 MiB scratch write each (cold caches; 0: none)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="first run a plain float32 copy kernel over this many MiB (three times), "
                         "the reference dispatch for calibrating HBM byte counters")
    ap.add_argument("--subset", type=int, default=0,
                    help="map_prune's candidate subset: -1 never, 0 automatic (default), n > 0 that many tokens")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the pruning stage is per image with no exchange "
              "between GPUs, so several GPUs would each run the same kernels on their share of "
              "the images (use --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_06411_amd as mp
    from workloads import get_config, make_inputs
    from workloads.configs import SWEEP_K

    cfg = get_config(args.workload)
    x = make_inputs(cfg)
    dev = torch.device("cuda:0")
    d = _upload(mp, torch, dev, x, cfg)
    if args.copy_calibration_mib > 0:
        src = torch.ones(args.copy_calibration_mib << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)  # reads and writes copy_calibration_mib MiB each
        torch.cuda.synchronize()
        del src, dst

    head, out = measure_prune(mp, torch, dev, cfg, x, d, args.steps, args.warmup, subset=args.subset,
                              per_step=args.percentile_steps, workload_key=args.workload, cold=args.cold_steps)
    sumM = int(x["t_off"][-1])
    line = {
        "metric": METRIC, "value": head["value"], "unit": "images/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
        "us_per_image": head["us_per_image"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic (seeded mixture, random-init predictor)",
        "config": {"workload": head["workload"], "global_batch": cfg.B, "seq_len": cfg.N,
                   "parallelism": "single GPU", "subset_tokens": head["subset_tokens"]},
        "wall_s_timed": head["wall_s_timed"], "step_us": head.get("step_us"),
        "step_us_cold": head.get("step_us_cold"), "kernels": head["kernels"],
        "dominant_kernel": head["dominant_kernel"], "roofline": head["roofline"],
        "roofline_mfma": head["roofline_mfma"], "hbm_stages": head["hbm_stages"],
    }
    line["assembly"] = assembly_bench(args, mp, torch, dev, out, d["T"], d["pos_t"], x["t_off"], cfg)
    if not args.no_streams:
        line["concurrent_streams"] = [concurrent_streams(mp, torch, dev, cfg, x, d, args.steps, args.warmup, n)
                                      for n in (2, 3, 4)]
    if not args.no_train:
        line["training_step"] = train_bench(mp, torch, dev, cfg, x, d, min(args.steps, 20), min(args.warmup, 5))
    if not args.no_context:
        line["decoder_layer_context"] = decoder_layer_context(torch, dev, head["us_per_image"])
    if not args.no_teacher:
        line["teacher_selection"] = teacher_bench(args, mp, torch, dev)
    tiny_cfg, tiny_x = get_config("tiny"), None
    if not args.no_configs:
        # the other workloads: a few steps each (their inputs are generated here, so
        # each costs seconds of host time), one object per workload and K
        cfgs = [("tiny", tiny_cfg)] + [(f"sweep_K{k}", get_config("sweep", K=k, K0=k // 2)) for k in SWEEP_K] + \
               [("multiframe", get_config("multiframe"))]
        line["configs"] = {}
        sweep_x = None
        for key, c in cfgs:
            if key.startswith("sweep"):
                sweep_x = sweep_x if sweep_x is not None else make_inputs(c)
                cx = dict(sweep_x, cfg=c)
            else:
                cx = make_inputs(c)
            if key == "tiny":
                tiny_x = cx
            cd = _upload(mp, torch, dev, cx, c)
            r, _ = measure_prune(mp, torch, dev, c, cx, cd, steps=10, warmup=3)
            line["configs"][key] = r
            del cd
            torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        if tiny_x is None:
            tiny_x = make_inputs(tiny_cfg)
        line["cpu_baseline"] = cpu_baseline(x, cfg, tiny_x, tiny_cfg)
    print(json.dumps(line), flush=True)
    # the library holds no HIP object after a timing reset: nothing is left
    # for the runtime's teardown at exit
    mp.timing_reset()


if __name__ == "__main__":
    main()
