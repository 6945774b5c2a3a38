"""Benchmark of the MXFP4 backward hot path on one MI355X.

One step = the MXFP4 backward pass (RHT + stochastic-rounding quantisation of
all four operands, two scaled MXFP4 GEMMs, 16/9g rescale) of every linear layer
of one transformer block. The headline workload is the GPT-6.7B-shaped block:
16384 tokens, hidden 4096, linears QKV 4096->12288, proj 4096->4096, fc1
4096->16384, fc2 16384->4096 (13.19 TFLOP of backward GEMMs per step), g = 64,
dY heavy-tailed with 0.5% of its 32-element blocks scaled x1000
(workloads.CONFIGS["gpt6.7b"]); --config picks another block. The GPT-345M
block (4096 tokens, hidden 1024) is timed the same way as a secondary figure.
Inputs are seeded synthetic tensors, resident in HBM before the timed region.
Consecutive steps rotate through copies of the inputs held in distinct
buffers, at least 512 MB in all, so the 256 MB MALL cannot serve a step's
inputs from the step before (one GPT-6.7B input set is 2.4 GB on its own).

Printed: ONE JSON line with the contract fields, plus
* roofline: the kernel with the largest share of the step, timed per launch
  with HIP events on the stream it runs on (the library's kernel tracing, in a
  second pass of the same steps), against its roofline;
* kernels: per-kernel times, launches and achieved rates from that pass;
* baselines: BF16 (torch.matmul) and FP8 E4M3 (torch._scaled_mm) GEMMs of the
  same two backward products per linear, on the same device;
* cpu_baseline: the CPU oracle timed on a bounded sample of the same work;
* variants: the same step through mx_linear_backward_ex with the options a
  training framework uses (bf16 dX, dW accumulated into an FP32 main gradient,
  the bias gradient db).

--rht-overhead instead times the RHT overhead study of Sec. 4.2: C = A B^T at
(m, n, k) = (32768, 8192, 8192) and (16384, 28672, 28672) with both operands
quantised along k in every quantiser mode, with BF16 and FP8 baselines.
"""

import argparse
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

DEFAULT_CONFIG = "gpt6.7b"
SECONDARY_CONFIG = "gpt345m"
METRIC = "MXFP4 backward-GEMM TFLOP/s incl. RHT+SR quantize; quantize GB/s; % of peak"
HBM_PEAK_GBS = 8000.0
MXFP4_PEAK_TFLOPS = 10100.0
# Vector ALU issue peak: 256 CUs x 4 SIMDs x 16 lanes per clock x 2.4 GHz, in
# 32-bit lane operations per second (packed FP32 would double it; the library
# uses none).
VALU_PEAK_LANE_OPS = 256 * 4 * 16 * 2.4e9
QUANT_BYTES_PER_ELEM = 2.0 + 0.5 + 1.0 / 32.0     # bf16 in, two codes per byte, one scale per 32
SEED = 0x0345_0000_0000_0000
# HBM bytes per launch measured with rocprofv3 FETCH_SIZE / WRITE_SIZE passes of
# this benchmark (scaled by a copy of known size), with the hash of the kernel
# sources they were measured on; one file per workload.
def traffic_file(config):
    return os.path.join(ROOT, "profiles", f"hbm_traffic_{config}.json")


def kernel_source_hash():
    """Hash of every HIP source and header of the library."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2502_20586_amd", "csrc")
    for f in sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.h"))):
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_counter(config, kernel, key):
    """A per-launch counter figure of `kernel` (`hbm_bytes_per_launch`,
    `valu_insts_per_launch`) from the committed counter summary of `config`, or
    None if there is none or the kernels have changed since it was taken."""
    try:
        with open(traffic_file(config)) as fh:
            d = json.load(fh)
    except (OSError, ValueError):
        return None
    if d.get("source_hash") != kernel_source_hash():
        return None
    k = d.get("kernels", {}).get(kernel)
    return None if k is None else k.get(key)


def measured_traffic(config, kernel):
    return measured_counter(config, kernel, "hbm_bytes_per_launch")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--config", default=DEFAULT_CONFIG, choices=["gpt6.7b", "gpt1.3b", "gpt345m", "tiny"],
                    help="block whose backward is the headline step (default %(default)s)")
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the secondary GPT-345M step timing")
    ap.add_argument("--steps", type=int, default=100)
    # Default warm-up: as many steps as fill WARMUP_S seconds (at least 20). The
    # GPU's clocks take about half a second of load to settle: with 20 warm-up
    # steps (4 ms) the GPT-345M step timed 6% slower and twice as spread out.
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed warm-up steps (default: enough to fill %.1f s, at least 20)" % WARMUP_S)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the MFMA-ceiling measurement (FP4 MFMAs from registers) beside the GEMM roofline")
    ap.add_argument("--no-baselines", action="store_true", help="skip the BF16 / FP8 GEMM baselines")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the framework-option variants (profiles of the headline step alone)")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of CPU oracle work")
    ap.add_argument("--calib-copy", action="store_true",
                    help="after the timed region, one plain 256 MiB device copy (scale for HBM byte counters)")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the step: standalone quantiser and GEMM throughput sweep")
    ap.add_argument("--write-traffic", nargs="+", metavar="CSV",
                    help="write profiles/hbm_traffic_<config>.json from the counter_collection.csv files of a "
                         "rocprofv3 --pmc FETCH_SIZE run and a --pmc WRITE_SIZE run of this benchmark with "
                         "--calib-copy, then exit")
    ap.add_argument("--rht-overhead", action="store_true",
                    help="RHT overhead study: GEMMs at the paper's 7B / 70B shapes in every quantiser mode")
    ap.add_argument("--rht-variance", action="store_true",
                    help="variance of the SR inner-product estimator with and without the RHT (the figure of "
                         "Sec. 3.2) and the flush-to-zero statistic, through the HIP path")
    ap.add_argument("--co-schedule", action="store_true",
                    help="two independent block backwards (--config, default GPT-6.7B) on one stream and on two "
                         "streams")
    ap.add_argument("--configs", action="store_true",
                    help="instead of the step: GPT-1.3B (every g) and GPT-6.7B block backward end to end, "
                         "with BF16 / FP8 GEMM baselines on the same shapes")
    return ap.parse_args()


class Layer:
    def __init__(self, torch, name, fin, fout, dy, x, w):
        self.name, self.fin, self.fout = name, fin, fout
        dev = "cuda"
        self.t = dy.shape[0]
        self.dy = torch.from_numpy(dy.view(np.int16)).to(dev)
        self.x = torch.from_numpy(x.view(np.int16)).to(dev)
        self.w = torch.from_numpy(w.view(np.int16)).to(dev)
        self.dx = torch.empty((self.t, fin), dtype=torch.float32, device=dev)
        self.dw = torch.empty((fout, fin), dtype=torch.float32, device=dev)

    def flops(self):
        return 4 * self.t * self.fin * self.fout

    def quant_elements(self):
        """Elements of the four quantised operands: dY twice (along out and along
        the tokens), W and x once each."""
        return 2 * self.t * self.fout + self.fin * self.fout + self.fin * self.t


def gemm_attainable(layers, gemm_ms_per_step):
    """The GEMMs' attainable time per step: for each backward GEMM (dX: M, N, K =
    T, in, out; dW: out, in, T) the larger of its MFMA time at the MXFP4 peak and
    its HBM time at 8 TB/s for its algorithmic bytes (MXFP4 operands at 0.53125 B
    per element, FP32 output written once), summed over the step; `frac` is that
    over the measured GEMM time."""
    us, n_hbm, n_mfma = 0.0, 0, 0
    for L in layers:
        for m, n, k in ((L.t, L.fin, L.fout), (L.fout, L.fin, L.t)):
            t_mfma = 2.0 * m * n * k / (MXFP4_PEAK_TFLOPS * 1e12)
            t_hbm = ((m + n) * k * 0.53125 + 4.0 * m * n) / (HBM_PEAK_GBS * 1e9)
            us += max(t_mfma, t_hbm) * 1e6
            n_hbm += t_hbm > t_mfma
            n_mfma += t_hbm <= t_mfma
    return {"us_per_step": us, "frac": us / (gemm_ms_per_step * 1e3), "mfma_bound_gemms": n_mfma,
            "hbm_bound_gemms": n_hbm}


def step(mx, layers, g):
    for L in layers:
        mx.mx_linear_backward(L.dy, L.x, L.w, L.dx, L.dw, g, SEED)


# Seconds of untimed steps before timing when --warmup is not given.
WARMUP_S = 0.5


def warm_up(torch, run_step, min_steps=20, seconds=WARMUP_S):
    """Runs steps until `seconds` of wall time and `min_steps` steps have passed;
    returns the number of steps run."""
    n, t0 = 0, time.perf_counter()
    while n < min_steps or time.perf_counter() - t0 < seconds:
        for _ in range(10):
            run_step(n)
            n += 1
        torch.cuda.synchronize()
    return n


# Bytes of distinct inputs the timed steps rotate through: twice the MALL.
ROTATION_BYTES = 512 << 20


def input_sets(layers):
    """The layers and copies of them whose inputs (dY, x, W) live in distinct
    device buffers (outputs are shared), enough that all sets together hold at
    least ROTATION_BYTES of inputs."""
    per_set = sum((L.dy.numel() + L.x.numel() + L.w.numel()) * 2 for L in layers)
    n = max(1, -(-ROTATION_BYTES // per_set))
    sets = [layers]
    for _ in range(n - 1):
        copy = []
        for L in layers:
            c = Layer.__new__(Layer)
            c.__dict__.update(L.__dict__)
            c.dy, c.x, c.w = L.dy.clone(), L.x.clone(), L.w.clone()
            copy.append(c)
        sets.append(copy)
    return sets, per_set


def step_ex(torch, mx, layers, g, flags, with_db, mode=None):
    """The step through mx_linear_backward_ex (bf16 dX buffers, db buffers made
    on first use; dW is accumulated into when flags say so), in quantiser mode
    `mode` (default: the method, MX_MODE_RHT_SR)."""
    mode = mx.MX_MODE_RHT_SR if mode is None else mode
    for L in layers:
        if not hasattr(L, "dx16"):
            L.dx16 = torch.empty((L.t, L.fin), dtype=torch.int16, device="cuda")
            L.db = torch.zeros(L.fout, dtype=torch.float32, device="cuda")
        dx = L.dx16 if flags & mx.MX_BWD_DX_BF16 else L.dx
        mx.mx_linear_backward_ex(L.dy, L.x, L.w, dx, L.dw, L.db if with_db else None, g, SEED, mode, flags)


def variants(torch, mx, sets, g, steps, warmup, rounds=3):
    """ms per step of the framework options next to the plain step: every
    round times each kind for `steps` steps, in turn, and the median over the
    rounds is reported, so that clock drift does not favour any kind. Steps
    rotate through the input sets as the headline step does."""
    bf, acc = mx.MX_BWD_DX_BF16, mx.MX_BWD_ACCUMULATE
    # (name, flags, db, mode): the framework options, and the method with the
    # cheaper 8-bit dither (a different rounding rule, reported beside it)
    kinds = (("plain", None, False, None), ("ex_no_options", 0, False, None), ("bf16_dx", bf, False, None),
             ("bias_grad", 0, True, None), ("bf16_dx_accumulate_bias_grad", bf | acc, True, None),
             ("rht_sr8_noise", 0, False, mx.MX_MODE_RHT_SR8))

    def run(flags, with_db, mode, n):
        for i in range(n):
            layers = sets[i % len(sets)]
            if flags is None:
                step(mx, layers, g)
            else:
                step_ex(torch, mx, layers, g, flags, with_db, mode)

    for _, flags, with_db, mode in kinds:
        run(flags, with_db, mode, warmup)
    times = {name: [] for name, _, _, _ in kinds}
    for _ in range(rounds):
        for name, flags, with_db, mode in kinds:
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            run(flags, with_db, mode, steps)
            e1.record()
            torch.cuda.synchronize()
            times[name].append(e0.elapsed_time(e1) / steps)
    return {name: {"ms_per_step": float(np.median(t)), "rounds": t} for name, t in times.items()}


def rht_overhead(torch, mx, reps=10):
    """Sec. 4.2's RHT overhead estimate redone on MXFP4: C = A B^T with A [n, k]
    and B [m, k] quantised along k in each quantiser mode (no RHT and nearest
    rounding; SR; RHT + nearest; RHT + SR, the method), then one MXFP4 GEMM,
    through the public entry points (row-major operands). Baselines: BF16 GEMM,
    FP8 E4M3 GEMM (operands cast beforehand, and with torch's eager casts), and
    FP8 with an unfused RHT in torch (a bf16 GEMM with H_64 per 64-block, then the
    cast)."""
    import workloads
    cfg = workloads.RHT_OVERHEAD
    g = cfg["g"]
    modes = (("nr", mx.MX_MODE_NR), ("sr", mx.MX_MODE_SR), ("rht_nr", mx.MX_MODE_RHT_NR),
             ("rht_sr", mx.MX_MODE_RHT_SR))
    res = []

    def timed(fn):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    for si, (m, n, k) in enumerate(cfg["shapes"]):
        gen = torch.Generator(device="cuda").manual_seed(cfg["data_seed"] * 100 + si)
        a = torch.randn((n, k), device="cuda", generator=gen).to(torch.bfloat16)
        b = torch.randn((m, k), device="cuda", generator=gen).to(torch.bfloat16)
        ac = torch.empty((n, k // 2), dtype=torch.uint8, device="cuda")
        asc = torch.empty((n, k // 32), dtype=torch.uint8, device="cuda")
        bc = torch.empty((m, k // 2), dtype=torch.uint8, device="cuda")
        bsc = torch.empty((m, k // 32), dtype=torch.uint8, device="cuda")
        c = torch.empty((n, m), dtype=torch.float32, device="cuda")
        flops = 2.0 * m * n * k
        row = {"m": m, "n": n, "k": k, "g": g, "modes": {}}
        ab, bb = a.view(torch.int16), b.view(torch.int16)
        for name, mode in modes:
            def quant(mode=mode):
                mx.mx_quantize(ab, ac, asc, g, 0x0006_0000_0000_0000, mode)
                mx.mx_quantize(bb, bc, bsc, g, 0x0006_0000_0000_0001, mode)
            def full(quant=quant):
                quant()
                mx.mx_gemm_f4(ac, asc, bc, bsc, c)
            q_ms = timed(quant)
            t_ms = timed(full)
            row["modes"][name] = {"ms": t_ms, "quant_ms": q_ms, "tflops": flops / (t_ms * 1e-3) / 1e12}
        gemm_ms = timed(lambda: mx.mx_gemm_f4(ac, asc, bc, bsc, c))
        row["mxfp4_gemm_ms"] = gemm_ms
        md = row["modes"]
        row["overhead"] = {
            "rht_vs_sr": md["rht_sr"]["ms"] / md["sr"]["ms"] - 1.0,
            "rht_sr_vs_nr": md["rht_sr"]["ms"] / md["nr"]["ms"] - 1.0,
            "rht_sr_vs_gemm_alone": md["rht_sr"]["ms"] / gemm_ms - 1.0,
        }
        del c
        cb = torch.empty((n, m), dtype=torch.bfloat16, device="cuda")
        bt = b.t()
        row["bf16_ms"] = timed(lambda: torch.matmul(a, bt, out=cb))
        try:
            f8 = torch.float8_e4m3fn
            one = torch.ones((), device="cuda")
            a8, b8 = a.to(f8), b.to(f8)
            row["fp8_gemm_ms"] = timed(lambda: torch._scaled_mm(a8, b8.t(), scale_a=one, scale_b=one,
                                                                out_dtype=torch.bfloat16))
            def fp8_cast():
                torch._scaled_mm(a.to(f8), b.to(f8).t(), scale_a=one, scale_b=one, out_dtype=torch.bfloat16)
            row["fp8_with_cast_ms"] = timed(fp8_cast)
            sign = torch.ones(g, device="cuda")
            sign[torch.randperm(g, generator=torch.Generator().manual_seed(1))[: g // 2]] = -1
            hmat = torch.ones((1, 1), device="cuda")
            while hmat.shape[0] < g:
                hmat = torch.cat([torch.cat([hmat, hmat], 1), torch.cat([hmat, -hmat], 1)], 0)
            hs = (sign[:, None] * hmat / g ** 0.5).to(torch.bfloat16)   # diag(S) H / sqrt(g)
            def fp8_rht():
                ar = torch.matmul(a.view(-1, g), hs).view(n, k).to(f8)
                br = torch.matmul(b.view(-1, g), hs).view(m, k).to(f8)
                torch._scaled_mm(ar, br.t(), scale_a=one, scale_b=one, out_dtype=torch.bfloat16)
            row["fp8_rht_unfused_ms"] = timed(fp8_rht)
            row["fp8_rht_overhead_unfused"] = row["fp8_rht_unfused_ms"] / row["fp8_with_cast_ms"] - 1.0
            del a8, b8
        except Exception as e:  # report, do not hide
            row["fp8_error"] = repr(e)[:200]
        del cb
        res.append(row)
        print(f"[rht] (m,n,k)=({m},{n},{k}): " + ", ".join(f"{kk} {v['ms']:.3f} ms" for kk, v in md.items())
              + f"; gemm {gemm_ms:.3f} ms; RHT vs SR {100 * row['overhead']['rht_vs_sr']:.1f}%",
              file=sys.stderr, flush=True)
        del a, b, ac, asc, bc, bsc
        torch.cuda.empty_cache()
    return res


def rht_variance(torch, mx, draws=64, oracle_rows=256):
    """The variance study of Sec. 3.2 (its figure) through the HIP path, and
    the flush-to-zero statistic of Sec. 4.1.

    Variance: for every sample length b and outlier rate p, n = 4096 sample
    pairs A_i, B_i (rows of [n, b] matrices, workloads.mixture_vectors) are
    quantised by mx_quantize with `draws` independent noise draws (one sign
    vector), without the RHT (SR) and with it (RHT + SR, g = b up to 256, the
    blockwise g = 256 beyond), and multiplied by mx_gemm_f4; the diagonal of
    alpha C is the estimate alpha Q(A_i)^T Q(B_i) of A_i^T B_i. Reported: its
    sample variance over the draws, averaged over the rows, per mode, and the
    ratio SR / RHT + SR; beside it the oracle's exact variance (closed form
    from the rounding rule) averaged over the first `oracle_rows` rows, with
    the GPU's average over the same rows. Also the fraction of zero codes.

    Flush to zero: the GPT-6.7B QKV output gradient dY (heavy-tailed, with
    x1000 block outliers) quantised in each mode; fraction of its nonzero
    elements whose code is 0 (with the RHT: of all elements, the transformed
    values being nonzero)."""
    import oracle
    import workloads
    cfg = workloads.FIG2
    n = cfg["n"]
    rows = []
    modes = (("sr", mx.MX_MODE_SR, False), ("rht_sr", mx.MX_MODE_RHT_SR, True))
    for b in cfg["b"]:
        g = min(b, 256)
        for p in cfg["p"]:
            a_bits = workloads.mixture_vectors(n, b, p, [cfg["data_seed"], b, int(p * 1000), 0], cfg["outlier_var"])
            b_bits = workloads.mixture_vectors(n, b, p, [cfg["data_seed"], b, int(p * 1000), 1], cfg["outlier_var"])
            da = torch.from_numpy(a_bits.view(np.int16)).cuda()
            db = torch.from_numpy(b_bits.view(np.int16)).cuda()
            ac = torch.empty((n, b // 2), dtype=torch.uint8, device="cuda")
            asc = torch.empty((n, b // 32), dtype=torch.uint8, device="cuda")
            bc, bsc = torch.empty_like(ac), torch.empty_like(asc)
            c = torch.empty((n, n), dtype=torch.float32, device="cuda")
            hi = 0x0F26_0000_0000_0000 | (b << 32)
            row = {"b": b, "p": p, "g": g, "n": n, "draws": draws}
            for name, mode, rht in modes:
                est = torch.empty((draws, n), dtype=torch.float64, device="cuda")
                zeros = torch.zeros((), dtype=torch.float64, device="cuda")
                for d in range(draws):
                    mx.mx_quantize(da, ac, asc, g, hi | (2 * d), mode)
                    mx.mx_quantize(db, bc, bsc, g, hi | (2 * d + 1), mode)
                    mx.mx_gemm_f4(ac, asc, bc, bsc, c)
                    est[d] = torch.diagonal(c).double()
                    zeros += (((ac & 7) == 0).sum() + (((ac >> 4) & 7) == 0).sum()).double()
                est *= oracle.estimator_alpha(g, rht)
                var = est.var(dim=0).cpu().numpy()
                exact = oracle.inner_product_variance(a_bits[:oracle_rows], b_bits[:oracle_rows], g, hi, hi | 1, rht)
                row[name] = {"mean_var": float(var.mean()), "mean_var_first_rows": float(var[:oracle_rows].mean()),
                             "oracle_mean_var_first_rows": float(exact.mean()),
                             "zero_code_frac": float(zeros.item()) / (draws * n * b)}
            row["ratio_sr_over_rht"] = row["sr"]["mean_var"] / row["rht_sr"]["mean_var"]
            rows.append(row)
            print(f"[var] b={b} p={p}: SR {row['sr']['mean_var']:.4g} (oracle {row['sr']['oracle_mean_var_first_rows']:.4g}"
                  f" vs {row['sr']['mean_var_first_rows']:.4g}), RHT+SR {row['rht_sr']['mean_var']:.4g} (oracle "
                  f"{row['rht_sr']['oracle_mean_var_first_rows']:.4g} vs {row['rht_sr']['mean_var_first_rows']:.4g}), "
                  f"ratio {row['ratio_sr_over_rht']:.2f}", file=sys.stderr, flush=True)
            del da, db, ac, asc, bc, bsc, c
    # flush to zero on a GPT-6.7B output gradient
    dy, _, _ = workloads.linear_inputs("gpt6.7b", "qkv")
    t, fout = dy.shape
    ddy = torch.from_numpy(dy.view(np.int16)).cuda()
    nz = int(np.count_nonzero(dy & 0x7FFF))
    codes = torch.empty((t, fout // 2), dtype=torch.uint8, device="cuda")
    scales = torch.empty((t, fout // 32), dtype=torch.uint8, device="cuda")
    nonzero_in = torch.from_numpy(((dy & 0x7FFF) != 0).view(np.uint8)).cuda().view(t, fout // 2, 2)
    flush = {"tensor": "gpt6.7b qkv dY [16384, 12288]", "nonzero_elements": nz}
    for name, mode, rht in (("nr", mx.MX_MODE_NR, False), ("sr", mx.MX_MODE_SR, False),
                            ("rht_nr", mx.MX_MODE_RHT_NR, True), ("rht_sr", mx.MX_MODE_RHT_SR, True)):
        mx.mx_quantize(ddy, codes, scales, 64, 0x0F27_0000_0000_0000, mode)
        z = torch.stack([(codes & 7) == 0, ((codes >> 4) & 7) == 0], dim=-1)
        if rht:
            frac = float(z.sum().item()) / (t * fout)
        else:
            frac = float((z & nonzero_in.bool()).sum().item()) / nz
        flush[name] = frac
    # oracle's expected flush fraction (SR modes) on the first rows
    ids = np.arange(256)
    for name, rht in (("sr", False), ("rht_sr", True)):
        _, _, pz = oracle.sr_moments(dy[ids], 64, 0x0F27_0000_0000_0000, rht)
        mask = np.ones_like(pz, dtype=bool) if rht else (dy[ids] & 0x7FFF) != 0
        flush[name + "_oracle_first_256_rows"] = float(pz[mask].sum() / mask.sum())
    print(f"[var] flush to zero: {flush}", file=sys.stderr, flush=True)
    return {"variance": rows, "flush_to_zero": flush}


def co_schedule(torch, mx, config="gpt6.7b", reps=None, rounds=3):
    """Two independent block backwards (two micro-batches' worth of inputs and
    outputs; GPT-6.7B unless --config names another block), run back to back
    on one stream and concurrently on two streams of the same priority, the
    second stream taking the linears in reverse order so that its quantiser
    launches tend to meet the first stream's GEMM launches. A 256 x 256 GEMM
    workgroup holds a whole SIMD's registers (one wave per SIMD), so at
    GPT-6.7B the two kernels cannot share a CU: any gain comes from the
    hardware filling CUs that one launch leaves idle (launch tails, the tiles'
    synchronised store bursts) with the other stream's work. Smaller blocks
    run the 128 x 128 kernel (two workgroups per CU) and shorter launches."""
    cfg, layers = load_layers(torch, config)
    g = cfg["g"][0]
    if reps is None:   # about 40 ms or more per timed run
        reps = 10 if config == "gpt6.7b" else 100
    other = []
    for L in layers:
        c = Layer.__new__(Layer)
        c.__dict__.update(L.__dict__)
        c.dy, c.x, c.w = L.dy.clone(), L.x.clone(), L.w.clone()
        c.dx, c.dw = torch.empty_like(L.dx), torch.empty_like(L.dw)
        other.append(c)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()

    def run(seq_a, seq_b, n):
        cur = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(cur)
        sa.wait_stream(cur)
        sb.wait_stream(cur)
        for _ in range(n):
            for s, seq in ((sa, seq_a), (sb, seq_b)):
                for L in seq:
                    mx.mx_linear_backward(L.dy, L.x, L.w, L.dx, L.dw, g, SEED, stream=s)
        cur.wait_stream(sa)
        cur.wait_stream(sb)
        e1.record(cur)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    cases = {"one_stream": (layers + other, []), "two_streams_same_order": (layers, other),
             "two_streams_reversed": (layers, other[::-1])}
    for a, b in cases.values():
        run(a, b, max(3, reps // 2))
    times = {k: [] for k in cases}
    for _ in range(rounds):
        for k, (a, b) in cases.items():
            times[k].append(run(a, b, reps))
    med = {k: sorted(v)[len(v) // 2] for k, v in times.items()}
    for s in (sa, sb):
        mx.mx_release_workspace(s)
    hidden = layers[0].fin
    return {"workload": f"two {config} block backwards (T={cfg['tokens']}, hidden {hidden}, g={g}), "
                        "independent inputs",
            "ms_per_two_blocks": {k: round(v, 4) for k, v in med.items()},
            "all_rounds_ms": {k: [round(t, 4) for t in v] for k, v in times.items()},
            "gain_vs_one_stream": {k: round(med["one_stream"] / v - 1, 4) for k, v in med.items()
                                   if k != "one_stream"}}


def gemm_baselines(torch, layers, reps=10):
    """BF16 and FP8 (E4M3, per-tensor scales) GEMMs for dX = dY W and dW = dY^T x."""
    out = {}
    mats = []
    for L in layers:
        dyb = L.dy.view(torch.bfloat16)
        xb = L.x.view(torch.bfloat16)
        wb = L.w.view(torch.bfloat16)
        mats.append((dyb, wb.contiguous(), dyb.t().contiguous(), xb))
    flops = sum(L.flops() for L in layers)

    def timed(fn):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    def bf16():
        for a, b, at, x in mats:
            torch.matmul(a, b)
            torch.matmul(at, x)
    ms = timed(bf16)
    out["bf16"] = {"ms_per_step": ms, "tflops": flops / (ms * 1e-3) / 1e12}
    try:
        f8 = torch.float8_e4m3fn
        one = torch.ones((), device="cuda")
        def cast():
            # _scaled_mm wants A row-major and B column-major: pass B^T's storage transposed.
            return [(a.to(f8), b.t().contiguous().to(f8).t(), at.to(f8), x.t().contiguous().to(f8).t())
                    for a, b, at, x in mats]
        pre = cast()
        def fp8():
            for a, b, at, x in pre:
                torch._scaled_mm(a, b, scale_a=one, scale_b=one, out_dtype=torch.bfloat16)
                torch._scaled_mm(at, x, scale_a=one, scale_b=one, out_dtype=torch.bfloat16)
        ms = timed(fp8)
        cast_ms = timed(cast)
        out["fp8_e4m3"] = {"ms_per_step": ms, "tflops": flops / (ms * 1e-3) / 1e12,
                           "note": "GEMMs only; operands cast to E4M3 beforehand; bf16 outputs"}

        def fp8_f32():
            for a, b, at, x in pre:
                torch._scaled_mm(a, b, scale_a=one, scale_b=one, out_dtype=torch.float32)
                torch._scaled_mm(at, x, scale_a=one, scale_b=one, out_dtype=torch.float32)
        try:
            ms32 = timed(fp8_f32)
            out["fp8_e4m3_f32_out"] = {"ms_per_step": ms32, "tflops": flops / (ms32 * 1e-3) / 1e12,
                                       "note": "GEMMs only, FP32 dX and dW as the MXFP4 step writes them"}
        except Exception as e:  # report, do not hide
            out["fp8_e4m3_f32_out"] = {"error": repr(e)[:200]}
        out["fp8_e4m3_with_cast"] = {
            "ms_per_step": ms + cast_ms, "cast_ms": cast_ms, "tflops": flops / ((ms + cast_ms) * 1e-3) / 1e12,
            "note": "GEMMs plus torch's eager bf16 -> E4M3 operand preparation (dY, W^T, dY^T, x^T as "
                    "separate transpose and convert kernels; per-tensor scale 1, no amax pass)"}
        # The same casts at the HBM peak: 2 bytes read and 1 written per operand element.
        cast_bytes = sum(3.0 * (a.numel() + b.numel() + at.numel() + x.numel()) for a, b, at, x in mats)
        bound_ms = ms + cast_bytes / (HBM_PEAK_GBS * 1e9) * 1e3
        out["fp8_e4m3_cast_bound"] = {
            "ms_per_step": bound_ms, "cast_bytes": cast_bytes, "tflops": flops / (bound_ms * 1e-3) / 1e12,
            "note": "measured FP8 GEMMs plus the operand casts' bytes at 8 TB/s: a lower bound on an FP8 "
                    "backward that starts from bf16"}
    except Exception as e:  # report, do not hide
        out["fp8_e4m3"] = {"error": repr(e)[:200]}
    return out


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        return 1


def cpu_oracle_full(config, linears=None):
    """The oracle's Algorithm 3 (oracle.linear_backward: all four operands
    quantised whole, both GEMMs in FP64) timed in full on the named linears of a
    config (all of them by default)."""
    import oracle
    import workloads
    cfg = workloads.CONFIGS[config]
    t, g = cfg["tokens"], cfg["g"][0]
    secs, flops, elems, names = 0.0, 0, 0, []
    for name, fin, fout in cfg["linears"]:
        if linears and name not in linears:
            continue
        dy, x, w = workloads.linear_inputs(config, name)
        t0 = time.perf_counter()
        oracle.linear_backward(dy, x, w, g, SEED)
        secs += time.perf_counter() - t0
        flops += 4 * t * fin * fout
        elems += 2 * t * fout + fin * fout + fin * t
        names.append(name)
    return {"config": config, "linears": names, "seconds": secs, "gemm_flops": flops, "quant_elems": elems,
            "value": flops / secs / 1e12, "unit": "TFLOP/s"}


def cpu_baseline(config, budget_s):
    """The CPU oracle timed on this machine's host cores.

    * In full: the tiny single-linear config (256 tokens, 256 x 256) and the
      QKV linear of the GPT-345M block.
    * Sampled, for the headline block (whose oracle step runs for most of an
      hour): per linear, the oracle quantises whole rows of each of the four
      operands -- 64 logical rows of dY and dY^T, 256 of W^T and x^T per pass
      (quantisation is row-local, so a row sample is exact work) -- and
      multiplies the sampled rows of both GEMMs in FP64. Passes take the next
      rows (wrapping around) until about `budget_s` seconds of CPU work have
      run, the two full runs included. The step time is the measured
      per-element quantise time times the step's elements plus the measured
      per-FLOP GEMM time times its FLOPs. The skinny sampled GEMMs run BLAS
      below its full-size rate, so this estimate errs towards a slower
      oracle."""
    import oracle
    import workloads
    threads = _blas_threads()
    start = time.perf_counter()
    full = {"tiny": cpu_oracle_full("tiny"), "gpt345m_qkv": cpu_oracle_full("gpt345m", ["qkv"])}
    cfg = workloads.CONFIGS[config]
    t, g = cfg["tokens"], cfg["g"][0]
    q_elems_total = sum(2 * t * fout + fin * fout + fin * t for _, fin, fout in cfg["linears"])
    flops_total = sum(4 * t * fin * fout for _, fin, fout in cfg["linears"])
    q_time, q_elems, g_time, g_flops = 0.0, 0, 0.0, 0
    rows_a, rows_b = 64, 256
    inputs = {}
    passes = 0
    while passes == 0 or time.perf_counter() - start < budget_s:
        for name, fin, fout in cfg["linears"]:
            if name not in inputs:
                inputs[name] = workloads.linear_inputs(config, name)
            dy, x, w = inputs[name]
            # Logical rows of the four operands: dY [T, out], W^T [in, out],
            # dY^T [out, T], x^T [in, T]; a row of a transposed operand is a
            # column of the stored matrix. Pass p takes rows p * rows_a ...
            # (rows_a of dY and dY^T) and p * rows_b ... (rows_b of W^T, x^T).
            ra = (passes * rows_a) % (min(t, fout) - rows_a + 1)
            rb = (passes * rows_b) % (fin - rows_b + 1)
            ops = [(dy[ra:ra + rows_a], ra, 0), (np.ascontiguousarray(w[:, rb:rb + rows_b].T), rb, 1),
                   (np.ascontiguousarray(dy[:, ra:ra + rows_a].T), ra, 2),
                   (np.ascontiguousarray(x[:, rb:rb + rows_b].T), rb, 3)]
            qs = []
            for bits, r0, i in ops:
                ids = np.arange(r0, r0 + bits.shape[0])
                t0 = time.perf_counter()
                qs.append(oracle.quantize_rht_sr(bits, g, SEED ^ i, row_ids=ids))
                q_time += time.perf_counter() - t0
                q_elems += bits.size
            for a, b in ((qs[0], qs[1]), (qs[2], qs[3])):
                t0 = time.perf_counter()
                oracle.gemm_f64(a[0], a[1], b[0], b[1])
                g_time += time.perf_counter() - t0
                g_flops += 2 * a[0].shape[0] * b[0].shape[0] * a[0].shape[1]
        passes += 1
    del inputs
    est_s = q_elems_total * (q_time / q_elems) + flops_total * (g_time / g_flops)
    names = ", ".join(n for n, _, _ in cfg["linears"])
    return {
        "value": flops_total / est_s / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
        "host_cpus": os.cpu_count(),
        "sample": (f"{config} block step, sampled: in {passes} passes over the linears {names}, the oracle "
                   f"quantised {q_elems} elements (whole logical rows, per pass {rows_a} of dY and dY^T and "
                   f"{rows_b} of W^T and x^T) and ran {g_flops:.3g} FLOPs of the FP64 GEMMs on those rows; step "
                   f"time = per-element quantise time x {q_elems_total} elements + per-FLOP GEMM time x "
                   f"{flops_total:.4g} FLOPs = {est_s:.0f} s. Quantiser single-threaded numpy, GEMM BLAS on "
                   f"{threads} threads; {time.perf_counter() - start:.1f} s in all, the full runs and the generation "
                   f"of the sampled linears' inputs included"),
        "quant_elems_per_s": q_elems / q_time, "gemm_flops_per_s": g_flops / g_time, "est_step_s": est_s,
        "passes": passes, "full_runs": full,
    }


def sweep(torch, mx):
    """Standalone throughput: the quantiser on the sweep shapes (row-major and
    transposed reads, g = 64 and 256) and the GEMM on large shapes. Inputs rotate
    through enough distinct buffers (>= 1 GiB) that the 256 MB MALL cannot hold
    them. Returns a dict of results."""
    import workloads
    out = {"quantize": [], "gemm": []}

    def timed(fns, reps):
        for f in fns[:2]:
            f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(reps):
            fns[i % len(fns)]()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    for rows, cols in workloads.QUANT_SWEEP["shapes"]:
        nbuf = max(2, -(-(1 << 30) // (rows * cols * 2)))
        src = [torch.randn((rows, cols), device="cuda", dtype=torch.float32).to(torch.bfloat16).view(torch.int16)
               for _ in range(nbuf)]
        for g in workloads.QUANT_SWEEP["g"]:
            for transposed in (False, True):
                codes = torch.empty((rows, cols // 2), dtype=torch.uint8, device="cuda")
                scales = torch.empty((rows, cols // 32), dtype=torch.uint8, device="cuda")
                if transposed:    # logical [rows, cols] from storage [cols, rows]
                    srcs = [x.view(cols, rows) for x in src]
                    fns = [lambda x=x: mx.mx_rht_sr_quantize_t(x, codes, scales, g, 1) for x in srcs]
                else:
                    fns = [lambda x=x: mx.mx_rht_sr_quantize(x, codes, scales, g, 1) for x in src]
                ms = timed(fns, 20)
                gbs = rows * cols * QUANT_BYTES_PER_ELEM / (ms * 1e-3) / 1e9
                out["quantize"].append({"rows": rows, "cols": cols, "g": g, "transposed": transposed,
                                        "us": ms * 1e3, "gbs": gbs, "hbm_frac": gbs / HBM_PEAK_GBS})
                print(f"[sweep] quant {rows}x{cols} g={g} t={transposed}: {ms*1e3:.1f} us {gbs:.0f} GB/s",
                      file=sys.stderr, flush=True)
        del src
    # A plain device copy of a known size, for scaling HBM byte counters.
    src = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    ms = timed([lambda: dst.copy_(src)], 10)
    out["copy"] = {"bytes_read": src.numel() * 4, "bytes_written": dst.numel() * 4, "us": ms * 1e3,
                   "gbs": 2 * src.numel() * 4 / (ms * 1e-3) / 1e9}
    print(f"[sweep] copy 1 GiB: {ms*1e3:.1f} us {out['copy']['gbs']:.0f} GB/s", file=sys.stderr, flush=True)
    del src, dst
    shapes = [(16384, 4096, 16384), (16384, 16384, 4096), (4096, 16384, 16384), (32768, 8192, 8192),
              (8192, 8192, 8192)]
    for m, n, k in shapes:
        def mxop(rows):
            c = torch.randint(0, 256, (rows, k // 2), dtype=torch.uint8, device="cuda")
            s = torch.randint(120, 134, (rows, k // 32), dtype=torch.uint8, device="cuda")
            return c, s
        a, b = mxop(m), mxop(n)
        cbuf = torch.empty((m, n), dtype=torch.float32, device="cuda")
        ms = timed([lambda: mx.mx_gemm_f4(*a, *b, cbuf)], 10)
        tf = 2 * m * n * k / (ms * 1e-3) / 1e12
        out["gemm"].append({"M": m, "N": n, "K": k, "us": ms * 1e3, "tflops": tf,
                            "mfma_frac": tf / MXFP4_PEAK_TFLOPS})
        print(f"[sweep] gemm {m}x{n}x{k}: {ms*1e3:.1f} us {tf:.0f} TFLOP/s", file=sys.stderr, flush=True)
        del a, b, cbuf
    return out


def config_runs(torch, mx, steps=10, warmup=3):
    """Block backward (all four linears) of the GPT-1.3B config at every g and of
    the GPT-6.7B config, timed like the headline step, with per-kernel times from
    the library's tracing and BF16 / FP8 GEMM baselines on the same shapes."""
    import workloads
    out = {}
    for config in ("gpt1.3b", "gpt6.7b"):
        cfg = workloads.CONFIGS[config]
        t0 = time.perf_counter()
        layers = [Layer(torch, name, fin, fout, *workloads.linear_inputs(config, name))
                  for name, fin, fout in cfg["linears"]]
        torch.cuda.synchronize()
        print(f"[configs] {config}: inputs ready in {time.perf_counter() - t0:.1f} s", file=sys.stderr, flush=True)
        flops = sum(L.flops() for L in layers)
        res = {"tokens": cfg["tokens"], "linears": [[n_, i_, o_] for n_, i_, o_ in cfg["linears"]],
               "gemm_flops_per_step": flops, "quant_elements_per_step": sum(L.quant_elements() for L in layers),
               "by_g": {}}
        # Settle the clocks on this config's step before its first timing.
        warm_up(torch, lambda i: step(mx, layers, cfg["g"][0]), min_steps=warmup)
        for g in cfg["g"]:
            for _ in range(warmup):
                step(mx, layers, g)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(steps):
                step(mx, layers, g)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / steps
            mx.mx_profile_start()
            for _ in range(steps):
                step(mx, layers, g)
            torch.cuda.synchronize()
            prof = mx.mx_profile_stop()
            q_ms = sum(v["total_ms"] for k, v in prof.items() if k.startswith("quant")) / steps
            # algorithmic bytes as the library counts them (each input read once)
            qbytes = sum(v["work"] for k, v in prof.items() if k.startswith("quant")) / steps
            g_ms = sum(v["total_ms"] for k, v in prof.items() if k.startswith("gemm") or k == "splitk_reduce") / steps
            res["by_g"][str(g)] = {
                "ms_per_step": ms, "tflops": flops / (ms * 1e-3) / 1e12,
                "quant_ms": q_ms, "quant_bytes_per_step": qbytes, "quant_gbs": qbytes / (q_ms * 1e-3) / 1e9,
                "gemm_ms": g_ms, "gemm_tflops": flops / (g_ms * 1e-3) / 1e12,
                "kernels": {k: {"avg_us": v["total_ms"] * 1e3 / v["launches"], "launches_per_step": v["launches"] / steps}
                            for k, v in prof.items()}}
            print(f"[configs] {config} g={g}: {ms:.3f} ms/step {flops / (ms * 1e-3) / 1e12:.0f} TFLOP/s "
                  f"(quantise {q_ms:.3f} ms, GEMMs {g_ms:.3f} ms)", file=sys.stderr, flush=True)
        g0 = "64" if "64" in res["by_g"] else next(iter(res["by_g"]))
        # One input set holds more than twice the MALL at these sizes.
        res["variants_g" + g0] = variants(torch, mx, [layers], int(g0), steps, warmup)
        print(f"[configs] {config} g={g0} options: " + ", ".join(
            f"{k} {v['ms_per_step']:.3f} ms" for k, v in res["variants_g" + g0].items()), file=sys.stderr, flush=True)
        base = gemm_baselines(torch, layers, reps=5)
        res["baselines"] = base
        ms0 = res["by_g"][g0]["ms_per_step"]
        for name, b in base.items():
            if "ms_per_step" in b:
                res[f"speedup_vs_{name}_g{g0}"] = b["ms_per_step"] / ms0
        print(f"[configs] {config} baselines: " + ", ".join(
            f"{k} {v.get('ms_per_step', float('nan')):.3f} ms" for k, v in base.items()), file=sys.stderr, flush=True)
        out[config] = res
        del layers
        torch.cuda.empty_cache()
    return out


KERNEL_TAGS = (("quant_kernel<64", "quant_g64"), ("gemm_ring_kernel<128", "gemm_128x128r"),
               ("gemm_ring_kernel<256", "gemm_256x256"), ("gemm_f4_kernel", "gemm_128x128"),
               ("reduce_splits", "splitk_reduce"), ("colsum_reduce", "colsum_reduce"))


def _kernel_key(name):
    for tag, short in KERNEL_TAGS:
        if tag in name:
            return short
    return None


def write_traffic(config, fetch_csv, write_csv, *sq_csvs):
    """HBM bytes per launch of each library kernel from two rocprofv3 counter
    passes. Each counter is scaled by the ratio of the true bytes of the plain
    256 MiB device copy that --calib-copy appends to what the counter reads for
    that copy (FETCH_SIZE and WRITE_SIZE are in KiB). Further passes (SQ / GRBM
    counters such as SQ_INSTS_VALU, SQ_INSTS_MFMA, SQ_VALU_MFMA_BUSY_CYCLES,
    SQ_BUSY_CYCLES, GRBM_GUI_ACTIVE) are averaged per launch as they are."""
    import csv
    copy_bytes = float(1 << 28)

    def per_kernel(path, counter=None, need_copy=True):
        sums, counts, copy = {}, {}, []
        for r in csv.DictReader(open(path)):
            if counter is not None and r["Counter_Name"] != counter:
                continue
            name, v = r["Kernel_Name"], float(r["Counter_Value"])
            if "copyBuffer" in name:
                copy.append(v)
                continue
            key = _kernel_key(name)
            if key:
                k2 = key if counter is not None else (key, r["Counter_Name"])
                # one row per dispatch and counter
                sums[k2] = sums.get(k2, 0.0) + v
                counts[k2] = counts.get(k2, 0) + 1
        if not need_copy:
            return {k: (sums[k] / counts[k], counts[k]) for k in sums}, 1.0
        if not copy:
            raise SystemExit(f"{path}: no copy kernel (run the benchmark with --calib-copy)")
        scale = copy_bytes / (max(copy) * 1024.0)
        return {k: (sums[k] / counts[k], counts[k]) for k in sums}, scale

    fetch, fscale = per_kernel(fetch_csv, "FETCH_SIZE")
    write, wscale = per_kernel(write_csv, "WRITE_SIZE")
    kernels = {}
    for k in sorted(set(fetch) & set(write)):
        kernels[k] = {"launches_counted": fetch[k][1], "fetch_kib_per_launch": fetch[k][0],
                      "write_kib_per_launch": write[k][0],
                      "hbm_bytes_per_launch": (fetch[k][0] * fscale + write[k][0] * wscale) * 1024.0}
    for path in sq_csvs:
        extra, _ = per_kernel(path, None, need_copy=False)
        for (k, cname), (v, _n) in extra.items():
            if k in kernels:
                kernels[k].setdefault("counters_per_launch", {})[cname] = v
                if cname == "SQ_INSTS_VALU":
                    kernels[k]["valu_insts_per_launch"] = v
    d = {"config": config, "source_hash": kernel_source_hash(), "fetch_scale": fscale, "write_scale": wscale,
         "kernels": kernels}
    with open(traffic_file(config), "w") as fh:
        json.dump(d, fh, indent=1)
    print(json.dumps(d, indent=1))


def load_layers(torch, config):
    import workloads
    cfg = workloads.CONFIGS[config]
    layers = [Layer(torch, name, fin, fout, *workloads.linear_inputs(config, name))
              for name, fin, fout in cfg["linears"]]
    torch.cuda.synchronize()
    return cfg, layers


def traced(torch, mx, sets, g, steps):
    """Per-kernel times of `steps` steps from the library's kernel tracing (HIP
    events recorded on each launch's own stream)."""
    mx.mx_profile_start()
    for i in range(steps):
        step(mx, sets[i % len(sets)], g)
    torch.cuda.synchronize()
    prof = mx.mx_profile_stop()
    kernels = {}
    for name, st in prof.items():
        d = {"ms_per_step": st["total_ms"] / steps, "launches_per_step": st["launches"] / steps,
             "avg_us": st["total_ms"] * 1e3 / st["launches"]}
        if st["work_is_flops"]:
            d["tflops"] = st["work"] / (st["total_ms"] * 1e-3) / 1e12
        else:
            d["gbs"] = st["work"] / (st["total_ms"] * 1e-3) / 1e9
        kernels[name] = d
    return prof, kernels


def roofline_of(config, prof, kernel, steps):
    """Roofline entry of one traced kernel: its algorithmic work per launch over
    its average launch time, against the MXFP4 MFMA peak (FLOP work) or HBM
    (byte work); traffic from the committed counter summary when its kernel
    sources are current."""
    st = prof[kernel]
    secs = st["total_ms"] * 1e-3
    if st["work_is_flops"]:
        achieved = st["work"] / secs / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": MXFP4_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / MXFP4_PEAK_TFLOPS}
    else:
        achieved = st["work"] / secs / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS}
    roof["traffic"] = measured_traffic(config, kernel)
    roof.update({"kernel": kernel, "launches_per_step": st["launches"] / steps,
                 "avg_us": st["total_ms"] * 1e3 / st["launches"], "per_launch": st["work"] / st["launches"],
                 "work_unit": "FLOP" if st["work_is_flops"] else "byte"})
    return roof


def alu_roofline_of(config, prof, kernel, elems_per_step, steps):
    """The quantiser is bound by vector ALU issue, not HBM: its counted VALU
    wavefront instructions (64 lanes each) per launch over the launch time,
    against the VALU issue peak (None without a current counter summary).
    elems_per_step: quantised elements per step (for the per-element count)."""
    valu = measured_counter(config, kernel, "valu_insts_per_launch")
    if valu is None or kernel not in prof:
        return None
    st = prof[kernel]
    avg_s = st["total_ms"] * 1e-3 / st["launches"]
    lane_ops = valu * 64.0
    r = {"bound": "alu", "kernel": kernel, "achieved": lane_ops / avg_s, "peak": VALU_PEAK_LANE_OPS,
         "unit": "lane-op/s", "frac": lane_ops / avg_s / VALU_PEAK_LANE_OPS, "lane_ops_per_launch": lane_ops}
    if not st["work_is_flops"]:
        r["lane_ops_per_element"] = lane_ops / (elems_per_step * steps / st["launches"])
    return r


def main():
    args = parse()
    if args.write_traffic:
        if len(args.write_traffic) < 2:
            raise SystemExit("--write-traffic FETCH_CSV WRITE_CSV [COUNTER_CSV ...]")
        write_traffic(args.config, *args.write_traffic)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); this build has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2502_20586_amd as mx
    import workloads
    mx.load_library()
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.sweep:
        print(json.dumps({"sweep": sweep(torch, mx)}))
        return
    if args.configs:
        print(json.dumps({"configs": config_runs(torch, mx)}))
        return
    if args.rht_overhead:
        print(json.dumps({"rht_overhead": rht_overhead(torch, mx)}))
        return
    if args.rht_variance:
        print(json.dumps({"rht_variance": rht_variance(torch, mx)}))
        return
    if args.co_schedule:
        print(json.dumps({"co_schedule": co_schedule(torch, mx, args.config)}))
        return
    config = args.config
    t0 = time.perf_counter()
    cfg, layers = load_layers(torch, config)
    g = cfg["g"][0]
    print(f"[bench] inputs ready ({config}, {time.perf_counter() - t0:.1f} s)", file=sys.stderr, flush=True)

    sets, set_bytes = input_sets(layers)
    if args.warmup is None:
        args.warmup = warm_up(torch, lambda i: step(mx, sets[i % len(sets)], g))
    else:
        for i in range(args.warmup):
            step(mx, sets[i % len(sets)], g)
    torch.cuda.synchronize()
    print(f"[bench] warm-up {args.warmup} steps", file=sys.stderr, flush=True)
    # Events between consecutive steps give the per-step spread; the value is
    # the whole timed region over the number of steps.
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    ev[0].record()
    for i in range(args.steps):
        step(mx, sets[i % len(sets)], g)
        ev[i + 1].record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms = ev[0].elapsed_time(ev[-1]) / args.steps
    step_times = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps))
    pct = lambda q: step_times[min(len(step_times) - 1, int(q * len(step_times)))]
    flops = sum(L.flops() for L in layers)
    value = flops / (ms * 1e-3) / 1e12
    print(f"[bench] timed {args.steps} steps: {ms:.4f} ms/step, {value:.0f} TFLOP/s", file=sys.stderr, flush=True)

    # Second pass of the same steps with the library's kernel tracing on.
    prof, kernels = traced(torch, mx, sets, g, args.steps)
    dom = max(prof, key=lambda k: prof[k]["total_ms"])
    roof = roofline_of(config, prof, dom, args.steps)
    quant_ms = sum(v["total_ms"] for k, v in prof.items() if k.startswith("quant"))
    quant_bytes = sum(v["work"] for k, v in prof.items() if k.startswith("quant"))
    gemm_ms = sum(v["total_ms"] for k, v in prof.items() if k.startswith("gemm") or k == "splitk_reduce")
    qk = max((k for k in prof if k.startswith("quant")), key=lambda k: prof[k]["total_ms"], default=None)
    hidden = {"gpt6.7b": 4096, "gpt1.3b": 2048, "gpt345m": 1024, "tiny": 256}[config]
    res = {
        "metric": METRIC, "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "mxfp4", "data": "synthetic",
        "config": {"workload": f"{config}_block_backward", "tokens": cfg["tokens"], "hidden": hidden,
                   "linears": [[n_, i_, o_] for n_, i_, o_ in cfg["linears"]], "g": g,
                   "gemm_flops_per_step": flops, "parallelism": "none"},
        "quantize_gbs": quant_bytes / (quant_ms * 1e-3) / 1e9,
        "quantize_ms_per_step": quant_ms / args.steps,
        "gemm_ms_per_step": gemm_ms / args.steps,
        "gemm_tflops": flops * args.steps / (gemm_ms * 1e-3) / 1e12,
        "gemm_attainable": gemm_attainable(layers, gemm_ms / args.steps),
        "mfma_peak_frac": value / MXFP4_PEAK_TFLOPS,
        "roofline": roof,
        "quantize_roofline": roofline_of(config, prof, qk, args.steps) if qk else None,
        "alu_roofline": alu_roofline_of(config, prof, qk, sum(L.quant_elements() for L in layers), args.steps)
                        if qk else None,
        "kernels": kernels,
        "kernel_source_hash": kernel_source_hash(),
        "wall_s_timed": t_wall,
        "step_ms_p10_p50_p90": [pct(0.1), pct(0.5), pct(0.9)],
        "input_rotation": {"sets": len(sets), "input_bytes_per_set": set_bytes},
    }
    if roof["bound"] == "mfma" and not args.no_ceiling:
        # What the GEMM could reach at best: FP4 MFMAs back to back from
        # registers on every CU, at the clock the chip holds under that load.
        try:
            tf, ghz = mx.mx_measure_mfma_peak()
            res["mfma_ceiling"] = {"tflops": tf, "clock_ghz": ghz,
                                   "what": "FP4 32x32x64 scaled MFMAs from registers, 16 independent tiles per wave, "
                                           "one 4-wave workgroup per CU, no memory traffic"}
            roof["frac_of_mfma_ceiling"] = roof["achieved"] / tf
            print(f"[bench] MFMA ceiling {tf:.0f} TFLOP/s at {ghz:.2f} GHz", file=sys.stderr, flush=True)
        except mx.MxError as e:  # a diagnostic: report it, keep the line
            res["mfma_ceiling"] = {"error": str(e)[:200]}
    if not args.no_variants:
        print("[bench] framework option variants", file=sys.stderr, flush=True)
        res["variants"] = variants(torch, mx, sets, g, max(10, args.steps // 2), min(args.warmup, 10))
    if args.calib_copy:
        src = torch.empty(1 << 26, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        res["calib_copy_bytes"] = {"read": src.numel() * 4, "written": dst.numel() * 4}
        del src, dst
    if not args.no_baselines:
        print("[bench] bf16 / fp8 baselines", file=sys.stderr, flush=True)
        res["baselines"] = gemm_baselines(torch, layers)
        res["speedups"] = {f"vs_{k}": v["ms_per_step"] / ms for k, v in res["baselines"].items()
                           if "ms_per_step" in v}
    del sets, layers
    torch.cuda.empty_cache()
    if not args.no_secondary and config != SECONDARY_CONFIG:
        # The GPT-345M block, timed the same way (its GEMMs are bound by their
        # FP32 output writes, its quantiser launches are short).
        cfg2, layers2 = load_layers(torch, SECONDARY_CONFIG)
        sets2, _ = input_sets(layers2)
        warm_up(torch, lambda i: step(mx, sets2[i % len(sets2)], cfg2["g"][0]), seconds=0.25)
        n2 = max(args.steps, 50)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(n2):
            step(mx, sets2[i % len(sets2)], cfg2["g"][0])
        e1.record()
        torch.cuda.synchronize()
        ms2 = e0.elapsed_time(e1) / n2
        flops2 = sum(L.flops() for L in layers2)
        prof2, kern2 = traced(torch, mx, sets2, cfg2["g"][0], n2)
        gemm_ms2 = sum(v["total_ms"] for k, v in prof2.items() if k.startswith("gemm") or k == "splitk_reduce") / n2
        sec = {"workload": f"{SECONDARY_CONFIG}_block_backward", "steps": n2, "ms_per_step": ms2,
               "tflops": flops2 / (ms2 * 1e-3) / 1e12, "kernels": kern2,
               "gemm_attainable": gemm_attainable(layers2, gemm_ms2)}
        if not args.no_baselines:
            sec["baselines"] = gemm_baselines(torch, layers2)
            sec["speedups"] = {f"vs_{k}": v["ms_per_step"] / ms2 for k, v in sec["baselines"].items()
                               if "ms_per_step" in v}
        res["secondary"] = sec
        print(f"[bench] secondary {SECONDARY_CONFIG}: {ms2:.4f} ms/step", file=sys.stderr, flush=True)
        del sets2, layers2
        torch.cuda.empty_cache()
    if not args.no_cpu:
        print("[bench] cpu oracle baseline", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(config, args.cpu_budget)
    print(json.dumps(res))


if __name__ == "__main__":
    main()
