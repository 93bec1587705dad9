"""Benchmark of the Gaunt tensor product hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload edge|edge16|tiny|manybody|sweep|highdeg|mix] [--L L]
                    [--backward | --weighted] [--no-cpu-baseline] [--gpus 1]

Default: the edge workload (B=65536 edges x C=128 channels, L1=L2=Lout=6,
x2 = radial weights x real SH of the edge direction), fp32.  One step is one
gtp_full over the whole batch.  Prints one JSON line with the throughput in
(b,c)-products/s, the roofline of the kernel (its launch duration measured
with HIP events on the stream it runs on; reported against whichever roof,
fp32 compute or HBM, the kernel comes closer to, with the other alongside)
and the fp64 oracle timed on the
host cores on a bounded sample of the same workload.  Before the warmup
steps the box's roofs are measured with the library's probes (MFMA and VALU
fp32 rates, the two-reads-one-write HBM stream; --no-roof-probe skips them);
after the edge workload, the L = 32 degree sweep is timed the same way and
reported as l32_sweep (--no-l32 skips it).  --backward times
gtp_full_backward (both input gradients) on the same inputs instead,
--weighted gtp_full_weighted with per-degree weights.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Gaunt TP (b,c)-products/sec at L=6 fp32; % HBM/MFMA roofline on 1 MI355X"
PEAK_FP32_TFLOPS = 157.3  # MI355X published fp32 vector / matrix peak
PEAK_HBM_GBS = 8000.0     # MI355X HBM3E

# Flops per (b,c)-product of the paper's Fourier method counted for an
# FFT-based real-form convolution (sparse change of basis, min(direct, FFT)
# convolution, projection to Lout): the figures the 50 % targets were set
# with, reported as context only (the kernels run a formulation with fewer
# flops, whose own count sets the roofline).
FFT_FORMULATION_FLOPS = {2: 745, 4: 6403, 6: 25785, 8: 71349, 16: 346034, 32: 1549020, 64: 7442286}
FFT_FORMULATION_FLOPS_MANYBODY = 2200

# Flops per product of the thread-per-product kernel at equal degrees
# L1 = L2 = Lout = L (fp32 inputs) as it runs: 2 FMA + MUL + ADD per lane (one
# lane is one product).  L = 4, 6, 8: the SQ_INSTS_VALU_FMA_F32 / _MUL_F32 /
# _ADD_F32 counters per wave; the others: the same count read off the
# kernel's instruction stream, which is loop-free per lane and equals the
# counters where both exist.  Below the structural count of the formulation
# (formulation_flops) because the compiler folds twiddles of +-1 and constant
# products.
SMALL_KERNEL_FLOPS = {1: 80, 2: 422, 3: 1224, 4: 2648, 5: 4232, 6: 7446, 7: 11392, 8: 17652}
# the stepwise many-body chain L = 2, nu = 3, Lout = 3 (one kernel), counted the same way
STEPWISE_FLOPS_L2_NU3_LOUT3 = 829


def kernel_flops(L1: int, L2: int, Lout: int) -> int:
    """Algorithmic flops per product of the kernel that runs (L1, L2, Lout):
    the executed count of the thread-per-product kernel for equal degrees up
    to 8, else the formulation's structural count (which leaves out the
    matrix cores' padding rows and columns)."""
    if L1 == L2 == Lout and L1 in SMALL_KERNEL_FLOPS:
        return SMALL_KERNEL_FLOPS[L1]
    return formulation_flops(L1, L2, Lout)


def formulation_flops(L1: int, L2: int, Lout: int) -> int:
    """Flops per product of the formulation the kernels implement (Sec. 3.2
    with the convolution theorem on a real-form sampling grid): theta nodes
    t_j = j pi / (U + 1), interior nodes in U / 2 mirror pairs plus two poles;
    phi samples NP = 4 Q with the 4-fold sample symmetry; an FMA counts 2.
      theta synthesis, per input t: K_t FMA per mirror pair (even/odd partial
        sums), 2 adds per m-part and pair (node and mirror), 2 FMA per degree
        at the poles;
      phi synthesis, per input and interior node: 2 L_t FMA per sample set;
      sample products and folds: 28 flops per node and sample set;
      phi analysis: (2 Le + 1) FMA per node and sample set;
      mirror combination: 2 adds per moment and pair;
      theta analysis: (Le + 1)^2 FMA per pair, 2 FMA per degree at the poles."""
    U = L1 + L2
    Le = min(Lout, U)
    NP = (U + Le + 1 + 3) // 4 * 4
    sets = NP // 4 + 1
    pairs = U / 2
    f = 0.0
    for Lt in (L1, L2):
        K = (Lt + 1) ** 2
        f += 2 * K * pairs + 2 * (2 * Lt + 1) * pairs + 4 * (Lt + 1)
        f += 4 * Lt * sets * U
    f += 28 * U * sets
    f += 2 * (2 * Le + 1) * sets * U
    f += 2 * (2 * Le + 1) * pairs
    f += 2 * (Le + 1) ** 2 * pairs + 4 * (Le + 1)
    return int(round(f))


def _fft_flops(N: int, nonzero_in: int = -1) -> int:
    """Flops of the in-register radix-2 complex DFT of length N (gtp_fft.hpp):
    4 per butterfly (a complex add and subtract) plus the twiddle products
    (6 for a general one, 4 for an odd multiple of an eighth turn, none for a
    quarter turn)."""
    f, length = 0, 2
    while length <= N:
        half = length // 2
        for j in range(half):
            if j == 0 or 4 * j == length or 4 * j == 3 * length:
                tw = 0
            elif (8 * j) % length == 0:
                tw = 4
            else:
                tw = 6
            f += (N // length) * (4 + tw)
        length *= 2
    return f


def fft_variant_flops(L: int) -> int:
    """Flops per product of the matrix-core kernel's radix-FFT variant
    (L1 = L2 = Lout = L in {16, 32, 64}): the theta stages as in the DFT form, and
    per pass of 16 theta nodes the three FFT stages of phi_fft -- 16 N2
    column DFTs of length N1 with their twiddle powers and products, 16 N1 row
    DFTs of length N2 with the sample products and the real forward transform
    (a length-N2/2 DFT and N2/2 + 1 recombinations), 8 (N2/2 + 1) pairs of
    forward column DFTs of length N1."""
    NF = 64 if L <= 16 else (128 if L <= 32 else 256)
    N1 = 8 if L <= 32 else 16
    N2 = NF // N1
    U = 2 * L
    pairs = U / 2
    K = (L + 1) ** 2
    theta = 2 * (2 * K * pairs + 2 * (2 * L + 1) * pairs + 4 * (L + 1)) + 2 * (L + 1) ** 2 * pairs + 4 * (L + 1)
    col = _fft_flops(N1) + 6 * (N1 - 2) + 6 * (N1 - 1)
    row = _fft_flops(N2) + N2 + _fft_flops(N2 // 2) + (N2 // 2 + 1) * 10 + 6 * (N2 // 2 - 1) + 6 * (N2 // 2)
    fwd = 2 * _fft_flops(N1) + 4 * 2 * (L + 1) / (N2 // 2 + 1)
    per_pass = 16 * N2 * col + 16 * N1 * row + 8 * (N2 // 2 + 1) * fwd
    return int(round(theta + (L // 8) * per_pass))


def escn_flops(L: int, C: int) -> float:
    """Flops per product of the rotated-frame convolution (L1 = L2 = Lout = L;
    Sec. 3.3, eq. sh2fs-escn): x' = D x and y = D^T y' (sum_l (2l+1)^2 FMA each);
    per mirror pair of the NT = 2L + 1 theta nodes: K FMA of synthesis, 2 adds
    per m-part for the two nodes, the zonal filter (L + 1 FMA, 2 adds), 2
    multiplies and 2 adds per m-part, K FMA of analysis; plus the edge's
    rotation matrices, shared by its C channels: T = Z(-b) J Z(-a) (6 flops
    per entry) and D = J^T T ((2l+1)^3 FMA per degree).  An FMA counts 2."""
    K = (L + 1) ** 2
    parts = 2 * L + 1
    pairs = L + 1
    rot = 2 * sum((2 * l + 1) ** 2 for l in range(L + 1))
    per_pair = 2 * K + 2 * parts + 2 * (L + 1) + 2 + 4 * parts + 2 * K
    per_edge = sum(6 * (2 * l + 1) ** 2 + 2 * (2 * l + 1) ** 3 for l in range(L + 1))
    return 2 * rot + pairs * per_pair + per_edge / C


def nsh(L):
    return (L + 1) * (L + 1)


# device-side sources every kernel depends on (the host dispatch in
# gtp_api.hip does not change a kernel's memory traffic), and those of single
# kernel files (build-time constants, their tables)
SHARED_SOURCES = ["gtp_ct.hpp", "gtp_device.hpp", "gtp_tables.cpp", "gtp_tables.hpp"]
KERNEL_SOURCES = {
    "gtp_small.hip": ["gen_small_consts.cpp", "gtp_small.hpp"],
    "gtp_escn.hip": ["gen_small_consts.cpp", "gtp_escn.hpp", "gtp_escn_tables.cpp", "gtp_escn_tables.hpp"],
    "gtp_wave.hip": ["gtp_fft.hpp"],
    "gtp_escn_wave.hip": ["gtp_escn.hpp", "gtp_escn_tables.cpp", "gtp_escn_tables.hpp"],
}


# degree triples with a thread-per-product kernel of their own
OWN_SMALL_TRIPLES = {(a, a, a) for a in range(1, 9)} | {(2, 2, 3), (3, 2, 3), (1, 2, 2), (2, 1, 3)}


def padded_kernel(L1: int, L2: int, Lout: int):
    """(kernel, roofline bound, source file) that runs a degree triple with no
    kernel of its own: the dot product for Lout = 0, else the equal-degree
    kernel of the padded degree A = max(L1, L2, min(Lout, L1 + L2))."""
    if Lout == 0:
        return "k_dot0", "hbm", "gtp_generic.hip"
    A = max(1, L1, L2, min(Lout, L1 + L2))
    if A <= 8:
        return f"k_full_small_pad<{A}>", "alu", "gtp_small.hip"
    W = 16 if A <= 16 else (32 if A <= 32 else 64)
    return ("k_full_wave4" if W > 32 else "k_full_wave") + f" (padded to L = {W})", "mfma", "gtp_wave.hip"


def fused_backward(degrees, conv: str = "auto") -> bool:
    """Whether gtp_full_backward computes both gradients in one launch
    (k_bwd_small: equal degrees 1..7 on the thread-per-product kernel)."""
    return (degrees is not None and degrees[0] == degrees[1] == degrees[2] and 1 <= degrees[0] <= 7
            and conv not in ("generic", "direct"))


def dominant_kernel(workload: str, L: int, escn: bool = False, conv: str = "auto", degrees=None):
    """(kernel, roofline bound, source file) of the kernel that dominates a workload."""
    if degrees is not None and workload == "sweep" and conv == "auto" and tuple(degrees) not in OWN_SMALL_TRIPLES \
            and not (degrees[0] == degrees[1] == degrees[2] and degrees[0] in (16, 32, 64)):
        return padded_kernel(*degrees)
    if conv == "fft" and workload in ("sweep", "highdeg") and L in (16, 32, 64):
        return ("k_full_wave4_fft" if L > 32 else "k_full_wave (FFT)"), "alu", "gtp_wave.hip"
    if escn:
        # both kernels of the step (rotation matrices, then the product): one unit
        if L == 16:
            # one kernel: the rotations applied from the edge angles
            return "k_conv_escn_wave", "mfma", "gtp_escn_wave.hip"
        return "k_escn_rot+k_conv_escn", "alu", "gtp_escn.hip"
    if workload == "mix":
        # pair products (thread per product) and the mix on the matrix cores in one kernel
        return "k_mix_fused", "alu", "gtp_small.hip"
    if workload in ("sweep", "highdeg", "edge16") and (L >= 16 or workload == "highdeg"):
        return ("k_full_wave4" if L > 32 else "k_full_wave"), "mfma", "gtp_wave.hip"
    if workload == "manybody":
        return "k_self_stepwise_small", "alu", "gtp_small.hip"
    return "k_full_small", "alu", "gtp_small.hip"


def kernel_sources_sha(kernel_source: str) -> str:
    """Hash of the sources that make up one kernel's launch path."""
    h = hashlib.sha256()
    for f in sorted(SHARED_SOURCES + KERNEL_SOURCES.get(kernel_source, []) + [kernel_source]):
        with open(os.path.join(ROOT, "paper_2401_10216_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_key(workload: str, L: int, degrees=None) -> str:
    if workload == "sweep" and degrees is not None and len(set(degrees)) > 1:
        return "sweep_{}_{}_{}".format(*degrees)
    return f"sweep_L{L}" if workload == "sweep" else workload


def load_traffic(key: str, kernel_source: str):
    """HBM bytes per launch from committed rocprofv3 FETCH_SIZE / WRITE_SIZE
    counters, if they were taken on the current sources of the kernel."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        d = json.load(open(path)).get(key)
    except Exception:
        return None
    if not d or d.get("kernel_sha") != kernel_sources_sha(kernel_source):
        return None
    return d.get("bytes_per_launch")


def pair_step(args, torch, gtp, inputs, plan, t1, t2, y, idx_cfg):
    """The timed step of a pair workload: gtp_full, or with --backward the
    gradients of <dy, gtp_full(x1, x2)> in both inputs for a seeded dy.
    Returns (step, rows(idx) -> the device result rows of products idx,
    oracle_of(O, idx, a, b) -> fn computing the same rows on the host, the
    output tensors the step writes)."""
    L1, L2, Lout = plan.L1, plan.L2, plan.Lout
    if getattr(args, "weighted", False):
        # one row of per-degree weights shared by every channel (w_l1 w_l2 w_l)
        rng = inputs.rng_for(idx_cfg, 300)
        w = [rng.standard_normal((1, L + 1)).astype("float32") for L in (L1, L2, Lout)]
        tw = [torch.from_numpy(v).to(y.device) for v in w]

        def step():
            gtp.gtp_full_weighted(plan, t1, t2, tw[0], tw[1], tw[2], False, y=y)

        def oracle_of(O, idx, a, b):
            return lambda: O.gtp_weighted(a, b, w[0][0], w[1][0], w[2][0], L1, L2, Lout)
        return step, (lambda idx: y.view(-1, y.shape[-1])[torch.from_numpy(idx).to(y.device)]), oracle_of, (y,)
    if not args.backward:
        def step():
            gtp.gtp_full(plan, t1, t2, y)

        def oracle_of(O, idx, a, b):
            if max(L1, L2, Lout) <= 8:
                return lambda: O.gtp(a, b, L1, L2, Lout)
            return lambda: O.gtp_grid(a, b, L1, L2, Lout)
        return step, (lambda idx: y.view(-1, y.shape[-1])[torch.from_numpy(idx).to(y.device)]), oracle_of, (y,)
    B, C = int(t1.shape[0]), int(t1.shape[1])
    d = inputs.output_gradient(idx_cfg, (B, C, nsh(Lout)))
    dy = torch.from_numpy(d).to(y.device)
    dx1 = torch.empty((B, C, nsh(L1)), dtype=torch.float32, device=y.device)
    dx2 = torch.empty((B, C, nsh(L2)), dtype=torch.float32, device=y.device)

    def step():
        gtp.gtp_full_backward(plan, t1, t2, dy, dx1=dx1, dx2=dx2)

    def result(idx):
        ti = torch.from_numpy(idx).to(y.device)
        return torch.cat([dx1.view(B * C, -1)[ti], dx2.view(B * C, -1)[ti]], dim=1)

    def oracle_of(O, idx, a, b):
        dd = d.reshape(B * C, -1)[idx].astype("float64")
        return lambda: np.concatenate(O.gtp_vjp(a, b, dd, L1, L2, Lout), axis=1)
    return step, result, oracle_of, (dx1, dx2)


def make_workload(args, torch, gtp, inputs):
    """Returns (step callable, products per step, description dict, alg flops, alg bytes, oracle sample fn)."""
    dev = torch.device("cuda:0")
    w = args.workload
    if w in ("edge", "edge16"):
        # edge16: the edge shape at L = 16 with 8192 edges (1.2 GB per
        # coefficient tensor)
        B, C, L = (65536, 128, 6) if w == "edge" else (8192, 128, 16)
        x1, r, h = inputs.edge_inputs(B, C, L, index=2 if w == "edge" else 7)
        t1 = torch.from_numpy(x1).to(dev)
        tr = torch.from_numpy(r.astype("float32")).to(dev)
        th = torch.from_numpy(h).to(dev)
        t2 = gtp.gtp_sh_filter(L, tr, th)
        del th
        plan = gtp.Plan(L, L, L)
        y = torch.empty((B, C, nsh(L)), dtype=torch.float32, device=dev)
        step, result, oracle_of, _ = pair_step(args, torch, gtp, inputs, plan, t1, t2, y, 2 if w == "edge" else 7)
        if args.escn:
            # the same product from (x1, r, h) in the edge's rotated frame
            del t2
            th = torch.from_numpy(h).to(dev)

            def step():
                gtp.gtp_conv_escn(plan, t1, tr, th, y=y)

        def oracle_sample(O, idx):
            deg = inputs.degree_of_index(L)
            bi, ci = idx // C, idx % C
            a = x1[bi, ci].astype("float64")
            bref = h[bi, ci][:, deg] * O.real_sh_xyz(L, r[bi])
            return oracle_of(O, idx, a, bref), result

        desc = {"workload": f"{w}: B={B} edges x C={C} channels, L1=L2=Lout={L}, x1~N(0,1), "
                            "x2 = h[b,c,l] * Y_lm(r_b), r_b uniform on S^2, h~N(0,1)",
                "B": B, "C": C, "L1": L, "L2": L, "Lout": L, "in_dtype": "f32"}
        if args.escn:
            desc["workload"] += "; gtp_conv_escn from (x1, r, h): rotated edge frame, m = 0 filter"
            # per product: rotation in (sum (2l+1)^2 FMA), zonal theta product, rotation out;
            # bytes: x1 and y, h, and the edge vector shared by C channels
            return step, B * C, desc, (escn_flops(L, C), FFT_FORMULATION_FLOPS[L]), 4 * (2 * nsh(L) + L + 1) + 12.0 / C, \
                oracle_sample, 2 if w == "edge" else 7
        return step, B * C, desc, (kernel_flops(L, L, L), FFT_FORMULATION_FLOPS[L]), 4 * (2 * nsh(L) + nsh(L)), \
            oracle_sample, 2 if w == "edge" else 7
    if (args.backward or args.weighted) and w not in ("edge", "tiny", "sweep", "highdeg"):
        raise SystemExit("--backward / --weighted apply to the pair workloads (edge, tiny, sweep, highdeg)")
    if args.backward and args.weighted:
        raise SystemExit("--backward and --weighted are separate benchmarks")
    if args.escn and (w not in ("edge", "edge16") or args.backward or args.weighted):
        raise SystemExit("--escn applies to the edge workloads' forward product")
    if w in ("tiny", "sweep", "highdeg"):
        if w == "tiny":
            B, C, L, idx_cfg = 1024, 1, 2, 1
            x1, x2 = inputs.pair_inputs(1, B, C, L, L)
        elif w == "sweep" and args.degrees:
            # unequal degrees: the sweep's batch shape, iid N(0,1) of each degree
            L1d, L2d, Lod = (int(v) for v in args.degrees.split(","))
            B, C, idx_cfg = 2048, 128, 4
            rng = inputs.rng_for(4, 10 * (L1d + 100 * L2d + 10000 * Lod))
            x1 = inputs.normal(rng, (B, C, nsh(L1d)))
            x2 = inputs.normal(rng, (B, C, nsh(L2d)))
            L = L1d
        elif w == "sweep":
            L = args.L
            B, C, idx_cfg = 2048, 128, 4
            x1, x2 = inputs.sweep_inputs(L)
        else:
            B, C, L, idx_cfg = 32768, 64, 16, 5
            b1, b2, x1, x2 = inputs.highdeg_inputs(B, C, L)
        if w == "highdeg":
            t1 = torch.from_numpy(b1.view("int16")).to(dev).view(torch.bfloat16)
            t2 = torch.from_numpy(b2.view("int16")).to(dev).view(torch.bfloat16)
            in_bytes = 2
        else:
            t1 = torch.from_numpy(x1).to(dev)
            t2 = torch.from_numpy(x2).to(dev)
            in_bytes = 4
        flags = {"auto": 0, "direct": gtp.GTP_CONV_DIRECT, "generic": gtp.GTP_FORCE_GENERIC,
                 "fft": gtp.GTP_CONV_FFT, "dft": gtp.GTP_CONV_DFT}[args.conv]
        L1, L2, Lo = (L1d, L2d, Lod) if (w == "sweep" and args.degrees) else (L, L, L)
        plan = gtp.Plan(L1, L2, Lo, flags)
        if args.products:
            # crossover runs: the first N products, as [N, 1, K]
            C = 1
            B = min(args.products, t1.shape[0] * t1.shape[1])
            t1 = t1.reshape(-1, nsh(L1))[:B].reshape(B, 1, -1)
            t2 = t2.reshape(-1, nsh(L2))[:B].reshape(B, 1, -1)
            x1 = x1.reshape(-1, nsh(L1))[:B].reshape(B, 1, -1)
            x2 = x2.reshape(-1, nsh(L2))[:B].reshape(B, 1, -1)
        y = torch.empty((B, C, nsh(Lo)), dtype=torch.float32, device=dev)
        step, result, oracle_of, _ = pair_step(args, torch, gtp, inputs, plan, t1, t2, y, idx_cfg)

        def oracle_sample(O, idx):
            a = x1.reshape(B * C, -1)[idx].astype("float64")
            b = x2.reshape(B * C, -1)[idx].astype("float64")
            return oracle_of(O, idx, a, b), result

        degs = f"L1=L2=Lout={L}" if (L1, L2) == (L, L) and Lo == L else f"L1={L1}, L2={L2}, Lout={Lo}"
        desc = {"workload": f"{w}: B={B} x C={C}, {degs}, iid N(0,1)" + (" rounded to bf16" if w == "highdeg" else ""),
                "B": B, "C": C, "L1": L1, "L2": L2, "Lout": Lo, "in_dtype": "bf16" if w == "highdeg" else "f32"}
        if args.conv != "auto":
            desc["conv"] = args.conv
        fl = kernel_flops(L1, L2, Lo)
        if args.conv == "fft" and L1 == L2 == Lo and L in (16, 32, 64):
            fl = fft_variant_flops(L)
        return step, B * C, desc, (fl, FFT_FORMULATION_FLOPS.get(L) if (L1, L2, Lo) == (L, L, L) else None), \
            in_bytes * (nsh(L1) + nsh(L2)) + 4 * nsh(Lo), oracle_sample, idx_cfg
    if w == "manybody":
        N, C, L, nu, Lout = 1728, 256, 2, 3, 3
        x = inputs.manybody_inputs(N, C, L)
        tx = torch.from_numpy(x).to(dev)
        y = torch.empty((N, C, nsh(Lout)), dtype=torch.float32, device=dev)

        def step():
            gtp.gtp_selfproduct(tx, L, nu, Lout, gtp.GTP_SELF_STEPWISE, y)

        def oracle_sample(O, idx):
            a = x.reshape(N * C, -1)[idx].astype("float64")
            return (lambda: O.selfproduct(a, L, nu, Lout, "stepwise")), \
                (lambda ix: y.view(N * C, -1)[torch.from_numpy(ix).to(y.device)])

        desc = {"workload": "manybody: 64 molecules x 27 atoms = 1728 nodes, C=256, L=2, nu=3 stepwise, Lout=3, "
                            "x~N(0,1)/sqrt(2l+1)", "B": N, "C": C, "L": L, "nu": nu, "Lout": Lout, "in_dtype": "f32"}
        return step, N * C, desc, (STEPWISE_FLOPS_L2_NU3_LOUT3, FFT_FORMULATION_FLOPS_MANYBODY), 4 * (nsh(L) + nsh(Lout)), \
            oracle_sample, 3
    if w == "mix":
        cfg = inputs.WORKLOADS["mix"]
        B, C, L = cfg["B"], cfg["C"], cfg["L1"]
        x1, x2, W = inputs.mix_inputs(B, C, L)
        t1 = torch.from_numpy(x1).to(dev)
        t2 = torch.from_numpy(x2).to(dev)
        tw = torch.from_numpy(W).to(dev)
        plan = gtp.Plan(L, L, L)
        y = torch.empty((B, C, nsh(L)), dtype=torch.float32, device=dev)

        def step():
            gtp.gtp_channel_mix(plan, t1, t2, tw, y=y)

        def oracle_sample(O, idx):
            # idx indexes pair products (b, c1, c2); the oracle computes the
            # whole batch entries b they fall in
            bs = np.unique(idx // (C * C))
            rows = lambda ix: y[torch.from_numpy(bs).to(y.device)].reshape(len(bs), -1)
            return (lambda: O.channel_mix(x1[bs], x2[bs], W, L, L, L).reshape(len(bs), -1)), rows, len(bs) * C * C

        desc = {"workload": "mix: channel mixing y[b,co] = sum_{c1,c2} W[co,c1,c2] GTP(x1[b,c1], x2[b,c2]), "
                            "B=8192, C1=C2=Co=32, L1=L2=Lout=6, x~N(0,1), W~N(0,1/C^2)",
                "B": B, "C": C, "L1": L, "L2": L, "Lout": L, "in_dtype": "f32"}
        # per pair product: the product itself and 2 Co K flops of the mix; bytes: x1, x2, y over C^2 pairs
        return step, B * C * C, desc, (kernel_flops(L, L, L) + 2 * C * nsh(L), None), \
            4.0 * nsh(L) * 3 * C / (C * C), oracle_sample, 6
    raise SystemExit(f"unknown workload {w}")


def cpu_baseline(O, inputs, oracle_sample, total, idx_cfg, budget_s=15.0):
    """Time the oracle on a seeded subsample sized to roughly budget_s seconds,
    on every host core this process may run on (its CPU affinity set): the
    oracle's BLAS thread pool is sized to that count."""
    try:
        cpus = len(os.sched_getaffinity(0))
    except AttributeError:
        cpus = os.cpu_count() or 1
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        limits = threadpool_limits(limits=cpus)
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        limits, threads = None, cpus
    n = min(1024, total)
    while True:
        idx = inputs.sample_indices(idx_cfg, total, n)
        got_sample = oracle_sample(O, idx)
        fn, rows = got_sample[0], got_sample[1]
        done = got_sample[2] if len(got_sample) > 2 else n  # products the oracle call covers
        t0 = time.perf_counter()
        ref = fn()
        dt = time.perf_counter() - t0
        if dt >= 0.6 * budget_s or n >= total:
            break
        n = int(min(total, max(2 * n, n * budget_s / max(dt, 1e-3))))
    if limits is not None:
        limits.restore_original_limits()
    # rows(idx) gathers the device results of exactly these products (each
    # index < total, checked on the host first)
    assert idx.size and 0 <= idx.min() and idx.max() < total
    got = rows(idx).cpu().numpy()
    err = O.max_rel_err(got, ref)
    host = None
    try:
        with open("/proc/cpuinfo") as fh:
            host = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), None)
    except OSError:
        pass
    out = {"value": done / dt, "unit": "products/s", "cores": int(threads), "kind": "oracle", "host": host,
           "host_cpus_in_affinity": cpus, "nproc": os.cpu_count(),
           "sample": f"{done} seeded products of the same workload, fp64 numpy oracle (dense real-Gaunt contraction), "
                     f"{dt:.2f} s", "max_rel_err_gpu_vs_oracle": err, "one_core": None}
    # the same oracle on one core, on a smaller seeded subsample (about a
    # quarter of the time above if the threads scaled perfectly)
    try:
        from threadpoolctl import threadpool_limits
    except Exception:
        return out
    n1 = max(16, min(total, n // max(1, 4 * int(threads))))
    idx1 = inputs.sample_indices(idx_cfg + 50, total, n1)
    got1 = oracle_sample(O, idx1)
    done1 = got1[2] if len(got1) > 2 else n1
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        got1[0]()
        dt1 = time.perf_counter() - t0
    out["one_core"] = {"value": done1 / dt1, "unit": "products/s", "cores": 1,
                       "sample": f"{done1} seeded products, {dt1:.2f} s"}
    return out


def stream_roofs(args, torch, gtp):
    """The HBM roof as the chip reaches it: 1 GiB read-only, write-only and
    copy sweeps and a two-read-one-write sweep (the pair products' mix: 1 GiB
    read, 0.5 GiB written) by the library's streaming probes (16-byte
    accesses, non-temporal stores, one contiguous chunk per workgroup), and
    torch's device copy, each timed with HIP events on the launch stream;
    then the fp32 rates the chip delivers under load (the library's compute
    probes: VALU FMA chains and 16x16x4 MFMA chains, 8 waves per SIMD).
    Also the calibration workload of the FETCH_SIZE / WRITE_SIZE counters
    (k_probe_copy moves a known 1 GiB each way)."""
    nbytes = 1 << 30
    dev = torch.device("cuda:0")
    src = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    out = {"workload": "copy: HBM streaming roofs on 1 GiB buffers", "bytes": nbytes}
    probes = [("read", lambda: gtp.gtp_stream_probe(0, src, sink), nbytes),
              ("write", lambda: gtp.gtp_stream_probe(1, None, dst), nbytes),
              ("copy", lambda: gtp.gtp_stream_probe(2, src, dst), 2 * nbytes),
              ("read2_write1", lambda: gtp.gtp_stream_probe(3, src, dst), nbytes + nbytes // 2),
              ("torch_copy", lambda: dst.copy_(src), 2 * nbytes)]
    def timed(fn):
        for _ in range(args.warmup):
            fn()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(args.steps):
            fn()
        ev1.record(stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / args.steps

    for name, fn, moved in probes:
        ms = timed(fn)
        out[name] = {"ms": round(ms, 4), "GBps": round(moved / (ms * 1e-3) / 1e9, 1),
                     "frac_of_8TBps": round(moved / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
    # the fp32 rates under load (VALU FMA chains, 16x16x4 MFMA chains)
    for name, mode, iters in (("valu_fma_f32", 0, 1 << 14), ("mfma_f32", 1, 1 << 12)):
        flops = gtp.gtp_compute_probe(mode, iters, sink)
        ms = timed(lambda: gtp.gtp_compute_probe(mode, iters, sink))
        out[name] = {"ms": round(ms, 4), "TFLOPs": round(flops / (ms * 1e-3) / 1e12, 2),
                     "frac_of_157_3": round(flops / (ms * 1e-3) / 1e12 / PEAK_FP32_TFLOPS, 4)}
    print(json.dumps(out), flush=True)


def measure_roofs(torch, gtp):
    """The roofs of this box, measured before the workload's warmup steps by
    the library's probes (HIP events on the launch stream): the
    two-reads-one-write stream (1 GiB read, 0.5 GiB written: the byte mix of
    a product's two inputs and its output) and the fp32 rates under load (VALU
    FMA chains, 16x16x4 MFMA chains).  About 0.35 s of GPU work; the stream
    runs last, the load closest to the kernels' own."""
    nbytes = 1 << 30
    dev = torch.device("cuda:0")
    src = torch.empty(nbytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty(nbytes // 8, dtype=torch.float32, device=dev)
    sink = torch.zeros(1, dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()

    def timed(fn, warm, reps):
        for _ in range(warm):
            fn()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for _ in range(reps):
            fn()
        ev1.record(stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / reps

    out = {}
    for name, mode, iters in (("mfma_f32_TFLOPs", 1, 1 << 12), ("valu_fma_f32_TFLOPs", 0, 1 << 14)):
        flops = gtp.gtp_compute_probe(mode, iters, sink)
        ms = timed(lambda: gtp.gtp_compute_probe(mode, iters, sink), 10, 60)
        out[name] = round(flops / (ms * 1e-3) / 1e12, 2)
    ms = timed(lambda: gtp.gtp_stream_probe(3, src, dst), 100, 400)
    out["read2_write1_GBps"] = round((nbytes + nbytes // 2) / (ms * 1e-3) / 1e9, 1)
    del src, dst
    return out


def l32_sweep(args, torch, gtp, inputs):
    """The degree-32 product measured in the same run as the edge workload:
    the L = 32 degree sweep (B = 2048 x C = 128 products, iid N(0,1), fp32,
    the matrix-core kernel k_full_wave<32>), with the same warmup and step
    counts, after the edge workload's timed region: its kernel time on the
    launch stream, its fraction of the fp32 peak at the kernel's flop count
    and its HBM traffic when the committed counters match the sources (its
    parity with the oracle is the GPU tests')."""
    sa = argparse.Namespace(**vars(args))
    sa.workload, sa.L, sa.degrees, sa.products, sa.conv = "sweep", 32, "", 0, "auto"
    sa.backward = sa.weighted = sa.escn = False
    step, products, desc, alg_flops, alg_bytes, oracle_sample, idx_cfg = make_workload(sa, torch, gtp, inputs)
    for _ in range(args.warmup):
        step()
    stream = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    kernel_ms = ev0.elapsed_time(ev1) / args.steps
    achieved = alg_flops[0] * products / (kernel_ms * 1e-3) / 1e12
    return {"workload": desc["workload"], "kernel": "k_full_wave", "kernel_ms": round(kernel_ms, 5),
            "products_per_s": products / (kernel_ms * 1e-3),
            "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(achieved / PEAK_FP32_TFLOPS, 4), "alg_flops_per_product": alg_flops[0],
                         "traffic": load_traffic("sweep_L32", "gtp_wave.hip"),
                         "alg_bytes_per_launch": alg_bytes * products}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="edge")
    ap.add_argument("--L", type=int, default=32)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-roof-probe", action="store_true",
                    help="skip the same-box roof measurement before the warmup steps")
    ap.add_argument("--no-l32", action="store_true",
                    help="with the edge workload: skip the L = 32 degree sweep measured after it")
    ap.add_argument("--conv", choices=["auto", "direct", "generic", "fft", "dft"], default="auto",
                    help="step-2 algorithm for the convolution crossover: auto (the measured fastest), direct "
                         "(fused direct real-form convolution), generic (workgroup-per-product convolution "
                         "theorem, the direct kernel's structural twin), fft (convolution theorem with radix-2 FFT "
                         "phi transforms), dft (convolution theorem with direct symmetric DFT phi transforms)")
    ap.add_argument("--backward", action="store_true",
                    help="time the backward pass (gtp_full_backward: both input gradients for a seeded dy) "
                         "of a pair workload instead of gtp_full")
    ap.add_argument("--weighted", action="store_true",
                    help="time gtp_full_weighted (per-degree weights w_l1 w_l2 w_l shared by all channels) of a "
                         "pair workload instead of gtp_full")
    ap.add_argument("--escn", action="store_true",
                    help="edge workload through gtp_conv_escn (the product with the SH filter taken in each edge's "
                         "rotated frame from x1, r, h) instead of gtp_full with a prebuilt filter")
    ap.add_argument("--degrees", default="",
                    help="L1,L2,Lout of the sweep workload (its batch shape) instead of --L for all three")
    ap.add_argument("--products", type=int, default=0,
                    help="use only the first N products of a pair workload (crossover runs of slow variants)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the Gaunt tensor product shards over (b,c) with no exchange, "
              "and the benchmark runs on a single MI355X (--gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2401_10216_amd import gtp, inputs
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    gtp.lib()  # fails loudly if the HIP library is not built
    if args.workload == "copy":
        stream_roofs(args, torch, gtp)
        return
    step, products, desc, alg_flops, alg_bytes, oracle_sample, idx_cfg = make_workload(args, torch, gtp, inputs)

    measured = None if args.no_roof_probe else measure_roofs(torch, gtp)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # average launch duration on the launch stream (a backward step is one
    # launch for both gradients at equal degrees up to 7, else two launches
    # of the forward kernel, one per input gradient)
    degs = (desc["L1"], desc["L2"], desc["Lout"]) if "L2" in desc else None
    fused = args.backward and fused_backward(degs, args.conv)
    launches = 2 if args.backward and not fused else 1
    if args.weighted and alg_flops:
        # one multiply per input and output coefficient on top of the product
        alg_flops = (alg_flops[0] + 3 * nsh(desc["L1"]), alg_flops[1])
    if args.backward and alg_flops:
        # per launch (equal degrees): dy (fp32) and one input in, one gradient
        # out; fused: dy and both inputs in, both gradients out, two products
        K = nsh(desc["L1"])
        es = 2 if desc.get("in_dtype") == "bf16" else 4
        if fused:
            alg_bytes = (4 + 2 * es + 2 * 4) * K
            alg_flops = (2 * alg_flops[0], alg_flops[1] and 2 * alg_flops[1])
        else:
            alg_bytes = (4 + es + 4) * K
    kernel_ms = ev0.elapsed_time(ev1) / args.steps / launches
    value = products * args.steps / wall

    roof = None
    if alg_flops:
        alg_flops, fft_flops = alg_flops
        achieved = alg_flops * products / (kernel_ms * 1e-3) / 1e12
        kname, bound, ksrc = dominant_kernel(args.workload, desc.get("L1", desc.get("L", 0)), args.escn, args.conv,
                                             degs)
        if fused:
            kname = "k_bwd_small"
        suffix = "_backward" if args.backward else ("_weighted" if args.weighted else ("_escn" if args.escn else ""))
        if args.conv != "auto":
            suffix += "_" + args.conv
        tb = load_traffic(traffic_key(args.workload, desc.get("L1", 0), degs) + suffix, ksrc)
        # fp32 peak: packed VALU and dense fp32 MFMA are both 157.3 TFLOP/s on MI355X
        comp = {"bound": bound, "achieved": round(achieved, 3), "peak": PEAK_FP32_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_FP32_TFLOPS, 4), "alg_flops_per_product": alg_flops,
                "fft_formulation_flops_per_product": fft_flops}
        hbm_gbs = alg_bytes * products / (kernel_ms * 1e-3) / 1e9
        hbm = {"bound": "hbm", "achieved": round(hbm_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
               "frac": round(hbm_gbs / PEAK_HBM_GBS, 4), "alg_bytes_per_product": alg_bytes}
        # the kernel is bound by the roof it is closer to: that one is reported,
        # the other rides along ("hbm" or "compute")
        if hbm["frac"] > comp["frac"]:
            roof = dict(hbm, compute=comp)
        else:
            roof = dict(comp, hbm=hbm)
        roof.update({"traffic": tb, "kernel": kname, "kernel_ms": round(kernel_ms, 5)})
        if measured:
            # the kernel's HBM rate against the stream of its byte mix on this machine
            roof["measured"] = dict(measured, hbm_frac_of_measured=round(hbm_gbs / measured["read2_write1_GBps"], 4))

    cpu = None
    if not args.no_cpu_baseline:
        from oracle import gtp_oracle as O
        cpu = cpu_baseline(O, inputs, oracle_sample, products, idx_cfg)
    l32 = None
    if args.workload == "edge" and not (args.backward or args.weighted or args.escn or args.no_l32):
        l32 = l32_sweep(args, torch, gtp, inputs)

    metric = METRIC
    if args.workload == "mix":
        metric = "channel-mixing Gaunt TP (b,c1,c2) pair-products/sec at L=6 fp32, C=32; % ALU roofline on 1 MI355X"
    if args.escn:
        metric = "equivariant convolution (b,c)-products/sec at L=6 fp32, rotated edge frame; % ALU roofline on 1 MI355X"
    if args.weighted:
        metric = "weighted Gaunt TP (per-degree w_l1 w_l2 w_l) (b,c)-products/sec; % MFMA/ALU roofline on 1 MI355X"
        desc["workload"] = "weighted " + desc["workload"] + "; weights ~ N(0,1), one row for all channels"
    if args.backward:
        metric = "Gaunt TP backward (dx1 and dx2) (b,c)-products/sec; % MFMA/ALU roofline per launch on 1 MI355X"
        desc["workload"] = "backward of " + desc["workload"] + "; dy ~ N(0,1)"
        desc["launches_per_step"] = launches
    if "L1" in desc and args.workload != "mix":
        # the degrees the workload runs at (the headline's L = 6 otherwise)
        l1, l2, lo = desc["L1"], desc["L2"], desc["Lout"]
        metric = metric.replace("at L=6", f"at L={l1}" if l1 == l2 == lo else f"at (L1,L2,Lout)=({l1},{l2},{lo})")
    line = {"metric": metric, "value": value, "unit": "products/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": wall * 1e3 / args.steps, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic", "config": desc,
            "roofline": roof, "cpu_baseline": cpu}
    if l32 is not None:
        line["l32_sweep"] = l32
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
