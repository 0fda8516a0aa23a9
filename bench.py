"""Benchmark: effective ZGEMM TFLOP/s (8mnk / t) of 2M + Ozaki-II on one MI355X.

Workload (default): C = A B, m = n = k = 8192, complex128, entries
U(-0.5, 0.5) * exp(0.5 N(0, 1)) per part (the phi-distribution of the paper's
Section 6, phi = 0.5), N = 16 2M moduli (log2 M ~ 117.7) with the
Cauchy-Schwarz scaling rule: the setting whose accuracy matches native
complex128 on these inputs (the line reports both errors on the same sampled
entries; the max rule at N = 16 is about twice less accurate than native),
seeded synthetic data.  One step = one full zgemm_2m call (scaling,
residues + 2M pre, the 32 int8 GEMMs, 2M post + CRT + descale) with inputs
resident in HBM.

Prints ONE JSON line on stdout (diagnostics go to stderr); only the optional
``--sweep-n`` mode prints one line per moduli count.  The line carries
the roofline of the dominant kernel (the batched int8 GEMM, timed live with
HIP events recorded by the library on the call's stream), the CPU oracle timed
on a bounded sample of the same workload, native complex128 torch.matmul on
the same GPU for comparison, and the sampled accuracy against a double-double
reference.
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

PEAK_INT8_TOPS = 5000.0   # MI355X dense int8 MFMA, 5.0 POP/s
PEAK_HBM_GBS = 8000.0     # MI355X HBM3E, 8 TB/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in ("k_gemm.hip", "tile_schedule.h", "o2m_internal.h"):
        with open(os.path.join(ROOT, "paper_2609_05419_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_traffic(workload_key: str):
    """HBM bytes per launch of the int8 GEMM from the committed rocprofv3 PMC
    summary, if it was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "k3_gemm_i8_zgemm8192_n16_traffic.json")
    try:
        with open(path) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    if d.get("kernel_hash") != kernel_source_hash() or d.get("workload") != workload_key:
        return None
    return d.get("traffic_bytes_per_launch")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(a, b, n_moduli, rows, cols, scaling="max"):
    """The oracle (exact output of Algorithm 1) on a rows x cols block of C."""
    import oracle

    oracle.lib()  # build/load outside the timed region
    ent = [(i, j) for j in range(cols) for i in range(rows)]
    t0 = time.perf_counter()
    oracle.oq_zgemm(a, b, n_moduli, entries=ent, scaling=scaling)
    dt = time.perf_counter() - t0
    k = a.shape[1]
    threads = oracle.omp_threads()
    return {"value": 8.0 * len(ent) * k / dt / 1e12, "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle",
            "omp_threads": threads, "os_cpu_count": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": f"exact Algorithm-1 output (C oracle, OpenMP, {scaling} rule) on a {rows}x{cols} "
                      f"block of C, k={k}, {dt:.2f} s"}


def hbm_probe(torch) -> dict:
    """STREAM-like rates of plain torch kernels on 4 GiB (after the timed
    region): device copy (read + write), sum (read), fill (write)."""
    n = 4 << 30
    out = {}
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty(n, dtype=torch.uint8, device="cuda")
    x = src.view(torch.float64)
    tests = (("copy_GBs", lambda: dst.copy_(src), 2 * n), ("read_GBs", lambda: x.sum(), n),
             ("write_GBs", lambda: dst.fill_(3), n))
    for name, fn, nbytes in tests:
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        s = torch.cuda.Event(enable_timing=True)
        e = torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(5):
            fn()
        e.record()
        torch.cuda.synchronize()
        out[name] = round(nbytes / (s.elapsed_time(e) / 5 * 1e-3) / 1e9, 1)
    del src, dst, x
    torch.cuda.empty_cache()
    return out


def hbm_probe_hip(torch) -> dict:
    """HBM rates of the probe library's streaming kernels (16-byte accesses,
    2 GiB per buffer, the better of 1 and 4 chunks per thread): read only,
    write only, copy, 1 read : 2 writes (the residue step's mix at N = 16),
    2 reads : 1 write (the CRT's mix at N = 16)."""
    import ctypes
    path = os.path.join(ROOT, "paper_2609_05419_amd", "libo2m_probe.so")
    L = ctypes.CDLL(path)
    P = ctypes.c_void_p
    L.o2m_probe_hbm.argtypes = [ctypes.c_int, P, P, P, P, ctypes.c_size_t, ctypes.c_int, P, ctypes.c_void_p]
    L.o2m_probe_hbm.restype = ctypes.c_double
    n = 2 << 30
    bufs = [torch.empty(n, dtype=torch.uint8, device="cuda") for _ in range(4)]
    for x in bufs:
        x.fill_(7)
    sink = torch.empty(4096, dtype=torch.uint8, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    p = [x.data_ptr() for x in bufs]
    out = {}
    for name, kind in (("read_GBs", 0), ("write_GBs", 1), ("copy_GBs", 2), ("r1w2_GBs", 3), ("r2w1_GBs", 4)):
        out[name] = round(max(L.o2m_probe_hbm(kind, p[0], p[1], p[2], p[3], n, chunks, sink.data_ptr(), st)
                              for chunks in (1, 4)), 1)
    del bufs, sink
    torch.cuda.empty_cache()
    return out


def mfma_ceiling(torch) -> dict:
    """The int8 MFMA rate the chip sustains on register operands (no memory
    traffic), from the probe library: the practical ceiling of the int8 GEMM
    under the part's power budget (random operands), next to zero operands
    and the 32x32x32 instruction."""
    import ctypes
    path = os.path.join(ROOT, "paper_2609_05419_amd", "libo2m_probe.so")
    L = ctypes.CDLL(path)
    L.o2m_probe_int8_mfma.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    L.o2m_probe_int8_mfma.restype = ctypes.c_double
    blocks, iters = 2048, 512
    out = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    res = {}
    for name, variant in (("mfma16x16x64_random_TOPS", 0), ("mfma16x16x64_zero_TOPS", 1),
                          ("mfma32x32x32_random_TOPS", 2)):
        res[name] = round(L.o2m_probe_int8_mfma(variant, blocks, iters, out.data_ptr(), st), 1)
    L.o2m_probe_int8_mfma_residues.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                               ctypes.c_void_p, ctypes.c_void_p]
    L.o2m_probe_int8_mfma_residues.restype = ctypes.c_double
    clk = ctypes.c_double()
    res["mfma16x16x64_residues241_TOPS"] = round(
        L.o2m_probe_int8_mfma_residues(241, blocks, iters, out.data_ptr(), ctypes.addressof(clk), st), 1)
    res["residues241_clock_GHz"] = round(clk.value, 3)
    return res


def mfma_residue_mix(torch, moduli) -> dict:
    """The probe on the symmetric residues of each modulus the call uses, as
    the int8 GEMM meets them (equal work per modulus): N / sum(1 / rate)."""
    import ctypes
    path = os.path.join(ROOT, "paper_2609_05419_amd", "libo2m_probe.so")
    L = ctypes.CDLL(path)
    L.o2m_probe_int8_mfma_residues.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                               ctypes.c_void_p, ctypes.c_void_p]
    L.o2m_probe_int8_mfma_residues.restype = ctypes.c_double
    blocks, iters = 2048, 256
    out = torch.empty(blocks * 256, dtype=torch.int32, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    inv, clocks = 0.0, []
    for q in moduli:
        clk = ctypes.c_double()
        r = L.o2m_probe_int8_mfma_residues(min(q, 256), blocks, iters, out.data_ptr(), ctypes.addressof(clk), st)
        inv += 1.0 / r
        clocks.append(clk.value)
    return {"mfma16x16x64_residue_mix_TOPS": round(len(moduli) / inv, 1),
            "residue_mix_clock_GHz": round(sum(clocks) / len(clocks), 3)}


def error_curve() -> int:
    """Error against the unquantized product over the whole output (the
    accuracy-per-modulus curves): max |c~ - c| / (4 u k (|A||B|)_ij) (the
    tolerance holds when <= 1), max |c~ - c| / |c| and the componentwise
    maxima, for ZGEMM (1024^3, parts N(0,1)) at N = 6..22 and CGEMM (1024^3,
    parts U(-1,1)) at N = 4..10, under both scaling rules."""
    import torch

    import oracle
    import paper_2609_05419_amd as o2m
    import workloads

    dev = torch.device("cuda:0")

    def to_dev(x):
        return torch.from_numpy(np.ascontiguousarray(x.T)).to(dev).t()

    ta, tb = args.transa, args.transb
    if (ta, tb) != ("N", "N") and op not in ("zgemm", "cgemm"):
        print("--transa/--transb apply to zgemm and cgemm only", file=sys.stderr)
        return 2

    def stored(x, t):
        """The device matrix a caller stores for the operand x under op t."""
        return to_dev(x if t == "N" else (x.T if t == "T" else x.conj().T))

    def op_view(X, t):
        return X if t == "N" else (X.mT if t == "T" else X.mH)

    m = n = k = 1024
    sa, sb = workloads.config_seeds(2)
    for op, dist, dtype, u, Ns in (("zgemm", "normal", np.complex128, 2.0 ** -53, range(6, 23, 2)),
                                   ("cgemm", "uniform", np.complex64, 2.0 ** -24, range(4, 11))):
        a = workloads.complex_matrix(m, k, sa, dist=dist, dtype=dtype)
        b = workloads.complex_matrix(k, n, sb, dist=dist, dtype=dtype)
        a64, b64 = a.astype(np.complex128), b.astype(np.complex128)
        t0 = time.perf_counter()
        hi, lo = oracle.dd_gemm(a64, b64)
        absab = np.abs(a64) @ np.abs(b64)
        log(f"bench: dd reference {op} in {time.perf_counter() - t0:.1f} s")
        A, B = to_dev(a), to_dev(b)
        native = (torch.matmul(A, B)).cpu().numpy().astype(np.complex128)
        nerr = oracle.error_vs_reference(native, absab, hi, lo, k, u)
        print(json.dumps({"report": "error_curve", "op": op, "n_moduli": None, "scaling_rule": "native torch.matmul",
                          **{kk: nerr[kk] for kk in ("ratio", "maxrel", "maxrel_re", "maxrel_im", "zeros")}}), flush=True)
        fn = o2m.zgemm_2m if op == "zgemm" else o2m.cgemm_2m
        for rule in ("max", "cs"):
            for N in Ns:
                try:
                    C = fn(A, B, n_moduli=N, scaling=rule)
                except o2m.O2MError as e:
                    log(f"bench: {op} N={N} {rule}: {e}")
                    continue
                got = C.cpu().numpy().astype(np.complex128)
                err = oracle.error_vs_reference(got, absab, hi, lo, k, u)
                print(json.dumps({"report": "error_curve", "op": op, "m": m, "n": n, "k": k, "n_moduli": N,
                                  "scaling_rule": rule,
                                  **{kk: err[kk] for kk in ("ratio", "maxrel", "maxrel_re", "maxrel_im", "zeros")}}),
                      flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--op", choices=("zgemm", "cgemm", "zherk", "dsyrk", "zher2k", "dsyr2k"), default="zgemm")
    ap.add_argument("--scaling", choices=("max", "cs"), default="cs",
                    help="scaling rule: Cauchy-Schwarz (2-norm; default) or per-row maximum")
    ap.add_argument("--sweep-n", default="",
                    help="comma-separated moduli counts: one JSON line per N on the same inputs "
                         "(perf-vs-precision sweep; not the default single-line run)")
    ap.add_argument("--error-curve", action="store_true",
                    help="accuracy report instead of timing: ZGEMM 1024^3 N(0,1) and CGEMM 1024^3 "
                         "U(-1,1), every entry against the double-double oracle, for each moduli "
                         "count and scaling rule; one JSON line per point")
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--m", type=int, default=8192)
    ap.add_argument("--n", type=int, default=8192)
    ap.add_argument("--k", type=int, default=8192)
    ap.add_argument("--n-moduli", type=int, default=16)
    ap.add_argument("--transa", choices=["N", "T", "C"], default="N",
                    help="zgemm/cgemm: the stored A is op(A) itself, its transpose or its conjugate "
                         "transpose (zgemm_2m_op); the product is the same")
    ap.add_argument("--transb", choices=["N", "T", "C"], default="N")
    ap.add_argument("--uplo", choices=["L", "U"], default="L",
                    help="zherk/dsyrk/zher2k/dsyr2k: the triangle written")
    ap.add_argument("--phi", type=float, default=0.5)
    ap.add_argument("--accuracy-samples", type=int, default=1024,
                    help="output entries compared with the double-double reference (and native matmul)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-native", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only copy 1 GiB device-to-device twice (reference kernel for the "
                         "rocprofv3 FETCH_SIZE / WRITE_SIZE scale) and exit")
    args = ap.parse_args()

    if args.calibrate_copy:
        import torch
        n = 1 << 30
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty(n, dtype=torch.uint8, device="cuda")
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"bench: copied {n} bytes twice")
        return 0

    if args.error_curve:
        return error_curve()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: this build has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        return 2

    import torch

    import paper_2609_05419_amd as o2m
    import workloads

    op = args.op
    m, n, k, N = args.m, args.n, args.k, args.n_moduli
    if op in ("zherk", "dsyrk", "zher2k", "dsyr2k"):
        n = m
    rule = args.scaling
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    def to_dev(x):
        return torch.from_numpy(np.ascontiguousarray(x.T)).to(dev).t()

    ta, tb = args.transa, args.transb
    if (ta, tb) != ("N", "N") and op not in ("zgemm", "cgemm"):
        print("--transa/--transb apply to zgemm and cgemm only", file=sys.stderr)
        return 2

    def stored(x, t):
        """The device matrix a caller stores for the operand x under op t."""
        return to_dev(x if t == "N" else (x.T if t == "T" else x.conj().T))

    def op_view(X, t):
        return X if t == "N" else (X.mT if t == "T" else X.mH)

    cfg = {"zgemm": 3, "cgemm": 4, "zherk": 5, "dsyrk": 5, "zher2k": 5, "dsyr2k": 5}[op]
    sa, sb = workloads.config_seeds(cfg)
    log(f"bench: {op} m={m} n={n} k={k} N={N}: generating inputs")
    b = None
    if op == "zgemm":
        a = workloads.complex_matrix(m, k, sa, dist="phi", phi=args.phi)
        b = workloads.complex_matrix(k, n, sb, dist="phi", phi=args.phi)
        A, B = stored(a, ta), stored(b, tb)
        C = torch.empty((n, m), dtype=torch.complex128, device=dev).t()
        if (ta, tb) == ("N", "N"):
            call = lambda N: o2m.zgemm_2m(A, B, n_moduli=N, out=C, scaling=rule)
        else:
            call = lambda N: o2m.zgemm_2m_op(A, B, ta, tb, n_moduli=N, out=C, scaling=rule)
        flops, int8_per_n = 8.0 * m * n * k, 4.0 * m * n * k
        metric = ("effective ZGEMM TFLOP/s (8mnk/t) at m=n=k=8192 + int8 MFMA util %"
                  if (m, n, k) == (8192, 8192, 8192) else "effective ZGEMM TFLOP/s (8mnk/t)")
        desc = (f"zgemm_2m {m}x{n}x{k} complex128, parts U(-0.5,0.5)*exp({args.phi}*N(0,1)), "
                "{N} 2M moduli, int8 MFMA")
        pre_bytes = lambda N: (16.0 + 2 * N) * (m * k + k * n)
        scale_bytes = 16.0 * (m * k + k * n)
        post_bytes = lambda N: (2.0 * N + 16.0) * m * n
    elif op == "cgemm":
        a = workloads.complex_matrix(m, k, sa, dist="uniform", dtype=np.complex64)
        b = workloads.complex_matrix(k, n, sb, dist="uniform", dtype=np.complex64)
        A, B = stored(a, ta), stored(b, tb)
        C = torch.empty((n, m), dtype=torch.complex64, device=dev).t()
        if (ta, tb) == ("N", "N"):
            call = lambda N: o2m.cgemm_2m(A, B, n_moduli=N, out=C, scaling=rule)
        else:
            call = lambda N: o2m.cgemm_2m_op(A, B, ta, tb, n_moduli=N, out=C, scaling=rule)
        flops, int8_per_n = 8.0 * m * n * k, 4.0 * m * n * k
        metric = "effective CGEMM TFLOP/s (8mnk/t)"
        desc = f"cgemm_2m {m}x{n}x{k} complex64, parts U(-1,1), {{N}} 2M moduli, int8 MFMA"
        pre_bytes = lambda N: (8.0 + 2 * N) * (m * k + k * n)
        scale_bytes = 8.0 * (m * k + k * n)
        post_bytes = lambda N: (2.0 * N + 8.0) * m * n
    elif op == "zherk":
        a = workloads.complex_matrix(n, k, sa)
        A = to_dev(a)
        C = o2m.colmajor(torch.zeros((n, n), dtype=torch.complex128, device=dev))
        call = lambda N: o2m.zherk_2m(A, n_moduli=N, out=C, scaling=rule, uplo=args.uplo)
        flops, int8_per_n = 4.0 * n * n * k, 2.0 * n * n * k
        metric = "effective ZHERK TFLOP/s (4n^2k/t)"
        desc = f"zherk_2m n={n} k={k} complex128 N(0,1), {{N}} 2M moduli, lower triangle"
        pre_bytes = lambda N: (16.0 + 2 * N) * n * k
        scale_bytes = 16.0 * n * k
        post_bytes = lambda N: (N + 8.0) * n * n           # both triangles of C+ read, lower C written
    elif op == "dsyrk":
        a = workloads.real_matrix(n, k, sa)
        A = to_dev(a)
        C = o2m.colmajor(torch.zeros((n, n), dtype=torch.float64, device=dev))
        call = lambda N: o2m.dsyrk_2m(A, n_moduli=N, out=C, scaling=rule, uplo=args.uplo)
        flops, int8_per_n = 1.0 * n * n * k, 2.0 * n * n * ((k + 1) // 2)
        metric = "effective DSYRK TFLOP/s (n^2k/t)"
        desc = f"dsyrk_2m n={n} k={k} float64 N(0,1), {{N}} 2M moduli, lower triangle"
        pre_bytes = lambda N: (8.0 + N) * n * k
        scale_bytes = 8.0 * n * k
        post_bytes = lambda N: (N + 4.0) * n * n
    elif op == "zher2k":
        a = workloads.complex_matrix(n, k, sa)
        b = workloads.complex_matrix(n, k, sb)
        A, B = to_dev(a), to_dev(b)
        C = o2m.colmajor(torch.zeros((n, n), dtype=torch.complex128, device=dev))
        call = lambda N: o2m.zher2k_2m(A, B, n_moduli=N, out=C, scaling=rule, uplo=args.uplo)
        flops, int8_per_n = 8.0 * n * n * k, 4.0 * n * n * k   # N GEMMs n x n x 2k
        metric = "effective ZHER2K TFLOP/s (8n^2k/t)"
        desc = f"zher2k_2m n={n} k={k} complex128 N(0,1), {{N}} 2M moduli, lower triangle"
        pre_bytes = lambda N: (16.0 + 2 * N) * 2 * n * k
        scale_bytes = 16.0 * 2 * n * k
        post_bytes = lambda N: (N + 8.0) * n * n
    else:  # dsyr2k
        a = workloads.real_matrix(n, k, sa)
        b = workloads.real_matrix(n, k, sb)
        A, B = to_dev(a), to_dev(b)
        C = o2m.colmajor(torch.zeros((n, n), dtype=torch.float64, device=dev))
        call = lambda N: o2m.dsyr2k_2m(A, B, n_moduli=N, out=C, scaling=rule, uplo=args.uplo)
        flops, int8_per_n = 2.0 * n * n * k, 4.0 * n * n * ((k + 1) // 2)
        metric = "effective DSYR2K TFLOP/s (2n^2k/t)"
        desc = f"dsyr2k_2m n={n} k={k} float64 N(0,1), {{N}} 2M moduli, lower triangle"
        pre_bytes = lambda N: (8.0 + N) * 2 * n * k
        scale_bytes = 8.0 * 2 * n * k
        post_bytes = lambda N: (N + 4.0) * n * n
    if rule == "cs":
        desc += ", Cauchy-Schwarz scaling"   # one pass as well: maxima and sums of squares together
    a_host, b_host = a, b

    def run_one(N: int, with_extras: bool) -> dict:
        log(f"bench: N={N} warmup {args.warmup}")
        for _ in range(args.warmup):
            call(N)
        torch.cuda.synchronize()

        log(f"bench: N={N} timing {args.steps} steps")
        o2m.phase_timing(True)
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        for _ in range(args.steps):
            call(N)
        end.record(stream)
        torch.cuda.synchronize()
        ms = start.elapsed_time(end) / args.steps
        phases = o2m.phase_times()
        o2m.phase_timing(False)
        log(f"bench: {ms:.3f} ms/step, phases {phases}")

        value = flops / (ms * 1e-3) / 1e12
        gemm_ms = phases.get("int8_gemm", float("nan"))
        # int8 work: 2 GEMMs per 2M modulus; a hybrid set's 3M moduli take 3
        n2, n3 = min(N, 22), max(N - 22, 0)
        achieved = (n2 + 1.5 * n3) * int8_per_n / (gemm_ms * 1e-3) / 1e12
        workload_key = (f"{op} m{m} n{n} k{k} N{N} phi{args.phi}" + ("" if rule == "max" else f" {rule}")
                        + ("" if (ta, tb) == ("N", "N") else f" op{ta}{tb}"))
        roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_INT8_TOPS,
                    "unit": "TFLOP/s", "frac": round(achieved / PEAK_INT8_TOPS, 4),
                    "traffic": load_traffic(workload_key)}
        hbm = {
            "scale_GBs": round(scale_bytes / (phases["scale"] * 1e-3) / 1e9, 1),
            "residues_GBs": round(pre_bytes(N) / (phases["residues"] * 1e-3) / 1e9, 1),
            "crt_GBs": round(post_bytes(N) / (phases["crt"] * 1e-3) / 1e9, 1),
            "peak_GBs": PEAK_HBM_GBS,
        }

        native, native_sample = None, None
        ent = None
        if op in ("zgemm", "cgemm"):
            rng = np.random.default_rng(8)
            ent = [(int(i), int(j)) for i, j in zip(rng.integers(0, m, args.accuracy_samples),
                                                    rng.integers(0, n, args.accuracy_samples))]
        if with_extras and not args.no_native and op in ("zgemm", "cgemm"):
            try:
                An, Bn = op_view(A, ta), op_view(B, tb)
                for _ in range(2):
                    Cn = torch.matmul(An, Bn)
                torch.cuda.synchronize()
                s2 = torch.cuda.Event(enable_timing=True)
                e2 = torch.cuda.Event(enable_timing=True)
                reps = 3
                s2.record(stream)
                for _ in range(reps):
                    Cn = torch.matmul(An, Bn)
                e2.record(stream)
                torch.cuda.synchronize()
                nms = s2.elapsed_time(e2) / reps
                native = {"op": f"torch.matmul {A.dtype}".replace("torch.", ""), "ms": round(nms, 3),
                          "tflops": round(flops / (nms * 1e-3) / 1e12, 2)}
                Cnh = Cn.cpu().numpy()
                native_sample = np.array([Cnh[i, j] for i, j in ent])
                del Cn, Cnh
            except Exception as e:
                log(f"bench: native comparison skipped: {e}")

        # sampled accuracy against the double-double reference (GEMMs), and of
        # native torch.matmul on the same entries
        accuracy = None
        if ent is not None:
            try:
                import oracle
                Ch = C.cpu().numpy()
                got = np.array([Ch[i, j] for i, j in ent])
                a64, b64 = a_host.astype(np.complex128), b_host.astype(np.complex128)
                hi, lo = oracle.dd_gemm(a64, b64, entries=ent)
                absab = np.array([np.sum(np.abs(a64[i, :]) * np.abs(b64[:, j])) for i, j in ent])
                u = 2.0 ** -53 if op == "zgemm" else 2.0 ** -24
                err = oracle.error_vs_reference(got.astype(np.complex128), absab, hi, lo, k, u)
                exact = (oracle.oq_zgemm(a_host, b_host, N, entries=ent, scaling=rule) if op == "zgemm"
                         else oracle.oq_cgemm(a_host, b_host, N, entries=ent, scaling=rule))
                accuracy = {"sampled_entries": len(ent), "maxrel": err["maxrel"], "tol_ratio": err["ratio"],
                            "bit_exact_vs_oracle": bool(np.array_equal(got, exact))}
                if native_sample is not None:
                    nerr = oracle.error_vs_reference(native_sample.astype(np.complex128), absab, hi, lo, k, u)
                    accuracy["native_maxrel"] = nerr["maxrel"]
                    accuracy["native_tol_ratio"] = nerr["ratio"]
                    accuracy["at_most_native"] = bool(err["maxrel"] <= nerr["maxrel"])
            except Exception as e:  # accuracy is a report, not the metric
                log(f"bench: accuracy check skipped: {e}")

        ceiling = None
        if with_extras:
            hbm["practical"] = hbm_probe(torch)
            try:
                probe = hbm_probe_hip(torch)
                hbm["probe"] = probe
                hbm["scale_frac_of_probe_read"] = round(hbm["scale_GBs"] / probe["read_GBs"], 4)
                hbm["residues_frac_of_probe_r1w2"] = round(hbm["residues_GBs"] / probe["r1w2_GBs"], 4)
                hbm["crt_frac_of_probe_r2w1"] = round(hbm["crt_GBs"] / probe["r2w1_GBs"], 4)
            except (OSError, AttributeError) as e:
                log(f"bench: HBM probe skipped: {e}")
            try:
                ceiling = mfma_ceiling(torch)
                ceiling["gemm_frac_of_random_ceiling"] = round(achieved / ceiling["mfma16x16x64_random_TOPS"], 4)
                ceiling.update(mfma_residue_mix(torch, o2m.moduli(N)[0]))
                ceiling["gemm_frac_of_residue_mix_ceiling"] = round(
                    achieved / ceiling["mfma16x16x64_residue_mix_TOPS"], 4)
            except (OSError, AttributeError) as e:
                log(f"bench: MFMA probe skipped: {e}")

        cpu = None
        if with_extras and not args.no_cpu_baseline and op == "zgemm":
            log("bench: CPU oracle baseline on a sample")
            cpu = cpu_baseline(a_host, b_host, N, rows=min(m, 1024), cols=min(n, 1536), scaling=rule)

        return {
            "metric": metric,
            "value": round(value, 2),
            "unit": "TFLOP/s",
            "n_gpus": 1,
            "steps": args.steps,
            "warmup": args.warmup,
            "ms_per_step": round(ms, 4),
            "higher_is_better": True,
            "scaling": "weak",
            "vs_baseline": None,
            "dtype": "f64",
            "data": "synthetic",
            "config": {"workload": desc.format(N=N), "op": op, "m": m, "n": n, "k": k, "n_moduli": N,
                       "phi": args.phi if op == "zgemm" else None, "scaling_rule": rule,
                       **({} if (ta, tb) == ("N", "N") else {"transa": ta, "transb": tb}),
                       **({"uplo": args.uplo} if op in ("zherk", "dsyrk", "zher2k", "dsyr2k") else {}),
                       "parallelism": "single GPU"},
            "int8_mfma_util": round(achieved / PEAK_INT8_TOPS, 4),
            "int8_mfma_ceiling": ceiling,
            "phase_ms": {kk: round(v, 4) for kk, v in phases.items()},
            "hbm": hbm,
            "roofline": roofline,
            "cpu_baseline": cpu,
            "native_zgemm": native,
            "accuracy": accuracy,
        }

    if args.sweep_n:
        for i, Nv in enumerate(int(x) for x in args.sweep_n.split(",")):
            print(json.dumps(run_one(Nv, with_extras=(i == 0))), flush=True)
        return 0
    print(json.dumps(run_one(N, with_extras=True)), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
