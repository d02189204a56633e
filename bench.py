#!/usr/bin/env python3
"""Throughput of the SubZero+ hot path on one MI355X (OPT-13B-shaped stack).

One step is Alg. 3 with central differences over the whole synthetic stack:
  - subspace refresh of every U_i, V_i when t mod F == 0 (Eq. 11, Alg. 1);
  - for every weight matrix: the perturbed linear over the 2q query blocks
    (Eq. 4; prepare = the rank-r operands, apply = the fused GEMM);
  - the per-block squared loss of the last matrix's outputs against a fixed
    target and the central difference g_j (Eq. 3 per query);
  - the subspace Adam update of every matrix (Eqs. 6-10).
All inputs are synthetic, seeded, and resident in HBM before timing starts.
Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "perturbed-linear TFLOP/s (% MFMA peak); subspace update GB/s (% HBM peak)"
PEAK_BF16_TFLOPS = 2516.6  # 256 CU x 4 SIMD x 1024 FLOP/clk x 2.4 GHz, dense
PEAK_HBM_GBPS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_traffic_opt13b.json")
CSRC = os.path.join(ROOT, "paper_2608_15665_amd", "csrc")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def plinear_flops(T, m, n, r, q, nblk, nsigned):
    """Algorithmic FLOPs of one matrix's perturbed linear per step: the main products of all
    nblk blocks, the X_b V projections of all blocks, the rank-r terms of the nsigned perturbed
    blocks and the q products U Z_j."""
    return nblk * (2 * T * m * n + 2 * T * n * r) + nsigned * 2 * T * r * m + q * 2 * m * r * r


def apply_flops(T, m, n, r, q, nblk, nsigned):
    """Algorithmic FLOPs of the fused GEMM launch alone: X_b W^T and the rank-r terms."""
    return nblk * 2 * T * m * n + nsigned * 2 * T * r * m


def lora_flops(T, m, n, rl, r, q, nblk, nsigned):
    """Algorithmic FLOPs of one LoRA-adapted layer per step: the frozen-base products, the
    X_b [A^T | V_A] projections, the rank-(rl + r) terms of the perturbed blocks, and the per-block
    right factors scale [B' | s eps B' U_A Z_A]."""
    re = rl + r
    return (nblk * (2 * T * m * n + 2 * T * n * re) + nsigned * 2 * T * re * m
            + nsigned * m * (2 * r * rl + 2 * rl * r))


def lora_apply_flops(T, m, n, rl, r, q, nblk, nsigned):
    return nblk * 2 * T * m * n + nsigned * 2 * T * (rl + r) * m


def update_bytes(m, n, r, q, wbytes=2):
    """Algorithmic HBM bytes of one matrix's update: W read + write (bf16, or fp32 for the
    adapter factors), fp32 U and V, the q fp32 Z_j, and the two fp32 moments read + write."""
    return 2 * wbytes * m * n + 4 * r * (m + n) + 4 * q * r * r + 16 * r * r


def _region(text, start, end):
    i = text.index(start)
    return text[i:text.index(end, i) + len(end)]


def source_hash():
    """Hash of the source text the dominant kernel is built from: its argument struct, its
    MFMA and store helpers, the kernel with its launcher, and the 16-bit rounding helpers its
    epilogue uses."""
    gemm = open(os.path.join(CSRC, "zo_gemm.hip")).read()
    inc = open(os.path.join(CSRC, "zo_internal.h")).read()
    parts = [_region(gemm, "struct GemmArgs {", "};"),
             _region(gemm, "template <int OUT>\n__device__ __forceinline__ void store4(", "\n}\n"),
             _region(gemm, "template <int OUT>\n__device__ __forceinline__ void load8(", "\n}\n"),
             _region(gemm, "template <int OUT>\n__device__ __forceinline__ void store8(", "\n}\n"),
             _region(gemm, "__device__ __forceinline__ f32x16 mfma32(", "\n}\n"),
             _region(gemm, "constexpr int MAIN_RB = 128;", 'hipGetLastError(), "k_gemm_main");\n}'),
             _region(inc, "__device__ __forceinline__ bf16_t f32_to_bf16(", "\n}\n"),
             _region(inc, "__device__ __forceinline__ uint32_t pack_bf16x2(", "\n}\n"),
             _region(inc, "__device__ __forceinline__ uint16_t f32_to_f16(", "\n}\n"),
             _region(inc, "__device__ __forceinline__ uint32_t pack_f16x2(", "\n}\n")]
    h = hashlib.sha256()
    for p in parts:
        h.update(p.encode())
    return h.hexdigest()[:16]


class ZFeed:
    """The per-step coefficients Z_j of every perturbed factor (Alg. 3: one Gaussian r x r draw
    per query and matrix, keyed by step), drawn on the host inside the timed window.

    A worker thread draws step s + 1 into a pinned host buffer while the GPU runs step s (it is
    started once step s is enqueued); the
    copy to the device runs on a side stream, and the compute stream waits for it before the
    step's first use.  Two device slots alternate: the copy into a slot waits until the compute
    stream has finished the step that last read it, and the host buffer of a slot is refilled
    only after its previous copy has landed."""

    def __init__(self, seed, nfac, q, r, dev):
        import threading  # noqa: F401  (the executor below runs one worker thread)
        from concurrent.futures import ThreadPoolExecutor

        import torch
        self.seed, self.nfac, self.q, self.r = seed, nfac, q, r
        shape = (nfac, q, r, r)
        self.dev = [torch.empty(shape, dtype=torch.float32, device=dev) for _ in range(2)]
        self.host = [torch.empty(shape, dtype=torch.float32, pin_memory=True) for _ in range(2)]
        self.copy_stream = torch.cuda.Stream()
        self.copied = [None, None]
        self.freed = [None, None]
        self.pool = ThreadPoolExecutor(max_workers=1)
        self.pending = {}
        self.draw_s = {}
        self.h2d = {}
        self.nbytes = 4 * nfac * q * r * r
        self.cur = -1

    def _draw(self, s, slot):
        import zo_draws as zd
        ev = self.copied[slot]
        if ev is not None:
            ev.synchronize()
        t0 = time.perf_counter()
        h = self.host[slot].numpy()
        for i in range(self.nfac):
            h[i] = zd.z_draws(self.seed, s, i, self.q, self.r)
        self.draw_s[s] = time.perf_counter() - t0

    def request(self, s):
        if s not in self.pending:
            self.pending[s] = self.pool.submit(self._draw, s, s % 2)

    def acquire(self, s):
        """Device slot holding step s's Z, ordered before the compute stream's next work."""
        import torch
        slot = s % 2
        self.request(s)
        self.pending.pop(s).result()
        cs = self.copy_stream
        if self.freed[slot] is not None:
            cs.wait_event(self.freed[slot])
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(cs):
            e0.record(cs)
            self.dev[slot].copy_(self.host[slot], non_blocking=True)
            e1.record(cs)
        self.copied[slot] = e1
        torch.cuda.current_stream().wait_event(e1)
        self.h2d[s] = (e0, e1)
        self.cur = s
        return slot

    def release(self, slot):
        """The compute stream's work on this slot is enqueued: the next copy into it waits for it.
        Then starts the host draw of the next step.  The draw is requested only now, once the
        whole step is enqueued: a draw loop running beside the enqueue holds the interpreter lock
        in slices, and the enqueuing thread, which gives the lock up in every library call, waits
        out a slice each time (a 1.1 ms refresh call took up to 1.3 s beside a looping draw, and
        15 ms of GPU idling at a step's start in the benchmark).  This thread then blocks in the
        next acquire while the GPU runs the step just enqueued."""
        import torch
        ev = torch.cuda.Event()
        ev.record()
        self.freed[slot] = ev
        self.request(self.cur + 1)

    def report(self, steps):
        """Host draw and copy time of the given steps (ms per step)."""
        d = [self.draw_s[s] * 1e3 for s in steps if s in self.draw_s]
        c = [self.h2d[s][0].elapsed_time(self.h2d[s][1]) for s in steps if s in self.h2d]
        self.pool.shutdown(wait=True)
        return {"z_bytes_per_step": self.nbytes,
                "z_host_draw_ms_per_step": round(sum(d) / max(1, len(d)), 2),
                "z_h2d_ms_per_step": round(sum(c) / max(1, len(c)), 3),
                "z_h2d_gbs": round(self.nbytes * len(c) / max(1e-9, sum(c) * 1e-3) / 1e9, 1) if c else None,
                "in_timed_window": True,
                "how": "worker thread draws step s+1 on the host while step s runs (requested once step s "
                       "is enqueued); pinned buffer; copy on a side stream; the compute stream waits for it"}


def omega_host_draw(seed, panels, r, F, sample=6):
    """Host time of drawing one refresh's Gaussian panel inputs (Alg. 1 first step), estimated
    from the first `sample` panels (float64 draws, cast to fp32) scaled by element count; the
    timed steps build their panels on the device instead (rolled copies of one draw per row
    count), so this is reported, not timed in the window."""
    import zo_draws as zd
    rows = list(panels)
    tot = sum(rows) * r
    take = rows[:sample]
    t0 = time.perf_counter()
    for k, rw in enumerate(take):
        zd.f32(zd.draw(seed, "OMEGA_U", (999, k), (rw, r)))
    dt = time.perf_counter() - t0
    est = dt * tot / max(1, sum(take) * r)
    return {"panels": len(rows), "elements": tot, "fp32_bytes": 4 * tot,
            "host_draw_s_per_refresh_est": round(est, 3), "amortised_ms_per_step": round(est / F * 1e3, 2),
            "sample": f"{len(take)} panels drawn, scaled by element count"}


class ClockSampler:
    """Graphics clock of GPU 0 sampled from the power-management firmware's metrics table (the
    amdsmi library) every `period` seconds while `active` is set; None when the table cannot be
    read."""

    def __init__(self, period=0.2):
        import threading
        self.period = period
        self.samples = []
        self.active = threading.Event()
        self.stop = threading.Event()
        self.source = None
        self.h = None
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            hs = amdsmi.amdsmi_get_processor_handles()
            self.h = hs[0] if hs else None
            self.amdsmi = amdsmi
        except Exception as e:  # pragma: no cover - depends on the machine
            self.source = f"unavailable ({type(e).__name__})"
        self.th = threading.Thread(target=self._run, daemon=True)
        if self.h is not None:
            self.th.start()

    def _read(self):
        a = self.amdsmi
        try:
            mt = a.amdsmi_get_gpu_metrics_info(self.h)
            cl = mt.get("current_gfxclks")
            vals = [v for v in (cl if isinstance(cl, (list, tuple)) else []) if isinstance(v, (int, float))
                    and 0 < v < 10000]
            if vals:
                self.source = "amdsmi gpu_metrics current_gfxclks (mean over XCDs)"
                return sum(vals) / len(vals)
            for key in ("current_gfxclk", "average_gfxclk_frequency"):
                v = mt.get(key)
                if isinstance(v, (int, float)) and 0 < v < 10000:
                    self.source = f"amdsmi gpu_metrics {key}"
                    return float(v)
        except Exception:
            pass
        try:
            v = a.amdsmi_get_clock_info(self.h, a.AmdSmiClkType.GFX).get("clk")
            if isinstance(v, (int, float)) and 0 < v < 10000:
                self.source = "amdsmi clock_info GFX"
                return float(v)
        except Exception:
            pass
        return None

    def _run(self):
        while not self.stop.is_set():
            if self.active.is_set():
                v = self._read()
                if v is not None:
                    self.samples.append(v)
            time.sleep(self.period)

    def result(self):
        self.stop.set()
        if self.h is not None:
            self.th.join(timeout=2)
        if not self.samples:
            return {"median_mhz": None, "samples": 0, "source": self.source}
        s = sorted(self.samples)
        return {"median_mhz": round(s[len(s) // 2], 1), "min_mhz": round(s[0], 1), "max_mhz": round(s[-1], 1),
                "samples": len(s), "period_s": self.period, "source": self.source}


def clock_fields(achieved, sclk):
    """The MFMA peak at the observed clock (the datasheet figure is at 2.4 GHz) and the fraction
    of it reached."""
    mhz = sclk.get("median_mhz")
    if not mhz:
        return {}
    peak = PEAK_BF16_TFLOPS * mhz / 2400.0
    return {"peak_at_observed_sclk": round(peak, 1), "frac_at_observed_sclk": round(achieved / peak, 4)}


def copy_calibration():
    """A plain device copy of known size (for scaling the FETCH_SIZE / WRITE_SIZE counters)."""
    import torch
    nbytes = 1 << 30
    a = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda").normal_()
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": nbytes, "copy_calibration_bytes_written": nbytes,
                      "launches": 3}))


def shared_x_report(seed, T, m, n, r, q, nblk, dt, label, reps=5):
    """The shared-X variant (one X read by every block: the first layer's q, k, v, or the Tiny
    layer): X W^T once, then each block's rank-r term.  Timed as prepare + apply, and the apply
    alone against the two-term roofline max(MFMA time of one X W^T at the datasheet peak, HBM
    time of X, W and the nblk outputs at 8 TB/s).  For comparison, the same problem with X
    copied into every block (the per-block path, X W^T nblk times)."""
    import numpy as np
    import torch

    import paper_2608_15665_amd as zo
    import zo_draws as zd
    dev = "cuda"
    es = 4 if dt == torch.float32 else 2
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    X = torch.randn(T, n, device=dev, generator=g).to(dt)
    W = (0.02 * torch.randn(m, n, device=dev, generator=g)).to(dt)
    U = torch.linalg.qr(torch.randn(m, r, device=dev, generator=g))[0].contiguous()
    V = torch.linalg.qr(torch.randn(n, r, device=dev, generator=g))[0].contiguous()
    Z = torch.from_numpy(zd.z_draws(seed, 0, 0, q, r)).to(dev)
    bq, bs = [b // 2 for b in range(nblk)], [1 if b % 2 == 0 else -1 for b in range(nblk)]
    Xr = X.repeat(nblk, 1).contiguous()

    def timed(pl, what):
        pl.prepare()
        pl.apply()
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        e[0].record()
        for _ in range(reps):
            pl.prepare()
        e[1].record()
        for _ in range(reps):
            pl.apply()
        e[2].record()
        torch.cuda.synchronize()
        return e[0].elapsed_time(e[1]) / reps, e[1].elapsed_time(e[2]) / reps

    shared = zo.PerturbedLinear(X, W, U, V, Z, bq, bs, 1e-3, T, x_block_stride=0)
    prep_ms, app_ms = timed(shared, "shared")
    per_block = zo.PerturbedLinear(Xr, W, U, V, Z, bq, bs, 1e-3, T, x_block_stride=T * n)
    pb_prep, pb_app = timed(per_block, "per-block")
    peak = PEAK_BF16_TFLOPS if es == 2 else 157.3
    flops = 2.0 * T * m * n + 2.0 * T * n * r + nblk * 2.0 * T * r * m
    nbytes = es * (T * n + m * n + nblk * T * m)
    ideal_ms = max(2.0 * T * m * n / (peak * 1e9), nbytes / (PEAK_HBM_GBPS * 1e6))
    del X, W, Xr, shared, per_block
    torch.cuda.empty_cache()
    return {"shape": f"{label}: T={T} x m={m} x n={n}, r={r}, {nblk} blocks, {'fp32' if es == 4 else 'bf16'}",
            "apply_ms": round(app_ms, 4), "prepare_ms": round(prep_ms, 4),
            "two_term_ideal_ms": round(ideal_ms, 4), "frac_of_two_term": round(ideal_ms / app_ms, 4),
            "algorithmic_tflops": round(flops / (app_ms * 1e-3) / 1e12, 2),
            "per_block_path_apply_ms": round(pb_app, 4), "speedup_vs_per_block": round(pb_app / app_ms, 2)}


def practical_peaks(T, nblk, m, n, r, q, dt16):
    """What library kernels reach on this GPU in the same run: a plain GEMM of the workload's
    first shape (torch.matmul, i.e. hipBLASLt), a 2 GiB device copy and a 2 GiB in-place
    read-modify-write (torch elementwise add).  Context for the roofline fractions.

    The library GEMM and the fused perturbed-linear GEMM (zo_perturbed_linear_apply, same
    M = nblk T, m, n, plus its rank-r segment) are also timed head to head under sustained load:
    rounds of back-to-back launches of each, alternating, for about 2 s apiece after a warm-up,
    so that both run at the power-limited clock the timed steps see (a short burst on an idle GPU
    runs at a higher clock)."""
    import torch

    import paper_2608_15665_amd as zo
    import zo_draws as zd
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def timed(fn, reps):
        for _ in range(2):
            fn()
        a, b = ev(), ev()
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    M = nblk * T
    g = torch.Generator(device="cuda")
    g.manual_seed(1)
    X = torch.randn(M, n, device="cuda", generator=g).to(dt16)
    W = (0.02 * torch.randn(m, n, device="cuda", generator=g)).to(dt16)
    Y = torch.empty(M, m, device="cuda", dtype=dt16)
    ms_gemm = timed(lambda: torch.matmul(X, W.t(), out=Y), 5)
    U = torch.linalg.qr(torch.randn(m, r, device="cuda", generator=g))[0].contiguous()
    V = torch.linalg.qr(torch.randn(n, r, device="cuda", generator=g))[0].contiguous()
    Z = torch.from_numpy(zd.z_draws(1, 0, 0, q, r)).cuda()
    bq, bs = [b // 2 for b in range(nblk)], [1 if b % 2 == 0 else -1 for b in range(nblk)]
    pl = zo.PerturbedLinear(X, W, U, V, Z, bq, bs, 1e-3, T, x_block_stride=T * n, Y=Y)
    pl.prepare()
    lib_fn = lambda: torch.matmul(X, W.t(), out=Y)
    ours_fn = pl.apply
    flops_lib = 2.0 * M * m * n
    flops_ours = flops_lib + nblk * 2.0 * T * r * m
    reps = max(4, int(400.0 / max(ms_gemm, 1e-3)))  # ~0.4 s per round
    for _ in range(reps):  # warm-up to the sustained clock
        lib_fn()
        ours_fn()
    t_lib = t_ours = 0.0
    for _ in range(5):
        t_lib += timed(lib_fn, reps)
        t_ours += timed(ours_fn, reps)
    sustained = {"shape": f"{M}x{m}x{n}", "rounds": 5, "launches_per_round": reps,
                 "torch_matmul_tflops": round(flops_lib / (t_lib / 5) / 1e9, 1),
                 "k_gemm_main_tflops": round(flops_ours / (t_ours / 5) / 1e9, 1)}
    sustained["ratio"] = round(sustained["k_gemm_main_tflops"] / sustained["torch_matmul_tflops"], 4)
    del X, W, Y, U, V, Z, pl
    nbytes = 1 << 31
    a = torch.empty(nbytes // 2, dtype=dt16, device="cuda").normal_(generator=g)
    b = torch.empty_like(a)
    ms_copy = timed(lambda: b.copy_(a), 5)
    ms_rmw = timed(lambda: a.add_(1.0), 5)
    del a, b
    torch.cuda.empty_cache()
    return {"gemm_torch_matmul": {"shape": f"{M}x{m}x{n}", "tflops": round(flops_lib / ms_gemm / 1e9, 1),
                                  "note": "5 launches after 2, right after the timed steps"},
            "gemm_sustained_head_to_head": sustained,
            "copy_2gib_gbs": round(2 * nbytes / ms_copy / 1e6, 1),
            "inplace_rmw_2gib_gbs": round(2 * nbytes / ms_rmw / 1e6, 1)}


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([d.get("num_threads", 1) for d in threadpool_info() if d.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        return 1


def cpu_baseline(cfg, seed, budget_s, mat, lora, r, f16=False):
    """The float64 oracle on bounded samples of the same workload, on this host's cores: the
    perturbed linear (the metric's unit), the update (GB/s) and the refresh QR (ms per panel),
    each also with one BLAS thread."""
    import numpy as np
    import oracle
    import zo_draws as zd
    try:
        from threadpoolctl import threadpool_limits
    except Exception:  # pragma: no cover
        threadpool_limits = None
    threads = _blas_threads()
    T, q = cfg["T"], cfg["q"]
    m, n = mat[1], mat[2]
    rl, scale = zd.QWEN_LORA_RANK, zd.QWEN_LORA_ALPHA / zd.QWEN_LORA_RANK
    S = 256
    cast = zd.as_f16_values if f16 else zd.as_bf16_values
    rnd = oracle.round_f16 if f16 else oracle.round_bf16
    W = cast(zd.draw(seed, "W0", (m, n), (m, n), 0.02))[1]
    X0 = cast(zd.draw(seed, "X", (T, n, 0), (S, n)))[1]
    Om_U = zd.draw(seed, "OMEGA_U", (0, m), (m, r))
    Om_V = zd.draw(seed, "OMEGA_V", (0, n), (n, r))
    U, V = oracle.haar_qr(Om_U)[0], oracle.haar_qr(Om_V)[0]
    Z = zd.z_draws(seed, 0, 0, q, r).astype(np.float64)
    g = zd.draw(seed, "G", (0,), (q,))
    if lora:
        A = zd.f32(zd.draw(seed, "LORA_A", (0,), (rl, n), 0.02)).astype(np.float64)
        B = np.zeros((m, rl))
        UA = oracle.haar_qr(zd.draw(seed, "OMEGA_U", (1, rl), (rl, r)))[0]
        VB = oracle.haar_qr(zd.draw(seed, "OMEGA_V", (1, rl), (rl, r)))[0]

    def plinear_leg(budget, cap):
        flops, nb = 0.0, 0
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < budget and nb < cap:
            j, s = (nb // 2) % q, (1 if nb % 2 == 0 else -1)
            if lora:
                oracle.lora_perturbed_linear(X0, W, A, UA, V, Z[j], B, U, VB, Z[(j + 1) % q], s, 1e-3, scale)
                re = rl + r
                flops += 2 * S * m * n + 2 * S * n * re + 2 * S * re * m + 2 * m * (2 * r * rl + 2 * rl * r)
            else:
                oracle.perturbed_linear(X0, W, U, V, Z[j], s, 1e-3)
                flops += 2 * S * m * n + 2 * S * n * r + 2 * S * r * m + 2 * m * r * r
            nb += 1
        return flops / (time.perf_counter() - t0) / 1e12, nb

    M1 = np.zeros((r, r))
    M2 = np.zeros((r, r))
    if lora:  # the updated matrices are the fp32 adapter factors; A (rl x n) stands for them
        Wu, Uu, Vu, ubytes = A, UA, V, update_bytes(rl, n, r, q, 4)
        rnd = zd.f32
    else:
        Wu, Uu, Vu, ubytes = W, U, V, update_bytes(m, n, r, q)

    def update_leg(budget):
        k = 0
        t0 = time.perf_counter()
        while k < 1 or time.perf_counter() - t0 < budget:
            out = oracle.subspace_adam_update(Wu, Uu, Vu, Z, g, M1, M2, 1, 1e-3, 0.9, 0.95, 1e-8)
            rnd(out["W"])
            k += 1
        return ubytes * k / (time.perf_counter() - t0) / 1e9, k

    def qr_leg(budget):
        k = 0
        t0 = time.perf_counter()
        while k < 2 or time.perf_counter() - t0 < budget:
            oracle.haar_qr(Om_U if k % 2 == 0 else Om_V)
            k += 1
        return (time.perf_counter() - t0) / k * 1e3, k

    pl, nb = plinear_leg(budget_s * 0.45, 4096)
    ug, nu = update_leg(budget_s * 0.15)
    qm, nq = qr_leg(budget_s * 0.1)
    one = None
    if threadpool_limits is not None:
        with threadpool_limits(limits=1, user_api="blas"):
            pl1, nb1 = plinear_leg(budget_s * 0.15, 4096)
            ug1, nu1 = update_leg(budget_s * 0.08)
            qm1, nq1 = qr_leg(budget_s * 0.07)
        one = {"value": pl1, "update_gbs": round(ug1, 3), "qr_ms_per_panel": round(qm1, 2),
               "sample": f"{nb1} query blocks, {nu1} updates, {nq1} panels"}
    what = ("materialised A', B' and W + scale B' A', then X W'^T" if lora
            else "materialised W + s eps U Z V^T, then X W'^T")
    return {"value": pl, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "cores_visible": len(os.sched_getaffinity(0)),
            "update_gbs": round(ug, 3), "qr_ms_per_panel": round(qm, 2),
            "one_thread": one,
            "sample": f"float64 oracle: perturbed linear ({what}) on {nb} query blocks x {S} token rows of "
                      f"the {m}x{n} layer, algorithmic FLOPs / time; update (Zbar, Adam, W - lr U S V^T, "
                      f"rounding to the stored type) of {'the ' + str(rl) + 'x' + str(n) + ' adapter factor A' if lora else 'that matrix'} {nu} times, algorithmic bytes {ubytes} each / time; "
                      f"Householder QR with sign fix of the {m}x{r} and {n}x{r} panels, {nq} panels; "
                      f"cores = BLAS threads used; one_thread = the same legs with one BLAS thread"}


def attention_flops(T, seq_len, heads, dh, nblk):
    """Algorithmic FLOPs of causal attention per layer: q.k and p.v for the L(L+1)/2 visible
    (query, key) pairs of each sequence and head, in every block."""
    return nblk * (T // seq_len) * heads * 2 * 2 * dh * seq_len * (seq_len + 1) // 2


def run_decoder(args):
    """One SubZero+ step through real decoder layers: refresh (t mod F == 0), for every layer the
    forward of all 2q blocks (OPT family, zo_decoder_layer_forward: layer norm, the six perturbed
    linears with fused ReLU / residuals, causal attention; LLaMA family, zo_llama_layer_forward:
    RMS norm, rotary positions, the seven perturbed linears with the SwiGLU product and the
    residuals fused), the squared loss of the last hidden state against a fixed target, the
    estimate, and the subspace Adam update of every matrix of every layer."""
    import numpy as np
    import torch

    import paper_2608_15665_amd as zo
    import zo_draws as zd

    cfg = zd.CONFIGS[args.config]
    dec = cfg.get("decoder")
    if not dec:
        print(f"bench.py: --model decoder has no layer shape for {args.config}", file=sys.stderr)
        sys.exit(2)
    if dec.get("family") == "llama-lora":
        return run_decoder_lora(args, cfg, dec)
    llama = dec.get("family") == "llama"
    T, r, q = cfg["T"], cfg["r"], cfg["q"]
    if args.queries:
        q = args.queries
    if args.rank:
        r = args.rank
    d, heads, ffn, L = dec["d"], dec["heads"], dec["ffn"], dec["seq_len"]
    layers = cfg["layers"]
    forward = args.estimator == "forward"
    if forward:
        bq, bs = [0] + list(range(q)), [0] + [1] * q
    else:
        bq, bs = [b // 2 for b in range(2 * q)], [1 if b % 2 == 0 else -1 for b in range(2 * q)]
    nblk = len(bq)
    nsigned = sum(1 for v in bs if v != 0)
    eps, lr, b1, b2, ea, F = cfg["eps"], cfg["lr"], cfg["beta1"], cfg["beta2"], cfg["eps_adam"], cfg["F"]
    seed, dev = args.seed, "cuda"
    f16 = args.dtype == "fp16"
    dt16 = torch.float16 if f16 else torch.bfloat16
    t_setup = time.perf_counter()

    def to16(a64):
        if f16:
            return torch.from_numpy(zd.as_f16_values(a64)[0]).to(dev)
        return torch.from_numpy(zd.bf16_bits(zd.f32(a64)).view(np.int16)).view(dt16).to(dev)

    if llama:
        shapes = {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d), "gate": (ffn, d), "up": (ffn, d),
                  "down": (d, ffn)}
    else:
        shapes = {"q": (d, d), "k": (d, d), "v": (d, d), "o": (d, d), "fc1": (ffn, d), "fc2": (d, ffn)}
    nper = len(shapes)
    Wbase = {sh: to16(zd.draw(seed, "W0", sh, sh, 0.02)) for sh in set(shapes.values())}
    rows_set = sorted({d, ffn})
    Obase = {rw: torch.from_numpy(zd.f32(zd.draw(seed, "OMEGA_U", (rw, r), (rw, r)))).to(dev) for rw in rows_set}
    nsteps = args.warmup + args.steps
    mats, omegas, qouts, lns = [], [], [], []
    for l in range(layers):
        lm = {}
        for nm, (m, n) in shapes.items():
            idx = len(mats) * nper + len(lm)
            u = dict(W=torch.roll(Wbase[(m, n)], l, 0).contiguous(),
                     U=torch.empty((m, r), dtype=torch.float32, device=dev),
                     V=torch.empty((n, r), dtype=torch.float32, device=dev),
                     M1=torch.zeros((r, r), dtype=torch.float32, device=dev),
                     M2=torch.zeros((r, r), dtype=torch.float32, device=dev), m=m, n=n)
            for key, rw in (("U", m), ("V", n)):
                omegas.append(torch.roll(Obase[rw], 2 * idx + (key == "V"), 0).contiguous())
                qouts.append(u[key])
            lm[nm] = u
        mats.append(lm)
        g = torch.from_numpy(zd.f32(1.0 + 0.05 * zd.draw(seed, "W0", (l, 1), (4, d)))).to(dev)
        if llama:
            lns.append(dict(rms1_gamma=g[0].contiguous(), rms2_gamma=g[2].contiguous()))
        else:
            lns.append(dict(ln1_gamma=g[0].contiguous(), ln1_beta=(g[1] - 1.0).contiguous(),
                            ln2_gamma=g[2].contiguous(), ln2_beta=(g[3] - 1.0).contiguous()))
    del Wbase, Obase
    nmat = nper * layers
    zfeed = ZFeed(seed, nmat, q, r, dev)
    Z = zfeed.dev  # [slot][matrix, q, r, r]
    H0 = to16(zd.draw(seed, "X", (T, d, 0), (T, d)))
    Ystar = to16(zd.draw(seed, "X", (T, d, 1), (T, d)))
    Hbuf = [torch.empty((nblk * T, d), dtype=dt16, device=dev) for _ in range(2)]

    def layer_obj(t, l):
        lm = {nm: dict(W=u["W"], U=u["U"], V=u["V"], Z=Z[t][nper * l + i])
              for i, (nm, u) in enumerate(mats[l].items())}
        if llama:
            return zo.LlamaLayer(lm, lns[l], bq, bs, eps, T, L, heads)
        return zo.DecoderLayer(lm, lns[l], bq, bs, eps, T, L, heads)

    decs = [[layer_obj(sl, l) for l in range(layers)] for sl in range(2)]
    items = [[dict(W=u["W"], U=u["U"], V=u["V"], Z=Z[sl][nper * l + i], M1=u["M1"], M2=u["M2"])
              for l in range(layers) for i, u in enumerate(mats[l].values())] for sl in range(2)]
    torch.cuda.synchronize()
    log(f"setup {time.perf_counter() - t_setup:.1f} s; {layers} decoder layers; "
        f"{torch.cuda.memory_allocated() / 2**30:.1f} GiB on device")
    Ev = lambda: torch.cuda.Event(enable_timing=True)
    recs = []

    def step(t, s):
        rec = {"layers": [], "upd": None, "refresh": None}
        s = zfeed.acquire(s)
        if t % F == 0:
            e0, e1 = Ev(), Ev()
            e0.record()
            zo.subspace_refresh(omegas, r, out=qouts)
            e1.record()
            rec["refresh"] = (e0, e1)
        H = H0
        for l in range(layers):
            e0, e1 = Ev(), Ev()
            e0.record()
            H = decs[s][l](H, out=Hbuf[l % 2])
            e1.record()
            rec["layers"].append((e0, e1))
        Lb = zo.sq_loss(H, Ystar, nblk, T)
        g = zo.combine_forward(Lb, eps) if forward else zo.combine_central(Lb, eps)
        e0, e1 = Ev(), Ev()
        e0.record()
        zo.subspace_adam_update(items[s], g, t + 1, lr, b1, b2, ea)
        e1.record()
        zfeed.release(s)
        rec["upd"] = (e0, e1)
        return rec

    for s in range(args.warmup):
        step(s, s)
        torch.cuda.synchronize()
        log(f"warmup step {s} done")
    for lm in mats:
        for u in lm.values():
            u["M1"].zero_()
            u["M2"].zero_()
    zfeed.request(args.warmup)
    torch.cuda.synchronize()
    args.clk.active.set()
    t0 = time.perf_counter()
    for k in range(args.steps):
        recs.append(step(k, args.warmup + k))
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    args.clk.active.clear()
    log(f"timed {args.steps} steps in {t1 - t0:.2f} s")
    sclk = args.clk.result()
    draws = zfeed.report(range(args.warmup, args.warmup + args.steps))

    lin_layer = sum(plinear_flops(T, m, n, r, q, nblk, nsigned) for m, n in shapes.values())
    att_layer = attention_flops(T, L, heads, d // heads, nblk)
    lin_step = lin_layer * layers
    value = lin_step * args.steps / (t1 - t0) / 1e12
    layer_ms = [a.elapsed_time(b) for rc in recs for a, b in rc["layers"]]
    avg_layer = sum(layer_ms) / len(layer_ms)
    achieved = (lin_layer + att_layer) / (avg_layer * 1e-3) / 1e12
    upd_ms = sum(rc["upd"][0].elapsed_time(rc["upd"][1]) for rc in recs)
    upd_bytes = sum(update_bytes(u["m"], u["n"], r, q) for lm in mats for u in lm.values()) * args.steps
    upd_gbps = upd_bytes / (upd_ms * 1e-3) / 1e9
    ref_ms = [rc["refresh"][0].elapsed_time(rc["refresh"][1]) for rc in recs if rc["refresh"]]
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round((t1 - t0) / args.steps * 1e3, 2), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": args.dtype, "data": "synthetic",
        "config": {"workload": (f"{args.config}-shaped decoder: {layers} "
                                + ("pre-norm LLaMA-family layers (RMS norm, rotary positions, " if llama
                                   else "pre-LN layers (")
                                + f"d={d}, {heads} heads of {d // heads}, ffn={ffn}, "
                                + ("SwiGLU), every q, k, v, o, gate, up, down perturbed; " if llama
                                   else "ReLU), every q, k, v, o, fc1, fc2 perturbed; ")
                                + (f"{nblk} blocks (baseline + q={q} forward queries)" if forward
                                   else f"{nblk} query blocks (q={q}, +/-)")
                                + f" of T={T} tokens ({T // L} sequences x {L}); r={r}; {args.dtype}; "
                                  "value counts the perturbed-linear FLOPs of the step"),
                   "layers": layers, "d": d, "heads": heads, "ffn": ffn, "seq_len": L, "T": T, "r": r, "q": q,
                   "blocks": nblk, "estimator": args.estimator, "refresh_every": F},
        "roofline": {"kernel": ("zo_llama_layer_forward (one layer: 2 RMS norms, 2 rotations, 7 fused "
                                "perturbed GEMMs with their projections, causal attention)" if llama else
                                "zo_decoder_layer_forward (one layer: 2 layer norms, 6 fused perturbed GEMMs "
                                "with their projections, causal attention)"), "bound": "mfma",
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None,
                     "launches": len(layer_ms), "avg_launch_ms": round(avg_layer, 4),
                     "flops_per_launch_avg": lin_layer + att_layer, **clock_fields(achieved, sclk)},
        "sclk_timed_window": sclk,
        "host_draws": draws,
        "attention_flops_per_layer": att_layer,
        "update": {"kernel": "zo_subspace_adam_update (k_adam_rr + k_us + k_update_bf16)", "bound": "hbm",
                   "achieved": round(upd_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                   "frac": round(upd_gbps / PEAK_HBM_GBPS, 4), "ms_per_step": round(upd_ms / args.steps, 3)},
        "refresh_ms": round(ref_ms[0], 3) if ref_ms else None,
    }
    print(json.dumps(out), flush=True)


def run_decoder_lora(args, cfg, dec):
    """The decoder step of the LoRA scheme (Qwen-shaped LLaMA-family layers with grouped
    key/value heads): refresh of every adapter factor's subspace (t mod F == 0), the forward of
    all 2q blocks through every layer (zo_llama_lora_layer_forward: frozen k, o, gate, up, down;
    adapted q and v with both factors perturbed), the loss and estimate, and the subspace Adam
    update of the adapter factors (fp32)."""
    import numpy as np
    import torch

    import paper_2608_15665_amd as zo
    import zo_draws as zd

    T, r, q = cfg["T"], cfg["r"], cfg["q"]
    if args.queries:
        q = args.queries
    if args.rank:
        r = args.rank
    d, heads, kv, ffn, L = dec["d"], dec["heads"], dec["kv_heads"], dec["ffn"], dec["seq_len"]
    dkv = d // heads * kv
    rl, scale = zd.QWEN_LORA_RANK, zd.QWEN_LORA_ALPHA / zd.QWEN_LORA_RANK
    layers = cfg["layers"]
    forward = args.estimator == "forward"
    if forward:
        bq, bs = [0] + list(range(q)), [0] + [1] * q
    else:
        bq, bs = [b // 2 for b in range(2 * q)], [1 if b % 2 == 0 else -1 for b in range(2 * q)]
    nblk = len(bq)
    nsigned = sum(1 for v in bs if v != 0)
    eps, lr, b1, b2, ea, F = cfg["eps"], cfg["lr"], cfg["beta1"], cfg["beta2"], cfg["eps_adam"], cfg["F"]
    seed, dev = args.seed, "cuda"
    f16 = args.dtype == "fp16"
    dt16 = torch.float16 if f16 else torch.bfloat16
    t_setup = time.perf_counter()

    def to16(a64):
        if f16:
            return torch.from_numpy(zd.as_f16_values(a64)[0]).to(dev)
        return torch.from_numpy(zd.bf16_bits(zd.f32(a64)).view(np.int16)).view(dt16).to(dev)

    f32dev = lambda a64: torch.from_numpy(zd.f32(a64)).to(dev)
    shapes = {"q": (d, d), "k": (dkv, d), "v": (dkv, d), "o": (d, d), "gate": (ffn, d), "up": (ffn, d),
              "down": (d, ffn)}
    Wbase = {sh: to16(zd.draw(seed, "W0", sh, sh, 0.02)) for sh in set(shapes.values())}
    Obase = {rw: f32dev(zd.draw(seed, "OMEGA_U", (rw, r), (rw, r))) for rw in sorted({d, dkv, rl})}
    zeros_rr = lambda: torch.zeros((r, r), dtype=torch.float32, device=dev)
    nsteps = args.warmup + args.steps
    mats, factors, omegas, qouts, norms = [], [], [], [], []
    for l in range(layers):
        lm = {nm: dict(W=torch.roll(Wbase[sh], l, 0).contiguous()) for nm, sh in shapes.items()}
        for nm in ("q", "v"):
            m = shapes[nm][0]
            u = lm[nm]
            k = len(factors)
            u["A"] = f32dev(zd.draw(seed, "LORA_A", (l, nm == "v"), (rl, d), 0.02))
            u["B"] = torch.zeros((m, rl), dtype=torch.float32, device=dev)  # the usual LoRA start
            for key, rw in (("UA", rl), ("VA", d), ("UB", m), ("VB", rl)):
                omegas.append(torch.roll(Obase[rw], len(omegas), 0).contiguous())
                u[key] = torch.empty((rw, r), dtype=torch.float32, device=dev)
                qouts.append(u[key])
            factors.append(dict(W=u["A"], U=u["UA"], V=u["VA"], M1=zeros_rr(), M2=zeros_rr(), m=rl, n=d, z=k))
            factors.append(dict(W=u["B"], U=u["UB"], V=u["VB"], M1=zeros_rr(), M2=zeros_rr(), m=m, n=rl, z=k + 1))
            u["zi"] = k
        mats.append(lm)
        g = f32dev(1.0 + 0.05 * zd.draw(seed, "W0", (l, 1), (2, d)))
        norms.append(dict(rms1_gamma=g[0].contiguous(), rms2_gamma=g[1].contiguous()))
    del Wbase, Obase
    zfeed = ZFeed(seed, len(factors), q, r, dev)
    Z = zfeed.dev  # [slot][factor, q, r, r]
    H0 = to16(zd.draw(seed, "X", (T, d, 0), (T, d)))
    Ystar = to16(zd.draw(seed, "X", (T, d, 1), (T, d)))
    Hbuf = [torch.empty((nblk * T, d), dtype=dt16, device=dev) for _ in range(2)]
    ws = None

    def layer_obj(t, l):
        nonlocal ws
        lm = {}
        for nm, u in mats[l].items():
            if nm in ("q", "v"):
                lm[nm] = dict(W=u["W"], A=u["A"], UA=u["UA"], VA=u["VA"], ZA=Z[t][u["zi"]], B=u["B"], UB=u["UB"],
                              VB=u["VB"], ZB=Z[t][u["zi"] + 1])
            else:
                lm[nm] = dict(W=u["W"])
        o = zo.LlamaLoraLayer(lm, norms[l], bq, bs, eps, scale, T, L, heads, kv, rope_base=dec["rope_base"],
                              workspace=ws)
        ws = o.ws
        return o

    decs = [[layer_obj(sl, l) for l in range(layers)] for sl in range(2)]
    items = [[dict(W=f["W"], U=f["U"], V=f["V"], Z=Z[sl][f["z"]], M1=f["M1"], M2=f["M2"]) for f in factors]
             for sl in range(2)]
    torch.cuda.synchronize()
    log(f"setup {time.perf_counter() - t_setup:.1f} s; {layers} LoRA-scheme layers; "
        f"{torch.cuda.memory_allocated() / 2**30:.1f} GiB on device")
    Ev = lambda: torch.cuda.Event(enable_timing=True)
    recs = []

    def step(t, s):
        rec = {"layers": [], "upd": None, "refresh": None}
        s = zfeed.acquire(s)
        if t % F == 0:
            e0, e1 = Ev(), Ev()
            e0.record()
            zo.subspace_refresh(omegas, r, out=qouts)
            e1.record()
            rec["refresh"] = (e0, e1)
        H = H0
        for l in range(layers):
            e0, e1 = Ev(), Ev()
            e0.record()
            H = decs[s][l](H, out=Hbuf[l % 2])
            e1.record()
            rec["layers"].append((e0, e1))
        Lb = zo.sq_loss(H, Ystar, nblk, T)
        g = zo.combine_forward(Lb, eps) if forward else zo.combine_central(Lb, eps)
        e0, e1 = Ev(), Ev()
        e0.record()
        zo.subspace_adam_update(items[s], g, t + 1, lr, b1, b2, ea)
        e1.record()
        zfeed.release(s)
        rec["upd"] = (e0, e1)
        return rec

    for s in range(args.warmup):
        step(s, s)
        torch.cuda.synchronize()
        log(f"warmup step {s} done")
    for f in factors:
        f["M1"].zero_()
        f["M2"].zero_()
    zfeed.request(args.warmup)
    torch.cuda.synchronize()
    args.clk.active.set()
    t0 = time.perf_counter()
    for k in range(args.steps):
        recs.append(step(k, args.warmup + k))
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    args.clk.active.clear()
    log(f"timed {args.steps} steps in {t1 - t0:.2f} s")
    sclk = args.clk.result()
    draws = zfeed.report(range(args.warmup, args.warmup + args.steps))

    lin_layer = (lora_flops(T, d, d, rl, r, q, nblk, nsigned) + lora_flops(T, dkv, d, rl, r, q, nblk, nsigned)
                 + sum(nblk * 2 * T * m * n for nm, (m, n) in shapes.items() if nm not in ("q", "v")))
    att_layer = attention_flops(T, L, heads, d // heads, nblk)
    value = lin_layer * layers * args.steps / (t1 - t0) / 1e12
    layer_ms = [a.elapsed_time(b) for rc in recs for a, b in rc["layers"]]
    avg_layer = sum(layer_ms) / len(layer_ms)
    achieved = (lin_layer + att_layer) / (avg_layer * 1e-3) / 1e12
    upd_ms = sum(rc["upd"][0].elapsed_time(rc["upd"][1]) for rc in recs)
    upd_bytes = sum(update_bytes(f["m"], f["n"], r, q, 4) for f in factors) * args.steps
    upd_gbps = upd_bytes / (upd_ms * 1e-3) / 1e9
    ref_ms = [rc["refresh"][0].elapsed_time(rc["refresh"][1]) for rc in recs if rc["refresh"]]
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round((t1 - t0) / args.steps * 1e3, 2), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": args.dtype, "data": "synthetic",
        "config": {"workload": (f"{args.config}-shaped decoder: {layers} LLaMA-family layers of the LoRA scheme "
                                f"(RMS norm, rotary positions base {dec['rope_base']:g}, d={d}, {heads} query heads "
                                f"over {kv} key/value heads of {d // heads}, ffn={ffn}, SwiGLU), frozen k, o, gate, up, "
                                f"down, adapters r_L={rl} (scale {scale:g}) on q and v with both factors perturbed; "
                                + (f"{nblk} blocks (baseline + q={q} forward queries)" if forward
                                   else f"{nblk} query blocks (q={q}, +/-)")
                                + f" of T={T} tokens ({T // L} sequences x {L}); r={r}; {args.dtype}; value counts "
                                  "the linear-layer FLOPs of the step (adapted at rank r_L + r, frozen plain)"),
                   "layers": layers, "d": d, "heads": heads, "kv_heads": kv, "ffn": ffn, "seq_len": L, "T": T,
                   "lora_rank": rl, "r": r, "q": q, "blocks": nblk, "estimator": args.estimator, "refresh_every": F},
        "roofline": {"kernel": "zo_llama_lora_layer_forward (one layer: 2 RMS norms, 2 rotations, 2 adapted and 5 "
                               "frozen fused GEMMs, grouped causal attention)", "bound": "mfma",
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None,
                     "launches": len(layer_ms), "avg_launch_ms": round(avg_layer, 4),
                     "flops_per_launch_avg": lin_layer + att_layer, **clock_fields(achieved, sclk)},
        "sclk_timed_window": sclk,
        "host_draws": draws,
        "attention_flops_per_layer": att_layer,
        "update": {"kernel": "zo_subspace_adam_update on the fp32 adapter factors (latency-bound)", "bound": "hbm",
                   "achieved": round(upd_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                   "frac": round(upd_gbps / PEAK_HBM_GBPS, 4), "ms_per_step": round(upd_ms / args.steps, 3)},
        "refresh_ms": round(ref_ms[0], 3) if ref_ms else None,
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="opt-13b", choices=["opt-1.3b", "llama-7b", "opt-13b", "qwen-32b-lora"])
    ap.add_argument("--estimator", default="central", choices=["central", "forward"],
                    help="central: 2q blocks (+/-); forward: a baseline block and q perturbed blocks (Eq. 6)")
    ap.add_argument("--queries", type=int, default=0, help="queries per step (default: the config's q)")
    ap.add_argument("--rank", type=int, default=0, help="subspace rank r (default: the config's r)")
    ap.add_argument("--dtype", default="bf16", choices=["bf16", "fp16"],
                    help="weights and activations (fp16: the paper's precision for OPT-13B)")
    ap.add_argument("--model", default="stack", choices=["stack", "decoder"],
                    help="stack: the perturbed linears of every matrix on synthetic activations; decoder: "
                         "real decoder-layer forwards (OPT: layer norm, causal attention, ReLU MLP; llama-7b: "
                         "RMS norm, rotary positions, causal attention, SwiGLU MLP; qwen-32b-lora: the same with "
                         "grouped key/value heads, a frozen base and perturbed adapters on q and v; residuals)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle work for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the library GEMM / copy / read-modify-write reference timings")
    ap.add_argument("--copy-calibration", action="store_true", help="run only a 1 GiB device copy (counter scale)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU only (got --gpus {args.gpus}); the multi-GPU "
              "path (sharding by query, one all-gather of 2q losses per step) is a design, not built.",
              file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2608_15665_amd as zo
    import zo_draws as zd

    if args.copy_calibration:
        copy_calibration()
        return
    torch.cuda.set_device(0)
    zo.lib()
    args.clk = clk = ClockSampler()
    if args.model == "decoder":
        run_decoder(args)
        return
    cfg = zd.CONFIGS[args.config]
    lora = args.config.endswith("-lora")
    T, r, q = cfg["T"], cfg["r"], cfg["q"]
    if args.queries:
        q = args.queries
    if args.rank:
        r = args.rank
    forward = args.estimator == "forward"
    # Query blocks: central -- (j, +), (j, -); forward -- the baseline (sign 0), then (j, +).
    if forward:
        bq, bs = [0] + list(range(q)), [0] + [1] * q
    else:
        bq, bs = [b // 2 for b in range(2 * q)], [1 if b % 2 == 0 else -1 for b in range(2 * q)]
    nblk = len(bq)
    nsigned = sum(1 for v in bs if v != 0)
    L = cfg["layers"]
    eps, lr, b1, b2, ea, F = cfg["eps"], cfg["lr"], cfg["beta1"], cfg["beta2"], cfg["eps_adam"], cfg["F"]
    rl, scale = zd.QWEN_LORA_RANK, zd.QWEN_LORA_ALPHA / zd.QWEN_LORA_RANK
    seed = args.seed
    dev = "cuda"
    f16 = args.dtype == "fp16"
    dt16 = torch.float16 if f16 else torch.bfloat16
    zdt = zo.ZO_F16 if f16 else zo.ZO_BF16
    t_setup = time.perf_counter()

    def to_bf16(a64):
        """A float64 host draw as a device tensor of the run's 16-bit type."""
        if f16:
            return torch.from_numpy(zd.as_f16_values(a64)[0]).to(dev)
        bits = zd.bf16_bits(zd.f32(a64))
        return torch.from_numpy(bits.view(np.int16)).view(dt16).to(dev)

    def f32dev(a64):
        return torch.from_numpy(zd.f32(a64)).to(dev)

    # The perturbed matrices: every weight (full tuning) or the adapted q and v projections (LoRA).
    unit_mats = [mt for mt in cfg["mats"] if not lora or mt[0] in ("q", "v")]
    # Weights: one host draw per distinct shape; layer l holds it rolled by l rows (device side).
    shapes = sorted({(m, n) for _, m, n in unit_mats})
    Wbase = {sh: to_bf16(zd.draw(seed, "W0", sh, sh, 0.02)) for sh in shapes}
    # Activations: one base block per distinct n; block b rolled by b*floor(T/nblk) rows.
    ns = sorted({n for _, _, n in unit_mats})
    X = {}
    for n in ns:
        x0 = to_bf16(zd.draw(seed, "X", (T, n, 0), (T, n)))
        X[n] = torch.cat([torch.roll(x0, b * (T // nblk), 0) for b in range(nblk)]).contiguous()
        del x0
    Y = {m: torch.empty((nblk * T, m), dtype=dt16, device=dev) for m in sorted({m for _, m, _ in unit_mats})}
    rows_set = sorted({m for _, m, _ in unit_mats} | set(ns) | ({rl} if lora else set()))
    Obase = {rw: f32dev(zd.draw(seed, "OMEGA_U", (rw, r), (rw, r))) for rw in rows_set}
    zeros_rr = lambda: torch.zeros((r, r), dtype=torch.float32, device=dev)
    units, omegas, qouts = [], [], []
    for l in range(L):
        for name, m, n in unit_mats:
            idx = len(units)
            u = dict(name=f"{name}{l}", m=m, n=n, W=torch.roll(Wbase[(m, n)], l, 0).contiguous())
            # Panels (rows x r Gaussian inputs of the refresh) and their Haar factors.
            prow = [("UA", rl), ("VA", n), ("UB", m), ("VB", rl)] if lora else [("U", m), ("V", n)]
            for k, (key, rw) in enumerate(prow):
                omegas.append(torch.roll(Obase[rw], len(prow) * idx + k, 0).contiguous())
                u[key] = torch.empty((rw, r), dtype=torch.float32, device=dev)
                qouts.append(u[key])
            if lora:
                u["A"] = f32dev(zd.draw(seed, "LORA_A", (idx,), (rl, n), 0.02))
                u["B"] = torch.zeros((m, rl), dtype=torch.float32, device=dev)  # the usual LoRA start
                u["mom"] = [(zeros_rr(), zeros_rr()), (zeros_rr(), zeros_rr())]
            else:
                u["mom"] = [(zeros_rr(), zeros_rr())]
            units.append(u)
    del Wbase, Obase
    zper = 2 if lora else 1  # coefficient sets per unit (one per perturbed factor)
    zfeed = ZFeed(seed, zper * len(units), q, r, dev)
    Z = zfeed.dev  # [slot][factor, q, r, r]
    m_last = unit_mats[-1][1]
    Ystar = to_bf16(zd.draw(seed, "X", (T, m_last, 1), (T, m_last)))
    if lora:
        ws_need = max(zo.lib().zo_lora_perturbed_linear_workspace(T, m, n, rl, r, q, nblk, T * n, zdt)
                      for m, n in shapes)
    else:
        ws_need = max(zo.lib().zo_perturbed_linear_workspace(T, m, n, r, q, nblk, T * n, zdt)
                      for m, n in shapes)
    # q, k and v of a layer read the same input: their prepares run as one group (one pass
    # over X), so each keeps its own workspace until its apply.
    grouped = not lora and [nm for nm, _, _ in unit_mats][:3] == ["q", "k", "v"]
    wsets = [torch.empty(ws_need, dtype=torch.uint8, device=dev) for _ in range(3 if grouped else 1)]
    ws = wsets[0]
    gws = None
    if grouped:
        gneed = zo.lib().zo_perturbed_linear_group_workspace(3, T, unit_mats[0][2], r, q, nblk, T * unit_mats[0][2], zdt)
        gws = torch.empty(max(gneed, 1), dtype=torch.uint8, device=dev)

    def make_layer(t, i, u):
        if lora:
            return zo.LoraPerturbedLinear(X[u["n"]], u["W"], u["A"], u["UA"], u["VA"], Z[t][2 * i], u["B"], u["UB"],
                                          u["VB"], Z[t][2 * i + 1], bq, bs, eps, scale, T,
                                          x_block_stride=T * u["n"], Y=Y[u["m"]], workspace=ws)
        k = i % len(unit_mats)
        return zo.PerturbedLinear(X[u["n"]], u["W"], u["U"], u["V"], Z[t][i], bq, bs, eps, T,
                                  x_block_stride=T * u["n"], Y=Y[u["m"]],
                                  workspace=wsets[k] if grouped and k < 3 else ws)

    def make_items(t, i, u):
        if lora:
            (a1, a2), (c1, c2) = u["mom"]
            return [dict(W=u["A"], U=u["UA"], V=u["VA"], Z=Z[t][2 * i], M1=a1, M2=a2),
                    dict(W=u["B"], U=u["UB"], V=u["VB"], Z=Z[t][2 * i + 1], M1=c1, M2=c2)]
        (m1, m2), = u["mom"]
        return [dict(W=u["W"], U=u["U"], V=u["V"], Z=Z[t][i], M1=m1, M2=m2)]

    plins = [[make_layer(sl, i, u) for i, u in enumerate(units)] for sl in range(2)]
    items = [[it for i, u in enumerate(units) for it in make_items(sl, i, u)] for sl in range(2)]
    torch.cuda.synchronize()
    log(f"setup {time.perf_counter() - t_setup:.1f} s; {len(units)} perturbed layers; "
        f"{torch.cuda.memory_allocated() / 2**30:.1f} GiB on device")

    Ev = lambda: torch.cuda.Event(enable_timing=True)
    recs = []

    def step(t, s):
        """One SubZero+ step; s keys the step's Z draws (step t of the run)."""
        rec = {"gemm": [], "prep": [], "upd": None, "refresh": None}
        s = zfeed.acquire(s)
        if t % F == 0:
            e0, e1 = Ev(), Ev()
            e0.record()
            zo.subspace_refresh(omegas, r, out=qouts)
            e1.record()
            rec["refresh"] = (e0, e1)
        i = 0
        while i < len(units):
            g = 3 if grouped and i % len(unit_mats) == 0 else 1
            e0, e1 = Ev(), Ev()
            e0.record()
            if g == 3:
                zo.prepare_group(plins[s][i:i + 3], gws)
            else:
                plins[s][i].prepare()
            e1.record()
            rec["prep"].append((e0, e1))
            for k in range(i, i + g):
                mt = units[k]
                a0, a1 = Ev(), Ev()
                a0.record()
                plins[s][k].apply()
                a1.record()
                rec["gemm"].append((a0, a1, mt["m"], mt["n"]))
            i += g
        Lb = zo.sq_loss(Y[m_last], Ystar, nblk, T)
        g = zo.combine_forward(Lb, eps) if forward else zo.combine_central(Lb, eps)
        e0, e1 = Ev(), Ev()
        e0.record()
        zo.subspace_adam_update(items[s], g, t + 1, lr, b1, b2, ea)
        e1.record()
        zfeed.release(s)
        rec["upd"] = (e0, e1)
        return rec

    # Warm-up runs steps t = 0.. (t = 0 refreshes U, V); the moments are then reset and the
    # timed steps run t = 0..K-1 again, so the timed window holds exactly one refresh.
    for s in range(args.warmup):
        step(s, s)
        torch.cuda.synchronize()
        log(f"warmup step {s} done")
    for u in units:
        for m1, m2 in u["mom"]:
            m1.zero_()
            m2.zero_()
    zfeed.request(args.warmup)
    torch.cuda.synchronize()
    clk.active.set()
    t0 = time.perf_counter()
    for k in range(args.steps):
        recs.append(step(k, args.warmup + k))
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    clk.active.clear()
    log(f"timed {args.steps} steps in {t1 - t0:.2f} s")
    sclk = clk.result()
    draws = zfeed.report(range(args.warmup, args.warmup + args.steps))
    draws["omega"] = omega_host_draw(seed, [rw for o in omegas for rw in [o.shape[0]]], r, F)

    if lora:
        layer_flops = lambda m, n: lora_flops(T, m, n, rl, r, q, nblk, nsigned)
        launch_flops = lambda m, n: lora_apply_flops(T, m, n, rl, r, q, nblk, nsigned)
        unit_bytes = lambda m, n: update_bytes(rl, n, r, q, 4) + update_bytes(m, rl, r, q, 4)
    else:
        layer_flops = lambda m, n: plinear_flops(T, m, n, r, q, nblk, nsigned)
        launch_flops = lambda m, n: apply_flops(T, m, n, r, q, nblk, nsigned)
        unit_bytes = lambda m, n: update_bytes(m, n, r, q)
    step_flops = sum(layer_flops(u["m"], u["n"]) for u in units)
    value = step_flops * args.steps / (t1 - t0) / 1e12
    gemm_ms = sum(a.elapsed_time(b) for rc in recs for a, b, _, _ in rc["gemm"])
    gemm_flops = sum(launch_flops(m, n) for rc in recs for _, _, m, n in rc["gemm"])
    n_gemm = sum(len(rc["gemm"]) for rc in recs)
    prep_ms = sum(a.elapsed_time(b) for rc in recs for a, b in rc["prep"])
    upd_ms = sum(rc["upd"][0].elapsed_time(rc["upd"][1]) for rc in recs)
    upd_bytes = sum(unit_bytes(u["m"], u["n"]) for u in units) * args.steps
    ref_ms = [rc["refresh"][0].elapsed_time(rc["refresh"][1]) for rc in recs if rc["refresh"]]
    per_shape = {}
    for rc in recs:
        for a, b, m, n in rc["gemm"]:
            d = per_shape.setdefault(f"{m}x{n}", [0.0, 0.0, 0])
            d[0] += a.elapsed_time(b)
            d[1] += launch_flops(m, n)
            d[2] += 1
    achieved = gemm_flops / (gemm_ms * 1e-3) / 1e12
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        tr = json.load(open(TRAFFIC_FILE))
        key = f"{args.config}/{args.estimator}/q={q}/r={r}/{args.dtype}"
        if tr.get("source_hash") == source_hash() and tr.get("workload_key") == key:
            traffic = tr.get("bytes_per_launch")
    upd_gbps = upd_bytes / (upd_ms * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round((t1 - t0) / args.steps * 1e3, 2), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": args.dtype, "data": "synthetic",
        "config": {"workload": (f"{args.config}-shaped stack: {L} layers x "
                                + ", ".join(f"{nm} {m}x{n}" for nm, m, n in unit_mats)
                                + (f" (frozen {args.dtype} base, fp32 LoRA adapter r_L={rl}, alpha={int(scale * rl)}, "
                                   f"each factor in its own subspace)" if lora else "")
                                + (f"; {nblk} blocks (baseline + q={q} forward queries)" if forward
                                   else f"; {nblk} query blocks (q={q}, +/-)")
                                + f" of T={T} tokens; r={r}; {args.dtype} W and X"),
                   "layers": L, "perturbed_layers": len(units), "T": T, "r": r, "q": q, "blocks": nblk,
                   "estimator": args.estimator,
                   "refresh_every": F},
        "roofline": {"kernel": "k_gemm_main (zo_perturbed_linear_apply)", "bound": "mfma",
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic,
                     "launches": n_gemm, "avg_launch_ms": round(gemm_ms / n_gemm, 4),
                     "flops_per_launch_avg": gemm_flops / n_gemm, **clock_fields(achieved, sclk)},
        "sclk_timed_window": sclk,
        "host_draws": draws,
        "update": {"kernel": "zo_subspace_adam_update (k_adam_rr + k_us + "
                             + ("k_update_f32, fp32 adapter factors)" if lora else "k_update_bf16)"), "bound": "hbm",
                   "achieved": round(upd_gbps, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                   "frac": round(upd_gbps / PEAK_HBM_GBPS, 4), "ms_per_step": round(upd_ms / args.steps, 3)},
        "prepare_ms_per_step": round(prep_ms / args.steps, 3),
        "refresh_ms": round(ref_ms[0], 3) if ref_ms else None,
        "gemm_by_shape": {k: {"tflops": round(v[1] / (v[0] * 1e-3) / 1e12, 1), "avg_ms": round(v[0] / v[2], 3)}
                          for k, v in per_shape.items()},
    }
    del plins, items, X, Y, ws, units
    torch.cuda.empty_cache()
    if not args.no_peaks:
        _, m0, n0 = unit_mats[0]
        out["practical_peaks"] = practical_peaks(T, nblk, m0, n0, r, q, dt16)
        if not lora:
            tc = zd.TINY
            out["shared_x"] = [
                shared_x_report(seed, T, m0, n0, r, q, nblk, dt16, "first layer's q/k/v shape"),
                shared_x_report(seed, tc["T"], tc["m"], tc["n"], tc["r"], tc["q"], 2 * tc["q"], torch.float32,
                                "Tiny layer")]
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, seed, args.cpu_budget, unit_mats[0], lora, r, f16)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
