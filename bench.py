"""Throughput of the fused policy loss (forward + backward) on one MI355X.

One step = the whole hot path over one batch: task advantage normalisation
over the global batch of trajectories, then the fused LM-head / log-prob /
clipped-surrogate forward and its backward (dH, dW) over the packed
micro-batch.  Inputs are synthetic, drawn on the GPU before timing.

Prints one JSON line.  ``value`` is packed micro-batch tokens per second;
``mfma_frac`` is the executed matrix-core work of the step (four products of
2 * N_act * V * d flops: forward logits, backward recompute, dW, dH) per
second over the bf16 dense peak.  ``roofline`` describes the slowest of the
four matrix-core launches, timed with HIP events on the library's stream.
``cpu_baseline`` is the CPU oracle timed on a bounded sample of the same
workload's action tokens on this host.
"""
from __future__ import annotations

import argparse
import ctypes
import glob
import hashlib
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16 = 2.5e15          # MI355X dense bf16 matrix-core peak, FLOP/s
PEAK_F32 = 157.3e12
HBM_PEAK = 8.0e12
METRIC = "policy-loss fwd+bwd tokens/s and % of bf16 MFMA peak, 1 MI355X"
PHASES = ["forward logits + lse", "backward logit recompute -> G", "dW = G^T H (+ dH = G W in the same launch for bf16)", "dH = G W (separate launch)"]


class HipEvents:
    """Raw hipEvent_t handles (the library records them on its own stream)."""

    def __init__(self, n: int):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.arr = (ctypes.c_void_p * n)()
        for i in range(n):
            ev = ctypes.c_void_p()
            rc = self.hip.hipEventCreate(ctypes.byref(ev))
            if rc != 0:
                raise RuntimeError(f"hipEventCreate failed: {rc}")
            self.arr[i] = ev

    def slice_ptr(self, start: int):
        return ctypes.cast(ctypes.byref(self.arr, start * ctypes.sizeof(ctypes.c_void_p)),
                           ctypes.c_void_p).value

    def elapsed_ms(self, a: int, b: int) -> float:
        ms = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(ms), self.arr[a], self.arr[b])
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed: {rc}")
        return float(ms.value)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


class ClockSampler:
    """Samples the shader clock the driver reports (the starred line of
    pp_dpm_sclk in sysfs) from a background thread while the steps run: the
    sustained clock under this load, against which the published peak (quoted
    at 2.4 GHz) is rescaled, and the board power next to its cap (hwmon), which
    shows whether that clock is set by the power limit.  Reports None where the
    files are not readable."""

    def __init__(self, period_s: float = 0.01):
        import glob
        import threading
        files = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.path = files[0] if files else None
        # board power (microwatts) and its cap from the same card's hwmon node
        self.power_path = self.cap_path = None
        if self.path:
            hw = os.path.join(os.path.dirname(self.path), "hwmon", "hwmon*")
            for name in ("power1_average", "power1_input"):
                found = sorted(glob.glob(os.path.join(hw, name)))
                if found and self._read_int(found[0]) is not None:
                    self.power_path = found[0]
                    break
            caps = sorted(glob.glob(os.path.join(hw, "power1_cap")))
            self.cap_path = caps[0] if caps else None
        self.period = period_s
        self.samples = []
        self.power = []
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)

    def _read(self):
        import re
        try:
            with open(self.path) as f:
                for line in f:
                    m = re.search(r"(\d+)\s*Mhz\s*\*", line)
                    if m:
                        return int(m.group(1))
        except OSError:
            return None
        return None

    @staticmethod
    def _read_int(path):
        try:
            with open(path) as f:
                return int(f.read().strip())
        except (OSError, ValueError):
            return None

    def _run(self):
        while not self._stop.is_set():
            v = self._read()
            if v is not None:
                self.samples.append(v)
            if self.power_path:
                w = self._read_int(self.power_path)
                if w is not None and w > 0:
                    self.power.append(w * 1e-6)
            self._stop.wait(self.period)

    def __enter__(self):
        if self.path:
            self._thread.start()
        return self

    def __exit__(self, *exc):
        if self.path:
            self._stop.set()
            self._thread.join()

    def summary(self):
        if not self.samples:
            return None
        a = np.array(self.samples, dtype=np.float64)
        return {"mean": float(a.mean()), "min": float(a.min()), "max": float(a.max()),
                "samples": int(a.size), "source": self.path}

    def power_summary(self):
        """Board power in W over the timed steps, beside the cap the driver
        enforces (None where hwmon does not expose them)."""
        if not self.power:
            return None
        a = np.array(self.power, dtype=np.float64)
        cap = self._read_int(self.cap_path) if self.cap_path else None
        return {"mean": float(a.mean()), "min": float(a.min()), "max": float(a.max()),
                "cap": cap * 1e-6 if cap else None, "samples": int(a.size),
                "source": self.power_path}


def kernel_sources_digest() -> str:
    """sha256 over the HIP sources and the build script (counters go stale when these change)."""
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2510_04206_amd", "csrc", "*")))
    files.append(os.path.join(ROOT, "paper_2510_04206_amd", "build.py"))
    for f in files:
        h.update(os.path.relpath(f, ROOT).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def committed_traffic(workload: str, kernel: str):
    """L2-to-fabric bytes per launch of `kernel` on `workload` from a committed counter summary.

    The summaries under profiles/ carry one line ``traffic-record: {json}`` with
    the sources digest they were measured on; a record whose digest differs from
    the current sources is stale and ignored (traffic is then reported as null).
    """
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        with open(path) as fh:
            for line in fh:
                if not line.startswith("traffic-record: "):
                    continue
                rec = json.loads(line[len("traffic-record: "):])
                if (rec.get("workload") == workload and rec.get("kernel") == kernel
                        and rec.get("sources_sha256") == kernel_sources_digest()):
                    return rec
    return None


def host_cpu_info():
    """What this process may run on: the host's logical CPUs, the CPUs in its
    affinity mask, the cgroup CPU quota (cgroup v2 cpu.max, in CPUs; None when
    unlimited or unreadable) and the CPU model from /proc/cpuinfo."""
    info = {"host_cpus": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0)),
            "cgroup_cpu_quota": None, "cpu_model": None}
    try:
        with open("/sys/fs/cgroup/cpu.max") as f:
            quota, period = f.read().split()[:2]
        if quota != "max":
            info["cgroup_cpu_quota"] = float(quota) / float(period)
    except (OSError, ValueError):
        pass
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    info["cpu_model"] = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return info


def cpu_baseline(w, adv_tok_host, n_sample, n_act, T):
    """The oracle's fwd+bwd on the first n_sample action tokens, scaled to the micro-batch.

    The oracle runs one thread per CPU this process may use: the affinity mask,
    capped by the cgroup CPU quota when there is one (more threads than the
    quota only time-slice)."""
    import oracle
    act = np.nonzero(w.mask)[0][:n_sample]
    H = w.H[torch.from_numpy(act).to(w.H.device)].cpu()
    W = w.W.cpu()
    info = host_cpu_info()
    threads = info["affinity_cpus"]
    if info["cgroup_cpu_quota"]:
        threads = min(threads, max(1, int(info["cgroup_cpu_quota"])))
    t0 = time.perf_counter()
    oracle.policy_loss(H, W, w.token_id[act], np.ones(len(act), np.uint8), adv_tok_host[act],
                       w.old_logp[act], eps_lo=w.spec.eps_lo, eps_hi=w.spec.eps_hi,
                       n_norm=n_act, nthreads=threads)
    dt = time.perf_counter() - t0
    per_token = dt / len(act)
    return {"value": T / (per_token * n_act), "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": f"fwd+bwd (logp, loss, dH, dW) of {len(act)} of the micro-batch's {n_act} "
                      f"action tokens over the full V={w.V}, d={w.d} in fp64 took {dt:.2f} s on "
                      f"{threads} threads; value = T / (time per action token * N_act)",
            "seconds": dt, **info}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=3, help="1..5; 3 is the 32B-shaped batch")
    ap.add_argument("--cpu-tokens", type=int, default=128,
                    help="action tokens in the oracle's timed sample (0 skips it)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="before the steps, copy a buffer of this many MiB once (a kernel of known "
                         "traffic, to scale the FETCH_SIZE / WRITE_SIZE counters of a profiling run)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path; "
              "each GPU of a data-parallel job would run this step on its own micro-batch.",
              file=sys.stderr)
        sys.exit(2)

    import paper_2510_04206_amd as P
    from paper_2510_04206_amd import _binding as B
    from workloads import gen

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t0 = time.perf_counter()
    w = gen.config(args.workload, device=dev)
    log(f"workload {w.spec.name}: T={w.T} N_act={w.n_act} T_g={w.T_g} n_traj={w.n_traj} "
        f"(generated in {time.perf_counter() - t0:.1f} s)")
    V, d, T, n_act = w.V, w.d, w.T, w.n_act
    dtype = w.H.dtype
    code = P.AGRL_BF16 if dtype == torch.bfloat16 else P.AGRL_F32
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    g_traj, g_mask = t(w.g_traj_id), t(w.g_mask)
    traj_task, traj_group, reward = t(w.traj_task), t(w.traj_group), t(w.reward)
    token_id, mask, old = t(w.token_id), t(w.mask), t(w.old_logp)
    H, W = w.H, w.W

    n_traj, n_task = w.n_traj, w.n_task
    act_count = torch.empty(n_traj, dtype=torch.int32, device=dev)
    task_count = torch.empty(n_task, dtype=torch.int64, device=dev)
    task_mean = torch.empty(n_task, dtype=torch.float32, device=dev)
    task_std = torch.empty(n_task, dtype=torch.float32, device=dev)
    adv_traj = torch.empty(n_traj, dtype=torch.float32, device=dev)
    adv_tok = torch.empty(w.T_g, dtype=torch.float32, device=dev)
    adv_mb = adv_tok[:T]        # the micro-batch is the global stream's first T tokens
    # member-range scratch of the advantage stages (groups, then tasks)
    adv_opt = B.agrl_options()
    ranges = torch.empty(2 * (w.n_group + n_task), dtype=torch.int32, device=dev)
    adv_opt.adv_ranges = ranges.data_ptr()

    K, Wm = args.steps, args.warmup
    events = HipEvents(8 * (K + Wm))
    opt = B.agrl_options()
    pl = P.PolicyLoss(T, d, V, dtype, max_act=n_act, eps_low=w.spec.eps_lo,
                      eps_high=w.spec.eps_hi, opt=opt, device=dev)
    log(f"workspace {pl.ws_bytes / 2**30:.2f} GiB")

    # per step: start, advantage normalisation done, end (torch's current stream,
    # which is the one the library enqueues on)
    marks = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K + Wm)]

    def step(i):
        opt.phase_events = events.slice_ptr(8 * i)
        marks[i][0].record()
        B.agrl_task_adv_norm(w.T_g, n_traj, n_task, w.n_group, g_traj, g_mask, traj_task,
                             traj_group, reward, adv_opt, act_count, task_count, task_mean,
                             task_std, adv_traj, adv_tok)
        marks[i][1].record()
        pl.forward(H, W, token_id, mask, adv_mb, old)
        pl.backward(H, W, token_id, mask, adv_mb, old)
        marks[i][2].record()

    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for i in range(Wm):
        step(i)
    torch.cuda.synchronize()
    if P.agrl_get_device_error() != 0:
        raise RuntimeError("device error flag set during warm-up")
    log(f"warm-up done; loss {pl.loss.item():.6g}")
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with ClockSampler() as clock:
        start.record()
        for i in range(Wm, Wm + K):
            step(i)
        end.record()
        torch.cuda.synchronize()
    sclk = clock.summary()
    board_power = clock.power_summary()
    total_ms = start.elapsed_time(end)
    ms = total_ms / K
    if P.agrl_get_device_error() != 0:
        raise RuntimeError("device error flag set during timing")

    # the forward-only log-prob pass over the same batch (outside the step)
    lp = P.TokenLogprob(T, d, V, dtype, max_act=n_act, device=dev)
    for _ in range(2):
        lp(H, W, token_id, mask)
    lp_marks = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
    for i in range(5):
        lp_marks[i].record()
        lp(H, W, token_id, mask)
    lp_marks[5].record()
    torch.cuda.synchronize()
    lp_ms = float(np.median([lp_marks[i].elapsed_time(lp_marks[i + 1]) for i in range(5)]))
    del lp

    step_ms = np.array([marks[i][0].elapsed_time(marks[i][2]) for i in range(Wm, Wm + K)])
    adv_ms = np.array([marks[i][0].elapsed_time(marks[i][1]) for i in range(Wm, Wm + K)])
    # advantage normalisation: the count pass and the broadcast each read traj_id and
    # the mask (5 B per global token); the broadcast writes adv_tok (4 B)
    adv_bytes = 14.0 * w.T_g
    gemm_flops = 2.0 * n_act * V * d
    # the backward walks the vocabulary in chunks; its phase events bracket the
    # last chunk's launches
    vc = pl.vocab_chunk
    n_chunks = -(-V // vc)
    nv_last = V - (n_chunks - 1) * vc
    chunk_flops = 2.0 * n_act * nv_last * d
    phase_ms = [float(np.mean([events.elapsed_ms(8 * i + 2 * p, 8 * i + 2 * p + 1)
                               for i in range(Wm, Wm + K)])) for p in range(4)]
    peak = PEAK_BF16 if code == P.AGRL_BF16 else PEAK_F32
    # products per bracketed launch: dW and dH share one launch when phase 3 is empty
    grouped = phase_ms[3] < 0.05          # an empty event pair reads a few microseconds
    prods = [1, 1, 2 if grouped else 1, 0 if grouped else 1]
    per_launch = [gemm_flops] + [chunk_flops * n for n in prods[1:]]
    rates = [f / (ms_ * 1e-3) if f > 0 else 0.0 for f, ms_ in zip(per_launch, phase_ms)]
    # the dominant kernel: most time per step (launch time x launches per step)
    per_step = [phase_ms[0], phase_ms[1] * n_chunks, phase_ms[2] * n_chunks, phase_ms[3] * n_chunks]
    dom = int(np.argmax(per_step))
    achieved = per_launch[dom] / (phase_ms[dom] * 1e-3)
    kernel_names = ["gemm_bf16_kernel<EpiLseCols>", "gemm_bf16_kernel<EpiLogitGrad>",
                    "gemm_bf16_kernel<EpiStore>", "gemm_bf16_kernel<EpiStore>"]
    if code != P.AGRL_BF16:
        kernel_names = [k.replace("gemm_bf16_kernel", "gemm_nt_kernel") for k in kernel_names]
    dom_kernel = kernel_names[dom]
    rec = committed_traffic(w.spec.name, dom_kernel + (" grouped" if grouped and dom == 2 else ""))
    step_flops = 4 * gemm_flops
    log("phases (ms): " + ", ".join(f"{n}: {m:.3f}" for n, m in zip(PHASES, phase_ms)))

    out = {
        "metric": METRIC,
        "value": T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": ms,
        "ms_per_step_median": float(np.median(step_ms)),
        "ms_per_step_min": float(step_ms.min()),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if code == P.AGRL_BF16 else "f32",
        "data": "synthetic",
        "config": {"workload": w.spec.name, "T": T, "N_act": n_act, "V": V, "d": d,
                   "T_g": w.T_g, "n_traj": n_traj, "n_task": n_task,
                   "vocab_chunk": vc, "vocab_chunks": n_chunks},
        "action_tokens_per_s": n_act / (ms * 1e-3),
        "model_tflops": 6.0 * n_act * V * d / (ms * 1e-3) / 1e12,
        "mfma_tflops": step_flops / (ms * 1e-3) / 1e12,
        "mfma_frac": step_flops / (ms * 1e-3) / peak,
        "adv_norm": {"us": float(np.median(adv_ms)) * 1e3,
                     "GBps": adv_bytes / (float(np.median(adv_ms)) * 1e-3) / 1e9,
                     "bytes": adv_bytes, "T_g": w.T_g},
        "logprob_pass": {"ms": lp_ms, "tokens_per_s": T / (lp_ms * 1e-3),
                         "mfma_frac": 2.0 * n_act * V * d / (lp_ms * 1e-3) / (
                             PEAK_BF16 if code == P.AGRL_BF16 else PEAK_F32)},
        "gemm_launches_per_step": {"fwd": 1, "recompute": n_chunks,
                                   "dW+dH" if grouped else "dW": n_chunks},
        "gemm_ms": dict(zip(["fwd", "recompute", "dW+dH" if grouped else "dW", "dH"], phase_ms)),
        "gemm_tflops": dict(zip(["fwd", "recompute", "dW+dH" if grouped else "dW", "dH"],
                                [r / 1e12 for r in rates])),
        "roofline": {"kernel": f"{dom_kernel} ({PHASES[dom]})", "bound": "mfma",
                     "achieved": achieved / 1e12, "peak": peak / 1e12, "unit": "TFLOP/s",
                     "frac": achieved / peak,
                     "traffic": rec["bytes_per_launch"] if rec else None,
                     "traffic_unit": "bytes per launch between the L2 caches and the fabric "
                                     "(reads + writes; Infinity Cache hits included, so an upper "
                                     "bound on HBM traffic): rocprofv3 FETCH_SIZE and WRITE_SIZE "
                                     "scaled by a copy kernel of known size",
                     "flops_per_launch": per_launch[dom]},
        "sclk_mhz": sclk,
        "board_power_w": board_power,
    }
    if sclk:
        # the published peak is quoted at 2.4 GHz: the same fractions at the
        # shader clock sampled during the timed steps
        at_clock = peak * sclk["mean"] / 2400.0
        out["mfma_frac_at_sampled_clock"] = step_flops / (ms * 1e-3) / at_clock
        out["roofline"]["frac_at_sampled_clock"] = achieved / at_clock
    if args.cpu_tokens > 0:
        adv_host = adv_tok[:T].cpu().numpy()
        log(f"timing the oracle on {args.cpu_tokens} action tokens ...")
        out["cpu_baseline"] = cpu_baseline(w, adv_host, args.cpu_tokens, n_act, T)
        out["speedup_vs_cpu_baseline"] = out["value"] / out["cpu_baseline"]["value"]
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
