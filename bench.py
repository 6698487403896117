"""Benchmark of the Aspis detect-and-aggregate step on one MI355X.

One step = the whole hot path over one round of replica gradients already
resident in HBM: pairwise agreement of every file's r replicas, the host
clique of Algorithm 3, the selection of Algorithm 1 and the coordinate-wise
median -- one call of aspis_detect_aggregate.

Default workload: K=15 workers, r=3, f=455 files, d=11,200,000 fp32
coordinates (ResNet-18 sized), optimal attack of Theorem 1 with 4 colluding
ALIE adversaries; 61.15 GB of replicas.  Inputs are synthetic and seeded
(synth/), written on the GPU before timing.

Prints ONE JSON line.  `value` is replica-gradient GB/s (f*r*d*4 bytes per
step / step time).  `roofline` reports the dominant kernel (the single-pass
agreement + median kernel) from HIP events recorded on its stream inside the
library; `read_ceiling` is a linear read of the same tensor with the same
loads (the part's ceiling for this allocation); `cpu_baseline` times the
oracle on the host over the same replicas: one thread on a coordinate slice,
and every coordinate on the host's threads, whose output is compared with
the GPU's (`parity_all_coordinates`).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "replica-gradient GB/s through detect+median (K=15,r=3,d=11.2M); % of HBM peak"
KERNEL_SOURCES = ["paper_2108_02416_amd/csrc/aspis_kernels.hip",
                  "paper_2108_02416_amd/csrc/aspis_internal.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_fused_K15_r3_d11.2M.json")


def kernel_hash(texts=None) -> str:
    """Hash of the kernel code, comments and whitespace ignored (a comment
    edit does not invalidate the counters taken on that code)."""
    import re
    h = hashlib.sha256()
    if texts is None:
        texts = []
        for p in KERNEL_SOURCES:
            with open(os.path.join(ROOT, p), encoding="utf-8") as fh:
                texts.append(fh.read())
    for t in texts:
        t = re.sub(r"//[^\n]*", "", t)
        h.update(" ".join(t.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic(per_launch_bytes_alg: float):
    """HBM bytes per launch of the dominant kernel from committed rocprofv3
    counter runs, if they were taken on the current kernel source."""
    try:
        with open(TRAFFIC_FILE) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("kernel_sha") != kernel_hash():
        return None
    return t.get("bytes_per_launch")


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            return next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")),
                        None)
    except OSError:
        return None


def cpu_baseline(torch, wl, chunk_of, d, gpu_out, gpu_sel, sample_coords: int, full: bool,
                 mode: str = "median"):
    """The oracle, as it stands, timed on the host's cores over the same
    replicas the GPU step consumed (chunk_of(k0, n) reads coordinates
    [k0, k0+n) of every replica back from the device tensor as float32
    [f, r, n]; the read-back is not timed):

      single   one thread, coordinates [0, sample_coords) (Algorithm 3
               then Algorithm 1 on that slice, as one call of oracle.run)
      full     every coordinate on min(16, nproc) threads through the
               chunk-parallel driver: agreement over all d (pass 1), then
               detection and selection, then the reduction (pass 2)

    Returns the cpu_baseline object and the parity verdicts (the oracle's
    output against the GPU's: on the slice, and on every coordinate)."""
    import numpy as np

    import oracle
    from oracle import parallel as oracle_parallel

    K, r, q, f = wl.K, wl.r, wl.q, wl.f

    def same(got, ref, by_mean):
        if not by_mean:
            return bool(np.array_equal(got.view(np.uint32), ref.view(np.uint32)))
        ref = ref.astype(np.float64)
        return bool(np.all(np.abs(got.astype(np.float64) - ref)
                           <= 1e-6 * np.maximum(np.abs(ref), 1e-30)))

    n1 = min(sample_coords, d)
    g = chunk_of(0, n1)
    t0 = time.perf_counter()
    res = oracle.run(g, K, r, q, mode=mode)
    dt1 = time.perf_counter() - t0
    slice_mean = mode == "mean" or (mode == "paper" and res["clique"]["success"])
    # comparable only where the slice alone detects what the whole vector
    # does (an adversary that deviates only past the slice changes the
    # selection): None otherwise; the full pass below checks every coordinate
    parity_slice = (same(gpu_out[:n1], res["out"], slice_mean)
                    if np.array_equal(res["sel"], gpu_sel) else None)
    single = {"value": round(g.nbytes / dt1 / 1e9, 4), "unit": "GB/s", "cores": 1,
              "seconds": round(dt1, 2),
              "sample": f"coordinates [0,{n1}) ({g.nbytes / 1e9:.2f} GB of replicas), one thread"}
    del g
    out = {"kind": "oracle", "cpu_model": _cpu_model(), "single_thread": single}
    parity_full = None
    if full:
        nthreads = oracle_parallel.workers()
        s = oracle.assign(K, r)
        step = max(1024, (1 << 30) // (f * r * 4))
        timed = 0.0
        alpha = np.ones((f, r * (r - 1) // 2), dtype=np.uint8)
        for k0 in range(0, d, step):
            n = min(step, d - k0)
            h = chunk_of(k0, n)
            t0 = time.perf_counter()
            alpha &= oracle_parallel.agreement(h, nthreads)
            timed += time.perf_counter() - t0
        t0 = time.perf_counter()
        det = oracle.detect(None, s, K, q, alpha=alpha)
        cl = det["clique"]
        sel, kept = oracle.select(s, det["vote"], cl["success"], cl["honest"])
        by_mean = mode == "mean" or (mode == "paper" and cl["success"])
        reduce_fn = (oracle_parallel.mean_by_coordinates if by_mean
                     else oracle_parallel.median_by_coordinates)
        timed += time.perf_counter() - t0
        parity_full = bool(np.array_equal(sel, gpu_sel))
        for k0 in range(0, d, step):
            n = min(step, d - k0)
            h = chunk_of(k0, n)
            t0 = time.perf_counter()
            o = reduce_fn(h, sel, nthreads)
            timed += time.perf_counter() - t0
            parity_full = parity_full and same(gpu_out[k0:k0 + n], o, by_mean)
        nbytes = float(f * r * d * 4)
        out.update({"value": round(nbytes / timed / 1e9, 4), "unit": "GB/s", "cores": nthreads,
                    "seconds": round(timed, 2),
                    "sample": f"the whole workload: all {d} coordinates, {nbytes / 1e9:.2f} GB "
                              f"of replicas, on {nthreads} threads (chunk-parallel driver; "
                              f"device read-back not timed)"})
    else:
        out.update({k: single[k] for k in ("value", "unit", "cores", "sample")})
    return out, parity_slice, parity_full


def read_ceiling(torch, aspis, grads, reps: int = 5) -> dict:
    """A linear read of the replica tensor itself (aspis_read_probe: the
    same non-temporal 16-byte loads as the single pass), timed with HIP
    events on the current stream: the bandwidth ceiling of the part for
    this allocation.  Median of `reps` reads after two warm-ups."""
    sink = aspis.read_probe(grads)
    for _ in range(2):
        aspis.read_probe(grads, sink)
    ts = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        aspis.read_probe(grads, sink)
        b.record()
        b.synchronize()
        ts.append(a.elapsed_time(b))
    ms = sorted(ts)[reps // 2]
    nbytes = grads.numel() * grads.element_size() // 16 * 16
    return {"ms": round(ms, 4), "GB/s": round(nbytes / (ms / 1e3) / 1e9, 1), "bytes": nbytes}


def copy_probe(torch, aspis, dev, nbytes: int = 1 << 32) -> int:
    """Kernels of known traffic for scaling the FETCH_SIZE / WRITE_SIZE
    counters: an elementwise negation (reads and writes nbytes) and the
    library's read probe (reads nbytes)."""
    src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)
        aspis.read_probe(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes, "launches": 3,
                      "copy_kernel": "torch.neg (reads and writes copy_probe_bytes)",
                      "read_kernel": "read_probe_kernel (reads copy_probe_bytes)"}), flush=True)
    return 0


def simulate_tables() -> int:
    """Host-only: aspis_simulate / aspis_detox over the settings of the
    paper's Section 5 (Tables 1-3, the K=50 sweep of Figure 3) and the
    K=100, r=5 graphs of the clique-timing tables; prints one JSON line."""
    from paper_2108_02416_amd import aspis
    aspis.lib()   # load before timing

    def row(K, r, q, attack):
        t0 = time.perf_counter()
        res = aspis.simulate(K, r, q, attack)
        wall = (time.perf_counter() - t0) * 1e3
        det = aspis.detox(K, r, q, attack)[1] if K % r == 0 else None
        return {"K": K, "r": r, "q": q, "attack": attack, "files": res["files"],
                "distorted": res["distorted"], "epsilon": round(res["epsilon"], 6),
                "epsilon_baseline": round(res["epsilon_baseline"], 6),
                "epsilon_detox": None if det is None else round(det, 6),
                "success": res["success"], "omega": res["omega"],
                "n_maximum": res["n_maximum"], "n_maximal": res["n_maximal"],
                "ms_clique": round(res["ms_clique"], 4),
                "ms_files": round(res["ms_files"], 3), "ms_wall": round(wall, 3)}

    tables = [row(K, 3, q, a) for K, qmax in ((15, 7), (21, 10), (24, 11))
              for a in ("optimal", "weak") for q in range(2, qmax + 1)]
    k50 = [row(50, 3, q, a) for a in ("optimal", "weak") for q in range(1, 25)]
    k100 = [row(100, 5, q, a) for a in ("weak", "optimal") for q in (5, 15, 25, 35, 45)]
    print(json.dumps({"mode": "simulate", "host_threads": min(16, os.cpu_count() or 1),
                      "tables_1_3": tables, "k50_r3": k50, "k100_r5": k100}), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=3)
    ap.add_argument("--seed", type=int, default=428)
    ap.add_argument("--two-pass", action="store_true", help="force the two-pass path")
    ap.add_argument("--alie-z", type=float, default=None,
                    help="ALIE shift z of the colluders' value mu - z*sigma (default: the "
                         "workload's, 1.0); z = 0 puts it at the honest mean, next to the median")
    ap.add_argument("--dist", choices=["normal", "student3", "tied"], default=None,
                    help="honest gradient distribution (default: the workload's); tied: every "
                         "value shares its high 16 bits, the worst case of half-key tiles")
    ap.add_argument("--keys", choices=["auto", "half", "full"], default="auto",
                    help="median tiles: chosen by the library's tie probe (auto), half keys "
                         "wherever the plan has them, or full 32-bit keys")
    ap.add_argument("--mode", choices=["median", "mean", "paper"], default="median",
                    help="reduction: median (default), mean, or paper (mean when detection "
                         "succeeds, else median)")
    ap.add_argument("--layout", choices=["file", "worker"], default="file",
                    help="replicas as one [f][r][d] tensor (file) or as the workers' uploads "
                         "[K][l][d] (worker, aspis_detect_aggregate_wm)")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the linear read of the replica tensor after the timed steps")
    ap.add_argument("--cpu-sample", type=int, default=1 << 20,
                    help="coordinates of the oracle's single-threaded CPU-baseline slice "
                         "(0 = skip the CPU baseline)")
    ap.add_argument("--no-cpu-full", action="store_true",
                    help="skip the oracle over every coordinate on the host's threads")
    ap.add_argument("--adversary-late", type=int, default=0, metavar="P",
                    help="the adversaries send honest values on coordinates [0, P) and distort "
                         "only after (Section 4.2's adversary, who knows the protocol): with the "
                         "prefix probe (--probe prefix) and P past it every step's guess misses "
                         "(0 = off; 65536 is past any prefix)")
    ap.add_argument("--adversary-sparse", type=int, default=0, metavar="N",
                    help="the adversaries send honest values everywhere but at N coordinates "
                         "drawn (seeded) from [65536, d): a probe rarely sees them, and the "
                         "guess misses (0 = off)")
    ap.add_argument("--adversary-ids", choices=["seeded", "high"], default="seeded",
                    help="which workers collude: the workload's seeded choice, or the q "
                         "highest-numbered (with D the q lowest under Theorem 1's attack), so "
                         "that an honest worker holds slot 0 of every distorted file")
    ap.add_argument("--probe", choices=["spread", "prefix"], default="spread",
                    help="the coordinates the guess is taken from: blocks drawn per call "
                         "(default) or the prefix (ASPIS_FLAG_PROBE_PREFIX)")
    ap.add_argument("--simulate", action="store_true",
                    help="instead of the step, run the host distortion-fraction simulator over "
                         "the paper's tables (K=15, 21, 24), the K=50 sweep and the K=100, r=5 "
                         "clique-timing setting")
    ap.add_argument("--copy-probe", action="store_true",
                    help="instead of the step, run a plain copy kernel and the read probe "
                         "over 4 GiB (the reference sizes for HBM counter calibration)")
    args = ap.parse_args()
    if args.simulate:
        return simulate_tables()
    if args.gpus != 1:
        print(f"bench.py: the benchmark runs on one GPU; --gpus {args.gpus} is not supported",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import synth
    from paper_2108_02416_amd import aspis

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    dev = torch.device("cuda:0")
    if args.copy_probe:
        return copy_probe(torch, aspis, dev)
    wl = synth.WORKLOADS[args.workload]
    if args.alie_z is not None:
        import dataclasses
        wl = dataclasses.replace(wl, alie_z=args.alie_z)
    if args.dist is not None:
        import dataclasses
        wl = dataclasses.replace(wl, dist={"normal": synth.DIST_NORMAL,
                                           "student3": synth.DIST_STUDENT3,
                                           "tied": synth.DIST_TIED}[args.dist])
    K, r, q, d, f = wl.K, wl.r, wl.q, wl.d, wl.f
    subsets = aspis.assign(K, r)
    ids = ({} if args.adversary_ids == "seeded" else
           {"adversaries": list(range(K - q, K)), "disagree_set": list(range(q))})
    role, worker, A, D = synth.make_roles(wl, subsets, seed=args.seed, **ids)
    t_gen = time.perf_counter()
    grads = torch.empty((f, r, d), dtype=torch.float32, device=dev)
    synth.fill_device(role, worker, grads, wl.dist, seed=args.seed, alie_z=wl.alie_z)
    if args.adversary_late > 0:
        # the same generator with every replica honest, over the first P
        # coordinates (it is counter-based: coordinate k has the same value
        # in a tensor of any length)
        P = min(args.adversary_late, d)
        clean = torch.empty((f, r, P), dtype=torch.float32, device=dev)
        synth.fill_device(np.zeros_like(role), worker, clean, wl.dist, seed=args.seed,
                          alie_z=wl.alie_z)
        grads[:, :, :P].copy_(clean)
        del clean
    sparse = None
    if args.adversary_sparse > 0:
        # honest replicas everywhere, then the attack's values back at N
        # coordinates past the longest probe prefix
        lo = min(65536, d - 1)
        sparse = sorted({lo + synth.u32(args.seed, 13, j) % (d - lo)
                         for j in range(args.adversary_sparse)})
        idx = torch.tensor(sparse, dtype=torch.int64, device=dev)
        kept = grads.index_select(2, idx)
        synth.fill_device(np.zeros_like(role), worker, grads, wl.dist, seed=args.seed,
                          alie_z=wl.alie_z)
        grads.index_copy_(2, idx, kept)
        del kept, idx
    if args.layout == "worker":
        # the same replicas in the order the workers upload them
        l_files = f * r // K
        rows = torch.from_numpy(aspis.worker_rows(K, r).reshape(-1).astype(np.int64)).to(dev)
        upload = torch.empty((K * l_files, d), dtype=torch.float32, device=dev)
        upload.index_copy_(0, rows, grads.view(f * r, d))
        del grads, rows
        torch.cuda.empty_cache()
        grads = upload.view(K, l_files, d)
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t_gen
    print(f"# workload {wl.name}: f={f} replicas {wl.replica_bytes() / 1e9:.2f} GB, "
          f"generated on GPU in {t_gen:.1f} s; adversaries {A}", file=sys.stderr, flush=True)

    bufs = aspis.DetectBuffers.empty(f, K, dev)
    out = torch.empty(d, dtype=torch.float32, device=dev)
    sel = torch.empty(f, dtype=torch.int32, device=dev)
    ws = aspis.workspace(K, r, d, dev)
    flags = (aspis.FLAG_TIMING | (aspis.FLAG_TWO_PASS if args.two_pass else 0)
             | {"auto": 0, "half": aspis.FLAG_HALF_KEYS, "full": aspis.FLAG_FULL_KEYS}[args.keys]
             | (aspis.FLAG_PROBE_PREFIX if args.probe == "prefix" else 0))

    def step():
        return aspis.detect_aggregate(grads, K, r, q, mode=args.mode, flags=flags, bufs=bufs,
                                      out=out, sel_out=sel, ws=ws, layout=args.layout)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stats = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step_out = step()
        stats.append(step_out["stats"])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps
    replica_bytes = float(f * r * d * 4)
    value = replica_bytes / (ms_step / 1e3) / 1e9
    last = stats[-1]
    print(f"# per-step stats (last): {last}", file=sys.stderr, flush=True)

    # dominant kernel: the single-pass kernel (or, two-pass, detect+reduce)
    ms_kernel = float(np.mean([s["ms_main"] for s in stats]))
    res = step_out["clique"]
    by_mean = args.mode == "mean" or (args.mode == "paper" and bool(res.success))
    red = "mean" if by_mean else "median"
    if last["fused"]:
        alg_bytes = replica_bytes + d * 4.0 + f * 4.0
        if by_mean:
            kname = "fused_mean_kernel"
        else:
            kname = (f"fused_ws_kernel, {last['tile_cols']}-column "
                     + ("half-key" if last["half_keys"] else "full-key") + " tiles")
        kname = f"single-pass agreement + {red} kernel (one read): {kname}"
    else:
        alg_bytes = replica_bytes + step_out["n_selected"] * d * 4.0 + d * 4.0
        kname = f"agree_kernel + {red}_kernel (two reads)"
    achieved = alg_bytes / (ms_kernel / 1e3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic(alg_bytes), "kernel": kname,
                "kernel_ms": round(ms_kernel, 4), "algorithmic_bytes": alg_bytes}

    ceiling = None
    if not args.no_ceiling:
        ceiling = read_ceiling(torch, aspis, grads)
        ceiling["kernel_frac"] = round(achieved / ceiling["GB/s"], 4)
        ceiling["step_frac"] = round(value / ceiling["GB/s"], 4)

    fallback = None
    missed = [s for s in stats if s["fused"] and not s["speculation_hit"]]
    if missed:
        # the reduction redone after the steps' wrong guesses: whole, or
        # (same files, same median) the tile groups the moved files touch
        ms_fb = float(np.mean([s["ms_fallback"] for s in missed]))
        groups = [s["repair_groups"] for s in missed]
        fallback = {"steps_missed": len(missed), "ms": round(ms_fb, 4),
                    "repair_groups": groups[-1]}
        if groups[-1] < 0:
            fb_bytes = step_out["n_selected"] * d * 4.0 + d * 4.0
            fallback.update({
                "kernel": f"{red} rerun over the final selection"
                          + (f" ({last['tile_cols']}-column tiles)" if not by_mean else ""),
                "algorithmic_bytes": fb_bytes,
                "achieved": round(fb_bytes / (ms_fb / 1e3) / 1e9, 1), "unit": "GB/s",
                "frac": round(fb_bytes / (ms_fb / 1e3) / 1e9 / HBM_PEAK_GBS, 4)})
        else:
            tiles = "1024-column" if by_mean else f"{last['tile_cols']}-column"
            fallback["kernel"] = ("dirty_tiles_kernel (moved files' two replicas compared) + "
                                  f"{red} over the marked tile groups ({tiles} tiles)")

    cpu = None
    parity = {}
    if args.cpu_sample > 0:
        if args.layout == "file":
            def chunk_of(k0, n):
                return grads[:, :, k0:k0 + n].contiguous().cpu().numpy()
        else:
            rows_fm = torch.from_numpy(aspis.worker_rows(K, r).reshape(-1).astype(np.int64)).to(dev)
            flat = grads.view(-1, d)

            def chunk_of(k0, n):
                return flat[:, k0:k0 + n].index_select(0, rows_fm).view(f, r, n).cpu().numpy()
        cpu, p_slice, p_full = cpu_baseline(torch, wl, chunk_of, d, out.cpu().numpy(),
                                            sel.cpu().numpy(), args.cpu_sample,
                                            not args.no_cpu_full, args.mode)
        parity = {"parity_on_cpu_sample": p_slice, "parity_all_coordinates": p_full}

    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": ("synthetic (seeded Philox, written on the GPU): "
                 + {synth.DIST_STUDENT3: "Student-t(3)", synth.DIST_TIED: "tied (1 + 16 random bits)"}
                 .get(wl.dist, "N(0,0.01^2) (polar method)")
                 + f" honest gradients, {wl.distortion} adversaries"),
        "config": {"workload": wl.name, "K": K, "r": r, "q": q, "files": f, "d": d,
                   **({"adversary_late": min(args.adversary_late, d)}
                      if args.adversary_late > 0 else {}),
                   **({"adversary_sparse": len(sparse)} if sparse else {}),
                   **({"adversary_ids": args.adversary_ids}
                      if args.adversary_ids != "seeded" else {}),
                   **({"dist": args.dist} if args.dist else {}),
                   "layout": "[f][r][d]" if args.layout == "file" else "[K][l][d] (worker uploads)",
                   "attack": wl.attack, "distortion": wl.distortion,
                   **({"alie_z": wl.alie_z} if "alie" in wl.distortion else {}),
                   "replica_bytes": replica_bytes, "parallelism": "single GPU"},
        "frac_of_hbm_peak": round(value / HBM_PEAK_GBS, 4),
        "path": {"fused": bool(last["fused"]), "speculation_hit": bool(last["speculation_hit"]),
                 "steps_hit": sum(1 for s in stats if s["speculation_hit"]),
                 "probe": args.probe, "probe_blocks": int(last["probe_blocks"]),
                 "probe_coords": int(last["probe_coords"]),
                 "repair_groups": int(last["repair_groups"]),
                 "ms_probe": round(last["ms_probe"], 4),
                 "ms_fallback": round(last["ms_fallback"], 4),
                 "tile_columns": int(last["tile_cols"]), "half_keys": bool(last["half_keys"]),
                 "tie_rows": int(last["tie_rows"]), "keys": args.keys},
        "roofline": roofline,
        "fallback": fallback,
        "read_ceiling": ceiling,
        "cpu_baseline": cpu,
        **parity,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
