"""Benchmark of the LVSA hot path on one MI355X.

One step = one denoising step of the hot path on one attention layer:
the device mask builder rebuilds the block CSR for step s (Eq. 3 anchors,
Alg. 1 windows, block expansion) and the block-sparse attention kernel runs
over it, on synthetic bf16 Q/K/V of the Wan2.1-1.3B 6x-horizon layer shape
(12 heads, 121 latent frames x 30x52 tokens, head_dim 128, block 128,
C = 21, W = 6).  Successive steps sweep s = 0, 1, 2, ... so the anchors
rotate as in a denoising loop.  Inputs are resident in HBM before timing.

Prints ONE JSON line.  Besides the step throughput it reports the attention
call alone (hipEvents), the token-exact form of the same mask (Eq. 2 token
for token), the pattern variants of Sec. 2 (window rule, fixed vs rotating
anchors, a dedicated initial anchor: density and call time), the dense kernel
of the same design, the roofline position of the sparse kernel, and the CPU
oracle on a bounded sample.

    python bench.py [--steps K] [--warmup W] [--workload wan13_6x]
"""
import argparse
import hashlib
import re
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
METRIC = ("ms/attention call + effective TFLOP/s (kept blocks) and speedup vs "
          "dense, Wan-1.3B 6×")
ATTN_SRC = os.path.join(ROOT, "paper_2605_31057_amd", "csrc", "attention.hip")
PROFILES = os.path.join(ROOT, "profiles")
SPARSE_KERNEL = "attn_fwd_kernel<128, ATTN_BLOCK>"


def kept_flops(row_ptr, col_idx, n_tokens, block, heads, d=128):
    """4*d FLOP per (query, key) pair of real tokens over the kept blocks."""
    import numpy as np
    rp = np.asarray(row_ptr, dtype=np.int64)
    ci = np.asarray(col_idx, dtype=np.int64)
    nb = len(rp) - 1
    rows = np.minimum(block, n_tokens - np.arange(nb) * block)
    cols = np.minimum(block, n_tokens - ci * block)
    per_row = np.add.reduceat(cols, rp[:-1]) if len(ci) else np.zeros(nb)
    per_row = np.where(np.diff(rp) > 0, per_row, 0)
    return 4.0 * d * heads * float((rows * per_row).sum())


def eq2_pairs(frames_per_query, P, text, n_tokens):
    """(query, key) token pairs of Eq. 2: P*P per attended frame pair, plus
    every pair with a text query or a text key."""
    video = P * P * sum(frames_per_query)
    return float(video + (n_tokens - text) * text + text * n_tokens)


def median(xs):
    xs = sorted(xs)
    return xs[len(xs) // 2]


def time_calls(fn, n, warm):
    import torch
    for _ in range(warm):
        fn()
    evs = []
    for _ in range(n):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        evs.append((a, b))
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in evs]


def percentile(xs, q):
    xs = sorted(xs)
    return xs[min(len(xs) - 1, int(round(q * (len(xs) - 1))))]


def kernel_code_hash(path=ATTN_SRC):
    """sha256 of the kernel source's code: comments removed and whitespace
    collapsed, so that a change to the comments alone keeps the hash and any
    change to the code does not."""
    text = open(path, encoding="utf-8").read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    text = " ".join(text.split())
    return hashlib.sha256(text.encode()).hexdigest()


def traffic_from_profile(workload, kernel):
    """HBM bytes per launch of `kernel` at `workload` from the committed PMC
    summary of that workload (profiles/attn_pmc_<workload>.json), if it was taken
    on the current kernel code; else None."""
    path = os.path.join(PROFILES, f"attn_pmc_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("attention_code_sha256") != kernel_code_hash() or rec.get("workload") != workload:
        return None
    k = rec.get("kernels", {}).get(kernel)
    return None if k is None else k.get("hbm_bytes_per_launch")


def host_cores():
    """Logical CPUs this process may run on, and physical cores among them
    (from /proc/cpuinfo; None where it cannot be read)."""
    logical = len(os.sched_getaffinity(0))
    try:
        cores = set()
        phys = core = None
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("physical id"):
                    phys = line.split(":")[1].strip()
                elif line.startswith("core id"):
                    core = line.split(":")[1].strip()
                elif not line.strip() and core is not None:
                    cores.add((phys, core))
                    phys = core = None
        physical = len(cores) or None
    except OSError:
        physical = None
    return logical, physical


def metadata_costs(w, L, params, reps=200):
    """Sec. 2 metadata figures: Alg. 1 growth steps (max, mean over every
    query frame of every swept step), the per-frame window call and the host
    CSR rebuild."""
    grow = []
    for s in w.steps:
        grow += L.frame_sets(w.frames, s, params, growth=True)[4]
    T = w.frames
    t0 = time.perf_counter()
    for i in range(reps):
        L.frame_sets(w.frames, w.steps[i % len(w.steps)], params)
    per_frame_us = (time.perf_counter() - t0) / (reps * T) * 1e6
    t0 = time.perf_counter()
    for i in range(reps):
        L.frame_window(w.frames, w.steps[i % len(w.steps)], i % T, params)
    per_call_us = (time.perf_counter() - t0) / reps * 1e6
    return {
        "alg1_growth_max": max(grow),
        "alg1_growth_mean": sum(grow) / len(grow),
        "alg1_frames_counted": len(grow),
        "frame_window_us_per_frame": per_frame_us,
        "frame_window_us_per_call_via_python": per_call_us,
    }


def cpu_baseline(w, target_s, full_max_s=60.0):
    """The oracle (numpy fp32, host cores) at step 10, scaled to TFLOP/s on
    kept blocks: on sampled query blocks of head 0 (about target_s seconds),
    or, when the whole call would take at most full_max_s at the sampled
    rate (the Wan 1x layer), on every query block of every head."""
    import numpy as np
    from paper_2605_31057_amd.inputs import make_qkv
    from oracle import attention as OA
    from oracle import mask as M
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    logical, physical = host_cores()
    t0 = time.perf_counter()
    rp, ci = M.build_mask(w.frames, w.tokens_per_frame, w.block, 10,
                          C=w.budget_frames, W=w.window, tper=w.tper,
                          text=w.text_tokens)
    mask_s = time.perf_counter() - t0
    q, k, v = make_qkv(1, w.n_tokens, value_scale=w.value_scale)
    q, k, v = (x.float().numpy() for x in (q, k, v))
    rng = np.random.default_rng(0)
    order = rng.permutation(len(rp) - 1)
    done = []
    t0 = time.perf_counter()
    for qb in order:
        OA.block_sparse_attention(q, k, v, rp, ci, w.block, q_blocks=[int(qb)])
        done.append(int(qb))
        if time.perf_counter() - t0 >= target_s:
            break
    elapsed = time.perf_counter() - t0
    n = w.n_tokens
    flops = 0.0
    for qb in done:
        rows = min(w.block, n - qb * w.block)
        cols = sum(min(w.block, n - kb * w.block) for kb in ci[rp[qb]:rp[qb + 1]])
        flops += 4.0 * 128 * rows * cols
    total = kept_flops(rp, ci, w.n_tokens, w.block, w.heads)
    if total / (flops / elapsed) <= full_max_s:
        # The whole call, every head, every query block, timed as one run.
        qh, kh, vh = (x.float().numpy() for x in make_qkv(w.heads, w.n_tokens,
                                                           value_scale=w.value_scale))
        t0 = time.perf_counter()
        OA.block_sparse_attention(qh, kh, vh, rp, ci, w.block)
        elapsed = time.perf_counter() - t0
        sample = (f"the whole call: all {len(rp) - 1} query blocks of all {w.heads} heads "
                  f"(step 10, fp32 numpy masked softmax, {total:.3g} FLOP), {elapsed:.3g} s, "
                  f"run in full; oracle mask build {mask_s * 1e3:.0f} ms")
        flops = total
    else:
        sample = (f"{len(done)} of {len(rp) - 1} query blocks of head 0 of {w.heads} "
                  f"(step 10, fp32 numpy masked softmax), {elapsed:.1f} s; a rate "
                  f"measured on that sample: the whole call ({total:.3g} FLOP) would take "
                  f"{total / (flops / elapsed):.0f} s at it (extrapolated, not run); "
                  f"oracle mask build {mask_s * 1e3:.0f} ms")
    return {
        "value": flops / elapsed / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": sample,
        "threads": threads,
        "logical_cpus": logical,
        "physical_cores": physical,
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="wan13_6x")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-patterns", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--pmc", action="store_true",
                    help="counter-collection run: untimed block-sparse (3), token-exact "
                         "(2) and dense (1) launches at step 10 plus three 1 GiB copies "
                         "(the byte-counter calibration), for rocprofv3 --pmc")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the hot path is a single-GPU kernel; see the sharding notes in "
              "the design document).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2605_31057_amd as L
    from paper_2605_31057_amd.inputs import WORKLOADS, workload_qkv

    w = WORKLOADS[args.workload]
    params = L.Params(budget_frames=w.budget_frames, window=w.window, tper=w.tper,
                      text_tokens=w.text_tokens)
    if args.pmc:
        # Counter runs: the same shapes and value distribution drawn on the
        # device from a seeded generator (counters do not depend on values,
        # and drawing 40 heads on the host would dominate every pass).
        g = torch.Generator(device="cuda")
        g.manual_seed(16)
        q, k, v = (torch.randn((w.heads, w.n_tokens, 128), generator=g, device="cuda")
                   .mul_(w.value_scale).to(torch.bfloat16) for _ in range(3))
    else:
        print(f"[bench] {w.name}: generating inputs", file=sys.stderr, flush=True)
        q, k, v = (x.cuda() for x in workload_qkv(w))
    out = torch.empty_like(q)
    nb = w.n_blocks
    rp = torch.empty(nb + 1, dtype=torch.int32, device="cuda")
    ci = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    # Kept FLOP of every step s (host builder, outside the timed region).
    n_sweep = len(w.steps)
    flops_of, nnz_of = {}, {}
    for s in w.steps:
        csr = L.build_mask(w.frames, w.tokens_per_frame, w.block, s, params)
        hrp, hci = csr.arrays()
        flops_of[s] = kept_flops(hrp, hci, w.n_tokens, w.block, w.heads)
        nnz_of[s] = int(hrp[-1])
        csr.free()
    # Host rebuild time (Sec. 2 quotes the metadata cost per denoising step):
    # 20 rebuilds, cycling over the swept steps, after the ones above.
    host_us = []
    for i in range(20):
        t0 = time.perf_counter()
        L.build_mask(w.frames, w.tokens_per_frame, w.block, w.steps[i % n_sweep], params).free()
        host_us.append((time.perf_counter() - t0) * 1e6)
    dense_flops = kept_flops(np.arange(nb + 1) * nb, np.tile(np.arange(nb), nb),
                             w.n_tokens, w.block, w.heads)

    if args.pmc:
        s_ref = 10 if 10 in w.steps else w.steps[0]
        m = L.build_mask_device(w.frames, w.tokens_per_frame, w.block, s_ref, rp, ci,
                                params=params, stream=stream)
        for _ in range(3):
            L.attention(q, k, v, m, out=out, stream=stream)
        ent = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
        rpx = torch.empty(nb + 1, dtype=torch.int32, device="cuda")
        try:
            me = L.build_exact_mask_device(w.frames, w.tokens_per_frame, w.block, s_ref, rpx,
                                           ent, params=params, stream=stream)
            for _ in range(2):
                L.attention_exact(q, k, v, me, out=out, stream=stream)
        except L.LvsaError:
            pass
        if not args.no_dense:
            L.dense_attention(q, k, v, block=w.block, out=out, stream=stream)
        src = torch.empty(1 << 29, dtype=torch.int16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print("[bench] pmc launches done (copy calibration: 1 GiB read, 1 GiB "
              "written per copy)", file=sys.stderr, flush=True)
        return

    def step(i):
        s = w.steps[i % n_sweep]
        m = L.build_mask_device(w.frames, w.tokens_per_frame, w.block, s, rp, ci,
                                params=params, stream=stream)
        L.attention(q, k, v, m, out=out, stream=stream)
        return s

    print("[bench] warmup", file=sys.stderr, flush=True)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    print("[bench] timed steps", file=sys.stderr, flush=True)
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record()
    total_flops = 0.0
    for i in range(args.steps):
        s = step(args.warmup + i)
        total_flops += flops_of[s]
    t_end.record()
    torch.cuda.synchronize()
    ms_step = t_start.elapsed_time(t_end) / args.steps
    value = total_flops / args.steps / (ms_step * 1e-3) / 1e12

    # Attention call alone at step 10 and the device mask build alone.
    s_ref = 10 if 10 in flops_of else w.steps[0]
    m = L.build_mask_device(w.frames, w.tokens_per_frame, w.block, s_ref, rp, ci,
                            params=params, stream=stream)
    attn_ms = time_calls(lambda: L.attention(q, k, v, m, out=out, stream=stream),
                         20, 3)
    attn_med = median(attn_ms)
    spread = {"p10": percentile(attn_ms, 0.1), "p90": percentile(attn_ms, 0.9),
              "min": min(attn_ms), "max": max(attn_ms), "calls": len(attn_ms)}
    # Cold caches: before each timed call, overwrite a 1 GiB buffer (more than
    # the L2s and the 256 MB last-level cache hold) so Q, K, V start in HBM.
    flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    cold = []
    for _ in range(5):
        flush.fill_(1.0)
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        L.attention(q, k, v, m, out=out, stream=stream)
        b.record()
        torch.cuda.synchronize()
        cold.append(a.elapsed_time(b))
    del flush
    mask_ms = time_calls(lambda: L.build_mask_device(
        w.frames, w.tokens_per_frame, w.block, s_ref, rp, ci, params=params,
        stream=stream), 20, 3)
    print(f"[bench] attention {attn_med:.3f} ms", file=sys.stderr, flush=True)

    # Token-exact form (Eq. 2 token for token) at the same step: the same
    # kept blocks, with frame-edge parts of straddling blocks masked.
    ent = torch.empty(nb * nb, dtype=torch.int32, device="cuda")
    exact = {}
    try:
        me = L.build_exact_mask_device(w.frames, w.tokens_per_frame, w.block, s_ref,
                                       rp, ent, params=params, stream=stream)
    except L.LvsaError:
        me = None
    if me is not None:
        ex_med = median(time_calls(
            lambda: L.attention_exact(q, k, v, me, out=out, stream=stream), 20, 3))
        _, anc, lo, hi = L.frame_sets(w.frames, s_ref, params)
        per_frame = [len(set(anc) | set(range(lo[t], hi[t] + 1)))
                     for t in range(w.frames)]
        eq2_flops = 4.0 * 128 * w.heads * eq2_pairs(per_frame, w.tokens_per_frame,
                                                    w.text_tokens, w.n_tokens)
        host_ex = []
        for _ in range(5):
            t0 = time.perf_counter()
            L.build_mask(w.frames, w.tokens_per_frame, w.block, s_ref, params,
                         exact=True).free()
            host_ex.append((time.perf_counter() - t0) * 1e6)
        exact = {
            "exact_ms_per_call": ex_med,
            "exact_mask_build_host_us": median(host_ex),
            "exact_tflops_eq2_pairs": eq2_flops / (ex_med * 1e-3) / 1e12,
            "exact_vs_block_time": ex_med / attn_med,
            "token_density_step10": eq2_flops / (4.0 * 128 * w.heads * w.n_tokens ** 2),
        }
        print(f"[bench] exact attention {ex_med:.3f} ms", file=sys.stderr, flush=True)
        # The block form again, for the step loop's mask buffers.
        m = L.build_mask_device(w.frames, w.tokens_per_frame, w.block, s_ref, rp, ci,
                                params=params, stream=stream)

    # Pattern variants of Sec. 2 at the same step: window rule, fixed vs
    # rotating anchors, a dedicated initial anchor.  Block density, token
    # density (Eq. 2) and the block-sparse call time of each.
    variants = []
    if not args.no_patterns:
        print("[bench] pattern variants", file=sys.stderr, flush=True)
        names = {L.WINDOW_BASIC: "basic", L.WINDOW_ADAPTIVE: "adaptive",
                 L.WINDOW_EXPANDED: "expanded"}
        for mode, rotate, extra in [(L.WINDOW_EXPANDED, 1, 0), (L.WINDOW_ADAPTIVE, 1, 0),
                                    (L.WINDOW_BASIC, 1, 0), (L.WINDOW_EXPANDED, 0, 0),
                                    (L.WINDOW_EXPANDED, 1, 1)]:
            pv = L.Params(budget_frames=w.budget_frames, window=w.window, tper=w.tper,
                          window_mode=mode, rotate=rotate, extra_anchors=extra,
                          text_tokens=w.text_tokens)
            csr = L.build_mask(w.frames, w.tokens_per_frame, w.block, s_ref, pv)
            hrp, hci = csr.arrays()
            csr.upload(stream)
            mv = csr.device_mask()
            v_ms = median(time_calls(
                lambda: L.attention(q, k, v, mv, out=out, stream=stream), 10, 2))
            fl = kept_flops(hrp, hci, w.n_tokens, w.block, w.heads)
            tper, anc, lo, hi = L.frame_sets(w.frames, s_ref, pv)
            sizes = [len(set(anc) | set(range(lo[t], hi[t] + 1))) for t in range(w.frames)]
            variants.append({
                "window": names[mode], "rotate": bool(rotate), "extra_anchors": extra,
                "T_per": tper, "frames_per_query_min": min(sizes),
                "frames_per_query_max": max(sizes),
                "block_density": int(hrp[-1]) / (nb * nb),
                "token_density": eq2_pairs(sizes, w.tokens_per_frame, w.text_tokens,
                                           w.n_tokens) / w.n_tokens ** 2,
                "ms_per_call": v_ms, "tflops_kept": fl / (v_ms * 1e-3) / 1e12,
            })
            csr.free()

    dense = {}
    if not args.no_dense:
        print("[bench] dense", file=sys.stderr, flush=True)
        # Dense attention through the dense entry point, and through the
        # block-sparse kernel with a full mask (a window of T frames keeps
        # every block), timed in alternation (two calls of each, five
        # times) so that the board's clock drift weighs on both alike; the
        # speedup divides by the dense entry point.
        full = L.Params(budget_frames=w.budget_frames, window=w.frames, tper=w.frames,
                        text_tokens=w.text_tokens)
        mf = L.build_mask_device(w.frames, w.tokens_per_frame, w.block, s_ref, rp, ci,
                                 params=full, stream=stream)
        torch.cuda.synchronize()
        assert int(rp[-1]) == nb * nb, "full mask expected"
        d_all, f_all = [], []
        for rnd in range(5):
            d_all += time_calls(lambda: L.dense_attention(q, k, v, block=w.block, out=out,
                                                          stream=stream), 2, 1 if rnd == 0 else 0)
            f_all += time_calls(lambda: L.attention(q, k, v, mf, out=out, stream=stream),
                                2, 1 if rnd == 0 else 0)
        d_ms, f_ms = median(d_all), median(f_all)
        dense = {
            "dense_ms_per_call": d_ms,
            "dense_full_mask_ms_per_call": f_ms,
            "dense_tflops": dense_flops / (d_ms * 1e-3) / 1e12,
            "speedup_vs_dense": d_ms / attn_med,
            "inv_density": dense_flops / flops_of[s_ref],
        }

    achieved = flops_of[s_ref] / (attn_med * 1e-3) / 1e12
    traffic = traffic_from_profile(w.name, SPARSE_KERNEL)
    meta = metadata_costs(w, L, params)
    rec = {
        "metric": METRIC,
        "value": value,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "desc": w.desc,
            "heads": w.heads,
            "n_tokens": w.n_tokens,
            "head_dim": 128,
            "block": w.block,
            "mask": {"C": w.budget_frames, "W": w.window, "window": "expanded",
                     "rotate": True, "steps_swept": f"{w.steps[0]}..{w.steps[-1]}"},
            "parallelism": "single GPU",
        },
        "ms_per_attention_call": attn_med,
        "ms_per_attention_call_spread": spread,
        "ms_per_attention_call_cold_caches": median(cold),
        "attention_tflops_kept": achieved,
        "mask_build_device_us": median(mask_ms) * 1e3,
        "mask_build_host_us": median(host_us),
        "mask_build_host_us_p90": percentile(host_us, 0.9),
        **meta,
        "nnz_step10": nnz_of[s_ref],
        "block_density_step10": nnz_of[s_ref] / (nb * nb),
        **exact,
        **({"pattern_variants": variants} if variants else {}),
        **dense,
        "roofline": {
            "kernel": SPARSE_KERNEL,
            "bound": "mfma",
            "achieved": achieved,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS,
            "traffic": traffic,
        },
    }
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        rec["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
