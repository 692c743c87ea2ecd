#!/usr/bin/env python3
"""Benchmark of the BDLM attention hot path on one MI355X.

Headline: fused BDLM attention forward + backward at 32K context (batch 1,
L = 32768 clean + 32768 corrupted tokens, block size 64, 32 query / 8 KV heads,
head_dim 128, bf16 inputs, fp32 accumulation, bf16 outputs), seeded synthetic
N(0, 1) inputs resident in HBM before the timed region.  One step = one
bdlm_attn_fwd + one bdlm_attn_bwd call (tile classification, fused forward,
the query-major dQ kernel, which also forms D = rowsum(dO * O), and the
key-major dK/dV kernel).

value = useful TFLOP/s: valid query-key pairs of the mask (the paper's unit of
attention work, App. B) x (4 d forward + 10 d backward) FLOP, divided by the
measured step time.  Masked entries inside partly visible tiles and skipped
tiles are never counted.

Also reported on the same JSON line:
* roofline of the dominant kernel (the fused backward), timed per launch with
  HIP events the library records around each kernel on the launch stream;
* per-kernel averages of the step;
* one 256K CSBP rank's share (17 partial forwards, a 17-way LSE merge and the
  backward over the 17 key ranges) with the merge kernel's HBM roofline;
* the mask generalisations at full size (mask_ext): the 32K shape in a
  1,024-position sliding-window layer, and a drafter share of 2,048 draft
  blocks of 16 over 32K target features with sorted anchors;
* cpu_baseline: the fp64 oracle timed on this host on a bounded sample of the
  same workload (evenly spaced query rows of one head, forward + backward).

Only one GPU is used: --gpus N with N > 1 exits with a message.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "BDLM attn fwd+bwd useful TFLOP/s & MFMA util at 32K ctx, 1 MI355X"
PEAK_BF16_TFLOPS = 256 * 4096 * 2.4e9 / 1e12  # 256 CUs x 2048 bf16 FMA/clk/CU x 2 x 2.4 GHz = 2516.6
PEAK_HBM_GBS = 8000.0
# Sources each timed kernel is built from (a recorded counter value is only
# trusted while these are unchanged).
KERNEL_SOURCES = {
    "fwd_bf16": ["common.hpp", "device.hpp", "qtiles.hpp", "fwd_bf16.hip"],
    "bwd_dkdv_bf16": ["common.hpp", "device.hpp", "bwd_dkdv.hip"],
    "bwd_dq_bf16": ["common.hpp", "device.hpp", "qtiles.hpp", "bwd_dq.hip"],
}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_32k.json")


def strip_comments(src):
    """C++ source without its comments and blank lines (a comment edit leaves the hash alone)."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c == '"':  # string literal, copied whole
            j = i + 1
            while j < n and src[j] != '"':
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return "\n".join(ln.rstrip() for ln in "".join(out).splitlines() if ln.strip())


def kernel_source_hash(kernel):
    """Hash of a kernel's sources (comments stripped) and of their per-source compile options."""
    from paper_2609_19242_amd import build
    h = hashlib.sha256()
    for f in KERNEL_SOURCES.get(kernel, []):
        with open(os.path.join(ROOT, "paper_2609_19242_amd", "csrc", f), encoding="utf-8") as fh:
            h.update(strip_comments(fh.read()).encode())
        h.update(" ".join(build.EXTRA_FLAGS.get(f, [])).encode())
    return h.hexdigest()[:16]


def recorded_traffic(kernel):
    """HBM bytes per launch of `kernel` from rocprofv3 FETCH_SIZE/WRITE_SIZE runs, if taken on its current source."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f).get(kernel)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_sha256_16") != kernel_source_hash(kernel):
        return None
    return rec.get("hbm_bytes_per_launch")


def per_kernel(records):
    out = {}
    for name, ms in records:
        d = out.setdefault(name, [0.0, 0])
        d[0] += ms
        d[1] += 1
    return {k: {"avg_ms": v[0] / v[1], "launches": v[1]} for k, v in out.items()}


def bench_32k(torch, bd, synth, steps, warmup, reading=0):
    w = synth.WORKLOADS["32k"]
    dev = "cuda"
    q, k, v, do = synth.make_joint(w, device=dev)
    B, n, Hq, D = q.shape
    L, M = w.L, w.block_size
    p = bd.make_problem(B, L, M, Hq, w.kv_heads, D, torch.bfloat16, clean_intra=reading)
    r = bd.joint_ranges(L)
    pairs = bd.visible_pairs(p, r, r)
    fl = bd.useful_flops(pairs, Hq, B, D)
    o = torch.empty_like(q)
    lse = torch.empty((B, Hq, n), dtype=torch.float32, device=dev)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, r), dtype=torch.uint8, device=dev)

    def step():
        bd.joint_fwd(q, k, v, M, out=(o, lse), clean_intra=reading)
        bd.joint_bwd(q, k, v, o, lse, do, M, out=(dq, dk, dv), workspace=ws, clean_intra=reading)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    bd.timing_enable(True)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(steps):
        step()
        ev[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    bd.timing_enable(False)
    kern = per_kernel(bd.timing_collect())
    per_step = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(steps))
    ms = ev[0].elapsed_time(ev[steps]) / steps
    median_ms = per_step[steps // 2] if steps % 2 else 0.5 * (per_step[steps // 2 - 1] + per_step[steps // 2])
    assert torch.isfinite(o).all() and torch.isfinite(dq).all()
    # Algorithmic FLOP per valid pair of each kernel: forward 4d (Q K^T, P V);
    # dK/dV kernel 8d (Q K^T, dO V^T, P^T dO, dS^T Q); dQ kernel 6d (Q K^T and
    # dO V^T recomputed, dS K).  The useful total of a step stays 14d per pair.
    per_pair = {"fwd_bf16": 4, "bwd_dkdv_bf16": 8, "bwd_dq_bf16": 6}
    n_pairs = pairs * Hq * B
    for name, kd in kern.items():
        if name in per_pair:
            kd["flop_per_launch"] = per_pair[name] * D * n_pairs
            kd["tflops"] = kd["flop_per_launch"] / (kd["avg_ms"] * 1e-3) / 1e12
    dom = max(kern, key=lambda n: kern[n]["avg_ms"])
    achieved = kern[dom]["tflops"]
    roof = {"bound": "mfma", "kernel": dom, "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS, "traffic": recorded_traffic(dom),
            "flop_per_launch": kern[dom]["flop_per_launch"], "avg_launch_ms": kern[dom]["avg_ms"]}
    fwd_ms = kern["fwd_bf16"]["avg_ms"]
    bwd_ms = sum(kern[k]["avg_ms"] for k in ("bwd_pre", "bwd_dkdv_bf16", "bwd_dq_bf16") if k in kern)
    res = {"ms_per_step": ms, "median_ms_per_step": median_ms, "fwd_ms": fwd_ms, "bwd_ms": bwd_ms,
           "wall_s": wall, "pairs_per_head": pairs, "flops": fl, "kernels": kern,
           "roofline": roof, "value": fl["total"] / (median_ms * 1e-3) / 1e12,
           "mean_value": fl["total"] / (ms * 1e-3) / 1e12, "workload": w}
    del q, k, v, do, o, lse, dq, dk, dv, ws
    torch.cuda.empty_cache()
    return res


def bench_csbp(torch, bd, synth, steps, warmup):
    w = synth.WORKLOADS["csbp256k"]
    dev = "cuda"
    q, kl, vl, kc, vc, do = synth.make_csbp_rank(w, device=dev)
    Hq, D, n = w.heads, w.head_dim, w.local_tokens
    p = bd.make_problem(1, w.L, w.block_size, Hq, w.kv_heads, D, torch.bfloat16)
    qr = bd.Range(bd.CORRUPTED, w.local_pos0, n)
    krs = [bd.Range(bd.CORRUPTED, w.local_pos0, n)] + \
          [bd.Range(bd.CLEAN, s * w.shard_tokens, w.shard_tokens) for s in range(w.n_shards)]
    step_b = w.shard_tokens * w.kv_heads * D * 2
    ks = [kl.data_ptr()] + [kc.data_ptr() + s * step_b for s in range(w.n_shards)]
    vs = [vl.data_ptr()] + [vc.data_ptr() + s * step_b for s in range(w.n_shards)]
    dkl, dvl, dkc, dvc = (torch.empty_like(t) for t in (kl, vl, kc, vc))
    dks = [dkl.data_ptr()] + [dkc.data_ptr() + s * step_b for s in range(w.n_shards)]
    dvs = [dvl.data_ptr()] + [dvc.data_ptr() + s * step_b for s in range(w.n_shards)]
    J = len(krs)
    o_parts = [torch.empty_like(q) for _ in range(J)]
    l_parts = [torch.empty((1, Hq, n), dtype=torch.float32, device=dev) for _ in range(J)]
    om, dq = torch.empty_like(q), torch.empty_like(q)
    lm = torch.empty((1, Hq, n), dtype=torch.float32, device=dev)
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, [qr]), dtype=torch.uint8, device=dev)
    pairs = bd.visible_pairs(p, [qr], krs)
    fl = bd.useful_flops(pairs, Hq, 1, D)

    def step():
        for j in range(J):
            bd.attn_partial_fwd(p, qr, q, o_parts[j], l_parts[j], krs[j], ks[j], vs[j])
        bd.lse_merge(o_parts, l_parts, om, lm)
        bd.attn_bwd(p, [qr], [q], [om], [lm], [do], [dq], krs, ks, vs, dks, dvs, ws)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    bd.timing_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    bd.timing_enable(False)
    kern = per_kernel(bd.timing_collect())
    ms = e0.elapsed_time(e1) / steps
    # merge: algorithmic bytes.  Every part's LSE is read; O_j is read only where
    # w_j != 0, which here is every row of the non-empty parts.
    nonempty = int(sum(bool(torch.isfinite(l).any()) for l in l_parts))
    rows_h = n * Hq
    merge_bytes = nonempty * rows_h * D * 2 + J * rows_h * 4 + rows_h * D * 2 + rows_h * 4
    mms = kern["lse_merge"]["avg_ms"]
    gbs = merge_bytes / (mms * 1e-3) / 1e9
    res = {"workload": w.describe(), "ms_per_step": ms, "useful_tflops": fl["total"] / (ms * 1e-3) / 1e12,
           "pairs_per_head": pairs, "kernels": kern,
           "merge_roofline": {"bound": "hbm", "kernel": "lse_merge", "achieved": gbs, "peak": PEAK_HBM_GBS,
                              "unit": "GB/s", "frac": gbs / PEAK_HBM_GBS, "bytes_per_launch": merge_bytes,
                              "parts": J, "parts_read": nonempty}}

    # The whole rank operator: the rank's clean-shard queries as well (they attend
    # causally to the gathered clean shards), one multi-range forward launch for
    # them and one backward over both query ranges.
    own = synth.csbp_own_shard(w)
    S = w.shard_tokens
    qc, doc = synth.make_csbp_clean_queries(w, device=dev)
    qrc = bd.Range(bd.CLEAN, own * S, S)
    oc, dqc = torch.empty_like(qc), torch.empty_like(qc)
    lc = torch.empty((1, Hq, S), dtype=torch.float32, device=dev)
    ws2 = torch.empty(bd.attn_bwd_workspace_bytes(p, [qr, qrc]), dtype=torch.uint8, device=dev)
    pairs2 = bd.visible_pairs(p, [qr, qrc], krs)
    fl2 = bd.useful_flops(pairs2, Hq, 1, D)

    def rank_step():
        for j in range(J):
            bd.attn_partial_fwd(p, qr, q, o_parts[j], l_parts[j], krs[j], ks[j], vs[j])
        bd.lse_merge(o_parts, l_parts, om, lm)
        bd.attn_fwd(p, [qrc], [qc], [oc], [lc], krs, ks, vs)
        bd.attn_bwd(p, [qr, qrc], [q, qc], [om, oc], [lm, lc], [do, doc], [dq, dqc], krs, ks, vs, dks, dvs, ws2)

    for _ in range(warmup):
        rank_step()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        rank_step()
    e1.record()
    torch.cuda.synchronize()
    ms2 = e0.elapsed_time(e1) / steps
    res["rank_operator"] = {"workload": "the same rank plus its 16384 clean-shard queries (shard %d)" % own,
                            "ms_per_step": ms2, "useful_tflops": fl2["total"] / (ms2 * 1e-3) / 1e12,
                            "pairs_per_head": pairs2}
    return res


def _timed_steps(torch, bd, step, steps, warmup):
    """Warm up, then time ``steps`` calls of ``step`` with per-kernel HIP-event records."""
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    bd.timing_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    bd.timing_enable(False)
    return e0.elapsed_time(e1) / steps, per_kernel(bd.timing_collect())


def bench_ext(torch, bd, synth, steps, warmup):
    """The mask generalisations at full size: the 32K shape in a sliding-window
    layer (1,024 positions) and a DFlash2 drafter share (2,048 draft blocks of
    16 over 32K target features).  Useful TFLOP/s on their own valid pairs."""
    out = {}
    w = synth.WORKLOADS["32k-w1024"]
    q, k, v, do = synth.make_joint(w, device="cuda")
    L, M = w.L, w.block_size
    p = bd.make_problem(1, L, M, w.heads, w.kv_heads, w.head_dim, torch.bfloat16, window=w.window)
    r = bd.joint_ranges(L)
    pairs = bd.visible_pairs(p, r, r)
    o, lse = torch.empty_like(q), torch.empty((1, w.heads, 2 * L), dtype=torch.float32, device="cuda")
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, r), dtype=torch.uint8, device="cuda")

    def step_w():
        bd.joint_fwd(q, k, v, M, out=(o, lse), window=w.window)
        bd.joint_bwd(q, k, v, o, lse, do, M, out=(dq, dk, dv), workspace=ws, window=w.window)

    ms, kern = _timed_steps(torch, bd, step_w, steps, warmup)
    fl = bd.useful_flops(pairs, w.heads, 1, w.head_dim)
    out["window32k"] = {"workload": w.describe(), "ms_per_step": ms, "useful_tflops": fl["total"] / (ms * 1e-3) / 1e12,
                        "pairs_per_head": pairs, "kernels": kern}
    del q, k, v, do, o, lse, dq, dk, dv, ws
    torch.cuda.empty_cache()

    w = synth.WORKLOADS["drafter32k"]
    q, kd, vd, kt, vt, do, anchors = synth.make_drafter(w, device="cuda")
    nd = w.draft_blocks * w.block_size
    p = bd.make_problem(1, w.L, w.block_size, w.heads, w.kv_heads, w.head_dim, torch.bfloat16, clean_prefix=anchors)
    qr = [bd.Range(bd.CORRUPTED, 0, nd)]
    kr = [bd.Range(bd.CORRUPTED, 0, nd), bd.Range(bd.CLEAN, 0, w.L)]
    pairs = bd.visible_pairs(p, qr, kr)
    o, lse = torch.empty_like(q), torch.empty((1, w.heads, nd), dtype=torch.float32, device="cuda")
    dq = torch.empty_like(q)
    dks = [torch.empty_like(kd), torch.empty_like(kt)]
    dvs = [torch.empty_like(vd), torch.empty_like(vt)]
    ws = torch.empty(bd.attn_bwd_workspace_bytes(p, qr), dtype=torch.uint8, device="cuda")

    def step_d():
        bd.attn_fwd(p, qr, [q], [o], [lse], kr, [kd, kt], [vd, vt])
        bd.attn_bwd(p, qr, [q], [o], [lse], [do], [dq], kr, [kd, kt], [vd, vt], dks, dvs, ws)

    ms, kern = _timed_steps(torch, bd, step_d, steps, warmup)
    assert torch.isfinite(o).all() and torch.isfinite(dq).all()
    fl = bd.useful_flops(pairs, w.heads, 1, w.head_dim)
    out["drafter32k"] = {"workload": w.describe(), "ms_per_step": ms, "useful_tflops": fl["total"] / (ms * 1e-3) / 1e12,
                         "pairs_per_head": pairs, "kernels": kern}
    del q, kd, vd, kt, vt, do, anchors, o, lse, dq, dks, dvs, ws
    torch.cuda.empty_cache()
    return out


def bench_configs(torch, bd, synth, steps, warmup):
    """Step time of the other joint workloads: 4k (batch 2, block 32; bf16 outputs,
    single-term products, as the headline) and 128k (block 128, 64/8 heads, 1% of
    keys x8) in the arithmetic its parity needs: fp32 outputs and every P and dS
    product in two bf16 terms on the tiles holding a probability of 1/64 or more."""
    out = {}
    legs = (("4k", dict(), steps, warmup),
            ("128k", dict(out_f32=True, hilo=bd.HILO_ALL | bd.HILO_ADAPTIVE), max(2, steps // 4), 1))
    for name, arith, n_steps, n_warm in legs:
        w = synth.WORKLOADS[name]
        q, k, v, do = synth.make_joint(w, device="cuda")
        B, n, Hq, D = q.shape
        L, M = w.L, w.block_size
        p = bd.make_problem(B, L, M, Hq, w.kv_heads, D, torch.bfloat16, **arith)
        r = bd.joint_ranges(L)
        pairs = bd.visible_pairs(p, r, r)
        odt = torch.float32 if arith.get("out_f32") else torch.bfloat16
        o, lse = torch.empty(q.shape, dtype=odt, device="cuda"), torch.empty((B, Hq, n), dtype=torch.float32,
                                                                              device="cuda")
        dq, dk, dv = (torch.empty(t.shape, dtype=odt, device="cuda") for t in (q, k, v))
        ws = torch.empty(bd.attn_bwd_workspace_bytes(p, r), dtype=torch.uint8, device="cuda")

        def step():
            bd.joint_fwd(q, k, v, M, out=(o, lse), **arith)
            bd.joint_bwd(q, k, v, o, lse, do, M, out=(dq, dk, dv), workspace=ws, **arith)

        ms, kern = _timed_steps(torch, bd, step, n_steps, n_warm)
        fl = bd.useful_flops(pairs, Hq, B, D)
        desc = w.describe() + (", fp32 outputs, two-term P and dS products on tiles with P >= 1/64" if arith
                               else ", bf16 outputs")
        out[name] = {"workload": desc, "ms_per_step": ms, "steps": n_steps,
                     "useful_tflops": fl["total"] / (ms * 1e-3) / 1e12, "pairs_per_head": pairs, "kernels": kern}
        print(f"[bench] {name}: {ms:.3f} ms/step, {out[name]['useful_tflops']:.1f} useful TFLOP/s", flush=True)
        del q, k, v, do, o, lse, dq, dk, dv, ws
        torch.cuda.empty_cache()
    return out


def cpu_baseline(bd, synth, budget_s):
    """The fp64 oracle on the host: forward + backward of evenly spaced query rows of one head of the 32K workload."""
    import numpy as np
    import oracle
    w = synth.WORKLOADS["32k"]
    L, M, D = w.L, w.block_size, w.head_dim
    q, k, v, do = synth.make_joint(w, device="cpu")
    h = 0
    kv = h // (w.heads // w.kv_heads)
    k0 = k[:, :, kv:kv + 1].double().numpy()
    v0 = v[:, :, kv:kv + 1].double().numpy()
    r = oracle.joint_ranges(L)
    s_all, p_all = oracle.rows_of(r)
    chunk_rows = 64
    n_chunks = (2 * L) // chunk_rows
    order = np.random.default_rng(0).permutation(n_chunks)
    pairs = 0
    rows_done = 0
    cores = len(os.sched_getaffinity(0))
    from threadpoolctl import threadpool_limits, threadpool_info
    limiter = threadpool_limits(limits=cores, user_api="blas")
    blas_threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    t0 = time.perf_counter()
    for c in order:
        rows = list(range(c * chunk_rows, (c + 1) * chunk_rows))
        single = [(int(s_all[i]), int(p_all[i]), 1) for i in rows]
        qs, dos = q[:, rows, h:h + 1], do[:, rows, h:h + 1]
        O, LSE = oracle.fwd(qs, k0, v0, single, r, M)
        oracle.bwd(qs, k0, v0, O, LSE, dos, single, r, M)
        pairs += oracle.count_visible_pairs(single, r, M)
        rows_done += len(rows)
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    limiter.restore_original_limits()
    flops = 14 * D * pairs
    return {"value": flops / el / 1e12, "unit": "TFLOP/s", "cores": blas_threads, "cores_available": cores,
            "kind": "oracle",
            "sample": f"{rows_done} query rows (random 64-row chunks) x 1 head of the 32K workload, "
                      f"fp64 forward+backward over all their visible keys ({pairs} pairs) in {el:.1f} s",
            "seconds": el}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--cpu-budget-s", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-csbp", action="store_true")
    ap.add_argument("--no-ext", action="store_true", help="skip the sliding-window and drafter legs")
    ap.add_argument("--no-configs", action="store_true", help="skip the 4k and 128k workload legs")
    ap.add_argument("--configs-only", action="store_true",
                    help="time only the 4k and 128k joint workloads and print their result")
    ap.add_argument("--ext-only", action="store_true",
                    help="run only the sliding-window and drafter legs and print their result")
    ap.add_argument("--csbp-only", action="store_true",
                    help="run only the 256K CSBP leg and print its result (for per-workload kernel profiles)")
    ap.add_argument("--pmc-pass", action="store_true",
                    help="one 32K fwd+bwd step and a plain 1 GiB device copy, for rocprofv3 counter runs")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (the data-parallel hot path of one rank); "
              f"--gpus {args.gpus} / WORLD_SIZE={world} is not supported", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_19242_amd as bd
    import synth
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    bd.lib()  # fail loudly if the HIP library is missing

    if args.pmc_pass:
        # Counter runs: one warm step of every kernel, then a plain copy of known
        # size (2^30 bytes read, 2^30 written) that calibrates FETCH_SIZE / WRITE_SIZE.
        bench_32k(torch, bd, synth, 1, 1)
        src = torch.empty(1 << 29, dtype=torch.bfloat16, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print("[bench] pmc pass done", flush=True)
        return
    if args.configs_only:
        print(json.dumps({"configs": bench_configs(torch, bd, synth, args.steps, args.warmup)}), flush=True)
        return
    if args.ext_only:
        print(json.dumps({"ext": bench_ext(torch, bd, synth, args.steps, args.warmup)}), flush=True)
        return
    if args.csbp_only:
        res = bench_csbp(torch, bd, synth, args.steps, args.warmup)
        print(json.dumps({"csbp256k": res}), flush=True)
        return
    main_res = bench_32k(torch, bd, synth, args.steps, args.warmup)
    print(f"[bench] 32k: {main_res['median_ms_per_step']:.3f} ms/step (median), {main_res['value']:.1f} useful TFLOP/s",
          flush=True)
    blk = bench_32k(torch, bd, synth, max(3, args.steps // 2), 1, reading=1)
    block_reading = {"workload": blk["workload"].describe() + ", clean-to-clean block reading",
                     "median_ms_per_step": blk["median_ms_per_step"], "useful_tflops": blk["value"],
                     "pairs_per_head": blk["pairs_per_head"], "fwd_ms": blk["fwd_ms"], "bwd_ms": blk["bwd_ms"]}
    print(f"[bench] 32k block reading: {blk['median_ms_per_step']:.3f} ms/step, {blk['value']:.1f} useful TFLOP/s",
          flush=True)
    configs = None if args.no_configs else bench_configs(torch, bd, synth, args.steps, args.warmup)
    csbp = None if args.no_csbp else bench_csbp(torch, bd, synth, max(2, args.steps // 2), 1)
    if csbp:
        print(f"[bench] csbp256k: {csbp['ms_per_step']:.3f} ms/step; with clean-shard queries "
              f"{csbp['rank_operator']['ms_per_step']:.3f} ms/step", flush=True)
    ext = None if args.no_ext else bench_ext(torch, bd, synth, max(2, args.steps // 2), 1)
    if ext:
        print("[bench] " + "; ".join(f"{n}: {r['ms_per_step']:.3f} ms/step, {r['useful_tflops']:.1f} useful TFLOP/s"
                                     for n, r in ext.items()), flush=True)
    cpu = None if args.no_cpu_baseline else cpu_baseline(bd, synth, args.cpu_budget_s)
    w = main_res["workload"]
    line = {
        "metric": METRIC,
        "value": main_res["value"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_res["median_ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.describe(), "batch": w.batch, "L": w.L, "block_size": w.block_size,
                   "heads": w.heads, "kv_heads": w.kv_heads, "head_dim": w.head_dim, "clean_intra": "causal",
                   "parallelism": "single GPU"},
        "mfma_util_useful": main_res["value"] / PEAK_BF16_TFLOPS,
        "mean_ms_per_step": main_res["ms_per_step"],
        "value_from_mean_step": main_res["mean_value"],
        "fwd_ms": main_res["fwd_ms"],
        "bwd_ms": main_res["bwd_ms"],
        "fwd_useful_tflops": main_res["flops"]["fwd"] / (main_res["fwd_ms"] * 1e-3) / 1e12,
        "bwd_useful_tflops": main_res["flops"]["bwd"] / (main_res["bwd_ms"] * 1e-3) / 1e12,
        # the stricter convention: 12 d per valid pair (no S recompute in the backward)
        "useful_tflops_12d": main_res["value"] * 12 / 14,
        "useful_flop_per_step": main_res["flops"]["total"],
        "roofline": main_res["roofline"],
        "kernels": main_res["kernels"],
        "cpu_baseline": cpu,
        "block_reading_32k": block_reading,
        "csbp256k": csbp,
        "mask_ext": ext,
        "configs": configs,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
