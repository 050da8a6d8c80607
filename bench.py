"""Benchmark of the bounded-window restore path on one MI355X.

One step = one pass of the whole path over one request: probe (chunk keys +
store lookup), bind (begin kernel), every window's pinned-host -> ring copies
and install + verify kernels, and the device commit, ending when commit has
returned to the host.  The external tier is the library's pinned-host store,
filled before timing; destination pools are resident in HBM.

Prints ONE JSON line.  ``value`` is restored KV bytes per second (1e9 B/s):
n_hit x (bytes of one chunk's entries) x steps / timed seconds.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, published
# MI355X's host interface, PCIe Gen5 x16, per direction: 32 GT/s x 16 lanes
# x 128/130 encoding / 8 bits
LINK_PEAK_GBPS = 32 * 16 * 128 / 130 / 8


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", type=int, default=5, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--window", type=int, default=32, help="W in chunks; 0 = legacy whole-plan mode")
    ap.add_argument("--install-batch", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target oracle sample time")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 1 GiB device copy (for counter calibration)")
    ap.add_argument("--held-chunks", type=int, default=0,
                    help="profiling passes only: hold just the first N chunks (same launch shape)")
    ap.add_argument("--tier", choices=["pinned", "file"], default="pinned",
                    help="external tier holding the chunks: the pinned-host store or the file tier")
    ap.add_argument("--file-dir", default="", help="file tier directory (default /tmp/bsr_tier_<workload>)")
    ap.add_argument("--load-concurrency", type=int, default=4, help="file tier reader threads")
    ap.add_argument("--direct", action="store_true", help="file tier reads with O_DIRECT")
    ap.add_argument("--concurrency-sweep", default="",
                    help="file tier only: comma-separated load concurrencies to measure as well")
    ap.add_argument("--copy-engine", choices=["kernel", "sdma"], default="kernel",
                    help="staging copies by the library's kernel (default) or by the copy engine")
    ap.add_argument("--two-streams", action="store_true",
                    help="stage on the copy stream whatever the request's size (BSR_FLAG_TWO_STREAMS)")
    ap.add_argument("--only-group", default="",
                    help="profiling: install these groups of the workload alone (comma-separated indices), their "
                         "tensor counts scaled together so that a chunk holds as many bytes as the whole layout's "
                         "chunk (the same launch size)")
    ap.add_argument("--scatter-ceiling", action="store_true",
                    help="also measure a plain scattered copy of each group's block size at the install's "
                         "launch size (bsr_measure_scatter)")
    ap.add_argument("--requests", type=int, default=1,
                    help="requests bound at once under a global admission budget B = requests x ring "
                         "(each with its own ring and destination pools; windows interleaved)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (--gpus {args.gpus} "
              "requested); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_17826_amd import bsr
    from paper_2608_17826_amd.session import RestoreSession, group_dsts
    from workloads import generate, get_config
    from workloads.device import place

    w = get_config(args.workload)
    if args.only_group:
        w = groups_alone(w, [int(x) for x in args.only_group.split(",")])
    W = args.window
    log(f"[bench] workload {w.index} {w.name}: generating inputs")
    wi = generate(w)
    kinds = {"contig": bsr.BSR_KIND_CONTIG, "planar": bsr.BSR_KIND_PLANAR}
    layout = bsr.make_layout(w.chunk_tokens, [(s.block_tokens, s.n_tensors, s.record_bytes, kinds[s.kind],
                                               s.split_bytes) for s in w.groups])
    K = args.requests
    if K < 1 or K > bsr.BSR_MAX_BOUND_REQUESTS:
        print(f"--requests must be in 1..{bsr.BSR_MAX_BOUND_REQUESTS}", file=sys.stderr)
        sys.exit(2)
    slot = bsr.bsr_slot_bytes(layout)
    held_plan = w.held_chunks if not args.held_chunks else min(args.held_chunks, w.held_chunks)
    budget = 0 if K == 1 else K * (W or held_plan) * slot
    copy_flag = (bsr.BSR_FLAG_SDMA_COPIES if args.copy_engine == "sdma" else 0) | \
        (bsr.BSR_FLAG_TWO_STREAMS if args.two_streams else 0)
    ctx = bsr.bsr_ctx_create(layout, W, hip_device=0, install_batch=args.install_batch,
                             flags=bsr.BSR_FLAG_TIME_INSTALL | copy_flag, staging_budget_bytes=budget,
                             max_bound_requests=0 if K == 1 else K)
    stride = (slot + 4095) // 4096 * 4096
    held = w.held_chunks if not args.held_chunks else min(args.held_chunks, w.held_chunks)
    keys = bsr.bsr_chunk_keys(wi.salt, wi.tokens, w.chunk_tokens)
    file_dir = args.file_dir or f"/tmp/bsr_tier_{w.name}"
    t0 = time.time()
    if args.tier == "pinned":
        log(f"[bench] pinned store: {held} chunks x {slot} B")
        bsr.bsr_store_reserve(ctx, stride * (held + 1))
        # the prompt's chunks are stored together, back to back in the arena
        bsr.bsr_store_put_chunks(ctx, keys[:held], [wi.payloads(i) for i in range(held)])
    else:
        log(f"[bench] file tier {file_dir}: {held} chunks x {slot} B, load concurrency {args.load_concurrency}")
        bsr.bsr_store_reserve(ctx, stride)
        open_file_tier(bsr, ctx, file_dir, args.load_concurrency, args.direct)

        def put(i):
            bsr.bsr_file_tier_put_chunk(ctx, int(keys[i]), wi.payloads(i))
        with ThreadPoolExecutor(8) as ex:
            list(ex.map(put, range(held)))
    log(f"[bench] tier filled in {time.time() - t0:.1f}s")
    devs = [place(wi) for _ in range(K)]   # one set of destination pools per bound request
    torch.cuda.synchronize()
    dsts_all = [group_dsts(d.block_tables, d.tensor_bases, d.valid, wi.pool_blocks) for d in devs]
    dsts = dsts_all[0]

    sessions = [RestoreSession(ctx) for _ in range(K)]
    sess = sessions[0]
    chunk_payload = sum(s.n_tensors * w.chunk_tokens * s.record_bytes for s in w.groups)

    log("[bench] measuring pinned H2D bandwidth (1 GiB, best of 10: copy engine on 1 and 2 streams, staging kernel)")
    h2d_sdma = max(bsr.bsr_measure_h2d(ctx, 1 << 30, 1, 10), bsr.bsr_measure_h2d(ctx, 1 << 30, 2, 10))
    h2d_kernel = bsr.bsr_measure_stage(ctx, 1 << 30, 10)
    h2d = max(h2d_sdma, h2d_kernel)
    copy_gbps = measure_d2d_copy(torch)

    def step(rid):
        if K > 1:
            return step_concurrent(rid)
        n, _, _ = bsr.bsr_probe(ctx, rid, wi.salt, wi.tokens)
        t_r = time.perf_counter()
        out = sess.restore(rid, n, dsts)
        t_c = time.perf_counter()
        bsr.bsr_request_end(ctx, rid)
        assert out.fallback == 0 and out.exposed_tokens == n * w.chunk_tokens, out
        return n, out, t_c - t_r

    def step_concurrent(rid0):
        """K requests of the same prompt, bound together, windows interleaved round-robin."""
        rids = [rid0 * 100 + k for k in range(K)]
        ns = [bsr.bsr_probe(ctx, r, wi.salt, wi.tokens)[0] for r in rids]
        t_r = time.perf_counter()
        torch.cuda.current_stream().synchronize()
        for r, n_k, se, d in zip(rids, ns, sessions, dsts_all):
            se.bind(r, n_k, d)
        left = list(rids)
        while left:  # one window of each request in turn, as the library plans them
            for r in list(left):
                first, cnt = bsr.bsr_next_window(ctx, r)
                if cnt == 0:
                    left.remove(r)
                else:
                    bsr.bsr_restore_window(ctx, r, first, cnt)
        outs_k = [se.commit(r) for r, se in zip(rids, sessions)]
        t_c = time.perf_counter()
        for r, o, n_k in zip(rids, outs_k, ns):
            bsr.bsr_request_end(ctx, r)
            assert o.fallback == 0 and o.exposed_tokens == n_k * w.chunk_tokens, o
        merged = outs_k[0]
        for key in ("n_install_launches", "install_ms_total", "installed_bytes"):
            merged.stats[key] = sum(o.stats[key] for o in outs_k)
        merged.stats["peak_live_staging_bytes"] = sum(o.stats["peak_live_staging_bytes"] for o in outs_k)
        return ns[0], merged, t_c - t_r

    for i in range(args.warmup):
        log(f"[bench] warmup step {i}")
        step(1000 + i)
    torch.cuda.synchronize()
    log(f"[bench] timing {args.steps} steps")
    outs = []
    step_s = []
    t_start = time.perf_counter()
    for i in range(args.steps):
        t_i = time.perf_counter()
        outs.append(step(2000 + i))
        step_s.append(time.perf_counter() - t_i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    log(f"[bench] timed {args.steps} steps in {elapsed:.3f}s")

    n = outs[0][0]
    restored = K * n * chunk_payload
    value = restored * args.steps / elapsed / 1e9
    restore_only = restored * args.steps / sum(o[2] for o in outs) / 1e9
    launches = sum(o[1].stats["n_install_launches"] for o in outs)
    kern_ms = sum(o[1].stats["install_ms_total"] for o in outs)
    installed = sum(o[1].stats["installed_bytes"] for o in outs)
    avg_launch_ms = kern_ms / launches
    bytes_per_launch = 2 * installed / launches        # read staged + write paged
    achieved = bytes_per_launch / (avg_launch_ms * 1e-3) / 1e9
    st = outs[-1][1].stats

    # The staging kernel's rate, from one more restore, untimed, with its
    # launches stamped as well: stamps on the copy stream lengthen the gaps
    # between consecutive copies, so the timed steps stamp the installs only.
    bsr.bsr_set_timing(ctx, bsr.BSR_FLAG_TIME_INSTALL | bsr.BSR_FLAG_TIME_STAGE)
    stage_st = step(2900)[1].stats
    bsr.bsr_set_timing(ctx, bsr.BSR_FLAG_TIME_INSTALL)
    stage_launches, stage_ms, stage_bytes = (stage_st["n_stage_launches"], stage_st["stage_ms_total"],
                                             stage_st["stage_bytes"])

    if args.calibrate_copy:
        a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()

    traffic, traffic_src, traffic_direct = recorded_traffic(w.name, st["install_batch"])

    sweep = None
    if args.concurrency_sweep and args.tier == "file":
        sweep = []
        for conc in [int(x) for x in args.concurrency_sweep.split(",")]:
            c2 = bsr.bsr_ctx_create(layout, W, hip_device=0, install_batch=args.install_batch)
            bsr.bsr_store_reserve(c2, stride)
            open_file_tier(bsr, c2, file_dir, conc, args.direct)   # re-indexes the same files
            s2 = RestoreSession(c2)
            times, outs2 = [], []
            for i in range(args.warmup + args.steps):
                n2, _, _ = bsr.bsr_probe(c2, 3000 + i, wi.salt, wi.tokens)
                t_a = time.perf_counter()
                o2 = s2.restore(3000 + i, n2, dsts)
                t_b = time.perf_counter()
                bsr.bsr_request_end(c2, 3000 + i)
                assert o2.fallback == 0 and o2.exposed_tokens == n2 * w.chunk_tokens
                if i >= args.warmup:
                    times.append(t_b - t_a)
                    outs2.append(o2)
            sweep.append({"load_concurrency": conc,
                          "gbps": round(n2 * chunk_payload * len(times) / sum(times) / 1e9, 3),
                          "ms_per_restore": round(sum(times) / len(times) * 1e3, 1),
                          "peak_live_staging_bytes": outs2[-1].stats["peak_live_staging_bytes"],
                          "host_bounce_bytes": outs2[-1].stats["host_bounce_bytes"],
                          "file_tier_chunks": outs2[-1].stats["file_tier_chunks"]})
            log(f"[bench] load concurrency {conc}: {sweep[-1]}")
            del s2
            bsr.bsr_ctx_destroy(c2)

    staging_measured = measure_staging(torch, bsr, ctx, sess, wi, dsts, 9000) if K == 1 else None

    ceiling = None
    if args.scatter_ceiling:
        # the install's data per full launch, copied as plain scattered blocks of each group's size
        data = st["install_batch"] * chunk_payload
        ceiling = {"data_bytes_per_launch": data,
                   "note": "bsr_measure_scatter: best of 5, read + write bytes; the source read cold, or rewritten "
                           "right before each launch as the staging copy writes a slot before the install"}
        for spec in w.groups:
            bb = spec.block_tokens * spec.record_bytes
            if bb % 16 == 0 and str(bb) not in ceiling:
                cold = bsr.bsr_measure_scatter(ctx, bb, data, 5, 1)
                warm = bsr.bsr_measure_scatter(ctx, bb, data, 5, 1, bsr.BSR_SCATTER_WARM_SOURCE)
                ceiling[str(bb)] = {"cold_source_gbps": round(cold, 1), "cold_source_frac": round(cold / HBM_PEAK_GBPS, 4),
                                    "warm_source_gbps": round(warm, 1), "warm_source_frac": round(warm / HBM_PEAK_GBPS, 4)}
                log(f"[bench] scatter ceiling, {bb} B blocks: {cold:.1f} GB/s cold source, {warm:.1f} warm")

    cpu = None
    if not args.no_cpu_baseline and W > 0 and K == 1:
        cpu = cpu_baseline(wi, W, args.cpu_seconds)

    line = {
        "metric": "restored KV GB/s per GPU (512K tokens, W=32) + peak staging bytes; % H2D/HBM roofline",
        "value": round(value, 3),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3),
        "ms_per_step_median": round(sorted(step_s)[len(step_s) // 2] * 1e3, 3),
        "value_at_median_step": round(restored / sorted(step_s)[len(step_s) // 2] / 1e9, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": {
            "workload": f"{w.name}: {w.n_tokens} tokens, {n} chunks of {w.chunk_tokens} tokens restored, "
                        f"{len(w.groups)} groups / {sum(s.n_tensors for s in w.groups)} tensors, W={W}, "
                        "pinned-host tier -> W-slot HBM ring -> paged pools"
                        + (f"; {K} requests bound together, windows interleaved" if K > 1 else ""),
            "tokens": w.n_tokens, "chunks_restored": n, "window_chunks": W,
            "chunk_bytes": slot, "restored_bytes_per_step": restored,
            "install_batch": st["install_batch"],
            "requests": K,
            "profiling_subset": bool(args.held_chunks),
        },
        "roofline": {
            "bound": "hbm", "kernel": "k_install",
            "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic, "traffic_source": traffic_src,
            "traffic_reads_counted_directly": traffic_direct,
            "traffic_note": "HBM bytes per average launch of a 2,048-chunk restore: FETCH_SIZE and WRITE_SIZE "
                            "scaled by a plain 1 GiB copy's readings; the other figure counts read requests "
                            "by size (32/64/128 B) instead of scaling FETCH_SIZE",
            "bytes_per_launch": int(bytes_per_launch), "avg_launch_us": round(avg_launch_ms * 1e3, 2),
            "launches_timed": launches,
        },
        "roofline_stage": None if not (stage_launches and stage_ms) else {
            "bound": "host link", "kernel": "k_stage",
            "achieved": round(stage_bytes / (stage_ms * 1e-3) / 1e9, 3), "peak": round(LINK_PEAK_GBPS, 3),
            "unit": "GB/s", "frac": round(stage_bytes / (stage_ms * 1e-3) / 1e9 / LINK_PEAK_GBPS, 4),
            "frac_of_measured_link": round(stage_bytes / (stage_ms * 1e-3) / 1e9 / h2d, 4),
            "bytes_per_launch": int(stage_bytes / stage_launches),
            "avg_launch_us": round(stage_ms / stage_launches * 1e3, 2), "launches_timed": stage_launches,
            "note": "bytes read over the host link (pinned host memory -> ring) per ms of the staging kernel, "
                    "HIP events on the copy stream over one untimed restore after the timed steps; "
                    "peak = PCIe Gen5 x16 per direction after encoding",
        },
        "scatter_ceiling": ceiling,
        "hbm_copy_context": {
            "achieved": round(copy_gbps, 1), "unit": "GB/s", "frac": round(copy_gbps / HBM_PEAK_GBPS, 4),
            "measured_as": "torch copy_ of 1 GiB device to device (read + write bytes), best of 5",
        },
        "probe": {
            "ms_median": round(sorted(o[1].stats["probe_ns"] for o in outs)[len(outs) // 2] / 1e6, 3),
            "chunks": n, "note": "chunk keys + tier lookups on the host, inside each timed step",
        },
        "host_link": {
            "achieved": round(value, 3), "peak_measured": round(h2d, 3), "unit": "GB/s",
            "frac": round(value / h2d, 4), "restore_only_gbps": round(restore_only, 3),
            "copy_engine_gbps": round(h2d_sdma, 3), "staging_kernel_gbps": round(h2d_kernel, 3),
            "staging_copies": args.copy_engine,
            "measured_as": "faster of: best of 10 hipMemcpyAsync of 1 GiB from hipHostMalloc memory on 1 and "
                           "2 streams; best of 10 staging-kernel copies of 1 GiB from hipHostMalloc memory",
        },
        "staging": {
            "peak_live_staging_bytes": st["peak_live_staging_bytes"],
            "measured": staging_measured,
            "law_W_times_chunk_bytes": K * (W or n) * slot,
            "mode": "bounded window" if W else "legacy whole-plan (W=0)",
            "aux_device_bytes": st["aux_device_bytes"],
        },
        "cpu_baseline": cpu,
    }
    if K > 1:
        adm = bsr.bsr_admission_get(ctx)
        line["admission"] = {"requests_bound_together": K, "staging_budget_bytes": adm["staging_budget_bytes"],
                             "peak_bound_staging_bytes": adm["peak_bound_staging_bytes"],
                             "peak_n_bound": adm["peak_n_bound"], "n_refused": adm["n_refused"],
                             "aux_device_bytes": adm["aux_device_bytes"],
                             "note": "value is the aggregate over the bound requests; staging.peak_live_"
                                     "staging_bytes sums their rings"}
    if args.tier == "file":
        line["file_tier"] = {"dir": file_dir, "direct": bool(args.direct),
                             "load_concurrency": args.load_concurrency,
                             "host_bounce_bytes": st["host_bounce_bytes"],
                             "file_tier_chunks": st["file_tier_chunks"],
                             "concurrency_sweep": sweep}
    print(json.dumps(line), flush=True)
    bsr.bsr_ctx_destroy(ctx)


def groups_alone(w, gs):
    """Workload w with only the groups gs, their tensor counts scaled by one
    factor so that a chunk holds about as many bytes as the whole layout's
    chunk: install launches of the same size as the layout's, built from
    those groups' blocks alone, in the same byte shares among themselves."""
    import dataclasses

    if not gs or len(set(gs)) != len(gs) or not all(0 <= g < len(w.groups) for g in gs):
        raise SystemExit(f"--only-group: distinct group indices in 0..{len(w.groups) - 1}")
    per_token = sum(s.n_tensors * s.record_bytes for s in w.groups)
    sub = sum(w.groups[g].n_tensors * w.groups[g].record_bytes for g in gs)
    specs = tuple(dataclasses.replace(w.groups[g], n_tensors=max(1, round(w.groups[g].n_tensors * per_token / sub)))
                  for g in sorted(gs))
    nt = max(s.n_tensors for s in specs)
    base = max(w.base_records or 0, nt * w.chunk_tokens + w.held_chunks)
    name = "+".join(s.name for s in specs)
    return dataclasses.replace(w, name=f"{w.name}-{name}-alone", groups=specs, base_records=base,
                               failure=None, failure_group=None)


def measure_staging(torch, bsr, ctx, sess, wi, dsts, rid):
    """Eq. 1 measured across one more restore of the same request, untimed,
    after the timed steps (so the runtime's own one-time set-up is done).

    The ring is dropped and allocated again by the bind, inside the measured
    region, after the pools and the status block: torch's peak allocated
    bytes then grow by the ring alone if the restore adds no other device
    memory, and the device's free bytes (hipMemGetInfo) stay the same from
    bind to commit."""
    sess.release_ring()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_allocated()
    base_req = torch.cuda.memory_stats()["requested_bytes.all.current"]
    n, _, _ = bsr.bsr_probe(ctx, rid, wi.salt, wi.tokens)
    m = {}
    out = sess.restore(rid, n, dsts, after_bind=lambda: m.setdefault("free", torch.cuda.mem_get_info()[0]))
    free_commit = torch.cuda.mem_get_info()[0]
    bsr.bsr_request_end(ctx, rid)
    assert out.fallback == 0
    return {"peak_requested_growth_bytes": int(torch.cuda.memory_stats()["requested_bytes.all.peak"] - base_req),
            "peak_alloc_growth_bytes": int(torch.cuda.max_memory_allocated() - base),
            "device_free_bytes_change_bind_to_commit": int(m["free"] - free_commit),
            "measured_as": "one untimed restore after the timed steps: growth of torch's peak requested "
                           "bytes (and of its allocated bytes, which round a ring up to its 2 MiB segment "
                           "when the remainder is at most 1 MiB) from before the ring, allocated by its bind, "
                           "to after its commit; and the change of hipMemGetInfo free bytes from its bind to "
                           "its commit"}


def measure_d2d_copy(torch):
    """A plain device-to-device copy as context for the install kernel's HBM rate."""
    a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best = 0.0
    for _ in range(6):
        e0.record()
        b.copy_(a)
        e1.record()
        e1.synchronize()
        best = max(best, 2 * a.numel() / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del a, b
    return best


def host_cpu():
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return f"{model}, {os.cpu_count()} logical CPUs visible"


def open_file_tier(bsr, ctx, directory, concurrency, direct):
    bsr.bsr_file_tier_open(ctx, directory, concurrency, 0, bsr.BSR_FILE_DIRECT if direct else 0)


def kernel_code_sha256(lib_path=None):
    """SHA-256 of the gfx950 code object inside libbsr.so: the kernels as
    built.  Counters recorded against it hold exactly as long as the machine
    code does; documentation or host-side edits leave it unchanged.  The
    library is a clang offload bundle ("__CLANG_OFFLOAD_BUNDLE__", entry count,
    then offset / size / triple per entry).  None if it cannot be read."""
    import hashlib
    import struct

    path = lib_path or os.path.join(ROOT, "paper_2608_17826_amd", "libbsr.so")
    try:
        with open(path, "rb") as fh:
            data = fh.read()
    except OSError:
        return None
    i = data.find(b"__CLANG_OFFLOAD_BUNDLE__")
    if i < 0:
        return None
    (n,) = struct.unpack_from("<Q", data, i + 24)
    p = i + 32
    for _ in range(n):
        off, size, tlen = struct.unpack_from("<QQQ", data, p)
        p += 24
        triple = data[p:p + tlen].decode(errors="replace")
        p += tlen
        if triple.endswith("gfx950"):
            return hashlib.sha256(data[i + off:i + off + size]).hexdigest()
    return None


def recorded_traffic(workload_name, install_batch):
    """HBM bytes per k_install launch from the committed rocprofv3 counter
    summary, only if it was taken on the kernel code built here."""
    import glob
    import re

    sha = kernel_code_sha256()
    for path in glob.glob(os.path.join(ROOT, "profiles", "*.md")):
        for m in re.finditer(r"<!-- traffic-record ([^>]*) -->", open(path).read()):
            kv = dict(x.split("=", 1) for x in m.group(1).split())
            if (kv.get("kernel") == "k_install" and kv.get("workload") == workload_name
                    and int(kv.get("install_batch", -1)) == install_batch
                    and sha is not None and kv.get("kernel_code_sha256") == sha):
                return (int(kv["traffic_bytes_per_launch"]), os.path.relpath(path, ROOT),
                        int(kv["traffic_bytes_per_launch_reads_direct"])
                        if "traffic_bytes_per_launch_reads_direct" in kv else None)
    return None, None, None


def cpu_baseline(wi, W, target_s):
    """The oracle, on one CPU, on the first windows of the same workload.

    The calling thread is pinned to a single CPU while the oracle runs (its
    numpy work is elementwise and runs on that thread).  The sample restores
    whole windows (W chunks each) until about target_s seconds of oracle
    work; destination pools are compacted to the blocks the sample touches
    (block ids renumbered), which changes no arithmetic.
    """
    prev = os.sched_getaffinity(0)
    cpu = min(prev)
    os.sched_setaffinity(0, {cpu})
    try:
        out = _cpu_baseline_pinned(wi, W, target_s)
    finally:
        os.sched_setaffinity(0, prev)
    out["pinned_cpu"] = cpu
    return out


def _cpu_baseline_pinned(wi, W, target_s):
    import numpy as np

    import oracle

    w = wi.workload
    layout = oracle.OracleLayout.from_specs(w.chunk_tokens, w.groups)
    t0 = time.perf_counter()
    keys = oracle.chain_keys(wi.tokens, w.chunk_tokens, wi.salt)
    t_keys = time.perf_counter() - t0
    done, t_restore, windows = 0, 0.0, 0
    while t_restore < target_s and done < w.held_chunks:
        k = min(W, w.held_chunks - done)
        # a store holding this window's chunks, and compact pools
        store = oracle.OracleStore(layout.n_groups)
        for i in range(done, done + k):
            store.put_chunk(keys[i], wi.payloads(i))
        bts, pools, valid = [], [], []
        for g, spec in enumerate(w.groups):
            lo = done * w.chunk_tokens // spec.block_tokens
            hi = -(-((done + k) * w.chunk_tokens) // spec.block_tokens)
            bt = np.full(hi, -1, dtype=np.int64)
            bt[lo:hi] = np.arange(hi - lo)
            bts.append(bt)
            pools.append(np.zeros((spec.n_tensors, hi - lo, layout.block_bytes(g)), np.uint8))
            valid.append(np.zeros(hi - lo, np.uint8))
        sub_keys = [None] * done + keys[done:done + k]
        t1 = time.perf_counter()
        res = _restore_range(layout, store, sub_keys, done, k, W, bts, pools, valid)
        t_restore += time.perf_counter() - t1
        assert res.fail_reason == 0
        done += k
        windows += 1
    restored = done * layout.chunk_payload_bytes
    probe_share = t_keys * done / max(1, len(keys))
    return {"value": round(restored / (t_restore + probe_share) / 1e9, 4), "unit": "GB/s", "cores": 1,
            "kind": "oracle", "host": host_cpu(),
            "sample": f"first {done} of {w.held_chunks} chunks ({windows} windows of W={W}); "
                      f"{restored} bytes in {t_restore:.1f}s + pro-rated probe {probe_share:.2f}s"}


def _restore_range(layout, store, keys, first, k, W, bts, pools, valid):
    """Oracle windowed restore of chunks [first, first + k) (one window)."""
    import oracle

    # the oracle restores a prefix from chunk 0; shift the plan so the sample
    # window is its only window
    shifted_keys = keys[first:first + k]
    shifted_bts = []
    C = layout.chunk_tokens
    for g, gr in enumerate(layout.groups):
        lo_tok = first * C
        if lo_tok % gr.block_tokens == 0:
            shifted_bts.append(bts[g][lo_tok // gr.block_tokens:])
        else:
            raise ValueError("sample windows must start on a block boundary")
    return oracle.windowed_restore(layout, store, shifted_keys, k, W, shifted_bts, pools, valid)


if __name__ == "__main__":
    main()
