"""Benchmark: one verification round per step on one MI355X.

A step is the whole hot path on one batch: the KV-state preparation of the
arriving requests' blocks fused with verification attention (one pass that
reads each staged byte once), then spec_accept.  --unfused runs kv_gather and
verify_attention as two kernels instead.  Inputs (synthetic, seeded) are
resident in HBM before timing starts.  Prints ONE JSON line.

    python bench.py [--steps K] [--warmup W] [--workload verify_8b] [--unfused]
                    [--no-cpu-baseline]
    python bench.py --draft [--draft-steps 4] [--draft-vocab 151936]   (draft stage)
    python bench.py --h2d                                              (host-arena preparation)
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E peak, GB/s


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None,
                    help="verify_8b (default), or draft_decode with --draft")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--unfused", action="store_true",
                    help="kv_gather and verify_attention as separate kernels")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--ceiling", action="store_true",
                    help="only the HBM probe: one layer's fused-pass read/write mix on the workload "
                         "(verify_8b unless --workload names another), with "
                         "the written tiles placed four ways (gathered at the end of every "
                         "wave's sequence, spread through it, on a share of the waves, or "
                         "stored by waves that do not read), and the writes alone")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the practical-ceiling probe of the dominant kernel's access pattern")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device copy three times (counter calibration)")
    ap.add_argument("--h2d", action="store_true",
                    help="measure the preparation from a pinned host arena instead: H2D rate, "
                         "interference with the round (Eq. D.1) and exposed KV-ready wait of "
                         "double-banked rounds (Eq. G.1)")
    ap.add_argument("--draft", action="store_true",
                    help="time the draft stage instead (Eq. 1): --draft-steps single-query "
                         "decode steps (append, attention, sampling) on draft_decode")
    ap.add_argument("--phi", action="store_true",
                    help="profile the stage-time tables the scheduler uses (phi_s of Eq. 4): "
                         "one target round layer (fused pass + acceptance) and one 4-step draft "
                         "stage layer over a range of batch sizes; prints one JSON line")
    ap.add_argument("--schedule", action="store_true",
                    help="host-side scheduler (no GPU): batch-reconstruction decision latency "
                         "and a pool-scale simulation, the library against the oracle")
    ap.add_argument("--sweep", action="store_true",
                    help="every named round workload (tiny, draft_decode, verify_8b, knee, "
                         "full_depth streamed layer by layer), one JSON line each, each with "
                         "an oracle sample of --cpu-seconds")
    ap.add_argument("--draft-steps", type=int, default=4)
    ap.add_argument("--draft-vocab", type=int, default=151936)
    args = ap.parse_args()
    if args.workload is None:
        args.workload = "draft_decode" if args.draft else "verify_8b"
    return args


KERNEL_SRC = os.path.join(ROOT, "paper_2609_29364_amd", "csrc", "verify_attention.hip")


def measured_traffic(kernel):
    """HBM bytes per call of `kernel` from the committed counter runs, or None
    when the kernel source has changed since those counters were taken."""
    import hashlib
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", f"{kernel}_traffic.json")))
        digest = hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()
    except (OSError, ValueError):
        return None
    if rec.get("kernel_sha256") != digest:
        return None
    return rec.get("bytes_per_call")


def calibrate_copy():
    import torch
    n = 1 << 30
    a = torch.ones(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "device copy", "bytes_read": n, "bytes_written": n,
                      "dispatches": 3}), flush=True)


def describe(cfg):
    return {"workload": cfg.name, "bs": cfg.bs, "layers": cfg.num_layers,
            "q_heads": cfg.num_q_heads, "kv_heads": cfg.num_kv_heads, "head_dim": cfg.head_dim,
            "context": [cfg.ctx_lo, cfg.ctx_hi], "draft_len": [cfg.k_lo, cfg.k_hi],
            "arriving": cfg.n_arriving, "vocab": cfg.vocab, "block_size": cfg.block_size,
            "seed": cfg.seed}


def algorithmic_bytes(cfg, meta, acc_len=None):
    """Bytes each kernel must move at minimum (read + write), per step.

    gather: every staged block read and written (both planes).  attention:
    every visible K/V token of every request read once, Q read, O written.
    fused: the staged blocks read once and written once, the resident
    requests' tokens read once, Q read, O written.  accept: the target and
    draft rows acceptance reads (two rows at a rejection, the bonus row
    otherwise), the uniforms, tokens and outputs."""
    hkv, d, hq = cfg.num_kv_heads, cfg.head_dim, cfg.num_q_heads
    block_bytes = hkv * 16 * d * 2          # one plane of one block
    token_bytes = 2 * hkv * d * 2           # K and V of one token, all KV heads
    qo = 2 * meta.total_q * hq * d * 2
    staged = 2 * meta.n_pairs * block_bytes  # both planes
    gather = 2 * staged
    kv_tokens = int(meta.seq_lens.astype(np.int64).sum())
    resident_tokens = int(meta.seq_lens[~meta.arriving].astype(np.int64).sum())
    attn = kv_tokens * token_bytes + qo
    fused = resident_tokens * token_bytes + 2 * staged + qo
    accept = 0
    if cfg.vocab and acc_len is not None:
        rows = np.where(acc_len < meta.depth, 2, 1).sum()
        accept = int(rows) * cfg.vocab * 4 + meta.total_q * 4 * 3
    L = cfg.num_layers
    return {"gather": L * gather, "attention": L * attn, "fused": L * fused, "accept": accept}


def practical_ceiling(dev, read_bytes, write_bytes, reps=7, placement="end"):
    """What the memory system gives the attention pass's access pattern, measured
    by a kernel that only moves the same bytes (libnsd_probe.so): 4 KiB tiles at
    random positions, one persistent wave per SIMD with up to 32 KiB in flight,
    and (for the fused pass) the written share of the tiles stored back to
    random positions right after they are read.  Returns the read-only rate and
    the rate of the given read/write mix, in GB/s of bytes moved.

    placement of the written tiles (same bytes): "end" the last share of every
    wave's sequence (the fused pass's order); "spread" runs of 40 steps (one
    request's item) scattered through every wave's sequence; "waves" every tile
    of a share of the waves, the others only reading; "writer" the same number
    of tiles stored by a fifth wave per workgroup that does not read (the four
    readers only read), which also reports the writes alone."""
    import ctypes
    import torch
    from paper_2609_29364_amd.build import PROBE_LIB_PATH
    lib = ctypes.CDLL(PROBE_LIB_PATH)
    lib.nsd_probe_tiles.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                    ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                    ctypes.c_void_p]
    lib.nsd_probe_tiles_writer.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                           ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_void_p, ctypes.c_void_p]
    tile = 4096
    waves = 4 * torch.cuda.get_device_properties(dev).multi_processor_count
    steps = max(2, int(read_bytes / (waves * 4 * tile)))
    n = waves * steps * 4
    src_tiles = 2 * n
    rng = np.random.default_rng(0)
    src = torch.zeros(src_tiles * tile, dtype=torch.uint8, device=dev)
    dst = torch.zeros(n * tile, dtype=torch.uint8, device=dev)
    sink = torch.zeros(waves * 1024, dtype=torch.uint8, device=dev)
    ids = torch.as_tensor(rng.permutation(src_tiles)[:n].astype(np.int32), device=dev)
    # the fused pass gives every wave its share of the arriving requests after its
    # share of the resident ones: the written tiles are the last ones of every
    # wave's sequence
    frac = write_bytes / read_bytes if read_bytes else 0.0
    step_in_wave = (np.arange(n) // 4) % steps
    if placement in ("end", "writer"):
        written = step_in_wave >= steps - int(round(frac * steps))
    elif placement == "spread":
        written = ((np.arange(n) // 4 // 40) * 7919 % 1000) < frac * 1000
    elif placement == "waves":
        written = ((np.arange(n) // (4 * steps)) * 7919 % 1000) < frac * 1000
    else:
        raise ValueError(placement)
    dids = np.where(written, rng.permutation(n), -1).astype(np.int32)
    dids_d = torch.as_tensor(dids, device=dev)
    # "writer": the written tiles' destinations dealt to the workgroups' writer
    # waves in turn, -1 padding
    wgs = waves // 4
    wdst = dids[dids >= 0]
    write_per = max(1, -(-len(wdst) // wgs))
    wl = np.full(wgs * write_per, -1, np.int32)
    wl[:len(wdst)] = wdst
    wl_d = torch.as_tensor(wl.reshape(write_per, wgs).T.copy().reshape(-1), device=dev)
    stream = torch.cuda.current_stream(dev)
    sp = ctypes.c_void_p(stream.cuda_stream)

    def run(kind):
        if placement == "writer" and kind != "read":
            st = lib.nsd_probe_tiles_writer(src.data_ptr(), src_tiles, dst.data_ptr(), n,
                                            ids.data_ptr(), wl_d.data_ptr(), write_per, waves,
                                            0 if kind == "write" else steps, sink.data_ptr(), sp)
        else:
            st = lib.nsd_probe_tiles(src.data_ptr(), src_tiles, dst.data_ptr(), n,
                                     ids.data_ptr(), dids_d.data_ptr() if kind == "mix" else None,
                                     waves, steps, sink.data_ptr(), sp)
        if st != 0:
            raise RuntimeError(f"probe status {st}")

    out = {}
    kinds = [("read_only_gbs", "read"), ("mix_gbs", "mix")]
    if placement == "writer":
        kinds.append(("write_only_gbs", "write"))
    for key, kind in kinds:
        if kind != "read" and not write_bytes:
            out[key] = out["read_only_gbs"]
            continue
        run(kind)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        ev[0].record(stream)
        for k in range(reps):
            run(kind)
            ev[k + 1].record(stream)
        torch.cuda.synchronize()
        ms = float(np.median([ev[k].elapsed_time(ev[k + 1]) for k in range(reps)]))
        moved = (n * tile if kind != "write" else 0) + \
            (int(written.sum()) * tile if kind != "read" else 0)
        out[key] = round(moved / (ms * 1e-3) / 1e9, 1)
    out["write_share"] = round(float(written.mean()), 4)
    where = {"end": f"the last {written.mean():.1%} of every wave's tiles",
             "spread": f"{written.mean():.1%} of the tiles, in runs of 40 steps through every "
                       f"wave's sequence",
             "waves": f"every tile of {written.mean():.1%} of the waves",
             "writer": f"{written.mean():.1%} of the tiles, by a fifth wave per workgroup "
                       f"that does not read"}[placement]
    out["pattern"] = (f"random 4 KiB tiles, {waves} persistent waves, up to 32 KiB in flight "
                      f"per wave, {n * tile / 1e9:.2f} GB read"
                      + (f", {where} written back" if write_bytes else ""))
    del src, dst, sink, ids, dids_d, wl_d
    torch.cuda.empty_cache()
    return out


def host_facts():
    """The host the oracle runs on: usable cores, CPU model, BLAS pool size."""
    try:
        cores = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        cores = os.cpu_count() or 1
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas = 1
    return {"host_cores": cores, "cpu_model": model, "blas_threads": int(blas),
            "nproc": os.cpu_count()}


def cpu_baseline(cfg, meta, layer, acc_in, budget_s, threads=None):
    """The CPU oracle, untuned, on a bounded sample of the same round.

    threads: None runs with the BLAS pool the host provides; an integer limits
    it (threadpoolctl) for the duration of the sample."""
    import contextlib
    facts = host_facts()
    limit = contextlib.nullcontext()
    if threads is not None:
        from threadpoolctl import threadpool_limits
        limit = threadpool_limits(limits=int(threads))
    with limit:
        return _cpu_baseline(cfg, meta, layer, acc_in, budget_s, facts,
                             facts["blas_threads"] if threads is None else int(threads))


def _cpu_baseline(cfg, meta, layer, acc_in, budget_s, facts, threads):
    import oracle
    from workload.synth import logical_kv
    rng = np.random.default_rng(0)
    order = rng.permutation(cfg.bs)
    p = acc_in.p_target if acc_in is not None else None
    done, t_total, t_layer, t_acc = 0, 0.0, 0.0, 0.0
    u16 = lambda t: t.view(__import__("torch").int16).cpu().numpy()
    # passes over the round's requests (host copies not timed) until the time
    # budget is spent
    for r in (r for _ in range(1000) for r in order):
        if t_total >= budget_s and done >= 2:
            break
        # host copies of this request's inputs (not timed)
        nb = meta.nblk(r)
        k, v = logical_kv(meta, layer, r)
        k64, v64 = k.cpu().double().numpy(), v.cpu().double().numpy()
        a, b = int(meta.q_indptr[r]), int(meta.q_indptr[r + 1])
        q64 = layer.q[a:b].cpu().double().numpy()
        if meta.arriving[r]:
            ids = meta.stage_table[r, :nb]
            sk, sv = u16(layer.k_stage[ids])[None], u16(layer.v_stage[ids])[None]
            dk = np.zeros_like(sk)
            dv = np.zeros_like(sv)
        if acc_in is not None:
            kk = b - a - 1
            pr = acc_in.p_target[a:b].cpu().numpy()
            qr = acc_in.q_draft[a - r:a - r + kk].cpu().numpy()
            xr = acc_in.draft_tokens[a - r:a - r + kk].cpu().numpy()
            ur = acc_in.uniforms[a:b].cpu().numpy()
        t0 = time.perf_counter()
        if meta.arriving[r]:
            oracle.gather.kv_gather(sk, sv, dk, dv, np.arange(nb), np.arange(nb))
        oracle.attention.verify_attention_request(q64, k64, v64, 1.0 / np.sqrt(cfg.head_dim))
        t1 = time.perf_counter()
        if acc_in is not None:
            oracle.accept.accept_request(pr, qr, xr, ur)
        t2 = time.perf_counter()
        t_layer += t1 - t0
        t_acc += t2 - t1
        t_total += t2 - t0
        done += 1
    # a round of several layers repeats the per-layer work (layer 0's sample
    # stands for every layer) and accepts once
    per_req = (t_layer * cfg.num_layers + t_acc) / done
    return {"value": round(1.0 / per_req, 3), "unit": "requests/s", "cores": int(threads),
            "kind": "oracle", "host_cores": facts["host_cores"], "cpu_model": facts["cpu_model"],
            "threads_note": "cores = the BLAS threads the fp64 numpy oracle may use; the "
                            "oracle's own loops run on one Python thread",
            "sample": (f"{done} of {cfg.bs} requests" if done <= cfg.bs else
                       f"{done} requests ({done / cfg.bs:.1f} passes over the {cfg.bs})")
                      + f" of the {cfg.name} round (gather of their "
                      f"blocks if arriving, attention over all heads/queries, acceptance), "
                      f"{t_total:.1f} s of fp64 numpy"
                      + (f"; layer 0 timed, counted for all {cfg.num_layers} layers"
                         if cfg.num_layers > 1 else "")}


def h2d_bench(args):
    """Preparation from HostKV: one JSON line (not the headline metric).

    * h2d: the round's arriving KV copied from the pinned arena into a bank alone.
    * interference (Eq. D.1): mean round time (fused pass + acceptance) while the next
      round's H2D runs on the copy stream, against the same rounds with no copy.
    * pipeline (Eq. G.1): double-banked rounds, each needing its own H2D of the first n
      arriving requests' blocks; inputs ready at t = 0, the worker ready when the
      previous round ends, KV ready when its H2D ends; exposed wait = [KV ready -
      max(input ready, worker ready)]+ per round, and rounds/s."""
    import torch
    import paper_2609_29364_amd as nsd
    from paper_2609_29364_amd.hostkv import DoubleBank, h2d_plan
    from workload import CONFIGS, make_meta, make_layer, make_accept, make_hostkv

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = CONFIGS[args.workload]
    meta = make_meta(cfg)
    layer = make_layer(cfg, meta, 0, dev)
    acc_in = make_accept(cfg, meta, dev)
    host = make_hostkv(cfg, meta, layer)
    i32 = lambda a: torch.as_tensor(np.ascontiguousarray(a), dtype=torch.int32, device=dev)
    bt, st, sl, qi = (i32(meta.block_table), i32(meta.stage_table), i32(meta.seq_lens),
                      i32(meta.q_indptr))
    bb = layer.k_stage[0].numel() * 2
    plan_all = h2d_plan(host.extent, meta.stage_table, meta.arriving, meta.seq_lens, bb)
    bank = DoubleBank(layer.k_stage.shape, layer.v_stage.shape, dev)
    del layer.k_stage, layer.v_stage
    out = torch.empty_like(layer.q)
    ws = nsd.new_workspace(nsd.verify_attention_workspace_size(
        cfg.bs, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, meta.max_q, meta.max_seq_len), dev)
    acc_len = torch.empty(cfg.bs, dtype=torch.int32, device=dev)
    toks = torch.empty(meta.total_q, dtype=torch.int32, device=dev)
    acc_ws = torch.empty(max(1, nsd.accept_workspace_size(cfg.bs, max(cfg.vocab, 4))),
                         dtype=torch.uint8, device=dev)
    comp = torch.cuda.current_stream(dev)

    def round_(i):
        ks, vs = bank.bank(i)
        nsd.gather_verify_attention(layer.q, layer.k_pool, layer.v_pool, ks, vs, bt, st, sl, qi,
                                    meta.max_q, meta.max_seq_len, out=out, workspace=ws)
        if acc_in is not None:
            nsd.spec_accept(acc_in.p_target, acc_in.q_draft, acc_in.draft_tokens,
                            acc_in.uniforms, qi, cfg.k_hi, accepted_len=acc_len, out_tokens=toks,
                            workspace=acc_ws)

    ev = lambda: torch.cuda.Event(enable_timing=True)
    # H2D alone (both banks filled, so every round below reads valid staging)
    for i in range(2):
        bank.prepare(i, host.k, host.v, plan_all, plan_all)
    torch.cuda.synchronize()
    h2d_bytes = 2 * int(plan_all[:, 2].sum())
    t = []
    for _ in range(3):
        s0 = ev(); s0.record(bank.copy_stream)
        e1 = bank.prepare(0, host.k, host.v, plan_all, plan_all)
        torch.cuda.synchronize()
        t.append(s0.elapsed_time(e1))
    h2d_ms = float(np.median(t))

    # interference (Eq. D.1): rounds on bank 0 with and without bank 1 being filled
    def timed_rounds(n):
        e = [ev() for _ in range(n + 1)]
        e[0].record(comp)
        for k in range(n):
            round_(0)
            e[k + 1].record(comp)
        return e
    for _ in range(args.warmup):
        round_(0)
    torch.cuda.synchronize()
    eb = timed_rounds(args.steps)
    torch.cuda.synchronize()
    t_base = eb[0].elapsed_time(eb[-1]) / args.steps
    n_ov = max(4, int(h2d_ms / t_base * 0.8))     # rounds that fit inside one H2D
    s0 = ev(); s0.record(bank.copy_stream)
    e_h2d = bank.prepare(1, host.k, host.v, plan_all, plan_all)
    eo = timed_rounds(n_ov)
    torch.cuda.synchronize()
    # count only the rounds that ended before the copy did
    ends = [s0.elapsed_time(x) for x in eo]
    h_end = s0.elapsed_time(e_h2d)
    inside = [k for k in range(n_ov) if ends[k + 1] <= h_end]
    t_overlap = (float(np.mean([ends[k + 1] - ends[k] for k in inside])) if inside else None)

    # pipeline (Eq. G.1) for a few arrival volumes per round
    order = [r for r in range(meta.bs) if meta.arriving[r]]
    pipeline = []
    for n_arr in sorted({1, 4, 16, len(order)}):
        keep = np.zeros(meta.bs, dtype=bool)
        keep[order[:n_arr]] = True
        plan = h2d_plan(host.extent, meta.stage_table, keep, meta.seq_lens, bb)
        rounds = 12
        torch.cuda.synchronize()
        t0 = ev(); t0.record(comp)
        bank.copy_stream.wait_event(t0)
        h_ev, r_ev = [], []
        bank.prepare(0, host.k, host.v, plan, plan)
        h_ev.append(bank.ready(0))
        for i in range(rounds):
            if i + 1 < rounds:
                bank.prepare(i + 1, host.k, host.v, plan, plan)
                h_ev.append(bank.ready(i + 1))
            comp.wait_event(bank.ready(i))
            round_(i)
            bank.done(i, comp)
            e = ev(); e.record(comp); r_ev.append(e)
        torch.cuda.synchronize()
        H = [t0.elapsed_time(x) for x in h_ev]
        R = [t0.elapsed_time(x) for x in r_ev]
        W = [0.0] + R[:-1]
        E = [max(0.0, H[i] - W[i]) for i in range(rounds)]
        pipeline.append({"arriving_per_round": n_arr, "h2d_mb": round(2 * int(plan[:, 2].sum()) / 2**20, 2),
                         "exposed_wait_ms_mean": round(float(np.mean(E[1:])), 4),
                         "rounds_per_s": round((rounds - 1) / ((R[-1] - R[0]) * 1e-3), 1)})
    # closing the round: window append, committed lengths, suffix writeback to the arena
    kn = torch.randn((meta.total_q, cfg.num_kv_heads, cfg.head_dim), device=dev).to(torch.bfloat16)
    vn = torch.randn_like(kn)
    round_(0)
    new_len = nsd.commit_lengths(sl, qi, acc_len) if acc_in is not None else sl.clone()
    torch.cuda.synchronize()
    nl = new_len.cpu().numpy()
    host_len = meta.seq_lens - np.diff(meta.q_indptr)        # the window is new this round
    from paper_2609_29364_amd.hostkv import writeback_pairs
    wsrc, wdst = writeback_pairs(meta.block_table, host.extent, host_len, nl)
    wsrc_d, wdst_d = i32(wsrc), i32(wdst)
    close = {}
    for name, fn in (("append", lambda: nsd.kv_append(layer.k_pool, layer.v_pool, kn, vn, bt, sl, qi)),
                     ("commit", lambda: nsd.commit_lengths(sl, qi, acc_len, out=new_len)),
                     ("writeback", lambda: nsd.kv_writeback(layer.k_pool, layer.v_pool, host.k,
                                                            host.v, wsrc_d, wdst_d))):
        fn(); torch.cuda.synchronize()
        a, b = ev(), ev()
        a.record(comp)
        for _ in range(10):
            fn()
        b.record(comp)
        torch.cuda.synchronize()
        close[name + "_ms"] = round(a.elapsed_time(b) / 10, 4)
    wb_bytes = 2 * len(wsrc) * bb
    close["writeback_bytes"] = wb_bytes
    close["writeback_gbs"] = round(wb_bytes / (close["writeback_ms"] * 1e-3) / 1e9, 2)
    close["append_bytes"] = 2 * kn.numel() * 2
    res = {"mode": "h2d", "workload": cfg.name, "arriving": int(meta.arriving.sum()),
           "h2d": {"bytes": h2d_bytes, "ms": round(h2d_ms, 3),
                   "gbs": round(h2d_bytes / (h2d_ms * 1e-3) / 1e9, 2),
                   "chunk_bytes": nsd.DEFAULT_CHUNK, "copies_in_plan": int(len(plan_all))},
           "interference": {"t_base_ms": round(t_base, 4),
                            "t_overlap_ms": None if t_overlap is None else round(t_overlap, 4),
                            "rounds_inside_copy": len(inside),
                            "delta_t": None if t_overlap is None else round((t_overlap - t_base) / t_base, 4)},
           "pipeline": pipeline, "close": close,
           "bounded_submission": bounded_submission(args, nsd, torch, meta, layer, host, bank, bb,
                                                    plan_all, round_, comp, bt, sl, qi, acc_len,
                                                    wsrc, wdst)}
    print(json.dumps(res), flush=True)


def bounded_submission(args, nsd, torch, meta, layer, host, bank, bb, plan_all, round_, comp,
                       bt, sl, qi, acc_len, wsrc, wdst):
    """Bounded H2D submission (Appendix E.5) and the export step of the bank
    lifecycle (Eq. E.2/E.3), measured on one GPU.

    * head-of-line: while the whole arriving KV of a round (both planes) is
      restored into one bank by H2D copies -- all 32 MiB chunks queued at
      once, or submitted by a DMA thread that keeps at most a 32 or 64 MiB
      window in flight -- the other bank's writeback (the round's committed
      suffix, by SDMA D2H copies into the pinned arena) is submitted 1 ms later
      on its own stream: its latency from submission to completion, against the
      same writeback alone.
    * rounds with exports: double-banked rounds where round k+1's H2D and round
      k's export both overlap computation (Compute_k || H2D_k+1, Compute_k+1 ||
      D2H_k), with and without the window: rounds/s, exposed KV-ready wait
      (Eq. G.1) and the round time against rounds with no transfer (Eq. D.1)."""
    import threading
    ev = lambda: torch.cuda.Event(enable_timing=True)
    d2h = bank.d2h_stream
    block = bb
    # the writeback as SDMA copies: pool block -> arena block, both planes
    wb_k = np.stack([wsrc.astype(np.int64) * block, wdst.astype(np.int64) * block,
                     np.full(len(wsrc), block, np.int64)], axis=1)

    def writeback_sdma(stream):
        nsd.copy_plan(layer.k_pool, host.k, wb_k, stream=stream)
        nsd.copy_plan(layer.v_pool, host.v, wb_k, stream=stream)

    wsrc_d = torch.as_tensor(wsrc, dtype=torch.int32, device=comp.device)
    wdst_d = torch.as_tensor(wdst, dtype=torch.int32, device=comp.device)

    def writeback_kernel(stream):
        nsd.kv_writeback(layer.k_pool, layer.v_pool, host.k, host.v, wsrc_d, wdst_d)

    def wb_latency_ms():
        t0 = time.perf_counter()
        writeback_sdma(d2h)
        e = ev(); e.record(d2h)
        e.synchronize()
        return (time.perf_counter() - t0) * 1e3

    torch.cuda.synchronize()
    alone = float(np.median([wb_latency_ms() for _ in range(5)]))
    hol = {"writeback_bytes": 2 * int(wb_k[:, 2].sum()), "writeback_alone_ms": round(alone, 3)}
    windows = (("all_queued", None), ("window_32MiB", nsd.DEFAULT_CHUNK),
               ("window_64MiB", 2 * nsd.DEFAULT_CHUNK))
    for name, window in windows:
        lat, h2d_ms = [], []
        for _ in range(3):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            bank.prepare(1, host.k, host.v, plan_all, plan_all, window_bytes=window)
            time.sleep(1e-3)
            lat.append(wb_latency_ms())
            e = bank.ready(1)
            e.synchronize()
            h2d_ms.append((time.perf_counter() - t0) * 1e3)
        hol[name] = {"writeback_ms": round(float(np.median(lat)), 3),
                     "h2d_ms": round(float(np.median(h2d_ms)), 3)}

    # double-banked rounds with the export of each round's suffix
    def run_rounds(n, window, export):
        torch.cuda.synchronize()
        t0 = ev(); t0.record(comp)
        bank.copy_stream.wait_event(t0)
        h_ev, r_ev = [], []
        bank.prepare(0, host.k, host.v, plan_all, plan_all, window_bytes=window)
        for i in range(n):
            if i + 1 < n:
                bank.prepare(i + 1, host.k, host.v, plan_all, plan_all, window_bytes=window)
            bank.computing(i, comp)
            h_ev.append(bank.ready(i))
            round_(i)
            e = ev(); e.record(comp); r_ev.append(e)
            if export:
                bank.export(i, comp, export)
            else:
                bank.done(i, comp)
        torch.cuda.synchronize()
        H = [t0.elapsed_time(x) for x in h_ev]
        R = [t0.elapsed_time(x) for x in r_ev]
        W = [0.0] + R[:-1]
        E = [max(0.0, H[i] - W[i]) for i in range(n)]
        return {"rounds_per_s": round((n - 1) / ((R[-1] - R[0]) * 1e-3), 1),
                "exposed_wait_ms_mean": round(float(np.mean(E[1:])), 4)}

    rounds = {"export": "the round's committed suffix written back into the pinned arena by "
                        "the gather kernel through the arena's device alias, on the D2H stream"}
    for name, window in windows:
        rounds[name] = run_rounds(8, window, writeback_kernel)
    rounds["all_queued_no_export"] = run_rounds(8, None, None)

    # Eq. D.1 for the round while both an H2D and an export run: the export by
    # SDMA copies, or by the writeback kernel (which takes compute units)
    def timed(n):
        e = [ev() for _ in range(n + 1)]
        e[0].record(comp)
        for k in range(n):
            round_(0)
            e[k + 1].record(comp)
        return e
    torch.cuda.synchronize()
    eb = timed(args.steps)
    torch.cuda.synchronize()
    t_base = eb[0].elapsed_time(eb[-1]) / args.steps
    interference = {"t_base_ms": round(t_base, 4)}
    for kind, fn in (("sdma_export", writeback_sdma), ("kernel_export", writeback_kernel)):
        torch.cuda.synchronize()
        s0 = ev(); s0.record(bank.copy_stream)
        bank.prepare(1, host.k, host.v, plan_all, plan_all)
        stop = threading.Event()

        def exporter(fn=fn):
            torch.cuda.set_device(comp.device)
            while not stop.is_set():
                with torch.cuda.stream(d2h):
                    fn(d2h)
                e = ev(); e.record(d2h); e.synchronize()
        th = threading.Thread(target=exporter, daemon=True)
        th.start()
        n_ov = 8
        eo = timed(n_ov)
        e_h2d = bank.ready(1)
        torch.cuda.synchronize()
        stop.set()
        th.join()
        ends = [s0.elapsed_time(x) for x in eo]
        h_end = s0.elapsed_time(e_h2d)
        inside = [k for k in range(n_ov) if ends[k + 1] <= h_end]
        t_ov = float(np.mean([ends[k + 1] - ends[k] for k in inside])) if inside else None
        interference[kind] = {"t_overlap_ms": None if t_ov is None else round(t_ov, 4),
                              "rounds_inside_copy": len(inside),
                              "delta_t": None if t_ov is None else round((t_ov - t_base) / t_base, 4)}
    return {"head_of_line": hol, "rounds_with_export": rounds,
            "interference_h2d_and_export": interference}


def draft_bench(args):
    """The draft stage: one JSON line (not the headline metric).

    A step is one whole stage on one batch: preparation of the arriving
    requests (fused into step 0's attention pass, or --unfused as a gather
    first), then per proposal the append of the processed token's K/V, one
    query of attention per request over its cache, and the inverse-CDF draw of
    the proposal."""
    import torch
    import paper_2609_29364_amd as nsd
    from paper_2609_29364_amd.round import draft_stage, fused_tables
    from workload import CONFIGS, make_draft

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = CONFIGS[args.workload]
    K, V = args.draft_steps, args.draft_vocab
    dd = make_draft(cfg, K, V, dev)
    meta, layer = dd.meta, dd.layer
    i32 = lambda a: torch.as_tensor(np.ascontiguousarray(a), dtype=torch.int32, device=dev)
    bt, qi = i32(meta.block_table), i32(np.arange(cfg.bs + 1))
    st, src, dst = i32(meta.stage_table), i32(meta.src_ids), i32(meta.dst_ids)
    pool_table, stage_rows = fused_tables(bt, st)
    max_len = int(meta.seq_lens.max())
    ws = nsd.new_workspace(nsd.verify_attention_workspace_size(
        cfg.bs, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, 1, max_len), dev)
    out = torch.empty_like(dd.q)
    tok = torch.empty((cfg.bs, K), dtype=torch.int32, device=dev)
    sw = torch.empty(nsd.accept_workspace_size(cfg.bs, V), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    kp, vp, ks, vs = layer.k_pool, layer.v_pool, layer.k_stage, layer.v_stage

    def stage(ev=None):
        # the same calls as round.draft_stage, with events between the kernels
        if ev: ev[0].record(stream)
        if args.unfused:
            nsd.kv_gather(ks, vs, kp, vp, src, dst)
        for i in range(K):
            if ev: ev[1 + 3 * i].record(stream)
            if i == 0 and not args.unfused:
                nsd.kv_append(kp, vp, dd.k_new[0], dd.v_new[0], pool_table, dd.lens[0], qi)
                if ks.numel():
                    nsd.kv_append(ks, vs, dd.k_new[0], dd.v_new[0], stage_rows, dd.lens[0], qi)
            else:
                nsd.kv_append(kp, vp, dd.k_new[i], dd.v_new[i], bt, dd.lens[i], qi)
            if ev: ev[2 + 3 * i].record(stream)
            if i == 0 and not args.unfused:
                nsd.gather_verify_attention(dd.q[0], kp, vp, ks, vs, bt, st, dd.lens[0], qi, 1,
                                            max_len, out=out[0], workspace=ws)
            else:
                nsd.verify_attention(dd.q[i], kp, vp, bt, dd.lens[i], qi, 1, max_len, out=out[i],
                                     workspace=ws)
            if ev: ev[3 + 3 * i].record(stream)
            nsd.sample(dd.probs[:, i], dd.uniforms[i], out=tok[:, i], workspace=sw)
        if ev: ev[1 + 3 * K].record(stream)

    def library_stage():
        draft_stage(kp, vp, dd.q, dd.k_new, dd.v_new, dd.probs, dd.uniforms, bt, dd.lens, qi,
                    max_len, k_stage=ks, v_stage=vs, stage_table=None if args.unfused else st,
                    src_ids=src, dst_ids=dst, tokens=tok, out=out, workspace=ws,
                    append_tables=(pool_table, stage_rows), sample_workspace=sw)

    # the timed region: the library's draft stage, back to back
    for _ in range(args.warmup):
        library_stage()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(args.steps):
        library_stage()
    end.record(stream)
    torch.cuda.synchronize()
    ms_stage = start.elapsed_time(end) / args.steps
    # per-kernel breakdown from the same calls with events between them
    n_ev = 2 + 3 * K
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)]
           for _ in range(max(3, args.steps // 2))]
    for e in evs:
        stage(e)
    torch.cuda.synchronize()
    t = np.array([[e[j].elapsed_time(e[j + 1]) for j in range(n_ev - 1)] for e in evs]).mean(0)
    gather_ms = float(t[0])
    append_ms = t[1::3][:K]
    attn_ms = t[2::3][:K]
    sample_ms = t[3::3][:K]

    hkv, d, hq = cfg.num_kv_heads, cfg.head_dim, cfg.num_q_heads
    token_bytes = 2 * hkv * d * 2
    block_bytes = hkv * 16 * d * 2
    lens = dd.lens.cpu().numpy().astype(np.int64)
    qo = 2 * cfg.bs * hq * d * 2
    attn_bytes = [int(lens[i].sum()) * token_bytes + qo for i in range(K)]
    # step 0 of the fused path: resident tokens read, the staged blocks it covers read and written
    nb0 = -(-lens[0] // 16)
    arr = meta.arriving
    fused0 = (int(lens[0][~arr].sum()) * token_bytes + 2 * 2 * int(nb0[arr].sum()) * block_bytes
              + qo)
    sample_bytes = cfg.bs * V * 4 + cfg.bs * 8
    steady = [attn_bytes[i] / (attn_ms[i] * 1e-3) / 1e9 for i in range(1, K)]
    dom_ms = float(np.mean(attn_ms[1:])) if K > 1 else float(attn_ms[0])
    dom_bytes = float(np.mean(attn_bytes[1:])) if K > 1 else attn_bytes[0]
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    res = {
        "metric": "draft-stage requests/s (draft decode shape, K single-query steps); "
                  "achieved HBM TB/s",
        "mode": "draft",
        "value": round(cfg.bs / (ms_stage * 1e-3), 1), "unit": "requests/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_stage, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": describe(cfg) | {"draft_steps": K, "vocab": V},
        "path": "unfused" if args.unfused else "fused",
        "breakdown_ms": {"kv_gather": round(gather_ms, 5) if args.unfused else 0.0,
                         "kv_append": [round(float(x), 5) for x in append_ms],
                         "attention": [round(float(x), 5) for x in attn_ms],
                         "sample": [round(float(x), 5) for x in sample_ms]},
        "step0_fused_tbs": None if args.unfused else
                           round(fused0 / (attn_ms[0] * 1e-3) / 1e12, 3),
        "decode_attention_tbs": [round(x / 1e3, 3) for x in steady],
        "sample_tbs": round(sample_bytes / (float(np.mean(sample_ms)) * 1e-3) / 1e12, 3),
        "roofline": {"bound": "hbm", "kernel": "verify_attention (one query per request)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "alg_bytes_per_launch": int(dom_bytes)},
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = draft_cpu_baseline(cfg, dd, args.cpu_seconds)
    print(json.dumps(res), flush=True)


def phi_bench(args):
    """Stage times of our kernels against batch size (one layer): the target
    round on verify_8b-shaped requests (contexts U[1024, 4096], K = 4, 30 %
    arriving; fused preparation + attention, then acceptance) and the draft
    stage on draft_decode-shaped requests (contexts U[512, 2048], 25 %
    arriving, --draft-steps proposals over --draft-vocab tokens)."""
    import dataclasses
    import torch
    import paper_2609_29364_amd as nsd
    from paper_2609_29364_amd.round import draft_stage, fused_tables
    from workload import CONFIGS, make_meta, make_layer, make_accept, make_draft

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    i32 = lambda a: torch.as_tensor(np.ascontiguousarray(a), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)

    def timed(fn, n):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(n):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    target = {"sizes": [], "ms": []}
    for b in (1, 4, 8, 16, 32, 64, 128, 256, 512):
        cfg = dataclasses.replace(CONFIGS["verify_8b"], bs=b, n_arriving=int(round(0.3 * b)))
        meta = make_meta(cfg)
        lay = make_layer(cfg, meta, 0, dev)
        acc = make_accept(cfg, meta, dev)
        bt, st, sl, qi = (i32(meta.block_table), i32(meta.stage_table), i32(meta.seq_lens),
                          i32(meta.q_indptr))
        ws = nsd.new_workspace(nsd.verify_attention_workspace_size(
            b, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, meta.max_q, meta.max_seq_len), dev)
        out = torch.empty_like(lay.q)
        al = torch.empty(b, dtype=torch.int32, device=dev)
        tk = torch.empty(meta.total_q, dtype=torch.int32, device=dev)
        aw = torch.empty(nsd.accept_workspace_size(b, cfg.vocab), dtype=torch.uint8, device=dev)

        def round_():
            nsd.gather_verify_attention(lay.q, lay.k_pool, lay.v_pool, lay.k_stage, lay.v_stage,
                                        bt, st, sl, qi, meta.max_q, meta.max_seq_len, out=out,
                                        workspace=ws)
            nsd.spec_accept(acc.p_target, acc.q_draft, acc.draft_tokens, acc.uniforms, qi,
                            cfg.k_hi, accepted_len=al, out_tokens=tk, workspace=aw)
        target["sizes"].append(b)
        target["ms"].append(round(timed(round_, max(5, args.steps // 2)), 5))
        del meta, lay, acc, ws, out
        torch.cuda.empty_cache()
    draft = {"sizes": [], "ms": []}
    for b in (1, 16, 64, 128, 256, 512, 1024):
        cfg = dataclasses.replace(CONFIGS["draft_decode"], bs=b, n_arriving=b // 4)
        dd = make_draft(cfg, args.draft_steps, args.draft_vocab, dev)
        meta, lay = dd.meta, dd.layer
        bt, st = i32(meta.block_table), i32(meta.stage_table)
        qi = i32(np.arange(b + 1))
        tables = fused_tables(bt, st)
        max_len = int(meta.seq_lens.max())
        ws = nsd.new_workspace(nsd.verify_attention_workspace_size(
            b, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, 1, max_len), dev)
        out = torch.empty_like(dd.q)
        tok = torch.empty((b, args.draft_steps), dtype=torch.int32, device=dev)
        sw = torch.empty(nsd.accept_workspace_size(b, args.draft_vocab), dtype=torch.uint8,
                         device=dev)

        def stage_():
            draft_stage(lay.k_pool, lay.v_pool, dd.q, dd.k_new, dd.v_new, dd.probs, dd.uniforms,
                        bt, dd.lens, qi, max_len, k_stage=lay.k_stage, v_stage=lay.v_stage,
                        stage_table=st, tokens=tok, out=out, workspace=ws, append_tables=tables,
                        sample_workspace=sw)
        draft["sizes"].append(b)
        draft["ms"].append(round(timed(stage_, max(5, args.steps // 2)), 5))
        del dd, meta, lay, ws, out
        torch.cuda.empty_cache()
    print(json.dumps({"mode": "phi", "layers": 1, "draft_steps": args.draft_steps,
                      "draft_vocab": args.draft_vocab,
                      "target": target | {"workload": "verify_8b shapes, bs varied"},
                      "draft": draft | {"workload": "draft_decode shapes, bs varied"}}),
          flush=True)


# Stage profiles printed in Appendix C (batch-size profiling): one draft forward
# takes about 16 ms at batch 1 and 18 ms at 512, 38.6 ms at 1024, with SM
# activity 9.1 %, 86.8 % and 95.1 %; target verification at depth 4 reaches SM
# activity 74.1 % at 1 request, 87.5 % at 32, 93.2 % at 64 and 95.7 % at 128,
# taking 28.8 ms at 32, 46.3 ms at 64 and 82.8 ms at 128 (below 32 the time is
# taken as flat).  A draft stage is `depth` forwards.
PAPER_PHI_DRAFT_FWD = ([1, 512, 1024], [0.016, 0.018, 0.0386], [0.091, 0.868, 0.951])
PAPER_PHI_TARGET = ([1, 32, 64, 128], [0.0288, 0.0288, 0.0463, 0.0828],
                    [0.741, 0.875, 0.932, 0.957])


def schedule_bench(args):
    """Host scheduler: one JSON line (no GPU).

    * decision latency: one reconstruction over C candidates (predecessor ends
      and KV-ready times uniform over 10 ms, worker free at 5 ms, g = 0, Delta =
      30 ms), the library against the oracle;
    * simulation (Appendix H): 6 draft + 32 target workers, 4096 requests, 32
      rounds of depth 4, draft/target batch limits 512/32, window [1, 2.5] s,
      with the stage profiles printed in Appendix C, and with our kernels' own
      one-layer stage times (profiles/phi_tables.json, from bench.py --phi)."""
    import paper_2609_29364_amd.schedule as sch
    import oracle
    rng = np.random.default_rng(0)
    lat = []
    for c, bmax in ((1024, 32), (16384, 32), (16384, 512)):
        ids = np.arange(c, dtype=np.int32)
        e = rng.uniform(0, 0.01, c)
        k = rng.uniform(0, 0.01, c)
        el, kl = e.tolist(), k.tolist()
        t0 = time.perf_counter()
        n = 0
        while time.perf_counter() - t0 < 0.5:
            sch.reconstruct(ids, e, k, a_hat=0.005, b_max=bmax, g=0.0, delta=0.03)
            n += 1
        t_lib = (time.perf_counter() - t0) / n
        t0 = time.perf_counter()
        m = 0
        z = [0] * c
        while time.perf_counter() - t0 < 1.0 or m == 0:
            oracle.schedule.reconstruct(list(range(c)), el, kl, z, z, 0.005, 0, 0, bmax, 0.0, 0.03)
            m += 1
        t_or = (time.perf_counter() - t0) / m
        lat.append({"candidates": c, "b_max": bmax, "lib_us": round(t_lib * 1e6, 2),
                    "oracle_us": round(t_or * 1e6, 1)})
    depth = 4
    phi_d = (PAPER_PHI_DRAFT_FWD[0], [depth * x for x in PAPER_PHI_DRAFT_FWD[1]],
             PAPER_PHI_DRAFT_FWD[2])
    sims = []
    setups = [("paper Appendix C profiles", phi_d, PAPER_PHI_TARGET, (1.0, 2.5))]
    try:
        tab = json.load(open(os.path.join(ROOT, "profiles", "phi_tables.json")))
        # our kernels: one layer of each stage, full activity (every launch fills the chip)
        kd = (tab["draft"]["sizes"], [x * 1e-3 for x in tab["draft"]["ms"]],
              [1.0] * len(tab["draft"]["sizes"]))
        kt = (tab["target"]["sizes"], [x * 1e-3 for x in tab["target"]["ms"]],
              [1.0] * len(tab["target"]["sizes"]))
        setups.append(("our kernels, one layer per stage", kd, kt, (0.02, 0.08)))
    except (OSError, KeyError, ValueError):
        pass
    for name, pd, pt, window in setups:
        t0 = time.perf_counter()
        m, _ = sch.simulate(6, 32, 4096, 32, pd, pt, 512, 32, 0.0, 0.0, 0.03 * window[1] / 2.5,
                            0.03 * window[1] / 2.5, window, trace=False)
        wall = time.perf_counter() - t0
        sims.append({"profiles": name, "window_s": list(window),
                     "U": round(m["U"], 4), "S": round(m["S"], 4),
                     "round_rate": round(m["round_rate"], 1), "batches": m["batches"],
                     "wall_s": round(wall, 3), "batches_per_s": round(m["batches"] / wall, 1)})
    # the oracle on the first simulation (same inputs): equal metrics, its time
    t0 = time.perf_counter()
    mo, _ = oracle.schedule.simulate(6, 32, 4096, 32, phi_d, PAPER_PHI_TARGET, 512, 32, 0.0,
                                     0.0, 0.03, 0.03, (1.0, 2.5))
    t_or = time.perf_counter() - t0
    ml, _ = sch.simulate(6, 32, 4096, 32, phi_d, PAPER_PHI_TARGET, 512, 32, 0.0, 0.0, 0.03,
                         0.03, (1.0, 2.5), trace=False)
    res = {"mode": "schedule", "metric": "scheduling decision latency (us); simulated pool "
           "metrics (Eqs. H.1, H.2)", "decision_latency": lat, "simulation": sims,
           "oracle_metrics_equal": ml == mo,
           "cpu_baseline": {"value": round(mo["batches"] / t_or, 1), "unit": "batches/s",
                            "cores": 1, "kind": "oracle",
                            "sample": f"the oracle simulator on the first simulation above "
                                      f"({mo['batches']} batches), {t_or:.1f} s"}}
    print(json.dumps(res), flush=True)


def draft_cpu_baseline(cfg, dd, budget_s):
    """The draft-stage oracle, untuned, on a bounded sample of the requests."""
    import oracle
    from workload.synth import logical_kv
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = 1
    order = np.random.default_rng(0).permutation(cfg.bs)
    done, t_total = 0, 0.0
    scale = 1.0 / np.sqrt(cfg.head_dim)
    # passes over the requests until the time budget is spent
    for r in (r for _ in range(1000) for r in order):
        if t_total >= budget_s and done >= 2:
            break
        k, v = logical_kv(dd.meta, dd.layer, r)
        p = int(dd.prefix[r])
        args = (k[:p].double().cpu().numpy(), v[:p].double().cpu().numpy(),
                dd.q[:, r].double().cpu().numpy(), dd.k_new[:, r].double().cpu().numpy(),
                dd.v_new[:, r].double().cpu().numpy(), dd.probs[r].cpu().numpy(),
                dd.uniforms[:, r].cpu().numpy(), scale)
        t0 = time.perf_counter()
        oracle.draft.draft_request(*args)
        t_total += time.perf_counter() - t0
        done += 1
    return {"value": round(done / t_total, 3), "unit": "requests/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"{done} of {cfg.bs} requests" if done <= cfg.bs else
                       f"{done} requests ({done / cfg.bs:.1f} passes over the {cfg.bs})")
                      + f" of the {cfg.name} draft stage "
                      f"({dd.steps} steps: append, attention, sampling), {t_total:.1f} s of "
                      f"fp64 numpy"}


def ceiling_bench(args):
    """The probe alone on the fused pass's bytes for the workload: one JSON line
    with the read-only rate and the read + write-back rate for each placement
    of the written tiles."""
    import torch
    from workload import CONFIGS, make_meta
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = CONFIGS[args.workload]
    meta = make_meta(cfg)
    alg = algorithmic_bytes(cfg, meta)
    # one layer's pass (a many-layer round runs the same pass once per layer)
    layers = cfg.num_layers
    w = alg["gather"] // 2 // layers
    res = {"mode": "ceiling", "workload": cfg.name, "layers": layers,
           "read_bytes": alg["fused"] // layers - w, "write_bytes": w}
    for placement in ("end", "spread", "waves", "writer"):
        res[placement] = practical_ceiling(dev, res["read_bytes"], w, placement=placement)
    print(json.dumps(res), flush=True)


def sweep_bench(args):
    """Every named round workload, one JSON line each (the default bench line is
    verify_8b).  A step is the fused preparation + attention pass of every
    layer, then acceptance.  The 36-layer round does not fit in HBM at once, so
    it is streamed: each layer's inputs are generated (untimed), its pass is
    timed with HIP events, and the round time is the sum over the layers plus
    one acceptance."""
    import torch
    import paper_2609_29364_amd as nsd
    from workload import CONFIGS, make_meta, make_layer, make_accept

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    i32 = lambda a: torch.as_tensor(np.ascontiguousarray(a), dtype=torch.int32, device=dev)

    def timed(fn, warm, n):
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(n):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / n

    for name in ("tiny", "draft_decode", "verify_8b", "knee", "full_depth"):
        cfg = CONFIGS[name]
        meta = make_meta(cfg)
        bt, st, sl, qi = (i32(meta.block_table), i32(meta.stage_table), i32(meta.seq_lens),
                          i32(meta.q_indptr))
        ws = nsd.new_workspace(nsd.verify_attention_workspace_size(
            cfg.bs, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, meta.max_q,
            meta.max_seq_len), dev)
        reps = max(3, args.steps // 5) if cfg.num_layers > 1 else args.steps
        layer_ms = []
        lay0 = None
        for l in range(cfg.num_layers):
            lay = make_layer(cfg, meta, l, dev)
            out = torch.empty_like(lay.q)
            layer_ms.append(timed(lambda: nsd.gather_verify_attention(
                lay.q, lay.k_pool, lay.v_pool, lay.k_stage, lay.v_stage, bt, st, sl, qi,
                meta.max_q, meta.max_seq_len, out=out, workspace=ws), args.warmup, reps))
            if l == 0 and not args.no_cpu_baseline:
                lay0 = lay          # the oracle sample uses layer 0's inputs
            del lay, out
            if cfg.num_layers > 1:
                torch.cuda.empty_cache()
        acc_in = make_accept(cfg, meta, dev)
        acc_ms, acc_host, acc_cold_ms = 0.0, None, None
        if acc_in is not None:
            al = torch.empty(cfg.bs, dtype=torch.int32, device=dev)
            tk = torch.empty(meta.total_q, dtype=torch.int32, device=dev)
            aw = torch.empty(nsd.accept_workspace_size(cfg.bs, cfg.vocab), dtype=torch.uint8,
                             device=dev)
            accept = lambda: nsd.spec_accept(
                acc_in.p_target, acc_in.q_draft, acc_in.draft_tokens, acc_in.uniforms, qi,
                int(meta.depth.max()), accepted_len=al, out_tokens=tk, workspace=aw)
            acc_ms = timed(accept, args.warmup, args.steps)
            acc_host = al.cpu().numpy()
            # each call after a 1 GiB read, so none of its rows is left in the
            # infinity cache (as inside a round, after the attention passes)
            scrub = torch.ones(1 << 28, dtype=torch.float32, device=dev)
            sink = torch.empty((), dtype=torch.float32, device=dev)
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(args.steps)]
            for a, b in ev:
                torch.sum(scrub, dim=0, out=sink)
                a.record(stream)
                accept()
                b.record(stream)
            torch.cuda.synchronize()
            acc_cold_ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
            del scrub, sink
        alg = algorithmic_bytes(cfg, meta, acc_host)
        fused_ms = float(np.sum(layer_ms))
        round_ms = fused_ms + acc_ms
        res = {"mode": "sweep", "workload": name, "config": describe(cfg),
               "value": round(cfg.bs / (round_ms * 1e-3), 1), "unit": "requests/s",
               "ms_per_round": round(round_ms, 4),
               "fused_ms": round(fused_ms, 4), "accept_ms": round(acc_ms, 4),
               "fused_layer_ms": [round(x, 4) for x in layer_ms] if cfg.num_layers > 1 else None,
               "bytes": alg,
               "fused_tbs": round(alg["fused"] / (fused_ms * 1e-3) / 1e12, 3),
               "fused_frac": round(alg["fused"] / (fused_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
               "gather_attention_equiv_tbs": round((alg["gather"] + alg["attention"]) /
                                             (fused_ms * 1e-3) / 1e12, 3),
               "accept_tbs": (round(alg["accept"] / (acc_ms * 1e-3) / 1e12, 3)
                              if acc_ms > 0 else None),
               "accept_scrubbed_ms": (round(acc_cold_ms, 4) if acc_cold_ms else None),
               "accept_scrubbed_tbs": (round(alg["accept"] / (acc_cold_ms * 1e-3) / 1e12, 3)
                                       if acc_cold_ms else None),
               "timing": f"mean of {reps} back-to-back passes per layer after {args.warmup} "
                         f"warm-up, HIP events on the launching stream"}
        if name != "tiny" and not args.no_ceiling:
            # the probe on one layer's read/write mix (the tiny round is cache-resident)
            wb = alg["gather"] // 2 // cfg.num_layers
            c = practical_ceiling(dev, alg["fused"] // cfg.num_layers - wb, wb)
            res["probe_mix_gbs"] = c["mix_gbs"]
            res["probe_read_only_gbs"] = c["read_only_gbs"]
            res["fused_of_probe"] = round(alg["fused"] / (fused_ms * 1e-3) / 1e9 / c["mix_gbs"], 4)
        if lay0 is not None:
            res["cpu_baseline"] = cpu_baseline(cfg, meta, lay0, acc_in, args.cpu_seconds)
        print(json.dumps(res), flush=True)
        del meta, lay0, acc_in, ws
        torch.cuda.empty_cache()


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the verification round runs on one GPU: the library has no multi-GPU path; use --gpus 1"}))
        sys.exit(2)
    if args.schedule:
        schedule_bench(args)
        return
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.h2d:
        h2d_bench(args)
        return
    if args.draft:
        draft_bench(args)
        return
    if args.phi:
        phi_bench(args)
        return
    if args.sweep:
        sweep_bench(args)
        return
    if args.ceiling:
        ceiling_bench(args)
        return
    import torch
    import paper_2609_29364_amd as nsd
    from workload import CONFIGS, make_meta, make_layer, make_accept

    if not os.path.exists(nsd.LIB_PATH):
        from paper_2609_29364_amd.build import build
        build()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = CONFIGS[args.workload]
    if cfg.num_layers != 1:
        raise SystemExit("bench times single-layer workloads; the 36-layer round is a test case")
    meta = make_meta(cfg)
    layer = make_layer(cfg, meta, 0, dev)
    acc_in = make_accept(cfg, meta, dev)
    i32 = lambda a: torch.as_tensor(np.ascontiguousarray(a), dtype=torch.int32, device=dev)
    src, dst = i32(meta.src_ids), i32(meta.dst_ids)
    bt, sl, qi = i32(meta.block_table), i32(meta.seq_lens), i32(meta.q_indptr)
    kp, vp = layer.k_pool, layer.v_pool
    ks, vs = layer.k_stage, layer.v_stage
    st = i32(meta.stage_table)
    out = torch.empty_like(layer.q)
    ws_n = nsd.verify_attention_workspace_size(cfg.bs, cfg.num_q_heads, cfg.num_kv_heads,
                                               cfg.head_dim, meta.max_q, meta.max_seq_len)
    ws = nsd.new_workspace(ws_n, dev)
    acc_len = torch.empty(cfg.bs, dtype=torch.int32, device=dev)
    toks = torch.empty(meta.total_q, dtype=torch.int32, device=dev)
    acc_ws = torch.empty(max(1, nsd.accept_workspace_size(cfg.bs, max(cfg.vocab, 4))),
                         dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)

    def step(ev=None):
        if ev: ev[0].record(stream)
        if args.unfused:
            nsd.kv_gather(ks, vs, kp, vp, src, dst)
        if ev: ev[1].record(stream)
        if args.unfused:
            nsd.verify_attention(layer.q, kp, vp, bt, sl, qi, meta.max_q, meta.max_seq_len,
                                 out=out, workspace=ws)
        else:
            nsd.gather_verify_attention(layer.q, kp, vp, ks, vs, bt, st, sl, qi, meta.max_q,
                                        meta.max_seq_len, out=out, workspace=ws)
        if ev: ev[2].record(stream)
        if acc_in is not None:
            nsd.spec_accept(acc_in.p_target, acc_in.q_draft, acc_in.draft_tokens,
                            acc_in.uniforms, qi, cfg.k_hi, accepted_len=acc_len, out_tokens=toks,
                            workspace=acc_ws)
        if ev: ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # the timed region: K whole steps back to back, nothing else on the stream
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    start.record(stream)
    for i in range(args.steps):
        step()
    end.record(stream)
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms_total = start.elapsed_time(end)
    ms_step = ms_total / args.steps
    # per-kernel breakdown from the same steps run again with events between the
    # kernels (an event record adds a few microseconds, so it stays out of the
    # timed region)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    parts = np.array([[e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[2].elapsed_time(e[3])]
                      for e in evs])
    g_ms, a_ms, c_ms = parts.mean(0)
    # per-step spread, and the same steps after an untimed 1 GiB read that
    # evicts the 256 MB last-level cache (MALL) before each step (a read, so
    # the scrub leaves no dirty lines to be written back during the step): the
    # A/B shows how much of the back-to-back figure any cache carry-over explains
    scrub = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    scrub_sink = torch.empty((), dtype=torch.float32, device=dev)

    def per_step(scrubbed):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
        for i in range(args.steps):
            if scrubbed:
                torch.sum(scrub, dim=0, out=scrub_sink)
            ev[i][0].record(stream)
            step()
            ev[i][1].record(stream)
        torch.cuda.synchronize()
        return np.array([a.elapsed_time(b) for a, b in ev])

    t_plain, t_scrub = per_step(False), per_step(True)
    del scrub, scrub_sink
    spread = {"median": round(float(np.median(t_plain)), 5),
              "min": round(float(t_plain.min()), 5), "max": round(float(t_plain.max()), 5),
              "median_scrubbed": round(float(np.median(t_scrub)), 5),
              "min_scrubbed": round(float(t_scrub.min()), 5),
              "max_scrubbed": round(float(t_scrub.max()), 5),
              "scrub_bytes_read": 1 << 30,
              "scrub_effect": round(float(np.median(t_scrub) / np.median(t_plain) - 1.0), 4)}
    acc_host = acc_len.cpu().numpy() if acc_in is not None else None
    alg = algorithmic_bytes(cfg, meta, acc_host)
    # the dominant kernel: the fused pass, or attention when run unfused
    kern = "verify_attention" if args.unfused else "gather_verify_attention"
    kb = alg["attention"] if args.unfused else alg["fused"]
    step_bytes = (alg["gather"] + alg["attention"] if args.unfused else alg["fused"]) + alg["accept"]
    achieved = kb / (a_ms * 1e-3) / 1e9
    result = {
        "metric": "verify-round requests/s (8B-shaped layer, bs=256, K=4); achieved HBM TB/s",
        "value": round(cfg.bs / (ms_step * 1e-3), 1),
        "unit": "requests/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": describe(cfg),
        "path": "unfused" if args.unfused else "fused",
        "breakdown_ms": ({"kv_gather": round(g_ms, 5)} if args.unfused else {}) |
                        {kern: round(a_ms, 5), "spec_accept": round(c_ms, 5)},
        "step_ms": spread,
        "round_hbm_tbs": round(step_bytes / (ms_step * 1e-3) / 1e12, 3),
        # an equivalent rate, not an HBM rate: the bytes the separate gather and
        # attention kernels would move, over the time this path took for that work
        "gather_attention_equiv_tbs": round((alg["gather"] + alg["attention"]) /
                                            (((g_ms if args.unfused else 0.0) + a_ms) * 1e-3) /
                                            1e12, 3),
        "roofline": {"bound": "hbm", "kernel": kern, "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(kern),
                     "alg_bytes_per_launch": kb},
        "wall_s_timed": round(t_wall, 3),
    }
    if not args.no_ceiling:
        # the dominant kernel's own read/write mix: the fused pass writes the staged
        # blocks back; attention alone only reads
        w = 0 if args.unfused else alg["gather"] // 2
        ceil = practical_ceiling(dev, kb - w, w)
        c = ceil["mix_gbs"]
        result["roofline"]["practical"] = {"ceiling_gbs": c, "frac": round(achieved / c, 4),
                                           "read_only_gbs": ceil["read_only_gbs"],
                                           "pattern": ceil["pattern"]}
    if not args.no_cpu_baseline:
        base = cpu_baseline(cfg, meta, layer, acc_in, args.cpu_seconds)
        # one-thread figures on this workload and on the tiny round
        one = {cfg.name: cpu_baseline(cfg, meta, layer, acc_in, args.cpu_seconds / 3,
                                      threads=1)["value"]}
        tcfg = CONFIGS["tiny"]
        tmeta = make_meta(tcfg)
        tlay = make_layer(tcfg, tmeta, 0, dev)
        tacc = make_accept(tcfg, tmeta, dev)
        tiny = cpu_baseline(tcfg, tmeta, tlay, tacc, 1.0)
        one["tiny"] = cpu_baseline(tcfg, tmeta, tlay, tacc, 1.0, threads=1)["value"]
        base["one_thread_requests_per_s"] = one
        base["tiny_requests_per_s"] = tiny["value"]
        result["cpu_baseline"] = base
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
