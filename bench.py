"""Benchmark of the verify hot path on one MI355X.

One step = one replay of a captured hipGraph holding the whole path on one
batch: verify attention (stream-K kernel + combine kernel) for one attention
layer, then greedy acceptance (argmax kernel + prefix kernel).  Workload:
Qwen3-8B attention shape at concurrency 32 -- B=32 requests, 32 query / 8 KV
heads, head_dim 128, bf16 paged KV (page 16), contexts uniform in
[1024, 8192], verify lengths 1..16 (anchor + truncated geometric, p=0.25)
packed into capacity 256, acceptance over bf16 logits [256 x 151936] with
the planted geometric accept lengths.  Inputs are synthetic and seeded, and
resident in HBM before the timed region.

Prints one JSON line.  ``value`` = packed verify tokens per second of the
whole step (sum of live verify lengths / step time).  ``roofline`` is for
the dominant kernel (the stream-K attention kernel), timed with timing-only
HIP events (no system-scope fence) on its stream; ``cpu_baseline`` times the fp64 CPU oracle on a bounded sample.
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

METRIC = "packed verify tokens/s + HBM GB/s (% peak) per layer, Qwen3-8B shape, B=8/16/32"
UNIT = "packed verify tokens/s"
HBM_PEAK_GBPS = 8000.0
CONFIG_INDEX = 4
COUNTERS_FILE = os.path.join(ROOT, "profiles", "attn_streamk_config4_counters.json")
ATTN_SOURCE = os.path.join(ROOT, "paper_2609_37532_amd", "csrc", "attn.hip")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # the GPU's clocks take about 150 back-to-back steps to settle: the first
    # 50-step window after 10 warm-up steps ran 6-9% slower than the later ones
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=300)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle sample")
    ap.add_argument("--eager-only", type=int, default=0, metavar="N",
                    help="only run N eager steps (no graph, no timing, no CPU "
                         "baseline): the program that hardware-counter passes profile")
    ap.add_argument("--eager-attention", type=int, default=0, metavar="C",
                    help="with --eager-only N: run N eager verify-attention launches of "
                         "config C (2, 3 or 4), or of one layer of the 36-layer stress "
                         "run at its first step (5), with a 512 MB scrub before each, and "
                         "nothing else: the program that per-shape counter passes profile")
    ap.add_argument("--no-stress", action="store_true",
                    help="skip the 36-layer graph-replay stress measurement")
    ap.add_argument("--stress-steps", type=int, default=100)
    ap.add_argument("--no-next", action="store_true",
                    help="skip the next-row sections (stochastic verifier, DVL, bucket set)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only copy a 1 GiB device buffer three times: the plain copy "
                         "of known size that scales the hardware byte counters")
    return ap.parse_args()


def attention_bytes(attn, hkv, hq, d):
    """Algorithmic HBM bytes of one verify-attention launch: every live key's
    K and V once per KV head, q read and out written once per live row, plus
    the metadata (offsets, context lengths, the page-table entries used)."""
    k = attn.qlens.astype(np.int64)
    keys = attn.ctx_lens.astype(np.int64) + k
    live = k > 0
    kv = int((keys[live] * hkv * d * 2 * 2).sum())
    qo = int(k.sum()) * hq * d * 2 * 2
    pages = int(((keys[live] + 15) // 16).sum())
    meta = (attn.num_reqs + 1 + attn.num_reqs + pages) * 4
    return kv + qo + meta


def accept_bytes(acc, esize):
    """Algorithmic bytes of acceptance: live logit rows once, the draft
    tokens of live rows, offsets, and the two outputs."""
    live = int(acc.cu_qlens[-1])
    return live * acc.vocab * esize + live * 4 + (acc.num_reqs + 1) * 4 + 2 * acc.num_reqs * 4


def row_padding(qlens, group):
    """Inactive-row fractions of the batch under Eq. (2): rows(l, B) =
    B*ceil(l/B), padding = 1 - l/rows, summed over live requests.  The
    paper's tiles hold one request's l = k_i rows of one head (B = 128 native,
    B = 16 with tile routing); this kernel stacks the G heads that share a KV
    head, so its 16-row MFMA tiles hold l = G*k_i rows."""
    k = np.asarray(qlens, dtype=np.int64)
    k = k[k > 0]

    def pad(l, b):
        return 1.0 - float(l.sum()) / float((b * -(-l // b)).sum())
    return {"paper_128_row_tiles": round(pad(k, 128), 4),
            "paper_16_row_tiles": round(pad(k, 16), 4),
            "live_row_mfma_tiles": round(pad(group * k, 16), 4)}


def attention_flops(attn, hq, d):
    """q.k and p.v flops over the visible keys of every live row."""
    tot = 0
    for ctx, k in zip(attn.ctx_lens.astype(np.int64), attn.qlens.astype(np.int64)):
        vis = k * ctx + k * (k + 1) // 2  # sum_j (ctx + j + 1)
        tot += int(vis) * hq * 4 * d
    return tot


def counters_traffic(nbytes_alg):
    """HBM traffic from committed rocprofv3 counter runs, if they were taken
    on the current attention source; else None."""
    try:
        with open(COUNTERS_FILE) as f:
            c = json.load(f)
        src = hashlib.sha256(open(ATTN_SOURCE, "rb").read()).hexdigest()
        if c.get("attn_source_sha256") != src:
            return None
        return int(c["hbm_bytes_per_launch"])
    except Exception:
        return None


def cpu_threads():
    """Host threads for the all-cores oracle timing: the machine's CPU share (16
    per GPU, exported as OMP_NUM_THREADS there), never more than the CPUs."""
    n = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or 16
    return max(1, min(n, os.cpu_count() or 1))


def cpu_model():
    """The host CPU's model name (lscpu, else /proc/cpuinfo) and its logical CPUs."""
    import subprocess
    name = None
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.strip().startswith("Model name:"):
                name = line.split(":", 1)[1].strip()
                break
    except Exception:
        pass
    if name is None:
        try:
            for line in open("/proc/cpuinfo"):
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
        except Exception:
            name = "unknown"
    return {"model": name, "logical_cpus": os.cpu_count()}


def cpu_baseline(attn, acc, seconds):
    """fp64 oracle over the requests of the same batch (attention rows of a
    request + its acceptance rows), repeating passes over the batch for about
    ``seconds``: once on one thread, then with the requests of each pass
    spread over all host threads (independent oracle calls; ctypes releases
    the GIL).  Returns (all-cores result, single-thread result)."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    import workloads as W
    subs = []
    for i in range(attn.num_reqs):
        k = int(attn.qlens[i])
        if k == 0:
            continue
        o = int(attn.cu_qlens[i])
        subs.append((W.repack(attn, [i], capacity=k), acc.logits[o:o + k],
                     acc.draft_tokens[o:o + k], k))

    def one(sub, sub_logits, sub_draft, k):
        oracle.verify_attn(sub.q, sub.cu_qlens, sub.kv_pages, sub.page_table,
                           sub.ctx_lens, **sub.oracle_kwargs())
        oracle.accept(sub_logits, acc.dtype, np.array([0, k], np.int32), sub_draft)
        return k

    done_tokens, done_reqs, passes, t_total = 0, 0, 0, 0.0
    while t_total < seconds:
        for sub in subs:
            t0 = time.perf_counter()
            done_tokens += one(*sub)
            t_total += time.perf_counter() - t0
            done_reqs += 1
            if t_total >= seconds:
                break
        passes += 1
    host = cpu_model()
    single = {"value": done_tokens / t_total, "unit": UNIT, "cores": 1, "kind": "oracle",
              "cpu": host,
              "sample": "%d request-verifications (%d passes over the %d live requests of "
                        "the same batch, %d packed rows): fp64 attention over each "
                        "request's keys + acceptance of its rows, %.1f s, single thread"
                        % (done_reqs, passes, len(subs), done_tokens, t_total)}
    threads = cpu_threads()
    mt_tokens, mt_passes = 0, 0
    with ThreadPoolExecutor(max_workers=threads) as ex:
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < seconds / 2:
            mt_tokens += sum(ex.map(lambda sub: one(*sub), subs))
            mt_passes += 1
        wall = time.perf_counter() - t0
    multi = {"value": mt_tokens / wall, "unit": UNIT, "cores": threads, "kind": "oracle",
             "cpu": host,
             "sample": "%d whole passes over the %d live requests of the same batch (%d "
                       "packed rows): fp64 attention + acceptance per request, requests "
                       "spread over %d host threads, %.1f s wall"
                       % (mt_passes, len(subs), mt_tokens, threads, wall)}
    return multi, single


STRESS_WARMUP = 10


def stress_bench(steps):
    """The graph-replay stress run (36 layers, B=32, contexts growing from
    U[512, 4096]): per step, input staging outside the graph, one replay of
    the captured 36-layer verify + acceptance graph timed with HIP events on
    its stream, then the acceptance read back and the contexts grown.  Also
    checks every step's acceptance against the planted values."""
    import torch

    import workloads as W
    from workloads.stress import StressRun

    plan = W.StressPlan(steps=steps)
    run = StressRun(plan)
    st = plan.draw_step()
    run.stage(st)
    run.capture()
    # untimed warm-up: replays of the first step (the graph only reads the
    # staged inputs, so replaying it changes no state)
    for _ in range(STRESS_WARMUP):
        run.replay()
    torch.cuda.synchronize()
    times, tokens, kv_bytes, step_other, exact = [], 0, 0, 0, True
    hq, hkv, d = run.hq, run.hkv, run.d
    for step in range(steps):
        if step > 0:
            st = plan.draw_step()
            run.stage(st)
        keys = (run.ctx_host + st.qlens)[st.qlens > 0]
        kv_bytes += int(keys.sum()) * hkv * d * 2 * 2 * plan.num_layers
        live = int(st.qlens.sum())
        step_other += live * hq * d * 2 * 2 * plan.num_layers + live * plan.vocab * 2
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(run.stream)
        run.replay()
        e1.record(run.stream)
        a, nxt = run.finish(st)
        exact &= bool((a == st.planted_accept_len).all() and (nxt == st.planted_next).all())
        times.append(e0.elapsed_time(e1))
        tokens += int(st.qlens.sum())
    run.close()
    total_ms = float(np.sum(times))
    return {"workload": "36 layers (36 KV pools) of Qwen3-8B-shape verify attention + acceptance "
                        "over 151936 tokens, B=32, contexts from U[512,4096] growing by "
                        "accepted+1 per step, one hipGraph replay per step",
            "steps": steps, "ms_per_step": round(total_ms / steps, 4),
            "us_per_layer_incl_accept": round(total_ms / steps * 1e3 / plan.num_layers, 2),
            "packed_tokens_per_s": round(tokens / (total_ms * 1e-3), 1),
            "kv_gbps": round(kv_bytes / (total_ms * 1e-3) / 1e9, 1),
            "kv_frac": round(kv_bytes / (total_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
            "step_frac": round((kv_bytes + step_other) / (total_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
            "step_frac_counts": "KV of every layer + q/out rows + logits of live rows",
            "acceptance_exact_every_step": exact}


def configs_bench(reps=200):
    """Verify attention alone on the other attention presets (configs 2 and
    3: Qwen3-4B shape B=8 with full blocks over contexts U[256, 2048], and
    Qwen3-8B shape B=16 packed over U[512, 4096]) and config 4 for
    reference: per launch, HIP events around each kernel on its stream.
    Configs 2-3 (33 and 135 MB) would otherwise be served from the 256 MB
    Infinity Cache on repeated launches, so a 512 MB buffer is rewritten
    between launches (outside the event pairs) and every launch reads its
    KV from HBM."""
    import torch

    import paper_2609_37532_amd as dsv
    import workloads as W

    out = {}
    for idx in (2, 3, 4):
        attn = W.config_attn_inputs(idx)
        bf = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to("cuda").view(
            torch.bfloat16)
        i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to("cuda")
        q, kv = bf(attn.q), bf(attn.kv_pages)
        cu, pt, ctx = i32(attn.cu_qlens), i32(attn.page_table), i32(attn.ctx_lens)
        o = torch.zeros_like(q)
        dims = dsv.attn_dims(q, kv, pt, max_kv_len=attn.max_kv_len, scale=attn.scale)
        ws = dsv.alloc_workspace(dsv.verify_attn_workspace_bytes(dims), "cuda")
        s = torch.cuda.Stream()
        run = lambda: dsv.verify_attn(q, cu, kv, pt, ctx, o, dims=dims, workspace=ws, stream=s)
        scrub = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        for _ in range(5):
            run()
        torch.cuda.synchronize()
        with dsv.KernelTimer(max_launches=2 * reps + 8) as tm:
            for r in range(reps):
                with torch.cuda.stream(s):
                    scrub.fill_(r & 0xFF)
                run()
            torch.cuda.synchronize()
        t_split = tm.median_ms("attn_split") * 1e-3
        t_comb = tm.median_ms("attn_combine") * 1e-3 if tm.count("attn_combine") else 0.0
        nbytes = attention_bytes(attn, attn.num_kv_heads, attn.num_q_heads, attn.head_dim)
        toks = int(attn.qlens.sum())
        t_op = t_split + t_comb
        out["config_%d" % idx] = {
            "B": attn.num_reqs, "packed_tokens": toks, "algorithmic_bytes": nbytes,
            "attn_us": round(t_split * 1e6, 2), "combine_us": round(t_comb * 1e6, 2),
            "attn_gbps": round(nbytes / t_split / 1e9, 1),
            "attn_frac": round(nbytes / t_split / 1e9 / HBM_PEAK_GBPS, 4),
            "op_us": round(t_op * 1e6, 2),
            "op_gbps": round(nbytes / t_op / 1e9, 1),
            "op_frac": round(nbytes / t_op / 1e9 / HBM_PEAK_GBPS, 4),
            "us_per_layer": round(t_op * 1e6, 2),
            "packed_tokens_per_s_attention": round(toks / t_op, 1),
            "timing": "median of %d launches per kernel (timing-only HIP events)"
                      % tm.count("attn_split")}
        del q, kv, o, scrub
        torch.cuda.empty_cache()
    return out


def dvl_bench(launches=100, replays=10):
    """The decision step (Sec. III-C, Alg. 1, Eq. (5)) per launch: the
    acceptance predictor (1735-64-15), DVL allocate-and-pack, and the two
    back to back.  Each is ``launches`` calls captured in one hipGraph,
    replayed ``replays`` times and timed with HIP events on the capturing
    stream, for the B=32 bucket of the workload and two larger buckets.
    Inputs: make_predictor_inputs / make_dvl_inputs, all slots live.  One
    workgroup (DVL) or a few (predictor): bound by latency, not by HBM; the
    bytes are given for reference only."""
    import torch

    import paper_2609_37532_amd as dsv
    import workloads as W

    out = {}
    for n_bs in (32, 256, 1024):
        w = W.BLOCK_WIDTH
        rng = np.random.default_rng(W.SEED_BASE + 60 + n_bs)
        d = W.make_dvl_inputs(rng, n_bs=n_bs, n_live=n_bs)
        p = W.make_predictor_inputs(rng, n_bs=n_bs, n_live=n_bs)
        m_bs = w * n_bs // 2
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
        lg, tok, pos, ref = dev(d.pred_logits), dev(d.tokens), dev(d.positions), dev(d.kv_refs)
        feats, w1, b1, w2, b2 = (dev(x) for x in (p.features, p.w1, p.b1, p.w2, p.b2))
        ws_pred = dsv.alloc_workspace(dsv.predictor_workspace_bytes(n_bs, p.features.shape[1]),
                                      "cuda")
        nl = dev(np.array([n_bs], np.int32))
        z = lambda n: torch.zeros(n, dtype=torch.int32, device="cuda")
        k, cu, pt, pp, pr = z(n_bs), z(n_bs + 1), z(m_bs), z(m_bs), z(m_bs)
        s = torch.cuda.Stream()
        dvl = lambda: dsv.dvl_allocate_pack(lg, nl, tok, pos, ref, k, cu, pt, pp, pr, stream=s)
        pred = lambda: dsv.predictor_forward(feats, nl, w1, b1, w2, b2, lg, workspace=ws_pred,
                                             stream=s)
        both = lambda: (pred(), dvl())
        res = {}
        for name, fn in (("dvl", dvl), ("predictor", pred), ("predictor_then_dvl", both)):
            for _ in range(10):
                fn()
            torch.cuda.synchronize()
            g = dsv.Graph().capture(lambda: [fn() for _ in range(launches)], s)
            g.replay(s)
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(s)
            for _ in range(replays):
                g.replay(s)
            e1.record(s)
            torch.cuda.synchronize()
            g.close()
            res[name + "_us"] = round(e0.elapsed_time(e1) * 1e3 / (launches * replays), 2)
        nbytes = n_bs * (w - 1) * 4 + 3 * m_bs * 4 + 8 + (2 * n_bs + 1) * 4 + 3 * m_bs * 4
        res["dvl_algorithmic_bytes"] = nbytes
        out["n_bs_%d" % n_bs] = res
    out["bound"] = "latency (one workgroup for DVL; K-split tiles for the predictor)"
    out["timing"] = "%d launches in one hipGraph, %d replays, HIP events" % (launches, replays)
    return out


def bucket_bench(layers=4, reps=5):
    """The multi-bucket capture set (Sec. III-D, Alg. 2, Eqs. (13)-(15)):
    buckets {8, 16, 32, 64} sharing one attention and one acceptance
    workspace, each with a captured decision graph (predictor + DVL) and
    verify graph
    (``layers`` attention layers, Qwen3-8B shape, then acceptance over
    151,936 tokens).  Per bucket, at N = N_bs and at N = 3 N_bs / 4 (the rest
    sentinels): decision and verify replay times (HIP events on the replay
    stream, mean of ``reps`` steps; staging outside the timed region), plus
    the set's device memory.  Contexts U[1024, 8192] as in the workload."""
    import torch

    import paper_2609_37532_amd as dsv
    import workloads as W

    sizes = (8, 16, 32, 64)
    rng = np.random.default_rng(W.SEED_BASE + 80)
    hq, hkv, d, V = 32, 8, 128, 151936
    ctx_lo, ctx_hi = 1024, 8192
    pool = max(sizes)
    max_kv_len = ctx_hi + W.BLOCK_WIDTH
    max_pages = -(-max_kv_len // W.PAGE_SIZE)
    num_pages = pool * max_pages
    cache_map = rng.permutation(num_pages).astype(np.int32).reshape(pool, max_pages)
    ctx_all = rng.integers(ctx_lo, ctx_hi + 1, size=pool).astype(np.int32)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(W.SEED_BASE + 81)
    kv = [torch.randn((num_pages, 2, hkv, W.PAGE_SIZE * d), generator=gen, device="cuda",
                      dtype=torch.bfloat16) for _ in range(layers)]
    p0 = W.make_predictor_inputs(rng, n_bs=pool, n_live=pool)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
    pred = dict(w1=t(p0.w1), b1=t(p0.b1), w2=t(p0.w2), b2=t(p0.b2))
    bs = dsv.BucketSet(sizes, kv_pools=kv, max_pages=max_pages, max_kv_len=max_kv_len,
                       num_q_heads=hq, head_dim=d, vocab=V, predictor=pred)
    s = torch.cuda.Stream()
    bs.capture(s)
    rows = []
    for b in sizes:
        bk = bs[b]
        bk.q.normal_(generator=gen)
        bk.logits.normal_(generator=gen)
        for n in (b, 3 * b // 4):
            t_dec, t_ver, kv_tokens = [], [], 0
            for _ in range(reps):
                reqs = np.sort(rng.choice(pool, size=n, replace=False))
                dv = W.make_dvl_inputs(rng, n_bs=b, n_live=n)
                feats = W.make_predictor_inputs(rng, n_bs=b, n_live=n).features
                bk.stage_decision(n, feats, dv.tokens, dv.positions, dv.kv_refs)
                bk.stage_verify(n, ctx_all[reqs], cache_map[reqs])
                torch.cuda.synchronize()
                ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
                ev[0].record(s)
                bk.graph_dec.replay(s)
                ev[1].record(s)
                bk.graph_ver.replay(s)
                ev[2].record(s)
                torch.cuda.synchronize()
                t_dec.append(ev[0].elapsed_time(ev[1]))
                t_ver.append(ev[1].elapsed_time(ev[2]))
                kv_tokens += int(ctx_all[reqs].sum()) + 8 * n
            ver_ms = float(np.mean(t_ver))
            rows.append({"n_bs": b, "live": n, "capacity_rows": 8 * b,
                         "decision_replay_us": round(float(np.mean(t_dec)) * 1e3, 2),
                         "verify_replay_us": round(ver_ms * 1e3, 2),
                         "verify_us_per_layer_incl_accept": round(ver_ms * 1e3 / layers, 2),
                         "packed_tokens_per_s": round(8 * n / (ver_ms * 1e-3), 1),
                         "kv_gbps": round(kv_tokens / reps * hkv * d * 4 * layers
                                          / (ver_ms * 1e-3) / 1e9, 1)})
    mem = bs.memory()
    bs.close()
    del kv
    torch.cuda.empty_cache()
    return {"workload": "%d layers of Qwen3-8B-shape verify attention + acceptance over "
                        "151936 tokens per bucket; DVL lengths fill 8 rows per live request"
                        % layers,
            "steps": rows, "memory": mem["total"],
            "memory_per_bucket": [{k: m[k] for k in ("n_bs", "metadata_bytes",
                                                     "activation_bytes",
                                                     "graph_decision_bytes",
                                                     "graph_verify_bytes")}
                                  for m in mem["buckets"]]}


READ_PROBE_GRIDS = (512, 1024, 2048, 4096)


def read_ceiling(stream, pool_gib=4, reps=10):
    """The read rate scattered 4 KiB page tiles reach on this device, the
    ceiling the attention kernel is compared with beside the vendor peak.
    ``read_probe`` reads every tile of a 4 GiB pool once per launch in a
    seeded random order, alternating between two pools so that no launch
    finds the previous one's tiles in the 256 MB Infinity Cache; HIP events
    bracket ``reps`` launches per grid size, and the best grid is reported.
    Three orders: random tiles, random 64 KiB pages with their tiles in
    sequence, and address order.  ``peak_gbps`` is the highest of the three,
    the measured read peak."""
    import torch

    import paper_2609_37532_amd as dsv
    import workloads as W
    dev = torch.device("cuda", 0)
    n_tiles = pool_gib << 18
    nbytes = n_tiles * 4096
    pools = [torch.empty(nbytes, dtype=torch.uint8, device=dev) for _ in range(2)]
    for k, pool in enumerate(pools):
        pool.fill_(0x3c + k)
    gen = torch.Generator()
    gen.manual_seed(W.SEED_BASE + 77)
    pages = torch.randperm(n_tiles // 16, generator=gen).to(torch.int32)
    orders = {
        # every 4 KiB tile in a random order
        "random_tiles": torch.randperm(n_tiles, generator=gen).to(torch.int32).to(dev),
        # 64 KiB pages (16 tiles, one page of all eight KV heads' K or V) in a
        # random order, the tiles of a page one after another
        "random_pages": (pages[:, None] * 16 + torch.arange(16, dtype=torch.int32)).reshape(-1)
        .to(dev),
        "address_order": torch.arange(n_tiles, dtype=torch.int32, device=dev),
    }
    out = {"pool_bytes": nbytes, "tile_bytes": 4096, "kernel": "read_probe_kernel",
           "timing": "HIP events around %d launches per grid size, two pools alternating" % reps}
    with torch.cuda.stream(stream):
        for name, order in orders.items():
            per_grid = {}
            for grid in READ_PROBE_GRIDS:
                sink = torch.empty(grid, dtype=torch.int32, device=dev)
                for r in range(2):
                    dsv.read_probe(pools[r % 2], order, sink, stream=stream)
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                for r in range(reps):
                    dsv.read_probe(pools[r % 2], order, sink, stream=stream)
                e1.record(stream)
                torch.cuda.synchronize()
                per_grid[str(grid)] = round(nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)
            best = max(per_grid, key=per_grid.get)
            out[name] = {"gbps": per_grid[best], "grid": int(best), "per_grid_gbps": per_grid}
    out["peak_gbps"] = max(out[name]["gbps"] for name in orders)
    del pools, orders
    torch.cuda.empty_cache()
    return out


def copy_probe():
    """Three device-to-device copies of 1 GiB: reads and writes 2^30 bytes
    each, the known size against which FETCH_SIZE / WRITE_SIZE are scaled."""
    import torch
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda")
    src.fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n, "copies": 3}), flush=True)


def eager_attention(cfg, launches):
    """``launches`` eager verify-attention launches of one shape, each after a
    512 MB scrub (so the KV comes from HBM), for hardware-counter passes.
    cfg 2-4: the attention configs; 5: one layer of the stress run's first
    step (B=32, contexts U[512, 4096], verify lengths of that step)."""
    import torch

    import paper_2609_37532_amd as dsv
    import workloads as W
    dev = "cuda"
    if cfg == 5:
        plan = W.StressPlan(steps=1)
        st = plan.draw_step()
        gen = torch.Generator(device=dev)
        gen.manual_seed(W.SEED_BASE + 5)
        hq, hkv, d = 32, 8, 128
        kv = torch.randn((plan.num_pages, 2, hkv, W.PAGE_SIZE * d), generator=gen, device=dev,
                         dtype=torch.bfloat16)
        q = torch.randn((plan.capacity, hq, d), generator=gen, device=dev, dtype=torch.bfloat16)
        cu = torch.from_numpy(st.cu_qlens).to(dev)
        ctx = torch.from_numpy(plan.ctx0.astype(np.int32)).to(dev)
        pt = torch.from_numpy(plan.page_table).to(dev)
        max_kv_len, scale = plan.max_kv_len, 1.0 / np.sqrt(d)
    else:
        a = W.config_attn_inputs(cfg)
        bf = lambda x: torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).to(dev).view(
            torch.bfloat16)
        i32 = lambda x: torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(dev)
        q, kv = bf(a.q), bf(a.kv_pages)
        cu, pt, ctx = i32(a.cu_qlens), i32(a.page_table), i32(a.ctx_lens)
        max_kv_len, scale = a.max_kv_len, a.scale
    out = torch.zeros_like(q)
    dims = dsv.attn_dims(q, kv, pt, max_kv_len=max_kv_len, scale=scale)
    ws = dsv.alloc_workspace(dsv.verify_attn_workspace_bytes(dims), dev)
    scrub = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    for r in range(launches):
        scrub.fill_(r & 0xFF)
        dsv.verify_attn(q, cu, kv, pt, ctx, out, dims=dims, workspace=ws)
    torch.cuda.synchronize()
    print(json.dumps({"eager_attention_config": cfg, "launches": launches}), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(requested --gpus %d, WORLD_SIZE %d)" % (args.gpus, world), flush=True)
        sys.exit(2)

    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_probe:
        copy_probe()
        return

    import paper_2609_37532_amd as dsv
    import workloads as W

    dev = torch.device("cuda", 0)
    if args.eager_only and args.eager_attention:
        eager_attention(args.eager_attention, args.eager_only)
        return
    t0 = time.time()
    rng = W.config_rng(CONFIG_INDEX)
    attn = W.config_attn_inputs(CONFIG_INDEX, rng=rng)
    acc = W.config_accept_inputs(CONFIG_INDEX, attn.cu_qlens, rng)
    log("inputs generated in %.1f s: B=%d, sum k=%d, %d pages"
        % (time.time() - t0, attn.num_reqs, int(attn.qlens.sum()), attn.num_pages))

    def bf16(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(
            torch.bfloat16)

    def i32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)

    q, kv = bf16(attn.q), bf16(attn.kv_pages)
    cu, pt, ctx = i32(attn.cu_qlens), i32(attn.page_table), i32(attn.ctx_lens)
    out = torch.zeros_like(q)
    logits = bf16(acc.logits)
    draft = i32(acc.draft_tokens)
    a_len = torch.zeros(attn.num_reqs, dtype=torch.int32, device=dev)
    nxt = torch.zeros_like(a_len)
    dims = dsv.attn_dims(q, kv, pt, max_kv_len=attn.max_kv_len, scale=attn.scale)
    ws_attn = dsv.alloc_workspace(dsv.verify_attn_workspace_bytes(dims), dev)
    ws_acc = dsv.alloc_workspace(
        dsv.accept_workspace_bytes(acc.capacity, acc.num_reqs, acc.vocab), dev)
    stream = torch.cuda.Stream(device=dev)

    def step_on(s):
        dsv.verify_attn(q, cu, kv, pt, ctx, out, dims=dims, workspace=ws_attn, stream=s)
        dsv.accept(logits, cu, draft, a_len, nxt, workspace=ws_acc, stream=s)

    torch.cuda.synchronize()
    if args.eager_only:
        for _ in range(args.eager_only):
            step_on(stream)
        torch.cuda.synchronize()
        print(json.dumps({"eager_steps": args.eager_only}), flush=True)
        return
    step_on(stream)  # eager run once before capture
    torch.cuda.synchronize()
    graph = dsv.Graph().capture(lambda: step_on(stream), stream)
    log("graph captured")

    # ---- timed region: K graph replays of the whole step
    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            graph.replay(stream)
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for _ in range(args.steps):
            graph.replay(stream)
        ev1.record(stream)
        torch.cuda.synchronize()
    ms_step = ev0.elapsed_time(ev1) / args.steps
    tokens = int(attn.qlens.sum())
    value = tokens / (ms_step / 1e3)
    log("step %.1f us, %.0f tokens/s" % (ms_step * 1e3, value))

    # ---- kernel durations: HIP events around each kernel on its stream
    n_timed = max(args.steps, 200)
    for _ in range(3):
        step_on(stream)
    torch.cuda.synchronize()
    timer = dsv.KernelTimer(max_launches=4 * n_timed + 16)
    with timer:
        for _ in range(n_timed):
            step_on(stream)
        torch.cuda.synchronize()
    t_split = timer.median_ms("attn_split") * 1e-3
    t_comb = timer.median_ms("attn_combine") * 1e-3 if timer.count("attn_combine") else 0.0
    t_argmax = timer.median_ms("accept_argmax") * 1e-3
    t_prefix = timer.median_ms("accept_prefix") * 1e-3
    t_split_mean = timer.mean_ms("attn_split") * 1e-3

    hq, hkv, d = attn.num_q_heads, attn.num_kv_heads, attn.head_dim
    b_attn = attention_bytes(attn, hkv, hq, d)
    b_acc = accept_bytes(acc, 2)
    f_attn = attention_flops(attn, hq, d)
    achieved = b_attn / t_split / 1e9
    traffic = counters_traffic(b_attn)
    a_gbps = b_acc / t_argmax / 1e9

    result = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": UNIT,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; Qwen3-8B attention shapes, no weights)",
        "config": {
            "workload": "verify attention (1 layer) + greedy acceptance, Qwen3-8B shape, "
                        "B=32, 32q/8kv heads, head_dim 128, page 16, ctx U[1024,8192], "
                        "verify lengths 1..16 (geometric p=0.25) packed in capacity 256, "
                        "bf16 logits [256 x 151936]",
            "global_batch": attn.num_reqs,
            "packed_tokens": tokens,
            "kv_tokens": int((attn.ctx_lens + attn.qlens).sum()),
            "capacity": attn.capacity,
            "step": "one hipGraph replay: attn stream-K + combine + argmax + prefix",
            "row_padding_eq2": row_padding(attn.qlens, hq // hkv),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "attn_streamk_kernel<128>",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "algorithmic_bytes": b_attn,
            "launch_us": round(t_split * 1e6, 2),
            "launch_us_mean": round(t_split_mean * 1e6, 2),
            "timing": "timing-only HIP events (hipEventDisableSystemFence) around each "
                      "launch on its stream; median of %d launches" % timer.count("attn_split"),
            # the same bytes over whole operations, not the dominant kernel alone
            "attention_op_frac": round(b_attn / (t_split + t_comb) / 1e9 / HBM_PEAK_GBPS, 4),
            "acceptance_op_frac": round(b_acc / (t_argmax + t_prefix) / 1e9 / HBM_PEAK_GBPS, 4),
            "step_frac": round((b_attn + b_acc) / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
        },
        "operations": {
            "attention": {"kernels": "attn_streamk_kernel + attn_combine_kernel",
                          "us": round((t_split + t_comb) * 1e6, 2),
                          "algorithmic_bytes": b_attn,
                          "gbps": round(b_attn / (t_split + t_comb) / 1e9, 1),
                          "frac": round(b_attn / (t_split + t_comb) / 1e9 / HBM_PEAK_GBPS, 4)},
            "acceptance": {"kernels": "argmax_chunk_kernel + prefix_kernel",
                           "us": round((t_argmax + t_prefix) * 1e6, 2),
                           "algorithmic_bytes": b_acc,
                           "gbps": round(b_acc / (t_argmax + t_prefix) / 1e9, 1),
                           "frac": round(b_acc / (t_argmax + t_prefix) / 1e9 / HBM_PEAK_GBPS, 4)},
            "step": {"what": "one graph replay of all four kernels (ms_per_step)",
                     "us": round(ms_step * 1e3, 2), "algorithmic_bytes": b_attn + b_acc,
                     "gbps": round((b_attn + b_acc) / (ms_step * 1e-3) / 1e9, 1),
                     "frac": round((b_attn + b_acc) / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)},
        },
        "us_per_layer_attention": round((t_split + t_comb) * 1e6, 2),
        "attention_gbps": round(b_attn / (t_split + t_comb) / 1e9, 1),
        "attention_tflops": round(f_attn / (t_split + t_comb) / 1e12, 2),
        "accept": {"argmax_us": round(t_argmax * 1e6, 2), "prefix_us": round(t_prefix * 1e6, 2),
                   "algorithmic_bytes": b_acc, "argmax_gbps": round(a_gbps, 1),
                   "argmax_frac": round(a_gbps / HBM_PEAK_GBPS, 4),
                   "op_frac": round(b_acc / (t_argmax + t_prefix) / 1e9 / HBM_PEAK_GBPS, 4)},
        "combine_us": round(t_comb * 1e6, 2),
    }
    graph.close()

    log("read ceiling ...")
    ceiling = read_ceiling(stream)
    result["read_ceiling"] = ceiling
    result["roofline"]["measured_read_peak"] = ceiling["peak_gbps"]
    result["roofline"]["frac_of_measured_peak"] = round(achieved / ceiling["peak_gbps"], 4)

    log("configs 2-4 attention ...")
    result["attention_configs"] = configs_bench()
    if args.no_next:
        finish(args, result, attn, acc, torch)
        return
    # ---- the stochastic verifier (T = 1) on the same logits and offsets
    gen = torch.Generator(device=dev)
    gen.manual_seed(W.SEED_BASE + 90)
    uni = torch.rand((acc.capacity, 2), generator=gen, device=dev, dtype=torch.float32)
    ws_smp = dsv.alloc_workspace(
        dsv.accept_stochastic_workspace_bytes(acc.capacity, acc.num_reqs, acc.vocab), dev)
    smp = lambda: dsv.accept_stochastic(logits, cu, draft, uni, 1.0, a_len, nxt,
                                        workspace=ws_smp, stream=stream)
    for _ in range(3):
        smp()
    torch.cuda.synchronize()
    timer = dsv.KernelTimer(max_launches=2 * n_timed + 8)
    with timer:
        for _ in range(n_timed):
            smp()
        torch.cuda.synchronize()
    t_stats = timer.median_ms("sample_stats") * 1e-3
    t_draw = timer.median_ms("sample_draw") * 1e-3
    s_gbps = b_acc / t_stats / 1e9
    result["stochastic_accept"] = {
        "temperature": 1.0, "stats_us": round(t_stats * 1e6, 2),
        "draw_us": round(t_draw * 1e6, 2), "algorithmic_bytes": b_acc,
        "stats_gbps": round(s_gbps, 1), "stats_frac": round(s_gbps / HBM_PEAK_GBPS, 4),
        "timing": "timing-only HIP events around each launch, median of %d launches"
                  % timer.count("sample_stats")}

    del q, kv, logits, out
    torch.cuda.empty_cache()
    log("DVL allocate-and-pack ...")
    result["dvl"] = dvl_bench()
    log("bucket set ...")
    result["buckets"] = bucket_bench()
    finish(args, result, attn, acc, torch)


def finish(args, result, attn, acc, torch):
    """The stress run and the CPU baseline, then the JSON line."""
    torch.cuda.empty_cache()
    if not args.no_stress:
        log("stress run (36 layers, %d steps) ..." % args.stress_steps)
        result["stress"] = stress_bench(args.stress_steps)
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        result["cpu_baseline"], result["cpu_baseline_single_thread"] = cpu_baseline(
            attn, acc, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
