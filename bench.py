"""Throughput of the MoE-layer hot path on one MI355X.

One step = one pass of the whole path over one scheduling unit of the
Mixtral-8x7B-shaped layer (H 4096, 8 experts of SwiGLU width 14336, top-2):
two adjacent batches of T = 4096 tokens (8192 tokens) with 32-layer predicted
routes are rebatched by the token scheduler (moe_schedule), gated in one
launch (moe_route), and each new batch is grouped by expert (moe_permute), run
through its resident experts (moe_expert_ffn; all 8 resident) and combined
(moe_combine). Inputs are seeded synthetic data already resident in HBM; no
allocation happens inside the timed region.

Prints one JSON line (see the keys below). --gpus N > 1 is refused: this path
runs on one GPU.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/sec + grouped-FFN MFMA % of peak (bf16, Mixtral-shape)"
PEAK_BF16_TFLOPS = 2516.6      # MI355X dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 flop/clk
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--seed", type=int, default=2)
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="CPU budget of the oracle baseline sample (0 = skip)")
    p.add_argument("--copy-probe-mib", type=int, default=0,
                   help="after timing, run one plain device copy of this many MiB "
                        "(the calibration kernel of a counter run)")
    p.add_argument("--ece", action="store_true",
                   help="instead of the layer throughput, measure the expert cache engine: "
                        "a Qwen-shaped layer with 32 of 60 experts resident, misses loaded "
                        "from pinned host memory while the resident experts compute, and "
                        "PLEC against per-layer LRU hit ratios on synthetic predicted routes")
    p.add_argument("--decode-ts", action="store_true",
                   help="instead of the layer throughput, run decode-sized two-batch units "
                        "through the Qwen-shaped layer in input order and as the token "
                        "scheduler splits them")
    p.add_argument("--decode", action="store_true",
                   help="instead of the layer throughput, measure decode-sized batches of the "
                        "Mixtral-shaped layer (4 to 256 tokens, all 8 experts resident): "
                        "per-stage times and the expert weights' read bandwidth")
    p.add_argument("--ways", action="store_true",
                   help="instead of the layer throughput, measure B-way rebatching by "
                        "recursive bisection (B = 2 to 64 batches of 64 tokens, Qwen-shaped "
                        "24-layer predicted routes): time and active (layer, expert) pairs")
    p.add_argument("--stack", action="store_true",
                   help="instead of the one-layer throughput, run the dual-batch pipeline over "
                        "the 32-layer Mixtral-shaped stack (8192-token units, KV caches merged "
                        "and reindexed) with and without the scheduling stream overlapped")
    p.add_argument("--stack-layers", type=int, default=32)
    p.add_argument("--stack-units", type=int, default=3)
    p.add_argument("--stack-predictor", action="store_true",
                   help="with --stack: units carry token ids (16 sequences of 512) and each "
                        "unit's plan runs the routing path predictor (hidden 32, FFN 2048, "
                        "random weights) and the per-layer top-2 of its logits before the "
                        "token scheduler")
    p.add_argument("--rpp", action="store_true",
                   help="instead of the layer throughput, time the routing path predictor's "
                        "forward pass (16 sequences of 512 tokens, hidden 32, FFN 2048, random "
                        "weights) with Mixtral-shaped and Qwen-shaped heads")
    p.add_argument("--sched-sweep", action="store_true",
                   help="instead of the layer throughput, time the two-way token scheduler on "
                        "Mixtral-shaped 32-layer predicted routes from 1024 to 2^20 tokens: "
                        "us per call, Eq. 2 before and after, effective GB/s")
    p.add_argument("--route-grouped", action="store_true",
                   help="instead of the all-resident Mixtral-shaped layer, time the route-grouped "
                        "one: 8192 tokens scheduled into two batches by 32-layer predicted "
                        "routes, 4 of 8 experts resident per batch, misses flagged")
    p.add_argument("--qwen", action="store_true",
                   help="instead of the Mixtral-shaped layer, time the Qwen1.5-MoE-shaped one: "
                        "8192 tokens, 60 experts with a Zipf-skewed router, 32 resident, four "
                        "shared experts; the FFN also split at the ridge (315 rows)")
    p.add_argument("--deepseek", action="store_true",
                   help="instead of the Mixtral-shaped layer, time the DeepSeek-V2-Lite-shaped "
                        "one: 32768 tokens scheduled into two batches by 26-layer predicted "
                        "routes, 48 of 64 experts resident per batch, two shared experts")
    p.add_argument("--plec", action="store_true",
                   help="instead of the layer throughput, run batches through a stack of "
                        "Qwen-shaped MoE layers whose experts live in pinned host memory and a "
                        "device cache managed by PLEC with real-time correction; hit ratio "
                        "against per-layer LRU caches of the same total size")
    p.add_argument("--plec-cache", type=int, default=16,
                   help="with --plec: cache slots per layer (the LRU capacity; PLEC gets "
                        "layers x this many slots shared by all layers)")
    p.add_argument("--plec-batch", type=int, default=16,
                   help="with --plec: tokens per batch")
    p.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                   help="summarise two rocprofv3 counter_collection.csv files (FETCH_SIZE, "
                        "WRITE_SIZE) of a --copy-probe-mib run into the traffic file, then exit")
    return p.parse_args()


# HBM traffic of moe_expert_ffn, measured by counters on this workload; used
# only while the FFN source is the one the counters were taken on.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "expert_ffn_mixtral_T4096_traffic.txt")
FFN_SOURCE = os.path.join(ROOT, "paper_2410_17954_amd", "csrc", "ffn.hip")
FFN_KERNELS = ("ffn_tiles_kernel", "ffn_gemm_bf16_fast<0>", "ffn_gemm_bf16_fast<1>")


def ffn_source_digest():
    import hashlib
    with open(FFN_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def pmc_summary(fetch_csv, write_csv, copy_mib):
    """Per-launch HBM bytes of moe_expert_ffn from FETCH_SIZE and WRITE_SIZE
    (KiB per dispatch), each scaled by the ratio of true bytes to counter for
    the plain copy of copy_mib MiB in the same run."""
    import csv
    copy_bytes = copy_mib * 2**20

    def per_kernel(path, counter):
        acc = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            acc.setdefault(name, []).append(float(r["Counter_Value"]) * 1024.0)
        return acc

    out = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        acc = per_kernel(path, counter)
        copies = [max(v) for n, v in acc.items() if "copyBuffer" in n]
        probe = max(copies)
        factor = copy_bytes / probe
        ffn = 0.0
        for k in FFN_KERNELS:
            vals = [v for n, v in acc.items() if k in n]
            if not vals:
                raise SystemExit(f"no {k} dispatch in {path}")
            ffn += float(np.mean(vals[0])) * factor
        out[counter] = {"bytes_per_launch": ffn, "copy_probe_counter_bytes": probe,
                        "factor": factor}
    return out



def ece_report(args):
    """Expert cache engine measurement (one JSON line)."""
    import torch
    from paper_2410_17954_amd import ece, ops, synth

    dev = torch.device("cuda:0")
    cfg = synth.workload("qwen15_moe_layer")
    T, H, E, F, k, S = cfg["T"], cfg["H"], cfg["E"], cfg["F"], cfg["k"], cfg["S"]
    inp = synth.layer_inputs(cfg, args.seed, T=T, parts=("x", "router", "experts", "bias"))

    def up(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    def pinned(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).pin_memory()

    x = up(inp["x"])
    idx, gw, _ = ops.route(x, up(inp["w_router"]), k, bias=up(inp["bias"]))
    store = tuple(pinned(inp[n]) for n in ("w_gate", "w_up", "w_down"))
    # the prediction: each routed choice kept with probability 0.9, else
    # another expert; the resident set is its top S (PLEC's per-layer rule)
    g = np.random.default_rng(args.seed)
    act = idx.cpu().numpy()
    pred = np.where(g.random(act.shape) < 0.9, act, g.integers(0, E, size=act.shape))
    slot = ops.plan_slots(np.bincount(pred.ravel(), minlength=E), S)
    counts = np.bincount(act.ravel(), minlength=E)
    spare = 16                                   # slots beyond the resident set for corrections
    cache = tuple(torch.empty((S + spare,) + tuple(t.shape[1:]), dtype=torch.bfloat16, device=dev)
                  for t in store)
    res = [e for e in range(E) if slot[e] >= 0]
    misses = [e for e in range(E) if slot[e] < 0 and counts[e] > 0]
    ws = {"permute": ops.workspace_tensor(ops.permute_workspace(T, k, E), dev),
          "ffn": ops.workspace_tensor(ops.expert_ffn_workspace(T * k, H, F, E), dev)}
    y = torch.zeros((T, H), dtype=torch.bfloat16, device=dev)

    def reload():
        ops.load_experts(store, cache, res, slot[res])
        torch.cuda.synchronize()

    def timed(fn, n=7):
        reload()
        fn()                                     # warm-up (first use of the pinned pages, launches)
        torch.cuda.synchronize()
        out = []
        for _ in range(n):
            reload()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            out.append(e0.elapsed_time(e1))
        return float(np.median(out))

    # resident experts only (the misses stay missing)
    def resident_only():
        offs, rop, _, xp = ops.permute(x, idx, E, workspace=ws["permute"])
        yp = ops.expert_ffn(xp, offs, *cache, slot_of_expert=torch.from_numpy(slot).to(dev),
                            workspace=ws["ffn"])
        ops.combine(yp, idx, gw, rop, slot_of_expert=torch.from_numpy(slot).to(dev), y=y)

    def copies_only():
        for i in range(0, len(misses), spare):
            ops.load_experts(store, cache, misses[i:i + spare], list(range(S, S + len(misses[i:i + spare]))))

    slot_sp = slot.copy()
    def corrected():
        ece.run_layer(x, idx, gw, E, store, cache, slot_sp, y=y, workspaces=ws)

    t_res = timed(resident_only)
    t_copy = timed(copies_only)
    t_corr = timed(corrected)
    expert_bytes = 3 * H * F * 2
    miss_pairs = int(sum(counts[e] for e in misses))

    # hit ratios (Fig. 10's comparison, synthetic Switch-32-like routes)
    hit = []
    for bs in (4, 8, 16):
        for cs in (8, 16):
            L32, E32, B = 6, 32, 40
            act_r, pred_r = synth.predicted_and_actual_routes(B * bs, L32, E32, 1, 0.7, 1.1, 0.9,
                                                              seed=args.seed)
            def demand(r):
                d = np.zeros((L32, E32), np.int64)
                for l in range(L32):
                    np.add.at(d[l], r[:, l, 0].astype(np.int64), 1)
                return d
            ph = pn = 0
            acts = []
            for b in range(B):
                sl = slice(b * bs, (b + 1) * bs)
                a, p_ = demand(act_r[sl]), demand(pred_r[sl])
                acts.append(a)
                r = ops.plec_run(p_, a, cs * L32)
                ph += int(r["hits"].sum())
                pn += int(r["needed"].sum())
            lh, ln = ops.lru_run(np.stack(acts), cs)
            hit.append({"batch": bs, "cache_per_layer": cs, "plec": round(ph / pn, 4),
                        "lru": round(lh / ln, 4)})
    rec = {
        "metric": "expert cache engine: corrected-layer time, copy/compute overlap, hit ratios",
        "config": {"workload": f"Qwen1.5-MoE-shaped layer: T={T}, H={H}, E={E}, F={F}, top-{k}, "
                               f"{S} resident slots from a 0.9-accurate prediction, "
                               f"{len(misses)} missed experts ({miss_pairs} of {T * k} pairs)",
                   "store": "pinned host memory"},
        "resident_only_ms": round(t_res, 3),
        "miss_copies_ms": round(t_copy, 3),
        "miss_copy_GBps": round(len(misses) * expert_bytes / (t_copy * 1e-3) / 1e9, 1),
        "corrected_layer_ms": round(t_corr, 3),
        "overlap_ms": round(t_res + t_copy - t_corr, 3),
        "overlap_ideal_ms": round(min(t_res, t_copy), 3),
        "hit_ratio_synthetic_switch32": hit,
        "data": "synthetic",
    }
    print(json.dumps(rec))


def decode_report(args):
    """Decode-sized batches through route, permute, expert FFN and combine (one
    JSON line). The 2.8 GB of expert weights do not fit the 256 MB last-level
    cache, so each step reads them from HBM; a 512 MB fill before every step
    makes sure of it."""
    import torch
    from paper_2410_17954_amd import ops, synth

    dev = torch.device("cuda:0")
    cfg = synth.workload("mixtral8x7b_layer")
    H, E, F, k = cfg["H"], cfg["E"], cfg["F"], cfg["k"]
    Tmax = 256
    inp = synth.layer_inputs(cfg, args.seed, T=Tmax, parts=("x", "router", "experts"))

    def up(a):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)

    wr = up(inp["w_router"])
    wg, wu, wd = (up(inp[n]) for n in ("w_gate", "w_up", "w_down"))
    flush = torch.empty(512 * 2 ** 20 // 4, dtype=torch.float32, device=dev)
    out = []
    for T in (4, 16, 64, 128, 256):
        x = up(inp["x"][:T])
        ws_p = ops.workspace_tensor(ops.permute_workspace(T, k, E), dev)
        ws_f = ops.workspace_tensor(ops.expert_ffn_workspace(T * k, H, F, E), dev)
        idx = torch.empty((T, k), dtype=torch.int32, device=dev)
        gw = torch.empty((T, k), dtype=torch.float32, device=dev)
        offs = torch.empty(E + 1, dtype=torch.int32, device=dev)
        rop = torch.empty(T * k, dtype=torch.int32, device=dev)
        por = torch.empty(T * k, dtype=torch.int32, device=dev)
        xp = torch.empty((T * k, H), dtype=torch.bfloat16, device=dev)
        yp = torch.empty_like(xp)
        y = torch.empty_like(x)
        inc = torch.empty(T, dtype=torch.int32, device=dev)

        def step(ev):
            ev[0].record()
            ops.route(x, wr, k, topk_idx=idx, topk_w=gw)
            ev[1].record()
            ops.permute(x, idx, E, expert_offsets=offs, row_of_pair=rop, pair_of_row=por,
                        x_perm=xp, workspace=ws_p)
            ev[2].record()
            ops.expert_ffn(xp, offs, wg, wu, wd, y_perm=yp, workspace=ws_f)
            ev[3].record()
            ops.combine(yp, idx, gw, rop, y=y, incomplete=inc)
            ev[4].record()

        times = []
        for rep in range(args.warmup + 7):
            flush.fill_(float(rep))
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
            # the launches queue behind a short wait so that host time is not counted
            torch.cuda._sleep(1000000)
            step(ev)
            torch.cuda.synchronize()
            if rep >= args.warmup:
                times.append([ev[i].elapsed_time(ev[i + 1]) for i in range(4)])
        med = np.median(np.array(times), axis=0)
        counts = np.bincount(idx.cpu().numpy().ravel(), minlength=E)
        wbytes = int((counts > 0).sum()) * 3 * H * F * 2
        out.append({"tokens": T, "max_rows_per_expert": int(counts.max()),
                    "experts_used": int((counts > 0).sum()),
                    "route_ms": round(float(med[0]), 4), "permute_ms": round(float(med[1]), 4),
                    "ffn_ms": round(float(med[2]), 4), "combine_ms": round(float(med[3]), 4),
                    "step_ms": round(float(med.sum()), 4),
                    "ffn_weight_GBps": round(wbytes / (float(med[2]) * 1e-3) / 1e9, 1),
                    "ffn_hbm_frac": round(wbytes / (float(med[2]) * 1e-3) / 1e9 / PEAK_HBM_GBS, 3)})
    rec = {"metric": "decode-sized MoE-layer steps: stage times and expert-weight read bandwidth",
           "config": {"workload": f"Mixtral-8x7B-shaped layer: H={H}, E={E}, F={F}, top-{k}, "
                                  "all experts resident, weights read from HBM every step"},
           "steps": out, "data": "synthetic"}
    print(json.dumps(rec))


def decode_ts_report(args):
    """The token scheduler on decode-sized scheduling units (Sec. 3.3): two
    batches of B tokens whose predicted routes over L = 24 Qwen-shaped layers
    carry topic structure (two topics, each token on its own topic's Markov
    chain), run through all 24 layers (60 experts, top-4, every expert
    resident; shared experts and attention left out: their cost does not
    depend on the batching), once in input order and once as the scheduler
    splits the unit. Layer l has its own router, and its gating is boosted by
    4 towards the token's predicted layer-l route, so the experts a batch
    activates at each layer are the ones Eq. 2 counts. Expert weights cycle
    through 8 distinct sets (8.3 GB), so every layer reads its experts from
    HBM. Per order: Eq. 2 (active (layer, expert) pairs summed over the
    batches), the expert-weight bytes read, and the time of the two batches
    through the layers (moe_permute + moe_expert_ffn + moe_combine per layer
    and batch; routing is the same per token in both orders and is done
    beforehand), HIP events, median of 5 after warm-up, a 512 MB fill before
    each run; for the scheduled order also moe_schedule. One JSON line."""
    import torch
    from paper_2410_17954_amd import ops, synth

    dev = torch.device("cuda:0")
    cfg = synth.workload("qwen15_moe_layer")
    H, E, F, k, L = cfg["H"], cfg["E"], cfg["F"], cfg["k"], cfg["L"]
    topics, boost, n_sets = 2, 4.0, 8
    Bmax = 64
    g = torch.Generator(device=dev)
    g.manual_seed(args.seed)

    def normal(shape, std):
        return (torch.randn(shape, generator=g, device=dev) * std).to(torch.bfloat16)

    sets = [(normal((E, F, H), 0.02), normal((E, F, H), 0.02), normal((E, H, F), 0.02))
            for _ in range(n_sets)]
    routers = [normal((E, H), 0.02) for _ in range(L)]
    x_all = normal((2 * Bmax, H), 1.0)
    flush = torch.empty(512 * 2 ** 20 // 4, dtype=torch.float32, device=dev)
    wbytes_expert = 3 * H * F * 2
    out = []
    for B in (8, 16, 32, 64):
        N = 2 * B
        routes = synth.topic_routes(N, L, E, k, cfg["keep"], cfg["zipf"], topics, args.seed + B)
        x = x_all[:N].contiguous()
        rt = torch.from_numpy(np.ascontiguousarray(routes, dtype=np.uint8)).to(dev)
        idx_l, gw_l = [], []
        for l in range(L):
            bias = torch.from_numpy(synth.route_boost_bias(routes, l, E, boost)).to(dev)
            i_, w_, _ = ops.route(x, routers[l], k, bias=bias)
            idx_l.append(i_)
            gw_l.append(w_)
        idx_host = [i_.cpu().numpy() for i_ in idx_l]
        ws_s = ops.workspace_tensor(ops.schedule_workspace(N, L, E, k), dev)
        perm = torch.empty(N, dtype=torch.int32, device=dev)
        demand = torch.empty((2, L, E), dtype=torch.int32, device=dev)
        info = torch.empty(8, dtype=torch.int64, device=dev)
        ws_p = ops.workspace_tensor(ops.permute_workspace(B, k, E), dev)
        ws_f = ops.workspace_tensor(ops.expert_ffn_workspace(B * k, H, F, E), dev)
        offs = torch.empty(E + 1, dtype=torch.int32, device=dev)
        rop = torch.empty(B * k, dtype=torch.int32, device=dev)
        por = torch.empty(B * k, dtype=torch.int32, device=dev)
        xp = torch.empty((B * k, H), dtype=torch.bfloat16, device=dev)
        yp = torch.empty_like(xp)
        y = torch.empty((N, H), dtype=torch.bfloat16, device=dev)
        inc = torch.empty(B, dtype=torch.int32, device=dev)
        natural = torch.arange(N, dtype=torch.int32, device=dev)

        def through_layers(tids):
            for l in range(L):
                wg, wu, wd = sets[l % n_sets]
                ops.permute(x, idx_l[l], E, token_ids=tids, expert_offsets=offs, row_of_pair=rop,
                            pair_of_row=por, x_perm=xp, workspace=ws_p)
                ops.expert_ffn(xp, offs, wg, wu, wd, y_perm=yp, workspace=ws_f)
                ops.combine(yp, idx_l[l], gw_l[l], rop, token_ids=tids, y=y, incomplete=inc)

        rec = {"tokens_per_batch": B}
        for name in ("input_order", "scheduled"):
            t_sched, t_layers = [], []
            for rep in range(args.warmup + 5):
                flush.fill_(float(rep))
                torch.cuda._sleep(1000000)
                ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
                ev[0].record()
                if name == "scheduled":
                    ops.schedule(rt, E, perm=perm, demand=demand, info=info, workspace=ws_s)
                    order = perm
                else:
                    order = natural
                ev[1].record()
                for b in range(2):
                    through_layers(order[b * B:(b + 1) * B])
                ev[2].record()
                torch.cuda.synchronize()
                if rep >= args.warmup:
                    t_sched.append(ev[0].elapsed_time(ev[1]))
                    t_layers.append(ev[1].elapsed_time(ev[2]))
            o = order.cpu().numpy()
            pairs = 0
            for b in range(2):
                rows = o[b * B:(b + 1) * B]
                pairs += sum(int(np.unique(idx_host[l][rows]).size) for l in range(L))
            layers_ms = float(np.median(t_layers))
            wgb = pairs * wbytes_expert / 1e9
            rec[name] = {"active_layer_expert_pairs": pairs,
                         "expert_weight_GB": round(wgb, 2),
                         "layers_ms": round(layers_ms, 3),
                         "weight_GBps": round(wgb / (layers_ms * 1e-3), 1)}
            if name == "scheduled":
                rec[name]["schedule_ms"] = round(float(np.median(t_sched)), 4)
                rec[name]["eq2_predicted_before_after"] = [int(info[4].item()), int(info[5].item())]
        a_, s_ = rec["input_order"], rec["scheduled"]
        rec["speedup_with_schedule"] = round(a_["layers_ms"] / (s_["layers_ms"] + s_["schedule_ms"]), 3)
        out.append(rec)
    rec = {"metric": "token scheduling on decode-sized units: active (layer, expert) pairs, "
                     "expert-weight bytes and time through 24 layers, input order against "
                     "scheduled",
           "config": {"workload": f"Qwen1.5-MoE-shaped layers: L={L}, H={H}, E={E}, F={F}, "
                                  f"top-{k}, every expert resident, no shared experts or "
                                  f"attention; units of two batches; predicted routes with "
                                  f"{topics} topics (keep {cfg['keep']}, zipf {cfg['zipf']}), "
                                  f"gating boosted {boost} towards each layer's predicted route"},
           "units": out, "data": "synthetic"}
    print(json.dumps(rec))


def ways_report(args):
    """B-way token scheduling (moe_schedule_multi) on Qwen-shaped predicted
    routes: for B batches of 64 tokens, the time of one call (HIP events,
    median of 7) and the active (layer, expert) pairs summed over the batches
    (Eq. 2 generalised) for the input order cut into B contiguous batches and
    for the scheduled batches; once on the unstructured Markov routes and once
    on topic-structured ones (two topics, 16-token batches, synth.topic_routes).
    One JSON line."""
    import torch
    from paper_2410_17954_amd import ops, synth

    dev = torch.device("cuda:0")
    cfg = synth.workload("qwen15_moe_layer")
    L, E, k = cfg["L"], cfg["E"], cfg["k"]
    per_batch = 64                   # decode-sized batches: not every expert is hit
    out = []
    topics, topic_batch = 2, 16      # topic case: two topics, 16-token batches
    out_topics = []
    for B, structured in [(b, False) for b in (2, 4, 8, 16, 64)] + \
                         [(b, True) for b in (2, 4, 8, 16, 64)]:
        N = B * (topic_batch if structured else per_batch)
        if structured:
            routes = synth.topic_routes(N, L, E, k, cfg["keep"], cfg["zipf"], topics, args.seed)
        else:
            routes = synth.predicted_routes(N, L, E, k, cfg["keep"], cfg["zipf"], args.seed)
        rt = torch.from_numpy(np.ascontiguousarray(routes, dtype=np.uint8)).to(dev)
        ws = ops.workspace_tensor(ops.schedule_multi_workspace(N, L, E, k, B), dev)
        perm = torch.empty(N, dtype=torch.int32, device=dev)
        offs = torch.empty(B + 1, dtype=torch.int32, device=dev)
        demand = torch.empty((B, L, E), dtype=torch.int32, device=dev)
        info = torch.empty((B - 1, 8), dtype=torch.int64, device=dev)

        def call():
            ops.schedule_multi(rt, E, B, perm=perm, batch_offsets=offs, demand=demand, info=info,
                               workspace=ws)

        ts = []
        for rep in range(args.warmup + 7):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(1000000)
            e0.record()
            call()
            e1.record()
            torch.cuda.synchronize()
            if rep >= args.warmup:
                ts.append(e0.elapsed_time(e1))
        before = 0
        nb = N // B
        for b in range(B):
            r = routes[b * nb:(b + 1) * nb].astype(np.int64)
            act = np.zeros((L, E), dtype=bool)
            for l in range(L):
                act[l, np.unique(r[:, l, :])] = True
            before += int(act.sum())
        after = int((demand.cpu().numpy() > 0).sum())
        (out_topics if structured else out).append({"batches": B, "tokens": N, "ms": round(float(np.median(ts)), 4),
                    "active_pairs_input_order": before, "active_pairs_scheduled": after,
                    "experts_per_layer_per_batch_input": round(before / (B * L), 2),
                    "experts_per_layer_per_batch_scheduled": round(after / (B * L), 2)})
    rec = {"metric": "B-way token scheduling: time and active (layer, expert) pairs",
           "config": {"workload": f"Qwen1.5-MoE-shaped predicted routes: L={L}, E={E}, top-{k}, "
                                  f"batches of {per_batch} tokens, keep {cfg['keep']}, "
                                  f"zipf {cfg['zipf']}"},
           "steps": out,
           "steps_topic_routes": out_topics,
           "topic_routes": f"batches of {topic_batch} tokens, {topics} topics, each token on "
                           "one topic's Markov chain over its own expert popularity order, "
                           "topics mixed along the token axis",
           "data": "synthetic"}
    print(json.dumps(rec))


def sched_sweep_report(args):
    """Two-way token scheduler (moe_schedule) from 1024 to 2^20 tokens on
    Mixtral-shaped predicted routes (32 layers, 8 experts, top-2; the first N
    tokens of one 2^20-token draw), n1 = N / 2. Per size: the call's time (HIP
    events, median of 5 after 2 warm-ups, launches queued behind a short wait),
    rounds, Eq. 2 before and after, and an effective rate over the bytes the
    algorithm must move: one read of the routes, one write of perm, and
    (5 + 3 * rounds) passes over the packed paths (their write, the signature
    order, the input split's counts, m1, m2, then per round the deltas, the
    batch-1 counts and the centroid sums). One JSON line."""
    import torch
    from paper_2410_17954_amd import ops, synth

    dev = torch.device("cuda:0")
    cfg = synth.workload("mixtral8x7b_route_grouped")
    L, E, k = cfg["L"], cfg["E"], cfg["k"]
    W = (L * E + 63) // 64
    Nmax = 1 << 20
    routes = synth.predicted_routes(Nmax, L, E, k, cfg["keep"], cfg["zipf"], args.seed)
    rt_all = torch.from_numpy(np.ascontiguousarray(routes, dtype=np.uint8)).to(dev)
    out = []
    for lg in (10, 12, 13, 14, 16, 18, 20):
        N = 1 << lg
        rt = rt_all[:N]
        ws = ops.workspace_tensor(ops.schedule_workspace(N, L, E, k), dev)
        perm = torch.empty(N, dtype=torch.int32, device=dev)
        demand = torch.empty((2, L, E), dtype=torch.int32, device=dev)
        info = torch.empty(8, dtype=torch.int64, device=dev)
        ts = []
        for rep in range(2 + 5):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(1000000)
            e0.record()
            ops.schedule(rt, E, perm=perm, demand=demand, info=info, workspace=ws)
            e1.record()
            torch.cuda.synchronize()
            if rep >= 2:
                ts.append(e0.elapsed_time(e1))
        ms = float(np.median(ts))
        inf = info.cpu().numpy()
        iters = int(inf[0])
        nbytes = N * L * k + 4 * N + (5 + 3 * iters) * N * W * 8
        out.append({"tokens": N, "us": round(ms * 1e3, 1), "rounds": iters,
                    "converged": int(inf[1]), "obj_before": int(inf[4]),
                    "obj_after": int(inf[5]), "used_original": int(inf[6]),
                    "algorithmic_MB": round(nbytes / 1e6, 3),
                    "GB/s": round(nbytes / (ms * 1e-3) / 1e9, 1),
                    "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)})
    rec = {"metric": "two-way token scheduling: time per call and effective bandwidth by size",
           "config": {"workload": f"Mixtral-shaped predicted routes: L={L}, E={E}, top-{k}, "
                                  f"keep {cfg['keep']}, zipf {cfg['zipf']}; n1 = N / 2"},
           "steps": out, "data": "synthetic"}
    print(json.dumps(rec))


def _median_ms(torch, fn, reps=7):
    """Median of HIP-event times of fn() on the current stream (after one
    untimed call), each behind a short device sleep so that host launch time
    is not counted."""
    fn()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(1000000)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    return float(np.median(ts))


def _rate(nbytes, ms):
    return {"ms": round(ms, 4), "GB/s": round(nbytes / ms / 1e6, 1),
            "hbm_frac": round(nbytes / ms / 1e6 / PEAK_HBM_GBS, 3)}


def _mfma(flop, ms):
    return {"ms": round(ms, 4), "TFLOP/s": round(flop / ms / 1e9, 1),
            "mfma_frac": round(flop / ms / 1e9 / PEAK_BF16_TFLOPS, 3)}


def _weight_bound_split(torch, ops, xp, off, counts, slot_np, slot_w, ws_f, yp, H, F, E, dev,
                        ridge_rows=315):
    """The FFN of one batch run twice more outside the timed step, once with
    only the resident experts that have fewer than ridge_rows rows (below the
    ridge every weight byte serves fewer flops than HBM can feed the MFMA, so
    these experts are bound by reading their weights) and once with only the
    others: weight GB/s and HBM fraction of the first, TFLOP/s of the second."""
    small = np.array([slot_np[e] >= 0 and 0 < counts[e] < ridge_rows for e in range(E)])
    large = np.array([slot_np[e] >= 0 and counts[e] >= ridge_rows for e in range(E)])
    out = {"ridge_rows": ridge_rows}
    for name, sel in (("under_ridge", small), ("over_ridge", large)):
        if not sel.any():
            out[name] = None
            continue
        sl = np.where(sel, slot_np, -1).astype(np.int32)
        sl_d = torch.from_numpy(sl).to(dev)
        ms = _median_ms(torch, lambda: ops.expert_ffn(xp, off, *slot_w, slot_of_expert=sl_d,
                                                      y_perm=yp, workspace=ws_f))
        rows = int(counts[sel].sum())
        wbytes = 3.0 * H * F * 2 * int(sel.sum())
        rec = {"experts": int(sel.sum()), "rows": rows, "ms": round(ms, 4),
               "weight_GB/s": round(wbytes / ms / 1e6, 1),
               "weight_hbm_frac": round(wbytes / ms / 1e6 / PEAK_HBM_GBS, 3),
               **{k: v for k, v in _mfma(6.0 * H * F * rows, ms).items() if k != "ms"}}
        out[name] = rec
    return out


def scheduled_layer_report(args, name):
    """A route-grouped MoE layer (Mixtral-shaped with 4 of 8 experts resident,
    or DeepSeek-V2-Lite-shaped with 48 of 64 and shared experts): one step
    schedules N tokens into two batches by multi-layer predicted routes,
    routes all of them (router bias toward each token's predicted layer-0
    experts, so that prediction and routing mostly agree), then per batch
    permutes, runs the resident experts (the batch's S most demanded by
    prediction; the slot tables and slot weights are set up once, before the
    timed region, as the expert cache would hold them), gathers the batch for
    the shared experts and runs them (if any), and combines; tokens whose
    experts are not all resident are flagged (misses). Tokens/s, per-stage
    HIP-event times and rates (routed and shared FFN against the bf16 MFMA
    peak), and the FFN of one batch split at the ridge. One JSON line."""
    import torch
    from paper_2410_17954_amd import ops, synth

    dev = torch.device("cuda:0")
    cfg = synth.workload(name)
    N, H, E, F, k, L, S = (cfg[n] for n in ("T", "H", "E", "F", "k", "L", "S"))
    n_s = cfg["n_shared"]
    inp = synth.layer_inputs(cfg, cfg["seed"], T=N)
    routes = synth.predicted_routes(N, L, E, k, cfg["keep"], cfg["zipf"], cfg["seed"])
    bias = synth.route_boost_bias(routes, 0, E, cfg["boost"], inp.get("bias"))

    def up(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    x, wr, bias_d, routes_d = up(inp["x"]), up(inp["w_router"]), up(bias), up(routes)
    W = {n: up(inp[n]) for n in ("w_gate", "w_up", "w_down")}
    shared = (tuple(up(inp[n])[None] for n in ("shared_gate", "shared_up", "shared_down"))
              if n_s else None)
    n1 = N // 2
    T = N - n1
    perm = torch.empty(N, dtype=torch.int32, device=dev)
    demand = torch.empty((2, L, E), dtype=torch.int32, device=dev)
    info = torch.empty(8, dtype=torch.int64, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    ws_s = ops.workspace_tensor(ops.schedule_workspace(N, L, E, k), dev)
    ops.schedule(routes_d, E, perm=perm, demand=demand, info=info, workspace=ws_s, err=err)
    d_host = demand.cpu().numpy()
    slots, slot_d, slot_w = [], [], []
    for b in range(2):
        sl = ops.plan_slots(d_host[b, 0], S)
        res = torch.tensor([e for e in range(E) if sl[e] >= 0], dtype=torch.long, device=dev)
        slots.append(sl)
        slot_d.append(torch.from_numpy(sl).to(dev))
        slot_w.append(tuple(W[n].index_select(0, res).contiguous()
                            for n in ("w_gate", "w_up", "w_down")))
    del W
    idx = torch.empty((N, k), dtype=torch.int32, device=dev)
    gw = torch.empty((N, k), dtype=torch.float32, device=dev)
    R = T * k
    ws_p = ops.workspace_tensor(ops.permute_workspace(T, k, E), dev)
    ws_f = ops.workspace_tensor(ops.expert_ffn_workspace(R, H, F, E), dev)
    if n_s:
        ws_p1 = ops.workspace_tensor(ops.permute_workspace(T, 1, 1), dev)
        ws_f1 = ops.workspace_tensor(ops.expert_ffn_workspace(T, H, n_s * F, 1), dev)
        zeros1 = torch.zeros((N, 1), dtype=torch.int32, device=dev)
    bufs = []
    for b in range(2):
        bf = dict(off=torch.empty(E + 1, dtype=torch.int32, device=dev),
                  rop=torch.empty(R, dtype=torch.int32, device=dev),
                  por=torch.empty(R, dtype=torch.int32, device=dev),
                  xp=torch.empty((R, H), dtype=torch.bfloat16, device=dev),
                  yp=torch.empty((R, H), dtype=torch.bfloat16, device=dev),
                  inc=torch.empty(T, dtype=torch.int32, device=dev))
        if n_s:
            bf.update(off1=torch.empty(2, dtype=torch.int32, device=dev),
                      rop1=torch.empty(T, dtype=torch.int32, device=dev),
                      por1=torch.empty(T, dtype=torch.int32, device=dev),
                      xs=torch.empty((T, H), dtype=torch.bfloat16, device=dev),
                      ys=torch.empty((T, H), dtype=torch.bfloat16, device=dev))
        bufs.append(bf)
    y = torch.zeros((N, H), dtype=torch.bfloat16, device=dev)
    names = ["schedule", "route", "permute", "expert_ffn"]
    if n_s:
        names += ["shared_gather", "shared_ffn"]
    names += ["combine"]
    per_batch = len(names) - 2

    def step(ev=None):
        marks = []

        def mark():
            if ev is not None:
                e = torch.cuda.Event(enable_timing=True)
                e.record()
                marks.append(e)
        mark()
        ops.schedule(routes_d, E, perm=perm, demand=demand, info=info, workspace=ws_s, err=err)
        mark()
        ops.route(x, wr, k, bias=bias_d, topk_idx=idx, topk_w=gw)
        mark()
        for b in range(2):
            tok = perm[:n1] if b == 0 else perm[n1:]
            bf = bufs[b]
            ops.permute(x, idx, E, token_ids=tok, expert_offsets=bf["off"], row_of_pair=bf["rop"],
                        pair_of_row=bf["por"], x_perm=bf["xp"], workspace=ws_p)
            mark()
            ops.expert_ffn(bf["xp"], bf["off"], *slot_w[b], slot_of_expert=slot_d[b],
                           y_perm=bf["yp"], workspace=ws_f)
            mark()
            if n_s:
                ops.permute(x, zeros1, 1, token_ids=tok, expert_offsets=bf["off1"],
                            row_of_pair=bf["rop1"], pair_of_row=bf["por1"], x_perm=bf["xs"],
                            workspace=ws_p1)
                mark()
                ops.expert_ffn(bf["xs"], bf["off1"], *shared, y_perm=bf["ys"], workspace=ws_f1)
                mark()
            ops.combine(bf["yp"], idx, gw, bf["rop"], token_ids=tok, slot_of_expert=slot_d[b],
                        y_shared=bf["ys"] if n_s else None, y=y, incomplete=bf["inc"])
            mark()
        return marks

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    K = args.steps
    all_marks = []
    t0 = time.perf_counter()
    for _ in range(K):
        all_marks.append(step(True))
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / K
    st = {n: 0.0 for n in names}
    for m in all_marks:
        st["schedule"] += m[0].elapsed_time(m[1])
        st["route"] += m[1].elapsed_time(m[2])
        for b in range(2):
            base = 2 + per_batch * b
            for j, n in enumerate(names[2:]):
                st[n] += m[base + j].elapsed_time(m[base + j + 1])
    st = {n: v / K for n, v in st.items()}
    assert int(err.item()) == 0, "the scheduler flagged its result"
    idx_h = idx.cpu().numpy()
    perm_h = perm.cpu().numpy()
    resident_pairs = 0
    incomplete = 0
    for b, tok in enumerate((perm_h[:n1], perm_h[n1:])):
        hit = slots[b][idx_h[tok]] >= 0
        resident_pairs += int(hit.sum())
        incomplete += int((~hit).any(axis=1).sum())
    inc_dev = int(sum(int(bufs[b]["inc"].sum()) for b in range(2)))
    assert inc_dev == incomplete and torch.isfinite(y.float()).all().item()
    ffn_flop = 6.0 * H * F * resident_pairs
    bytes_route = N * H * 2 + E * H * 2 + N * E * 4 + N * k * 8
    bytes_perm = N * H * 2 + N * k * H * 2 + N * k * 12
    bytes_comb = N * k * H * 2 + (2 if n_s else 1) * N * H * 2 + N * k * 12
    inf = info.cpu().numpy()
    counts0 = np.diff(bufs[0]["off"].cpu().numpy().astype(np.int64))
    stages = {
        "schedule": {"ms": round(st["schedule"], 4), "iters": int(inf[0]),
                     "obj_before": int(inf[4]), "obj_after": int(inf[5])},
        "route": _rate(bytes_route, st["route"]),
        "permute": _rate(bytes_perm, st["permute"]),
        "expert_ffn": _mfma(ffn_flop, st["expert_ffn"]),
    }
    if n_s:
        stages["shared_gather"] = _rate(2 * N * H * 2, st["shared_gather"])
        stages["shared_ffn"] = _mfma(6.0 * H * (n_s * F) * N, st["shared_ffn"])
    stages["combine"] = _rate(bytes_comb, st["combine"])
    split = _weight_bound_split(torch, ops, bufs[0]["xp"], bufs[0]["off"], counts0, slots[0],
                                slot_w[0], ws_f, bufs[0]["yp"], H, F, E, dev)
    desc = {"mixtral8x7b_route_grouped": "Mixtral-8x7B-shaped", "deepseek_v2_lite_layer":
            "DeepSeek-V2-Lite-shaped"}[name]
    rec = {
        "metric": f"{desc} route-grouped MoE layer: tokens/s and per-stage rates",
        "value": N / (ms_step * 1e-3), "unit": "tokens/s", "ms_per_step": ms_step, "steps": K,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{desc} MoE layer: {N} tokens scheduled into two batches by "
                               f"{L}-layer predicted routes (keep {cfg['keep']}, zipf "
                               f"{cfg['zipf']}), H={H}, E={E}, F={F}, top-{k}, {S} of {E} "
                               f"experts resident per batch (misses flagged)"
                               + (f", {n_s} shared experts" if n_s else ""),
                   "router_boost": cfg["boost"]},
        "stages": stages,
        "batch0_ffn_by_ridge": split,
        "batch0_rows_per_expert": counts0.tolist(),
        "resident_pair_share": round(resident_pairs / (N * k), 4),
        "incomplete_tokens": incomplete,
    }
    print(json.dumps(rec))


def qwen_report(args):
    """Qwen1.5-MoE-shaped layer (H 2048, 60 routed experts of width 1408,
    top-4, Zipf(1.2)-skewed router, four shared experts as one FFN of width
    5632): one 8192-token batch per step is routed, permuted, run through the
    32 resident experts (the batch's 32 most routed: the expert cache with a
    perfect predictor; slot weights set up once, before the timed region),
    gathered for the shared experts, run through them, and combined. The
    routed experts' row counts fall off along the Zipf tail, so below about
    315 rows an expert is bound by reading its weights: the FFN is also timed
    with only those experts, and with only the others. One JSON line."""
    import torch
    from paper_2410_17954_amd import ops, synth

    dev = torch.device("cuda:0")
    cfg = synth.workload("qwen15_moe_layer")
    T, H, E, F, k, S, n_s = (cfg[n] for n in ("T", "H", "E", "F", "k", "S", "n_shared"))
    inp = synth.layer_inputs(cfg, cfg["seed"], T=T)

    def up(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    x, wr, bias_d = up(inp["x"]), up(inp["w_router"]), up(inp["bias"])
    W = {n: up(inp[n]) for n in ("w_gate", "w_up", "w_down")}
    shared = tuple(up(inp[n])[None] for n in ("shared_gate", "shared_up", "shared_down"))
    idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    gw = torch.empty((T, k), dtype=torch.float32, device=dev)
    ops.route(x, wr, k, bias=bias_d, topk_idx=idx, topk_w=gw)
    routed = np.bincount(idx.cpu().numpy().ravel(), minlength=E)
    slot = ops.plan_slots(routed, S)
    res = torch.tensor([e for e in range(E) if slot[e] >= 0], dtype=torch.long, device=dev)
    slot_w = tuple(W[n].index_select(0, res).contiguous() for n in ("w_gate", "w_up", "w_down"))
    del W
    slot_d = torch.from_numpy(slot).to(dev)
    R = T * k
    off = torch.empty(E + 1, dtype=torch.int32, device=dev)
    rop = torch.empty(R, dtype=torch.int32, device=dev)
    por = torch.empty(R, dtype=torch.int32, device=dev)
    xp = torch.empty((R, H), dtype=torch.bfloat16, device=dev)
    yp = torch.empty((R, H), dtype=torch.bfloat16, device=dev)
    off1 = torch.empty(2, dtype=torch.int32, device=dev)
    rop1 = torch.empty(T, dtype=torch.int32, device=dev)
    por1 = torch.empty(T, dtype=torch.int32, device=dev)
    ys = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
    inc = torch.empty(T, dtype=torch.int32, device=dev)
    y = torch.zeros((T, H), dtype=torch.bfloat16, device=dev)
    ws_p = ops.workspace_tensor(ops.permute_workspace(T, k, E), dev)
    ws_f = ops.workspace_tensor(ops.expert_ffn_workspace(R, H, F, E), dev)
    ws_f1 = ops.workspace_tensor(ops.expert_ffn_workspace(T, H, n_s * F, 1), dev)
    names = ["route", "permute", "expert_ffn", "shared_ffn", "combine"]

    def step(ev=None):
        marks = []

        def mark():
            if ev is not None:
                e = torch.cuda.Event(enable_timing=True)
                e.record()
                marks.append(e)
        mark()
        ops.route(x, wr, k, bias=bias_d, topk_idx=idx, topk_w=gw)
        mark()
        ops.permute(x, idx, E, expert_offsets=off, row_of_pair=rop, pair_of_row=por, x_perm=xp,
                    workspace=ws_p)
        mark()
        ops.expert_ffn(xp, off, *slot_w, slot_of_expert=slot_d, y_perm=yp, workspace=ws_f)
        mark()
        # the shared experts see the batch in token order: x itself, no gather
        ops.expert_ffn(x, off1, *shared, y_perm=ys, workspace=ws_f1)
        mark()
        ops.combine(yp, idx, gw, rop, slot_of_expert=slot_d, y_shared=ys, y=y, incomplete=inc)
        mark()
        return marks

    off1.copy_(torch.tensor([0, T], dtype=torch.int32))
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    K = args.steps
    all_marks = []
    t0 = time.perf_counter()
    for _ in range(K):
        all_marks.append(step(True))
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / K
    st = {n: sum(m[j].elapsed_time(m[j + 1]) for m in all_marks) / K
          for j, n in enumerate(names)}
    counts = np.diff(off.cpu().numpy().astype(np.int64))
    assert np.array_equal(counts, routed)
    resident_pairs = int(counts[slot >= 0].sum())
    incomplete = int((slot[idx.cpu().numpy()] < 0).any(axis=1).sum())
    assert int(inc.sum()) == incomplete and torch.isfinite(y.float()).all().item()
    bytes_route = T * H * 2 + E * H * 2 + T * E * 4 + T * k * 8 + E * 4
    bytes_perm = T * H * 2 + R * H * 2 + T * k * 12
    bytes_comb = R * H * 2 + 2 * T * H * 2 + T * k * 12
    split = _weight_bound_split(torch, ops, xp, off, counts, slot, slot_w, ws_f, yp, H, F, E,
                                dev)
    rec = {
        "metric": "Qwen1.5-MoE-shaped MoE layer: tokens/s and per-stage rates",
        "value": T / (ms_step * 1e-3), "unit": "tokens/s", "ms_per_step": ms_step, "steps": K,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"Qwen1.5-MoE-shaped MoE layer: one batch of {T} tokens, H={H}, "
                               f"E={E}, F={F}, top-{k}, router skewed by a Zipf({cfg['zipf_bias']})"
                               f"-ranked bias, {S} of {E} experts resident (the batch's most "
                               f"routed), {n_s} shared experts (one FFN of width {n_s * F})"},
        "stages": {
            "route": _rate(bytes_route, st["route"]),
            "permute": _rate(bytes_perm, st["permute"]),
            "expert_ffn": _mfma(6.0 * H * F * resident_pairs, st["expert_ffn"]),
            "shared_ffn": _mfma(6.0 * H * (n_s * F) * T, st["shared_ffn"]),
            "combine": _rate(bytes_comb, st["combine"]),
        },
        "ffn_by_ridge": split,
        "rows_per_resident_expert": sorted((int(c) for c in counts[slot >= 0]), reverse=True),
        "resident_pair_share": round(resident_pairs / R, 4),
        "incomplete_tokens": incomplete,
    }
    print(json.dumps(rec))


def plec_report(args):
    """Expert cache engine at run time (one JSON line): batches of
    --plec-batch tokens through L = 8 Qwen1.5-MoE-shaped layers (H 2048, 60
    experts of width 1408, top-4; residual, no attention) whose 480 experts
    (8.3 GB) live in pinned host memory; the device holds L x --plec-cache
    slots shared by all layers, run by PLEC from each batch's predicted
    routes (Markov routes, keep 0.7, Zipf 1.2), with misses corrected by
    copies on a second stream. The router of each layer is biased toward the
    batch's predicted experts so that prediction and routing mostly agree
    (the predictor's role); every batch's routes are cut from one draw, so
    the layers' expert popularity is the same model-wide. Reported: ms per
    batch, measured hits / needed
    per batch and in all, copies and PCIe bytes, and the hit ratio of
    per-layer LRU caches of --plec-cache experts on the same measured
    demands (moe_lru_run, kept across the batches)."""
    import torch
    from paper_2410_17954_amd import ece, ops, synth

    dev = torch.device("cuda:0")
    cfg = synth.workload("qwen15_moe_layer")
    H, E, F, k = cfg["H"], cfg["E"], cfg["F"], cfg["k"]
    L, T, CS = 8, args.plec_batch, args.plec_cache
    budget = L * CS
    n_batches = max(2, args.steps)
    g = torch.Generator(device=dev)
    g.manual_seed(args.seed)

    def host_stack(shape):
        out = torch.empty((L, E) + shape, dtype=torch.bfloat16).pin_memory()
        for l in range(L):
            out[l].copy_((torch.randn((E,) + shape, generator=g, device=dev) * 0.02)
                         .to(torch.bfloat16))
        return out
    store = (host_stack((F, H)), host_stack((F, H)), host_stack((H, F)))
    routers = [(torch.randn((E, H), generator=g, device=dev) * 0.02).to(torch.bfloat16)
               for _ in range(L)]
    cache = tuple(torch.zeros((budget,) + tuple(t.shape[2:]), dtype=torch.bfloat16, device=dev)
                  for t in store)
    copy = torch.cuda.Stream(device=dev)
    rows = []
    demands = []
    # one model: every batch's tokens come from one draw (one expert popularity
    # order per layer), cut into consecutive batches
    all_routes = synth.predicted_routes((n_batches + 1) * T, L, E, k, 0.7, 1.2,
                                        seed=1000 * args.seed)
    for b in range(n_batches + 1):             # batch 0: warm-up, not reported
        routes = all_routes[b * T:(b + 1) * T]
        pdem = np.zeros((L, E), np.int64)
        for l in range(L):
            np.add.at(pdem[l], routes[:, l, :].ravel().astype(np.int64), 1)
        biases = [torch.from_numpy(synth.route_boost_bias(routes, l, E, 3.0, None)).to(dev)
                  for l in range(L)]
        h = (torch.randn((T, H), generator=g, device=dev)).to(torch.bfloat16)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        st = ece.run_plec_stack(h, routers, store, cache, pdem, k, budget, biases=biases,
                                copy_stream=copy)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3
        if b == 0:
            continue
        demands.append(st["demand"])
        sim = ops.plec_run(pdem, st["demand"], budget)
        assert sim["hits"].tolist() == st["hits"] and sim["loads"] == st["loads"]
        rows.append({"ms": round(ms, 3), "hits": int(sum(st["hits"])),
                     "needed": int(sum(st["needed"])), "copies": int(st["loads"]),
                     "GB_copied": round(st["bytes_loaded"] / 1e9, 3)})
    hits = sum(r["hits"] for r in rows)
    needed = sum(r["needed"] for r in rows)
    lru_h, lru_n = ops.lru_run(np.stack(demands), CS)
    ms = [r["ms"] for r in rows]
    rec = {"metric": "expert cache engine: PLEC hit ratio and time per batch vs per-layer LRU",
           "config": {"workload": f"{L} Qwen1.5-MoE-shaped layers (H={H}, E={E}, F={F}, "
                                  f"top-{k}), experts in pinned host memory, batches of {T} "
                                  f"tokens, {budget} device slots shared by all layers (LRU: "
                                  f"{CS} per layer), predicted routes keep 0.7 / Zipf 1.2, "
                                  f"router bias +3 toward predicted experts",
                      "batches": len(rows)},
           "plec_hit_ratio": round(hits / needed, 4),
           "lru_hit_ratio_same_demands": round(lru_h / lru_n, 4),
           "ms_per_batch_median": round(float(np.median(ms)), 3),
           "copies_per_batch_mean": round(float(np.mean([r["copies"] for r in rows])), 1),
           "copy_GBps": round(sum(r["GB_copied"] for r in rows) / (sum(ms) * 1e-3), 2),
           "batches": rows, "data": "synthetic"}
    print(json.dumps(rec))


def stack_report(args):
    """Dual-batch pipeline over a stack of MoE layers (one JSON line).

    Units of 8192 tokens (two 4096-token batches) with 32-layer predicted
    routes; each unit is rebatched by the token scheduler, its two original
    batches' KV caches (Mixtral: 8 KV heads x 128 x K,V in bf16 = 4 KB per token
    and layer) merged and reindexed into the new layout, and both new batches
    run through the layer stack (RMS pre-normalised blocks, every expert of
    every layer resident in HBM: 32 x 2.8 GB). Timed with and without the next
    unit's scheduling and KV work on a second stream."""
    import torch
    from paper_2410_17954_amd import ops, pipeline, synth

    dev = torch.device("cuda:0")
    cfg = synth.workload("mixtral8x7b_route_grouped")
    H, E, F, k = cfg["H"], cfg["E"], cfg["F"], cfg["k"]
    L = args.stack_layers
    N = cfg["T"]                                   # one unit: two batches of N / 2
    kv_row = 8 * 128 * 2 * 2
    g = torch.Generator(device=dev)
    g.manual_seed(args.seed)

    def rnd(shape, scale):
        t = torch.empty(shape, dtype=torch.bfloat16, device=dev)
        t.normal_(0.0, scale, generator=g)
        return t

    layers = [(rnd((E, H), 0.02), rnd((E, F, H), 0.02), rnd((E, F, H), 0.02),
               rnd((E, H, F), 0.02)) for _ in range(L)]
    n_units = 1 + args.stack_units
    predictor = None
    if args.stack_predictor:
        dims = dict(vocab=32000, d_model=32, n_heads=4, d_ff=2048, n_enc=3, n_dec=3, L=L, E=E,
                    num_buckets=32, max_distance=128, eps=1e-6)
        pw = torch.randn(ops.rpp_weights_count(dims), generator=g, device=dev) * 0.1
        predictor = dict(weights=pw, dims=dims)

    def make_units(seed0):
        us = []
        for u in range(n_units):
            kv = [torch.randint(0, 256, (L, N // 2, kv_row), dtype=torch.uint8, device=dev,
                                generator=g) for _ in range(2)]
            if predictor is not None:
                ids = torch.randint(0, 32000, (16, N // 16), dtype=torch.int32, device=dev,
                                    generator=g)
                us.append(pipeline.Unit(h=rnd((N, H), 1.0), kv=kv, ids=ids))
                continue
            routes = synth.predicted_routes(N, L, E, k, cfg["keep"], cfg["zipf"], seed0 + u)
            us.append(pipeline.Unit(
                h=rnd((N, H), 1.0),
                routes=torch.from_numpy(np.ascontiguousarray(routes, dtype=np.uint8)).to(dev),
                kv=kv))
        return us

    out = {}
    state = {}
    for overlap in (True, False):
        units = make_units(args.seed * 1000)
        pl = pipeline.DualBatchPipeline(layers, k, E, N, overlap=overlap, predictor=predictor)
        pl.run(units[:1])                          # warm-up unit
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        pl.run(units[1:])
        torch.cuda.synchronize()
        out[overlap] = time.perf_counter() - t0
        hf = units[-1].h.float()
        state[overlap] = (bool(torch.isfinite(hf).all().item()), float(hf.abs().mean().item()))
        del units, pl
    # the scheduling work of one unit alone (token scheduler + KV merge/reindex)
    units = make_units(args.seed * 1000 + 7)
    pl = pipeline.DualBatchPipeline(layers, k, E, N, overlap=False, predictor=predictor)
    pl._plan(units[0])
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    pl._plan(units[1])
    e1.record()
    torch.cuda.synchronize()
    plan_ms = e0.elapsed_time(e1)
    toks = args.stack_units * N
    rec = {"metric": "dual-batch pipeline over a stack of MoE layers: tokens/s through all layers",
           "config": {"workload": f"Mixtral-8x7B-shaped stack: {L} layers, H={H}, E={E}, F={F}, "
                                  f"top-{k}, units of {N} tokens (2 batches of {N // 2}), "
                                  f"32-layer predicted routes, KV rows of {kv_row} B per token "
                                  f"and layer, every expert resident in HBM",
                      "units_timed": args.stack_units},
           "tokens_per_s_overlapped": round(toks / out[True], 1),
           "tokens_per_s_in_order": round(toks / out[False], 1),
           "ms_per_unit_overlapped": round(out[True] / args.stack_units * 1e3, 3),
           "ms_per_unit_in_order": round(out[False] / args.stack_units * 1e3, 3),
           "plan_ms_per_unit": round(plan_ms, 3),
           "plan": ("routing path predictor (16 x 512 tokens, hidden 32, FFN 2048) + top-2 per "
                    "layer + token scheduler + KV merge/reindex" if predictor is not None else
                    "token scheduler + KV merge/reindex (routes given)"),
           "kv_bytes_moved_per_unit": 2 * L * N * kv_row,
           "final_state_finite": state[True][0],
           "final_state_abs_mean": round(state[True][1], 3),
           "data": "synthetic"}
    print(json.dumps(rec))


def rpp_flops(dims, B, S):
    """Algorithmic flops of one forward: every multiply-add counted as 2."""
    d, dff, LE = dims["d_model"], dims["d_ff"], dims["L"] * dims["E"]
    M = B * S
    enc = dims["n_enc"] * M * (2 * d * 3 * d + 2 * d * d + 4 * d * dff + 4 * S * d)
    causal_keys = (S + 1) / 2                      # mean keys per query under the causal mask
    dec = dims["n_dec"] * M * (2 * d * 3 * d + 2 * d * d + 4 * causal_keys * d
                               + 2 * d * d + 4 * d * d + 2 * d * d + 4 * S * d + 4 * d * dff)
    return enc + dec + 2 * M * d * LE


def rpp_report(args):
    """Routing path predictor forward (one JSON line): tokens/s and float32
    TFLOP/s, HIP events around one call, median of 7."""
    import torch
    from paper_2410_17954_amd import ops

    dev = torch.device("cuda:0")
    B, S = 16, 512
    out = []
    for name, L, E in (("Mixtral-8x7B heads", 32, 8), ("Qwen1.5-MoE heads", 24, 60)):
        dims = dict(vocab=32000, d_model=32, n_heads=4, d_ff=2048, n_enc=3, n_dec=3, L=L, E=E,
                    num_buckets=32, max_distance=128, eps=1e-6)
        g = torch.Generator(device=dev)
        g.manual_seed(args.seed)
        w = torch.randn(ops.rpp_weights_count(dims), generator=g, device=dev) * 0.1
        ids = torch.randint(0, 32000, (B, S), generator=g, device=dev, dtype=torch.int32)
        ws = ops.workspace_tensor(ops.load_library().moe_rpp_workspace(
            B, S, ops.ctypes.byref(ops.rpp_dims(dims))), dev)
        probs = torch.empty((B, S, L, E), dtype=torch.float32, device=dev)
        err = torch.zeros(1, dtype=torch.int32, device=dev)
        ts = []
        for rep in range(args.warmup + 7):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(1000000)
            e0.record()
            ops.rpp_forward(ids, w, dims, probs=probs, err=err, workspace=ws)
            e1.record()
            torch.cuda.synchronize()
            if rep >= args.warmup:
                ts.append(e0.elapsed_time(e1))
        ms = float(np.median(ts))
        fl = rpp_flops(dims, B, S)
        out.append({"heads": name, "L": L, "E": E, "ms": round(ms, 4),
                    "tokens_per_s": round(B * S / (ms * 1e-3), 1),
                    "gflop": round(fl / 1e9, 2), "tflops_fp32": round(fl / (ms * 1e-3) / 1e12, 2),
                    "frac_of_fp32_peak": round(fl / (ms * 1e-3) / 1e12 / 157.3, 3),
                    "weights_MB_fp32": round(ops.rpp_weights_count(dims) * 4 / 1e6, 2)})
    rec = {"metric": "routing path predictor forward: tokens/s and float32 TFLOP/s",
           "config": {"workload": f"T5-style predictor, 3+3 layers, hidden 32, 4 heads, FFN 2048, "
                                  f"vocab 32000, {B} sequences x {S} tokens, random weights"},
           "steps": out, "data": "synthetic"}
    print(json.dumps(rec))


def main():
    args = parse()
    if args.pmc_summary:
        summ = pmc_summary(args.pmc_summary[0], args.pmc_summary[1], args.copy_probe_mib)
        rec = {"ffn_source_sha256": ffn_source_digest(),
               "traffic_bytes_per_launch": summ["FETCH_SIZE"]["bytes_per_launch"]
               + summ["WRITE_SIZE"]["bytes_per_launch"], **summ}
        print(json.dumps(rec))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this hot path runs on exactly one GPU; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.ece:
        ece_report(args)
        return
    if args.decode_ts:
        decode_ts_report(args)
        return
    if args.decode:
        decode_report(args)
        return
    if args.ways:
        ways_report(args)
        return
    if args.stack:
        stack_report(args)
        return
    if args.sched_sweep:
        sched_sweep_report(args)
        return
    if args.deepseek:
        scheduled_layer_report(args, "deepseek_v2_lite_layer")
        return
    if args.route_grouped:
        scheduled_layer_report(args, "mixtral8x7b_route_grouped")
        return
    if args.qwen:
        qwen_report(args)
        return
    if args.plec:
        plec_report(args)
        return
    if args.rpp:
        rpp_report(args)
        return
    import torch
    from paper_2410_17954_amd import ops, synth

    dev = torch.device("cuda:0")
    cfg = synth.workload("mixtral8x7b_layer")
    T, H, E, F, k, L = cfg["T"], cfg["H"], cfg["E"], cfg["F"], cfg["k"], cfg["L"]
    N = 2 * T                        # one scheduling unit = two adjacent batches
    n1 = N // 2

    t_gen = time.time()
    inp = synth.layer_inputs(cfg, args.seed, T=N, parts=("x", "router", "experts"))
    routes = synth.predicted_routes(N, L, E, k, cfg["keep"], cfg["zipf"], args.seed)

    def up(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    x = up(inp["x"])
    wr = up(inp["w_router"])
    wg, wu, wd = up(inp["w_gate"]), up(inp["w_up"]), up(inp["w_down"])
    routes_d = up(routes)
    gen_s = time.time() - t_gen

    # Outputs and workspaces, allocated once.
    perm = torch.empty(N, dtype=torch.int32, device=dev)
    demand = torch.empty((2, L, E), dtype=torch.int32, device=dev)
    info = torch.empty(8, dtype=torch.int64, device=dev)
    ws_sched = ops.workspace_tensor(ops.schedule_workspace(N, L, E, k), dev)
    idx = torch.empty((N, k), dtype=torch.int32, device=dev)
    gw = torch.empty((N, k), dtype=torch.float32, device=dev)
    R = T * k
    offs = [torch.empty(E + 1, dtype=torch.int32, device=dev) for _ in range(2)]
    rops = [torch.empty(R, dtype=torch.int32, device=dev) for _ in range(2)]
    pors = [torch.empty(R, dtype=torch.int32, device=dev) for _ in range(2)]
    xps = [torch.empty((R, H), dtype=torch.bfloat16, device=dev) for _ in range(2)]
    yps = [torch.empty((R, H), dtype=torch.bfloat16, device=dev) for _ in range(2)]
    incs = [torch.empty(T, dtype=torch.int32, device=dev) for _ in range(2)]
    ws_perm = ops.workspace_tensor(ops.permute_workspace(T, k, E), dev)
    ws_ffn = ops.workspace_tensor(ops.expert_ffn_workspace(R, H, F, E), dev)
    y = torch.zeros((N, H), dtype=torch.bfloat16, device=dev)
    # Resident set (expert-cache planning from predicted demand): with as many
    # slots as experts every expert is resident, whatever the demand.
    S = cfg["S"]
    assert S >= E
    slot = torch.arange(E, dtype=torch.int32, device=dev)
    batches = [perm[:n1], perm[n1:]]

    stage_names = ["schedule", "route", "permute", "expert_ffn", "combine"]

    def step(ev=None):
        def mark(i):
            if ev is not None:
                ev[i].record()
        mark(0)
        ops.schedule(routes_d, E, n1=n1, perm=perm, demand=demand, info=info,
                     workspace=ws_sched)
        mark(1)
        ops.route(x, wr, k, topk_idx=idx, topk_w=gw)
        mark(2)
        j = 3
        for b in range(2):
            tok = batches[b]
            ops.permute(x, idx, E, token_ids=tok, expert_offsets=offs[b], row_of_pair=rops[b],
                        pair_of_row=pors[b], x_perm=xps[b], workspace=ws_perm)
            mark(j)
            ops.expert_ffn(xps[b], offs[b], wg, wu, wd, slot_of_expert=slot, y_perm=yps[b],
                           workspace=ws_ffn)
            mark(j + 1)
            ops.combine(yps[b], idx, gw, rops[b], token_ids=tok, slot_of_expert=slot, y=y,
                        incomplete=incs[b])
            mark(j + 2)
            j += 3

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    K = args.steps
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(9)] for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(K):
        step(events[s])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1e3 / K

    def span(ev, a, b):
        return ev[a].elapsed_time(ev[b])

    def stage_ms(ev, ffn_launch_ms=None):
        t = {n: 0.0 for n in stage_names}
        t["schedule"] = span(ev, 0, 1)
        t["route"] = span(ev, 1, 2)
        prev = 2
        for b in range(2):
            base = 3 + 3 * b
            t["permute"] += span(ev, prev, base)
            d = span(ev, base, base + 1)
            t["expert_ffn"] += d
            if ffn_launch_ms is not None:
                ffn_launch_ms.append(d)
            t["combine"] += span(ev, base + 1, base + 2)
            prev = base + 2
        return t

    ffn_launch_ms = []
    per_step = [stage_ms(ev, ffn_launch_ms) for ev in events]
    st = {n: sum(t[n] for t in per_step) / K for n in stage_names}

    # Outside the timed region: the same step with every cache cold (a 512 MB
    # write before each step evicts the last-level cache), launches queued
    # behind a short wait so that host time is not counted; median of 5.
    flush = torch.empty(512 * 2 ** 20 // 4, dtype=torch.float32, device=dev)
    cold = []
    for rep in range(5):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(9)]
        torch.cuda._sleep(3000000)
        flush.fill_(float(rep))
        step(ev)
        torch.cuda.synchronize()
        cold.append(stage_ms(ev))
    st_cold = {n: float(np.median([t[n] for t in cold])) for n in stage_names}
    del flush

    ceilings = measured_ceilings(torch, ops, dev)

    if args.copy_probe_mib > 0:
        src = torch.empty(args.copy_probe_mib * 2**20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()

    info_h = info.cpu().numpy()
    inc_h = torch.cat(incs).cpu().numpy()
    assert inc_h.sum() == 0 and torch.isfinite(y.float()).all().item()

    # Algorithmic work.
    ffn_flops = 6.0 * H * F * R                     # per moe_expert_ffn launch
    ffn_ms = float(np.mean(ffn_launch_ms))
    achieved = ffn_flops / (ffn_ms * 1e-3) / 1e12
    bytes_route = N * H * 2 + E * H * 2 + N * k * 8
    bytes_perm = 2 * (T * H * 2 + R * H * 2 + T * k * 4 + R * 8)
    bytes_comb = 2 * (R * H * 2 + T * H * 2 + T * k * 12)
    stages = {
        "schedule": {"ms": st["schedule"], "obj_before": int(info_h[4]),
                     "obj_after": int(info_h[5]), "iters": int(info_h[0])},
        "route": {"ms": st["route"], "GB/s": bytes_route / st["route"] / 1e6,
                  "hbm_frac": bytes_route / st["route"] / 1e6 / PEAK_HBM_GBS},
        "permute": {"ms": st["permute"], "GB/s": bytes_perm / st["permute"] / 1e6,
                    "hbm_frac": bytes_perm / st["permute"] / 1e6 / PEAK_HBM_GBS},
        "expert_ffn": {"ms": st["expert_ffn"], "TFLOP/s": achieved,
                       "mfma_frac": achieved / PEAK_BF16_TFLOPS},
        "combine": {"ms": st["combine"], "GB/s": bytes_comb / st["combine"] / 1e6,
                    "hbm_frac": bytes_comb / st["combine"] / 1e6 / PEAK_HBM_GBS},
    }
    # the same fractions against what this chip measured (probe kernels, below)
    for name in ("route", "permute", "combine"):
        stages[name]["hbm_frac_measured"] = stages[name]["GB/s"] / ceilings["hbm_read_GBps"]
    # routing is one cold read of x while the cache holds the FFN's and
    # combine's dirty lines: the dirty-cache pass is its own ceiling (permute
    # and combine also write, and read data written just before)
    stages["route"]["frac_of_dirty_cache_read"] = (stages["route"]["GB/s"] /
                                                   ceilings["read_64MiB_dirty_GBps"])
    # permute and combine read and write: against the plain copy in that state
    for name in ("permute", "combine"):
        stages[name]["frac_of_dirty_cache_copy"] = (stages[name]["GB/s"] /
                                                    ceilings["copy_64MiB_dirty_GBps"])
    stages["expert_ffn"]["mfma_frac_measured"] = achieved / ceilings["mfma_bf16_TFLOPs"]

    out = {
        "metric": METRIC,
        "value": N / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) activations, N(0,0.02) weights, Markov predicted routes)",
        "config": {
            "workload": ("Mixtral-8x7B-shaped MoE layer, one scheduling unit of two adjacent "
                         "T=4096 batches (8192 tokens), H=4096, E=8, F=14336, top-2 renormalised, "
                         "all 8 experts resident, 32-layer predicted routes (keep 0.7, Zipf 1.1)"),
            "tokens_per_step": N, "T": T, "H": H, "E": E, "F": F, "k": k, "L": L,
            "resident": S, "parallelism": "single GPU",
        },
        "roofline": {
            "bound": "mfma",
            "kernel": "moe_expert_ffn (" + " + ".join(FFN_KERNELS) + ")",
            "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS, "traffic": measured_traffic(),
            "flop_per_launch": ffn_flops, "launch_ms": ffn_ms,
        },
        "stages": stages,
        "stages_cold_ms": {n: round(v, 4) for n, v in st_cold.items()},
        "measured_ceilings": ceilings,
        "setup_s": gen_s,
    }
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cpu_baseline(inp, routes, cfg, args.cpu_seconds)
    print(json.dumps(out))


def measured_ceilings(torch, ops, dev):
    """What this GPU reaches in practice, measured after the timed region with
    the library's probe kernels: a loop of dense bf16 32x32x16 MFMAs on every
    SIMD (random operands that keep changing, no memory traffic), and one
    streaming read of a 1 GiB buffer (larger than the last-level cache;
    median of 5 passes)."""
    lib = ops.load_library()
    st = torch.cuda.current_stream().cuda_stream
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    src = torch.randn(8 * 64 * 8, generator=g, device=dev).to(torch.bfloat16)
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    out_f = torch.empty(8 * cus * 256, dtype=torch.float32, device=dev)
    out_u = torch.empty(8 * cus * 256, dtype=torch.int32, device=dev)

    def timed(fn, n):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(n):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    iters = 256
    flops = lib.moe_probe_mfma_bf16(ops._ptr(src), iters, ops._ptr(out_f), out_f.numel(), st)
    if flops <= 0:
        raise RuntimeError("moe_probe_mfma_bf16 failed")
    ms = timed(lambda: lib.moe_probe_mfma_bf16(ops._ptr(src), iters, ops._ptr(out_f),
                                               out_f.numel(), st), 5)
    buf = torch.ones(2 ** 30, dtype=torch.uint8, device=dev)
    rms = timed(lambda: lib.moe_probe_read(ops._ptr(buf), buf.numel(), ops._ptr(out_u),
                                           out_u.numel(), st), 5)

    # One 64 MiB pass (a routed batch's activations) in three cache states:
    # warm (read just before), clean (a 512 MiB read evicted it) and dirty (a
    # 512 MiB write evicted it: the last-level cache holds dirty lines that are
    # written back during the pass, as after the expert FFN and combine).
    a = torch.ones(64 * 2 ** 20, dtype=torch.uint8, device=dev)
    big = buf[:512 * 2 ** 20]

    def read(t):
        lib.moe_probe_read(ops._ptr(t), t.numel(), ops._ptr(out_u), out_u.numel(), st)

    def state(prep):
        ts = []
        for rep in range(6):
            prep(rep)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            read(a)
            e1.record()
            torch.cuda.synchronize()
            if rep:
                ts.append(e0.elapsed_time(e1))
        return a.numel() / (float(np.median(ts)) * 1e-3) / 1e9
    warm = state(lambda rep: read(a))
    clean = state(lambda rep: read(big))
    dirty = state(lambda rep: big.fill_(rep))
    # a plain copy of 64 MiB into a second buffer after a 512 MiB write (the
    # state permute and combine run in: reads and writes, dirty lines to
    # write back); bytes counted read plus written
    dst = torch.empty_like(a)
    cts = []
    for rep in range(6):
        big.fill_(rep)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        if lib.moe_probe_copy(ops._ptr(a), ops._ptr(dst), a.numel(), st) != 0:
            raise RuntimeError("moe_probe_copy failed")
        e1.record()
        torch.cuda.synchronize()
        if rep:
            cts.append(e0.elapsed_time(e1))
    copy = 2 * a.numel() / (float(np.median(cts)) * 1e-3) / 1e9
    return {"mfma_bf16_TFLOPs": flops / (ms * 1e-3) / 1e12,
            "hbm_read_GBps": buf.numel() / (rms * 1e-3) / 1e9,
            "read_64MiB_warm_GBps": warm, "read_64MiB_clean_GBps": clean,
            "read_64MiB_dirty_GBps": dirty, "copy_64MiB_dirty_GBps": copy,
            "probes": "moe_probe_mfma_bf16 (4 waves per SIMD, 8 MFMA chains, "
                      f"{iters} rounds), moe_probe_read (1 GiB, one pass; 64 MiB after a "
                      "read of it, after a 512 MiB read, after a 512 MiB write), "
                      "moe_probe_copy (64 MiB to a second buffer after a 512 MiB write, "
                      "read + written bytes)"}


def measured_traffic():
    """HBM bytes per moe_expert_ffn launch from the counter summary, or None
    when there is none or the FFN source has changed since it was taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = next(json.loads(l) for l in f if l.startswith("{"))
    except (OSError, StopIteration, ValueError):
        return None
    if rec.get("ffn_source_sha256") != ffn_source_digest():
        return None
    return rec["traffic_bytes_per_launch"]


def cpu_baseline(inp, routes, cfg, budget_s):
    """The CPU oracle, unmodified, on a bounded sample of the same workload:
    the scheduler over the whole 8192-token unit, then the MoE layer on
    128-token chunks of the first new batch until the budget is spent. The
    rate is per token: 1 / (schedule time / N + layer time / sampled tokens)."""
    import oracle
    from paper_2410_17954_amd import synth
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max(int(i.get("num_threads", 1)) for i in threadpool_info()) \
            if threadpool_info() else 1
    except Exception:
        blas_threads = 1
    E, k = cfg["E"], cfg["k"]
    N = routes.shape[0]
    x = synth.values(inp["x"])
    wr = synth.values(inp["w_router"])
    wg, wu, wd = (synth.values(inp[n]) for n in ("w_gate", "w_up", "w_down"))
    t0 = time.perf_counter()
    perm, demand, info = oracle.schedule(routes, E)
    t_sched = time.perf_counter() - t0
    chunk = 128
    done = 0
    t_stage = {"route": 0.0, "permute": 0.0, "expert_ffn": 0.0, "combine": 0.0}
    slots = np.arange(E)
    while done < N and (sum(t_stage.values()) + t_sched) < budget_s:
        tok = perm[done:done + chunk]
        xb = np.asarray(x[tok], dtype=np.float64)
        # the composition of oracle.moe_layer, one stage at a time
        t1 = time.perf_counter()
        _, idx, w = oracle.route(xb, wr, k)
        t2 = time.perf_counter()
        offs, rop, _, xp = oracle.permute(xb, idx, E)
        t3 = time.perf_counter()
        yp, _ = oracle.expert_ffn(xp, offs, slots, wg, wu, wd)
        t4 = time.perf_counter()
        oracle.combine(np.nan_to_num(yp), idx, w, rop, None, slots, None, n_out=xb.shape[0])
        t5 = time.perf_counter()
        for name, dt in zip(t_stage, (t2 - t1, t3 - t2, t4 - t3, t5 - t4)):
            t_stage[name] += dt
        done += len(tok)
    t_layer = sum(t_stage.values())
    per_token = t_sched / N + t_layer / max(done, 1)
    rates = {"schedule": N / t_sched if t_sched > 0 else None}
    rates.update({n: (done / t if t > 0 else None) for n, t in t_stage.items()})
    return {"value": 1.0 / per_token, "unit": "tokens/s", "cores": blas_threads,
            "kind": "oracle",
            "sample": (f"scheduler over all {N} tokens ({t_sched:.2f} s) + MoE layer on "
                       f"{done} tokens in {chunk}-token chunks ({t_layer:.2f} s), float64"),
            "stage_tokens_per_s": rates,
            "affinity_cores": len(os.sched_getaffinity(0))}


if __name__ == "__main__":
    main()
