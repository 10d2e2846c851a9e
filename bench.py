#!/usr/bin/env python3
"""MoE-layer forward benchmark of the LorExperts / BTExperts hot path on one GPU.

Headline workload: the BTExperts tree layer (d=4096, f=1024, E=256 under 4
roots x 8 sub-dominants with rank-128 corrections, leaves with rank-64
corrections, top-8, bf16, T=8192 tokens, Gaussian router), the largest
configuration; the flat 30B-A3B-class prefill (d=2048, f=768, E=128 in 16
clusters of 8, rank 64, T=4096) and its decode-sized batch (T=64) follow as
extra objects, each with its own roofline (MFMA-bound prefill, HBM-bound
decode). Seeded synthetic inputs. One step = one call of the layer forward
(bucketing included, router excluded: ids and weights are inputs), with all
inputs resident in HBM; consecutive steps use independent copies of the
layer weights (round-robin over --rotate copies), so no step finds the
previous step's weights in the last-level cache.

Prints ONE JSON line: tokens/s of the whole layer, the roofline of the
dominant kernel (the longest per-step kernel; durations from HIP events
recorded around each launch on its launch stream, over K further steps) with
every kernel's own fraction beside it, the uncompressed dense-expert
comparator on the same shapes, and the CPU oracle timed on a bounded token
sample.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workloads 4,1,2]
  python bench.py --summarize-profile DIR --workloads I   (rocprofv3 CSVs -> profiles/)
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

PEAK_BF16_FLOPS = 2.5e15     # MI355X dense bf16 MFMA
PEAK_HBM_BYTES = 8.0e12      # MI355X HBM3E
RIDGE = PEAK_BF16_FLOPS / PEAK_HBM_BYTES


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workloads", default="4,1,2",
                    help="configurations to run, headline first (4 = BTExperts tree, 1 = flat prefill, "
                         "2 = flat decode, 3 = community-routed prefill, 5 = the paper's co-selected "
                         "cost example)")
    ap.add_argument("--config", type=int, default=None, help="run this one configuration only")
    ap.add_argument("--seed", type=int, default=None)
    ap.add_argument("--tokens", type=int, default=None, help="override the headline workload's token count")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense comparator")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-tokens", type=int, default=None,
                    help="tokens of the CPU oracle sample (default: 2048 for the tree, 4096 otherwise)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--rotate", type=int, default=5,
                    help="independent device copies of the layer weights, used round-robin by the "
                         "timed steps so that the 256 MB last-level cache cannot hold one step's weights "
                         "for the next (1 = a single copy)")
    ap.add_argument("--no-lo8", action="store_true",
                    help="no fp8 copy of the anchor down weights: the anchor down projection multiplies "
                         "both halves of its bf16 (hi, lo) input in bf16")
    ap.add_argument("--no-f16", action="store_true",
                    help="no fp16 copy of the anchor down weights: the anchor down projection keeps the fp8-lo "
                         "(or bf16 pair) path on every batch")
    ap.add_argument("--no-route", action="store_true", help="skip timing the GPU top-k router")
    ap.add_argument("--stage3", action="store_true",
                    help="also time Stage-3 factor production for one member at the flat workload's expert "
                         "shape (alignment cost, host assignment, randomized SVD factors of the three "
                         "projections), against the oracle on the host")
    ap.add_argument("--cluster", action="store_true",
                    help="also time router profiling + NPMI distance + k-medoids (Stages 1-2) on a calibration "
                         "routing of 64 x 2048 tokens, against the oracle on the host")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy 5 times (scales the "
                         "FETCH_SIZE / WRITE_SIZE counters to bytes)")
    ap.add_argument("--summarize-profile", default=None, metavar="DIR",
                    help="no GPU work: summarise the rocprofv3 runs under DIR (see profile_commands) into "
                         "profiles/ for the one workload given by --workloads")
    a = ap.parse_args()
    if a.config is not None:
        a.workloads = str(a.config)
    a.workload_list = [int(v) for v in a.workloads.split(",") if v.strip()]
    return a


def copy_calibration(torch):
    n = 1 << 30
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 5
    print(json.dumps({"copy_bytes": n, "ms": round(ms, 4), "read_plus_write_GBps": round(2 * n / ms / 1e6, 1)}),
          flush=True)


def kernel_work(name, P, rows, touched):
    """Algorithmic (flops, bytes) of one launch of kernel ``name`` (a batched
    launch "a+b" counts the sum of its parts).

    rows[l] / touched[l]: rows doing work and distinct nodes touched at level l.
    Bytes: the weights the launch must read (touched nodes once, bf16) plus
    its algorithmic activation input read once (x: T*d bf16; the per-row
    fp32 intermediates are not counted).
    """
    if "+" in name:
        parts = [kernel_work(n, P, rows, touched) for n in name.split("+")]
        return sum(p[0] for p in parts), sum(p[1] for p in parts)
    d, f, T = P["d"], P["f"], P["T"]
    if name in ("lowrank_gate_up_out_merged", "lowrank_down_out_merged", "lowrank_down_in_merged"):
        # one launch doing every correction level's product of that kind
        tag = {"lowrank_gate_up_out_merged": "lowrank_gate_up_out_l", "lowrank_down_out_merged": "lowrank_down_out_l",
               "lowrank_down_in_merged": "lowrank_down_in_l"}[name]
        parts = [kernel_work(f"{tag}{l}", P, rows, touched) for l in range(1, len(P["ranks"]))]
        return sum(p[0] for p in parts), sum(p[1] for p in parts)
    if name == "anchor_gate_up":
        return 4 * d * f * rows[0], 2 * f * d * 2 * touched[0] + T * d * 2
    if name == "anchor_down":
        return 2 * d * f * rows[0], d * f * 2 * touched[0]
    for tag in ("lowrank_gate_up_in_l", "lowrank_gate_up_out_l", "lowrank_down_in_l",
                "lowrank_down_out_l"):
        if name.startswith(tag):
            l = int(name[len(tag):])
            r = P["ranks"][l]
            if tag == "lowrank_gate_up_in_l":
                return 4 * r * d * rows[l], 2 * r * d * 2 * touched[l] + T * d * 2
            if tag == "lowrank_gate_up_out_l":
                return 4 * r * f * rows[l], 2 * f * r * 2 * touched[l]
            if tag == "lowrank_down_in_l":
                return 2 * r * f * rows[l], r * f * 2 * touched[l]
            return 2 * r * d * rows[l], d * r * 2 * touched[l]
    return 0, 0


def source_sha():
    h = hashlib.sha256()
    for fn in sorted(os.listdir(os.path.join(ROOT, "paper_2608_07814_amd", "csrc"))):
        with open(os.path.join(ROOT, "paper_2608_07814_amd", "csrc", fn), "rb") as fh:
            h.update(fn.encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_traffic(kernel, workload):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        db = json.load(open(path))
        ent = db.get(f"{kernel}@{workload}")
        if not ent or ent.get("source_sha") != source_sha():
            return None
        return ent["fetch_bytes_per_launch"] + ent["write_bytes_per_launch"]
    except Exception:
        return None


def clone_layer(dl):
    """Independent device copy of a DeviceLayer's weights (same routing structure)."""
    import dataclasses
    from paper_2608_07814_amd import lorex as lx
    names = ("a_gate", "b_gate", "a_up", "b_up", "a_down", "b_down") + lx.FACTOR_F16 + lx.FACTOR_PAD
    levels = [dataclasses.replace(lv, **{n: getattr(lv, n).clone() for n in names if getattr(lv, n) is not None})
              for lv in dl.levels]
    copies = {n: getattr(dl, n).clone() for n in ("anchor_down_f8", "anchor_down_f8_scale", "anchor_down_f16",
                                                   "anchor_down_f16_exp") if getattr(dl, n) is not None}
    return dataclasses.replace(dl, anchor_gate=dl.anchor_gate.clone(), anchor_up=dl.anchor_up.clone(),
                               anchor_down=dl.anchor_down.clone(), levels=levels, **copies)


def rotating(calls):
    """One step = the next prepared call, round-robin over the weight copies."""
    state = [0]

    def step():
        calls[state[0]]()
        state[0] = (state[0] + 1) % len(calls)
    return step


def step_percentiles(fn, steps, torch):
    """p10 / median / p90 of single-step times (events around each step)."""
    import numpy as np
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    t = np.array([a.elapsed_time(b) for a, b in ev])
    return dict(p10=round(float(np.percentile(t, 10)), 4), median=round(float(np.median(t)), 4),
                p90=round(float(np.percentile(t, 90)), 4))


def graph_timing(make_call, copies, a, torch):
    """The same forward captured once per weight copy into a HIP graph (torch's
    CUDAGraph API) and replayed in rotation: what a serving loop that cannot
    afford per-kernel launch latency runs. Returns ms per step."""
    graphs = []
    for c in copies:
        call = make_call(c)
        call()  # the first call on a stream outside capture (plans, device queries)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            make_call(c)()
        graphs.append(g)
    it = [0]

    def step():
        graphs[it[0] % len(graphs)].replay()
        it[0] += 1
    ms, _ = time_steps(step, a.steps, a.warmup, torch)
    return dict(ms_per_step=round(ms, 4), note="HIP graph replay of the same forward (launch latency removed)")


def time_steps(fn, steps, warmup, torch):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    return e0.elapsed_time(e1) / steps, wall


def bench_clustering(torch, np, lx, a):
    """Stages 1-2 on the GPU: firing / co-activation counts and the NPMI
    distance over a calibration routing (64 sequences x 2048 tokens, 128
    experts, top-8, community-structured: 16 groups of 8, 70% of slots in the
    token's home group), then k-medoids to 64 clusters (k = E / 2). Timed with
    events around the two calls; the oracle runs the same steps on the host."""
    from lxsynth import route_community
    from oracle import cluster as K
    E, k, N, C = 128, 8, 64 * 2048, 64
    members = [list(range(g * 8, g * 8 + 8)) for g in range(16)]
    ids = route_community(N, members, k, 0.7, 5).topk_ids
    ids_d = torch.from_numpy(np.ascontiguousarray(ids, np.int32)).cuda()
    fire, pair, dist = lx.coact_distance(ids_d, E)
    lx.kmedoids(dist, fire, C)
    torch.cuda.synchronize()
    reps = 20
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    e0.record()
    for _ in range(reps):
        lx.coact_distance(ids_d, E)
    e1.record()
    outs = None
    for _ in range(reps):
        outs = lx.kmedoids(dist, fire, C)
    e2.record()
    torch.cuda.synchronize()
    it = int(outs[3].cpu()[0])
    t0 = time.perf_counter()
    f0, p0 = K.coact_counts(ids, E)
    d0 = K.npmi_distance(f0, p0, N)
    K.kmedoids(d0, f0, C)
    cpu_s = time.perf_counter() - t0
    same = bool(np.array_equal(outs[0].cpu().numpy(), K.kmedoids(dist.cpu().numpy(),
                                                                 fire.cpu().numpy().view(np.uint32), C)[0]))
    return dict(tokens=N, E=E, k=k, C=C, coact_distance_us=round(e0.elapsed_time(e1) / reps * 1e3, 2),
                kmedoids_us=round(e1.elapsed_time(e2) / reps * 1e3, 2), kmedoids_update_rounds=it,
                ids_bytes=N * k * 4, cpu_oracle_s=round(cpu_s, 2), clusters_match_oracle=same)


def bench_stage3(torch, np, lx, layer):
    """Stage 3 for one member at the layer's expert shape (d, f, rank r,
    oversampling 10, 2 power iterations): a dominant and a member that is the
    dominant plus rank-r corrections with its neurons shuffled, both bf16.
    GPU: alignment cost, host assignment, factors of gate, up and down, and
    the activation-weighted factors on calibration activations; the oracle
    runs the same steps on the host."""
    from lxsynth import f32_to_bf16_bits
    from oracle import stage3 as S
    d, f, r, p = layer.d, layer.f, layer.levels[0].rank, 10
    rng = np.random.default_rng(3)
    s = np.sqrt(0.3 / np.sqrt(r * d))
    dom64 = [rng.standard_normal(sh) / np.sqrt(d) for sh in ((f, d), (f, d), (d, f))]
    cor = [(rng.standard_normal((a, r)) * s) @ (rng.standard_normal((r, b)) * s) for a, b in ((f, d), (f, d), (d, f))]
    inv = np.argsort(rng.permutation(f))
    bf = lambda x: f32_to_bf16_bits(np.asarray(x, np.float32))
    dom = [bf(x) for x in dom64]
    mem = [bf((dom64[0] + cor[0])[inv]), bf((dom64[1] + cor[1])[inv]), bf((dom64[2] + cor[2])[:, inv])]
    dev = lambda b: torch.from_numpy(b.view(np.int16)).cuda().view(torch.bfloat16)
    ddom, dmem = [dev(x) for x in dom], [dev(x) for x in mem]
    oms = [rng.standard_normal((w.shape[1], r + p)) for w in dom]
    doms = [torch.from_numpy(o).cuda() for o in oms]

    def factors(pd):
        for i in range(3):
            lx.lowrank_factors(ddom[i], dmem[i], r, doms[i], q=2, perm=pd, perm_axis=1 if i == 2 else 0)

    factors(torch.from_numpy(lx.assign(lx.align_cost(tuple(ddom), tuple(dmem)).cpu().numpy())[0]).cuda())  # warm-up
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    ev[0].record()
    cost = lx.align_cost(tuple(ddom), tuple(dmem))
    ev[1].record()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    perm, _ = lx.assign(cost.cpu().numpy())
    t_assign = time.perf_counter() - t0
    pd = torch.from_numpy(perm).cuda()
    torch.cuda.synchronize()
    ev[2].record()
    factors(pd)
    ev[3].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    perm0, _ = S.assign(S.align_cost(dom, mem, "bf16"))
    for i in range(3):
        S.factors(S.aligned_residual(dom[i], mem[i], perm0, 1 if i == 2 else 0, "bf16"), oms[i], r, q=2)
    cpu_s = time.perf_counter() - t1
    # activation-weighted fit of the same three projections on 4096
    # calibration rows (bf16 Gaussian activations of each projection's input)
    n_cal = 4096
    xs = [bf(rng.standard_normal((n_cal, w.shape[1]))) for w in dom]
    dxs = [dev(x) for x in xs]
    woms = [rng.standard_normal((n_cal, r + p)) for _ in dom]
    dwoms = [torch.from_numpy(o).cuda() for o in woms]

    def weighted(pd_):
        for i in range(3):
            lx.weighted_factors(ddom[i], dmem[i], r, dxs[i], dwoms[i], q=2, perm=pd_, perm_axis=1 if i == 2 else 0)

    weighted(pd)  # warm-up
    torch.cuda.synchronize()
    evw = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    evw[0].record()
    weighted(pd)
    evw[1].record()
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for i in range(3):
        S.weighted_factors(S.aligned_residual(dom[i], mem[i], perm0, 1 if i == 2 else 0, "bf16"),
                           S.to_f64(xs[i], "bf16"), woms[i], r, q=2)
    cpu_w = time.perf_counter() - t2
    return dict(d=d, f=f, r=r, oversampling=p, power_iterations=2,
                weighted_fit_calibration_rows=n_cal,
                weighted_factors_3_projections_us=round(evw[0].elapsed_time(evw[1]) * 1e3, 1),
                weighted_cpu_oracle_s=round(cpu_w, 2),
                align_cost_us=round(ev[0].elapsed_time(ev[1]) * 1e3, 1),
                align_cost_gflop=round(2 * f * f * 3 * d / 1e9, 2),
                assign_host_ms=round(t_assign * 1e3, 2),
                factors_3_projections_us=round(ev[2].elapsed_time(ev[3]) * 1e3, 1),
                permutation_matches_oracle=bool(np.array_equal(perm, perm0)),
                cpu_oracle_s=round(cpu_s, 2))


def roofline_of(name, P, rows, touched, avg_s):
    """Roofline of one kernel launch: bound by its own arithmetic intensity
    (algorithmic FLOPs / algorithmic bytes against the ridge point)."""
    fl, by = kernel_work(name, P, rows, touched)
    if not fl and not by:
        return None
    if fl and fl / max(by, 1) >= RIDGE:
        return dict(bound="mfma", achieved=round(fl / avg_s / 1e12, 2), peak=PEAK_BF16_FLOPS / 1e12,
                    unit="TFLOP/s", frac=round(fl / avg_s / PEAK_BF16_FLOPS, 4),
                    alg_flops_per_launch=fl, alg_bytes_per_launch=by)
    return dict(bound="hbm", achieved=round(by / avg_s / 1e9, 1), peak=PEAK_HBM_BYTES / 1e9,
                unit="GB/s", frac=round(by / avg_s / PEAK_HBM_BYTES, 4),
                alg_flops_per_launch=fl, alg_bytes_per_launch=by)


def run_workload(cfg_index, a, torch, np, lx, headline):
    """Time one configuration; returns (result dict, problem, prepared state)."""
    from lxsynth import make_problem
    from paper_2608_07814_amd import accounting as acc

    p = make_problem(cfg_index, seed=a.seed, T=a.tokens if headline else None)
    cfg = p.cfg
    T, k = p.T, p.k
    layer = p.layer
    dl = lx.to_device(layer, lo8=not a.no_lo8, f16=not a.no_f16)
    if layer.dtype == "bf16":
        xd = torch.from_numpy(p.x.view(np.int16)).cuda().view(torch.bfloat16)
    else:
        xd = torch.from_numpy(p.x).cuda()
    ids = torch.from_numpy(p.routing.topk_ids).cuda()
    w = torch.from_numpy(p.routing.topk_weights).cuda()
    kind = "flat" if layer.n_levels == 1 else "tree"
    ws = lx.alloc_workspace(dl, T, k, kind)
    out = torch.empty(T, layer.d, dtype=torch.float32, device="cuda")
    workload = cfg["name"] if not (headline and a.tokens) else f"{cfg['name']} at T={T}"

    # bucket counts for the algorithmic counts (before any timed region)
    n_lv = layer.n_levels
    rows, touched = [], []
    for l in range(n_lv + 1):
        _, off, _ = lx.bucket(dl, ids, l, workspace=ws)
        cnt = np.diff(off.cpu().numpy().astype(np.int64))
        if l > 0:
            cnt = np.where(layer.levels[l - 1].factor_of >= 0, cnt, 0)
        rows.append(int(cnt.sum()))
        touched.append(int((cnt > 0).sum()))
    ranks = [0] + [lv.rank for lv in layer.levels]
    lvrows = [acc.LevelRows(rank=ranks[l], rows=rows[l], nodes_touched=touched[l])
              for l in range(n_lv + 1)]
    work = acc.algorithmic_counts(layer.d, layer.f, lvrows, T, k)
    P = dict(d=layer.d, f=layer.f, T=T, ranks=ranks)

    copies = [dl] + [clone_layer(dl) for _ in range(max(a.rotate, 1) - 1)]
    call = rotating([lx.PreparedCall(c, xd, ids, w, out, ws, kind) for c in copies])

    ms, wall = time_steps(call, a.steps, a.warmup, torch)
    tokens_per_s = T / (ms * 1e-3)
    pct = step_percentiles(call, min(a.steps, 100), torch)
    graph = graph_timing(lambda c: lx.PreparedCall(c, xd, ids, w, out, ws, kind), copies, a, torch)

    # per-kernel durations: HIP events around every launch, on its stream
    lx.profile_reset()
    lx.profile_enable(True)
    for _ in range(a.steps):
        call()
    torch.cuda.synchronize()
    prof = lx.profile_read()  # launch order of one forward
    lx.profile_enable(False)

    kernels = {}
    tot_all = sum(v[1] for v in prof.values())
    for name, (n, tot) in prof.items():
        avg_s = tot / max(n, 1) * 1e-3
        rf = roofline_of(name, P, rows, touched, avg_s)
        kernels[name] = dict(launches=n, avg_us=round(avg_s * 1e6, 3), share=round(tot / tot_all, 4),
                             bound=rf["bound"] if rf else None, frac=rf["frac"] if rf else None,
                             achieved=rf["achieved"] if rf else None, unit=rf["unit"] if rf else None)
    # the dominant kernel: the longest per step
    dom = max(prof.items(), key=lambda kv: kv[1][1])[0]
    dom_avg_s = prof[dom][1] / prof[dom][0] * 1e-3
    roof = roofline_of(dom, P, rows, touched, dom_avg_s) or dict(bound="alu", achieved=None, peak=None, unit=None,
                                                                 frac=None)
    roof["kernel"] = dom
    roof["avg_launch_us"] = round(dom_avg_s * 1e6, 3)
    roof["traffic"] = load_traffic(dom, workload)
    roof["launches_per_step"] = len(prof)

    step_s = ms * 1e-3
    layer_perf = dict(alg_gflop=round(work["flops"] / 1e9, 2), alg_mbytes=round(work["bytes"] / 1e6, 1),
                      alg_tflops=round(work["flops"] / step_s / 1e12, 2),
                      frac_bf16_peak=round(work["flops"] / step_s / PEAK_BF16_FLOPS, 4),
                      alg_gbps=round(work["bytes"] / step_s / 1e9, 1),
                      frac_hbm_peak=round(work["bytes"] / step_s / PEAK_HBM_BYTES, 4),
                      rows_per_level=rows, nodes_touched=touched,
                      serial_kernel_us=round(tot_all / a.steps * 1e3, 2))

    dense = None
    if not a.no_dense and kind in ("flat", "tree"):
        # uncompressed comparator: every expert = its anchor + the A B of every
        # factor-carrying node on its path, rounded to bf16 (setup, untimed)
        def reconstruct(anchor, an, bn):
            wt = anchor.float()
            for lv in dl.levels:
                wt = wt[lv.parent.long()]
                fo = lv.factor_of.long()
                m = fo >= 0
                if bool(m.any()):
                    fi = fo[m]
                    wt[m] += torch.bmm(getattr(lv, an)[fi].float(), getattr(lv, bn)[fi].float())
            return wt.bfloat16().contiguous()

        dd = lx.DeviceLayer(E=layer.E, d=layer.d, f=layer.f, dtype="bf16",
                            anchor_gate=reconstruct(dl.anchor_gate, "a_gate", "b_gate"),
                            anchor_up=reconstruct(dl.anchor_up, "a_up", "b_up"),
                            anchor_down=reconstruct(dl.anchor_down, "a_down", "b_down"), levels=[])
        torch.cuda.empty_cache()
        if not a.no_lo8:
            dd = lx.attach_down_f8(dd)
        if not a.no_f16:
            dd = lx.attach_down_f16(dd)
        wsd = lx.alloc_workspace(dd, T, k, "dense")
        outd = torch.empty_like(out)
        dcopies = [dd] + [clone_layer(dd) for _ in range(max(a.rotate, 1) - 1)]
        dcall = rotating([lx.PreparedCall(c, xd, ids, w, outd, wsd, "dense") for c in dcopies])
        dms, _ = time_steps(dcall, a.steps, a.warmup, torch)
        # algorithmic work of the dense layer: every touched expert's three
        # matrices once, 6df FLOPs per routed slot
        ids_np = p.routing.topk_ids
        valid = ids_np[(ids_np >= 0) & (ids_np < layer.E)]
        e_touched = int(np.unique(valid).size)
        d_flops = 6 * layer.d * layer.f * int(valid.size)
        d_bytes = 3 * layer.d * layer.f * 2 * e_touched + T * layer.d * (2 + 4) + T * k * 8
        dense = dict(tokens_per_s=round(T / (dms * 1e-3), 1), ms_per_step=round(dms, 4),
                     speedup_of_compressed=round(dms / ms, 3),
                     alg_gflop=round(d_flops / 1e9, 2), alg_mbytes=round(d_bytes / 1e6, 1),
                     experts_touched=e_touched,
                     alg_flops_ratio=round(d_flops / work["flops"], 4),
                     alg_bytes_ratio=round(d_bytes / work["bytes"], 4))
        if cfg.get("routing") == "coselect":
            # per-token cost ratio of Sec. 5 (k experts sharing one dominant)
            dense["analytic_speedup"] = round(acc.closed_form_speedup(k, layer.f, layer.d, ranks[1]), 4)
        del dd, dcopies, dcall, wsd, outd
        torch.cuda.empty_cache()

    routed = None
    if not a.no_route and layer.dtype == "bf16" and layer.d % 128 == 0 and layer.E <= 512:
        # the unchanged top-k router on the GPU (lx_route_topk), alone and
        # chained with the forward on one stream (ids and weights stay in HBM)
        from lxsynth import make_router
        wr = torch.from_numpy(make_router(layer.d, layer.E, "bf16", p.seed).view(np.int16)).cuda() \
            .view(torch.bfloat16)
        rids = torch.empty(T, k, dtype=torch.int32, device="cuda")
        rw = torch.empty(T, k, dtype=torch.float32, device="cuda")
        rws = lx.route_workspace(T, layer.d, layer.E)
        lx.route_topk(xd, wr, k, ids=rids, weights=rw, workspace=rws)  # argument checks once
        rargs = (xd.data_ptr(), wr.data_ptr(), lx.LX_BF16, T, layer.d, layer.E, k, rids.data_ptr(),
                 rw.data_ptr(), rws.data_ptr(), rws.numel(), None)
        rfn = lx.lib().lx_route_topk
        route = lambda: rfn(*rargs)
        rms, _ = time_steps(route, a.steps, a.warmup, torch)
        fwd = [lx.PreparedCall(c, xd, rids, rw, out, ws, kind) for c in copies]
        chain = rotating([(lambda f=f: (route(), f())) for f in fwd])
        cms, _ = time_steps(chain, a.steps, a.warmup, torch)
        # the router's top-k fused into the bucketing (lx_route_moe_forward_tree)
        import ctypes
        L = lx.lib()
        fused = []
        for c in copies:
            desc = c.tree_struct()
            nws = int(L.lx_route_moe_tree_workspace_bytes(ctypes.byref(desc), T, k))
            fws = torch.empty(nws, dtype=torch.uint8, device="cuda")
            args = (ctypes.byref(desc), T, k, xd.data_ptr(), wr.data_ptr(), rids.data_ptr(), rw.data_ptr(),
                    out.data_ptr(), lx.LX_F32, fws.data_ptr(), nws, None)
            fused.append((desc, fws, args))
        ffn = L.lx_route_moe_forward_tree
        fcall = rotating([(lambda a_=f[2]: ffn(*a_)) for f in fused])
        fcall()
        torch.cuda.synchronize()
        fms, _ = time_steps(fcall, a.steps, a.warmup, torch)
        routed = dict(router_us=round(rms * 1e3, 3),
                      router_gflop=round(2 * T * layer.d * layer.E / 1e9, 3),
                      router_and_forward_ms=round(cms, 4),
                      router_and_forward_tokens_per_s=round(T / (cms * 1e-3), 1),
                      fused_router_forward_ms=round(fms, 4),
                      fused_router_forward_tokens_per_s=round(T / (fms * 1e-3), 1),
                      fused_saving_us=round((cms - fms) * 1e3, 2))
        del fused, fcall

    graph["tokens_per_s"] = round(T / (graph["ms_per_step"] * 1e-3), 1)
    res = dict(workload=workload, tokens_per_s=round(tokens_per_s, 1), ms_per_step=round(ms, 4), step_ms=pct,
               graph=graph,
               wall_s_timed=round(wall, 3), weight_copies=len(copies),
               config={"workload": workload, "T": T, "d": layer.d, "f": layer.f, "E": layer.E, "k": k,
                       "anchors": layer.n_anchors, "ranks": ranks[1:], "layer": kind, "seed": p.seed,
                       "out_dtype": "f32",
                       "anchor_down_copies": [c for c, off in (("fp8 lo (block-scaled)", a.no_lo8),
                                                               ("fp16 (token-scaled sums)", a.no_f16)) if not off],
                       "factor_copies": [] if a.no_f16 else ["fp16 (tile-scaled low-rank intermediates)"]},
               roofline=roof, layer_roofline=layer_perf, kernels=kernels, dense_comparator=dense,
               gpu_router=routed)
    del copies, call
    return res, p


def cpu_baseline(p, a, np):
    """The fp64 oracle on a bounded sample of the workload (host cores)."""
    from threadpoolctl import threadpool_info, threadpool_limits
    from oracle import moe as O
    layer = p.layer
    T = p.T
    # a bounded sample: the first n tokens, repeated until ~cpu_seconds of CPU work
    n = min(a.cpu_tokens or (2048 if layer.n_levels > 1 else 4096), T)
    reps, t0 = 0, time.perf_counter()
    while True:
        O.moe_forward(layer, p.x, p.routing.topk_ids, p.routing.topk_weights, tokens=np.arange(n))
        reps += 1
        dt = time.perf_counter() - t0
        if dt >= a.cpu_seconds or reps >= 64:
            break
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    # one core: a short sample (few tokens, one pass; the oracle reconstructs
    # every expert the sample touches, which dominates at small samples)
    n1 = max(1, min(n // 4, 16 if layer.n_levels > 1 else 1024))
    with threadpool_limits(limits=1):
        t1 = time.perf_counter()
        O.moe_forward(layer, p.x, p.routing.topk_ids, p.routing.topk_weights, tokens=np.arange(n1))
        dt1 = time.perf_counter() - t1
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            model = next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), None)
    except OSError:
        pass
    return dict(value=round(n * reps / dt, 2), unit="tokens/s", cores=int(threads), kind="oracle",
                sample=f"first {n} of {T} tokens of the same workload, {reps} passes, fp64 numpy "
                       f"oracle (dense reconstruction of every routed expert + per-slot SwiGLU), "
                       f"{dt:.1f} s wall", nproc=os.cpu_count(), cpu_model=model,
                single_core_value=round(n1 / dt1, 2),
                single_core_sample=f"first {n1} tokens, one pass, {dt1:.1f} s wall")


def main():
    a = parse()
    if a.summarize_profile:
        summarize_profile(a)
        return
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {a.gpus}); this implementation has no "
              "multi-GPU path.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2608_07814_amd import lorex as lx

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(3)
    torch.cuda.set_device(0)
    if a.copy_calibration:
        copy_calibration(torch)
        return
    results, head_p = [], None
    for i, c in enumerate(a.workload_list):
        print(f"[bench] workload {c}", file=sys.stderr, flush=True)
        r, p = run_workload(c, a, torch, np, lx, headline=(i == 0))
        results.append(r)
        if i == 0:
            head_p = p
        else:
            del p
        torch.cuda.empty_cache()
    head = results[0]

    clustering = None
    if a.cluster:
        clustering = bench_clustering(torch, np, lx, a)
    stage3 = None
    if a.stage3:
        from lxsynth import make_problem
        stage3 = bench_stage3(torch, np, lx, make_problem(1, T=16).layer)

    cpu = None
    if not a.no_cpu:
        print("[bench] cpu baseline", file=sys.stderr, flush=True)
        cpu = cpu_baseline(head_p, a, np)

    res = {
        "metric": "MoE-layer tokens/s (LorExperts / BTExperts forward, bucketing included)",
        "value": head["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": head["ms_per_step"],
        "step_ms": head["step_ms"],
        "graph": head["graph"],
        "weight_copies": head["weight_copies"],
        "wall_s_timed": head["wall_s_timed"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; Gaussian, community or co-selected routing; random-init weights)",
        "config": head["config"],
        "roofline": head["roofline"],
        "layer_roofline": head["layer_roofline"],
        "kernels": head["kernels"],
        "dense_comparator": head["dense_comparator"],
        "gpu_router": head["gpu_router"],
        "workloads": {r["workload"]: {k: r[k] for k in ("tokens_per_s", "ms_per_step", "step_ms", "graph", "roofline",
                                                         "layer_roofline", "kernels", "dense_comparator",
                                                         "gpu_router", "config")}
                      for r in results[1:]},
        "clustering": clustering,
        "stage3": stage3,
        "cpu_baseline": cpu,
        "kernel_sources_sha": source_sha(),
    }
    print(json.dumps(res), flush=True)


# ------------------------------------------------------------------ profiles
def profile_commands(c):
    """The rocprofv3 runs a profile summary is made from (run from the
    repository root on one MI355X after `cd /tmp && export TMPDIR=/tmp`;
    OUT is any output directory)."""
    b = f"python3 bench.py --workloads {c} --no-cpu --no-dense --no-route"
    return [
        ("trace", f"rocprofv3 --kernel-trace --stats -f csv -d OUT/trace_c{c} -o t -- {b} --steps 20 --warmup 5"),
        ("FETCH_SIZE", f"rocprofv3 --pmc FETCH_SIZE -f csv -d OUT/FETCH_SIZE_c{c} -o p -- {b} --steps 2 --warmup 1 "
                       f"--rotate 1"),
        ("WRITE_SIZE", f"rocprofv3 --pmc WRITE_SIZE -f csv -d OUT/WRITE_SIZE_c{c} -o p -- {b} --steps 2 --warmup 1 "
                       f"--rotate 1"),
        ("copy FETCH_SIZE", "rocprofv3 --pmc FETCH_SIZE -f csv -d OUT/FETCH_SIZE_copy -o p -- python3 bench.py "
                            "--copy-calibration"),
        ("copy WRITE_SIZE", "rocprofv3 --pmc WRITE_SIZE -f csv -d OUT/WRITE_SIZE_copy -o p -- python3 bench.py "
                            "--copy-calibration"),
    ]


def _csv(path):
    import csv
    with open(path) as fh:
        return list(csv.DictReader(fh))


def _find(d, sub, name):
    for root, _, files in os.walk(os.path.join(d, sub)):
        for f in files:
            if f.endswith(name):
                return os.path.join(root, f)
    raise FileNotFoundError(f"{sub}/*{name} under {d}")


def _counter_per_dispatch(path):
    by = {}
    for r in _csv(path):
        i = int(r["Dispatch_Id"])
        ent = by.setdefault(i, [r["Kernel_Name"], 0.0])
        ent[1] += float(r["Counter_Value"])
    return [(by[i][0], by[i][1]) for i in sorted(by)]


def summarize_profile(a):
    """rocprofv3 output (profile_commands) -> profiles/<workload>.md and the
    workload's entries of profiles/traffic.json. The library's kernels are the
    dispatches whose names carry its namespace; the last K x n of them are the
    benchmark's serialised per-kernel timing pass (K steps of n launches, in
    the launch order the benchmark's own JSON line lists)."""
    import statistics
    from lxsynth import config as _cfg
    c = a.workload_list[0]
    d = a.summarize_profile
    wl = _cfg(c)["name"]
    # the benchmark's JSON line of the trace run names the launches in order
    line = None
    with open(os.path.join(d, f"trace_c{c}.log")) as fh:
        for ln in fh:
            if ln.startswith("{"):
                line = json.loads(ln)
    if line is None:
        raise RuntimeError("no JSON line in the trace run's log")
    roles = list(line["kernels"].keys())
    n = len(roles)
    steps = int(line["steps"])
    tr = sorted(_csv(_find(d, f"trace_c{c}", "kernel_trace.csv")), key=lambda r: int(r["Dispatch_Id"]))
    lxr = [r for r in tr if "lx::" in r["Kernel_Name"]]
    ser = lxr[-steps * n:]
    dur = {r: [] for r in roles}
    for i, row in enumerate(ser):
        dur[roles[i % n]].append((int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) / 1e3)
    # whole forwards of the timed loops before the serialised pass (first to
    # last dispatch of each group of n)
    warm = int(line["warmup"])
    n_timed = warm + steps + min(steps, 100)
    timed = lxr[max(0, len(lxr) - steps * n - n_timed * n): len(lxr) - steps * n]
    fwd = []
    for g in range(len(timed) // n):
        grp = timed[g * n:(g + 1) * n]
        fwd.append((max(int(x["End_Timestamp"]) for x in grp) - min(int(x["Start_Timestamp"]) for x in grp)) / 1e3)

    def scale(ctr):
        vals = [v for nm, v in _counter_per_dispatch(_find(d, f"{ctr}_copy", "counter_collection.csv"))
                if "copy" in nm.lower() or "elementwise" in nm.lower()]
        return (1 << 30) / (statistics.median(vals) * 1024.0)

    sc = {ctr: scale(ctr) for ctr in ("FETCH_SIZE", "WRITE_SIZE")}
    cnt = {}
    for ctr in ("FETCH_SIZE", "WRITE_SIZE"):
        rows = [(nm, v) for nm, v in _counter_per_dispatch(_find(d, f"{ctr}_c{c}", "counter_collection.csv"))
                if "lx::" in nm]
        per = {r: [] for r in roles}
        # the counter runs end, like the trace run, with the serialised pass
        # of K forwards (same launch sequence)
        k_ctr = 2
        tail = rows[len(rows) - k_ctr * n:]
        for i, (_, v) in enumerate(tail):
            per[roles[i % n]].append(v * 1024.0 * sc[ctr])
        cnt[ctr] = {r: statistics.mean(v) if v else None for r, v in per.items()}
    # the sources the profiled run was built from (its JSON line records them)
    sha = line.get("kernel_sources_sha") or source_sha()
    lines = [f"# rocprofv3 kernel summary: {wl}", "",
             f"Kernel sources sha256[:16] = `{sha}`.", "",
             "Commands (from the repository root on one MI355X, after `cd /tmp && export TMPDIR=/tmp`; "
             "OUT is the output directory), then "
             f"`python3 bench.py --summarize-profile OUT --workloads {c}`:", ""]
    lines += [f"- {what}: `{cmd}`" for what, cmd in profile_commands(c)]
    lines += ["", f"FETCH_SIZE scale = {sc['FETCH_SIZE']:.4f} bytes per counted byte, WRITE_SIZE scale = "
                  f"{sc['WRITE_SIZE']:.4f} (a plain 1 GiB device copy reads and writes exactly 1 GiB).", "",
              f"Per-kernel rows: the last {steps} forwards of the trace (the benchmark's serialised per-kernel "
              f"timing pass, {n} launches each). Whole forward (first dispatch start to last dispatch end) over "
              f"the {len(fwd)} forwards of the timed loops: median {statistics.median(fwd):.1f} us, min "
              f"{min(fwd):.1f} us." if fwd else "", "",
              "| kernel (role) | dispatches | avg us | min us | max us | roofline of the benchmark run "
              "| HBM read MB/launch | HBM write MB/launch |",
              "|---|---:|---:|---:|---:|---|---:|---:|"]
    db_path = os.path.join(ROOT, "profiles", "traffic.json")
    db = json.load(open(db_path)) if os.path.exists(db_path) else {}
    db = {k: v for k, v in db.items() if not k.endswith("@" + wl)}
    tot = 0.0
    for r in roles:
        v = dur[r]
        kr = line["kernels"][r]
        rf = f"{kr['frac']:.3f} of {kr['bound']} ({kr['achieved']} {kr['unit']})" if kr.get("frac") else "-"
        fb, wb = cnt["FETCH_SIZE"][r], cnt["WRITE_SIZE"][r]
        tot += statistics.mean(v)
        lines.append(f"| {r} | {len(v)} | {statistics.mean(v):.2f} | {min(v):.2f} | {max(v):.2f} | {rf} | "
                     f"{fb / 1e6:.1f} | {wb / 1e6:.1f} |")
        db[f"{r}@{wl}"] = dict(avg_us=round(statistics.mean(v), 3), fetch_bytes_per_launch=int(fb),
                               write_bytes_per_launch=int(wb), source_sha=sha)
    dom = line["roofline"]["kernel"]
    lines += ["", f"Sum of per-role averages (serialised): {tot:.1f} us. Longest kernel in this trace: "
                  f"{max(roles, key=lambda r: statistics.mean(dur[r]))} "
                  f"({max(statistics.mean(dur[r]) for r in roles):.2f} us); the benchmark's dominant kernel: {dom}.",
              ""]
    out = os.path.join(ROOT, "profiles", f"forward_{wl}.md")
    with open(out, "w") as fh:
        fh.write("\n".join(lines))
    with open(db_path, "w") as fh:
        json.dump(dict(sorted(db.items())), fh, indent=1)
    print(out)


if __name__ == "__main__":
    main()
