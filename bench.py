"""SparSTAR hot-path benchmark on one MI355X.

A step is one full pass of the hot path over the 720p final-scale workload
(batch 1, 24 heads, head dim 128, 64-token blocks, 72,000 queries, 144,512 keys
= 72,000 preceding-clip + 512 text + 72,000 current, text blocks forced, 25%
budget): block pooling + scores + top-k selection (sparstar_score_blocks), then
the block-sparse attention forward (sparstar_sparse_attn_fwd).  Inputs are
seeded synthetic bf16 tensors already resident in HBM.

Prints ONE JSON line.  `value` is effective TFLOP/s of the step: FLOPs executed
on the selected blocks (4 * 64 * 64 * D per (query block, listed key block))
divided by the step time.  `roofline` reports the sparse forward call against
the bf16 MFMA peak, timed with HIP events on the stream it runs on; `traffic`
comes from the committed rocprofv3 counter summary when it was taken on the
current kernel source.  Also reported: the in-house dense forward on the same
shape, the retained attention mass of the selection against the token-wise
top-K bound (Section 4's diagnostic, on the synthetic inputs), the density sweep
(per-head budgets around 10 / 25 / 50%), the five-scale clip pyramid, and the
float64 CPU oracle timed on a bounded sample (`cpu_baseline`).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "ms and effective TFLOP/s per sparse attention call at 72k-query 720p scale"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "attn_fwd_sparse_720p_hbm.md")
ATTN_SOURCE = os.path.join(ROOT, "paper_2608_10519_amd", "csrc", "attn_fwd.hip")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def executed_flops(num_blocks: np.ndarray, last_entries: np.ndarray, lq: int, lk: int, block: int,
                   d: int) -> float:
    """Sum over (b, h, i) of 4 * rows_i * keys(A_i) * D, where rows_i is the
    number of real query rows of block i and keys(A_i) counts only real keys
    (the last key block may be partial; lists are ascending, so it is present
    exactly when it is the row's last entry)."""
    n_q, n_k = -(-lq // block), -(-lk // block)
    rows = np.full(n_q, float(block))
    rows[-1] = lq - (n_q - 1) * block
    short = block - (lk - (n_k - 1) * block)  # missing keys of the last key block
    keys = num_blocks.astype(np.float64) * block - short * ((last_entries == n_k - 1) & (num_blocks > 0))
    return float((keys * rows).sum()) * 4.0 * d


def traffic_from_profile() -> dict | None:
    """HBM bytes per launch of the sparse attention kernel from the committed
    counter summary, if it was measured on the current kernel source."""
    if not os.path.exists(TRAFFIC_SUMMARY):
        return None
    text = open(TRAFFIC_SUMMARY).read()
    src = hashlib.sha256(open(ATTN_SOURCE, "rb").read()).hexdigest()
    m_sha = re.search(r"kernel_source_sha256:\s*([0-9a-f]{64})", text)
    m_f = re.search(r"fetch_bytes_per_launch:\s*([0-9.eE+]+)", text)
    m_w = re.search(r"write_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not (m_sha and m_f and m_w) or m_sha.group(1) != src:
        return None
    return {"fetch": float(m_f.group(1)), "write": float(m_w.group(1))}


def _cpu_model() -> str:
    """The host CPU's model name with its family/model/stepping numbers (from
    /proc/cpuinfo where there is one)."""
    fields = {}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if ":" in line:
                    k, v = (x.strip() for x in line.split(":", 1))
                    fields.setdefault(k, v)
                if not line.strip() and fields:
                    break
    except OSError:
        pass
    name = fields.get("model name") or platform.processor() or platform.machine()
    ids = [f"{k} {fields[k]}" for k in ("cpu family", "model", "stepping") if k in fields]
    return f"{name} ({', '.join(ids)})" if ids else name


CPU_SELECTOR_HEADS = (0, 12)   # heads whose whole selector the oracle runs
CPU_ATTN_BLOCKS = 480           # (head, query block) pairs of the forward, spread over heads and blocks


def cpu_baseline(w, qb, kb, vb, keep_ref, total_flops: float, idx_gpu, num_gpu) -> dict:
    """The float64 oracle, as it stands, on a bounded sample of the headline
    workload: the whole selector of CPU_SELECTOR_HEADS, and the forward of
    CPU_ATTN_BLOCKS (head, query block) pairs spread over all heads and blocks.
    The per-head selector time and the per-block forward time are scaled to the
    whole call (24 heads x 1,125 blocks); the value is therefore extrapolated."""
    import oracle as O
    from synthetic import bf16_to_f64

    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=cores)
    except Exception:  # pragma: no cover
        limiter = None
    n_q = -(-w.lq // w.block)
    t_sel, agree = [], []
    for h in CPU_SELECTOR_HEADS:
        q, k = bf16_to_f64(qb[0, h]), bf16_to_f64(kb[0, h])
        t0 = time.perf_counter()
        lists, _, _, _ = O.select(q, k, w.block, w.density, keep_ref)
        t_sel.append(time.perf_counter() - t0)
        agree.append(sum(int(lists[i] == idx_gpu[0, h, i, : num_gpu[0, h, i]].tolist()) for i in range(n_q)) / n_q)
    rng = np.random.default_rng(7)
    pairs = sorted((int(h), int(i)) for h, i in zip(rng.integers(0, w.heads, CPU_ATTN_BLOCKS),
                                                      np.linspace(0, n_q - 1, CPU_ATTN_BLOCKS).astype(int)))
    t_att = 0.0
    cur, kv = None, None
    for h, i in pairs:
        if cur != h:
            cur, kv = h, (bf16_to_f64(qb[0, h]), bf16_to_f64(kb[0, h]), bf16_to_f64(vb[0, h]))
        q, k, v = kv
        rows = slice(i * w.block, min((i + 1) * w.block, w.lq))
        t0 = time.perf_counter()
        O.sparse_attention(q[rows], k, v, [idx_gpu[0, h, i, : num_gpu[0, h, i]].tolist()], w.block)
        t_att += time.perf_counter() - t0
    if limiter is not None:
        limiter.unregister()
    per_sel, per_blk = float(np.mean(t_sel)), t_att / len(pairs)
    est_s = w.heads * (per_sel + n_q * per_blk)
    return {
        "value": total_flops / est_s / 1e12,
        "unit": "TFLOP/s",
        "ms_per_call": est_s * 1e3,
        "cores": cores,
        "kind": "oracle",
        "method": "extrapolated",
        "sample": (f"extrapolated from a sample: the full selector of heads {list(CPU_SELECTOR_HEADS)} "
                   f"({n_q} rows each, {per_sel:.2f} s per head) and the forward of {len(pairs)} (head, query "
                   f"block) pairs spread over all heads and blocks ({per_blk * 1e3:.1f} ms each, on the GPU's "
                   f"lists), scaled to {w.heads} heads x {n_q} blocks; {sum(t_sel) + t_att:.1f} s of CPU work"),
        "cpu": _cpu_model(),
        "lists_equal_gpu_sampled_heads": float(np.mean(agree)),
    }


class Runner:
    """Device buffers and timed C-ABI calls for one workload shape."""

    def __init__(self, S, torch, w, qb, kb, vb, budget):
        self.S, self.torch, self.w = S, torch, w
        dev = torch.device("cuda:0")
        up = lambda bits: torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(dev)
        self.q, self.k, self.v = up(qb), up(kb), up(vb)
        seg = w.segments()
        self.keep = S.sparstar_clip_keep_ranges(2, seg["text"], seg["ref"])  # Eq. 3: later clips keep the text
        self.budget = budget
        B, H, Lq, D = self.q.shape
        Lk = self.k.shape[2]
        self.shape = (B, H, Lq, Lk, D)
        self.stride = S.sparstar_kv_stride(H, Lk, w.block, budget, self.keep)
        n_q = -(-Lq // w.block)
        self.num = torch.empty((B, H, n_q), dtype=torch.int32, device=dev)
        self.idx = torch.empty((B, H, n_q, self.stride), dtype=torch.int32, device=dev)
        self.ws = torch.empty(S.sparstar_score_workspace_bytes(B, H, Lq, Lk, D, w.block), dtype=torch.uint8,
                              device=dev)
        self.aws = torch.empty(max(1, S.sparstar_attn_workspace_bytes(B, H, Lq, Lk, D, w.block)), dtype=torch.uint8,
                               device=dev)
        self.o = torch.empty_like(self.q)
        self.lse = torch.empty((B, H, Lq), dtype=torch.float32, device=dev)

    def ev(self):
        return self.torch.cuda.Event(enable_timing=True)

    def score(self):
        self.S.sparstar_score_blocks(self.q, self.k, self.w.block, self.budget, self.keep, kv_stride=self.stride,
                                     workspace=self.ws, out=(self.num, self.idx))

    def sparse(self):
        self.S.sparstar_sparse_attn_fwd(self.q, self.k, self.v, self.num, self.idx, self.w.block, out=self.o,
                                        lse=self.lse, workspace=self.aws)

    def dense(self):
        self.S.sparstar_dense_attn_fwd(self.q, self.k, self.v, self.w.block, out=self.o, lse=self.lse,
                                       workspace=self.aws)

    def timed(self, fn, reps: int, warm: int = 1) -> list[float]:
        for _ in range(warm):
            fn()
        self.torch.cuda.synchronize()
        marks = [(self.ev(), self.ev()) for _ in range(reps)]
        for a, b in marks:
            a.record()
            fn()
            b.record()
        self.torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in marks]

    def flops(self) -> float:
        B, H, Lq, Lk, D = self.shape
        num = self.num.cpu().numpy()
        idx = self.idx.cpu().numpy()
        last = np.take_along_axis(idx, np.clip(num - 1, 0, None)[..., None].astype(np.int64), axis=-1)[..., 0]
        return executed_flops(num, last, Lq, Lk, self.w.block, D)

    def dense_flops(self) -> float:
        B, H, Lq, Lk, D = self.shape
        return 4.0 * B * H * Lq * Lk * D


MASS_DENSITIES = (0.25, 0.30, 0.50)
MASS_ROWS = 8


def attention_mass(r: "Runner", S, torch) -> dict:
    """Section 4's diagnostic on the bench inputs: the dense softmax mass each
    query's block selection keeps, exp(lse_sparse - lse_dense) for every query,
    and, on MASS_ROWS sampled queries per head, the token-wise bound (the mass
    of the same number of best single keys)."""
    B, H, Lq, Lk, D = r.shape
    b = r.w.block
    dev = r.q.device
    _, lse_all = S.sparstar_dense_attn_fwd(r.q, r.k, r.v, b, workspace=r.aws)
    rows = [int(x) for x in np.linspace(0, Lq - 1, MASS_ROWS)]
    ws = torch.empty(S.sparstar_token_topk_workspace_bytes(B, H, Lk, len(rows)), dtype=torch.uint8, device=dev)
    res, mass_ms = [], []
    for rho in MASS_DENSITIES:
        stride = S.sparstar_kv_stride(H, Lk, b, rho, r.keep)
        num, idx = S.sparstar_score_blocks(r.q, r.k, b, rho, r.keep, kv_stride=stride, workspace=r.ws)
        _, lse_sel = S.sparstar_sparse_attn_fwd(r.q, r.k, r.v, num, idx, b, workspace=r.aws)
        e0, e1 = r.ev(), r.ev()
        e0.record()
        mass = S.sparstar_retained_mass(lse_sel, lse_all)
        e1.record()
        torch.cuda.synchronize()
        mass_ms.append(e0.elapsed_time(e1))
        nb = num.cpu().numpy()
        ix = idx.cpu().numpy()
        n_tok = np.zeros((B, H, len(rows)), dtype=np.int32)
        for h in range(H):
            for j, t in enumerate(rows):
                lst = ix[0, h, t // b, : nb[0, h, t // b]]
                n_tok[0, h, j] = int(np.sum(np.minimum((lst + 1) * b, Lk) - lst * b))
        bound = S.sparstar_token_topk_mass(r.q, r.k, rows, torch.from_numpy(n_tok).to(dev), lse_all, workspace=ws)
        m = mass.cpu().numpy().astype(np.float64)
        bd = bound.cpu().numpy().astype(np.float64)
        ms_rows = m[:, :, rows]
        res.append({"density": rho, "block_mean": float(m.mean()), "block_min": float(m.min()),
                    "block_mean_sampled": float(ms_rows.mean()), "token_bound_mean_sampled": float(bd.mean()),
                    "gap_sampled": float((bd - ms_rows).mean())})
        del num, idx, lse_sel, mass
    return {"rows_sampled_per_head": len(rows), "by_density": res, "mass_kernel_ms": float(np.median(mass_ms)),
            "data": "synthetic (no trained model): absolute values are not the paper's"}


def _stats(xs) -> dict:
    return {"mean": float(np.mean(xs)), "median": float(np.median(xs)), "min": float(np.min(xs)),
            "p90": float(np.percentile(xs, 90))}


FLUSH_BYTES = 512 << 20  # larger than the L2s (8 x 4 MB) and the 256 MB last-level cache together


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--density", type=float, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-pyramid", action="store_true", help="skip both pyramid legs")
    ap.add_argument("--no-mid", action="store_true", help="skip the mid-scale leg")
    ap.add_argument("--no-warm", action="store_true", help="skip the warm-cache step timing")
    ap.add_argument("--no-b128", action="store_true", help="skip the 720p run at block size 128")
    ap.add_argument("--no-mass", action="store_true", help="skip the retained-attention-mass diagnostic")
    ap.add_argument("--no-graph", action="store_true", help="skip the graph-captured step timing")
    ap.add_argument("--gen-workers", type=int, default=None,
                    help="input-generation processes (default: up to 16; generation runs in-process "
                         "under a profiler regardless)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB -> 1 GiB fp32 copy kernel 3 times (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {args.gpus} is not supported (the hot path shards "
              "by head with no exchange between GPUs; the benchmark measures one GPU)", file=sys.stderr)
        return 2

    if args.copy_calibration:
        import torch

        n = 1 << 28  # 1 GiB of fp32
        x = torch.ones(n, dtype=torch.float32, device="cuda:0")
        y = torch.empty_like(x)
        for _ in range(3):
            torch.mul(x, 1.0, out=y)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration": {"read_bytes": 4 * n, "write_bytes": 4 * n, "launches": 3}}))
        return 0

    from synthetic import MID, P720, SWEEP, SWEEP_DENSITIES, generate, head_densities, pyramid_scales

    # all inputs are generated before the GPU is touched
    w = P720 if args.density is None else P720.with_(density=args.density)
    log(f"generating {w.name}: H={w.heads} D={w.head_dim} b={w.block} Lq={w.lq} Lk={w.lk} rho={w.density}")
    t0 = time.perf_counter()
    gw = args.gen_workers
    data = generate(w, workers=gw)
    w128 = w.with_(name="720p-b128", block=128)
    b128_data = None if args.no_b128 else generate(w128, workers=gw)
    sweep_data = None if args.no_sweep else generate(SWEEP, workers=gw)
    mid_data = None if args.no_mid else generate(MID, workers=gw)
    pyr = [] if args.no_pyramid else [(pw, sparse, generate(pw, workers=gw)) for pw, sparse in pyramid_scales()]
    log(f"generated in {time.perf_counter() - t0:.1f} s")

    import torch

    from paper_2608_10519_amd import sparstar as S

    S.load()
    r = Runner(S, torch, w, *data, w.density)
    B, H, Lq, Lk, D = r.shape
    flush_buf = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device="cuda:0")

    def flush():
        flush_buf.fill_(1)

    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        r.score()
        r.sparse()
    torch.cuda.synchronize()

    # The timed region: K steps, each after a 512 MiB write that evicts the L2s
    # and the last-level cache (cold caches, as the measurement protocol asks),
    # with HIP events around the selector call and the sparse forward call.
    log(f"timing {args.steps} steps (512 MiB cache flush before each)")
    marks = [(r.ev(), r.ev(), r.ev()) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for m in marks:
        flush()
        m[0].record()
        r.score()
        m[1].record()
        r.sparse()
        m[2].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    sel_ms = [m[0].elapsed_time(m[1]) for m in marks]
    att_ms = [m[1].elapsed_time(m[2]) for m in marks]
    step_ms = [a + b for a, b in zip(sel_ms, att_ms)]
    ms_step = float(np.median(step_ms))

    counts = r.num.cpu().numpy()
    flops = r.flops()
    att_avg = float(np.mean(att_ms))
    achieved = flops / (att_avg * 1e-3) / 1e12
    log(f"step median {ms_step:.3f} ms (min {np.min(step_ms):.3f}, p90 {np.percentile(step_ms, 90):.3f})  "
        f"selector {np.median(sel_ms):.3f} ms  sparse fwd {np.median(att_ms):.3f} ms ({achieved:.1f} TFLOP/s)")
    tr = traffic_from_profile()

    out = {
        "metric": METRIC,
        "value": flops / (ms_step * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded planted block structure, bf16)",
        "config": {
            "workload": "720p final scale: B=1, H=24, D=128, block 64, Lq=72000, Lk=144512 "
                        "(72000 preceding-clip + 512 text + 72000 current), text forced, budget 25%",
            "density": w.density,
            "kv_blocks_per_row": int(counts.max()),
            "executed_tflop": flops / 1e12,
        },
        "timing": {
            "protocol": "HIP events around each call; a 512 MiB write before each of the K timed steps "
                        "(cold L2 and last-level cache); ms_per_step is the median step",
            "step_ms": _stats(step_ms),
            "wall_ms_per_step_incl_flush": wall * 1e3 / args.steps,
        },
        "breakdown_ms": {
            "score_blocks": float(np.median(sel_ms)),
            "score_blocks_stats": _stats(sel_ms),
            "sparse_attn_fwd": float(np.median(att_ms)),
            "sparse_attn_fwd_stats": _stats(att_ms),
        },
        "roofline": {
            "bound": "mfma",
            "kernel": "sparse forward call (attn_fwd_kernel<128,64,sparse,split> + attn_merge_kernel)",
            "achieved": achieved,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS,
            "traffic": None if tr is None else tr["fetch"] + tr["write"],
        },
    }
    if tr is not None:
        out["roofline"]["traffic_detail_bytes"] = tr
    read_bytes = 2.0 * B * H * (Lq + Lk) * D  # Q and K, bf16, read once by the pooling kernel
    out["breakdown_ms"]["score_blocks_hbm_TBps"] = read_bytes / (np.median(sel_ms) * 1e-3) / 1e12

    if not args.no_warm:
        # the same step with warm caches (no flush), for comparison
        wm = [(r.ev(), r.ev(), r.ev()) for _ in range(args.steps)]
        for m in wm:
            m[0].record()
            r.score()
            m[1].record()
            r.sparse()
            m[2].record()
        torch.cuda.synchronize()
        wsel = [m[0].elapsed_time(m[1]) for m in wm]
        watt = [m[1].elapsed_time(m[2]) for m in wm]
        out["timing"]["warm"] = {"step_ms": _stats([a + b for a, b in zip(wsel, watt)]),
                                 "score_blocks_ms": _stats(wsel), "sparse_attn_fwd_ms": _stats(watt)}
        log(f"warm: step {np.median(wsel) + np.median(watt):.3f} ms, selector {np.median(wsel):.3f} ms")

    n_k = -(-Lk // w.block)
    if n_k <= S.FUSED_MAX_BLOCKS:
        # the selector with scores and selection fused in one kernel (S kept in
        # LDS), on lists of its own
        fnum, fidx = torch.empty_like(r.num), torch.empty_like(r.idx)

        def fused():
            S.sparstar_score_blocks(r.q, r.k, w.block, r.budget, r.keep, kv_stride=r.stride, workspace=r.ws,
                                    out=(fnum, fidx), fused=True)

        f_ms = r.timed(fused, reps=10, warm=2)
        out["breakdown_ms"]["score_blocks_fused"] = float(np.median(f_ms))
        log(f"fused score/select selector: {np.median(f_ms):.3f} ms (separate kernels {np.median(sel_ms):.3f} ms)")
        del fnum, fidx

    if not args.no_graph:
        # the same step captured once in a HIP graph (both calls only launch
        # kernels on the stream) and replayed K times
        log("graph-captured step")
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            r.score()
            r.sparse()
            torch.cuda.synchronize()
            with torch.cuda.graph(graph, stream=side):
                r.score()
                r.sparse()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            graph.replay()
        torch.cuda.synchronize()
        g_ms = (time.perf_counter() - t0) * 1e3 / args.steps
        out["graph"] = {"ms_per_step_warm": g_ms}
        log(f"graph step {g_ms:.3f} ms (warm)")
        del graph

    dense_ms = None
    if not args.no_dense:
        log("dense comparison")
        dense_ms = float(np.median(r.timed(r.dense, 3)))
        out["dense"] = {
            "ms": dense_ms,
            "tflops": r.dense_flops() / (dense_ms * 1e-3) / 1e12,
            "speedup_sparse_step": dense_ms / ms_step,
            "speedup_sparse_fwd_only": dense_ms / float(np.median(att_ms)),
        }
        log(f"dense {dense_ms:.2f} ms -> speedup {dense_ms / ms_step:.2f}x (step)")

    if not args.no_mass:
        log("retained attention mass (selection vs token-wise top-K bound)")
        out["attention_mass"] = attention_mass(r, S, torch)
        for row in out["attention_mass"]["by_density"]:
            log(f"  rho={row['density']}: block top-k keeps {row['block_mean']:.4f} of the dense mass "
                f"(sampled rows {row['block_mean_sampled']:.4f}, token bound {row['token_bound_mean_sampled']:.4f})")

    def cold_timed(rr, fn, reps):
        """Event times of fn, each rep after the cache flush."""
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            flush()
            a, b = rr.ev(), rr.ev()
            a.record()
            fn()
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        return ts

    if mid_data is not None:
        log("mid scale (11,520 queries against 84,032 keys)")
        rm = Runner(S, torch, MID, *mid_data, MID.density)
        sc = cold_timed(rm, rm.score, 10)
        sp = cold_timed(rm, rm.sparse, 10)
        fl = rm.flops()
        mB, mH, mLq, mLk, mD = rm.shape
        mbytes = 2.0 * mB * mH * (mLq + mLk) * mD
        out["mid"] = {"workload": "mid scale: B=1, H=24, D=128, block 64, Lq=11520, Lk=84032 (72000 preceding-"
                                  "clip + 512 text + 11520 current), text forced, budget 25%",
                      "score_ms": float(np.median(sc)), "sparse_fwd_ms": float(np.median(sp)),
                      "executed_tflop": fl / 1e12, "tflops": fl / (np.median(sp) * 1e-3) / 1e12,
                      "scoring_read_bytes": mbytes, "score_hbm_TBps": mbytes / (np.median(sc) * 1e-3) / 1e12,
                      "kv_blocks_per_row": int(rm.num.max().item())}
        log(f"  mid: score {np.median(sc):.3f} ms, sparse {np.median(sp):.3f} ms ({out['mid']['tflops']:.0f} TFLOP/s)")
        del rm

    if b128_data is not None:
        log("720p at the paper's deployed block size 128")
        rb = Runner(S, torch, w128, *b128_data, w128.density)
        sc = float(np.median(rb.timed(rb.score, 5)))
        sp = float(np.median(rb.timed(rb.sparse, 5)))
        dn = float(np.median(rb.timed(rb.dense, 2)))
        fl = rb.flops()
        out["block_128"] = {"score_ms": sc, "sparse_fwd_ms": sp, "executed_tflop": fl / 1e12,
                            "tflops": fl / (sp * 1e-3) / 1e12, "kv_blocks_per_row": int(rb.num.max().item()),
                            "dense_ms": dn, "dense_tflops": rb.dense_flops() / (dn * 1e-3) / 1e12,
                            "speedup_vs_dense_step": dn / (sc + sp)}
        log(f"  b=128: score {sc:.3f} ms, sparse {sp:.2f} ms ({fl / (sp * 1e-3) / 1e12:.0f} TFLOP/s), dense {dn:.1f} ms")
        del rb

    if sweep_data is not None:
        log("density sweep (per-head budgets U[0.5, 1.5] x rho)")
        rows = []
        for rho in SWEEP_DENSITIES:
            budgets = head_densities(SWEEP, rho).tolist()
            rs = Runner(S, torch, SWEEP, *sweep_data, budgets)
            sc = float(np.median(rs.timed(rs.score, 5)))
            sp = float(np.median(rs.timed(rs.sparse, 5)))
            fl = rs.flops()
            row = {"density": rho, "score_ms": sc, "sparse_fwd_ms": sp, "step_ms": sc + sp,
                   "executed_tflop": fl / 1e12, "tflops": fl / (sp * 1e-3) / 1e12,
                   "scoring_overhead": sc / sp}
            if dense_ms is not None:
                row["speedup_vs_dense_step"] = dense_ms / (sc + sp)
                row["speedup_vs_dense_fwd"] = dense_ms / sp
            rows.append(row)
            log(f"  rho={rho}: score {sc:.2f} ms, sparse {sp:.2f} ms ({row['tflops']:.0f} TFLOP/s)")
            del rs
        out["sweep"] = rows

    if pyr:
        # the configured pyramid (dense scales 1-3, fresh selection at 25% on
        # scales 4-5), then the paper's scale-wise density schedule: the four
        # finest scales sparsified at (0.625, 0.1875, 0.1875, 0.09375), looked
        # up by query length (sparstar_scale_densities), the coarsest dense
        lqs = [pw.lq for pw, _, _ in pyr]
        sched = S.sparstar_scale_densities(lqs, S.PAPER_720P_FINEST_DENSITIES)
        for leg, modes in (("pyramid", [(0.25 if sp_ else None) for _, sp_, _ in pyr]),
                           ("pyramid_paper_schedule", sched)):
            log(f"clip pyramid: {leg}")
            scales, total, dense_total = [], 0.0, 0.0
            for (pw, _, pdata), rho in zip(pyr, modes):
                rp = Runner(S, torch, pw.with_(density=rho if rho is not None else pw.density), *pdata,
                            rho if rho is not None else pw.density)
                dn_ms = float(np.median(rp.timed(rp.dense, 2)))
                if rho is not None:
                    ms = float(np.median(rp.timed(lambda: (rp.score(), rp.sparse()), 3)))
                    fl = rp.flops()
                else:
                    ms, fl = dn_ms, rp.dense_flops()
                total += ms
                dense_total += dn_ms
                scales.append({"lq": pw.lq, "lk": pw.lk, "density": rho, "mode": "dense" if rho is None else "sparse",
                               "ms": ms, "dense_ms": dn_ms, "executed_tflop": fl / 1e12})
                log(f"  Lq={pw.lq}: {'dense' if rho is None else f'rho={rho}'} {ms:.2f} ms (dense {dn_ms:.2f} ms)")
                del rp
            out[leg] = {"total_ms": total, "all_dense_ms": dense_total, "speedup_vs_all_dense": dense_total / total,
                        "scales": scales}

    if not args.no_cpu_baseline:
        log("cpu baseline (the oracle on a bounded sample, extrapolated)")
        import oracle as O

        seg = w.segments()
        keep_ref = O.keep_ranges_for_clip(2, seg["text"], seg["ref"])
        out["cpu_baseline"] = cpu_baseline(w, *data, keep_ref, flops, r.idx.cpu().numpy(), counts)
        log(f"cpu baseline {out['cpu_baseline']['value']:.4f} TFLOP/s ({out['cpu_baseline']['sample']})")

    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
