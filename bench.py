"""Benchmark of batched Traversal Verification on one MI355X.

Workload: 256 trees x 64 draft nodes (65 rows per tree; irregular BFS trees of
depth 7, branching 1-4 with P(k) proportional to 2^-k), V = 128256, bfloat16
target and draft logits (target N(0, 3^2) plus +6 on 1% of the ids per row,
draft = target + N(0, 1.5^2)), temperature 1, children drawn from the draft
without replacement (the paper's sibling mode). Every step uses fresh seeds; the
inputs are generated on the GPU outside the timed region (about 8.5 GB of
logits per step).

A step is one tv_verify call over the whole batch. The timed region holds
exactly --steps calls, each bracketed by HIP events on the stream the kernel
runs on, with the device synchronised before and after. Prints one JSON line.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0       # MI355X HBM3E
SLEEP_CYCLES = 2_000_000     # about 1 ms of GPU clock ahead of each timed launch
CFG = 5
PROFILE_COUNTERS = os.path.join(ROOT, "profiles", "tv_verify_256trees_n64_v128256_hbm_counters.md")
PROFILE_TRACE = os.path.join(ROOT, "profiles", "tv_verify_256trees_n64_v128256_kernel_trace.md")
CSRC = os.path.join(ROOT, "paper_2505_12398_amd", "csrc")
HEADER = os.path.join(ROOT, "include", "tv.h")
METRIC = ("verified trees/sec + achieved HBM GB/s (% peak), 64-node trees, V=128256, bf16")


def kernel_hash() -> str:
    """Hash of every source the library is built from (the kernels, their
    launch code and the C-ABI) and of its header: a profile taken on other
    sources no longer describes the library built from these."""
    h = hashlib.sha256()
    for path in sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC)) + [HEADER]:
        h.update(os.path.basename(path).encode())
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _profile_value(path, key):
    """A number from a committed rocprofv3 summary, if the summary was taken on
    the sources as they are now; else None."""
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    t = re.search(rf"{key}:\s*([0-9.eE+]+)", text)
    if not m or not t or m.group(1) != kernel_hash():
        return None
    return float(t.group(1))


def measured_traffic():
    """HBM bytes per launch from the committed rocprofv3 counter summary."""
    return _profile_value(PROFILE_COUNTERS, "hbm_bytes_per_launch")


def traced_kernel_us():
    """Mean duration of the verify kernel alone (no initialisation kernel, no
    launch gap) from the committed rocprofv3 kernel trace."""
    return _profile_value(PROFILE_TRACE, "verify_kernel_mean_us")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def algorithmic_bytes(counters, vocab, elem_bytes, num_nodes, status=None):
    """Bytes the method must move for one launch: both rows of every consulted
    node, the accepted leaf's target row, both rows again per residual update,
    plus the per-node inputs and outputs. Counters of trees whose status is
    not OK are excluded (an error tree reports zeros)."""
    if status is not None:
        counters = counters[status == 0]
    c = counters.sum(dim=0).tolist()
    row = vocab * elem_bytes
    B = counters.shape[0]
    small = B * num_nodes * (4 + 4 + 4 + 1 + 4) + B * 4 * (4 + TV_NUM_COUNTERS)
    return {
        "compulsory": 2 * row * c[0] + row * c[2],
        "rescan": 2 * row * c[1],
        "small": small,
        "total": 2 * row * c[0] + row * c[2] + 2 * row * c[1] + small,
    }


TV_NUM_COUNTERS = 4


_CPU_TREES = None


def _one_thread():
    """Pool initialiser: one BLAS/OpenMP thread per worker process, so that
    `workers` processes use `workers` cores."""
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)


def _oracle_idx(b):
    """The oracle on tree b of the trees the parent process holds (inherited
    by fork, never sent); returns the result without its V-vector."""
    trees, T, mode = _CPU_TREES
    r = _oracle_one((trees[b], T, mode))
    r.y_weights = None
    return r


def cpu_baseline(batch, gpu_outs: dict, sample: int, workers: int):
    """The oracle on the first `sample` trees of one step, on host cores, with
    parity of those trees against each of the GPU outputs (by label). The
    trees are copied to host memory before the clock starts and the workers
    inherit them, so the time is the oracle's own."""
    global _CPU_TREES
    import multiprocessing as mp

    import workloads as W
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import parity  # noqa: E402  (test infrastructure: oracle comparison)

    _CPU_TREES = ([W.tree_numpy(batch, b) for b in range(sample)], batch["temperature"],
                  batch["mode"])
    try:
        t0 = time.perf_counter()
        with mp.get_context("fork").Pool(workers, initializer=_one_thread) as pool:
            refs = pool.map(_oracle_idx, range(sample), chunksize=1)
        dt = time.perf_counter() - t0
    finally:
        _CPU_TREES = None
    reps = {}
    for label, gpu_out in gpu_outs.items():
        g = parity.host_outputs(gpu_out)
        rep = parity.ParityReport()
        for b, ref in enumerate(refs):
            kind, msg, worst = parity.compare_tree(g, b, ref, False, False, "bf16")
            rep.record(kind, msg, worst, f"{label} tree {b}")
        reps[label] = rep
    return sample / dt, dt, reps


def commit_leg(last, stream, steps: int = 20) -> dict:
    """Times tv_commit_paths (the accepted-path commit) on the outputs of the
    last timed verification and checks every tree against the oracle's
    committed sequence."""
    import numpy as np
    import torch

    import paper_2505_12398_amd as tv
    from oracle import tv_oracle as O
    batch, out = last
    B, n1 = batch["parents"].shape
    max_len = 16
    times = []
    for _ in range(steps):
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(SLEEP_CYCLES)
        ev0.record(stream)
        pn, pt, pl = tv.commit_paths(batch["parents"], batch["tokens"], out, max_len,
                                     stream=stream.cuda_stream)
        ev1.record(stream)
        torch.cuda.synchronize()
        times.append(ev0.elapsed_time(ev1))
    par, tok = batch["parents"].cpu().numpy(), batch["tokens"].cpu().numpy()
    acc, y = out.accepted_node.cpu().numpy(), out.bonus_token.cpu().numpy()
    pt_h, pl_h = pt.cpu().numpy(), pl.cpu().numpy()
    exact = 0
    for b in range(B):
        _, toks = O.committed_sequence(par[b], tok[b], int(acc[b]), int(y[b]))
        exact += int(pl_h[b] == len(toks) and list(pt_h[b, :len(toks)]) == toks)
    return {"us_per_step": 1000.0 * sum(times) / len(times), "trees": B, "max_len": max_len,
            "bound": "launch latency (a few bytes per tree)",
            "parity": {"trees": B, "exact": exact}}


def deep_leg(steps: int, mode: int, stream, elem: int, V: int) -> dict:
    """tv_verify (no theta: early rejection) on Sequoia-scale trees: 8 trees of
    767 draft nodes (depth about 30), V=128256 bf16, fresh seeds per launch,
    with the oracle on one tree of the last launch."""
    import numpy as np
    import torch

    import paper_2505_12398_amd as tv
    import workloads as W
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import parity  # noqa: E402  (test infrastructure: oracle comparison)
    times, nbytes, acc = [], [], []
    out = batch = None
    for s in range(steps + 2):
        batch = W.make_deep_batch(step=s, device=torch.device("cuda", 0), mode=mode, vocab=V)
        B, n1 = batch["parents"].shape
        ws, _ = tv.workspace_tensor(B, n1, V, batch["target"].device)
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(SLEEP_CYCLES)
        ev0.record(stream)
        out = tv.verify_batch(batch["parents"], batch["tokens"], batch["target"], batch["draft"],
                              batch["temperature"], batch["uniforms"], mode, want_nodes=False,
                              want_counters=True, stream=stream.cuda_stream, workspace=ws)
        ev1.record(stream)
        torch.cuda.synchronize()
        if s >= 2:                     # two untimed warmup launches
            times.append(ev0.elapsed_time(ev1))
            nbytes.append(algorithmic_bytes(out.counters, V, elem, n1)["total"])
            acc.append(out.accept_len.float().mean().item() + 1.0)
    ms = sum(times) / len(times)
    alg = sum(nbytes) / len(nbytes)
    gpu = parity.host_outputs(tv.verify_batch(
        batch["parents"], batch["tokens"], batch["target"], batch["draft"],
        batch["temperature"], batch["uniforms"], mode, want_nodes=True, want_theta=False))
    kind, msg, _ = parity.compare_tree(gpu, 0, parity.oracle_tree(batch, 0, False), False, False,
                                       "bf16")
    B, n1 = batch["parents"].shape
    depth = max(int(W.node_depths(p).max()) for p in batch["parents"].cpu().numpy())
    return {"workload": W.DEEP_NAME, "trees": B, "nodes_per_tree": n1, "max_depth": depth,
            "ms_per_step": ms, "trees_per_s": B / (ms * 1e-3),
            "algorithmic_bytes_per_launch": alg, "achieved_GBps": alg / (ms * 1e-3) / 1e9,
            "frac": alg / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, "accept_len_mean": sum(acc) / len(acc),
            "parity_tree0": kind if kind != "fail" else f"fail: {msg}"}


def sampler_leg(batch, steps: int, stream, elem: int) -> dict:
    """Times tv_draft_tokens (the device draft-tree sampler) on the trees and
    draft logits of one benchmark step with fresh uniforms per launch, and
    checks 16 trees against the oracle. Algorithmic bytes: one read of the
    draft row of every node that has children."""
    import numpy as np
    import torch

    import paper_2505_12398_amd as tv
    import workloads as W
    from oracle import draft_sampler as DS
    par = batch["parents"]
    B, n1 = par.shape
    V = batch["draft"].shape[-1]
    par_h = par.cpu().numpy()
    internal = sum(len(set(row[1:].tolist())) for row in par_h)
    alg = internal * V * elem
    times = []
    for s in range(steps):
        rng = np.random.default_rng(1000 + s)
        u = torch.as_tensor(W.uniforms_np(rng, (B, n1)), device=par.device)
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(SLEEP_CYCLES)
        ev0.record(stream)
        tok, st = tv.draft_tokens(par, batch["draft"], batch["temperature"], u, batch["mode"],
                                  stream=stream.cuda_stream)
        ev1.record(stream)
        torch.cuda.synchronize()
        times.append(ev0.elapsed_time(ev1))
    ms = sum(times) / len(times)
    tok_h, st_h, u_h = tok.cpu().numpy(), st.cpu().numpy(), u.cpu().numpy()
    exact = near = fail = 0
    for b in range(0, B, max(1, B // 16)):
        rows = batch["draft"][b].detach().cpu()
        rows = rows.view(torch.int16).numpy().view(np.uint16) if rows.dtype == torch.bfloat16 \
            else rows.numpy()
        ref = DS.draw_tree_tokens(par_h[b], rows, batch["temperature"], u_h[b], batch["mode"])
        if st_h[b] == ref.status and np.array_equal(tok_h[b], ref.tokens):
            exact += 1
        elif st_h[b] == ref.status and ref.margin < 1e-6:
            near += 1
        else:
            fail += 1
    gbps = alg / (ms * 1e-3) / 1e9
    return {"ms_per_step": ms, "trees_per_s": B / (ms * 1e-3), "rows_with_children": internal,
            "algorithmic_bytes_per_launch": alg, "achieved_GBps": gbps,
            "frac": gbps / HBM_PEAK_GBPS, "bound": "hbm",
            "kernel": "sample_kernel<uint16_t, FastArith> (tv_draft_tokens)",
            "parity_sample": {"trees": exact + near + fail, "exact": exact, "near_ties": near,
                              "failures": fail}}


def config_leg(cfg_id: int, steps: int, tl_steps: int, mode: int, stream, batch=None,
               label=None) -> dict:
    """One workload at its full size (or ``batch`` trees of it): tv_verify on
    the timed path (no theta: early rejection) over ``steps`` launches with
    fresh seeds, the token-level verifier over ``tl_steps`` launches on the
    same trees and uniforms, algorithmic bytes and acceptance lengths. A
    512 MiB buffer is written before each timed launch so that the launch reads
    its rows from HBM, not from the 256 MiB cache in front of it."""
    import torch

    import paper_2505_12398_amd as tv
    import workloads as W
    cfg = W.CONFIGS[cfg_id]
    dev = torch.device("cuda", 0)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    B = batch or cfg.batch
    n1, V = cfg.n_nodes + 1, cfg.vocab
    elem = 2 if cfg.dtype == "bf16" else 4
    ws, _ = tv.workspace_tensor(B, n1, V, dev)
    res = {"tv": [], "tl": []}
    for s in range(max(steps, tl_steps) + 1):          # launch 0 is an untimed warmup
        bt = W.make_batch(cfg_id, step=30_000 + s, device=dev, mode=mode, batch=B, seed=2)
        for tl in (False, True):
            if s > (tl_steps if tl else steps):
                continue
            flush.fill_(s & 0xFF)
            torch.cuda.synchronize()
            ev0 = torch.cuda.Event(enable_timing=True)
            ev1 = torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(SLEEP_CYCLES)
            ev0.record(stream)
            out = tv.verify_batch(bt["parents"], bt["tokens"], bt["target"], bt["draft"],
                                  bt["temperature"], bt["uniforms"], mode, tokenlevel=tl,
                                  want_nodes=False, want_counters=True,
                                  stream=stream.cuda_stream, workspace=ws)
            ev1.record(stream)
            torch.cuda.synchronize()
            if s == 0:
                continue
            st = out.status
            if int((st != tv.TV_TREE_OK).sum().item()):
                raise RuntimeError(f"config {cfg_id}: trees with error status")
            res["tl" if tl else "tv"].append(
                (ev0.elapsed_time(ev1), algorithmic_bytes(out.counters, V, elem, n1, st)["total"],
                 out.accept_len.float().mean().item() + 1.0))
        del bt
    del flush

    def mean(xs):
        return sum(xs) / max(1, len(xs))
    ms = mean([r[0] for r in res["tv"]])
    alg = mean([r[1] for r in res["tv"]])
    acc_tv = mean([r[2] for r in res["tv"][:tl_steps]])
    acc_tl = mean([r[2] for r in res["tl"]])
    gbps = alg / (ms * 1e-3) / 1e9
    return {"workload": label or cfg.name, "trees": B, "rows_per_tree": n1, "vocab": V,
            "dtype": cfg.dtype, "temperature": cfg.temperature, "steps": steps,
            "ms_per_step": ms, "trees_per_s": B / (ms * 1e-3),
            "algorithmic_bytes_per_launch": alg, "achieved_GBps": gbps,
            "frac": gbps / HBM_PEAK_GBPS,
            "tokenlevel_ms_per_step": mean([r[0] for r in res["tl"]]),
            "accept_len_mean": {"traversal": acc_tv, "tokenlevel": acc_tl,
                                "delta_pct": 100.0 * (acc_tv / acc_tl - 1.0) if acc_tl else None},
            "cache": "512 MiB written before each launch (cold rows)"}


MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak


def lmhead_leg(steps: int, stream) -> dict:
    """tv_lmhead_stats at the size of one verification step of the large-batch
    workload: 16640 rows (256 trees x 65 nodes), hidden 4096 (Llama-3-8B),
    V = 128256, bf16, T = 1: logits plus their row statistics in one kernel.
    Roofline: bf16 MFMA FLOPs (2 M N K). Four sampled rows are checked
    against the oracle (exact products; statistics of the written logits)."""
    import numpy as np
    import torch

    import paper_2505_12398_amd as tv
    import oracle.lmhead as LM
    dev = torch.device("cuda", 0)
    M, K, N = 16640, 4096, 128256
    g = torch.Generator(device=dev).manual_seed(11)
    x = torch.randn((M, K), generator=g, device=dev).to(torch.bfloat16)
    w = (torch.randn((N, K), generator=g, device=dev) * (3.0 / K ** 0.5)).to(torch.bfloat16)
    out = (torch.empty((M, N), dtype=torch.bfloat16, device=dev),
           torch.empty(M, dtype=torch.float32, device=dev),
           torch.empty(M, dtype=torch.float64, device=dev))
    times = []
    for i in range(steps + 1):
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        tv.lmhead_stats(x, w, 1.0, stream=stream.cuda_stream, out=out)
        e1.record(stream)
        torch.cuda.synchronize()
        if i:
            times.append(e0.elapsed_time(e1))
    ms = sum(times) / len(times)
    flops = 2.0 * M * N * K
    tflops = flops / (ms * 1e-3) / 1e12
    # a library GEMM without the statistics, for context
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    y = x @ w.T
    e0.record(stream)
    for _ in range(3):
        y = x @ w.T
    e1.record(stream)
    torch.cuda.synchronize()
    lib_ms = e0.elapsed_time(e1) / 3
    del y
    # parity of sampled rows
    rows = [0, 4097, 9000, M - 1]
    def bits(t):
        return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    xb, wb = bits(x[rows]), bits(w)
    exact = LM.logits(xb, wb)
    bound = LM.accumulation_bound(xb, wb)
    got = bits(out[0][rows])
    gz = LM.to_f64(got)
    ok_logits = bool(np.all(np.abs(gz - exact) <= 2.0 ** -8 * np.abs(exact)
                            + 2.0 * K * 2.0 ** -24 * bound + 1e-30))
    m, ssum = LM.row_stats(got, 1.0)
    gm = out[1][rows].cpu().numpy().astype(np.float64)
    gs = out[2][rows].cpu().numpy()
    rel = float(np.max(np.abs(gs - ssum) / ssum))
    del x, w, out
    torch.cuda.empty_cache()
    return {"workload": "LM head 16640 rows x hidden 4096 x V 128256 bf16 (one 256-tree step)",
            "ms_per_step": ms, "tflops": tflops,
            "roofline": {"bound": "mfma", "achieved": tflops, "peak": MFMA_BF16_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": tflops / MFMA_BF16_PEAK_TFLOPS,
                         "kernel": "lmhead_kernel (tv_lmhead_stats)"},
            "library_gemm_without_statistics": {"ms": lib_ms,
                                                "tflops": flops / (lib_ms * 1e-3) / 1e12,
                                                "what": "torch matmul (hipBLASLt), logits only"},
            "parity_sample": {"rows": len(rows), "logits_within_bound": ok_logits,
                              "row_max_exact": bool(np.array_equal(gm, m)),
                              "row_sum_max_rel_err": rel}}


def verify_stats_leg(steps: int, mode: int, stream, workers: int) -> dict:
    """tv_verify_stats on the large-batch workload: the row statistics are given
    (as an LM head with fused statistics produces them; here computed from the
    synthetic logits outside the timed region), so the verifier reads rows
    only for residual updates and Y. Algorithmic bytes: both rows per executed
    residual update, the accepted leaf's target row, the small per-node data.
    16 trees of the last step are checked against the oracle."""
    import torch

    import paper_2505_12398_amd as tv
    import workloads as W
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import parity  # noqa: E402  (test infrastructure: oracle comparison)
    dev = torch.device("cuda", 0)
    cfg = W.CONFIGS[CFG]
    B, n1, V = cfg.batch, cfg.n_nodes + 1, cfg.vocab
    ws, _ = tv.workspace_tensor(B, n1, V, dev)

    def stats_of(z, T):
        zf = z.double()
        m = zf.amax(dim=-1)
        s = torch.exp((zf - m.unsqueeze(-1)) / float(T)).sum(dim=-1)
        return m.float().contiguous(), s.contiguous()

    times, nbytes, acc = [], [], []
    last = None
    for s_ in range(steps + 2):
        bt = W.make_batch(CFG, step=40_000 + s_, device=dev, mode=mode, seed=3)
        tm, ts = stats_of(bt["target"], bt["temperature"])
        dm, ds = stats_of(bt["draft"], bt["temperature"])
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(SLEEP_CYCLES)
        e0.record(stream)
        out = tv.verify_batch(bt["parents"], bt["tokens"], bt["target"], bt["draft"],
                              bt["temperature"], bt["uniforms"], mode, want_nodes=False,
                              want_counters=True, stream=stream.cuda_stream, workspace=ws,
                              stats=(tm, ts, dm, ds))
        e1.record(stream)
        torch.cuda.synchronize()
        if s_ >= 2:
            times.append(e0.elapsed_time(e1))
            c = out.counters[out.status == 0].sum(dim=0).tolist()
            row = V * 2
            nbytes.append(2 * row * c[1] + row * c[2] + B * n1 * 17 + B * 32)
            acc.append(out.accept_len.float().mean().item() + 1.0)
            last = (bt, (tm, ts, dm, ds))
        del bt
    ms = sum(times) / len(times)
    alg = sum(nbytes) / len(nbytes)
    bt, stats = last
    g = parity.host_outputs(tv.verify_batch(bt["parents"], bt["tokens"], bt["target"],
                                            bt["draft"], bt["temperature"], bt["uniforms"], mode,
                                            want_nodes=True, want_theta=False, stats=stats))
    trees = list(range(0, B, B // 16))
    refs = parity.oracle_many(bt, trees, tokenlevels=(False,), workers=workers)[False]
    rep = parity.check(bt, False, trees=trees, refs=refs, gpu=g, theta=False, label="stats")
    gbps = alg / (ms * 1e-3) / 1e9
    return {"workload": cfg.name + " with the row statistics given (tv_verify_stats)",
            "ms_per_step": ms, "trees_per_s": B / (ms * 1e-3),
            "algorithmic_bytes_per_launch": alg, "achieved_GBps": gbps,
            "frac": gbps / HBM_PEAK_GBPS, "accept_len_mean": sum(acc) / len(acc),
            "parity_sample": {"trees": rep.trees, "exact": rep.exact,
                              "near_ties": rep.near_ties, "failures": len(rep.failures)}}


def _oracle_one(args):
    (par, tok, zb, zs, u), T, mode = args
    from oracle import verify_tree
    return verify_tree(par, tok, zb, zs, T, u, mode)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--cpu-sample", type=int, default=256,
                    help="trees of one step verified by the CPU oracle (0: skip); the "
                         "default, the whole last step, is 10-20 s of host work")
    ap.add_argument("--cpu-workers", type=int, default=0)
    ap.add_argument("--mode", choices=["without", "with"], default="without")
    ap.add_argument("--tokenlevel-steps", type=int, default=20)
    ap.add_argument("--parity-steps", type=int, default=0,
                    help="also check every tree of this many more steps against the oracle "
                         "(timed path: no theta, early rejection)")
    ap.add_argument("--deep-steps", type=int, default=8,
                    help="timed launches on Sequoia-scale trees (8 trees x 768 nodes, V=128256)")
    ap.add_argument("--sampler-steps", type=int, default=20,
                    help="timed launches of the draft-tree token sampler on the same trees")
    ap.add_argument("--config-steps", type=int, default=10,
                    help="timed launches per smaller workload (chain, binary tree, irregular "
                         "tree) and of the one-tree latency leg (0: skip them)")
    ap.add_argument("--lmhead-steps", type=int, default=3,
                    help="timed launches of the LM head with fused statistics (0: skip)")
    ap.add_argument("--stats-steps", type=int, default=20,
                    help="timed launches of the verifier with row statistics given (0: skip)")
    ap.add_argument("--copy-calibration-gib", type=float, default=0.0,
                    help="only run plain device-to-device copies of this size (to scale "
                         "the FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the verification of independent trees needs no "
              "collectives, and only --gpus 1 is supported.", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2505_12398_amd as tv
    import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration_gib > 0:
        n = int(args.copy_calibration_gib * (1 << 30)) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_per_launch": n * 4, "launches": 3}), flush=True)
        return
    tv.load_library()
    mode = W.WITHOUT_REPLACEMENT if args.mode == "without" else W.WITH_REPLACEMENT
    cfg = W.CONFIGS[CFG]
    B, n1, V = cfg.batch, cfg.n_nodes + 1, cfg.vocab
    elem = 2
    stream = torch.cuda.current_stream(dev)

    workspace, _ = tv.workspace_tensor(B, n1, V, dev)

    def one_step(step, tokenlevel=False):
        batch = W.make_batch(CFG, step=step, device=dev, mode=mode, seed=1)
        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        # a spin kernel keeps the stream busy while the host enqueues the
        # launch, so the events time the GPU work and not the host's call
        torch.cuda._sleep(SLEEP_CYCLES)
        ev0.record(stream)
        out = tv.verify_batch(batch["parents"], batch["tokens"], batch["target"],
                              batch["draft"], batch["temperature"], batch["uniforms"], mode,
                              tokenlevel=tokenlevel, want_nodes=False, want_counters=True,
                              stream=stream.cuda_stream, workspace=workspace)
        ev1.record(stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1), batch, out

    for w in range(args.warmup):
        one_step(10_000 + w)
        print(f"warmup {w + 1}/{args.warmup}", file=sys.stderr, flush=True)

    times, nbytes, acc_tv, statuses = [], [], [], []
    last = None
    for s in range(args.steps):
        ms, batch, out = one_step(s)
        times.append(ms)
        if int((out.status == tv.TV_TREE_ABORTED).sum().item()):
            raise RuntimeError("a timed launch gave up (TV_TREE_ABORTED)")
        nb = algorithmic_bytes(out.counters, V, elem, n1, out.status)
        nbytes.append(nb)
        acc_tv.append(out.accept_len.float().mean().item() + 1.0)
        statuses.append(int((out.status != tv.TV_TREE_OK).sum().item()))
        if s == args.steps - 1:
            last = (batch, out)
        if (s + 1) % 10 == 0:
            print(f"step {s + 1}/{args.steps}: {ms:.3f} ms", file=sys.stderr, flush=True)

    ms_mean = sum(times) / len(times)
    srt = sorted(times)
    alg_total = sum(b["total"] for b in nbytes) / len(nbytes)
    achieved = alg_total / (ms_mean * 1e-3) / 1e9
    traffic = measured_traffic()
    kernel_us = traced_kernel_us()

    # token-level baseline on the same trees and uniforms (common random numbers)
    tl_times, acc_tl, acc_tv_same = [], [], []
    for s in range(args.tokenlevel_steps):
        ms, batch, out = one_step(s, tokenlevel=True)
        tl_times.append(ms)
        acc_tl.append(out.accept_len.float().mean().item() + 1.0)
        acc_tv_same.append(acc_tv[s] if s < len(acc_tv) else float("nan"))

    res = {
        "metric": METRIC,
        "value": B / (ms_mean * 1e-3),
        "unit": "trees/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_mean,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 terms, f64 accumulation and state (bf16 inputs)",
        "data": "synthetic (seeded, generated on the GPU; fresh seeds every step)",
        "config": {
            "workload": cfg.name + " (256 trees x 65 rows x V=128256 bf16 target+draft, "
                        "T=1, siblings without replacement)" if mode == W.WITHOUT_REPLACEMENT
            else cfg.name + " (siblings i.i.d.)",
            "batch": B, "rows_per_tree": n1, "vocab": V, "input_dtype": "bf16",
            "temperature": cfg.temperature, "mode": args.mode + "_replacement",
            "parallelism": "single GPU; each tree verified by a group of workgroups "
                           "(3 per tree at 256 trees) that run its traversal redundantly "
                           "and split every vocabulary pass into stripes",
        },
        "ms_p50": srt[len(srt) // 2],
        "ms_p90": srt[min(len(srt) - 1, int(0.9 * len(srt)))],
        "roofline": {
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": alg_total,
            "kernel": "verify_kernel<uint16_t, FastArith, 128> (tv_verify)",
            "timing": "HIP events around each tv_verify call (initialisation kernel, launch "
                      "gap and verify kernel)",
            "kernel_only": None if kernel_us is None else {
                "verify_kernel_mean_us": kernel_us,
                "achieved": alg_total / (kernel_us * 1e-6) / 1e9,
                "frac": alg_total / (kernel_us * 1e-6) / 1e9 / HBM_PEAK_GBPS,
                "source": "committed rocprofv3 kernel trace of these sources"},
            "sources_sha256_16": kernel_hash(),
        },
        "nominal_input_GBps": 2 * B * n1 * V * elem / (ms_mean * 1e-3) / 1e9,
        "trees_with_error_status": sum(statuses),
        "accept_len_mean": {
            "traversal": sum(acc_tv) / len(acc_tv),
            "tokenlevel": sum(acc_tl) / max(1, len(acc_tl)),
            "traversal_same_steps": sum(acc_tv_same) / max(1, len(acc_tv_same)),
        },
        "tokenlevel_ms_per_step": sum(tl_times) / max(1, len(tl_times)),
    }
    if acc_tl:
        res["accept_len_mean"]["delta_pct"] = 100.0 * (
            res["accept_len_mean"]["traversal_same_steps"] / res["accept_len_mean"]["tokenlevel"]
            - 1.0)

    if last is not None:
        res["commit_paths"] = commit_leg(last, stream)

    if args.deep_steps > 0:
        res["deep_trees"] = deep_leg(args.deep_steps, mode, stream, elem, V)

    if args.config_steps > 0:
        res["configs"] = {}
        for cid in (2, 3, 4):
            res["configs"][str(cid)] = config_leg(cid, args.config_steps,
                                                  max(1, args.config_steps // 2), mode, stream)
            print(f"config {cid} leg done", file=sys.stderr, flush=True)
        res["single_tree_latency"] = config_leg(
            CFG, 2 * args.config_steps, args.config_steps, mode, stream, batch=1,
            label=cfg.name.replace("B256", "B1") + " (one tree per call: latency)")
        print("single-tree leg done", file=sys.stderr, flush=True)

    if args.stats_steps > 0:
        res["verify_with_stats"] = verify_stats_leg(args.stats_steps, mode, stream,
                                                    args.cpu_workers or min(16, os.cpu_count() or 1))
        print("verify-with-statistics leg done", file=sys.stderr, flush=True)

    if args.lmhead_steps > 0:
        res["lmhead"] = lmhead_leg(args.lmhead_steps, stream)
        print("LM-head leg done", file=sys.stderr, flush=True)

    if args.sampler_steps > 0 and last is not None:
        res["draft_sampler"] = sampler_leg(last[0], args.sampler_steps, stream, elem)

    if args.parity_steps > 0:
        import multiprocessing as mp
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        import parity  # noqa: E402  (test infrastructure: oracle comparison)
        workers = args.cpu_workers or min(16, os.cpu_count() or 1)
        tot = parity.ParityReport()
        for k in range(args.parity_steps):
            batch = W.make_batch(CFG, step=20_000 + k, device=dev, mode=mode, seed=1)
            out = tv.verify_batch(batch["parents"], batch["tokens"], batch["target"],
                                  batch["draft"], batch["temperature"], batch["uniforms"], mode,
                                  want_nodes=True, want_theta=False, want_counters=True)
            g = parity.host_outputs(out)
            trees = [W.tree_numpy(batch, b) for b in range(B)]
            with mp.get_context("fork").Pool(workers) as pool:
                refs = pool.map(_oracle_one, [(t, batch["temperature"], mode) for t in trees])
            for b, ref in enumerate(refs):
                kind, msg, worst = parity.compare_tree(g, b, ref, False, False, "bf16")
                tot.record(kind, msg, worst, f"step {k} tree {b}")
            print(f"parity step {k + 1}/{args.parity_steps}: {tot.summary()}", file=sys.stderr,
                  flush=True)
            del batch, out
        res["parity_steps"] = {"steps": args.parity_steps, "trees": tot.trees,
                               "exact": tot.exact, "zero_rate_boundary": tot.zero_rate,
                               "near_ties": tot.near_ties,
                               "failures": len(tot.failures)}
        if tot.failures:
            print("\n".join(tot.failures[:5]), file=sys.stderr)

    if args.cpu_sample > 0 and last is not None:
        workers = args.cpu_workers or min(16, os.cpu_count() or 1)
        sample = min(args.cpu_sample, B)
        batch, _ = last
        # the timed configuration (no theta output: early rejection), with node
        # states for the comparison; and once more with theta, for its accuracy
        outs = {theta: tv.verify_batch(batch["parents"], batch["tokens"], batch["target"],
                                       batch["draft"], batch["temperature"], batch["uniforms"],
                                       mode, want_nodes=True, want_theta=theta,
                                       want_counters=True)
                for theta in (False, True)}
        torch.cuda.synchronize()
        tps, secs, reps = cpu_baseline(batch, {"timed": outs[False], "theta": outs[True]},
                                       sample, workers)
        # one process, one core: the oracle on the first trees, in this process
        n_single = min(8, B)
        single = [W.tree_numpy(batch, b) for b in range(n_single)]
        from threadpoolctl import threadpool_limits
        with threadpool_limits(1):
            t0 = time.perf_counter()
            for t in single:
                _oracle_one((t, batch["temperature"], mode))
            per_core = n_single / (time.perf_counter() - t0)
        res["cpu_baseline"] = {
            "value": tps, "unit": "trees/s", "cores": workers, "kind": "oracle",
            "sample": f"first {sample} trees of timed step {args.steps - 1} "
                      f"({secs:.1f} s wall, float64 numpy, one process per core)",
            "per_core": {"value": per_core, "unit": "trees/s",
                         "sample": f"first {n_single} trees of the same step, one process, "
                                   "one BLAS thread"},
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
        }
        rep, rth = reps["timed"], reps["theta"]
        res["parity_sample"] = {"trees": rep.trees, "exact": rep.exact,
                                "near_ties": rep.near_ties, "failures": len(rep.failures),
                                "zero_rate_boundary": rep.zero_rate,
                                "with_theta": {"exact": rth.exact, "near_ties": rth.near_ties,
                                               "zero_rate_boundary": rth.zero_rate,
                                               "failures": len(rth.failures),
                                               "max_theta_rel_err": rth.max_theta_rel,
                                               "max_theta_abs_err": rth.max_theta_abs}}
        for r in (rep, rth):
            if r.failures:
                print("\n".join(r.failures[:5]), file=sys.stderr)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
