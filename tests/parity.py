"""Parity of the HIP verifiers against the CPU oracle, tree by tree.

Rule: status, then the accept/reject decision of every node the oracle tested,
in the oracle's order, then the accepted node, tau, Y and the counters must be
identical. At the first decision that differs, the tree counts as a near-tie
(and the rest of it is not compared) if the oracle's |u - theta| < 1e-6; for Y,
if u*W lies within 1e-6*W of a CDF boundary. Any other difference is a
failure. Acceptance probabilities (theta of tested nodes, p_init) must agree
within 1e-5 relative for float32 logits and 2e-3 relative for bfloat16 logits
(plus 1e-7 absolute for values near zero).

Outputs without theta come from tv_verify with early rejection: their residual
update counter is compared with the oracle's count of executed updates under
that rule; a difference there is a near-tie if the rule's own comparison
u[j] >= p(j) had an oracle margin below 1e-6.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

import paper_2505_12398_amd as tv
import workloads as W
from oracle import verify_tree, verify_tree_tokenlevel

BAND = 1e-6
THETA_RTOL = {"f32": 1e-5, "bf16": 2e-3}
THETA_ATOL = 1e-7


@dataclass
class ParityReport:
    trees: int = 0
    exact: int = 0
    near_ties: int = 0
    zero_rate: int = 0            # exact trees with a zero-rate boundary difference (see compare_tree)
    failures: list = field(default_factory=list)
    max_theta_rel: float = 0.0
    max_theta_abs: float = 0.0

    def add(self, other: "ParityReport"):
        self.trees += other.trees
        self.exact += other.exact
        self.near_ties += other.near_ties
        self.zero_rate += other.zero_rate
        self.failures += other.failures
        self.max_theta_rel = max(self.max_theta_rel, other.max_theta_rel)
        self.max_theta_abs = max(self.max_theta_abs, other.max_theta_abs)

    def record(self, kind: str, msg: str, worst, label: str):
        """Counts one compared tree (the result of compare_tree)."""
        self.trees += 1
        self.max_theta_rel = max(self.max_theta_rel, worst[0])
        self.max_theta_abs = max(self.max_theta_abs, worst[1])
        if kind in ("exact", "zero_rate"):
            self.exact += 1
            self.zero_rate += kind == "zero_rate"
        elif kind == "near_tie":
            self.near_ties += 1
        else:
            self.failures.append(f"{label}: {msg}")

    def summary(self):
        zr = f" ({self.zero_rate} at the zero-rate boundary)" if self.zero_rate else ""
        return (f"{self.trees} trees: {self.exact} exact{zr}, {self.near_ties} near-ties, "
                f"{len(self.failures)} failures, max theta err {self.max_theta_rel:.2e} rel "
                f"{self.max_theta_abs:.2e} abs")


def host_outputs(out: tv.VerifyOutputs):
    def h(t):
        return None if t is None else t.detach().cpu().numpy()
    return {k: h(getattr(out, k)) for k in ("accept_len", "accepted_node", "bonus_token",
                                             "status", "node_state", "node_theta", "p_init",
                                             "counters")}


def _theta_ok(g, r, rtol):
    return abs(float(g) - float(r)) <= rtol * abs(float(r)) + THETA_ATOL


_REJ, _PRU = tv.TV_NODE_REJECTED, tv.TV_NODE_PRUNED


def compare_tree(g: dict, b: int, ref, tokenlevel: bool, check_p_init: bool,
                 dtype: str = "f32"):
    """Returns (kind, message, (max_rel, max_abs) theta error) with kind in
    exact / zero_rate / near_tie / fail.

    zero_rate: every decision, the accepted node, tau and Y are identical, and
    the only differences are nodes that one side prunes (its rate is exactly
    0, the residual mass of Eq. (e1) having vanished) while the other tests
    them with a rate below the 1e-6 band, and the work counters that follow
    from that. Whether a mass far below rounding level is exactly zero is
    decided by rounding; such a node is rejected either way (a pruned node is
    a node rejected with rate 0), so its state counts as REJECTED on both
    sides."""
    rtol = THETA_RTOL[dtype]
    worst = [0.0, 0.0]
    if int(g["status"][b]) != ref.status:
        return "fail", f"status gpu {g['status'][b]} oracle {ref.status}", worst
    if ref.status != tv.TV_TREE_OK:
        ok = (g["accept_len"][b] == -1 and g["accepted_node"][b] == -1
              and g["bonus_token"][b] == -1)
        return ("exact", "", worst) if ok else ("fail", "error tree without sentinels", worst)
    state = g["node_state"][b]
    theta = None if g["node_theta"] is None else g["node_theta"][b]
    early = theta is None and not tokenlevel
    boundary = []          # nodes pruned on one side, tested below the band on the other
    for node in ref.test_order:
        want = ref.node_state[node]
        if state[node] != want:
            if want == _REJ and state[node] == _PRU and ref.node_theta[node] < BAND:
                boundary.append(node)
                continue
            if ref.margins[node] < BAND:
                return "near_tie", f"node {node} margin {ref.margins[node]:.2e}", worst
            gth = "-" if theta is None else f"{theta[node]:.9g}"
            return ("fail", f"node {node} state gpu {state[node]} oracle {want} "
                    f"theta gpu {gth} oracle {ref.node_theta[node]:.9g} "
                    f"u-margin {ref.margins[node]:.2e}", worst)
        if theta is None:
            continue
        th_r = float(ref.node_theta[node])
        err = abs(float(theta[node]) - th_r)
        worst[1] = max(worst[1], err)
        if th_r != 0.0:
            worst[0] = max(worst[0], err / abs(th_r))
        if not _theta_ok(theta[node], th_r, rtol):
            return "fail", f"node {node} theta gpu {theta[node]!r} oracle {th_r!r}", worst
    tested = set(ref.test_order)
    for node in range(len(state)):
        if node in tested or state[node] == ref.node_state[node]:
            continue
        if (ref.node_state[node] == _PRU and state[node] == _REJ
                and (theta is None or float(theta[node]) < BAND)):
            boundary.append(node)
            continue
        return ("fail", f"node states differ: gpu {state.tolist()} oracle "
                f"{ref.node_state.tolist()}", worst)
    if theta is not None:
        pruned = (ref.node_state == _PRU) & (state == _PRU)
        if not np.all(theta[pruned] == 0.0):
            return "fail", "pruned nodes must report theta 0", worst
        untested = ref.node_state == tv.TV_NODE_UNTESTED
        if not np.all(theta[untested] == -1.0):
            return "fail", "untested nodes must report theta -1", worst
    if int(g["accepted_node"][b]) != ref.accepted_node or int(g["accept_len"][b]) != ref.accept_len:
        return ("fail", f"accepted gpu {g['accepted_node'][b]}/{g['accept_len'][b]} oracle "
                f"{ref.accepted_node}/{ref.accept_len}", worst)
    if g["counters"] is not None:
        want = np.array(ref.counters_early if early else ref.counters)
        got = g["counters"][b]
        if not np.array_equal(got, want):
            others = [k for k in range(len(want)) if k != 1]
            if boundary and got[2] == want[2]:
                pass        # consulted rows, updates and tests follow the boundary nodes
            elif (early and ref.early_margin < BAND
                    and np.array_equal(got[others], want[others])):
                return "near_tie", f"early rejection margin {ref.early_margin:.2e}", worst
            else:
                return "fail", f"counters gpu {got.tolist()} oracle {want.tolist()}", worst
    if check_p_init and g["p_init"] is not None and not tokenlevel:
        for i, (a, r) in enumerate(zip(g["p_init"][b], ref.p_init)):
            if not _theta_ok(a, r, rtol):
                return "fail", f"p_init[{i}] gpu {a!r} oracle {r!r}", worst
    if int(g["bonus_token"][b]) != ref.bonus_token:
        if ref.y_margin < BAND:
            return "near_tie", f"Y margin {ref.y_margin:.2e}", worst
        return ("fail", f"Y gpu {g['bonus_token'][b]} oracle {ref.bonus_token} "
                f"margin {ref.y_margin:.2e}", worst)
    if boundary:
        return "zero_rate", f"nodes {sorted(boundary)} at the zero-rate boundary", worst
    return "exact", "", worst


def oracle_tree(batch: dict, b: int, tokenlevel: bool):
    par, tok, zb, zs, u = W.tree_numpy(batch, b)
    fn = verify_tree_tokenlevel if tokenlevel else verify_tree
    return fn(par, tok, zb, zs, batch["temperature"], u, batch["mode"])


def run_gpu(batch: dict, tokenlevel: bool, p_init: bool = False, theta: bool = True):
    """Runs a verifier on the whole batch; without ``theta`` tv_verify applies
    early rejection."""
    out = tv.verify_batch(batch["parents"], batch["tokens"], batch["target"], batch["draft"],
                          batch["temperature"], batch["uniforms"], batch["mode"],
                          tokenlevel=tokenlevel, want_p_init=p_init, want_theta=theta)
    return host_outputs(out)


_POOL_DATA = None


def _pool_oracle(args):
    b, tokenlevel = args
    par, tok, zb, zs, u, T, mode = _POOL_DATA
    fn = verify_tree_tokenlevel if tokenlevel else verify_tree
    r = fn(par[b], tok[b], zb[b], zs[b], T, u[b], mode)
    r.y_weights = None           # not compared; keeps the result small to send back
    return r


def host_batch(batch: dict):
    """Host copies of a whole batch for the oracle (bf16 logits as uint16 bits)."""
    import torch

    def rows(t):
        t = t.detach().cpu()
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16)
        return t.numpy()

    return (batch["parents"].cpu().numpy(), batch["tokens"].cpu().numpy(),
            rows(batch["target"]), rows(batch["draft"]), batch["uniforms"].cpu().numpy(),
            batch["temperature"], batch["mode"])


def oracle_many(batch: dict, trees, tokenlevels=(False, True), workers: int = 16,
                host=None) -> dict:
    """Oracle results of the listed trees for each verifier, computed by a pool
    of forked worker processes that only run the numpy oracle (the inputs are
    copied to host memory first and inherited, never sent). Returns
    {tokenlevel: [results in the order of trees]}."""
    import multiprocessing as mp
    global _POOL_DATA
    _POOL_DATA = host if host is not None else host_batch(batch)
    trees = list(trees)
    jobs = [(b, tl) for tl in tokenlevels for b in trees]
    try:
        with mp.get_context("fork").Pool(workers) as pool:
            res = pool.map(_pool_oracle, jobs, chunksize=1)
    finally:
        _POOL_DATA = None
    n = len(trees)
    return {tl: res[k * n:(k + 1) * n] for k, tl in enumerate(tokenlevels)}


def check(batch: dict, tokenlevel: bool, trees=None, p_init: bool = False,
          gpu: dict | None = None, label: str = "", theta: bool = True,
          refs=None) -> ParityReport:
    """Run the HIP verifier on the whole batch (unless ``gpu`` outputs are
    given) and compare the listed trees (all by default) with the oracle
    (computed here, or given in ``refs`` in the order of ``trees``)."""
    if gpu is None:
        gpu = run_gpu(batch, tokenlevel, p_init, theta)
    B = batch["parents"].shape[0]
    rep = ParityReport()
    for k, b in enumerate(range(B) if trees is None else trees):
        ref = oracle_tree(batch, b, tokenlevel) if refs is None else refs[k]
        kind, msg, worst = compare_tree(gpu, b, ref, tokenlevel, p_init,
                                        batch.get("dtype", "f32"))
        rep.record(kind, msg, worst, f"{label} tree {b}")
    return rep


def from_numpy(parents, tokens, target, draft, uniforms, temperature, mode, device,
               dtype="f32"):
    """Batch dict from host arrays (target/draft float64 are cast to the dtype)."""
    import torch
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    return {
        "parents": torch.as_tensor(np.ascontiguousarray(parents), dtype=torch.int32,
                                   device=device),
        "tokens": torch.as_tensor(np.ascontiguousarray(tokens), dtype=torch.int32,
                                  device=device),
        "target": torch.as_tensor(np.asarray(target, np.float32), device=device).to(tdt),
        "draft": torch.as_tensor(np.asarray(draft, np.float32), device=device).to(tdt),
        "uniforms": torch.as_tensor(np.asarray(uniforms, np.float32), device=device),
        "temperature": temperature, "mode": mode, "dtype": dtype,
    }
