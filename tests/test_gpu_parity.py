"""HIP verifiers against the CPU oracle on the same seeded inputs (needs an
MI355X). Every call goes through the C-ABI library via its ctypes binding."""

import numpy as np
import pytest
import torch

import paper_2505_12398_amd as tv
import parity
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda"
MODES = [W.WITHOUT_REPLACEMENT, W.WITH_REPLACEMENT]


def assert_clean(rep, label):
    print(f"{label}: {rep.summary()}", flush=True)
    assert not rep.failures, "\n".join(rep.failures[:10])
    assert rep.max_theta_abs < parity.BAND, rep.summary()
    assert rep.near_ties <= max(1, rep.trees // 100), rep.summary()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tv.load_library()
    yield


# --------------------------------------------------------------------------
# The paper's example and the tiny exact-check workload
# --------------------------------------------------------------------------

@pytest.mark.parametrize("tokenlevel", [False, True])
def test_worked_example(tokenlevel):
    """Sec. 3.2 tree, V = 3 float32 (rows are 12 bytes: every row is misaligned
    and handled by the scalar head/tail path), 256 random uniform vectors."""
    par, tok, zb, zs, T = W.worked_example()
    rng = np.random.default_rng(0)
    B = 256
    u = W.uniforms_np(rng, (B, 6))
    u[0, 1:] = np.float32(1 - 2 ** -24)          # all rejections on tree 0
    batch = parity.from_numpy(np.tile(par, (B, 1)), np.tile(tok, (B, 1)),
                              np.tile(zb, (B, 1, 1)), np.tile(zs, (B, 1, 1)), u, T,
                              W.WITHOUT_REPLACEMENT, DEV)
    rep = parity.check(batch, tokenlevel, p_init=not tokenlevel, label="worked")
    assert_clean(rep, f"worked example tokenlevel={tokenlevel}")
    g = parity.run_gpu(batch, tokenlevel)
    if not tokenlevel:
        assert list(g["node_state"][0]) == [0, 2, 1, 2, 2, 2]
        np.testing.assert_allclose(g["node_theta"][0], [-1, 0, 1, 2 / 3, 7 / 11, 1 / 2],
                                   rtol=1e-6)
        # updates after X3, X4, X1 and X5 (counter 1)
        assert g["counters"][0][1] == 4
        # without theta: the update after X4 is skipped (p(X1) = 1/11 <= u(X1))
        rep = parity.check(batch, False, label="worked-early", theta=False)
        assert_clean(rep, "worked example, early rejection")
        g = parity.run_gpu(batch, False, theta=False)
        assert g["node_theta"] is None
        assert list(g["node_state"][0]) == [0, 2, 1, 2, 2, 2]
        assert g["counters"][0][1] == 3


@pytest.mark.parametrize("tokenlevel", [False, True])
@pytest.mark.parametrize("mode", MODES)
def test_tiny_context_model(mode, tokenlevel):
    """V = 8, complete binary tree of depth 2, context-keyed target N(0, 2^2)
    and draft target + N(0, 1), T = 1, seed 0; 512 trees drawn per mode."""
    m = W.ContextModel(8, seed=0)
    par = W.binary_parents(2)
    rng = np.random.default_rng(100 + mode)
    B = 512
    P, TK, ZB, ZS = [], [], [], []
    for _ in range(B):
        tok, zb, zs = W.draw_context_tree(rng, m, par, 1.0, mode)
        P.append(par)
        TK.append(tok)
        ZB.append(zb)
        ZS.append(zs)
    u = W.uniforms_np(rng, (B, len(par)))
    batch = parity.from_numpy(np.stack(P), np.stack(TK), np.stack(ZB), np.stack(ZS), u, 1.0,
                              mode, DEV)
    rep = parity.check(batch, tokenlevel, p_init=not tokenlevel, label="tiny")
    assert_clean(rep, f"tiny mode={mode} tokenlevel={tokenlevel}")
    if not tokenlevel:
        rep = parity.check(batch, False, label="tiny-early", theta=False)
        assert_clean(rep, f"tiny mode={mode} early rejection")


# --------------------------------------------------------------------------
# Reduced-vocabulary versions of the workloads: every tree compared, the
# vocabulary spans many 64-vector blocks and ends in a ragged tail.
# --------------------------------------------------------------------------

@pytest.mark.parametrize("tokenlevel", [False, True])
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("cfg,vocab,batch", [(2, 32003, 16), (3, 20011, 12), (4, 12347, 8),
                                             (5, 16381, 24)])
def test_configs_reduced(cfg, vocab, batch, mode, tokenlevel):
    bt = W.make_batch(cfg, step=1, device=DEV, mode=mode, batch=batch, vocab=vocab)
    rep = parity.check(bt, tokenlevel, p_init=not tokenlevel, label=f"cfg{cfg}")
    assert_clean(rep, f"cfg{cfg} V={vocab} mode={mode} tokenlevel={tokenlevel}")
    if not tokenlevel:
        rep = parity.check(bt, False, label=f"cfg{cfg}-early", theta=False)
        assert_clean(rep, f"cfg{cfg} V={vocab} mode={mode} early rejection")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_temperature_and_dtype(dtype):
    """Config-3 shape at T = 0.7 and T = 1.9 in both dtypes."""
    for T in (0.7, 1.9):
        bt = W.make_batch(3, step=2, device=DEV, mode=W.WITHOUT_REPLACEMENT, batch=8,
                          vocab=4099)
        bt["temperature"] = T
        tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
        bt["target"] = bt["target"].to(tdt)
        bt["draft"] = bt["draft"].to(tdt)
        bt["dtype"] = dtype
        for tl in (False, True):
            rep = parity.check(bt, tl, p_init=not tl, label=f"T{T}")
            assert_clean(rep, f"T={T} {dtype} tokenlevel={tl}")


# --------------------------------------------------------------------------
# Full-size workloads, in the launch configuration the benchmark times
# --------------------------------------------------------------------------

def _check_all(bt, label, trees=None, workers=16, p_init=False):
    """Every listed tree (all by default) of a full-size batch against the
    oracle (computed by a pool of host processes), for Traversal Verification
    with theta, without theta (early rejection, as the benchmark runs it) and
    for the token-level verifier."""
    B = bt["parents"].shape[0]
    trees = list(range(B)) if trees is None else list(trees)
    refs = parity.oracle_many(bt, trees, workers=workers)
    for tl in (False, True):
        rep = parity.check(bt, tl, trees=trees, refs=refs[tl], p_init=p_init and not tl,
                           label=label)
        assert_clean(rep, f"{label} tokenlevel={tl}")
    rep = parity.check(bt, False, trees=trees, refs=refs[False], theta=False,
                       label=f"{label}-early")
    assert_clean(rep, f"{label} early rejection")


@pytest.mark.parametrize("cfg", [2, 3, 4, 5])
def test_configs_full_size(cfg):
    """Every tree of each workload at its full size, both sibling modes (the
    large-batch workload: all 256 trees of a step per mode)."""
    for mode in MODES:
        bt = W.make_batch(cfg, step=3, device=DEV, mode=mode)
        _check_all(bt, f"cfg{cfg} full mode={mode}")
        del bt
        torch.cuda.empty_cache()


@pytest.mark.parametrize("cfg,batch", [(3, None), (5, 64)])
def test_low_temperature_full_vocab(cfg, batch):
    """T = 0.2, the lowest temperature of the paper's sweep (Table 4), at the
    full vocabulary in bf16 (the fast element path, where log2(e)/T is rounded
    to fp32 and multiplies larger exponents): the binary-tree workload (32
    trees) and 64 trees of the large-batch shape, both sibling modes. At this
    temperature chain rates fall far below rounding level, and whether a
    residual mass that small is exactly zero (the node's children pruned) is
    decided by rounding: such trees count as exact at the zero-rate boundary
    when everything else agrees (parity.compare_tree)."""
    for mode in MODES:
        bt = W.make_batch(cfg, step=8, device=DEV, mode=mode, batch=batch)
        bt["temperature"] = 0.2
        # drafted tokens must come from the draft at the temperature verified
        bt["tokens"] = W.draw_tokens(bt["parents"].cpu().numpy(), bt["draft"], 0.2, mode,
                                     W._seed(0, cfg, 8, 33))
        _check_all(bt, f"cfg{cfg} T=0.2 mode={mode}", p_init=True)
        del bt
        torch.cuda.empty_cache()


@pytest.mark.parametrize("batch", [512, 1024])
def test_large_batches_with_helpers(batch):
    """Batches beyond one tree per group: groups of one workgroup, groups that
    verify two trees in turn, and helpers joining running groups (sampled
    trees, all statuses)."""
    bt = W.make_batch(5, step=5, device=DEV, mode=W.WITHOUT_REPLACEMENT, batch=batch,
                      vocab=16400)
    gpu = parity.run_gpu(bt, False, False)
    assert (gpu["status"] == tv.TV_TREE_OK).all()
    trees = list(range(0, batch, batch // 48)) + [batch - 1]
    rep = parity.check(bt, False, trees=trees, gpu=gpu, label=f"B{batch}")
    assert_clean(rep, f"batch {batch}")
    gpu = parity.run_gpu(bt, False, False, theta=False)
    rep = parity.check(bt, False, trees=trees, gpu=gpu, label=f"B{batch}-early", theta=False)
    assert_clean(rep, f"batch {batch} early rejection")


# --------------------------------------------------------------------------
# Edge cases
# --------------------------------------------------------------------------

def _rand_batch(rng, parents, vocab, dtype="f32", mode=W.WITH_REPLACEMENT, T=1.0,
                scale=2.0):
    B, n1 = parents.shape
    zb = rng.normal(0, scale, (B, n1, vocab))
    zs = zb + rng.normal(0, 1.0, (B, n1, vocab))
    tok = np.zeros((B, n1), np.int32)
    for b in range(B):
        for i in range(1, n1):
            tok[b, i] = rng.integers(0, vocab)
        if mode == W.WITHOUT_REPLACEMENT:
            kids = {}
            for i in range(1, n1):
                kids.setdefault(parents[b, i], []).append(i)
            for p, ks in kids.items():
                tok[b, ks] = rng.choice(vocab, len(ks), replace=False)
    u = W.uniforms_np(rng, (B, n1))
    return parity.from_numpy(parents, tok, zb, zs, u, T, mode, DEV, dtype)


@pytest.mark.parametrize("tokenlevel", [False, True])
def test_root_only_and_tiny_vocab(tokenlevel):
    rng = np.random.default_rng(1)
    for vocab in (2, 3, 5, 17):
        bt = _rand_batch(rng, np.full((16, 1), -1, np.int32), vocab)
        rep = parity.check(bt, tokenlevel, p_init=not tokenlevel, label=f"root V{vocab}")
        assert_clean(rep, f"root-only V={vocab}")
        par = np.tile(np.array([-1, 0, 0, 1], np.int32), (16, 1))
        bt = _rand_batch(rng, par, vocab)
        rep = parity.check(bt, tokenlevel, p_init=not tokenlevel, label=f"small V{vocab}")
        assert_clean(rep, f"small tree V={vocab}")
        if not tokenlevel:
            rep = parity.check(bt, False, label=f"small V{vocab} early", theta=False)
            assert_clean(rep, f"small tree V={vocab} early rejection")


def test_large_trees():
    """1024-node trees: a random recursive tree and a 1023-deep chain."""
    rng = np.random.default_rng(2)
    n1 = tv.TV_MAX_NODES
    par = np.zeros((4, n1), np.int32)
    par[:, 0] = -1
    for b in range(3):
        for i in range(1, n1):
            par[b, i] = rng.integers(max(0, i - 8), i)
    par[3] = np.arange(-1, n1 - 1)
    for tl in (False, True):
        bt = _rand_batch(rng, par, 64, mode=W.WITH_REPLACEMENT, scale=0.3)
        rep = parity.check(bt, tl, label="large")
        assert_clean(rep, f"1024-node trees tokenlevel={tl}")
        if not tl:
            rep = parity.check(bt, False, label="large-early", theta=False)
            assert_clean(rep, "1024-node trees, early rejection")


@pytest.mark.parametrize("mode", MODES)
def test_deep_trees(mode):
    """Sequoia-scale trees (767 draft nodes, depth about 30, hundreds of
    internal nodes) with the large-batch logit law at a reduced vocabulary
    (V = 4099, fp32): every tree, both verifiers, with and without theta."""
    bt = W.make_deep_batch(batch=4, vocab=4099, step=1, device=DEV, mode=mode, dtype="f32")
    for tl in (False, True):
        rep = parity.check(bt, tl, label=f"deep mode={mode} tl={tl}")
        assert_clean(rep, f"deep trees mode={mode} tokenlevel={tl}")
    rep = parity.check(bt, False, label=f"deep-early mode={mode}", theta=False)
    assert_clean(rep, f"deep trees mode={mode} early rejection")


@pytest.mark.parametrize("mode", MODES)
def test_deep_trees_full_vocab(mode):
    """Sequoia-scale trees at their benchmark shape: the 8 trees of one launch
    (767 draft nodes, depth about 30) at V = 128256 bf16 (the fast element
    path), both verifiers, with and without theta."""
    bt = W.make_deep_batch(step=2, device=DEV, mode=mode)
    _check_all(bt, f"deep full-V mode={mode}", workers=8)
    del bt
    torch.cuda.empty_cache()


def test_unconsulted_nonfinite_row():
    """Error reporting for a row the traversal never consults (a documented
    difference between the eager oracle and the lazy kernels). With identical
    models the first leaf (node 7 of a binary tree of depth 3) is accepted and
    only the rows of nodes 0, 1, 3 are consulted. A NaN planted in the target
    row of node 2 (internal, off that path): with p_init the verifier reads
    every row with children and reports NONFINITE, as the oracle does; without
    p_init it never reads the row, and its outputs equal those of the clean
    input."""
    rng = np.random.default_rng(9)
    par = np.tile(W.binary_parents(3), (8, 1))
    bt = _rand_batch(rng, par, 20000, dtype="bf16")
    bt["draft"] = bt["target"].clone()
    clean = parity.run_gpu(bt, False, p_init=False)
    rep = parity.check(bt, False, gpu=clean, label="clean")
    assert_clean(rep, "identical models, clean")
    tgt = bt["target"].clone()
    tgt[:, 2, 123] = float("nan")
    bad = dict(bt, target=tgt)
    with_pinit = parity.run_gpu(bad, False, p_init=True)
    assert (with_pinit["status"] == tv.TV_TREE_NONFINITE).all()
    for b in range(8):
        assert parity.oracle_tree(bad, b, False).status == tv.TV_TREE_NONFINITE
    without = parity.run_gpu(bad, False, p_init=False)
    for k in ("status", "accept_len", "accepted_node", "bonus_token", "node_state",
              "node_theta", "counters"):
        assert np.array_equal(without[k], clean[k]), k


def test_abandoned_launch_reports_sentinels(monkeypatch):
    """The bounded wait: with a wait limit of 0 ms (TV_WAIT_LIMIT_MS) a launch
    is abandoned at its first wait that is not satisfied at once, and every
    kernel exits. Each tree then reports either TV_TREE_ABORTED with the
    sentinel outputs (-1, node states 0, theta and p_init -1, counters 0) or,
    if it finished first, its verified result; a following call with the
    normal limit on the same workspace is clean."""
    bt = W.make_batch(5, step=9, device=DEV, mode=W.WITHOUT_REPLACEMENT, batch=64,
                      vocab=32768)
    B, n1 = bt["parents"].shape
    ws, _ = tv.workspace_tensor(B, n1, 32768, DEV)
    monkeypatch.setenv("TV_WAIT_LIMIT_MS", "0")
    out = tv.verify_batch(bt["parents"], bt["tokens"], bt["target"], bt["draft"],
                          bt["temperature"], bt["uniforms"], bt["mode"], want_p_init=True,
                          workspace=ws)
    torch.cuda.synchronize()
    g = parity.host_outputs(out)
    monkeypatch.delenv("TV_WAIT_LIMIT_MS")
    aborted = g["status"] == tv.TV_TREE_ABORTED
    print(f"abandoned launch: {int(aborted.sum())} of {B} trees aborted", flush=True)
    assert aborted.sum() >= 1
    assert np.all((g["status"] == tv.TV_TREE_OK) | aborted)
    for k in ("accept_len", "accepted_node", "bonus_token"):
        assert np.all(g[k][aborted] == -1), k
    assert np.all(g["node_state"][aborted] == 0)
    assert np.all(g["node_theta"][aborted] == -1.0)
    assert np.all(g["p_init"][aborted] == -1.0)
    assert np.all(g["counters"][aborted] == 0)
    done = np.nonzero(~aborted)[0].tolist()
    if done:
        rep = parity.check(bt, False, trees=done, gpu=g, p_init=True, label="abandoned")
        assert_clean(rep, "trees finished before the abandon")
    g2 = parity.run_gpu(bt, False, p_init=True)
    assert (g2["status"] == tv.TV_TREE_OK).all()
    rep = parity.check(bt, False, trees=[0, 21, 42, 63], gpu=g2, p_init=True, label="after")
    assert_clean(rep, "call after an abandoned launch")


def test_batch_beyond_one_grid_of_trees():
    """300000 two-node trees (more trees than the initialisation grid has
    threads, so its per-tree loop strides): every tree verified, sampled trees
    against the oracle."""
    rng = np.random.default_rng(10)
    B, V = 300_000, 8
    par = np.tile(np.array([-1, 0], np.int32), (B, 1))
    zb = rng.normal(0, 2, (B, 2, V)).astype(np.float32)
    zs = (zb + rng.normal(0, 1, (B, 2, V))).astype(np.float32)
    tok = np.zeros((B, 2), np.int32)
    tok[:, 1] = rng.integers(0, V, B)
    u = W.uniforms_np(rng, (B, 2))
    bt = parity.from_numpy(par, tok, zb, zs, u, 1.0, W.WITH_REPLACEMENT, DEV)
    g = parity.run_gpu(bt, False, p_init=True)
    assert (g["status"] == tv.TV_TREE_OK).all()
    assert set(np.unique(g["accepted_node"]).tolist()) <= {0, 1}
    trees = list(range(0, B, 997)) + [B - 1]
    rep = parity.check(bt, False, trees=trees, gpu=g, p_init=True, label="B300000")
    assert_clean(rep, "300000 trees")


def test_identical_models_accept_first_leaf():
    rng = np.random.default_rng(3)
    par = np.tile(W.binary_parents(3), (8, 1))
    bt = _rand_batch(rng, par, 1000, dtype="bf16")
    bt["draft"] = bt["target"].clone()
    g = parity.run_gpu(bt, False, p_init=True)
    assert np.all(g["accepted_node"] == 7) and np.all(g["accept_len"] == 3)
    assert np.all(g["p_init"] == 1.0)
    rep = parity.check(bt, False, gpu=g, p_init=True, label="identical")
    assert_clean(rep, "identical models")


@pytest.mark.parametrize("tokenlevel", [False, True])
def test_error_trees(tokenlevel):
    rng = np.random.default_rng(4)
    par = np.tile(np.array([-1, 0, 0, 1, 1, 2], np.int32), (6, 1))
    bt = _rand_batch(rng, par, 50, mode=W.WITHOUT_REPLACEMENT)
    P = bt["parents"].clone()
    K = bt["tokens"].clone()
    P[1, 3] = 3                 # not < i
    P[2, 0] = 0                 # root parent must be -1
    K[3, 4] = 50                # token out of range
    K[4, 2] = K[4, 1]           # duplicate siblings (without replacement)
    bt["parents"], bt["tokens"] = P, K
    tgt = bt["target"].clone()
    tgt[5, 0, 7] = float("nan")  # NaN in the root's target row (always read)
    bt["target"] = tgt
    g = parity.run_gpu(bt, tokenlevel, p_init=not tokenlevel)
    assert list(g["status"]) == [tv.TV_TREE_OK, tv.TV_TREE_BAD_PARENT, tv.TV_TREE_BAD_PARENT,
                                 tv.TV_TREE_BAD_TOKEN, tv.TV_TREE_DUP_SIBLING,
                                 tv.TV_TREE_NONFINITE]
    for b in range(1, 6):
        assert g["accept_len"][b] == -1 and g["bonus_token"][b] == -1
        assert np.all(g["node_state"][b] == 0) and np.all(g["node_theta"][b] == -1)
    rep = parity.check(bt, tokenlevel, gpu=g, p_init=not tokenlevel, label="errors")
    assert_clean(rep, "error trees")


def test_masked_vocabulary_and_misaligned_base():
    """Logits with -inf entries (masked tokens) and tensors whose base address is
    2 bytes past a 16-byte boundary (every row starts misaligned)."""
    rng = np.random.default_rng(5)
    par = np.tile(W.binary_parents(2), (16, 1))
    B, n1, V = 16, 7, 1031
    bt = _rand_batch(rng, par, V, dtype="bf16", mode=W.WITHOUT_REPLACEMENT)
    mask = torch.as_tensor(rng.random((B, n1, V)) < 0.2, device=DEV)
    toks = bt["tokens"].long()
    pidx = bt["parents"].long().clamp(min=0)
    for t in ("target", "draft"):
        x = bt[t].clone()
        x[mask] = float("-inf")
        # drafted tokens keep a finite draft logit at their parent
        bidx = torch.arange(B, device=DEV).unsqueeze(1).expand(B, n1)
        x[bidx[:, 1:], pidx[:, 1:], toks[:, 1:]] = bt[t][bidx[:, 1:], pidx[:, 1:], toks[:, 1:]]
        flat = torch.empty(B * n1 * V + 8, dtype=x.dtype, device=DEV)
        view = flat[1:1 + B * n1 * V].view(B, n1, V)
        view.copy_(x)
        bt[t] = view
    assert bt["target"].data_ptr() % 16 == 2
    for tl in (False, True):
        rep = parity.check(bt, tl, p_init=not tl, label="masked")
        assert_clean(rep, f"masked+misaligned tokenlevel={tl}")


def test_deterministic():
    bt = W.make_batch(5, step=4, device=DEV, mode=W.WITHOUT_REPLACEMENT, batch=64, vocab=50000)
    a = parity.run_gpu(bt, False, p_init=True)
    b = parity.run_gpu(bt, False, p_init=True)
    for k in a:
        if a[k] is not None:
            assert np.array_equal(a[k], b[k]), k


def test_repeated_launches_with_helpers_agree():
    """The full 256-tree, V=128256 batch, launched several times: helpers join
    at timing-dependent points, so the last bits of the sums may differ, but
    every decision, accepted node, Y and status must be the same, and the
    acceptance probabilities the same to well within the fp32 tolerance."""
    bt = W.make_batch(5, step=7, device=DEV, mode=W.WITHOUT_REPLACEMENT, batch=256)
    runs = [parity.run_gpu(bt, False) for _ in range(4)]
    a = runs[0]
    assert (a["status"] == tv.TV_TREE_OK).all()
    for b in runs[1:]:
        for k in ("status", "accept_len", "accepted_node", "bonus_token", "node_state"):
            assert np.array_equal(a[k], b[k]), k
        th_a, th_b = a["node_theta"], b["node_theta"]
        assert np.allclose(th_a, th_b, rtol=1e-6, atol=1e-9)
    rep = parity.check(bt, False, trees=[0, 85, 170, 255], gpu=a, label="repeat")
    assert_clean(rep, "repeated launches")
    del bt
    torch.cuda.empty_cache()
