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

@pytest.mark.parametrize("cfg,trees", [(2, None), (3, None), (4, None), (5, list(range(0, 256, 8)))])
def test_configs_full_size(cfg, trees):
    for mode in MODES:
        bt = W.make_batch(cfg, step=3, device=DEV, mode=mode)
        for tl in (False, True):
            rep = parity.check(bt, tl, trees=trees, label=f"cfg{cfg}-full")
            assert_clean(rep, f"cfg{cfg} full mode={mode} tokenlevel={tl}")
        rep = parity.check(bt, False, trees=trees, label=f"cfg{cfg}-full-early", theta=False)
        assert_clean(rep, f"cfg{cfg} full mode={mode} early rejection")
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
