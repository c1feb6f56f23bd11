"""The device draft-tree token sampler (tv_draft_tokens) against the CPU oracle
on the same seeded inputs (needs an MI355X). Tokens are integers decided by
floating point: they must be identical, except where the oracle's u*W lies
within 1e-6*W of a CDF boundary (a near-tie, counted)."""

import numpy as np
import pytest
import torch

import paper_2505_12398_amd as tv
import parity
import workloads as W
from oracle import draft_sampler as DS

pytestmark = pytest.mark.gpu
DEV = "cuda"
MODES = [W.WITHOUT_REPLACEMENT, W.WITH_REPLACEMENT]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tv.load_library()
    yield


def _host_rows(t, b):
    t = t[b].detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def check_sampler(parents, draft, T, uniforms, mode, trees=None, label=""):
    """Runs the sampler on the whole batch and compares the listed trees with
    the oracle. Returns (exact, near_ties)."""
    tok, st = tv.draft_tokens(parents, draft, T, uniforms, mode)
    torch.cuda.synchronize()
    tok, st = tok.cpu().numpy(), st.cpu().numpy()
    par_h, u_h = parents.cpu().numpy(), uniforms.cpu().numpy()
    B = parents.shape[0]
    exact = near = 0
    for b in (range(B) if trees is None else trees):
        ref = DS.draw_tree_tokens(par_h[b], _host_rows(draft, b), T, u_h[b], mode)
        assert st[b] == ref.status, f"{label} tree {b}: status gpu {st[b]} oracle {ref.status}"
        if np.array_equal(tok[b], ref.tokens):
            exact += 1
        elif ref.margin < parity.BAND:
            near += 1
        else:
            raise AssertionError(f"{label} tree {b}: tokens gpu {tok[b].tolist()} oracle "
                                 f"{ref.tokens.tolist()} margin {ref.margin:.2e}")
    n = exact + near
    print(f"{label}: {n} trees, {exact} exact, {near} near-ties", flush=True)
    assert near <= max(1, n // 100), (label, exact, near)
    return exact, near


def _random_trees(rng, B, n1, max_back=4):
    par = np.zeros((B, n1), np.int32)
    par[:, 0] = -1
    for b in range(B):
        for i in range(1, n1):
            par[b, i] = rng.integers(max(0, i - max_back), i)
    return par


@pytest.mark.parametrize("mode", MODES)
def test_tiny_vocabularies(mode):
    """V in {2, 3, 5, 17} float32 (rows misaligned for odd V), random trees of
    9 nodes; without replacement some nodes have more children than tokens
    (DEGENERATE)."""
    rng = np.random.default_rng(10 + mode)
    for V in (2, 3, 5, 17):
        B, n1 = 64, 9
        par = _random_trees(rng, B, n1)
        zs = rng.normal(0, 2.0, (B, n1, V)).astype(np.float32)
        u = W.uniforms_np(rng, (B, n1))
        check_sampler(torch.as_tensor(par, device=DEV), torch.as_tensor(zs, device=DEV), 1.0,
                      torch.as_tensor(u, device=DEV), mode, label=f"V={V} mode={mode}")


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("cfg,vocab,batch,dtype", [(2, 32003, 16, "f32"), (3, 20011, 12, "bf16"),
                                                   (4, 12347, 8, "bf16"), (5, 16381, 24, "bf16"),
                                                   (5, 4099, 24, "f32")])
def test_config_shapes_reduced(cfg, vocab, batch, dtype, mode):
    """The benchmark's tree shapes and logit laws at reduced vocabularies
    (ragged tails), both element paths, every tree compared."""
    bt = W.make_batch(cfg, step=7, device=DEV, mode=mode, batch=batch, vocab=vocab)
    draft = bt["draft"].to(torch.bfloat16 if dtype == "bf16" else torch.float32).contiguous()
    rng = np.random.default_rng(cfg * 100 + vocab)
    u = torch.as_tensor(W.uniforms_np(rng, tuple(bt["parents"].shape)), device=DEV)
    check_sampler(bt["parents"], draft, bt["temperature"], u, mode,
                  label=f"cfg{cfg} V={vocab} {dtype} mode={mode}")


def test_full_size_sampled():
    """256 trees x 65 nodes, V = 128256 bf16 (the benchmark's shape), 16
    sampled trees per mode."""
    for mode in MODES:
        bt = W.make_batch(5, step=8, device=DEV, mode=mode)
        rng = np.random.default_rng(55 + mode)
        u = torch.as_tensor(W.uniforms_np(rng, tuple(bt["parents"].shape)), device=DEV)
        check_sampler(bt["parents"], bt["draft"], bt["temperature"], u, mode,
                      trees=list(range(0, 256, 16)), label=f"full mode={mode}")
        del bt
        torch.cuda.empty_cache()


def test_error_trees():
    """A backward-pointing link violated, a NaN in a row with children, and a
    root with three children over two tokens without replacement."""
    rng = np.random.default_rng(12)
    B, n1, V = 4, 5, 2
    par = np.tile(np.array([-1, 0, 0, 0, 1], np.int32), (B, 1))
    par[1, 3] = 4
    zs = rng.normal(0, 1.0, (B, n1, V)).astype(np.float32)
    zs[2, 0, 1] = np.nan
    u = W.uniforms_np(rng, (B, n1))
    args = (torch.as_tensor(par, device=DEV), torch.as_tensor(zs, device=DEV), 1.0,
            torch.as_tensor(u, device=DEV))
    tok, st = tv.draft_tokens(*args, W.WITHOUT_REPLACEMENT)
    st = st.cpu().tolist()
    assert st == [tv.TV_TREE_DEGENERATE, tv.TV_TREE_BAD_PARENT, tv.TV_TREE_NONFINITE,
                  tv.TV_TREE_DEGENERATE]
    assert (tok.cpu().numpy() == -1).all()
    check_sampler(*args, W.WITHOUT_REPLACEMENT, label="errors w/o")
    tok, st = tv.draft_tokens(*args, W.WITH_REPLACEMENT)
    assert st.cpu().tolist() == [0, tv.TV_TREE_BAD_PARENT, tv.TV_TREE_NONFINITE, 0]
    check_sampler(*args, W.WITH_REPLACEMENT, label="errors with")
    # a NaN row (the root's) and a row with three children over two tokens
    par2 = torch.as_tensor(np.array([[-1, 0, 1, 1, 1]], np.int32), device=DEV)
    zs2 = torch.as_tensor(rng.normal(0, 1.0, (1, 5, V)).astype(np.float32), device=DEV)
    zs2[0, 0, 0] = float("nan")
    u2 = torch.as_tensor(W.uniforms_np(rng, (1, 5)), device=DEV)
    tok, st = tv.draft_tokens(par2, zs2, 1.0, u2, W.WITHOUT_REPLACEMENT)
    assert st.cpu().tolist() == [tv.TV_TREE_DEGENERATE]
    check_sampler(par2, zs2, 1.0, u2, W.WITHOUT_REPLACEMENT, label="mixed errors")


@pytest.mark.parametrize("mode", MODES)
def test_drawn_trees_verify(mode):
    """End to end on the device: trees drawn by tv_draft_tokens in one sibling
    mode are verified by tv_verify in the same mode (siblings never repeat
    without replacement, so no DUP_SIBLING), with parity against the oracle."""
    bt = W.make_batch(5, step=9, device=DEV, mode=mode, batch=24, vocab=16381)
    rng = np.random.default_rng(77 + mode)
    u = torch.as_tensor(W.uniforms_np(rng, tuple(bt["parents"].shape)), device=DEV)
    tok, st = tv.draft_tokens(bt["parents"], bt["draft"], bt["temperature"], u, mode)
    assert (st == tv.TV_TREE_OK).all()
    t = tok.clone()
    t[:, 0] = 0
    bt["tokens"] = t.contiguous()
    rep = parity.check(bt, False, label=f"drawn-verify mode={mode}")
    print(f"drawn trees mode={mode}: {rep.summary()}", flush=True)
    assert not rep.failures, "\n".join(rep.failures[:5])


@pytest.mark.parametrize("mode", MODES)
def test_peaked_rows(mode):
    """Rows where one token holds most of the mass (its logit raised by 12
    above the row's N(0, 3^2) values, so it holds more than half of the
    tempered draft at T = 1), V = 128256 bf16: the fast path's chunk sums
    are fp32 sums of unit sums whatever share of the row a chunk has; draws
    must still match the oracle (near-ties aside). 24 random 9-node trees."""
    rng = np.random.default_rng(23)
    B, n1, V = 24, 9, 128256
    par = np.zeros((B, n1), np.int32)
    par[:, 0] = -1
    for b in range(B):
        for i in range(1, n1):
            par[b, i] = rng.integers(max(0, i - 3), i)
    z = rng.normal(0.0, 3.0, (B, n1, V)).astype(np.float32)
    hot = rng.integers(0, V, (B, n1))
    for b in range(B):
        for i in range(n1):
            z[b, i, hot[b, i]] = z[b, i].max() + 12.0
    draft = torch.as_tensor(z, device=DEV).to(torch.bfloat16)
    u = torch.as_tensor(W.uniforms_np(rng, (B, n1)), device=DEV)
    check_sampler(torch.as_tensor(par, device=DEV), draft, 1.0, u, mode,
                  label=f"peaked mode={mode}")

@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("V,dtype,B", [(151936, "bf16", 12), (100003, "f32", 12),
                                       (1 << 20, "bf16", 4)])
def test_chunks_of_several_blocks(V, dtype, B, mode):
    """Vocabularies whose chunks span several 8-unit blocks, so that a chunk's
    running maximum (and frame) rises inside the chunk: 16 units per chunk at
    V = 151936 bf16 (the irregular N=60 workload's vocabulary) and V = 100003
    fp32 (odd: misaligned rows), 64 units per chunk at the largest bf16
    vocabulary, 2^20. Random 9-node trees, rows N(0, 2^2), every tree
    compared."""
    rng = np.random.default_rng(V % 1000 + 31 * mode)
    n1 = 9
    par = _random_trees(rng, B, n1, max_back=3)
    z = torch.as_tensor(rng.normal(0.0, 2.0, (B, n1, V)).astype(np.float32), device=DEV)
    draft = z.to(torch.bfloat16) if dtype == "bf16" else z
    u = W.uniforms_np(rng, (B, n1))
    check_sampler(torch.as_tensor(par, device=DEV), draft.contiguous(), 1.0,
                  torch.as_tensor(u, device=DEV), mode, label=f"V={V} {dtype} mode={mode}")
    del z, draft
    torch.cuda.empty_cache()

@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("T,V,dtype", [(0.2, 128256, "bf16"), (2.0, 128256, "bf16"),
                                       (0.2, 4099, "f32")])
def test_temperatures(T, V, dtype, mode):
    """The lowest temperature of the paper's sweep (Table 4), T = 0.2, where
    k = log2(e)/T multiplies exponents by five and the integer frames take
    large steps, and a high one, T = 2, on both element paths: the
    benchmark's tree shapes and logit law, 16 trees, every tree compared."""
    bt = W.make_batch(5, step=11, device=DEV, mode=mode, batch=16, vocab=V)
    draft = bt["draft"].to(torch.bfloat16 if dtype == "bf16" else torch.float32).contiguous()
    rng = np.random.default_rng(int(T * 10) + V + mode)
    u = torch.as_tensor(W.uniforms_np(rng, tuple(bt["parents"].shape)), device=DEV)
    check_sampler(bt["parents"], draft, T, u, mode, label=f"T={T} V={V} {dtype} mode={mode}")
    del bt, draft
    torch.cuda.empty_cache()
