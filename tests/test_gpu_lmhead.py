"""The LM head with fused row statistics (tv_lmhead_stats) and the verifier
that takes them (tv_verify_stats), against the oracle (needs an MI355X).

Logits: each must lie within the rounding of its exact value (oracle.lmhead
.logits, float64): bf16 rounding (2^-9 relative, to nearest even, taken as
2^-8 here) plus float32 accumulation of K products (K 2^-24 times the sum of
the products' magnitudes). Statistics: the row maximum must equal the maximum
of the logits the kernel wrote, and the sum must match the oracle's
sum exp((z - max) / T) of those same logits within 1e-5 relative (float32
terms). Verification with the statistics given: tree by tree against the
oracle on the same logits."""

import numpy as np
import pytest
import torch

import oracle.lmhead as LM
import paper_2505_12398_amd as tv
import parity
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tv.load_library()
    yield


def _bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def _check_logits(x, w, z_gpu, rows=None):
    """Kernel logits (bf16 tensor) against the exact products within the
    rounding bound; ``rows`` restricts the check to sampled rows."""
    xb, wb = _bits(x), _bits(w)
    if rows is not None:
        xb = xb[rows]
    exact = LM.logits(xb, wb)
    bound = LM.accumulation_bound(xb, wb)
    K = xb.shape[1]
    got = _bits(z_gpu if rows is None else z_gpu[rows])
    gz = LM.to_f64(got)
    tol = 2.0 ** -8 * np.abs(exact) + 2.0 * K * 2.0 ** -24 * bound + 1e-30
    err = np.abs(gz - exact)
    worst = float((err / tol).max())
    assert np.all(err <= tol), f"logit error {worst:.3f} x the bound"
    nearest = torch.as_tensor(exact).to(torch.bfloat16).double().numpy()
    same = float(np.mean(gz == nearest))
    return got, worst, same


def _check_stats(got_bits, row_max, row_sum, T):
    m, s = LM.row_stats(got_bits, T)
    gm = row_max.detach().cpu().numpy().astype(np.float64)
    gs = row_sum.detach().cpu().numpy()
    assert np.array_equal(gm, m), "row maximum differs from the maximum of the logits"
    rel = np.abs(gs - s) / s
    assert np.all(rel < 1e-5), float(rel.max())
    return float(rel.max())


@pytest.mark.parametrize("M,K,N,T", [(37, 72, 301, 1.0), (130, 200, 1000, 0.7),
                                     (300, 4096, 2053, 1.9), (257, 512, 4097, 0.2),
                                     (1, 8, 2, 1.0)])
def test_lmhead_ragged_tiles(M, K, N, T):
    """Row, column and K tails (none of M, N a multiple of 128, K of 64), the
    lowest temperature of the paper's sweep (T = 0.2, Table 4), and the
    smallest shapes the library takes (one row, K = 8, V = 2)."""
    g = torch.Generator(device=DEV).manual_seed(M * 7 + N)
    x = torch.randn((M, K), generator=g, device=DEV).to(torch.bfloat16)
    w = (torch.randn((N, K), generator=g, device=DEV) * (3.0 / K ** 0.5)).to(torch.bfloat16)
    z, rm, rs = tv.lmhead_stats(x, w, T)
    torch.cuda.synchronize()
    got, worst, same = _check_logits(x, w, z)
    rel = _check_stats(got, rm, rs, T)
    print(f"lmhead M={M} K={K} N={N} T={T}: worst {worst:.3f} of the bound, "
          f"{same:.4f} equal to the rounded exact value, stats rel err {rel:.2e}", flush=True)


def test_lmhead_rounding_is_nearest_even():
    """Integer inputs whose products and fp32 sums are exact (|sum| < 2^24),
    with sums of up to 13 significant bits: the bf16 rounding is then the only
    rounding, and every logit must be the exact sum rounded to nearest even
    (torch's float32 -> bfloat16 conversion), bit for bit. Ties occur (sums
    with 9 significant bits whose last is 1) and must round to even."""
    M, K, N = 130, 96, 515
    g = torch.Generator(device="cpu").manual_seed(41)
    x = torch.randint(-12, 13, (M, K), generator=g).float()
    w = torch.randint(-12, 13, (N, K), generator=g).float()
    z, _, _ = tv.lmhead_stats(x.to(DEV).to(torch.bfloat16), w.to(DEV).to(torch.bfloat16), 1.0)
    torch.cuda.synchronize()
    exact = x.double() @ w.double().T
    assert exact.abs().max() < 2 ** 24
    want = exact.float().to(torch.bfloat16)
    got = z.cpu()
    assert torch.equal(got.view(torch.int16), want.view(torch.int16)), \
        int((got.view(torch.int16) != want.view(torch.int16)).sum())
    ties = int(((exact.abs().long() % 2 == 1) & (exact.abs() >= 256) & (exact.abs() < 512)).sum())
    print(f"lmhead rounding: {M * N} logits equal to the nearest-even rounding, {ties} ties", flush=True)
    assert ties > 0


def test_lmhead_misaligned_logits():
    """Logits written into a buffer that starts 2 bytes past a 16-byte
    boundary (the element-by-element store path), N a multiple of 8: equal bit
    for bit to the same call into an aligned buffer, statistics included."""
    M, K, N = 300, 136, 1024
    g = torch.Generator(device=DEV).manual_seed(17)
    x = torch.randn((M, K), generator=g, device=DEV).to(torch.bfloat16)
    w = (torch.randn((N, K), generator=g, device=DEV) * 0.3).to(torch.bfloat16)
    z0, m0, s0 = tv.lmhead_stats(x, w, 0.9)
    flat = torch.zeros(M * N + 1, dtype=torch.bfloat16, device=DEV)
    z1 = flat[1:].view(M, N)
    assert z1.data_ptr() % 16 == 2
    out = (z1, torch.empty(M, device=DEV), torch.empty(M, dtype=torch.float64, device=DEV))
    tv.lmhead_stats(x, w, 0.9, out=out)
    torch.cuda.synchronize()
    assert torch.equal(z1.view(torch.int16), z0.view(torch.int16))
    assert torch.equal(out[1], m0) and torch.equal(out[2], s0)
    assert flat[0].item() == 0.0      # nothing written before the buffer


def test_lmhead_benchmark_shape_sampled_rows():
    """The benchmark's shape: 16640 rows (256 trees x 65 nodes), hidden 4096,
    V = 128256; 24 sampled rows checked against the exact products, every
    row's statistics against the oracle's on the kernel's logits of 48 rows."""
    M, K, N = 16640, 4096, 128256
    g = torch.Generator(device=DEV).manual_seed(5)
    x = torch.randn((M, K), generator=g, device=DEV).to(torch.bfloat16)
    w = (torch.randn((N, K), generator=g, device=DEV) * (3.0 / K ** 0.5)).to(torch.bfloat16)
    z, rm, rs = tv.lmhead_stats(x, w, 1.0)
    torch.cuda.synchronize()
    rows = [0, 1, 127, 128, 129, 4095, 8191, 8192, 12000, 16511, 16512, 16639] + \
        list(range(3001, 3013))
    got, worst, same = _check_logits(x, w, z, rows)
    rel = _check_stats(got, rm[rows], rs[rows], 1.0)
    more = list(range(0, M, M // 48))
    rel2 = _check_stats(_bits(z[more]), rm[more], rs[more], 1.0)
    print(f"lmhead benchmark shape: worst {worst:.3f} of the bound, {same:.4f} equal, "
          f"stats rel err {max(rel, rel2):.2e}", flush=True)
    del x, w, z
    torch.cuda.empty_cache()


def test_lmhead_nonfinite_rows():
    """A NaN or an infinity in a row's hidden state makes that row's sum
    non-finite and leaves the other rows as they were."""
    M, K, N = 64, 128, 500
    g = torch.Generator(device=DEV).manual_seed(9)
    x = torch.randn((M, K), generator=g, device=DEV).to(torch.bfloat16)
    w = (torch.randn((N, K), generator=g, device=DEV) * 0.2).to(torch.bfloat16)
    _, rm0, rs0 = tv.lmhead_stats(x, w, 1.0)
    x2 = x.clone()
    x2[3, 5] = float("nan")
    x2[40, 0] = float("inf")
    _, rm, rs = tv.lmhead_stats(x2, w, 1.0)
    rs_h, rs0_h = rs.cpu().numpy(), rs0.cpu().numpy()
    assert not np.isfinite(rs_h[3]) and not np.isfinite(rs_h[40])
    keep = [i for i in range(M) if i not in (3, 40)]
    assert np.array_equal(rs_h[keep], rs0_h[keep])


def _stats_np(bt):
    """Oracle row statistics of a batch's target and draft rows, as tensors."""
    host = parity.host_batch(bt)
    T = bt["temperature"]
    out = []
    for rows in (host[2], host[3]):
        m, s = LM.row_stats(rows, T)
        out += [torch.as_tensor(m.astype(np.float32), device=DEV),
                torch.as_tensor(s, device=DEV)]
    return tuple(out), host


@pytest.mark.parametrize("mode", [W.WITHOUT_REPLACEMENT, W.WITH_REPLACEMENT])
def test_verify_stats_benchmark_workload(mode):
    """tv_verify_stats on the full large-batch workload (256 trees, V=128256
    bf16) with the oracle's row statistics: every tree against the oracle
    (with theta, and without: early rejection)."""
    bt = W.make_batch(5, step=13, device=DEV, mode=mode)
    stats, host = _stats_np(bt)
    B = bt["parents"].shape[0]
    refs = parity.oracle_many(bt, range(B), tokenlevels=(False,), host=host)[False]
    for theta in (True, False):
        g = parity.host_outputs(tv.verify_batch(
            bt["parents"], bt["tokens"], bt["target"], bt["draft"], bt["temperature"],
            bt["uniforms"], mode, want_theta=theta, want_p_init=theta, stats=stats))
        rep = parity.check(bt, False, trees=list(range(B)), refs=refs, gpu=g, theta=theta,
                           p_init=theta, label=f"verify_stats mode={mode} theta={theta}")
        print(f"verify_stats mode={mode} theta={theta}: {rep.summary()}", flush=True)
        assert not rep.failures, "\n".join(rep.failures[:10])
        assert rep.near_ties <= max(1, B // 100)
        assert rep.max_theta_abs < parity.BAND, rep.summary()
    del bt
    torch.cuda.empty_cache()


def test_lmhead_then_verify_stats_pipeline():
    """The two model layers and the verifier end to end: 32 trees of the
    large-batch shape (65 rows each); target logits from one LM head (hidden
    512, V = 32003), draft logits from a perturbed copy of it; children drawn
    from the draft on the device (tv_draft_tokens); then tv_verify_stats on
    the statistics the LM heads produced, tree by tree against the oracle on
    the logits they produced."""
    B, n1, K, V = 32, 65, 512, 32003
    g = torch.Generator(device=DEV).manual_seed(77)
    parents = torch.as_tensor(W.make_parents(W.CONFIGS[5], B, (0, 5, 77)), device=DEV)
    h = torch.randn((B, n1, K), generator=g, device=DEV).to(torch.bfloat16)
    wt = torch.randn((V, K), generator=g, device=DEV) * (3.0 / K ** 0.5)
    wd = wt + torch.randn((V, K), generator=g, device=DEV) * (1.5 / K ** 0.5)
    zt, tm, ts = tv.lmhead_stats(h, wt.to(torch.bfloat16), 1.0)
    zd, dm, ds = tv.lmhead_stats(h, wd.to(torch.bfloat16), 1.0)
    u = torch.randint(0, 2 ** 24, (B, n1), generator=g, device=DEV).float() * 2.0 ** -24
    ud = torch.randint(0, 2 ** 24, (B, n1), generator=g, device=DEV).float() * 2.0 ** -24
    mode = W.WITHOUT_REPLACEMENT
    tok, st = tv.draft_tokens(parents, zd, 1.0, ud, mode)
    assert (st == tv.TV_TREE_OK).all()
    bt = {"parents": parents, "tokens": tok, "target": zt, "draft": zd, "uniforms": u,
          "temperature": 1.0, "mode": mode, "dtype": "bf16"}
    # the statistics the LM heads produced are those of the logits they wrote
    for z, m, s in ((zt, tm, ts), (zd, dm, ds)):
        _check_stats(_bits(z.reshape(B * n1, V)), m.reshape(-1), s.reshape(-1), 1.0)
    stats = (tm, ts, dm, ds)
    refs = parity.oracle_many(bt, range(B), tokenlevels=(False,))[False]
    g_out = parity.host_outputs(tv.verify_batch(parents, tok, zt, zd, 1.0, u, mode,
                                                want_p_init=True, stats=stats))
    rep = parity.check(bt, False, trees=list(range(B)), refs=refs, gpu=g_out, p_init=True,
                       label="pipeline")
    print(f"lmhead -> verify_stats pipeline: {rep.summary()}", flush=True)
    assert not rep.failures, "\n".join(rep.failures[:10])
    assert rep.near_ties <= 1
    assert rep.max_theta_abs < parity.BAND, rep.summary()


@pytest.mark.parametrize("cfg,vocab", [(2, None), (3, 4099), (4, 20000)])
@pytest.mark.parametrize("mode", [W.WITHOUT_REPLACEMENT, W.WITH_REPLACEMENT])
def test_verify_stats_other_workloads(cfg, vocab, mode):
    """tv_verify_stats with the oracle's row statistics on the other workloads:
    the precise element path (fp32 logits of the chain workload; bf16 logits
    below 16384 tokens, the binary-tree workload at V = 4099, T = 0.7) and the
    fast one on the irregular workload at V = 20000; every tree against the
    oracle, with theta (no early rejection) and without."""
    bt = W.make_batch(cfg, step=17, device=DEV, mode=mode, vocab=vocab)
    stats, host = _stats_np(bt)
    B = bt["parents"].shape[0]
    refs = parity.oracle_many(bt, range(B), tokenlevels=(False,), host=host)[False]
    for theta in (True, False):
        g = parity.host_outputs(tv.verify_batch(
            bt["parents"], bt["tokens"], bt["target"], bt["draft"], bt["temperature"],
            bt["uniforms"], mode, want_theta=theta, want_p_init=theta, stats=stats))
        rep = parity.check(bt, False, trees=list(range(B)), refs=refs, gpu=g, theta=theta,
                           p_init=theta, label=f"verify_stats cfg{cfg} mode={mode} theta={theta}")
        print(f"verify_stats cfg{cfg} V={bt['target'].shape[-1]} mode={mode} theta={theta}: "
              f"{rep.summary()}", flush=True)
        assert not rep.failures, "\n".join(rep.failures[:10])
        assert rep.near_ties <= max(1, B // 100)


def test_verify_stats_bad_statistics():
    """Statistics that cannot normalise a consulted row (the root's, which every
    tree with children consults): a NaN target sum, a zero draft sum, an
    infinite target maximum, a -inf draft maximum. Each such tree reports
    TV_TREE_NONFINITE with the sentinel outputs; the other trees of the launch
    match the oracle."""
    bt = W.make_batch(5, step=21, device=DEV, mode=W.WITHOUT_REPLACEMENT, batch=8, vocab=32768)
    stats, host = _stats_np(bt)
    tmax, tsum, dmax, dsum = [s.clone() for s in stats]
    tsum[1, 0] = float("nan")
    dsum[2, 0] = 0.0
    tmax[3, 0] = float("inf")
    dmax[4, 0] = float("-inf")
    g = parity.host_outputs(tv.verify_batch(
        bt["parents"], bt["tokens"], bt["target"], bt["draft"], bt["temperature"],
        bt["uniforms"], bt["mode"], want_theta=True, want_p_init=True,
        stats=(tmax, tsum, dmax, dsum)))
    for b in (1, 2, 3, 4):
        assert g["status"][b] == tv.TV_TREE_NONFINITE, (b, g["status"][b])
        assert g["accept_len"][b] == -1 and g["accepted_node"][b] == -1
        assert g["bonus_token"][b] == -1
    good = [0, 5, 6, 7]
    refs = parity.oracle_many(bt, good, tokenlevels=(False,), host=host)[False]
    rep = parity.check(bt, False, trees=good, refs=refs, gpu=g, theta=True, p_init=True,
                       label="verify_stats bad statistics")
    assert not rep.failures, "\n".join(rep.failures[:10])
