"""The accepted-path commit (tv_commit_paths) against the oracle's committed
sequence (Def. def2) on the verifier's own outputs, bit-exact (needs an
MI355X)."""

import numpy as np
import pytest
import torch

import paper_2505_12398_amd as tv
import parity
import workloads as W
from oracle import tv_oracle as O

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tv.load_library()
    yield


def expected(par, tok, out, max_len):
    B = par.shape[0]
    acc, y, st = (out.accepted_node.cpu().numpy(), out.bonus_token.cpu().numpy(),
                  out.status.cpu().numpy())
    pn = np.full((B, max_len), -1, np.int32)
    pt = np.full((B, max_len + 1), -1, np.int32)
    pl = np.zeros(B, np.int32)
    for b in range(B):
        if st[b] != tv.TV_TREE_OK:
            continue
        nodes, toks = O.committed_sequence(par[b], tok[b], int(acc[b]), int(y[b]))
        if len(nodes) > max_len:
            pl[b] = tv.TV_COMMIT_OVERFLOW
            continue
        pn[b, :len(nodes)] = nodes
        pt[b, :len(toks)] = toks
        pl[b] = len(toks)
    return pn, pt, pl


def check(bt, out, max_len):
    pn, pt, pl = tv.commit_paths(bt["parents"], bt["tokens"], out, max_len)
    want = expected(bt["parents"].cpu().numpy(), bt["tokens"].cpu().numpy(), out, max_len)
    for got, w, name in zip((pn, pt, pl), want, ("path_nodes", "path_tokens", "path_len")):
        np.testing.assert_array_equal(got.cpu().numpy(), w, err_msg=name)
    return pl.cpu().numpy()


@pytest.mark.parametrize("tokenlevel", [False, True])
def test_commit_after_verify(tokenlevel):
    """256 benchmark-shaped trees (V reduced to 16381): the commit of the
    verifier's outputs equals the oracle's, and the verifier itself matches the
    oracle; a max_len below some trees' depth reports overflow."""
    bt = W.make_batch(5, step=4, device=DEV, mode=W.WITHOUT_REPLACEMENT, vocab=16381)
    out = tv.verify_batch(bt["parents"], bt["tokens"], bt["target"], bt["draft"],
                          bt["temperature"], bt["uniforms"], bt["mode"], tokenlevel=tokenlevel)
    rep = parity.check(bt, tokenlevel, trees=list(range(0, 256, 16)),
                       gpu=parity.host_outputs(out), label="commit")
    assert not rep.failures, rep.failures[:3]
    pl = check(bt, out, 8)
    assert (pl == out.accept_len.cpu().numpy() + 1).all()
    pl = check(bt, out, 1)
    assert (pl == tv.TV_COMMIT_OVERFLOW).any()
    check(bt, out, 0)


def test_commit_edge_cases():
    """Error trees give length 0; an accepted node out of range or a link that
    does not point back gives TV_COMMIT_INCONSISTENT; the root accepted gives
    Y alone."""
    par = torch.tensor([[-1, 0, 1, 1], [-1, 0, 1, 1], [-1, 0, 2, 1], [-1, 0, 1, 1]],
                       dtype=torch.int32, device=DEV)
    tok = torch.tensor([[0, 5, 6, 7]] * 4, dtype=torch.int32, device=DEV)
    out = tv.VerifyOutputs(
        accept_len=torch.zeros(4, dtype=torch.int32, device=DEV),
        accepted_node=torch.tensor([3, 9, 2, 0], dtype=torch.int32, device=DEV),
        bonus_token=torch.tensor([11, 12, 13, 14], dtype=torch.int32, device=DEV),
        status=torch.tensor([0, 0, 0, tv.TV_TREE_OK], dtype=torch.int32, device=DEV))
    pn, pt, pl = tv.commit_paths(par, tok, out, 3)
    assert pl.cpu().tolist() == [3, tv.TV_COMMIT_INCONSISTENT, tv.TV_COMMIT_INCONSISTENT, 1]
    assert pn.cpu().tolist()[0] == [1, 3, -1] and pt.cpu().tolist()[0] == [5, 7, 11, -1]
    assert pt.cpu().tolist()[3] == [14, -1, -1, -1]
    out.status[0] = tv.TV_TREE_NONFINITE
    pn, pt, pl = tv.commit_paths(par, tok, out, 3)
    assert pl.cpu().tolist()[0] == 0 and pt.cpu().tolist()[0] == [-1] * 4
