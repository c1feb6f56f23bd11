"""tv_verify_noalloc (the library's own device scratch, no workspace argument)
against tv_verify (the caller's workspace) on the same inputs, through the
C-ABI: two calls in a row, the second smaller than the first, so that the
second runs on scratch the first left behind. Both must also match the CPU
oracle tree by tree (needs an MI355X)."""

import numpy as np
import pytest
import torch

import paper_2505_12398_amd as tv
import parity
import workloads as W

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _outputs(B, n1, dev):
    i32 = dict(dtype=torch.int32, device=dev)
    return tv.VerifyOutputs(
        accept_len=torch.full((B,), -7, **i32), accepted_node=torch.full((B,), -7, **i32),
        bonus_token=torch.full((B,), -7, **i32), status=torch.full((B,), -7, **i32),
        node_state=torch.full((B, n1), 9, dtype=torch.int8, device=dev),
        node_theta=torch.full((B, n1), 9.0, dtype=torch.float32, device=dev),
        p_init=torch.full((B, n1), 9.0, dtype=torch.float32, device=dev),
        counters=torch.full((B, tv.TV_NUM_COUNTERS), -7, **i32))


def _call(fn, bt, out, **extra):
    B, n1 = bt["parents"].shape
    V = bt["target"].shape[-1]
    dtype = tv.TV_DTYPE_BF16 if bt["target"].dtype == torch.bfloat16 else tv.TV_DTYPE_F32
    st = fn(B, n1, V, bt["parents"], bt["tokens"], bt["target"], bt["draft"], dtype,
            bt["temperature"], bt["uniforms"], bt["mode"], out.accept_len, out.accepted_node,
            out.bonus_token, out.status, out.node_state, out.node_theta, out.p_init,
            out.counters, stream=torch.cuda.current_stream().cuda_stream, **extra)
    assert st == tv.TV_OK, tv.tv_status_string(st)
    return parity.host_outputs(out)


def _check_pair(bt, label):
    B, n1 = bt["parents"].shape
    V = bt["target"].shape[-1]
    a = _call(tv.tv_verify_noalloc, bt, _outputs(B, n1, DEV))
    ws, nbytes = tv.workspace_tensor(B, n1, V, DEV)
    b = _call(tv.tv_verify, bt, _outputs(B, n1, DEV), workspace=ws, workspace_bytes=nbytes)
    torch.cuda.synchronize()
    assert (a["status"] == tv.TV_TREE_OK).all(), label
    for k in ("status", "accept_len", "accepted_node", "bonus_token", "node_state",
              "counters"):
        assert np.array_equal(a[k], b[k]), (label, k)
    for k in ("node_theta", "p_init"):
        assert np.allclose(a[k], b[k], rtol=1e-6, atol=1e-9), (label, k)
    rep = parity.check(bt, False, p_init=True, gpu=a, label=label)
    print(f"{label}: {rep.summary()}", flush=True)
    assert not rep.failures, "\n".join(rep.failures[:10])
    assert rep.near_ties <= max(1, rep.trees // 100), rep.summary()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tv.load_library()
    yield


def test_noalloc_matches_workspace_entry_point_twice():
    # first call: 64 trees of the 64-node benchmark shape, bf16, V = 32003
    big = W.make_batch(5, step=11, device=DEV, mode=W.WITHOUT_REPLACEMENT, batch=64,
                       vocab=32003)
    _check_pair(big, "noalloc 64 trees bf16")
    # second call, smaller: 12 complete binary trees, fp32, V = 20011, i.i.d. siblings
    small = W.make_batch(3, step=12, device=DEV, mode=W.WITH_REPLACEMENT, batch=12,
                         vocab=20011)
    small["target"] = small["target"].float()
    small["draft"] = small["draft"].float()
    small["dtype"] = "f32"
    _check_pair(small, "noalloc 12 trees f32")
