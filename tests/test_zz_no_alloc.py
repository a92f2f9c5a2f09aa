"""The loss head that allocates nothing (digest_softmax_xent_static, whose
partial sums live in the library's fixed device array) against the
workspace entry point digest_softmax_xent: the same kernels and the same
block partition, so the outputs must agree bit for bit (and with the oracle
within rtol 1e-4 / atol 1e-5), on two calls in a row, the second smaller,
plus the size limit and argument errors.  Called through the C ABI."""
import ctypes

import numpy as np
import pytest

import oracle
from paper_2206_00057_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def workspace_loss(n, C, logits, labels):
    """digest_softmax_xent of a partition of n rows (no entries, no halo)."""
    from paper_2206_00057_amd import digest as D
    h = D.digest_partition_create(n, np.zeros(n + 1, np.int64), np.zeros(0, np.int64),
                                  np.zeros(0, np.float32), np.arange(n, dtype=np.int64),
                                  np.zeros(0, np.int64), [C, C])
    ws = torch.empty(max(h.workspace_bytes, 256), dtype=torch.uint8, device="cuda")
    D.digest_partition_bind_workspace(h, ws)
    dl = torch.full((n, C), float("nan"), device="cuda")
    loss = torch.full((1,), float("nan"), device="cuda")
    D.digest_softmax_xent(h, logits, labels, dl, loss)
    return host(dl), host(loss)


def static_loss(n, C, logits, labels, stream=None):
    from paper_2206_00057_amd import digest as D
    dl = torch.full((n, C), float("nan"), device="cuda")
    loss = torch.full((1,), float("nan"), device="cuda")
    st = D.lib().digest_softmax_xent_static(
        ctypes.c_int64(n), ctypes.c_int32(C), ctypes.c_void_p(logits.data_ptr()),
        ctypes.c_void_p(labels.data_ptr()), ctypes.c_void_p(dl.data_ptr()),
        ctypes.c_void_p(loss.data_ptr()),
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream if stream is None else stream))
    assert st == D.OK, D.lib().digest_last_error()
    return host(dl), host(loss)


@pytest.mark.parametrize("C", [7, 47, 130])
def test_static_loss_matches_workspace_entry_point(C):
    from paper_2206_00057_amd import digest as D
    # the second call is smaller: the partial sums of the first stay in the
    # array and must not leak into it
    for n, seed in ((306_250, 1), (1_001, 2)):
        logits = synth.normal((n, C), seed=seed, scale=3.0)
        labels = np.random.default_rng(seed).integers(0, C, n).astype(np.int32)
        dlog, dlab = dev(logits), dev(labels)
        ref_dl, ref_loss = workspace_loss(n, C, dlog, dlab)
        got_dl, got_loss = static_loss(n, C, dlog, dlab)
        np.testing.assert_array_equal(got_dl.view(np.uint32), ref_dl.view(np.uint32))
        np.testing.assert_array_equal(got_loss.view(np.uint32), ref_loss.view(np.uint32))
        # the Python binding of the same call
        dl2 = torch.empty(n, C, device="cuda")
        loss2 = torch.empty(1, device="cuda")
        D.digest_softmax_xent_static(dlog, dlab, dl2, loss2)
        np.testing.assert_array_equal(host(dl2).view(np.uint32), ref_dl.view(np.uint32))
        np.testing.assert_array_equal(host(loss2).view(np.uint32), ref_loss.view(np.uint32))
        o_loss, o_dl = oracle.softmax_xent(logits, labels)
        err = np.abs(got_dl.astype(np.float64) - o_dl)
        assert not (err > 1e-5 + 1e-4 * np.abs(o_dl)).any()
        assert abs(float(got_loss[0]) - o_loss) <= 1e-5 + 1e-4 * abs(o_loss)


def test_static_loss_rejects_bad_arguments():
    from paper_2206_00057_amd import digest as D
    L = D.lib()
    buf = torch.zeros(16, device="cuda")
    p = ctypes.c_void_p(buf.data_ptr())
    limit = 262144 * 16   # 47 classes: 16 rows per partial sum
    assert L.digest_softmax_xent_static(limit + 1, 47, p, p, p, p, None) == D.EINVAL
    assert b"static scratch" in L.digest_last_error()
    assert L.digest_softmax_xent_static(-1, 47, p, p, p, p, None) == D.EINVAL
    assert L.digest_softmax_xent_static(4, 0, p, p, p, p, None) == D.EINVAL
    assert L.digest_softmax_xent_static(4, 47, None, p, p, p, None) == D.EINVAL
    assert L.digest_softmax_xent_static(4, 47, p, p, p, None, None) == D.EINVAL
    # no rows: loss 0, nothing else touched
    loss = torch.full((1,), float("nan"), device="cuda")
    assert L.digest_softmax_xent_static(0, 47, None, None, None,
                                        ctypes.c_void_p(loss.data_ptr()), None) == D.OK
    assert float(host(loss)[0]) == 0.0
