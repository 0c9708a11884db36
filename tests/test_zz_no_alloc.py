"""sao_clipped_loss_noalloc, the entry point whose scratch is the library's static
per-device array, against sao_clipped_loss with a caller workspace (the same
kernels, so every output must agree bit for bit) and against the oracle.

Three calls in a row share the device's one scratch array: a batch large enough
to use every block of partials, with N counted in the scratch; then a smaller
batch, which must not see anything the first left behind; then one with the
caller's N. All calls go through the C ABI (ctypes), on the current stream.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_07508_amd as sao

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return sao.lib()


def _inputs(T, seed, eps_low, eps_high):
    rng = np.random.default_rng(seed)
    lro = rng.uniform(-6.0, -0.01, T).astype(np.float32)
    # log-ratios spread across both band edges
    d = rng.normal(0.0, 0.3, T)
    lp = (lro.astype(np.float64) + d).astype(np.float32)
    adv = rng.normal(0.0, 1.0, T).astype(np.float32)
    mask = (rng.random(T) < 0.7).astype(np.uint8)
    return lp, lro, adv, mask


def _call(L, fn_name, arrays, T, eps_low, eps_high, n_dev, ws=None):
    lp, lro, adv, mask = arrays
    loss = torch.zeros(2, dtype=torch.float64, device="cuda")
    counts = torch.zeros(5, dtype=torch.int64, device="cuda")
    g = torch.full((T,), float("nan"), dtype=torch.float32, device="cuda")
    flags = torch.full((T,), 255, dtype=torch.uint8, device="cuda")
    st = torch.cuda.current_stream().cuda_stream
    p = lambda t: None if t is None else t.data_ptr()  # noqa: E731
    common = [p(lp), p(lro), p(adv), p(mask), T, eps_low, eps_high, p(n_dev), p(loss), p(g), p(flags), p(counts)]
    if fn_name == "sao_clipped_loss_noalloc":
        code = L.sao_clipped_loss_noalloc(*common, st)
    else:
        code = L.sao_clipped_loss(*common, p(ws), ws.numel(), st)
    assert code == 0, L.sao_last_error_message()
    torch.cuda.synchronize()
    return loss.cpu().numpy(), g.cpu().numpy(), flags.cpu().numpy(), counts.cpu().numpy()


@pytest.mark.parametrize("T1,T2", [(5_000_000, 1_000), (2_100_000, 70_003)])
def test_noalloc_matches_workspace_entry_point(L, T1, T2):
    eps_low, eps_high = 0.2, 0.28
    results = []
    for i, (T, with_n) in enumerate(((T1, False), (T2, False), (T2, True))):
        host = _inputs(T, 100 + i + T1 % 7, eps_low, eps_high)
        dev = [torch.from_numpy(x).cuda() for x in host]
        N = int(host[3].sum())
        n_dev = torch.tensor([N], dtype=torch.int64, device="cuda") if with_n else None
        ws = torch.empty(sao.workspace_size(2, T, 1, 1, 1), dtype=torch.uint8, device="cuda")
        got = _call(L, "sao_clipped_loss_noalloc", dev, T, eps_low, eps_high, n_dev)
        want = _call(L, "sao_clipped_loss", dev, T, eps_low, eps_high, n_dev, ws=ws)
        # the same kernels on the same inputs: bit-identical
        assert np.array_equal(got[0].view(np.int64), want[0].view(np.int64)), (got[0], want[0])
        assert np.array_equal(got[1].view(np.int32), want[1].view(np.int32))
        assert np.array_equal(got[2], want[2]) and np.array_equal(got[3], want[3])
        # and the oracle's bars: flags and counts exact, loss and g within fp32 weight rounding
        rl, rg, rf, rc = oracle.dis_loss(*host, eps_low, eps_high, N)
        assert np.array_equal(got[2], rf) and np.array_equal(got[3], rc)
        used = rf == 1
        rho = np.exp(host[0].astype(np.float64) - host[1])
        scale = (np.abs(rho * host[2] * host[0])[used].sum() / N, np.abs(rho * host[2])[used].sum() / N)
        for k in range(2):
            assert abs(got[0][k] - rl[k]) <= 1e-5 * max(abs(rl[k]), scale[k])
        assert (np.abs(got[1] - rg) <= 1e-5 * np.abs(rg) + 1e-15).all()
        results.append(got)
    # the smaller batch is not the first one's prefix result
    assert results[1][3][0] == int(_inputs(T2, 101 + T1 % 7, eps_low, eps_high)[3].sum())
