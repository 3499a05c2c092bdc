"""GPU parity of the token-importance indicators (Sec. 3.3) against the
oracle: hidden-state family (delta-norm of Eq. 3, norm, variance,
cosine-delta) in fp16 and bf16, and the key/value norm, through the C ABI.

Tolerance, from the arithmetic: the kernels sum squares and products in fp32,
each lane a chain of at most 128 terms, then a 64-lane butterfly, so a sum of
non-negative terms is within (128 + 6) * 2^-24 < 1e-5 of its value relative;
a norm's square root halves that.  1 - cos loses the same relative accuracy
of cos as an absolute error (about 3 * 8e-6), hence an absolute 3e-5."""
import numpy as np
import pytest

from oracle import oracle as O

pytestmark = pytest.mark.gpu

RTOL, COS_ATOL = 1e-5, 3e-5


def _close(got, want, ind):
    atol = COS_ATOL if ind == O.COSINE_DELTA else 0.0
    d = np.abs(got.astype(np.float64) - want)
    lim = RTOL * np.abs(want) + atol
    assert np.all(d <= lim), "max excess %.3g at %d" % ((d - lim).max(), int(np.argmax(d - lim)))


def _states(rng, m, B, T, d, bf16):
    import torch
    x = rng.standard_normal((m + 1, B, T, d)).astype(np.float32)
    x *= rng.uniform(0.2, 3.0, (m + 1, B, T, 1)).astype(np.float32)       # layers and tokens differ in scale
    x[1:] = x[:1] + 0.3 * x[1:]                                          # correlated layers (cos near 1)
    t = torch.from_numpy(x).to(torch.bfloat16 if bf16 else torch.float16)
    bits = t.view(torch.int16).numpy().view(np.uint16) if bf16 else t.numpy()
    return t, bits


@pytest.mark.parametrize("bf16", [False, True])
@pytest.mark.parametrize("d", [8, 520, 4096, 8192])
@pytest.mark.parametrize("ind", [O.DELTA_NORM, O.NORM, O.VARIANCE, O.COSINE_DELTA])
def test_hidden_indicators(ind, d, bf16):
    import paper_2608_28911_amd as P
    rng = np.random.default_rng(ind * 100 + d + bf16)
    m, B, T = (4 if ind in (O.DELTA_NORM, O.COSINE_DELTA) else 2), 2, 37
    t, bits = _states(rng, m, B, T, d, bf16)
    got = P.score_hidden(ind, t.cuda()).cpu().numpy()
    for b in range(B):
        want = O.score_hidden(ind, np.ascontiguousarray(bits[:, b]), bf16=bf16)
        _close(got[b], want, ind)


def test_hidden_strided_layout_and_m0():
    """States stored token-major ([B][T][m+1][d]) and read through strides;
    the norm with m = 0 reads the only state."""
    import torch
    import paper_2608_28911_amd as P
    rng = np.random.default_rng(11)
    m, B, T, d = 3, 3, 70, 1024
    x = torch.from_numpy(rng.standard_normal((B, T, m + 1, d)).astype(np.float16))
    view = x.cuda().permute(2, 0, 1, 3)                                  # (m+1, B, T, d), strided
    for ind in (O.DELTA_NORM, O.COSINE_DELTA, O.VARIANCE):
        got = P.score_hidden(ind, view).cpu().numpy()
        for b in range(B):
            _close(got[b], O.score_hidden(ind, np.ascontiguousarray(x[b].permute(1, 0, 2).numpy())), ind)
    got = P.score_hidden("norm", view[m:]).cpu().numpy()
    for b in range(B):
        _close(got[b], O.score_hidden(O.NORM, np.ascontiguousarray(x[b, :, m:].permute(1, 0, 2).numpy())), O.NORM)


def test_hidden_rejects_bad_shapes():
    import ctypes
    import torch
    import paper_2608_28911_amd as P
    from paper_2608_28911_amd import _abi
    h = torch.zeros((2, 1, 4, 16), dtype=torch.float16, device="cuda")
    s = torch.zeros((1, 4), dtype=torch.float32, device="cuda")
    f = _abi.lib().semkv_score_hidden
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    assert f(0, p(h), 0, 0, 1, 4, 16, 64, 64, 16, p(s), None) == -1         # delta-norm needs m >= 1
    assert f(9, p(h), 0, 1, 1, 4, 16, 64, 64, 16, p(s), None) == -1         # unknown indicator
    assert f(1, p(h), 0, 1, 1, 4, 12, 64, 64, 16, p(s), None) == -1         # d not a multiple of 8
    assert f(1, p(h), 0, 1, 1, 4, 16384, 64, 64, 16, p(s), None) == -2      # d above 8192
    assert f(1, p(h), 2, 1, 1, 4, 16, 64, 64, 16, p(s), None) == -1         # unknown dtype
    with pytest.raises(P.SemKVError):
        P.score_hidden("delta_norm", h[:1])


@pytest.mark.parametrize("T", [1, 63, 200])
def test_kv_norm(T):
    import torch
    from tests import gpu_util as U
    from workloads import get_config
    cfgw = get_config(0, n_layers=3, batch=2, n_kv_heads=2, n_q_heads=8)
    cache = U.make_cache(cfgw, max(T, 64), n_layers=3, max_new=0)
    rng = np.random.default_rng(T)
    big = rng.standard_normal((3, 2, 2, T + 5, 128)).astype(np.float16)  # padded tokens: strided view
    X = torch.from_numpy(big).cuda()[:, :, :, 2:T + 2]
    got = cache.score_kv_norm(X).cpu().numpy()
    for b in range(2):
        rows = np.ascontiguousarray(big[:, b, :, 2:T + 2].reshape(6, T, 128))
        _close(got[b], O.score_kv_norm(rows), O.NORM)


def test_delta_norm_at_the_headline_shape_sampled():
    """Eq. (3) over the last 4 layers of a 4096-wide model for a 32768-token
    prompt (the grid bench.py times), checked on 96 sampled tokens."""
    import torch
    import paper_2608_28911_amd as P
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    H = torch.randn((5, 1, 32768, 4096), generator=g, device="cuda", dtype=torch.float32).half()
    got = P.score_hidden("delta_norm", H)
    idx = torch.from_numpy(np.random.default_rng(0).choice(32768, 96, replace=False)).cuda()
    sample = H[:, 0].index_select(1, idx).cpu().numpy()
    _close(got[0].index_select(0, idx).cpu().numpy(), O.score_hidden(O.DELTA_NORM, sample), O.DELTA_NORM)
