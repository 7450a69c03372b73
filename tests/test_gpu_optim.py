"""GPU parity of fastrl_adamw_step against the fp64 oracle on the same float32 inputs.
Bars (float32 arithmetic against float64): theta within 2.5e-7 |theta| + 1e-5 lr, m and v
within 1e-6 relative; the bfloat16 copy bit-exact against round-to-nearest-even of the
library's own float32 theta."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def fr():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_36932_amd as m
    return m


def _check(th, m, v, ref, lr, m_prev, g, b1=0.9, gs=1.0):
    """float32 rounding bounds: m = b1 m' + (1 - b1) g can cancel, so its error is bounded
    by the size of its terms, not of the result; v's terms are non-negative."""
    rt, rm, rv = ref
    th, m, v = (x.double().cpu().numpy() for x in (th, m, v))
    m_scale = b1 * np.abs(m_prev) + (1 - b1) * np.abs(g * gs)
    assert np.all(np.abs(m - rm) <= 4e-7 * m_scale + 1e-30)
    assert np.all(np.abs(v - rv) <= 1e-6 * np.abs(rv) + 1e-38)
    assert np.all(np.abs(th - rt) <= 2.5e-7 * np.abs(rt) + 1e-5 * lr)


@pytest.mark.parametrize("n", [1, 7, 4096, 1_000_003])
@pytest.mark.parametrize("hp", [dict(), dict(lr=1e-3, betas=(0.8, 0.95), eps=1e-6,
                                             weight_decay=0.1, grad_scale=0.5)])
def test_adamw_steps_match_oracle(fr, n, hp):
    rng = np.random.default_rng(n)
    th = torch.from_numpy((0.02 * rng.normal(size=n)).astype(np.float32)).to(DEV)
    m = torch.zeros(n, dtype=torch.float32, device=DEV)
    v = torch.zeros(n, dtype=torch.float32, device=DEV)
    wb = torch.empty(n, dtype=torch.bfloat16, device=DEV)
    lr = hp.get("lr", 1e-6)
    b1, b2 = hp.get("betas", (0.9, 0.999))
    for t in range(1, 4):
        g = torch.from_numpy((1e-3 * rng.normal(size=n)).astype(np.float32)).to(DEV)
        # the library takes its scalars as float32: the oracle gets the same values
        f = lambda x: float(np.float32(x))
        ref = oracle.adamw_step(th.double().cpu().numpy(), g.double().cpu().numpy(),
                                m.double().cpu().numpy(), v.double().cpu().numpy(), t,
                                lr=f(lr), beta1=f(b1), beta2=f(b2), eps=f(hp.get("eps", 1e-8)),
                                weight_decay=f(hp.get("weight_decay", 1e-2)),
                                grad_scale=f(hp.get("grad_scale", 1.0)))
        m_prev, g_host = m.double().cpu().numpy(), g.double().cpu().numpy()
        st = torch.zeros(1, dtype=torch.int32, device=DEV)
        fr.adamw_step(th, g, m, v, step=t, w_bf16=wb, status=st, **hp)
        torch.cuda.synchronize()
        assert st.item() == 0
        _check(th, m, v, ref, lr, m_prev, g_host, b1, hp.get("grad_scale", 1.0))
        assert torch.equal(wb, th.bfloat16())


def test_adamw_full_lm_head_size_sampled(fr):
    """W of the 7B shape (152064 x 3584 float32 master weights): sampled elements."""
    V, d = 152064, 3584
    n = V * d
    gen = torch.Generator(device=DEV).manual_seed(5)
    th = 0.02 * torch.randn(n, generator=gen, device=DEV)
    g = 1e-3 * torch.randn(n, generator=gen, device=DEV)
    m = 1e-4 * torch.randn(n, generator=gen, device=DEV)
    v = (1e-7 * torch.rand(n, generator=gen, device=DEV)).contiguous()
    idx = torch.from_numpy(np.random.default_rng(0).choice(n, 100_000, replace=False)).to(DEV)
    before = [x[idx].double().cpu().numpy() for x in (th, g, m, v)]
    wb = torch.empty(n, dtype=torch.bfloat16, device=DEV)
    fr.adamw_step(th, g, m, v, step=7, w_bf16=wb)
    torch.cuda.synchronize()
    f = lambda x: float(np.float32(x))
    ref = oracle.adamw_step(before[0], before[1], before[2], before[3], 7, lr=f(1e-6),
                            beta1=f(0.9), beta2=f(0.999), eps=f(1e-8), weight_decay=f(1e-2))
    _check(th[idx], m[idx], v[idx], ref, 1e-6, before[2], before[1])
    assert torch.equal(wb[idx], th[idx].bfloat16())
    del th, g, m, v, wb
    torch.cuda.empty_cache()


def test_nonfinite_gradient_flags_status(fr):
    n = 1000
    th = torch.zeros(n, device=DEV)
    g = torch.zeros(n, device=DEV)
    g[17] = float("nan")
    m, v = torch.zeros(n, device=DEV), torch.zeros(n, device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    fr.adamw_step(th, g, m, v, step=1, status=st)
    torch.cuda.synchronize()
    assert st.item() & 0x80
    assert torch.isnan(th[17]) and not torch.isnan(th[16])
