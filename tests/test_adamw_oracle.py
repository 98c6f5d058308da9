"""Pins of the AdamW oracle: closed forms of the moment averages and of the
first step, the zero-gradient case, and the library optimizer (torch's
AdamW in fp64) on the same state."""
import numpy as np
import pytest

from oracle.mathref import adamw_step
from workloads import adamw_program, adamw_worklist
from workloads.tensors import adamw_inputs

torch = pytest.importorskip("torch")

HP = dict(lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, wd=0.01)


def test_zero_gradient_only_decays():
    ai = adamw_inputs(seed=1, n=256)
    z = np.zeros(256)
    p1, m1, v1 = adamw_step(ai.p, z, z, z, t=5, **HP)
    assert np.array_equal(m1, z) and np.array_equal(v1, z)
    assert np.allclose(p1, ai.p.astype(np.float64) * (1 - HP["lr"] * HP["wd"]), rtol=1e-15, atol=0)


def test_first_step_closed_form():
    """From zero moments at t = 1 the corrected moments are g and g^2, so the
    step is lr * (g / (|g| + eps) + wd p): about lr times the sign of g."""
    ai = adamw_inputs(seed=2, n=4096)
    z = np.zeros(4096)
    g = ai.g.astype(np.float64)
    p1, _, _ = adamw_step(ai.p, g, z, z, t=1, **HP)
    p0 = ai.p.astype(np.float64)
    want = p0 - HP["lr"] * (g / (np.abs(g) + HP["eps"]) + HP["wd"] * p0)
    assert np.allclose(p1, want, rtol=1e-13, atol=1e-18)


def test_constant_gradient_moment_closed_forms():
    """With a constant gradient from zero moments, m_t = (1 - b1^t) g and
    v_t = (1 - b2^t) g^2 (sums of geometric series), so the bias-corrected
    moments stay g and g^2 at every step."""
    g = np.linspace(-0.05, 0.05, 101)
    p = np.full(101, 0.3)
    m = np.zeros(101)
    v = np.zeros(101)
    for t in range(1, 30):
        p, m, v = adamw_step(p, g, m, v, t=t, **HP)
        assert np.allclose(m, (1 - HP["b1"] ** t) * g, rtol=1e-12, atol=1e-18)
        assert np.allclose(v, (1 - HP["b2"] ** t) * g * g, rtol=1e-12, atol=1e-20)


def test_matches_library_adamw():
    """torch.optim.AdamW in fp64 from the same state one step before t."""
    ai = adamw_inputs(seed=3, n=5000)
    t = 10
    P = torch.nn.Parameter(torch.from_numpy(ai.p.astype(np.float64)).clone())
    opt = torch.optim.AdamW([P], lr=HP["lr"], betas=(HP["b1"], HP["b2"]), eps=HP["eps"], weight_decay=HP["wd"])
    P.grad = torch.from_numpy(ai.g.astype(np.float64))
    st = opt.state[P]
    st["step"] = torch.tensor(float(t - 1), dtype=torch.float64)
    st["exp_avg"] = torch.from_numpy(ai.m.astype(np.float64)).clone()
    st["exp_avg_sq"] = torch.from_numpy(ai.v.astype(np.float64)).clone()
    opt.step()
    p1, m1, v1 = adamw_step(ai.p, ai.g, ai.m, ai.v, t=t, **HP)
    # the library forms m' as m + (1 - b1)(g - m) (a lerp): equal up to fp64
    # rounding of terms of size |m|, |g| ~ 1e-2
    assert np.allclose(st["exp_avg"].numpy(), m1, rtol=1e-13, atol=1e-16)
    assert np.allclose(st["exp_avg_sq"].numpy(), v1, rtol=1e-13, atol=1e-19)
    assert np.allclose(P.detach().numpy(), p1, rtol=1e-13, atol=1e-16)


def test_adamw_worklist_covers_chunks_once():
    for n, chunk, n_wg in ((1 << 20, 1024, 256), (1000, 256, 3), (4096, 512, 20), (12, 256, 2)):
        base, tt = adamw_worklist(n, chunk, n_wg)
        n_chunks = -(-n // chunk)
        seen = np.zeros(n_chunks, np.int64)
        for w in range(n_wg):
            seen[base[w]:base[w] + int(tt.per_wg[w][1][0])] += 1
        assert np.all(seen == 1)


def test_adamw_program_offsets():
    assert sorted({k for _, _, k in adamw_program().deps}) == [0, 2]
