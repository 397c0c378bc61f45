"""Pins for the oracle's LAMB step (LAMB with layer-wise trust ratio, as
used by Section 3.1 and the sahajBERT-XL appendix).

* trust ratio forced to 1 and no weight decay: torch.optim.Adam (float64);
* trust ratio forced to 1 with decoupled weight decay: torch.optim.AdamW;
* closed forms at the first step from zero moments (hand-derived fixtures),
  one with weight decay on one tensor of two, so that the trust ratio's
  ||u|| includes the decay term and r != 1;
* an independent float64 numpy statement of the textbook update, within the
  fp32 rounding error;
* the trust-ratio fallback rules (zero norm, non-adaptive tensor)."""

import json
import os

import numpy as np
import pytest
import torch

import oracle

F = np.float32


def _tensors(rng, sizes):
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    return off


@pytest.mark.parametrize("wd,opt", [(0.0, "adam"), (0.01, "adamw")])
def test_unit_trust_equals_adam(wd, opt):
    rng = np.random.default_rng(11)
    sizes = [64, 1000, 8, 4096]
    off = _tensors(rng, sizes)
    P = int(off[-1])
    flags = np.full(len(sizes), 3, np.uint8)
    x0 = (rng.standard_normal(P) * 0.02).astype(F)
    lr, b1, b2, eps = 1e-3, 0.9, 0.999, 1e-6
    x, m, v = x0.copy(), np.zeros(P, F), np.zeros(P, F)
    p = torch.nn.Parameter(torch.tensor(x0, dtype=torch.float64))
    # torch receives the same fp32 hyper-parameters the oracle rounds to
    kw = dict(lr=float(F(lr)), betas=(float(F(b1)), float(F(b2))), eps=float(F(eps)))
    o = (torch.optim.Adam([p], weight_decay=0.0, **kw) if opt == "adam"
         else torch.optim.AdamW([p], weight_decay=float(F(wd)), **kw))
    for step in range(1, 4):
        g = (rng.standard_normal(P) * 1e-3).astype(F)
        cfg = oracle.lamb_cfg(lr, b1, b2, eps, wd, step=step, force_unit_trust=True)
        x, m, v, trust = oracle.lamb(x, m, v, g, off, flags, cfg)
        assert np.all(trust == 1)
        p.grad = torch.tensor(g, dtype=torch.float64)
        o.step()
    ref = p.detach().numpy()
    disp = np.max(np.abs(ref - x0))
    assert np.max(np.abs(x - ref)) <= 1e-5 * disp + 2 * np.max(np.spacing(np.abs(x0)))
    st = o.state[p]
    mr, vr = st["exp_avg"].numpy(), st["exp_avg_sq"].numpy()
    # moments: a few fp32 roundings per step, relative to their magnitude
    assert np.max(np.abs(m - mr)) <= 1e-6 * np.max(np.abs(mr))
    assert np.max(np.abs(v - vr)) <= 1e-6 * np.max(np.abs(vr))


def test_golden_closed_forms(golden_dir):
    d = json.load(open(os.path.join(golden_dir, "lamb_examples.json")))
    for c in d["cases"]:
        n = len(c["x"])
        off = np.array(c.get("offsets", [0, n]), np.uint64)
        flags = np.array(c.get("flags", [3]), np.uint8)
        cfg = oracle.lamb_cfg(c["lr"], c["beta1"], c["beta2"], c["eps"],
                              c["weight_decay"], step=c["step"])
        x, m, v, trust = oracle.lamb(np.array(c["x"], F), np.array(c["m"], F),
                                     np.array(c["v"], F), np.array(c["g"], F), off, flags, cfg)
        assert np.allclose(x, c["x_new"], rtol=0, atol=c["atol_x"]), c["derivation"]
        assert np.allclose(m, c["m_new"], rtol=c["rtol_moments"], atol=0)
        assert np.allclose(v, c["v_new"], rtol=c["rtol_moments"], atol=0)
        assert np.allclose(trust, np.atleast_1d(c["trust"]), rtol=c["rtol_trust"], atol=0), c["derivation"]


def lamb64(x, m, v, g, off, flags, lr, b1, b2, eps, wd, t, unit=False):
    """Textbook LAMB in float64 (independent of the C oracle)."""
    b1, b2, lr, eps, wd = (float(F(a)) for a in (b1, b2, lr, eps, wd))
    x, m, v, g = (a.astype(np.float64) for a in (x, m, v, g))
    m2 = b1 * m + (1 - b1) * g
    v2 = b2 * v + (1 - b2) * g * g
    u = (m2 / (1 - b1 ** t)) / (np.sqrt(v2 / (1 - b2 ** t)) + eps)
    xn = x.copy()
    rs = []
    for k in range(len(flags)):
        s = slice(int(off[k]), int(off[k + 1]))
        uk = u[s] + (wd if flags[k] & 1 else 0.0) * x[s]
        X, U = np.linalg.norm(x[s]), np.linalg.norm(uk)
        r = X / U if (flags[k] & 2 and X > 0 and U > 0 and not unit) else 1.0
        rs.append(r)
        xn[s] = x[s] - lr * r * uk
    return xn, m2, v2, np.array(rs)


@pytest.mark.parametrize("step", [1, 2, 10, 1000])
def test_against_float64_textbook(step):
    rng = np.random.default_rng(step)
    sizes = [8, 128, 128, 5000, 4096, 64]
    off = _tensors(rng, sizes)
    P = int(off[-1])
    flags = np.array([3, 2, 2, 3, 1, 0], np.uint8)
    x = (rng.standard_normal(P) * 0.02).astype(F)
    x[int(off[1]):int(off[2])] = 1.0
    x[int(off[2]):int(off[3])] = 0.0          # zero tensor: trust ratio 1
    m = (rng.standard_normal(P) * 1e-4).astype(F)
    v = ((rng.standard_normal(P) * 1e-3) ** 2).astype(F)
    g = (rng.standard_normal(P) * 1e-3).astype(F)
    args = (1e-3, 0.9, 0.999, 1e-6, 0.01)
    cfg = oracle.lamb_cfg(*args, step=step)
    xo, mo, vo, tr = oracle.lamb(x, m, v, g, off, flags, cfg)
    xr, mr, vr, rr = lamb64(x, m, v, g, off, flags, *args, step)
    assert np.max(np.abs(mo - mr)) <= 1e-6 * np.max(np.abs(mr))
    assert np.max(np.abs(vo - vr)) <= 1e-6 * np.max(np.abs(vr))
    assert np.allclose(tr, rr, rtol=1e-5, atol=0)
    assert tr[2] == 1.0 and tr[4] == 1.0 and tr[5] == 1.0   # zero x, non-adaptive
    dx_o = xo.astype(np.float64) - x
    dx_r = xr - x
    assert np.max(np.abs(dx_o - dx_r)) <= 1e-5 * np.max(np.abs(dx_r)) + 2 * np.max(np.spacing(np.abs(x)))


def test_zero_update_direction_keeps_ratio_one():
    # g = m = 0 and no decay: u = 0, so ||u|| = 0 and r falls back to 1; x is unchanged
    P = 256
    x = np.linspace(-1, 1, P).astype(F)
    cfg = oracle.lamb_cfg(1e-2, 0.9, 0.999, 1e-6, 0.0, step=3)
    xo, mo, vo, tr = oracle.lamb(x, np.zeros(P, F), np.full(P, 1e-6, F), np.zeros(P, F),
                                 np.array([0, P], np.uint64), np.array([3], np.uint8), cfg)
    assert tr[0] == 1.0 and np.array_equal(xo, x)


def test_lamb_rejects_bad_table():
    cfg = oracle.lamb_cfg(step=1)
    z = np.zeros(16, F)
    for off in ([0, 8, 15], [1, 16], [0, 9, 8, 16]):
        with pytest.raises(oracle.OracleError):
            oracle.lamb(z, z, z, z, np.array(off, np.uint64), np.full(len(off) - 1, 3, np.uint8), cfg)
    with pytest.raises(oracle.OracleError):
        oracle.lamb(z, z, z, z, np.array([0, 16], np.uint64), np.array([3], np.uint8),
                    oracle.lamb_cfg(step=0))
