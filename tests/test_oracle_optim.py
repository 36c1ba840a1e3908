"""Pins for the oracle's optimizer steps.

* AdamW with FP32 states against torch.optim.AdamW (an independent
  implementation; the paper aligns its reference path to PyTorch AdamW).
* Adafactor with FP32 states against Hugging Face's Adafactor (same options
  the paper's reference path uses), plus the rank-1 closed form.
* CAME: the official implementation is not available here, so the CAME oracle
  is pinned by closed forms (beta1 = 0; a uniform gradient; a rank-1
  gradient; 20 steps with beta1 = 0.9 for constant gradients and sign flips),
  by its second-moment path against the (HF-pinned) Adafactor oracle at t = 1,
  and, for gradients of varying magnitude over 20 steps, by the symmetries its
  definition implies (row / column permutation, negation, scaling by 2,
  transposition).
* Dormant entries (exact zeros) keep code 0 and a pure weight-decay
  trajectory, as the exact-zero invariant (section 4.2) implies.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import AL8, AL16, FP32, UF8, State
from paper_2608_22322_amd import synth


def _grads(rows, cols, steps, seed, sigma=1e-3, zero_frac=0.0):
    out = []
    for t in range(1, steps + 1):
        g = synth.normal_f32(synth.grad_key(seed, t), rows * cols, sigma,
                             synth.mask_key(seed), zero_frac)
        out.append(g)
    return out


def _param(n, seed, sigma=0.02):
    return synth.normal_f32(synth.param_key(seed), n, sigma)


# ----------------------------------------------------------------------- AdamW
@pytest.mark.parametrize("shape", [(64, 96), (1, 1000)])
def test_adamw_fp32_matches_torch(shape):
    rows, cols = shape
    n = rows * cols
    steps = 100
    p0 = _param(n, 1)
    grads = _grads(rows, cols, steps, 2, zero_frac=0.05)
    cfg = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, wd=0.01)

    p = p0.copy()
    m, v = State(FP32, n), State(FP32, n)
    for t, g in enumerate(grads, 1):
        oracle.adamw_step(p, g, m, v, t, **cfg)

    tp = torch.nn.Parameter(torch.from_numpy(p0.copy()))
    opt = torch.optim.AdamW([tp], lr=cfg["lr"], betas=(cfg["beta1"], cfg["beta2"]), eps=cfg["eps"],
                            weight_decay=cfg["wd"], foreach=False)
    for g in grads:
        tp.grad = torch.from_numpy(g.copy())
        opt.step()
    ref = tp.detach().numpy()
    assert np.abs(p - ref).max() <= 1e-5 * 0.2  # the paper's alignment tolerance is 1e-5
    assert np.linalg.norm(p - ref) / np.linalg.norm(ref) < 2e-6
    st = opt.state[tp]
    np.testing.assert_allclose(m.codes, st["exp_avg"].numpy(), rtol=1e-4, atol=1e-10)
    np.testing.assert_allclose(v.codes, st["exp_avg_sq"].numpy(), rtol=1e-4, atol=1e-16)


def test_adamw_dormant_entries():
    """Exact-zero gradients from a zero state: codes stay 0 and p follows (1 - lr wd)^t."""
    rows, cols = 16, 256
    n = rows * cols
    p0 = _param(n, 3)
    mk = synth.mask_key(4)
    mask = synth.normal_f32(synth.grad_key(4, 1), n, 1e-3, mk, 0.05) == 0
    p = p0.copy()
    m = State(UF8, n, 256)
    v = State(AL8, n, 256, float(np.float32(2 * math.log2(1e-8))))
    lr, wd = 1e-3, 0.01
    for t in range(1, 8):
        g = synth.normal_f32(synth.grad_key(4, t), n, 1e-3)
        if t <= 5:
            g[mask] = 0.0
        oracle.adamw_step(p, g, m, v, t, lr=lr, wd=wd)
        if t <= 5:
            assert np.all(m.codes[mask] == 0) and np.all(v.codes[mask] == 0)
            want = p0[mask].astype(np.float64) * (1 - lr * wd) ** t
            np.testing.assert_allclose(p[mask], want, rtol=4e-7 * t, atol=0)
            assert np.all(v.codes[~mask] > 0)
        else:
            assert np.all(v.codes > 0)


def test_adamw_first_live_step_from_zero_state():
    """An entry whose gradient was exactly zero so far has decoded state exactly 0, so on its first
    nonzero gradient the moments reduce to m = fl32((1 - beta1) g), v = fl32((1 - beta2) g^2)."""
    n = 4096
    p = _param(n, 31)
    m, v = State(FP32, n), State(FP32, n)
    b1, b2 = 0.9, 0.999
    zero = np.zeros(n, np.float32)
    for t in (1, 2, 3):
        oracle.adamw_step(p, zero, m, v, t, beta1=b1, beta2=b2)
        assert not m.codes.any() and not v.codes.any()
    g = synth.normal_f32(synth.grad_key(31, 4), n, 1e-3)
    oracle.adamw_step(p, g, m, v, 4, beta1=b1, beta2=b2)
    g64 = g.astype(np.float64)
    assert np.array_equal(m.codes, ((1.0 - b1) * g64).astype(np.float32))
    assert np.array_equal(v.codes, ((1.0 - b2) * (g64 * g64)).astype(np.float32))


def test_adamw_quantized_close_to_fp32():
    """AL8 second moment + UF8 momentum stays close to the FP32 trajectory (qualitative)."""
    n = 256 * 64
    p0 = _param(n, 5)
    grads = _grads(64, 256, 50, 6)
    pf, pq = p0.copy(), p0.copy()
    mf, vf = State(FP32, n), State(FP32, n)
    mq, vq = State(UF8, n, 256), State(AL8, n, 256, float(np.float32(2 * math.log2(1e-8))))
    for t, g in enumerate(grads, 1):
        oracle.adamw_step(pf, g, mf, vf, t)
        oracle.adamw_step(pq, g, mq, vq, t)
    rel = np.linalg.norm(pq - pf) / np.linalg.norm(pf - p0)
    assert rel < 0.02, rel


# ------------------------------------------------------------------- Adafactor
def _hf_adafactor(p0, rows, cols, grads, lr=1e-3):
    from transformers.optimization import Adafactor

    shape = (rows, cols) if rows > 1 else (cols,)
    tp = torch.nn.Parameter(torch.from_numpy(p0.copy().reshape(shape)))
    opt = Adafactor([tp], lr=lr, eps=(1e-30, 1e-3), clip_threshold=1.0, decay_rate=-0.8, beta1=None,
                    weight_decay=0.0, scale_parameter=False, relative_step=False, warmup_init=False)
    for g in grads:
        tp.grad = torch.from_numpy(g.copy().reshape(shape))
        opt.step()
    return tp.detach().numpy().reshape(-1), opt.state[tp]


@pytest.mark.parametrize("shape", [(48, 80), (1, 777)])
def test_adafactor_fp32_matches_hf(shape):
    rows, cols = shape
    n = rows * cols
    steps = 60
    p0 = _param(n, 7)
    grads = _grads(rows, cols, steps, 8, zero_frac=0.02)
    p = p0.copy()
    if rows > 1:
        vr, vc, v = State(FP32, rows), State(FP32, cols), None
    else:
        vr, vc, v = None, None, State(FP32, n)
    for t, g in enumerate(grads, 1):
        oracle.adafactor_step(p, g, rows, cols, vr, vc, v, t)
    ref, st = _hf_adafactor(p0, rows, cols, grads)
    assert np.abs(p - ref).max() <= 2e-6
    assert np.linalg.norm(p - ref) / np.linalg.norm(ref) < 2e-6
    if rows > 1:
        np.testing.assert_allclose(vr.codes, st["exp_avg_sq_row"].numpy(), rtol=2e-6)
        np.testing.assert_allclose(vc.codes, st["exp_avg_sq_col"].numpy(), rtol=2e-6)
    else:
        np.testing.assert_allclose(v.codes, st["exp_avg_sq"].numpy(), rtol=2e-6)


def test_adafactor_first_step_factors_are_exact_means():
    """At t = 1 the decay 1 - t^-0.8 is 0, so R and C are the exactly rounded row and column means of
    g^2 + eps1 (reference sums by math.fsum; a transposed reduction fails on a non-square matrix)."""
    rows, cols = 12, 37
    g = _grads(rows, cols, 1, 33, zero_frac=0.05)[0]
    p = _param(rows * cols, 34)
    vr, vc = State(FP32, rows), State(FP32, cols)
    oracle.adafactor_step(p, g, rows, cols, vr, vc, None, 1, lr=1e-3, eps1=1e-30)
    g2 = g.astype(np.float64).reshape(rows, cols) ** 2 + 1e-30
    want_r = np.array([math.fsum(g2[i]) / cols for i in range(rows)]).astype(np.float32)
    want_c = np.array([math.fsum(g2[:, j]) / rows for j in range(cols)]).astype(np.float32)
    assert np.array_equal(vr.codes, want_r)
    assert np.array_equal(vc.codes, want_c)


def test_adafactor_rank1_closed_form():
    """g_ij = a_i b_j: the factored estimate is exact, so at t = 1 the clipped update is sign(g)."""
    rng = np.random.default_rng(21)
    rows, cols = 24, 40
    # power-of-two factors keep |g| = a_i b_j exact in fp32
    a = np.exp2(rng.integers(-12, -8, rows)).astype(np.float64)
    b = np.exp2(rng.integers(-2, 2, cols)).astype(np.float64)
    sgn = np.where(rng.random(rows * cols) < 0.5, -1.0, 1.0)
    g = (np.outer(a, b).reshape(-1) * sgn).astype(np.float32)
    p0 = _param(rows * cols, 9)
    for codec in (FP32, AL16):
        p = p0.copy()
        oracle.adafactor_step(p, g, rows, cols, State(codec, rows, 128, -99.66), State(codec, cols, 128, -99.66),
                              None, 1, lr=1e-3)
        upd = (p0.astype(np.float64) - p) / 1e-3
        tol = 1e-4 if codec == FP32 else 3e-4
        np.testing.assert_allclose(upd, sgn, rtol=tol, atol=tol)


# ------------------------------------------------------------------------ CAME
def _came_states(rows, cols, codec=FP32, mcodec=FP32):
    n = rows * cols
    if rows > 1:
        return dict(m=State(mcodec, n, 256), vr=State(codec, rows, 128, -99.66), vc=State(codec, cols, 128, -99.66),
                    v=None, cr=State(codec, rows, 128, -53.15), cc=State(codec, cols, 128, -53.15))
    return dict(m=State(mcodec, n, 256), vr=None, vc=None, v=State(codec, n, 128, -99.66), cr=None, cc=None)


def test_came_beta1_zero_closed_form():
    """beta1 = 0: m = clipped update, residual == eps2, so from zero confidence
    R'_t = C'_t = (1 - beta3^t) eps2 and p -= lr * uhat / sqrt((1 - beta3^t) eps2). With beta2 = 0 the clipped
    update uhat is Hugging Face Adafactor's at decay_rate 0 (beta2_t = 1 - t^0 = 0, the factors of the
    current gradient only), so every step is held to that independent implementation."""
    from transformers.optimization import Adafactor

    rows, cols = 20, 36
    n = rows * cols
    p0 = _param(n, 11)
    grads = _grads(rows, cols, 5, 12)
    st = _came_states(rows, cols)
    beta3, eps2 = 0.9999, 1e-16
    lr = 1e-13  # the confidence scale 1/sqrt((1 - beta3^t) eps2) is about 1e10 / sqrt(t)
    p = p0.copy()
    tp = torch.nn.Parameter(torch.from_numpy(p0.copy().reshape(rows, cols)))
    hf = Adafactor([tp], lr=1e-3, eps=(1e-30, 1e-3), clip_threshold=1.0, decay_rate=0.0, beta1=None,
                   weight_decay=0.0, scale_parameter=False, relative_step=False, warmup_init=False)
    for t, g in enumerate(grads, 1):
        before = p.copy()
        oracle.came_step(p, g, rows, cols, t=t, beta1=0.0, beta2=0.0, lr=lr, beta3=beta3, eps2=eps2, **st)
        c_expect = (1 - beta3**t) * eps2
        np.testing.assert_allclose(st["cr"].codes, np.float32(c_expect), rtol=1e-6)
        np.testing.assert_allclose(st["cc"].codes, np.float32(c_expect), rtol=1e-6)
        upd = (before.astype(np.float64) - p) / lr * math.sqrt(c_expect)
        hp = tp.detach().numpy().reshape(-1).astype(np.float64).copy()
        tp.grad = torch.from_numpy(g.copy().reshape(rows, cols))
        hf.step()
        ref = (hp - tp.detach().numpy().reshape(-1)) / 1e-3  # HF's clipped update of this step
        # both updates are read back through an fp32 parameter: ~1e-6 relative of p per read
        tol = 4 * float(np.spacing(np.float32(np.abs(p0).max()))) / 1e-3
        np.testing.assert_allclose(upd, ref, rtol=1e-4, atol=tol)
        assert np.abs(ref).max() > 0.1


def test_came_uniform_gradient_closed_form():
    """Uniform g = c: uhat = sign(c); m = (1-beta1) sign(c); residual beta1^2 + eps2 everywhere;
    p -= lr (1-beta1) sign(c) / sqrt((1-beta3)(beta1^2 + eps2))."""
    for rows, cols in ((16, 32), (1, 300)):
        n = rows * cols
        p0 = _param(n, 13)
        c = np.float32(-3e-4)
        g = np.full(n, c, np.float32)
        st = _came_states(rows, cols)
        p = p0.copy()
        b1, b3, e2, lr = 0.9, 0.9999, 1e-16, 1e-4
        oracle.came_step(p, g, rows, cols, t=1, beta1=b1, beta3=b3, eps2=e2, lr=lr, **st)
        if rows > 1:
            want = lr * (1 - b1) * -1.0 / math.sqrt((1 - b3) * (b1 * b1 + e2))
        else:
            want = lr * (1 - b1) * -1.0  # 1-D tensors: update = momentum, no confidence
        # p is fp32: the observed step carries one rounding of p
        ulp_p = float(np.spacing(np.abs(p0)).max())
        np.testing.assert_allclose(p0.astype(np.float64) - p, want, rtol=1e-5, atol=ulp_p)


def test_came_rank1_closed_form():
    rng = np.random.default_rng(23)
    rows, cols = 12, 20
    a = np.exp2(rng.integers(-12, -8, rows)).astype(np.float64)
    b = np.exp2(rng.integers(-2, 2, cols)).astype(np.float64)
    sgn = np.where(rng.random(rows * cols) < 0.5, -1.0, 1.0)
    g = (np.outer(a, b).reshape(-1) * sgn).astype(np.float32)
    p0 = _param(rows * cols, 15)
    st = _came_states(rows, cols)
    p = p0.copy()
    b1, b3, e2, lr = 0.9, 0.9999, 1e-16, 1e-4
    oracle.came_step(p, g, rows, cols, t=1, beta1=b1, beta3=b3, eps2=e2, lr=lr, **st)
    want = lr * (1 - b1) * sgn / math.sqrt((1 - b3) * (b1 * b1 + e2))
    np.testing.assert_allclose(p0.astype(np.float64) - p, want, rtol=1e-4)


def test_came_second_moment_path_matches_adafactor_at_t1():
    """With beta2 = 0 CAME's factored V equals Adafactor's at t = 1 (beta2_t = 0); with beta1 = 0 its
    update is that clipped update scaled by 1/sqrt((1 - beta3) eps2)."""
    for rows, cols in ((30, 44), (1, 500)):
        n = rows * cols
        p0 = _param(n, 17)
        g = _grads(rows, cols, 1, 18, zero_frac=0.02)[0]
        pa = p0.copy()
        fac = rows > 1
        oracle.adafactor_step(pa, g, rows, cols, State(FP32, rows) if fac else None,
                              State(FP32, cols) if fac else None, None if fac else State(FP32, n), 1, lr=1e-3)
        ua = (p0.astype(np.float64) - pa) / 1e-3
        st = _came_states(rows, cols)
        pc = p0.copy()
        oracle.came_step(pc, g, rows, cols, t=1, beta1=0.0, beta2=0.0, lr=1e-4, **st)
        uc = (p0.astype(np.float64) - pc) / 1e-4
        scale = math.sqrt((1 - 0.9999) * 1e-16) if fac else 1.0
        np.testing.assert_allclose(uc * scale, ua, rtol=5e-3, atol=5e-3 * np.abs(ua).max())


# ----------------------------------------------- CAME over many steps with beta1 > 0 (closed forms)
# A constant gradient g_ij = s_ij a_i b_j (|s| = 1; a uniform gradient is a = b = const) makes every
# factored estimate exact: R_t = (1 - beta2^t) a_i^2 mean(b^2), C_t = (1 - beta2^t) b_j^2 mean(a^2) (plus
# eps1), so u = g / sqrt(R_i C_j / mean R) = s / sqrt(1 - beta2^t), whose RMS exceeds the clip threshold
# 1 for every finite t: the clipped update is exactly s. Then m_t is the EMA of s from zero, the residual
# (s - m_t)^2 + eps2 is the same for every element, the confidence factors are uniform, and
# p_t = p_{t-1} - lr m_t / sqrt(R'_t) with R'_t = (1 - beta3) sum_k beta3^(t-k) (r_k + eps2).
# A sign change of the gradient at step k (s -> -s) keeps all of this (r_k then grows), and probes the
# momentum carried across steps, including through its UF8 code.

def _came_closed_form(signs_t, b1, b2, b3, e2, lr):
    """(m_t, R'_t, p-update_t) per step for the clipped update signs_t[t-1] * s (uniform per step)."""
    T = len(signs_t)
    m = []
    for t in range(1, T + 1):
        # m_t = (1 - b1) sum_{j<=t} b1^(t-j) sigma_j
        m.append(sum((1 - b1) * b1 ** (t - j) * signs_t[j - 1] for j in range(1, t + 1)))
    r = [(signs_t[t - 1] - m[t - 1]) ** 2 for t in range(1, T + 1)]
    R = [sum((1 - b3) * b3 ** (t - k) * (r[k - 1] + e2) for k in range(1, t + 1)) for t in range(1, T + 1)]
    upd = [lr * m[t] / math.sqrt(R[t]) for t in range(T)]
    return m, R, upd


@pytest.mark.parametrize("kind", ["uniform", "rank1", "flip", "row1"])
@pytest.mark.parametrize("codecs", ["fp32", "uf8_al16"])
def test_came_multistep_closed_form(kind, codecs):
    """20 CAME steps with beta1 = 0.9 > 0 against the closed form above: momentum, confidence factors and the
    parameter trajectory, with FP32 states and with UF8 momentum + AL16 factors (a block of equal values is
    coded exactly by UF8, and by AL16 up to the fp32 rounding of its l_min: ~1e-6 relative per decode)."""
    rng = np.random.default_rng(41)
    rows, cols, T, k_flip = (1, 300, 20, 0) if kind == "row1" else (16, 48, 20, 8 if kind == "flip" else 0)
    n = rows * cols
    if kind == "rank1":
        a = np.exp2(rng.integers(-12, -8, rows)).astype(np.float64)
        b = np.exp2(rng.integers(-2, 2, cols)).astype(np.float64)
        s = np.where(rng.random(n) < 0.5, -1.0, 1.0)
        mag = np.outer(a, b).reshape(-1)
    else:
        s = np.full(n, -1.0)
        mag = np.full(n, 3e-4)
    b1, b2, b3, e2, lr = 0.9, 0.999, 0.9999, 1e-16, 1e-4
    sig = [(-1.0 if (k_flip and t >= k_flip) else 1.0) for t in range(1, T + 1)]
    m_cf, R_cf, upd_cf = _came_closed_form(sig, b1, b2, b3, e2, lr)
    if kind == "row1":  # 1-D semantics (rows == 1): update = lr m_t, no confidence factors
        upd_cf = [lr * x for x in m_cf]
    mc, fc = (FP32, FP32) if codecs == "fp32" else (UF8, AL16)
    st = _came_states(rows, cols, codec=fc, mcodec=mc)
    p0 = _param(n, 43)
    p = p0.copy()
    total = np.zeros(n)
    tol = 2e-6 if codecs == "fp32" else 5e-5
    for t in range(1, T + 1):
        g = (mag * s * sig[t - 1]).astype(np.float32)
        before = p.copy()
        oracle.came_step(p, g, rows, cols, t=t, beta1=b1, beta2=b2, beta3=b3, eps2=e2, lr=lr, **st)
        step_upd = before.astype(np.float64) - p
        total += step_upd
        # momentum: m_t s in every element
        m_dec = st["m"].decode() if mc == UF8 else st["m"].codes[:n]
        # m is rounded to fp32 every step (|m| <= 1): its absolute error grows by at most an ulp of 1 per step,
        # which matters where the flipped momentum crosses zero
        m_atol = t * 2.0**-23
        np.testing.assert_allclose(m_dec, m_cf[t - 1] * s, rtol=tol, atol=m_atol, err_msg=f"m at t={t}")
        if mc == UF8:
            assert np.all(np.abs(st["m"].codes[:n]) == 127), t
        if rows > 1:
            for key in ("cr", "cc"):
                dec = st[key].decode() if fc == AL16 else st[key].codes
                np.testing.assert_allclose(dec, R_cf[t - 1], rtol=tol * t, err_msg=f"{key} at t={t}")
        # per-step update, read back through an fp32 parameter (one rounding of |p| <= 0.1)
        ulp = float(np.spacing(np.float32(np.abs(p0).max() + 0.1)))
        u_atol = 2 * ulp + (lr * m_atol / math.sqrt(R_cf[t - 1]) if rows > 1 else lr * m_atol)
        np.testing.assert_allclose(step_upd, upd_cf[t - 1] * s, rtol=tol * t, atol=u_atol,
                                   err_msg=f"update at t={t}")
    np.testing.assert_allclose(total, sum(upd_cf) * s, rtol=tol * T, atol=T * u_atol)
    if kind == "flip":
        # the momentum has turned: m_T s = -(1 - b1^(T-k+1)) + b1^(T-k+1) m_{k-1} < 0
        assert m_cf[-1] < 0 < m_cf[k_flip - 2]


def test_came_staggered_sign_flips_closed_form():
    """Rank-1 magnitudes a_i b_j with per-element signs that flip at element-specific steps k_ij: the second
    moment and the clip stay exact (|g| does not change, so uhat = the current sign), but the momentum,
    the residual and therefore the confidence factors R'_i, C'_j now differ by row and by column. Their
    values follow from the definitions: m = EMA(beta1) of the signs, residual (sign - m)^2 + eps2, R' / C' =
    EMA(beta3) of its row / column means, update lr m / sqrt(R'_i C'_j / mean R'). A transposed or
    misindexed confidence factor, a residual taken against the previous momentum, or a clip applied after
    the momentum each fail it. FP32 states, 20 steps."""
    rng = np.random.default_rng(47)
    rows, cols, T = 16, 48, 20
    b1, b2, b3, e2, lr = 0.9, 0.999, 0.9999, 1e-16, 1e-4
    a = np.exp2(rng.integers(-12, -8, rows)).astype(np.float64)
    b = np.exp2(rng.integers(-2, 2, cols)).astype(np.float64)
    s0 = np.where(rng.random((rows, cols)) < 0.5, -1.0, 1.0)
    k = rng.integers(2, 14, (rows, cols))  # the step from which element (i, j) has the opposite sign
    sig = np.stack([np.where(t >= k, -s0, s0) for t in range(1, T + 1)])  # [T, rows, cols]
    m = np.zeros((T, rows, cols))
    for t in range(T):  # m_t = (1 - b1) sum_{l <= t} b1^(t - l) sigma_l
        m[t] = sum((1 - b1) * b1 ** (t - l) * sig[l] for l in range(t + 1))
    r = (sig - m) ** 2 + e2
    Rp = np.stack([sum((1 - b3) * b3 ** (t - l) * r[l].mean(axis=1) for l in range(t + 1)) for t in range(T)])
    Cp = np.stack([sum((1 - b3) * b3 ** (t - l) * r[l].mean(axis=0) for l in range(t + 1)) for t in range(T)])
    assert np.ptp(Rp[-1]) > 1e-3 * Rp[-1].mean() and np.ptp(Cp[-1]) > 1e-3 * Cp[-1].mean()  # not uniform
    st = _came_states(rows, cols)
    p0 = _param(rows * cols, 49)
    p = p0.copy()
    mag = np.outer(a, b)
    for t in range(1, T + 1):
        g = (mag * sig[t - 1]).reshape(-1).astype(np.float32)
        before = p.copy()
        oracle.came_step(p, g, rows, cols, t=t, beta1=b1, beta2=b2, beta3=b3, eps2=e2, lr=lr, **st)
        tol = 2e-6 * t
        np.testing.assert_allclose(st["m"].codes[: rows * cols], m[t - 1].reshape(-1), rtol=tol, atol=t * 2.0**-23)
        np.testing.assert_allclose(st["cr"].codes, Rp[t - 1], rtol=tol, err_msg=f"R' at t={t}")
        np.testing.assert_allclose(st["cc"].codes, Cp[t - 1], rtol=tol, err_msg=f"C' at t={t}")
        S = np.outer(Rp[t - 1], Cp[t - 1]) / Rp[t - 1].mean()
        want = lr * m[t - 1] / np.sqrt(S)
        ulp = float(np.spacing(np.float32(np.abs(p0).max() + 0.1)))
        atol = 2 * ulp + lr * t * 2.0**-23 / np.sqrt(S.min())
        np.testing.assert_allclose(before.astype(np.float64) - p, want.reshape(-1), rtol=tol, atol=atol,
                                   err_msg=f"update at t={t}")


# -------------------------------------- CAME over many steps: symmetries that hold for any gradient
# Constant gradients give closed forms; for gradients that vary in magnitude from step to step the step
# is pinned by what the method's definition implies for every input. With FP32 states and exact sums,
# the step commutes with permuting rows or columns (the factors, the means, the clip's RMS and the
# confidence are sums over rows / columns) and with negating the gradient (uhat, m and the update change
# sign; V, the residual and the confidence do not), bit for bit; scaling the gradient by 2 (eps1 = 0)
# leaves uhat, m, the confidence and the update unchanged and scales V by exactly 4; transposing the
# gradient swaps the roles of rows and columns (equal up to the fp32 roundings of the factor means). A
# factor indexed by the wrong side, a residual against the previous momentum, a missing normalisation or
# a sign slip breaks one of them.

def _came_run(g_steps, rows, cols, p0, **kw):
    st = _came_states(rows, cols, codec=FP32, mcodec=FP32)
    p = p0.copy()
    for t, g in enumerate(g_steps, 1):
        oracle.came_step(p, g, rows, cols, t=t, **kw, **st)
    return p, st


def _varying_grads(rows, cols, T, seed):
    """Gradients whose row and column scales change from step to step (so the factors, the clip and the
    confidence are far from uniform), with exact zeros."""
    rng = np.random.default_rng(seed)
    out = []
    for t in range(1, T + 1):
        a = np.exp2(rng.uniform(-3, 3, rows))[:, None]
        b = np.exp2(rng.uniform(-3, 3, cols))[None, :]
        g = (rng.standard_normal((rows, cols)) * a * b * 1e-3).astype(np.float32)
        g[rng.random((rows, cols)) < 0.03] = 0.0
        out.append(g)
    return out


def test_came_multistep_permutation_equivariance():
    rows, cols, T = 24, 40, 20
    rng = np.random.default_rng(51)
    gs = _varying_grads(rows, cols, T, 52)
    p0 = _param(rows * cols, 53).reshape(rows, cols)
    pr, pc = rng.permutation(rows), rng.permutation(cols)
    kw = dict(beta1=0.9, lr=1e-4)
    p, st = _came_run([g.ravel() for g in gs], rows, cols, p0.ravel(), **kw)
    q, sq = _came_run([np.ascontiguousarray(g[pr][:, pc]).ravel() for g in gs], rows, cols,
                      np.ascontiguousarray(p0[pr][:, pc]).ravel(), **kw)
    assert np.array_equal(p.reshape(rows, cols)[pr][:, pc], q.reshape(rows, cols))
    assert np.array_equal(st["m"].codes.reshape(rows, cols)[pr][:, pc], sq["m"].codes.reshape(rows, cols))
    for key, perm in (("vr", pr), ("cr", pr), ("vc", pc), ("cc", pc)):
        assert np.array_equal(st[key].codes[perm], sq[key].codes), key
    # the factors are far from uniform: the test sees the indexing
    assert np.ptp(st["cr"].codes) > 0.1 * st["cr"].codes.mean() and np.ptp(st["vc"].codes) > st["vc"].codes.mean()


def test_came_multistep_sign_equivariance():
    rows, cols, T = 24, 40, 20
    gs = _varying_grads(rows, cols, T, 54)
    zero = np.zeros(rows * cols, np.float32)
    kw = dict(beta1=0.9, lr=1e-4)
    p, st = _came_run([g.ravel() for g in gs], rows, cols, zero, **kw)
    q, sq = _came_run([(-g).ravel() for g in gs], rows, cols, zero, **kw)
    assert np.array_equal(q, -p) and np.abs(p).max() > 0
    assert np.array_equal(sq["m"].codes, -st["m"].codes)
    for key in ("vr", "vc", "cr", "cc"):
        assert np.array_equal(st[key].codes, sq[key].codes), key


def test_came_multistep_scale_invariance():
    rows, cols, T = 24, 40, 20
    gs = _varying_grads(rows, cols, T, 55)
    for g in gs:  # eps1 = 0: a zero row or column would divide by zero
        g[g == 0] = np.float32(1e-4)
    p0 = _param(rows * cols, 56)
    kw = dict(beta1=0.9, lr=1e-4, eps1=0.0)
    p, st = _came_run([g.ravel() for g in gs], rows, cols, p0, **kw)
    q, sq = _came_run([(2 * g).ravel() for g in gs], rows, cols, p0, **kw)
    assert np.array_equal(p, q) and np.array_equal(st["m"].codes, sq["m"].codes)
    for key in ("cr", "cc"):
        assert np.array_equal(st[key].codes, sq[key].codes), key
    for key in ("vr", "vc"):
        assert np.array_equal(4 * st[key].codes, sq[key].codes), key


def test_came_multistep_transposition():
    rows, cols, T = 24, 40, 20
    gs = _varying_grads(rows, cols, T, 57)
    p0 = _param(rows * cols, 58).reshape(rows, cols)
    kw = dict(beta1=0.9, lr=1e-4)
    p, st = _came_run([g.ravel() for g in gs], rows, cols, p0.ravel(), **kw)
    q, sq = _came_run([np.ascontiguousarray(g.T).ravel() for g in gs], cols, rows,
                      np.ascontiguousarray(p0.T).ravel(), **kw)
    # V and the confidence of one side are the other's, up to fp32 roundings propagated over 20 steps
    for a, b in (("vr", "vc"), ("cr", "cc"), ("vc", "vr"), ("cc", "cr")):
        np.testing.assert_allclose(st[a].codes, sq[b].codes, rtol=1e-5, err_msg=a)
    np.testing.assert_allclose(st["m"].codes.reshape(rows, cols), sq["m"].codes.reshape(cols, rows).T,
                               rtol=1e-4, atol=1e-6)
    upd_p = p0.astype(np.float64) - p.reshape(rows, cols)
    upd_q = p0.astype(np.float64) - q.reshape(cols, rows).T
    np.testing.assert_allclose(upd_q, upd_p, rtol=1e-3, atol=1e-3 * np.abs(upd_p).max())
