"""Pins for the APOLLO oracle (oracle/apollo.py): the paper states APOLLO only in words, and the
official implementation is not available here, so the oracle is held to what the definitions fix:

* storage: the projected layout (rank 256, the smaller side projected, full AdamW states for the
  embedding, LM head and 1-D tensors) reproduces Table 4's APOLLO FP32 optimizer state, 2078.7 MiB;
* the projection, by brute force (exact sums of exact products) and with selection matrices;
* the moments: with an identity projection APOLLO's projected direction is AdamW's, checked against
  torch.optim.AdamW's update over three steps;
* the channel scale at step 1 in closed form (R / (|R| + eps) per element);
* the norm-growth limiter's closed form (growth capped at gamma from the previous norm);
* exact zeros: an all-zero channel gets scale 0 (no update) and keeps code 0;
* the two projection sides agree under transposition.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import AL8, FP32, UF8, State
from oracle import apollo as oap
from paper_2608_22322_amd import apollo, synth
from paper_2608_22322_amd.workloads import tinyllama_shapes

MiB = 2.0**20


def _g(rows, cols, key, sigma=1e-3, zero_frac=0.0, mkey=0):
    return synth.normal_f32(key, rows * cols, sigma, mkey, zero_frac)


def _states(C, r, codes=False):
    n = C * r
    if codes:
        floor = float(np.float32(2 * math.log2(1e-8)))
        return State(UF8, n, 256), State(AL8, n, 2048, floor)
    return State(FP32, n), State(FP32, n)


def test_table4_apollo_fp32_state_reproduced():
    b = apollo.state_bytes(tinyllama_shapes(), rank=256)
    assert round(b / MiB, 1) == 2078.7


@pytest.mark.parametrize("shape", [(5, 7), (9, 4)])
def test_projection_brute_force(shape):
    rows, cols = shape
    right, C, L = oap.layout(rows, cols)
    r = 3
    g = synth.to_bf16_bits(_g(rows, cols, synth.grad_key(0, 1)))
    g64 = oap.bf16_to_f64(g)
    P = synth.proj_matrix(0, 0, L, r)
    R = oap.project(g64, rows, cols, P)
    G = g64.reshape(rows, cols)
    for c in range(C):
        for k in range(r):
            terms = [(G[c, l] if right else G[l, c]) * float(P[l, k]) for l in range(L)]  # exact products
            assert R[c, k] == np.float32(math.fsum(terms))


def test_selection_projection_picks_inputs():
    rows, cols = 12, 8  # right: channels = rows, L = cols
    sel = [5, 0, 7]
    P = np.zeros((cols, 3), np.float32)
    for k, l in enumerate(sel):
        P[l, k] = 1.0
    g = _g(rows, cols, synth.grad_key(1, 1))
    R = oap.project(g.astype(np.float64), rows, cols, P)
    assert np.array_equal(R, g.reshape(rows, cols)[:, sel])


def test_identity_projection_gives_the_adamw_direction():
    # rows >= cols with r = L and Pi = I: R = G, so the projected direction is AdamW's update direction
    rows, cols = 16, 8
    C, r = rows, cols
    P = np.eye(cols, dtype=np.float32)
    m, v = _states(C, r)
    prev = np.zeros(1, np.float32)
    p = np.zeros(rows * cols, np.float32)
    tp = torch.nn.Parameter(torch.zeros(rows * cols))
    opt = torch.optim.AdamW([tp], lr=1.0, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.0, foreach=False)
    for t in range(1, 4):
        g = _g(rows, cols, synth.grad_key(2, t))
        out = oap.apollo_step(p, g, rows, cols, P, m, v, t, prev, gamma=0.0)
        with torch.no_grad():
            tp.zero_()  # no weight decay: the parameter value does not enter the update
        tp.grad = torch.from_numpy(g.copy())
        opt.step()
        d = -tp.detach().numpy().reshape(rows, cols)  # torch's AdamW direction (fp32 arithmetic)
        assert np.allclose(out["Rt"], d, rtol=2e-6, atol=0)
        ref_s = np.sqrt((d.astype(np.float64) ** 2).sum(1)) / (np.sqrt((g.reshape(rows, cols).astype(np.float64)
                                                                         ** 2).sum(1)) + 1e-8)
        assert np.allclose(out["s"], ref_s, rtol=2e-6, atol=0)


def test_step1_channel_scale_closed_form():
    rows, cols, r = 6, 40, 16  # left: channels = columns, L = rows
    right, C, L = oap.layout(rows, cols)
    g = _g(rows, cols, synth.grad_key(3, 1))
    P = synth.proj_matrix(3, 0, L, r)
    m, v = _states(C, r)
    prev = np.zeros(1, np.float32)
    p = _g(rows, cols, synth.param_key(3), 0.02)
    p0 = p.copy()
    out = oap.apollo_step(p, g, rows, cols, P, m, v, 1, prev, lr=1e-4, gamma=0.0)
    R = out["R"].astype(np.float64)
    eps = 1e-8
    # at t = 1 the bias-corrected moments are R and R^2: the direction is R / (|R| + eps)
    s = np.sqrt(((R / (np.abs(R) + eps)) ** 2).sum(1)) / (np.sqrt((R ** 2).sum(1)) + 1e-8)
    assert np.allclose(out["s"], s, rtol=1e-6, atol=0)
    # the update scales each channel (column) of G by s_c
    upd = (p0.astype(np.float64) - p.astype(np.float64)).reshape(rows, cols) / 1e-4
    G = g.reshape(rows, cols).astype(np.float64)
    assert np.allclose(upd, G * s[None, :], rtol=2e-3, atol=1e-9)


def test_limiter_closed_form():
    rows, cols, r = 32, 16, 8
    right, C, L = oap.layout(rows, cols)
    P = synth.proj_matrix(4, 0, L, r)
    g1 = _g(rows, cols, synth.grad_key(4, 1))
    g2 = _g(rows, cols, synth.grad_key(4, 2))
    runs = {}
    for name, gamma, prev0 in (("free", 0.0, None), ("capped", 1.01, "small"), ("loose", 1.01, "large")):
        m, v = _states(C, r)
        prev = np.zeros(1, np.float32)
        p = np.zeros(rows * cols, np.float32)
        oap.apollo_step(p, g1, rows, cols, P, m, v, 1, prev, lr=1.0, gamma=gamma)
        if prev0 == "small":
            prev[0] = np.float32(prev[0] * 0.25)
        elif prev0 == "large":
            prev[0] = np.float32(prev[0] * 100.0)
        pv = prev[0]
        p[:] = 0.0
        out = oap.apollo_step(p, g2, rows, cols, P, m, v, 2, prev, lr=1.0, gamma=gamma)
        runs[name] = (p.copy(), out, pv, prev[0])
    pf, of, _, _ = runs["free"]
    pc, oc, pv, after = runs["capped"]
    lam = (of["norm"] / (float(pv) + 1e-8)) / 1.01
    assert lam > 1.0 and math.isclose(oc["lam"], lam, rel_tol=1e-12)
    assert after == np.float32(of["norm"] / lam)  # the stored norm grows by exactly gamma
    assert math.isclose(float(after), 1.01 * float(pv), rel_tol=1e-6)
    assert np.allclose(pc, (pf.astype(np.float64) / lam).astype(np.float32), rtol=1e-6, atol=0)
    pl, ol, _, _ = runs["loose"]
    assert ol["lam"] == 1.0 and np.array_equal(pl, pf)


def test_zero_channel_is_left_alone():
    rows, cols, r = 20, 10, 8  # right: channels = rows
    right, C, L = oap.layout(rows, cols)
    g = _g(rows, cols, synth.grad_key(5, 1)).reshape(rows, cols)
    g[3] = 0.0
    P = synth.proj_matrix(5, 0, L, r)
    m, v = _states(C, r, codes=True)
    p = _g(rows, cols, synth.param_key(5), 0.02)
    p0 = p.copy()
    prev = np.zeros(1, np.float32)
    out = oap.apollo_step(p, g.ravel(), rows, cols, P, m, v, 1, prev, wd=0.1)
    assert out["s"][3] == 0.0
    assert np.array_equal(p.reshape(rows, cols)[3], (p0.reshape(rows, cols)[3].astype(np.float64)
                                                     * (1 - 1e-4 * 0.1)).astype(np.float32))
    assert np.all(m.codes[3 * r:4 * r] == 0) and np.all(v.codes[3 * r:4 * r] == 0)
    assert np.all(v.codes[:3 * r] != 0)


def test_transpose_symmetry():
    rows, cols, r = 6, 24, 8  # left projection; its transpose (24 x 6) takes the right one
    g = _g(rows, cols, synth.grad_key(6, 1)).reshape(rows, cols)
    P = synth.proj_matrix(6, 0, rows, r)
    p = _g(rows, cols, synth.param_key(6), 0.02).reshape(rows, cols)
    a_p, b_p = p.ravel().copy(), p.T.ravel().copy()
    a_m, a_v = _states(cols, r, codes=True)
    b_m, b_v = _states(cols, r, codes=True)
    a_prev, b_prev = np.zeros(1, np.float32), np.zeros(1, np.float32)
    for t in (1, 2):
        gt = g * t
        oa = oap.apollo_step(a_p, gt.ravel(), rows, cols, P, a_m, a_v, t, a_prev)
        ob = oap.apollo_step(b_p, np.ascontiguousarray(gt.T).ravel(), cols, rows, P, b_m, b_v, t, b_prev)
        assert np.array_equal(oa["R"], ob["R"]) and np.array_equal(oa["s"], ob["s"])
    assert np.array_equal(a_p.reshape(rows, cols), b_p.reshape(cols, rows).T)
    assert np.array_equal(a_m.codes, b_m.codes) and np.array_equal(a_v.codes, b_v.codes)


@pytest.mark.parametrize("shape", [(24, 16), (16, 24)])
def test_channel_permutation_equivariance(shape):
    """Permuting the channels of the gradient and the parameter (rows when rows >= cols, else columns)
    with the projection fixed permutes R, both moments, the direction and the channel scales, and leaves
    the limiter's norm unchanged (its sum is exact), so 5 steps give the permuted parameter bit for bit:
    each channel's scale reads only its own row of R and of the direction."""
    rows, cols = shape
    r = 8
    right, C, L = oap.layout(rows, cols)
    rng = np.random.default_rng(71)
    perm = rng.permutation(C)
    P = synth.proj_matrix(71, 0, L, r)
    p0 = _g(rows, cols, synth.param_key(71), 0.02).reshape(rows, cols)

    def chan(x):  # x: rows x cols
        return x[perm] if right else x[:, perm]

    a_p, b_p = p0.ravel().copy(), np.ascontiguousarray(chan(p0)).ravel()
    a_m, a_v = _states(C, r)
    b_m, b_v = _states(C, r)
    a_prev, b_prev = np.zeros(1, np.float32), np.zeros(1, np.float32)
    for t in range(1, 6):
        g = _g(rows, cols, synth.grad_key(72, t), zero_frac=0.05).reshape(rows, cols)
        sc = np.exp2(rng.integers(-2, 3, C)).astype(np.float32)  # channel magnitudes that vary by step
        g = g * (sc[:, None] if right else sc[None, :])
        oa = oap.apollo_step(a_p, g.ravel(), rows, cols, P, a_m, a_v, t, a_prev)
        ob = oap.apollo_step(b_p, np.ascontiguousarray(chan(g)).ravel(), rows, cols, P, b_m, b_v, t, b_prev)
        assert np.array_equal(oa["R"][perm], ob["R"]) and np.array_equal(oa["s"][perm], ob["s"]), t
        assert a_prev[0] == b_prev[0], t
    assert np.array_equal(chan(a_p.reshape(rows, cols)), b_p.reshape(rows, cols))
    for a, b in ((a_m, b_m), (a_v, b_v)):
        assert np.array_equal(a.codes.reshape(C, r)[perm], b.codes.reshape(C, r))
    assert np.ptp(oa["s"]) > 0.1 * np.abs(oa["s"]).mean()  # the scales differ by channel
