"""Update-domain and temporal diagnostics (section 3.2, Eq. update_error; section 5).

E_upd = ||U(S_hat, G) - U(S, G)||_2 / (||U(S, G)||_2 + eps): the update an optimizer
step produces from a state reconstructed from its codes, S_hat, against the update from
the exact state S, for the same gradient G. Both updates come from the library's step
kernels (the reference run uses FP32 states, the other the state codes produced by
al_quantize from the same values), starting from zero parameters so the parameters
after the step are the updates themselves; al_diff_norms forms the two sums of squares.

state_error is the relative reconstruction error of one vector under a state code, and
ema_drift the temporal probe of section 5: two trajectories of the same optimizer over
the same gradients, one with FP32 states and one with the codes under test, compared
after K steps in the state domain (relative L2 drift of each decoded state) and in the
update domain (E_upd of step K).
"""
from __future__ import annotations

import math

from . import (FP32, ParamState, Spec, StateSpec, adafactor_step, adafactor_workspace_bytes, adamw_step,
               adamw_workspace_bytes,               alloc_state, came_step, came_workspace_bytes, dequantize, diff_norms, DIFF_NORMS_OUT, quantize,
               tensor_array)

ROLES = ("m", "v", "vr", "vc", "cr", "cc")
KINDS = ("adamw", "adafactor", "came")


def _role_spec(kind: str, cfg, role: str) -> StateSpec:
    if role == "m":
        return cfg.m
    if role in ("cr", "cc"):
        return cfg.conf
    return cfg.v


def _spec(ss: StateSpec) -> Spec:
    return Spec(ss.codec, ss.block, ss.log_floor)


def _role_len(st, role: str) -> int:
    if role in ("m", "v"):
        return st.rows * st.cols
    return st.rows if role in ("vr", "cr") else st.cols


def _cfg_copy(kind: str, cfg, fp32: bool = False, lr: float | None = None):
    out = type(cfg).from_buffer_copy(cfg)
    if fp32:
        for n in {"adamw": ("m", "v"), "adafactor": ("v",), "came": ("m", "v", "conf")}[kind]:
            ss = getattr(cfg, n)
            setattr(out, n, StateSpec(FP32, ss.block, ss.log_floor))
    if lr is not None:
        out.lr = lr
    return out


def _fp32_cfg(kind: str, cfg):
    return _cfg_copy(kind, cfg, fp32=True)


class _Stepper:
    """One optimizer kind over a fixed tensor list: descriptor array and workspace built once."""

    def __init__(self, kind: str, states, cfgs, device):
        import torch

        self.kind, self.states = kind, states
        self.arr = tensor_array(states)
        fn = {"adamw": adamw_workspace_bytes, "adafactor": adafactor_workspace_bytes,
              "came": came_workspace_bytes}[kind]
        nbytes = max(fn(states, c, arr=self.arr) for c in cfgs)
        self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)

    def __call__(self, cfg, t: int, stream=None) -> None:
        if self.kind == "adamw":
            adamw_step(self.states, cfg, t, self.ws, stream=stream, arr=self.arr)
        elif self.kind == "adafactor":
            adafactor_step(self.states, cfg, t, self.ws, stream=stream, arr=self.arr)
        else:
            came_step(self.states, cfg, t, self.ws, stream=stream, arr=self.arr)


def _run(kind: str, states, cfg, t: int, device, stream) -> None:
    _Stepper(kind, states, [cfg], device)(cfg, t, stream)


class _Norms:
    """Running sums of ||a - b||^2 and ||b||^2 over device vector pairs (al_diff_norms)."""

    def __init__(self, device):
        import torch

        self.out = torch.empty(DIFF_NORMS_OUT, dtype=torch.float64, device=device)
        self.num = self.den = 0.0

    def add(self, a, b, stream=None) -> None:
        diff_norms(a, b, self.out, stream=stream)
        s = self.out[:2].cpu()
        self.num += float(s[0])
        self.den += float(s[1])

    def rel(self, eps: float = 0.0) -> float:
        return math.sqrt(self.num) / (math.sqrt(self.den) + eps)


def update_error(kind: str, ref_states, cfg, t: int, eps: float = 1e-30, stream=None) -> float:
    """E_upd of one step (kind: 'adamw', 'adafactor', 'came') over a tensor list.

    ref_states: ParamState list whose state buffers (m, v, vr, vc, cr, cc as the optimizer
    uses them) hold the exact states in FP32; grad holds G; param is ignored. cfg: the
    optimizer config with the state codes under test (its FP32 counterpart is derived). The
    reference states are not modified."""
    import torch

    if kind not in KINDS:
        raise ValueError(kind)
    device = ref_states[0].grad.device
    ref, quant = [], []
    for st in ref_states:
        n = st.rows * st.cols
        r = ParamState(torch.zeros(max(n, 4), dtype=torch.float32, device=device), st.grad, st.rows, st.cols)
        q = ParamState(torch.zeros(max(n, 4), dtype=torch.float32, device=device), st.grad, st.rows, st.cols)
        for role in ROLES:
            buf = getattr(st, role)
            if buf is None:
                continue
            length = _role_len(st, role)
            setattr(r, role, buf.clone())
            ss = _role_spec(kind, cfg, role)
            if ss.codec == FP32:
                setattr(q, role, buf.clone())
                continue
            codes, meta = alloc_state(length, _spec(ss), device)
            quantize(ss.codec, buf[:length], ss.block, ss.log_floor, codes, meta, stream=stream)
            setattr(q, role, codes)
            setattr(q, role + "_meta", meta)
        ref.append(r)
        quant.append(q)
    _run(kind, ref, _fp32_cfg(kind, cfg), t, device, stream)
    _run(kind, quant, cfg, t, device, stream)
    acc = _Norms(device)
    for r, q, st in zip(ref, quant, ref_states):
        n = st.rows * st.cols
        acc.add(q.param[:n], r.param[:n], stream=stream)
    return acc.rel(eps)


def state_error(x, spec: Spec, stream=None) -> float:
    """Relative reconstruction error ||dec(enc(x)) - x||_2 / ||x||_2 of one float32 device vector
    under a state code (al_quantize, then al_dequantize). Exact zeros decode to zero, so they add
    nothing to either norm."""
    import torch

    n = x.numel()
    if spec.codec == FP32 or n == 0:
        return 0.0
    codes, meta = alloc_state(n, spec, x.device)
    quantize(spec.codec, x, spec.block, spec.log_floor, codes, meta, stream=stream)
    y = torch.empty(max(n, 4), dtype=torch.float32, device=x.device)
    dequantize(spec.codec, codes, meta, n, spec.block, y, stream=stream)
    acc = _Norms(x.device)
    acc.add(y[:n], x, stream=stream)
    return acc.rel()


def _attach(kind: str, sts, cfg, device) -> None:
    roles = {"adamw": ("m", "v"), "adafactor": ("v",), "came": ("m", "v", "conf")}[kind]
    specs = {r: getattr(cfg, r) for r in roles}
    for st in sts:
        n = st.rows * st.cols
        if kind in ("adamw", "came"):
            st.m, st.m_meta = alloc_state(n, _spec(specs["m"]), device)
        if kind == "adamw" or st.rows <= 1:
            st.v, st.v_meta = alloc_state(n, _spec(specs["v"]), device)
            continue
        st.vr, st.vr_meta = alloc_state(st.rows, _spec(specs["v"]), device)
        st.vc, st.vc_meta = alloc_state(st.cols, _spec(specs["v"]), device)
        if kind == "came":
            st.cr, st.cr_meta = alloc_state(st.rows, _spec(specs["conf"]), device)
            st.cc, st.cc_meta = alloc_state(st.cols, _spec(specs["conf"]), device)


def ema_drift(kind: str, shapes, cfg, steps: int, grad_fn, grads, eps: float = 1e-30, stream=None) -> dict:
    """Temporal probe (section 5): K = steps optimizer steps from zero states over the gradients
    grad_fn supplies, once with FP32 states and once with cfg's state codes.

    shapes: (rows, cols) per tensor; grads: one device gradient buffer per tensor (float32 or
    bfloat16 as cfg says, at least rows * cols elements); grad_fn(t) refills them for step t
    (1-based). Steps 1..K-1 run with lr = 0, so both trajectories see the same gradients and
    only their states evolve; step K starts from zero parameters with cfg's lr, so the two
    parameter vectors are the two updates. Returns {"drift": {role: ||dec(S_hat_K) - S_K|| /
    ||S_K||}, "update_error": E_upd of step K}; roles with FP32 codes are left out of drift."""
    import torch

    if kind not in KINDS:
        raise ValueError(kind)
    if steps < 1:
        raise ValueError("steps must be >= 1")
    device = grads[0].device
    mk = lambda: [ParamState(torch.zeros(max(r * c, 4), dtype=torch.float32, device=device), g, r, c)
                  for (r, c), g in zip(shapes, grads)]
    ref, quant = mk(), mk()
    cfg_ref = _cfg_copy(kind, cfg, fp32=True)
    _attach(kind, ref, cfg_ref, device)
    _attach(kind, quant, cfg, device)
    cfg_ref0, cfg0 = _cfg_copy(kind, cfg_ref, lr=0.0), _cfg_copy(kind, cfg, lr=0.0)
    run_ref = _Stepper(kind, ref, [cfg_ref, cfg_ref0], device)
    run_q = _Stepper(kind, quant, [cfg, cfg0], device)
    for t in range(1, steps + 1):
        grad_fn(t)
        last = t == steps
        run_ref(cfg_ref if last else cfg_ref0, t, stream)
        run_q(cfg if last else cfg0, t, stream)
    upd = _Norms(device)
    drift = {}
    for r, q, (rows, cols) in zip(ref, quant, shapes):
        n = rows * cols
        upd.add(q.param[:n], r.param[:n], stream=stream)
        for role in ROLES:
            if getattr(q, role) is None:
                continue
            ss = _role_spec(kind, cfg, role)
            if ss.codec == FP32:
                continue
            length = _role_len(q, role)
            y = torch.empty(max(length, 4), dtype=torch.float32, device=device)
            dequantize(ss.codec, getattr(q, role), getattr(q, role + "_meta"), length, ss.block, y, stream=stream)
            drift.setdefault(role, _Norms(device)).add(y[:length], getattr(r, role)[:length], stream=stream)
    return {"drift": {k: v.rel() for k, v in drift.items()}, "update_error": upd.rel(eps)}


def apollo_update_error(tensors, cfg, t: int, eps: float = 1e-30, stream=None) -> float:
    """E_upd of one APOLLO step (al_apollo_step) over projected tensors.

    tensors: (grad, rows, cols, proj, m, v) per tensor, all device tensors: grad G, the projection
    (L x rank fp32) and the exact projected moments m, v in FP32 (rank * C elements each). cfg: an
    APOLLO config with the state codes under test (its FP32 counterpart is derived). Both runs start
    from zero parameters with the limiter off (it only rescales a tensor's whole update), so the
    parameters after the step are the two updates -lr g s_c. The inputs are not modified."""
    import torch

    from . import ApolloCfg, apollo_step, apollo_tensor_array, apollo_workspace_bytes

    device = tensors[0][0].device
    ref_cfg = ApolloCfg.from_buffer_copy(cfg)
    ref_cfg.m = StateSpec(FP32, cfg.m.block, cfg.m.log_floor)
    ref_cfg.v = StateSpec(FP32, cfg.v.block, cfg.v.log_floor)
    ref_cfg.gamma = 0.0
    q_cfg = ApolloCfg.from_buffer_copy(cfg)
    q_cfg.gamma = 0.0
    ref_items, q_items, keep = [], [], []
    for g, rows, cols, proj, m, v in tensors:
        n = rows * cols
        pr = torch.zeros(max(n, 4), dtype=torch.float32, device=device)
        pq = torch.zeros(max(n, 4), dtype=torch.float32, device=device)
        ref_items.append((pr, g, rows, cols, proj, m.clone(), None, v.clone(), None, None))
        length = m.numel()
        coded = []
        for buf, ss in ((m, cfg.m), (v, cfg.v)):
            if ss.codec == FP32:
                coded += [buf.clone(), None]
                continue
            codes, meta = alloc_state(length, _spec(ss), device)
            quantize(ss.codec, buf[:length], ss.block, ss.log_floor, codes, meta, stream=stream)
            coded += [codes, meta]
        q_items.append((pq, g, rows, cols, proj, coded[0], coded[1], coded[2], coded[3], None))
        keep.append((pr, pq, n))
    for items, c in ((ref_items, ref_cfg), (q_items, q_cfg)):
        arr = apollo_tensor_array(items)
        nbytes = apollo_workspace_bytes(arr, len(items), c)
        ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        apollo_step(arr, len(items), c, t, ws, stream)
    acc = _Norms(device)
    for pr, pq, n in keep:
        acc.add(pq[:n], pr[:n], stream=stream)
    return acc.rel(eps)


__all__ = ["update_error", "state_error", "ema_drift", "apollo_update_error"]
