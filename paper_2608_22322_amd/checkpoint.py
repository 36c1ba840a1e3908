"""Optimizer-state checkpoints and state-precision migration (section 7.1).

A checkpoint keeps every state in its coded form -- codes, block metadata and the code
type (codec, block size, log floor) -- so saving and loading is exact and training resumes
bit for bit. Migration re-codes a state under another spec (for instance AL8 -> AL16) by
decoding it with al_dequantize and encoding the values with al_quantize.

File format: one safetensors file. Tensor "t{i}.{role}" holds the codes (or FP32 values),
"t{i}.{role}.meta" the block metadata; the JSON header metadata holds, per tensor, its name,
shape and per-role spec, plus the optimizer kind and step.

APOLLO (save_apollo / load_apollo) keeps the projected moments "p{i}.m", "p{i}.v" (+ ".meta") and
the limiter state "p{i}.norm" of every projected tensor, the full AdamW states "t{i}.m", "t{i}.v" of
the others, and in the header the rank, codes, refresh gap and seed: the projection itself is not
stored, it is drawn again from the seeded stream of its refresh period.
"""
from __future__ import annotations

import json

from . import AL8, AL16, FP32, UF8, Spec, alloc_state, dequantize, quantize

ROLES = ("m", "v", "vr", "vc", "cr", "cc")
_CODECS = {FP32: "FP32", AL8: "AL8", AL16: "AL16", UF8: "UF8"}
_BY_NAME = {v: k for k, v in _CODECS.items()}


def _role_len(st, role: str) -> int:
    if role in ("m", "v"):
        return st.rows * st.cols
    return st.rows if role in ("vr", "cr") else st.cols


def save(path: str, states, specs, names, kind: str, step: int) -> None:
    """Write the coded states of a tensor list.

    states: ParamState list; specs: per tensor, a dict role -> Spec for the roles it holds;
    names: tensor names; kind: optimizer kind; step: the last completed step."""
    from safetensors.torch import save_file

    tensors, info = {}, []
    for i, (st, sp, name) in enumerate(zip(states, specs, names)):
        roles = {}
        for role in ROLES:
            buf = getattr(st, role)
            if buf is None:
                continue
            s = sp[role]
            tensors[f"t{i}.{role}"] = buf.detach().contiguous().cpu()
            meta = getattr(st, role + "_meta")
            if meta is not None:
                tensors[f"t{i}.{role}.meta"] = meta.detach().contiguous().cpu()
            roles[role] = {"codec": _CODECS[s.codec], "block": int(s.block), "log_floor": float(s.log_floor),
                           "n": _role_len(st, role)}
        info.append({"name": name, "rows": int(st.rows), "cols": int(st.cols), "roles": roles})
    header = {"format": "al-optimizer-state/1", "kind": kind, "step": str(int(step)), "tensors": json.dumps(info)}
    save_file(tensors, path, metadata=header)


def load(path: str, states, device="cuda"):
    """Load coded states into a ParamState list of the same tensors (shapes checked); returns
    (kind, step, specs) with specs per tensor as dicts role -> Spec."""
    from safetensors import safe_open

    with safe_open(path, framework="pt") as f:
        header = f.metadata()
        if header.get("format") != "al-optimizer-state/1":
            raise ValueError(f"{path}: not an optimizer-state checkpoint")
        info = json.loads(header["tensors"])
        if len(info) != len(states):
            raise ValueError(f"{path}: {len(info)} tensors, expected {len(states)}")
        specs = []
        for i, (st, ti) in enumerate(zip(states, info)):
            if (ti["rows"], ti["cols"]) != (st.rows, st.cols):
                raise ValueError(f"{path}: tensor {i} ({ti['name']}) shape {ti['rows']}x{ti['cols']} "
                                 f"!= {st.rows}x{st.cols}")
            sp = {}
            for role, r in ti["roles"].items():
                setattr(st, role, f.get_tensor(f"t{i}.{role}").to(device))
                key = f"t{i}.{role}.meta"
                setattr(st, role + "_meta", f.get_tensor(key).to(device) if key in f.keys() else None)
                sp[role] = Spec(_BY_NAME[r["codec"]], r["block"], r["log_floor"])
            specs.append(sp)
    return header["kind"], int(header["step"]), specs


def migrate(st, role: str, old: Spec, new: Spec, stream=None) -> None:
    """Re-code one state of a ParamState from spec old to spec new (e.g. AL8 -> AL16, AL16 -> AL8,
    FP32 <-> AL). Values are decoded to fp32 and encoded again; FP32 states are taken as is."""
    import torch

    n = _role_len(st, role)
    buf, meta = getattr(st, role), getattr(st, role + "_meta")
    device = buf.device
    if old.codec == FP32:
        x = buf
    else:
        x = torch.empty(max(n, 4), dtype=torch.float32, device=device)
        dequantize(old.codec, buf, meta, n, old.block, x, stream=stream)
    if new.codec == FP32:
        setattr(st, role, x if old.codec != FP32 else buf)
        setattr(st, role + "_meta", None)
        return
    codes, nmeta = alloc_state(n, new, device)
    quantize(new.codec, x[:n], new.block, new.log_floor, codes, nmeta, stream=stream)
    setattr(st, role, codes)
    setattr(st, role + "_meta", nmeta)


def _spec_json(ss) -> dict:
    return {"codec": _CODECS[ss.codec], "block": int(ss.block), "log_floor": float(ss.log_floor)}


def save_apollo(path: str, drv, names, step: int) -> None:
    """Write the state of an apollo.ApolloStep after `step` completed steps."""
    from safetensors.torch import save_file

    tensors, proj, full = {}, [], []
    for k, (i, L, pj) in enumerate(drv.proj):
        _, _, rows, cols, _, m, mm, v, vm, ns = drv.items[k]
        tensors[f"p{i}.m"] = m.detach().cpu()
        tensors[f"p{i}.v"] = v.detach().cpu()
        if mm is not None:
            tensors[f"p{i}.m.meta"] = mm.detach().cpu()
        if vm is not None:
            tensors[f"p{i}.v.meta"] = vm.detach().cpu()
        tensors[f"p{i}.norm"] = ns.detach().cpu()
        proj.append({"index": i, "name": names[i], "rows": int(rows), "cols": int(cols)})
    for i, st in zip(drv.full_idx, drv.full_states):
        for role in ("m", "v"):
            tensors[f"t{i}.{role}"] = getattr(st, role).detach().cpu()
            meta = getattr(st, role + "_meta")
            if meta is not None:
                tensors[f"t{i}.{role}.meta"] = meta.detach().cpu()
        full.append({"index": i, "name": names[i], "rows": int(st.rows), "cols": int(st.cols)})
    c = drv.cfg
    header = {"format": "al-apollo-state/1", "step": str(int(step)), "rank": str(int(c.rank)),
              "gap": str(int(drv.gap)), "seed": str(int(drv.seed)), "m": json.dumps(_spec_json(c.m)),
              "v": json.dumps(_spec_json(c.v)), "projected": json.dumps(proj), "full": json.dumps(full)}
    save_file(tensors, path, metadata=header)


def load_apollo(path: str, drv, names) -> int:
    """Copy a saved APOLLO state into an ApolloStep built over the same tensor list (same names, shapes,
    rank, codes, gap and seed); the buffers are overwritten in place. Returns the saved step; the next
    step() draws the projection of its refresh period again."""
    from safetensors import safe_open

    c = drv.cfg
    with safe_open(path, framework="pt") as f:
        h = f.metadata()
        if h.get("format") != "al-apollo-state/1":
            raise ValueError(f"{path}: not an APOLLO optimizer-state checkpoint")
        want = {"rank": str(int(c.rank)), "gap": str(int(drv.gap)), "seed": str(int(drv.seed)),
                "m": json.dumps(_spec_json(c.m)), "v": json.dumps(_spec_json(c.v))}
        for key, val in want.items():
            if h[key] != val:
                raise ValueError(f"{path}: {key} {h[key]} != {val}")
        proj, full = json.loads(h["projected"]), json.loads(h["full"])
        if [p["index"] for p in proj] != [i for i, _, _ in drv.proj] or \
                [p["index"] for p in full] != list(drv.full_idx):
            raise ValueError(f"{path}: the projected / full tensor sets differ")
        for p in proj + full:
            if p["name"] != names[p["index"]]:
                raise ValueError(f"{path}: tensor {p['index']} is {p['name']}, expected {names[p['index']]}")
        for k, (i, L, pj) in enumerate(drv.proj):
            _, _, rows, cols, _, m, mm, v, vm, ns = drv.items[k]
            if (proj[k]["rows"], proj[k]["cols"]) != (rows, cols):
                raise ValueError(f"{path}: tensor {i} shape differs")
            for buf, key in ((m, f"p{i}.m"), (mm, f"p{i}.m.meta"), (v, f"p{i}.v"), (vm, f"p{i}.v.meta"),
                             (ns, f"p{i}.norm")):
                if buf is not None:
                    buf.copy_(f.get_tensor(key).to(buf.device))
        for k, (i, st) in enumerate(zip(drv.full_idx, drv.full_states)):
            if (full[k]["rows"], full[k]["cols"]) != (st.rows, st.cols):
                raise ValueError(f"{path}: tensor {i} shape differs")
            for role in ("m", "v"):
                getattr(st, role).copy_(f.get_tensor(f"t{i}.{role}").to(st.param.device))
                meta = getattr(st, role + "_meta")
                if meta is not None:
                    meta.copy_(f.get_tensor(f"t{i}.{role}.meta").to(st.param.device))
    drv._epoch = None
    return int(h["step"])


__all__ = ["save", "load", "migrate", "save_apollo", "load_apollo"]
