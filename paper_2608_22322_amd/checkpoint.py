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

import numpy as np

from . import AL8, AL16, FP32, UF8, Spec, alloc_state, dequantize, quantize

ROLES = ("m", "v", "vr", "vc", "cr", "cc")
_CODECS = {FP32: "FP32", AL8: "AL8", AL16: "AL16", UF8: "UF8"}
_BY_NAME = {v: k for k, v in _CODECS.items()}
_SAFE_DTYPES = {"F32": "float32", "U8": "uint8", "I16": "int16", "I8": "int8"}


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


def _layout(n: int, spec: Spec):
    """(code dtype name, code elements, meta floats) that alloc_state gives an n-element state: the sizes the
    kernels index."""
    from . import code_bytes, meta_floats

    if spec.codec == FP32:
        return "float32", max(n, 1), 0
    dt = {AL8: "uint8", AL16: "int16", UF8: "int8"}[spec.codec]
    elems = code_bytes(spec.codec, n, spec.block) // (2 if spec.codec == AL16 else 1)
    return dt, max(elems, 1), max(meta_floats(spec.codec, n, spec.block), 4)


def load(path: str, states, specs, kind: str | None = None):
    """Copy a checkpoint's coded states into the existing state buffers of a ParamState list.

    states: the same tensors (shapes checked), with their state buffers already allocated for `specs` (for
    instance by alloc_state or grouping.attach_states); specs: per tensor, a dict role -> Spec the caller
    will step with; kind: the optimizer kind expected (None: any). The checkpoint must hold exactly those
    roles with the same codec, block and log floor, and each stored array must have the dtype and size of
    the destination buffer, at least the size the spec needs. The buffers are overwritten in place
    (copy_), so descriptor arrays and steppers built over them stay valid. Returns (kind, step)."""
    from safetensors import safe_open

    with safe_open(path, framework="pt") as f:
        header = f.metadata()
        if header.get("format") != "al-optimizer-state/1":
            raise ValueError(f"{path}: not an optimizer-state checkpoint")
        if kind is not None and header["kind"] != kind:
            raise ValueError(f"{path}: optimizer {header['kind']}, expected {kind}")
        info = json.loads(header["tensors"])
        if len(info) != len(states) or len(specs) != len(states):
            raise ValueError(f"{path}: {len(info)} tensors, expected {len(states)} (with {len(specs)} specs)")
        keys = set(f.keys())
        plan = []
        for i, (st, ti, want) in enumerate(zip(states, info, specs)):
            tag = f"{path}: tensor {i} ({ti['name']})"
            if (ti["rows"], ti["cols"]) != (st.rows, st.cols):
                raise ValueError(f"{tag} shape {ti['rows']}x{ti['cols']} != {st.rows}x{st.cols}")
            if set(ti["roles"]) != set(want):
                raise ValueError(f"{tag} holds roles {sorted(ti['roles'])}, expected {sorted(want)}")
            for role, r in ti["roles"].items():
                w = want[role]
                got = Spec(_BY_NAME[r["codec"]], int(r["block"]), float(r["log_floor"]))
                same = got.codec == w.codec and (w.codec == FP32 or (
                    got.block == w.block and np.float32(got.log_floor) == np.float32(w.log_floor)))
                if not same:
                    raise ValueError(f"{tag} {role}: saved as {r['codec']} block {r['block']} floor "
                                     f"{r['log_floor']}, expected {_CODECS[w.codec]} block {w.block} floor "
                                     f"{w.log_floor}")
                n = _role_len(st, role)
                if int(r["n"]) != n:
                    raise ValueError(f"{tag} {role}: {r['n']} elements, expected {n}")
                dt, ncode, nmeta = _layout(n, w)
                parts = [(role, f"t{i}.{role}", ncode, dt)]
                if nmeta:
                    parts.append((role + "_meta", f"t{i}.{role}.meta", nmeta, "float32"))
                elif f"t{i}.{role}.meta" in keys:
                    raise ValueError(f"{tag} {role}: metadata stored for an FP32 state")
                for attr, key, need, want_dt in parts:
                    dst = getattr(st, attr)
                    if dst is None:
                        raise ValueError(f"{tag} {attr}: no buffer to load into (allocate the states first)")
                    if key not in keys:
                        raise ValueError(f"{tag}: {key} missing")
                    sl = f.get_slice(key)
                    shape, sdt = sl.get_shape(), sl.get_dtype()
                    numel = int(np.prod(shape)) if shape else 1
                    if str(dst.dtype) != "torch." + want_dt or _SAFE_DTYPES.get(sdt) != want_dt:
                        raise ValueError(f"{tag} {attr}: dtype {sdt} / buffer {dst.dtype}, expected {want_dt}")
                    if numel != dst.numel() or numel < need:
                        raise ValueError(f"{tag} {attr}: {numel} stored elements, buffer {dst.numel()}, "
                                         f"at least {need} needed")
                    plan.append((dst, key))
        for dst, key in plan:  # every check passed: overwrite in place
            dst.copy_(f.get_tensor(key).to(dst.device))
    return header["kind"], int(header["step"])


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
