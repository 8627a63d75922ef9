"""Stand-in weight loaders of the trainer and rollout engines, written with
torch slicing.

Each style function takes the checkpoint as {name: tensor} and returns one
rank's local tensors, built from whole-tensor torch operations (chunk, cat,
stack, t, flatten) rather than from placements. They serve two purposes: an
independent statement of what each parallelism style stores (pinning the
declared placements), and the black-box loader whose copies source-map probing
observes. Copies here never change values.
"""

from __future__ import annotations

import torch


def _ckpt_names(model):
    fam, L = model["family"], model["num_layers"]
    names = []
    if fam in ("dense", "mixtral"):
        names.append("embed")
    for layer in range(L):
        p = f"layers.{layer}."
        if fam in ("dense", "mixtral"):
            names += [p + n for n in ("attn_norm", "q", "k", "v", "o", "mlp_norm")]
        if fam == "dense":
            names += [p + n for n in ("gate", "up", "down")]
            continue
        names.append(p + "router")
        if fam == "moe_only":
            names += [p + "shared.gate", p + "shared.up", p + "shared.down"]
        for e in range(model["num_experts"]):
            names += [f"{p}experts.{e}.{n}" for n in ("gate", "up", "down")]
    if fam in ("dense", "mixtral"):
        names += ["final_norm", "lm_head"]
    return names


def fsdp_flat(model, par, T, rank):
    """FSDP1-style flat units, each padded to a multiple of the degree."""
    fsdp, ep = par.get("fsdp", 1), par.get("ep", 1)
    f = rank % fsdp
    ep_i = (rank // fsdp) % ep
    fam = model["family"]
    units = []
    if fam in ("dense", "mixtral"):
        units.append(["embed"])
    for layer in range(model["num_layers"]):
        p = f"layers.{layer}."
        mine = [n for n in _ckpt_names(model) if n.startswith(p)]
        if fam == "dense":
            units.append(mine)
            continue
        units.append([n for n in mine if ".experts." not in n])
        per = model["num_experts"] // ep
        units.append([n for n in mine if ".experts." in n and per * ep_i <= int(n.split(".")[3]) < per * (ep_i + 1)])
    if fam in ("dense", "mixtral"):
        units.append(["final_norm", "lm_head"])
    out = []
    for names in units:
        flat = torch.cat([T[n].flatten() for n in names])
        pad = (-flat.numel()) % fsdp
        flat = torch.cat([flat, flat.new_zeros(pad)])
        out.append(flat.chunk(fsdp)[f])
    return out


def megatron(model, par, T, rank):
    tp, ep = par.get("tp", 1), par.get("ep", 1)
    tr = par.get("transposed_row_parallel", False)
    r = rank % tp
    ep_i = (rank // tp) % ep
    fam = model["family"]
    hd = model.get("head_dim", 0)
    out = []

    def rowpar(w):
        s = w.chunk(tp, dim=1)[r]
        return s.t().contiguous() if tr else s

    if fam in ("dense", "mixtral"):
        out.append(T["embed"].chunk(tp)[r])
    for layer in range(model["num_layers"]):
        p = f"layers.{layer}."
        if fam in ("dense", "mixtral"):
            out.append(T[p + "attn_norm"])
            nkv, nq = model["num_kv_heads"], model["num_heads"]
            qg = T[p + "q"].reshape(nkv, nq // nkv * hd, -1)
            kg = T[p + "k"].reshape(nkv, hd, -1)
            vg = T[p + "v"].reshape(nkv, hd, -1)
            groups = torch.cat([qg, kg, vg], dim=1).chunk(tp)[r]
            out.append(groups.reshape(-1, groups.shape[-1]))
            out.append(rowpar(T[p + "o"]))
            out.append(T[p + "mlp_norm"])
        if fam == "dense":
            out.append(torch.cat([T[p + "gate"].chunk(tp)[r], T[p + "up"].chunk(tp)[r]]))
            out.append(rowpar(T[p + "down"]))
            continue
        out.append(T[p + "router"])
        if fam == "moe_only":
            out += [T[p + "shared.gate"], T[p + "shared.up"], rowpar(T[p + "shared.down"])]
        el = model["num_experts"] // ep
        es = range(ep_i * el, (ep_i + 1) * el)
        out.append(torch.stack([T[f"{p}experts.{e}.gate"] for e in es]))
        out.append(torch.stack([T[f"{p}experts.{e}.up"] for e in es]))
        out.append(torch.stack([rowpar(T[f"{p}experts.{e}.down"]) for e in es]))
    if fam in ("dense", "mixtral"):
        out.append(T["final_norm"])
        out.append(T["lm_head"].chunk(tp)[r])
    return out


def serving(model, par, T, rank):
    """Serving-style locals (quantised tensors are returned before quantisation
    and are followed by None in place of their scale tensor)."""
    tp, ep = par.get("tp", 1), par.get("ep", 1)
    q = bool(par.get("quant"))
    r = rank % tp
    ep_i = (rank // tp) % ep
    fam = model["family"]
    out = []

    def lin(x):
        out.append(x)
        if q:
            out.append(None)

    if fam in ("dense", "mixtral"):
        out.append(T["embed"].chunk(tp)[r])
    for layer in range(model["num_layers"]):
        p = f"layers.{layer}."
        if fam in ("dense", "mixtral"):
            out.append(T[p + "attn_norm"])
            lin(torch.cat([T[p + "q"].chunk(tp)[r], T[p + "k"].chunk(tp)[r], T[p + "v"].chunk(tp)[r]]))
            lin(T[p + "o"].chunk(tp, dim=1)[r])
            out.append(T[p + "mlp_norm"])
        if fam == "dense":
            lin(torch.cat([T[p + "gate"].chunk(tp)[r], T[p + "up"].chunk(tp)[r]]))
            lin(T[p + "down"].chunk(tp, dim=1)[r])
            continue
        out.append(T[p + "router"])
        if fam == "moe_only":
            lin(torch.cat([T[p + "shared.gate"].chunk(tp)[r], T[p + "shared.up"].chunk(tp)[r]]))
            lin(T[p + "shared.down"].chunk(tp, dim=1)[r])
        el = model["num_experts"] // ep
        es = range(ep_i * el, (ep_i + 1) * el)
        lin(torch.stack([torch.cat([T[f"{p}experts.{e}.gate"].chunk(tp)[r], T[f"{p}experts.{e}.up"].chunk(tp)[r]])
                         for e in es]))
        lin(torch.stack([T[f"{p}experts.{e}.down"].chunk(tp, dim=1)[r] for e in es]))
    if fam in ("dense", "mixtral"):
        out.append(T["final_norm"])
        out.append(T["lm_head"].chunk(tp)[r])
    return out


STYLES = {"fsdp_flat": fsdp_flat, "megatron": megatron, "serving": serving}


def ckpt_shapes(model):
    h = model["hidden"]
    fam = model["family"]
    shapes = {}
    for n in _ckpt_names(model):
        leaf = n.split(".")[-1]
        if n in ("embed", "lm_head"):
            s = (model["vocab"], h)
        elif leaf in ("attn_norm", "mlp_norm") or n == "final_norm":
            s = (1, h)
        elif leaf == "q":
            s = (model["num_heads"] * model["head_dim"], h)
        elif leaf in ("k", "v"):
            s = (model["num_kv_heads"] * model["head_dim"], h)
        elif leaf == "o":
            s = (h, model["num_heads"] * model["head_dim"])
        elif leaf == "router":
            s = (model["num_experts"], h)
        elif n.endswith("shared.gate") or n.endswith("shared.up"):
            s = (model["ffn"] * model["num_shared_experts"], h)
        elif n.endswith("shared.down"):
            s = (h, model["ffn"] * model["num_shared_experts"])
        elif leaf in ("gate", "up"):
            s = (model["ffn"], h)
        elif leaf == "down":
            s = (h, model["ffn"])
        else:
            raise KeyError(n)
        shapes[n] = s
    assert fam in ("dense", "mixtral", "moe_only")
    return shapes
