"""Run a workload's steps through the oracle (CPU) or the HIP library (GPU)
from the same initial bytes, and compare."""
from __future__ import annotations

import numpy as np

from oracle import kvx_oracle
from paper_2606_31093_amd.workloads import (normal_bf16_bytes, prefill_bytes, random_bytes,
                                            value_side)


def initial_bytes(wl) -> dict:
    """CPU initial contents: values in the first source side, prefill elsewhere."""
    out = {}
    vs = value_side(wl)
    for name, spec in wl.sides.items():
        if name == vs:
            out[name] = (normal_bf16_bytes(spec.nbytes, wl.value_seed) if spec.e == 2
                         else random_bytes(spec.nbytes, wl.value_seed))
        else:
            pad = (-spec.nbytes) % 8
            out[name] = prefill_bytes(spec.nbytes + pad, wl.prefill_tag)[: spec.nbytes].copy()
    return out


def run_oracle(wl, init: dict, reqs_override=None) -> tuple[dict, list]:
    """Apply every step with the oracle; returns (final bytes, error bits per step)."""
    O = kvx_oracle.default()
    mem = {k: v.copy() for k, v in init.items()}
    errs = []
    for i, st in enumerate(wl.steps):
        reqs = st.reqs if reqs_override is None else reqs_override[i]
        S, D = wl.sides[st.src], wl.sides[st.dst]
        if st.op == "transfer" and st.slice is not None:
            e = O.transfer_slice(mem[st.src], S, mem[st.dst], D, st.slice, st.src_pt, st.dst_pt, reqs)
        elif st.op == "transfer":
            e = O.transfer(mem[st.src], S, mem[st.dst], D, st.src_pt, st.dst_pt, reqs)
        elif st.op == "gather" and st.slice is not None:
            e = O.gather_slice(mem[st.src], S, mem[st.dst], D, st.slice, st.src_pt, reqs)
        elif st.op == "gather":
            e = O.gather(mem[st.src], S, mem[st.dst], D, st.src_pt, reqs)
        elif st.slice is not None:
            e = O.scatter_slice(mem[st.src], S, mem[st.dst], D, st.slice, st.dst_pt, reqs)
        else:
            e = O.scatter(mem[st.src], S, mem[st.dst], D, st.dst_pt, reqs)
        errs.append(e)
    return mem, errs


def run_gpu(wl, init: dict, raw_reqs=None, planned=None, library=None) -> tuple[dict, list]:
    """Apply every step with libkvx on cuda:0.  ``raw_reqs`` may give kvx_req
    record arrays (numpy structured) per step instead of the (n, 6) rows.
    With ``planned``, transfer steps go through kvx_transfer_planned, in
    ``library`` (a build from kvx.load; default the product library), with
    their plan: ``planned`` takes the host plan (int64 array), its pages and
    tokens and returns the three to pass (the same, or altered)."""
    import torch

    from paper_2606_31093_amd import kvx

    dev = torch.device("cuda", 0)
    mem = {}
    for name, arr in init.items():
        t = torch.from_numpy(arr.copy())
        if name in wl.host_sides:
            h = torch.empty(arr.nbytes, dtype=torch.uint8, pin_memory=True)
            h.copy_(t)
            mem[name] = h
        else:
            mem[name] = t.to(dev)
    errs = []
    for i, st in enumerate(wl.steps):
        if raw_reqs is not None:
            reqs = torch.from_numpy(raw_reqs[i].view(np.uint8).copy()).to(dev)
        else:
            reqs = kvx.device_reqs(st.reqs, dev)
        err = torch.zeros(1, dtype=torch.int32, device=dev)
        S, D = wl.sides[st.src], wl.sides[st.dst]
        spt = kvx.device_table(st.src_pt, dev) if st.src_pt is not None else None
        dpt = kvx.device_table(st.dst_pt, dev) if st.dst_pt is not None else None
        if st.op == "transfer" and planned is not None and not st.layer_group:
            buf, pages, tokens = kvx.host_plan(raw_reqs[i] if raw_reqs is not None else st.reqs,
                                               S.T, D.T)
            buf, pages, tokens = planned(buf, pages, tokens)
            kvx.kvx_transfer_planned(mem[st.src], S, mem[st.dst], D, spt, dpt, reqs,
                                     torch.from_numpy(buf).to(dev), pages, tokens, st.slice, err,
                                     library=library)
        elif st.op == "transfer" and st.layer_group:
            n_layers = st.slice[2] if st.slice is not None else S.L
            events = [torch.cuda.Event() for _ in range(-(-n_layers // st.layer_group))]
            if planned is not None:
                buf, pages, tokens = planned(*kvx.host_plan(
                    raw_reqs[i] if raw_reqs is not None else st.reqs, S.T, D.T))
                kvx.kvx_transfer_layered_planned(mem[st.src], S, mem[st.dst], D, spt, dpt, reqs,
                                                 st.layer_group, events, torch.from_numpy(buf).to(dev),
                                                 pages, tokens, st.slice, err, library=library)
            else:
                kvx.kvx_transfer_layered(mem[st.src], S, mem[st.dst], D, spt, dpt, reqs,
                                         st.layer_group, events, st.slice, err)
        elif st.op == "transfer" and st.slice is not None:
            kvx.kvx_transfer_slice(mem[st.src], S, mem[st.dst], D, st.slice, spt, dpt, reqs, err)
        elif st.op == "transfer":
            kvx.kvx_transfer(mem[st.src], S, mem[st.dst], D, spt, dpt, reqs, err)
        elif st.op == "gather" and st.slice is not None:
            kvx.kvx_gather_slice(mem[st.src], S, mem[st.dst], D, st.slice, spt, reqs, err)
        elif st.op == "gather":
            kvx.kvx_gather(mem[st.src], S, mem[st.dst], D, spt, reqs, err)
        elif st.slice is not None:
            kvx.kvx_scatter_slice(mem[st.src], S, mem[st.dst], D, st.slice, dpt, reqs, err)
        else:
            kvx.kvx_scatter(mem[st.src], S, mem[st.dst], D, dpt, reqs, err)
        torch.cuda.synchronize()
        errs.append(int(err.item()) & 0xFFFFFFFF)
    out = {k: v.cpu().numpy() for k, v in mem.items()}
    return out, errs


def assert_same(got: dict, want: dict, what: str = "") -> None:
    for name in want:
        a, b = got[name], want[name]
        if not np.array_equal(a, b):
            bad = np.nonzero(a != b)[0]
            raise AssertionError(f"{what} side {name}: {len(bad)} of {a.size} bytes differ; "
                                 f"first offsets {bad[:8].tolist()}")

