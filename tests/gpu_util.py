"""Helpers for the GPU tests: run the HIP library on a workload and compare
with the oracle at the stated tolerances.  No attention arithmetic here."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2405_19888_amd import (Decoder, parrot_validate_inputs, parrot_validate_nested_inputs,
                                  problem_from_host)
from workloads.gen import TORCH_DTYPES

# Tolerances: max |out_gpu - out_ref| over all elements (fp32-accumulated
# results of fp16 / fp32 inputs 2e-3, bf16 inputs 8e-3); lse relative error
# |d| / max(1, |ref|) <= 1e-4.  fp32 inputs also meet a tighter 1e-5.
OUT_TOL = {"float16": 2e-3, "bfloat16": 8e-3, "float32": 2e-3}
OUT_TOL_INTERNAL = {"float32": 1e-5}
LSE_RTOL = 1e-4
# A second, internal bar on the whole output: ||out - ref||_2 / ||ref||_2.  It
# sees a systematic error spread thinly over many elements (a dropped key in
# every row, a biased rounding) that the max-abs bar lets through.
REL_L2 = {"float16": 2e-3, "bfloat16": 1e-2, "float32": 1e-5}


def problem_for(plan, num_prefix_blocks=None, num_suffix_blocks=None):
    return problem_from_host(
        num_heads=plan.heads, head_dim=plan.head_dim, block_size=plan.block_size,
        dtype=TORCH_DTYPES[plan.dtype], sm_scale=plan.sm_scale, group_ids=plan.group_ids,
        prefix_lens=plan.prefix_lens, suffix_lens=plan.suffix_lens,
        prefix_table_stride=plan.prefix_tables.shape[1],
        suffix_table_stride=plan.suffix_tables.shape[1],
        num_prefix_blocks=num_prefix_blocks or plan.num_blocks,
        num_suffix_blocks=num_suffix_blocks or plan.num_blocks,
        prefix_parents=plan.prefix_parents if plan.nested else None)


def run_gpu(plan, dev: dict, shared: bool = True, problem=None, poison: bool = True,
            decoder: Decoder = None, nested: bool = None):
    """Validate inputs on the device, poison outputs and workspace, run, sync.
    Nested plans go through the nested-group entry point (unless `nested` is
    False: then the groups are taken as flat)."""
    nested = plan.nested if nested is None else nested
    prob = problem or problem_for(plan)
    dec = decoder or Decoder(prob)
    scratch = torch.zeros(16, dtype=torch.int32, device="cuda")
    if nested:
        parrot_validate_nested_inputs(prob, dev["prefix_tables"], dev["prefix_lens"],
                                      dev["prefix_parents"], dev["suffix_tables"],
                                      dev["suffix_lens"], dev["group_ids"], scratch)
    else:
        parrot_validate_inputs(prob, dev["prefix_tables"], dev["prefix_lens"],
                               dev["suffix_tables"], dev["suffix_lens"], dev["group_ids"], scratch)
    if poison:
        dec.out.fill_(float("nan"))
        dec.lse.fill_(float("nan"))
        dec.workspace.fill_(0xFF)          # every float slot reads as NaN
    out, lse = dec(dev, shared=shared, nested=nested)
    torch.cuda.synchronize()
    return out, lse


def to_np(out, lse):
    return out.detach().double().cpu().numpy(), lse.detach().double().cpu().numpy()


def oracle_for(batch_like, plan, requests=None, pools=None):
    """The oracle on a batch (host tensors) or on device pools (gathered blocks only)."""
    q = batch_like["q"] if isinstance(batch_like, dict) else batch_like.q
    kp = pools[0] if pools else batch_like.k_pool
    vp = pools[1] if pools else batch_like.v_pool
    return oracle.shared_prefix_decode(
        q.cpu() if isinstance(q, torch.Tensor) else q, kp, vp, kp, vp, plan.prefix_tables,
        plan.prefix_lens, plan.suffix_tables, plan.suffix_lens, plan.group_ids, plan.sm_scale,
        requests=requests, prefix_parents=plan.prefix_parents if plan.nested else None)


def assert_close(out, lse, ref_out, ref_lse, dtype: str, what: str = "", out_tol=None,
                 rel_l2=None):
    """Element-wise comparison with the oracle; ``out_tol`` / ``rel_l2``
    replace the dtype's internal bars for inputs whose logits are far from unit
    scale (the caller states the derivation)."""
    out = np.asarray(out, dtype=np.float64)
    lse = np.asarray(lse, dtype=np.float64)
    assert np.all(np.isfinite(out)), f"{what}: non-finite output"
    assert np.all(np.isfinite(lse)), f"{what}: non-finite lse"
    err = np.max(np.abs(out - ref_out)) if out.size else 0.0
    lerr = np.max(np.abs(lse - ref_lse) / np.maximum(1.0, np.abs(ref_lse))) if lse.size else 0.0
    tol = out_tol if out_tol is not None else OUT_TOL_INTERNAL.get(dtype, OUT_TOL[dtype])
    assert err <= tol, f"{what}: max |out err| {err:.3e} > {tol:.1e}"
    assert lerr <= LSE_RTOL, f"{what}: max lse rel err {lerr:.3e} > {LSE_RTOL:.0e}"
    ref_norm = float(np.linalg.norm(ref_out))
    if ref_norm > 0.0:
        rel = float(np.linalg.norm(out - ref_out)) / ref_norm
        bar = rel_l2 if rel_l2 is not None else REL_L2[dtype]
        assert rel <= bar, f"{what}: relative L2 of out {rel:.3e} > {bar:.0e}"
    return err, lerr


def prefill_rows_for(plan, offsets):
    from paper_2405_19888_amd import prefill_rows_from_host
    return prefill_rows_from_host(offsets, plan.group_ids, plan.num_groups,
                                  plan.prefix_parents if plan.nested else None)


def run_prefill(plan, dev: dict, offsets, problem=None, rows=None, poison: bool = True,
                nested: bool = None, keep: list = None):
    """Validate the prefill inputs on the device, poison outputs and
    workspace, run the prefill entry point, sync.  `keep` (a list) receives
    the Prefiller, whose workspace shows which path ran: the single pass
    writes none of it."""
    from paper_2405_19888_amd import Prefiller, parrot_validate_prefill_inputs
    nested = plan.nested if nested is None else nested
    prob = problem or problem_for(plan)
    rows = rows or prefill_rows_for(plan, offsets)
    pre = Prefiller(prob, rows)
    scratch = torch.zeros(16, dtype=torch.int32, device="cuda")
    parrot_validate_prefill_inputs(prob, rows, dev["query_offsets"], dev["prefix_tables"],
                                   dev["prefix_lens"], dev["prefix_parents"] if nested else None,
                                   dev["suffix_tables"], dev["suffix_lens"], dev["group_ids"],
                                   scratch)
    if poison:
        pre.out.fill_(float("nan"))
        pre.lse.fill_(float("nan"))
        pre.workspace.fill_(0xFF)
    out, lse = pre(dev, nested=nested)
    torch.cuda.synchronize()
    if keep is not None:
        keep.append(pre)
    return out, lse


def workspace_untouched(pre) -> bool:
    """True when no byte of the prefill workspace changed from the 0xFF poison."""
    return bool(torch.all(pre.workspace.view(torch.uint8) == 0xFF).item())


def oracle_prefill_for(batch, plan, q_rows, offsets, rows=None, pools=None):
    kp = pools[0] if pools else batch.k_pool
    vp = pools[1] if pools else batch.v_pool
    return oracle.shared_prefix_prefill(
        q_rows.cpu(), offsets, kp, vp, kp, vp, plan.prefix_tables, plan.prefix_lens,
        plan.suffix_tables, plan.suffix_lens, plan.group_ids, plan.sm_scale, rows=rows,
        prefix_parents=plan.prefix_parents if plan.nested else None)
