"""The allocation-free decode entry point (the library's fixed partial-result
array instead of a caller workspace) against parrot_shared_prefix_decode on
the same inputs: two calls in a row, the second with a smaller batch, each
bitwise equal to the workspace entry point and within the oracle bar."""
import math
import sys

import numpy as np
import pytest
import torch

from gpu_util import assert_close, oracle_for, problem_for, run_gpu, to_np
from workloads import build_plan, get_config, make_batch, make_plan

pytestmark = pytest.mark.gpu


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def _noalloc(plan, dev):
    from paper_2405_19888_amd import parrot_shared_prefix_decode_noalloc
    R, H, D = plan.num_requests, plan.heads, plan.head_dim
    out = torch.full((R, H, D), float("nan"), dtype=dev["q"].dtype, device="cuda")
    lse = torch.full((R, H), float("nan"), dtype=torch.float32, device="cuda")
    parrot_shared_prefix_decode_noalloc(
        problem_for(plan), dev["q"], dev["k_pool"], dev["v_pool"], dev["k_pool"], dev["v_pool"],
        dev["prefix_tables"], dev["prefix_lens"], dev["suffix_tables"], dev["suffix_lens"],
        dev["group_ids"], out, lse)
    torch.cuda.synchronize()
    return out, lse


def _small_plan():
    rng = np.random.default_rng(3)
    return build_plan(heads=4, head_dim=128, block_size=16, dtype="float16",
                      group_of_request=[0, 0, 1, -1, 1, 0], prefix_lens=[300, 17],
                      suffix_lens=[5, 0, 140, 33, 16, 260], sm_scale=1 / math.sqrt(128),
                      shuffle=True, rng=rng)


def test_noalloc_matches_workspace_entry_twice():
    """C2 (LLaMA-7B layer, 1 x 32, P = 2048), then a 6-request batch: the
    second call reuses the array the first one filled."""
    for name, plan in (("llama7b_g32_p2048", make_plan(get_config("c2"))),
                       ("small mixed batch", _small_plan())):
        say("noalloc", name)
        batch = make_batch(plan, seed=9)
        dev = batch.to("cuda")
        ref_out, ref_lse = run_gpu(plan, dev, shared=True)
        ref_out, ref_lse = ref_out.clone(), ref_lse.clone()
        out, lse = _noalloc(plan, dev)
        assert torch.equal(out, ref_out) and torch.equal(lse, ref_lse), name
        assert_close(*to_np(out, lse), *oracle_for(batch, plan), plan.dtype, f"noalloc {name}")


def test_noalloc_rejects_batches_above_the_array():
    """A call whose partial results exceed the fixed array is refused before
    any launch, with the workspace error."""
    from paper_2405_19888_amd import ParrotError, parrot_shared_prefix_decode_noalloc
    from paper_2405_19888_amd.binding import PARROT_ERR_WORKSPACE_TOO_SMALL
    say("noalloc too large")
    plan = make_plan(get_config("c5"))
    prob = problem_for(plan)
    z = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    zi = torch.zeros(16, dtype=torch.int32, device="cuda")
    zf = torch.zeros(16, dtype=torch.float32, device="cuda")
    with pytest.raises(ParrotError, match="fixed array") as e:
        parrot_shared_prefix_decode_noalloc(prob, z, z, z, z, z, zi, zi, zi, zi, zi, z, zf)
    assert e.value.status == PARROT_ERR_WORKSPACE_TOO_SMALL
