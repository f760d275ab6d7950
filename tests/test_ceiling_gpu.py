"""The measurement aids.  The read-bandwidth probe (parrot_hbm_read_ceiling)
reads every 16-byte piece of its buffer exactly once: its XOR fold equals the
XOR of all words computed on the host, for every launch shape it supports,
including sizes that leave a ragged tail for the unrolled loop.  The
matrix-core issue probe (parrot_mfma_issue_ceiling) runs for every vector
share it is built for."""
import sys

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("spans", [False, True], ids=["grid_stride", "wave_spans"])
@pytest.mark.parametrize("n16", [1, 7, 64, 4096 + 3, 3 * 256 * 16 + 5, 1 << 20])
@pytest.mark.parametrize("loads", [4, 8, 16])
def test_read_probe_folds_every_word(n16, loads, spans):
    from paper_2405_19888_amd import parrot_hbm_read_ceiling
    print("[case] read probe", n16, "pieces,", loads, "loads per thread, spans", spans, flush=True)
    sys.stdout.flush()
    rng = np.random.default_rng(n16 + loads)
    words = rng.integers(0, 2 ** 32, size=4 * n16, dtype=np.uint64).astype(np.uint32)
    buf = torch.from_numpy(words.view(np.int32)).to("cuda")
    expect = int(np.bitwise_xor.reduce(words))
    for workgroups in (1, 3, 256):
        sink = torch.zeros(1, dtype=torch.int32, device="cuda")
        parrot_hbm_read_ceiling(buf, sink, workgroups, loads, wave_spans=spans)
        torch.cuda.synchronize()
        got = int(sink.cpu().numpy().view(np.uint32)[0])
        assert got == expect, (n16, loads, workgroups, spans)


@pytest.mark.parametrize("valu_x4", [0, 8, 10, 11, 12, 16])
def test_mfma_issue_probe_runs_and_is_deterministic(valu_x4):
    """The matrix-core issue probe completes for every vector share it is built
    for, on a partial and a full grid, and folds the same value on two runs of
    the same shape (registers only: the result depends on nothing else)."""
    from paper_2405_19888_amd import ParrotTrace, parrot_mfma_issue_ceiling
    print("[case] mfma issue probe, valu_x4", valu_x4, flush=True)
    for workgroups, iters in ((3, 17), (256, 64)):
        sinks = []
        for _ in range(2):
            sink = torch.zeros(1, dtype=torch.int32, device="cuda")
            e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            for x in e:
                x.record()
            torch.cuda.synchronize()
            parrot_mfma_issue_ceiling(sink, workgroups, iters, valu_x4,
                                      trace=ParrotTrace(*[x.cuda_event for x in e]))
            torch.cuda.synchronize()
            assert e[0].elapsed_time(e[1]) > 0.0
            sinks.append(int(sink.item()))
        assert sinks[0] == sinks[1], (valu_x4, workgroups, iters)
