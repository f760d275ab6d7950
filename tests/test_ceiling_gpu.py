"""The read-bandwidth probe (parrot_hbm_read_ceiling) reads every 16-byte
piece of its buffer exactly once: its XOR fold equals the XOR of all words
computed on the host, for every launch shape it supports, including sizes
that leave a ragged tail for the unrolled loop."""
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
