"""The measuring probes behind the bench's practical ceilings run to completion
and write nothing (their sink keeps its value); they compute nothing of the
method, so there is no oracle to compare with."""

import pytest
import torch

from paper_2606_21848_amd import binding as kb
from tests.parity import say

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("nbytes,workgroups", [(16, 1), (4096, 3), (1 << 20, 1024), ((1 << 24) + 48, 8192)])
def test_probe_read_runs_and_writes_nothing(lib, nbytes, workgroups):
    say(f"probe_read bytes={nbytes} workgroups={workgroups}")
    buf = torch.zeros(nbytes // 4, dtype=torch.int32, device=DEV)  # folds to zero: no store
    sink = torch.full((1,), 7, dtype=torch.int32, device=DEV)
    kb.probe_read(buf, sink, workgroups)
    torch.cuda.synchronize()
    assert int(sink.item()) == 7


@pytest.mark.parametrize("iters,workgroups", [(1, 1), (50, 256)])
def test_probe_mfma_runs_and_writes_nothing(lib, iters, workgroups):
    say(f"probe_mfma iters={iters} workgroups={workgroups}")
    sink = torch.full((1,), 3.0, dtype=torch.float32, device=DEV)
    flop = kb.probe_mfma(sink, iters, workgroups)
    torch.cuda.synchronize()
    assert float(sink.item()) == 3.0
    assert flop == workgroups * 4 * iters * 16 * 16 * 16 * 32 * 2
