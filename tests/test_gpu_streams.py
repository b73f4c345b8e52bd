"""Calls on different streams: every call uses the library's one workspace, so
switching streams must order the new stream after the work already queued on
the previous one.  Two DGEMMs queued back to back on two torch streams (default
priority) must give the bits each gives alone."""
import numpy as np
import pytest
import torch

import seeded_inputs as S

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def emu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_04663_amd as E
    E.lib()
    return E


def test_two_streams_share_the_workspace_in_order(emu):
    n = 2048
    A1 = torch.from_numpy(S.make("uniform", 951, (n, n), np.float64)).cuda()
    B1 = torch.from_numpy(S.make("uniform", 952, (n, n), np.float64)).cuda()
    A2 = torch.from_numpy(S.make("wide", 953, (n, n), np.float64)).cuda()
    B2 = torch.from_numpy(S.make("wide", 954, (n, n), np.float64)).cuda()
    ref1 = emu.dgemm(A1, B1, 21).clone()
    ref2 = emu.dgemm(A2, B2, 6).clone()
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    C1 = torch.empty_like(ref1)
    C2 = torch.empty_like(ref2)
    torch.cuda.synchronize()
    for _ in range(3):
        with torch.cuda.stream(s1):
            emu.dgemm(A1, B1, 21, C=C1)         # long call
        with torch.cuda.stream(s2):
            emu.dgemm(A2, B2, 6, C=C2)          # would overwrite the planes C1 reads
        torch.cuda.synchronize()
        assert torch.equal(C1, ref1) and torch.equal(C2, ref2)
    emu.lib().emu_set_stream(None)
