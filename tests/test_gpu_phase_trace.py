"""The phase-trace build (libcompkv_trace.so, compkv_phase_trace_set): its fused step computes exactly what
the normal library computes, and its records are well formed (every workgroup of both launches stamped,
in order, with a known role). The normal library refuses the trace."""
import numpy as np
import pytest
import torch

import paper_2609_26300_amd as P
import paper_2609_26300_amd.binding as B
from paper_2609_26300_amd import build as lib_build
from gpu_case import make_case

pytestmark = pytest.mark.gpu


def test_normal_library_refuses_the_trace():
    with pytest.raises(P.CompkvError):
        P.compkv_phase_trace_set(None, None)


@pytest.mark.parametrize("name", ["tiny_4k", "llama8b_32k", "long_16k_b8"])
def test_traced_step_matches_and_stamps_every_workgroup(name):
    c = make_case(name, "chunked_exact")
    print(f"\n[phase trace {name}]", flush=True)
    c.build_stats()
    ref = c.decode_step()
    torch.cuda.synchronize()
    rec1 = torch.zeros(1 << 18, dtype=torch.int64, device="cuda")
    rec2 = torch.zeros(1 << 18, dtype=torch.int64, device="cuda")
    saved = (B._lib, B.LIB_PATH)
    try:
        B._lib, B.LIB_PATH = None, lib_build.TRACE_LIB
        P.compkv_phase_trace_set(rec1, rec2)
        got = c.decode_step()
        torch.cuda.synchronize()
        P.compkv_phase_trace_set(None, None)
    finally:
        B._lib, B.LIB_PATH = saved
    for k in ("sel", "n_sel", "blk_logit", "out", "lse"):
        assert torch.equal(got[k], ref[k]), k
    units = c.dims.batch * c.dims.n_kv_heads
    for rec, roles in ((rec1, (1, 2)), (rec2, (1, 2))):
        r = rec.cpu().numpy().view(np.uint64).reshape(-1, 16)
        r = r[r[:, 15] != 0]
        assert len(r) >= 2 * units
        assert set(np.unique(r[:, 1]).tolist()) <= set(roles)
        assert np.all(r[:, 0] <= r[:, 15])
        for s in range(2, 14):  # every stamped phase lies between the workgroup's start and end (14 holds its placement)
            m = r[:, s] != 0
            assert np.all((r[m, s] >= r[m, 0]) & (r[m, s] <= r[m, 15])), s
    a = rec1.cpu().numpy().view(np.uint64).reshape(-1, 16)
    b = rec2.cpu().numpy().view(np.uint64).reshape(-1, 16)
    a, b = a[a[:, 15] != 0], b[b[:, 15] != 0]
    assert np.sum(a[:, 1] == 2) == units  # one last-block workgroup per unit
    assert a[:, 15].max() <= b[:, 0].min()  # the fused launch starts after the chunk launch ends
