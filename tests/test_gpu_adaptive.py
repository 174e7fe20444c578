"""GPU parity with a per-layer window size: the adaptive compression ratio
across layers that the paper names as future work (Sec. VI).

Every layer's pooling, prefill and decode run through the library with that
layer's own window, so each layer's cache has its own compressed length.  The
60 s stack (b=64) with windows 2/4/8 by depth is checked on sampled outputs
against the oracle at each layer's window; a layer of it must also give the
same bits as the same layer of a stack with that window everywhere.
"""
import pytest
import torch

from helpers import TOL, f64, gather
from paper_2607_06827_amd import inputs
from paper_2607_06827_amd.workload import Job
from test_gpu_workloads import assert_ok, check_decode, check_pool, check_prefill

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

LAYERS = [0, 13, 14, 17, 18, 23, 24, 27]


def test_adaptive_stack_sampled():
    wl = inputs.ADAPTIVE_W_60S
    job = Job(wl, layers=LAYERS, keep_decode=True)
    for i, l in enumerate(LAYERS):
        w = wl.window(l) if l >= wl.l0 else 1
        assert job.prefill_clen[i] == wl.prefix_len + -(-wl.speech_len // w)
    errs = []
    for l in (13, 14, 18, 27):
        job.run_prefill(layers=[l])
        torch.cuda.synchronize()
        check_prefill(job, job.layers.index(l), [7, 50], errs)
    job.run()
    torch.cuda.synchronize()
    for i in range(len(LAYERS)):
        assert int(job.cache_len_out[i][0]) == job.prefill_clen[i]
        for b in (0, 41):
            check_decode(job, i, b, (0, 127), errs)
        check_pool(job, i, [41], errs)
    assert_ok(errs, TOL["bf16"], wl.name)


@pytest.mark.parametrize("layer", [17, 23, 27])
def test_adaptive_layer_matches_uniform(layer):
    """A layer depends only on its own window: its cache and decode outputs
    equal, bit for bit, those of the same layer in a stack whose every
    compressed layer uses that window."""
    wl = inputs.ADAPTIVE_W_60S
    a = Job(wl, layers=[layer], keep_decode=True)
    u = Job(inputs.STACK_60S.with_(w=wl.window(layer)), layers=[layer], keep_decode=True,
            share_inputs=a)
    a.run()
    u.run()
    torch.cuda.synchronize()
    assert a.prefill_clen == u.prefill_clen
    L = a.prefill_clen[0] + wl.decode_steps
    for b in (0, 63):
        ka, va = gather(a.caches[0], b, L)
        ku, vu = gather(u.caches[0], b, L)
        assert torch.equal(ka, ku) and torch.equal(va, vu)
    assert torch.equal(a.decode_out, u.decode_out)
    assert torch.equal(a.prefill_out, u.prefill_out)
