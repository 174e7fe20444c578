"""GPU parity on the five synthetic workloads, at their full sizes.

tiny fp32 (1 layer, b=1), 30 s layer (b=32) and prefill (b=8, 1596 queries
over 471 keys) are checked on every output; the 28-layer 60 s stack (b=64) and
the 10-minute decode (b=16, w in {2,4,8}) are run whole, in the launch
configuration the benchmark times, and checked on sampled (layer, step,
sequence) outputs the oracle computes one by one; the 10-minute prefill
(7532 rows) on two whole sequences of a full and a pooled layer.

Each check is helpers.fwd_err (the per-element bound plus each vector's scale
and bias).  Beside it every workload prints the worst RMS-only figure
(max |x - ref| / rms(ref) per vector) and the tensor-wide one
(max |x - ref| / rms(ref) over a whole checked tensor), which are reported,
not gated, for bf16 (fp32 is gated by the RMS-only form).
"""
import numpy as np
import pytest
import torch

import oracle
from helpers import (TOL, f64, fwd_err, fwd_parts, gather, oracle_decode_for, oracle_pool_for,
                     oracle_prefill_for, rms_err, tensor_err)
from paper_2607_06827_amd import inputs
from paper_2607_06827_amd.workload import Job

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def record(errs, kind, layer, where, x, ref, dtype):
    """One parity check: (kind, layer, where, fwd_err, parts, rms-only,
    tensor-wide)."""
    parts = fwd_parts(x, ref, dtype)
    errs.append((kind, layer, where, fwd_err(x, ref, dtype), parts, rms_err(x, ref),
                 tensor_err(x, ref)))


def check_pool(job, i, bs, errs):
    for b in bs:
        kh, vh, clen = oracle_pool_for(job, i, b)
        L = int(clen[0])
        gk, gv = gather(job.caches[i], b, L)
        record(errs, "pool_k", job.layers[i], b, f64(gk), kh[0, :L], job.wl.dtype)
        record(errs, "pool_v", job.layers[i], b, f64(gv), vh[0, :L], job.wl.dtype)


def check_prefill(job, i, bs, errs):
    ref, ref_lse = oracle_prefill_for(job, i, bs)
    R = job.wl.prefill_len
    got = f64(job.prefill_out[bs])
    record(errs, "prefill", job.layers[i], tuple(bs), got[:, :R], ref[:, :R], job.wl.dtype)


def check_decode(job, i, b, steps, errs):
    pooled = oracle_pool_for(job, i, b)
    for s in steps:
        ref, _ = oracle_decode_for(job, i, b, s, pooled)
        got = f64(job.decode_out_at(i, s)[b])
        record(errs, "decode", job.layers[i], (b, s), got, ref, job.wl.dtype)


def assert_ok(errs, tol, name):
    worst = max(errs, key=lambda e: e[3])
    print(f"{name}: {len(errs)} checks, worst {worst[:4]} {worst[4]}", flush=True)
    for kind in sorted({e[0] for e in errs}):
        es = [e for e in errs if e[0] == kind]
        print(f"{name} {kind}: fwd_err {max(e[3] for e in es):.3e} element "
              f"{max(e[4]['elem'] for e in es):.3e} scale {max(e[4]['scale'] for e in es):.2e} "
              f"bias {max(e[4]['bias'] for e in es):.2e} per-head scale "
              f"{max(e[4]['group_scale'] for e in es):.1e} bias {max(e[4]['group_bias'] for e in es):.1e} "
              f"rms-only {max(e[5] for e in es):.3e} "
              f"tensor-wide {max(e[6] for e in es):.3e}", flush=True)
    bad = [e[:4] for e in errs if not e[3] <= tol]
    assert not bad, f"{name}: {len(bad)} checks above {tol}: {bad[:8]}"


def test_tiny_fp32_everything():
    wl = inputs.TINY_F32
    job = Job(wl, keep_decode=True)
    job.run()
    torch.cuda.synchronize()
    errs = []
    check_pool(job, 0, [0], errs)
    check_prefill(job, 0, [0], errs)
    check_decode(job, 0, 0, range(wl.decode_steps), errs)
    assert_ok(errs, TOL["f32"], wl.name)


def test_layer_30s_everything():
    wl = inputs.LAYER_30S
    job = Job(wl, keep_decode=True)
    job.run()
    torch.cuda.synchronize()
    errs = []
    bs = list(range(wl.batch))
    check_pool(job, 0, bs, errs)
    check_prefill(job, 0, bs, errs)
    # every decode step of every sequence, batched through the oracle
    kh, vh, clen = oracle.pool(f64(job.k_raw[0]), f64(job.v_raw[0]), [wl.prefix_len] * wl.batch,
                               [wl.speech_len] * wl.batch, [0] * wl.batch, wl.w, 0, job.l0,
                               f64(job.gate[0]))
    L0 = int(clen[0])
    K = np.concatenate([kh[:, :L0], f64(job.k_new[0]).transpose(1, 0, 2, 3)], axis=1)
    V = np.concatenate([vh[:, :L0], f64(job.v_new[0]).transpose(1, 0, 2, 3)], axis=1)
    for s in range(wl.decode_steps):
        ref, _ = oracle.decode(f64(job.q_dec[0][s]), K, V, [L0 + s + 1] * wl.batch, job.scale)
        record(errs, "decode", 0, s, f64(job.decode_out_at(0, s)), ref, "bf16")
    assert_ok(errs, TOL["bf16"], wl.name)


def test_prefill_1500_everything():
    wl = inputs.PREFILL_1500
    job = Job(wl)
    job.run()
    torch.cuda.synchronize()
    errs = []
    bs = list(range(wl.batch))
    check_pool(job, 0, bs, errs)
    assert job.prefill_clen[0] == 471
    check_prefill(job, 0, bs, errs)
    assert_ok(errs, TOL["bf16"], wl.name)


def test_stack_60s_sampled():
    wl = inputs.STACK_60S
    job = Job(wl, keep_decode=True)
    errs = []
    # prefill outputs share one buffer across layers: check a few layers as they run
    for l in (0, 13, 14, 27):
        job.run_prefill(layers=[l])
        torch.cuda.synchronize()
        check_prefill(job, job.layers.index(l), [5], errs)
    job.run()
    torch.cuda.synchronize()
    for i in range(wl.num_layers):
        for b in (0, 37, 63):
            check_decode(job, i, b, (0, 63, 127), errs)
        check_pool(job, i, [37], errs)
    assert_ok(errs, TOL["bf16"], wl.name)


@pytest.mark.parametrize("w", [2, 4, 8])
def test_long_10min_sampled(w):
    wl = inputs.LONG_10MIN.with_(w=w)
    job = Job(wl, layers=[0, 13, 14, 27], with_prefill=False, keep_decode=True)
    job.run()
    torch.cuda.synchronize()
    errs = []
    for i in range(len(job.layers)):
        for b in (0, 9, 15):
            check_decode(job, i, b, (0, 127, 255), errs)
        check_pool(job, i, [9], errs)
    assert_ok(errs, TOL["bf16"], f"{wl.name}-w{w}")


def test_long_10min_prefill_sampled():
    """Prefill at the 10-minute workload's full size (b=16, 32 + 7500 rows,
    w=4): a full layer (7532 keys, causal) and a pooled layer (1907 keys), in
    the launch configuration the benchmark uses, checked on two whole
    sequences against the oracle."""
    wl = inputs.LONG_10MIN.with_(decode_steps=0)
    job = Job(wl, layers=[0, 14])
    errs = []
    for l in (0, 14):
        job.run_prefill(layers=[l])
        torch.cuda.synchronize()
        check_prefill(job, job.layers.index(l), [0, 15], errs)
        check_pool(job, job.layers.index(l), [15], errs)
    assert_ok(errs, TOL["bf16"], f"{wl.name}-prefill")
