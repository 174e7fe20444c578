"""The synthetic inputs have the structure the workloads call for."""
import math

import numpy as np
import pytest
import torch

from paper_2607_06827_amd import inputs


def test_ar1_matches_its_recursion():
    eps = torch.randn(3, 200, 5, generator=torch.Generator().manual_seed(0))
    rho = 0.9
    x = inputs.ar1(eps, rho, chunk=16).double()
    ref = torch.empty_like(x)
    ref[:, 0] = eps[:, 0].double()
    c = math.sqrt(1 - rho * rho)
    for t in range(1, 200):
        ref[:, t] = rho * ref[:, t - 1] + c * eps[:, t].double()
    assert torch.allclose(x, ref, atol=1e-4)


def test_speech_frames_are_locally_redundant():
    """Adjacent speech frames correlate at about rho (the local similarity
    the paper measures between adjacent speech positions), text does not."""
    wl = inputs.LAYER_30S.with_(batch=4)
    k, v = inputs.raw_kv(wl, layer=0)
    P, T = wl.prefix_len, wl.speech_len
    sp = k[:, P:P + T].float().reshape(4, T, -1)
    a, b = sp[:, :-1].reshape(-1), sp[:, 1:].reshape(-1)
    corr = float(torch.corrcoef(torch.stack([a, b]))[0, 1])
    assert abs(corr - wl.rho) < 0.01
    assert abs(float(sp.std()) - 1.0) < 0.02
    tx = k[:, :P].float().reshape(4, P, -1)
    corr_t = float(torch.corrcoef(torch.stack([tx[:, :-1].reshape(-1), tx[:, 1:].reshape(-1)]))[0, 1])
    assert abs(corr_t) < 0.02
    assert k.dtype == torch.bfloat16 and k.shape == (4, P + T, 8, 128)


def test_inputs_are_seeded_and_streams_independent():
    wl = inputs.TINY_F32
    k1, v1 = inputs.raw_kv(wl, 0)
    k2, v2 = inputs.raw_kv(wl, 0)
    assert torch.equal(k1, k2) and torch.equal(v1, v2)
    assert not torch.equal(k1, v1)
    k3, _ = inputs.raw_kv(wl, 1)
    assert not torch.equal(k1, k3)
    assert not torch.equal(inputs.decode_q(wl, 0, 0), inputs.decode_q(wl, 0, 1))
    u = inputs.gate(wl, 0)
    assert u.dtype == torch.float32 and u.shape == (2, 64)
    assert abs(float(u.std()) * math.sqrt(64) - 1.0) < 0.2
    assert not inputs.gate(wl, 0, scale=0.0).any()


def test_bf16_rounding_happens_once():
    wl = inputs.LAYER_30S.with_(batch=2)
    q = inputs.prefill_q(wl, 0)
    assert q.dtype == torch.bfloat16
    assert torch.equal(q, q.float().to(torch.bfloat16))


def test_block_table_is_a_permutation():
    bt, total = inputs.block_table(4, 7, seed=3, spare_pages=5)
    assert bt.shape == (4, 7) and total == 33
    flat = bt.reshape(-1).numpy()
    assert len(set(flat.tolist())) == 28 and flat.min() >= 0 and flat.max() < 33
    ident, _ = inputs.block_table(2, 3, seed=3, shuffle=False)
    assert ident.reshape(-1).tolist() == list(range(6))


def test_workload_shapes():
    assert [w.prefill_len for w in inputs.WORKLOADS] == [68, 407, 782, 7532, 1596]
    assert inputs.PREFILL_1500.prefix_len + inputs.PREFILL_1500.speech_len + inputs.PREFILL_1500.suffix_len == 1596
    assert np.all([w.num_q_heads % w.num_kv_heads == 0 for w in inputs.WORKLOADS])


def test_per_layer_windows():
    wl = inputs.ADAPTIVE_W_60S
    assert [wl.window(l) for l in (13, 14, 17, 18, 23, 24, 27)] == [1, 2, 2, 4, 4, 8, 8]
    assert inputs.STACK_60S.window(20) == inputs.STACK_60S.w
    with pytest.raises(ValueError):
        inputs.STACK_60S.with_(w_layers=(4,) * 27)
    with pytest.raises(ValueError):
        inputs.STACK_60S.with_(w_layers=(0,) + (4,) * 27)
