"""GPU checks of the HIP graph cache on an MSA-row-attention step
(LayerNorm + projections, pair bias, attention, output projection, and the
backward of all of them).

* a replayed graph gives bitwise the results of the same step run eagerly
  (every kernel is deterministic), over several replays with new input
  values copied into the static buffers between them and eager work and
  synchronisations in between;
* one capture per key; a second shape gets its own graph; with capacity 1
  the older graph is evicted and captured again when its key returns.
"""
import pytest
import torch

from paper_2404_11068_amd import graph as gr

pytestmark = pytest.mark.gpu


def _snapshot(step):
    return {k: v.detach().clone() for k, v in step.outputs().items()}


def test_replay_matches_eager_over_new_inputs():
    s = torch.cuda.Stream()
    step = gr.MSARowAttentionStep(N=4, L=64, seed=1)
    cache = gr.GraphCache(capacity=4)
    gen = torch.Generator(device="cpu").manual_seed(7)
    for it in range(4):
        print("\n[case] replay", it, flush=True)
        if it:
            step.m.copy_(torch.randn(step.m.shape, generator=gen).to(torch.bfloat16))
            step.z.copy_(torch.randn(step.z.shape, generator=gen).to(torch.bfloat16))
            step.d_m_out.copy_(torch.randn(step.d_m_out.shape, generator=gen).to(torch.bfloat16))
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            step.record(s)
        torch.cuda.synchronize()
        eager = _snapshot(step)
        for v in step.outputs().values():
            v.zero_()
        torch.cuda.synchronize()
        captured = cache.run(step.key(), step.record, s)
        assert captured == (it == 0)
        torch.cuda.synchronize()
        for k, v in step.outputs().items():
            assert torch.equal(v, eager[k]), (it, k)
        _ = torch.randn(1000, device="cuda").sum()  # unrelated eager work between replays
    assert len(cache) == 1 and cache.captures == 1


def test_keys_and_eviction():
    s = torch.cuda.Stream()
    a = gr.MSARowAttentionStep(N=2, L=32, seed=2)
    b = gr.MSARowAttentionStep(N=3, L=64, seed=3)
    cache = gr.GraphCache(capacity=2)
    assert cache.run(a.key(), a.record, s) and cache.run(b.key(), b.record, s)
    assert not cache.run(a.key(), a.record, s) and len(cache) == 2
    small = gr.GraphCache(capacity=1)
    assert small.run(a.key(), a.record, s)
    assert small.run(b.key(), b.record, s)       # evicts a
    assert small.run(a.key(), a.record, s)       # captured again
    assert len(small) == 1 and small.captures == 3
    torch.cuda.synchronize()
    ref = _snapshot(a)
    with torch.cuda.stream(s):
        a.record(s)
    torch.cuda.synchronize()
    for k, v in a.outputs().items():
        assert torch.equal(v, ref[k]), k
