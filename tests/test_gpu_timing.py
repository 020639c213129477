"""The per-kernel timing hook (`specdec_time_kernel`) on a small bf16 model.

The hook re-runs the last pass's launches layer after layer.  It must refuse
kinds no pass has recorded, return a positive duration for every recorded
kind, and leave the committed context intact: a verify of the same drafts
after timing gives bit-identical logits (the re-run Q|K|V launches only
rewrite the cache entries that the verify writes again).
"""
import math

import numpy as np
import pytest

from paper_2608_10362_amd import binding, synth
from tests.gpu_util import i32, install_context, log, torch_cuda

pytestmark = pytest.mark.gpu


def test_time_kernel_cycles_layers_and_keeps_the_context():
    torch = torch_cuda()
    shape, n_layers, lengths, g = synth.LLAMA_1B, 3, [200, 75], 4
    B = len(lengths)
    capacity = 256
    W = synth.make_weights(shape, n_layers=n_layers)
    ctx = synth.make_kv_context(shape, n_layers, lengths)
    dw = binding.DeviceWeights(shape, W)
    target = binding.Model(dw, n_layers, max_rows=B * (g + 1), max_ctx=capacity)
    with pytest.raises(binding.SpecdecError):  # nothing recorded yet
        binding.specdec_time_kernel(target, "gate_up", reps=2)
    kv = binding.KVCache(target, B, capacity)
    install_context(kv, ctx, lengths, n_layers, shape.dtype)
    pend = synth.make_prompt(1, shape.vocab, batch=B, seed=41)[:, 0]
    state = (np.asarray(lengths, np.int32), np.stack([np.zeros(B, np.int32), pend], 1), np.ones(B, np.int32))
    kv.set_state(*state)
    drafts = i32(synth.make_prompt(g, shape.vocab, batch=B, seed=42))
    logits = torch.empty((B, g + 1, shape.vocab), dtype=torch.float32, device="cuda")
    binding.specdec_verify(target, kv, g, drafts, g, logits)
    before = logits.cpu().numpy().copy()

    times = {}
    for kind in ("embed", "qkv", "attention", "o_proj", "gate_up", "down", "lm_head"):
        us = binding.specdec_time_kernel(target, kind, reps=2 * n_layers + 1)
        assert math.isfinite(us) and us > 0.0, (kind, us)
        times[kind] = us
    with pytest.raises(binding.SpecdecError):  # bf16: RoPE and the KV append run in the Q|K|V epilogue
        binding.specdec_time_kernel(target, "rope_append", reps=1)
    log(f"time_kernel us: { {k: round(v, 2) for k, v in times.items()} }")

    kv.set_state(*state)
    binding.specdec_verify(target, kv, g, drafts, g, logits)
    after = logits.cpu().numpy()
    assert kv.read_state()["status"] == 0
    assert np.array_equal(before, after)


def test_stream_read_reads_and_writes_nothing():
    """The streaming-read ceiling probe over a buffer whose size is not a whole
    number of its chunks: it runs, and it never writes its sink for real data."""
    torch = torch_cuda()
    buf = torch.ones((64 << 20) + 123, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    binding.specdec_stream_read(buf, sink)
    binding.specdec_stream_read(buf, sink, nbytes=5000)
    torch.cuda.synchronize()
    assert int(sink.item()) == 0
