"""Draft reload into a resident slot (the draft cache of Sec. 3.3, Alg. 2, on
one GPU): a draft run from weights copied into a slot from pinned host memory
on a side stream must compute exactly what the same draft computes from the
resident target image (same bytes, same kernels: bitwise equal)."""
import numpy as np
import pytest

from paper_2608_10362_amd import binding, synth
from tests.gpu_util import install_context, log, torch_cuda

pytestmark = pytest.mark.gpu


def _draft_step(model, ctx, lengths, k, shape, pending_tok, T):
    torch = torch_cuda()
    kv = binding.KVCache(model, 1, 384)
    install_context(kv, ctx, lengths, k, shape.dtype)
    kv.set_state(np.asarray(lengths, np.int32), [[0, pending_tok]], [1])
    g = 4
    d = torch.zeros((1, g), dtype=torch.int32, device="cuda")
    q = torch.zeros((1, g, shape.vocab), dtype=torch.float32, device="cuda")
    lo = torch.empty((1, shape.vocab), dtype=torch.float32, device="cuda")
    for s in range(g):
        binding.specdec_draft_step(model, kv, g, s, T, 5, 1, None, q if T > 0 else None, d, g, lo if s == 0 else None)
    return lo, d, q


def test_draft_reload_into_slot_matches_resident_draft():
    torch = torch_cuda()
    shape = synth.LLAMA_1B
    W = synth.make_weights(shape, n_layers=3)
    dw = binding.DeviceWeights(shape, W)
    slot = binding.DraftSlot(dw, max_layers=2)
    copy = torch.cuda.Stream()
    lengths = [300]
    ctx = synth.make_kv_context(shape, 2, lengths)
    for k, T in ((2, 1.0), (1, 0.0), (2, 0.0)):
        log(f"reload {k}-layer draft into the slot (T={T})")
        sent = slot.load_async(k, copy)
        slot.event.wait()  # the current stream waits on the device; the host does not block
        resident = binding.Model(dw, k, max_rows=2, max_ctx=384)
        in_slot = binding.Model(dw, k, max_rows=2, max_ctx=384, packed=slot.slot)
        lo_r, d_r, q_r = _draft_step(resident, ctx, lengths, k, shape, 17, T)
        lo_s, d_s, q_s = _draft_step(in_slot, ctx, lengths, k, shape, 17, T)
        torch.cuda.synchronize()
        assert slot.event.query()
        off, nb = binding.packed_range(slot.shape, 0, k)
        assert sent == nb
        assert torch.equal(slot.slot[:off + nb], dw.packed[:off + nb])
        assert torch.equal(lo_r, lo_s) and torch.equal(d_r, d_s)
        if T > 0:
            assert torch.equal(q_r, q_s)
