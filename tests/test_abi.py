"""The C-ABI library loads, exports what include/specdec.h declares, and
validates arguments on the host (no GPU needed: nothing here launches)."""
import ctypes
import os
import re

import pytest

from paper_2608_10362_amd import binding, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.LIB_PATH):
        from paper_2608_10362_amd import build
        build.build()
    return binding.lib()


def _declared():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            txt = open(os.path.join(ROOT, "include", fn)).read()
            names |= set(re.findall(r"SPECDEC_API[^;(]*?\b(specdec_\w+)\s*\(", txt))
    return sorted(names)


def test_header_declares_the_four_hot_path_calls():
    names = _declared()
    for n in ("specdec_draft_step", "specdec_verify", "specdec_accept", "specdec_kv_commit"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert len(names) >= 21
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(binding._SIGS), "binding signatures out of sync with the header"


def test_status_strings(lib):
    for code, text in binding.STATUS.items():
        assert binding.specdec_status_string(code) == text


def test_sizes_and_shape_validation(lib):
    d = binding.make_desc(synth.LLAMA_7B)
    ws = lib.specdec_workspace_bytes(ctypes.byref(d), 5, 4096)
    assert ws > 0 and ws % 256 == 0
    assert lib.specdec_kv_bytes(ctypes.byref(d), 32, 1, 2048) == 32 * 32 * 2 * 2048 * 128 * 2
    assert lib.specdec_kv_state_count(16) == 68
    bad = binding.make_desc(synth.LLAMA_7B)
    bad.head_dim = 96
    assert lib.specdec_workspace_bytes(ctypes.byref(bad), 5, 4096) == 0
    bad = binding.make_desc(synth.LLAMA_7B)
    bad.n_kv_heads = 5
    assert lib.specdec_workspace_bytes(ctypes.byref(bad), 5, 4096) == 0


def test_model_create_argument_errors(lib):
    d = binding.make_desc(synth.TINY)
    h = ctypes.c_void_p()
    w = binding.Weights()
    fake = ctypes.c_void_p(256)  # never dereferenced: creation fails before any use
    # null weights struct
    assert lib.specdec_model_create(ctypes.byref(d), None, 1, None, 0, 8, 128, fake, 1 << 30, ctypes.byref(h)) == -1
    # null per-layer arrays
    assert lib.specdec_model_create(ctypes.byref(d), ctypes.byref(w), 1, None, 0, 8, 128, fake, 1 << 30,
                                    ctypes.byref(h)) == -1
    # too many layers
    assert lib.specdec_model_create(ctypes.byref(d), ctypes.byref(w), 3, None, 0, 8, 128, fake, 1 << 30,
                                    ctypes.byref(h)) == -1
    # unsupported shape
    bad = binding.make_desc(synth.TINY)
    bad.d_model = 100
    assert lib.specdec_model_create(ctypes.byref(bad), ctypes.byref(w), 1, None, 0, 8, 128, fake, 1 << 30,
                                    ctypes.byref(h)) == -2
    # workspace too small
    arr = (ctypes.c_void_p * 2)(256, 256)
    pp = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
    w2 = binding.Weights(256, 256, 256, *([pp] * 9))
    assert lib.specdec_model_create(ctypes.byref(d), ctypes.byref(w2), 1, None, 0, 8, 128, fake, 16,
                                    ctypes.byref(h)) == -1
    # a float32 model takes no packed image; a bf16 model needs one of the right size
    assert lib.specdec_model_create(ctypes.byref(d), ctypes.byref(w2), 1, fake, 1 << 30, 8, 128, fake, 1 << 30,
                                    ctypes.byref(h)) == -1
    d16 = binding.make_desc(synth.LLAMA_1B)
    need = lib.specdec_packed_bytes(ctypes.byref(d16), 2)
    assert need > 0 and lib.specdec_packed_bytes(ctypes.byref(d), 1) == 0
    assert lib.specdec_model_create(ctypes.byref(d16), ctypes.byref(w2), 2, fake, need - 1, 8, 128, fake, 1 << 40,
                                    ctypes.byref(h)) == -1
    assert lib.specdec_pack_weights(ctypes.byref(d), ctypes.byref(w2), 1, fake, 1 << 30, None) == -6
    assert not h.value


def test_call_argument_errors_before_any_launch(lib):
    kv = binding.KV()
    # null handles / buffers are rejected synchronously
    assert lib.specdec_verify(None, ctypes.byref(kv), 4, None, 4, None, None) == -1
    assert lib.specdec_draft_step(None, ctypes.byref(kv), 4, 0, 1.0, 0, 0, None, None, None, None, 4, None,
                                  None) == -1
    fake = ctypes.c_void_p(256)
    ws = lib.specdec_accept_workspace_bytes(1, 4, 100)
    assert ws > 0 and lib.specdec_accept_workspace_bytes(1, 40, 100) == 0
    assert lib.specdec_accept(0, 4, 100, 0, 1.0, None, None, None, 4, None, 0, 0, None, None, None, None, fake, ws,
                              None) == -1
    assert lib.specdec_accept(1, 4, 100, 7, 1.0, fake, fake, fake, 4, None, 0, 0, None, fake, fake, None, fake, ws,
                              None) == -1
    assert lib.specdec_accept(1, 40, 100, 0, 1.0, fake, fake, fake, 40, None, 0, 0, None, fake, fake, None, fake, ws,
                              None) == -6
    # the workspace is required and must be large enough
    assert lib.specdec_accept(1, 4, 100, 0, 1.0, fake, fake, fake, 4, None, 0, 0, None, fake, fake, None, None, ws,
                              None) == -1
    assert lib.specdec_accept(1, 4, 100, 0, 1.0, fake, fake, fake, 4, None, 0, 0, None, fake, fake, None, fake, ws - 1,
                              None) == -1
    # the no-allocation accept: the same argument errors, and a request beyond its
    # static scratch is refused before any HIP call
    assert lib.specdec_accept_noalloc(0, 4, 100, 0, 1.0, None, None, None, 4, None, 0, 0, None, None, None, None,
                                      None) == -1
    assert lib.specdec_accept_noalloc(1, 40, 100, 0, 1.0, fake, fake, fake, 40, None, 0, 0, None, fake, fake, None,
                                      None) == -6
    assert lib.specdec_accept_workspace_bytes(200, 8, 200000) > binding.ACCEPT_NOALLOC_SCRATCH_BYTES
    assert lib.specdec_accept_noalloc(200, 8, 200000, 0, 1.0, fake, fake, fake, 8, None, 0, 0, None, fake, fake, None,
                                      None) == -8
    # a step word must be 8-byte aligned
    odd = ctypes.c_void_p(260)
    assert lib.specdec_accept(1, 4, 100, 0, 1.0, fake, fake, fake, 4, None, 0, 0, odd, fake, fake, None, fake, ws,
                              None) == -1
    assert lib.specdec_accept_noalloc(1, 4, 100, 0, 1.0, fake, fake, fake, 4, None, 0, 0, odd, fake, fake, None,
                                      None) == -1
    # the commit counter sits after the status word and one unused word
    assert lib.specdec_kv_step_word(ctypes.byref(kv)) is None
    kv.state = 4096
    kv.batch = 3
    assert lib.specdec_kv_step_word(ctypes.byref(kv)) == 4096 + 4 * (4 * 3 + 2)
    assert lib.specdec_kv_step_word(None) is None
    kv = binding.KV()
    assert lib.specdec_stream_read(None, 1024, fake, None) == -1
    assert lib.specdec_stream_read(ctypes.c_void_p(257), 1024, fake, None) == -1  # (16-byte alignment)
    assert lib.specdec_kv_commit(ctypes.byref(kv), 4, 0, None, None, 4, None, None) == -1
    assert lib.specdec_sample(1, 10, None, 10, None, 0, 0, 0, 0, None, None) == -1
    assert lib.specdec_draw_u32(1, 0, 0, 0x10000, 0, ctypes.c_void_p(256), None) == -1


def test_packed_range_tiles_the_image(lib):
    shape = synth.LLAMA_1B.with_layers(3)
    d = binding.make_desc(shape)
    total = lib.specdec_packed_bytes(ctypes.byref(d), 3)
    head_off, _ = binding.packed_range(shape, 0, 1)
    prev_end = head_off
    for layer in range(3):
        off, nb = binding.packed_range(shape, layer, 1)
        assert off == prev_end and nb > 0
        prev_end = off + nb
    assert prev_end == total
    off, nb = binding.packed_range(shape, 0, 2)
    assert off == head_off and off + nb == lib.specdec_packed_bytes(ctypes.byref(d), 2)
    # the LM head region is its [V, d] bf16 image, 256-byte aligned
    assert head_off == -(-shape.vocab * shape.d_model * 2 // 256) * 256
    off_t, nb_t = ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.specdec_packed_range(ctypes.byref(d), 2, 2, ctypes.byref(off_t), ctypes.byref(nb_t)) == -1
    assert lib.specdec_packed_range(ctypes.byref(d), -1, 1, ctypes.byref(off_t), ctypes.byref(nb_t)) == -1
    assert lib.specdec_packed_range(ctypes.byref(d), 0, 1, None, ctypes.byref(nb_t)) == -1
    d32 = binding.make_desc(synth.TINY)
    assert lib.specdec_packed_range(ctypes.byref(d32), 0, 1, ctypes.byref(off_t), ctypes.byref(nb_t)) == -6


def test_reload_calls_reject_bad_arguments(lib):
    fake = ctypes.c_void_p(256)
    assert lib.specdec_event_create(None) == -1
    assert lib.specdec_event_destroy(None) == -1
    assert lib.specdec_load_async(None, fake, 16, None, fake) == -1
    assert lib.specdec_load_async(fake, fake, 0, None, fake) == -1
    assert lib.specdec_load_async(fake, fake, 16, None, None) == -1
    assert lib.specdec_stream_wait_event(None, None) == -1
    assert lib.specdec_event_query(None, None) == -1


def test_int4_image_sizes_and_format_errors(lib):
    fake = ctypes.c_void_p(256)
    h = ctypes.c_void_p()
    d16 = binding.make_desc(synth.LLAMA_7B)
    bf = lib.specdec_packed_bytes_fmt(ctypes.byref(d16), 2, 0)
    q4 = lib.specdec_packed_bytes_fmt(ctypes.byref(d16), 2, 1)
    assert bf == lib.specdec_packed_bytes(ctypes.byref(d16), 2)
    # two 7B layers (2 x 202.4M weights) at 4 bits + 1/64 scale overhead, plus the bf16 LM head
    head = 32000 * 4096 * 2
    layer_w = 4 * 4096 * 4096 + 3 * 4096 * 11008
    assert abs((q4 - head) - 2 * layer_w * (0.5 + 2 / 128)) < 1e5
    assert abs((bf - head) - 2 * layer_w * 2) < 1e5
    assert lib.specdec_packed_bytes_fmt(ctypes.byref(d16), 2, 7) == 0
    assert lib.specdec_packed_bytes_fmt(ctypes.byref(binding.make_desc(synth.TINY)), 1, 1) == 0
    arr = (ctypes.c_void_p * 2)(256, 256)
    pp = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
    w2 = binding.Weights(256, 256, 256, *([pp] * 9))
    # unknown format; INT4 handles run at most 64 rows per pass
    assert lib.specdec_pack_weights_fmt(ctypes.byref(d16), ctypes.byref(w2), 2, 5, fake, q4, None) == -1
    assert lib.specdec_model_create_fmt(ctypes.byref(d16), ctypes.byref(w2), 2, 5, fake, q4, 8, 128, fake, 1 << 40,
                                        ctypes.byref(h)) == -1
    assert lib.specdec_model_create_fmt(ctypes.byref(d16), ctypes.byref(w2), 2, 1, fake, q4, 65, 128, fake, 1 << 40,
                                        ctypes.byref(h)) == -6
    assert lib.specdec_model_create_fmt(ctypes.byref(d16), ctypes.byref(w2), 2, 1, fake, q4 - 1, 8, 128, fake,
                                        1 << 40, ctypes.byref(h)) == -1
    assert not h.value
